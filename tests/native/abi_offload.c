/* Offload through the C ABI from C, with no Python and no torch.
 *
 * A KV block manager with a host pool (cw_bm_create_with_host_pool) serves four
 * sessions (two of them sharing a 32-token prefix group) on a 12-block device
 * pool and a 6-block host pool over fifteen admissions, so blocks are evicted to
 * the host, dropped when it is full and swapped back when their session
 * resumes.  Each admission's swap lists run through cw_kv_swap_out and then
 * cw_kv_swap_in (pinned host pools), and each step through cw_step_attention,
 * whose new tokens are the sessions' own K/V.  Checks, per step:
 *  - the output and lse equal, bit for bit, the same step run on a second pool
 *    built on the host from the sessions' own K/V (so every page the step reads
 *    holds what the block table says it holds);
 *  - after the step, every position of every admitted request holds that
 *    session's K/V in the slot its table gives;
 * and over the run that there were swap-outs, swap-ins and drops.
 * Prints "ok" and exits 0 on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "cw.h"
#include "cw_policy.h"

#define FAIL(...)                                   \
  do {                                              \
    fprintf(stderr, "FAIL line %d: ", __LINE__);    \
    fprintf(stderr, __VA_ARGS__);                   \
    fprintf(stderr, "\n");                          \
    exit(1);                                        \
  } while (0)
#define CHECK_HIP(x)                                                          \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) FAIL("%s: %s", #x, hipGetErrorString(e_));          \
  } while (0)
#define CHECK_CW(x)                                                           \
  do {                                                                        \
    cw_status_t s_ = (x);                                                     \
    if (s_ != CW_OK) FAIL("%s: %s (%s)", #x, cw_status_string(s_),            \
                          cw_last_error_message());                           \
  } while (0)

enum {
  P = 16, HKV = 2, G = 4, HQ = HKV * G, D = 64,
  NDEV = 12, NHOST = 6, NSESS = 4, SHARED = 32,
  MAXB = 8, MAXCTX = MAXB * P, MAXROWS = 2
};
#define ROW (HKV * D)                    /* one token's K (or V) across kv heads */
#define PAGE_ELEMS ((size_t)HKV * P * D) /* one page of one pool */

static const int32_t kGroup[NSESS] = {-1, -1, 0, 0};
/* admissions: session, input tokens, eviction value at release; steps of one or two */
static const int kSteps[][MAXROWS][3] = {
    {{0, 40, 3}}, {{1, 50, 1}}, {{2, 45, 2}}, {{3, 40, 5}}, {{0, 30, 4}},
    {{1, 20, 2}, {0, 10, 9}}, {{2, 30, 1}}, {{3, 25, 2}}, {{1, 30, 3}}, {{0, 20, 1}},
    {{2, 20, 6}}, {{3, 30, 2}}, {{1, 25, 4}}, {{0, 15, 3}},
};
#define NSTEPS ((int)(sizeof(kSteps) / sizeof(kSteps[0])))

static uint64_t rng = 0x13198A2E03707344ull;
static uint16_t next_bf16(void) { /* a bf16 uniform in [-2, 2) */
  rng = rng * 6364136223846793005ull + 1442695040888963407ull;
  float f = (float)((rng >> 40) & 0xFFFFFF) / (float)(1 << 22) - 2.0f;
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
static void fill(uint16_t* dst, size_t n) {
  for (size_t i = 0; i < n; ++i) dst[i] = next_bf16();
}

/* the sessions' own K and V: [session][position][kv head][D]; the group's
 * members hold the same rows for the shared prefix */
static uint16_t lk[NSESS][MAXCTX][ROW], lv[NSESS][MAXCTX][ROW];

static size_t slot_at(int page, int h, int slot) { return (((size_t)page * HKV + h) * P + slot) * D; }

int main(void) {
  CHECK_CW(cw_init());
  fill(&lk[0][0][0], sizeof(lk) / 2);
  fill(&lv[0][0][0], sizeof(lv) / 2);
  for (int s = 0; s < NSESS; ++s)
    if (kGroup[s] >= 0 && s != 2) { /* session 2 leads group 0 */
      memcpy(lk[s], lk[2], (size_t)SHARED * ROW * 2);
      memcpy(lv[s], lv[2], (size_t)SHARED * ROW * 2);
    }

  cw_block_manager_t* bm = NULL;
  if (cw_bm_create_with_host_pool(NDEV, P, 0, &bm) != CW_ERR_UNSUPPORTED) FAIL("empty host pool accepted");
  CHECK_CW(cw_bm_create_with_host_pool(NDEV, P, NHOST, &bm));
  for (int s = 0; s < NSESS; ++s) CHECK_CW(cw_bm_add_session(bm, s, kGroup[s], kGroup[s] >= 0 ? SHARED : 0));

  const size_t pool_elems = (size_t)NDEV * PAGE_ELEMS, host_elems = (size_t)NHOST * PAGE_ELEMS;
  uint16_t* garbage = malloc(pool_elems * 2);
  uint16_t* ref_k = malloc(pool_elems * 2);
  uint16_t* ref_v = malloc(pool_elems * 2);
  uint16_t* got_k = malloc(pool_elems * 2);
  uint16_t* got_v = malloc(pool_elems * 2);
  fill(garbage, pool_elems);
  void *kp, *vp, *rkp, *rvp, *kh, *vh;
  CHECK_HIP(hipMalloc(&kp, pool_elems * 2));
  CHECK_HIP(hipMalloc(&vp, pool_elems * 2));
  CHECK_HIP(hipMalloc(&rkp, pool_elems * 2));
  CHECK_HIP(hipMalloc(&rvp, pool_elems * 2));
  CHECK_HIP(hipMemcpy(kp, garbage, pool_elems * 2, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(vp, garbage, pool_elems * 2, hipMemcpyHostToDevice));
  CHECK_HIP(hipHostMalloc(&kh, host_elems * 2, hipHostMallocDefault));
  CHECK_HIP(hipHostMalloc(&vh, host_elems * 2, hipHostMallocDefault));
  memset(kh, 0xFF, host_elems * 2);
  memset(vh, 0xFF, host_elems * 2);

  const int max_t = MAXROWS * MAXCTX;
  void *q, *kn, *vn, *dbt, *out_a, *out_b, *lse_a, *lse_b, *sws;
  CHECK_HIP(hipMalloc(&q, (size_t)max_t * HQ * D * 2));
  CHECK_HIP(hipMalloc(&kn, (size_t)max_t * ROW * 2));
  CHECK_HIP(hipMalloc(&vn, (size_t)max_t * ROW * 2));
  CHECK_HIP(hipMalloc(&dbt, sizeof(int32_t) * MAXROWS * MAXB));
  CHECK_HIP(hipMalloc(&out_a, (size_t)max_t * HQ * D * 2));
  CHECK_HIP(hipMalloc(&out_b, (size_t)max_t * HQ * D * 2));
  CHECK_HIP(hipMalloc(&lse_a, (size_t)max_t * HQ * 4));
  CHECK_HIP(hipMalloc(&lse_b, (size_t)max_t * HQ * 4));
  const size_t sws_bytes = cw_swap_workspace_bytes(MAXB);
  CHECK_HIP(hipMalloc(&sws, sws_bytes));
  uint16_t* hq = malloc((size_t)max_t * HQ * D * 2);
  uint16_t* hkn = malloc((size_t)max_t * ROW * 2);
  uint16_t* hvn = malloc((size_t)max_t * ROW * 2);
  uint16_t* oa = malloc((size_t)max_t * HQ * D * 2);
  uint16_t* ob = malloc((size_t)max_t * HQ * D * 2);
  float* la = malloc((size_t)max_t * HQ * 4);
  float* lb = malloc((size_t)max_t * HQ * 4);
  hipStream_t st;
  CHECK_HIP(hipStreamCreate(&st));
  const float scale = 1.0f / sqrtf((float)D);

  int64_t ctx[NSESS] = {0};
  long n_out = 0, n_in = 0, n_evicted = 0, n_cached = 0;
  for (int stp = 0; stp < NSTEPS; ++stp) {
    int rows = 0, sess[MAXROWS];
    int32_t table[MAXROWS][MAXB], blocks[MAXROWS], lp[MAXROWS], ls[MAXROWS], end[MAXROWS];
    for (int r = 0; r < MAXROWS && kSteps[stp][r][1] > 0; ++r, ++rows) {
      const int s = kSteps[stp][r][0], tin = kSteps[stp][r][1];
      int32_t od[MAXB], oh[MAXB], ih[MAXB], idv[MAXB];
      cw_bm_swaps_t sw = {od, oh, ih, idv, MAXB, 0, 0};
      int64_t cached, evicted;
      CHECK_CW(cw_bm_admit_swaps(bm, s, ctx[s], tin, 0, table[r], MAXB, &blocks[r], &cached, &evicted, &sw));
      if (sw.n_out > 0)
        CHECK_CW(cw_kv_swap_out(kp, vp, NULL, NULL, NDEV, kh, vh, NULL, NULL, NHOST, od, oh, sw.n_out, HKV, D,
                                P, CW_KV_BF16, sws, sws_bytes, st));
      if (sw.n_in > 0)
        CHECK_CW(cw_kv_swap_in(kh, vh, NULL, NULL, NHOST, kp, vp, NULL, NULL, NDEV, ih, idv, sw.n_in, HKV, D, P,
                               CW_KV_BF16, sws, sws_bytes, st));
      sess[r] = s;
      lp[r] = (int32_t)cached;
      end[r] = (int32_t)(ctx[s] + tin);
      ls[r] = end[r] - lp[r];
      if (blocks[r] != (end[r] + P - 1) / P) FAIL("step %d: %d blocks for %d tokens", stp, blocks[r], end[r]);
      n_out += sw.n_out;
      n_in += sw.n_in;
      n_evicted += evicted;
      n_cached += cached;
    }
    /* the step's inputs: q at random, the new tokens the sessions' own K/V */
    int T = 0;
    int32_t bt[MAXROWS * MAXB];
    for (int r = 0; r < rows; ++r) {
      for (int j = 0; j < MAXB; ++j) bt[r * MAXB + j] = j < blocks[r] ? table[r][j] : 0x7FFFFFFF;
      memcpy(hkn + (size_t)T * ROW, lk[sess[r]][lp[r]], (size_t)ls[r] * ROW * 2);
      memcpy(hvn + (size_t)T * ROW, lv[sess[r]][lp[r]], (size_t)ls[r] * ROW * 2);
      T += ls[r];
    }
    fill(hq, (size_t)T * HQ * D);
    CHECK_HIP(hipMemcpy(q, hq, (size_t)T * HQ * D * 2, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(kn, hkn, (size_t)T * ROW * 2, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(vn, hvn, (size_t)T * ROW * 2, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(dbt, bt, sizeof(int32_t) * rows * MAXB, hipMemcpyHostToDevice));
    /* the reference pool: garbage except the prefixes, written from the sessions' K/V */
    memcpy(ref_k, garbage, pool_elems * 2);
    memcpy(ref_v, garbage, pool_elems * 2);
    for (int r = 0; r < rows; ++r)
      for (int pos = 0; pos < lp[r]; ++pos)
        for (int h = 0; h < HKV; ++h) {
          const size_t at = slot_at(table[r][pos / P], h, pos % P);
          memcpy(ref_k + at, &lk[sess[r]][pos][h * D], D * 2);
          memcpy(ref_v + at, &lv[sess[r]][pos][h * D], D * 2);
        }
    CHECK_HIP(hipMemcpy(rkp, ref_k, pool_elems * 2, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(rvp, ref_v, pool_elems * 2, hipMemcpyHostToDevice));
    const size_t ws_bytes = cw_step_workspace_bytes(lp, ls, rows, HKV, G, D, P, CW_KV_BF16);
    if (ws_bytes == 0) FAIL("workspace query failed");
    void* ws = NULL;
    CHECK_HIP(hipMalloc(&ws, ws_bytes));
    CHECK_CW(cw_step_attention(q, kn, vn, kp, vp, NULL, NULL, dbt, MAXB, NDEV, lp, ls, rows, HKV, G, D, P, scale,
                               CW_KV_BF16, out_a, lse_a, ws, ws_bytes, st));
    CHECK_CW(cw_step_attention(q, kn, vn, rkp, rvp, NULL, NULL, dbt, MAXB, NDEV, lp, ls, rows, HKV, G, D, P,
                               scale, CW_KV_BF16, out_b, lse_b, ws, ws_bytes, st));
    CHECK_HIP(hipStreamSynchronize(st));
    CHECK_HIP(hipFree(ws));
    CHECK_HIP(hipMemcpy(oa, out_a, (size_t)T * HQ * D * 2, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(ob, out_b, (size_t)T * HQ * D * 2, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(la, lse_a, (size_t)T * HQ * 4, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(lb, lse_b, (size_t)T * HQ * 4, hipMemcpyDeviceToHost));
    if (memcmp(oa, ob, (size_t)T * HQ * D * 2) != 0) FAIL("step %d: output differs from the reference pool's", stp);
    if (memcmp(la, lb, (size_t)T * HQ * 4) != 0) FAIL("step %d: lse differs from the reference pool's", stp);
    for (int i = 0; i < T * HQ; ++i)
      if (!isfinite(la[i])) FAIL("step %d: lse %d not finite", stp, i);
    /* every position of every admitted request in its slot */
    CHECK_HIP(hipMemcpy(got_k, kp, pool_elems * 2, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(got_v, vp, pool_elems * 2, hipMemcpyDeviceToHost));
    for (int r = 0; r < rows; ++r)
      for (int pos = 0; pos < end[r]; ++pos)
        for (int h = 0; h < HKV; ++h) {
          const size_t at = slot_at(table[r][pos / P], h, pos % P);
          if (memcmp(got_k + at, &lk[sess[r]][pos][h * D], D * 2) != 0 ||
              memcmp(got_v + at, &lv[sess[r]][pos][h * D], D * 2) != 0)
            FAIL("step %d: session %d position %d not in its slot", stp, sess[r], pos);
        }
    for (int r = 0; r < rows; ++r) {
      ctx[sess[r]] = end[r];
      CHECK_CW(cw_bm_release(bm, sess[r], (double)kSteps[stp][r][2]));
    }
  }
  if (n_out == 0 || n_in == 0 || n_evicted <= n_out || n_cached == 0)
    FAIL("the run did not exercise offload: %ld out, %ld in, %ld evicted, %ld cached", n_out, n_in, n_evicted,
         n_cached);
  int64_t free_host, held_host;
  CHECK_CW(cw_bm_host_stats(bm, &free_host, &held_host));
  if (free_host + held_host != NHOST) FAIL("host pool accounting");
  CHECK_CW(cw_bm_destroy(bm));

  CHECK_HIP(hipStreamDestroy(st));
  void* bufs[] = {kp, vp, rkp, rvp, q, kn, vn, dbt, out_a, out_b, lse_a, lse_b, sws};
  for (size_t i = 0; i < sizeof(bufs) / sizeof(bufs[0]); ++i) CHECK_HIP(hipFree(bufs[i]));
  CHECK_HIP(hipHostFree(kh));
  CHECK_HIP(hipHostFree(vh));
  free(garbage), free(ref_k), free(ref_v), free(got_k), free(got_v);
  free(hq), free(hkn), free(hvn), free(oa), free(ob), free(la), free(lb);
  printf("ok: %d steps, %ld swap-outs, %ld swap-ins, %ld evictions, %ld cached tokens\n", NSTEPS, n_out, n_in,
         n_evicted, n_cached);
  return 0;
}
