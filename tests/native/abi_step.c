/* Native use of the C ABI from C, with no Python and no torch.
 *
 * A KV block manager hands out the block tables of a two-sequence serving step
 * (two sessions sharing a 32-token prefix group): session 0 extends its
 * 100-token context by 37 tokens, session 1 decodes one token after 60.  Pools
 * and new tokens are filled on the host with a fixed pseudo-random pattern and
 * copied to the device, and cw_step_attention runs the step.  Checks:
 *  - the step's rows equal, bit for bit, cw_extend_attention of the extending
 *    sequence alone and cw_decode_attention of the decoding one (rows and lse);
 *  - every output is finite;
 *  - the pools hold the new tokens' K/V in the slots the tables give, and every
 *    other slot is unchanged;
 *  - invalid calls return their status codes and leave a message.
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

enum { P = 16, HKV = 2, G = 4, HQ = HKV * G, D = 128, NPAGES = 64, MAXB = 16 };

static uint64_t rng = 0x243F6A8885A308D3ull;
static float next_value(void) { /* uniform in [-2, 2) */
  rng = rng * 6364136223846793005ull + 1442695040888963407ull;
  return (float)((rng >> 40) & 0xFFFFFF) / (float)(1 << 22) - 2.0f;
}
static uint16_t to_bf16(float f) { /* round to nearest even */
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
static void fill(uint16_t* dst, size_t n) {
  for (size_t i = 0; i < n; ++i) dst[i] = to_bf16(next_value());
}
static int finite_bf16(uint16_t b) { return (b & 0x7F80u) != 0x7F80u; }

static void* dev_copy(const void* host, size_t bytes) {
  void* d = NULL;
  CHECK_HIP(hipMalloc(&d, bytes));
  CHECK_HIP(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
  return d;
}

int main(void) {
  CHECK_CW(cw_init());

  /* ---- the block manager: two sessions sharing a 32-token prefix */
  cw_block_manager_t* bm = NULL;
  CHECK_CW(cw_bm_create(NPAGES, P, &bm));
  CHECK_CW(cw_bm_add_session(bm, 0, 0, 32));
  CHECK_CW(cw_bm_add_session(bm, 1, 0, 32));
  int32_t table[2][MAXB], blocks[2];
  int64_t cached[2], evicted;
  CHECK_CW(cw_bm_admit(bm, 0, 0, 100, 0, table[0], MAXB, &blocks[0], &cached[0], &evicted));
  CHECK_CW(cw_bm_release(bm, 0, 1.0));
  CHECK_CW(cw_bm_admit(bm, 1, 0, 60, 0, table[1], MAXB, &blocks[1], &cached[1], &evicted));
  if (cached[1] != 32) FAIL("session 1 found %lld cached tokens, expected the shared 32", (long long)cached[1]);
  CHECK_CW(cw_bm_release(bm, 1, 2.0));
  /* the step: both admitted together (their shared blocks are resident) */
  CHECK_CW(cw_bm_admit(bm, 0, 100, 37, 0, table[0], MAXB, &blocks[0], &cached[0], &evicted));
  CHECK_CW(cw_bm_admit(bm, 1, 60, 1, 0, table[1], MAXB, &blocks[1], &cached[1], &evicted));
  if (table[0][0] != table[1][0] || table[0][1] != table[1][1]) FAIL("shared prefix blocks differ");
  const int32_t lp[2] = {(int32_t)cached[0], (int32_t)cached[1]};
  const int32_t ls[2] = {100 + 37 - lp[0], 60 + 1 - lp[1]};
  if (lp[0] != 100 || ls[0] != 37 || lp[1] != 60 || ls[1] != 1)
    FAIL("unexpected lengths %d+%d, %d+%d", lp[0], ls[0], lp[1], ls[1]);
  const int stride = MAXB;
  int32_t bt[2 * MAXB];
  for (int b = 0; b < 2; ++b)
    for (int j = 0; j < MAXB; ++j) bt[b * MAXB + j] = j < blocks[b] ? table[b][j] : 0x7FFFFFFF;
  CHECK_CW(cw_bm_destroy(bm));

  /* ---- inputs */
  const int T = ls[0] + ls[1];
  const size_t n_q = (size_t)T * HQ * D, n_new = (size_t)T * HKV * D;
  const size_t n_pool = (size_t)NPAGES * HKV * P * D;
  uint16_t* hq = malloc(n_q * 2);
  uint16_t* hk = malloc(n_new * 2);
  uint16_t* hv = malloc(n_new * 2);
  uint16_t* hkp = malloc(n_pool * 2);
  uint16_t* hvp = malloc(n_pool * 2);
  fill(hq, n_q);
  fill(hk, n_new);
  fill(hv, n_new);
  fill(hkp, n_pool);
  fill(hvp, n_pool);
  void* q = dev_copy(hq, n_q * 2);
  void* kn = dev_copy(hk, n_new * 2);
  void* vn = dev_copy(hv, n_new * 2);
  void* kp = dev_copy(hkp, n_pool * 2);
  void* vp = dev_copy(hvp, n_pool * 2);
  void* dbt = dev_copy(bt, sizeof(bt));
  void *out_step, *out_ext, *out_dec, *lse_step, *lse_ext, *lse_dec;
  CHECK_HIP(hipMalloc(&out_step, n_q * 2));
  CHECK_HIP(hipMalloc(&out_ext, (size_t)ls[0] * HQ * D * 2));
  CHECK_HIP(hipMalloc(&out_dec, (size_t)HQ * D * 2));
  CHECK_HIP(hipMalloc(&lse_step, (size_t)T * HQ * 4));
  CHECK_HIP(hipMalloc(&lse_ext, (size_t)ls[0] * HQ * 4));
  CHECK_HIP(hipMalloc(&lse_dec, (size_t)HQ * 4));
  const float scale = 1.0f / sqrtf((float)D);
  size_t ws_bytes = cw_step_workspace_bytes(lp, ls, 2, HKV, G, D, P, CW_KV_BF16);
  const size_t ws_ext = cw_extend_workspace_bytes(lp, ls, 1, HKV, G, D, P);
  const size_t ws_dec = cw_decode_workspace_bytes(lp + 1, 1, HKV, G, D, P, CW_KV_BF16);
  if (ws_ext > ws_bytes) ws_bytes = ws_ext;
  if (ws_dec > ws_bytes) ws_bytes = ws_dec;
  if (ws_bytes == 0) FAIL("workspace query failed");
  void* ws = NULL;
  CHECK_HIP(hipMalloc(&ws, ws_bytes));
  hipStream_t st;
  CHECK_HIP(hipStreamCreate(&st));

  /* ---- the step, then each sequence through its own entry point */
  CHECK_CW(cw_step_attention(q, kn, vn, kp, vp, NULL, NULL, dbt, stride, NPAGES, lp, ls, 2, HKV, G, D, P,
                             scale, CW_KV_BF16, out_step, lse_step, ws, ws_bytes, st));
  CHECK_HIP(hipStreamSynchronize(st));
  CHECK_CW(cw_extend_attention(q, kn, vn, kp, vp, NULL, NULL, dbt, stride, NPAGES, lp, ls, 1, HKV, G, D, P,
                               scale, CW_KV_BF16, out_ext, lse_ext, ws, ws_bytes, st));
  CHECK_HIP(hipStreamSynchronize(st));
  const size_t row = (size_t)ls[0];
  CHECK_CW(cw_decode_attention((const uint16_t*)q + row * HQ * D, (const uint16_t*)kn + row * HKV * D,
                               (const uint16_t*)vn + row * HKV * D, kp, vp, NULL, NULL,
                               (const int32_t*)dbt + stride, stride, NPAGES, lp + 1, 1, HKV, G, D, P, scale,
                               CW_KV_BF16, out_dec, lse_dec, ws, ws_bytes, st));
  CHECK_HIP(hipStreamSynchronize(st));

  uint16_t* o_step = malloc(n_q * 2);
  uint16_t* o_ext = malloc(row * HQ * D * 2);
  uint16_t* o_dec = malloc((size_t)HQ * D * 2);
  float* l_step = malloc((size_t)T * HQ * 4);
  float* l_ext = malloc(row * HQ * 4);
  float* l_dec = malloc((size_t)HQ * 4);
  CHECK_HIP(hipMemcpy(o_step, out_step, n_q * 2, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(o_ext, out_ext, row * HQ * D * 2, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(o_dec, out_dec, (size_t)HQ * D * 2, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(l_step, lse_step, (size_t)T * HQ * 4, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(l_ext, lse_ext, row * HQ * 4, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(l_dec, lse_dec, (size_t)HQ * 4, hipMemcpyDeviceToHost));
  for (size_t i = 0; i < n_q; ++i)
    if (!finite_bf16(o_step[i])) FAIL("step output %zu not finite", i);
  if (memcmp(o_step, o_ext, row * HQ * D * 2) != 0) FAIL("extend rows differ from the step's");
  if (memcmp(o_step + row * HQ * D, o_dec, (size_t)HQ * D * 2) != 0) FAIL("decode row differs from the step's");
  if (memcmp(l_step, l_ext, row * HQ * 4) != 0 || memcmp(l_step + row * HQ, l_dec, (size_t)HQ * 4) != 0)
    FAIL("lse differs");
  for (int i = 0; i < T * HQ; ++i)
    if (!isfinite(l_step[i])) FAIL("lse %d not finite", i);

  /* ---- the pools: new tokens in their slots, nothing else changed */
  uint16_t* gk = malloc(n_pool * 2);
  CHECK_HIP(hipMemcpy(gk, kp, n_pool * 2, hipMemcpyDeviceToHost));
  size_t written = 0;
  for (int b = 0, r0 = 0; b < 2; r0 += ls[b], ++b)
    for (int i = 0; i < ls[b]; ++i) {
      const int pos = lp[b] + i, page = bt[b * MAXB + pos / P], slot = pos % P;
      for (int h = 0; h < HKV; ++h) {
        const size_t at = (((size_t)page * HKV + h) * P + slot) * D;
        const size_t from = ((size_t)(r0 + i) * HKV + h) * D;
        if (memcmp(gk + at, hk + from, D * 2) != 0) FAIL("new key of sequence %d token %d not in its slot", b, i);
        memcpy(hkp + at, hk + from, D * 2); /* expected pool */
        written += D;
      }
    }
  if (memcmp(gk, hkp, n_pool * 2) != 0) FAIL("a pool slot outside the new tokens changed");
  if (written != n_new) FAIL("slot count");

  /* ---- invalid calls: status codes, nothing enqueued */
  if (cw_step_attention(NULL, kn, vn, kp, vp, NULL, NULL, dbt, stride, NPAGES, lp, ls, 2, HKV, G, D, P, scale,
                        CW_KV_BF16, out_step, lse_step, ws, ws_bytes, st) != CW_ERR_NULL)
    FAIL("NULL q accepted");
  if (cw_last_error_message()[0] == '\0') FAIL("no error message");
  if (cw_step_attention(q, kn, vn, kp, vp, NULL, NULL, dbt, stride, NPAGES, lp, ls, 2, HKV, G, 96, P, scale,
                        CW_KV_BF16, out_step, lse_step, ws, ws_bytes, st) != CW_ERR_UNSUPPORTED)
    FAIL("head_dim 96 accepted");
  const int32_t bad_ls[2] = {37, -1};
  if (cw_step_attention(q, kn, vn, kp, vp, NULL, NULL, dbt, stride, NPAGES, lp, bad_ls, 2, HKV, G, D, P, scale,
                        CW_KV_BF16, out_step, lse_step, ws, ws_bytes, st) != CW_ERR_BAD_LENS)
    FAIL("negative length accepted");
  if (cw_step_attention(q, kn, vn, kp, vp, NULL, NULL, dbt, stride, NPAGES, lp, ls, 2, HKV, G, D, P, scale,
                        CW_KV_BF16, out_step, lse_step, ws, 16, st) != CW_ERR_WORKSPACE)
    FAIL("small workspace accepted");
  CHECK_HIP(hipStreamSynchronize(st));

  CHECK_HIP(hipStreamDestroy(st));
  void* bufs[] = {q, kn, vn, kp, vp, dbt, out_step, out_ext, out_dec, lse_step, lse_ext, lse_dec, ws};
  for (size_t i = 0; i < sizeof(bufs) / sizeof(bufs[0]); ++i) CHECK_HIP(hipFree(bufs[i]));
  free(hq), free(hk), free(hv), free(hkp), free(hvp), free(o_step), free(o_ext), free(o_dec);
  free(l_step), free(l_ext), free(l_dec), free(gk);
  printf("ok: step of %d tokens (extend %d after %d, decode after %d), shared prefix pages %d %d\n", T, ls[0],
         lp[0], lp[1], bt[0], bt[1]);
  return 0;
}
