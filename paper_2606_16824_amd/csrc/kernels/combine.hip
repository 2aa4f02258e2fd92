// Split-K merge of extend / decode partials.
#include <hip/hip_runtime.h>

#include "../cw_internal.h"
#include "../plan_expand.h"

namespace cw {
namespace {

constexpr float kLn2 = 0.69314718055994531f;
constexpr int kFewParts = 4;  // the one-slice merge loads up to this many partials at once

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// PER consecutive bf16 elements of a partial's O row, as fp32.
template <int PER>
__device__ __forceinline__ void load_part(const uint16_t* base, size_t elem, float (&v)[PER]) {
  static_assert(PER == 2 || PER == 4, "two or four elements per lane");
  if constexpr (PER == 4) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(base + elem);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
    const uint32_t w = *reinterpret_cast<const uint32_t*>(base + elem);
    v[0] = __uint_as_float(w << 16);
    v[1] = __uint_as_float(w & 0xFFFF0000u);
  }
}

// Merges the split-K partials of query rows: weights 2^(m_c - max m),
// O = sum w_c O_c / sum w_c l_c.  A workgroup of 256 lanes covers ROWS rows;
// each row's SLICES slices of 32 lanes fold every SLICES-th partial with an
// online merge, then the slices are merged through LDS (SLICES = 1 for a few
// partials per row, 8 for many).  Fixed order, no atomics.
template <int D, int SLICES, bool AP>
__global__ __launch_bounds__(256) void combine_kernel(ExtendParams p, PlanArg<AP> ap) {
  constexpr int ROWS = 8 / SLICES;
  constexpr int PER = D / 32;  // dims per lane
  __shared__ float sh_o[ROWS][SLICES][D];
  __shared__ float sh_m[ROWS][SLICES], sh_l[ROWS][SLICES];
  const int wg_per_group = (p.part_rows + ROWS - 1) / ROWS;
  const int grp = blockIdx.x / wg_per_group;
  const int rsub = threadIdx.x / (32 * SLICES);
  const int lr = (blockIdx.x % wg_per_group) * ROWS + rsub;
  const CombineGroup cg = [&]() {
    if constexpr (AP) {
      if (p.ap_desc > 0) {  // a decode plan in compact form: the group is rebuilt (each wave searches)
        const ExpandDesc& d = *reinterpret_cast<const ExpandDesc*>(ap.bytes + p.ap_desc);
        const DecodeRec* rec = reinterpret_cast<const DecodeRec*>(ap.bytes + d.rec_off);
        const int b = wave_last_at_most(d.n_seqs, grp, static_cast<int>(threadIdx.x % 64),
                                        [&](int k) { return rec[k].group_off; });
        return expand_group_at(rec, grp, b, d.rows);
      }
    }
    return plan_ptr<AP>(ap, p.ap_groups, p.groups)[grp];
  }();
  const bool active = lr < cg.rows;
  const int slice = (threadIdx.x / 32) % SLICES, d0 = (threadIdx.x % 32) * PER;

  float m = -INFINITY, L = 0.f, acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  if (SLICES == 1 && active && cg.n_parts <= kFewParts) {
    // few partials (at most kFewParts): every load is issued before the first
    // use, so a row waits for one memory latency instead of one per partial
    float mc[kFewParts], lc[kFewParts], oc[kFewParts][PER];
#pragma unroll
    for (int c = 0; c < kFewParts; ++c) {
      mc[c] = -INFINITY;
      lc[c] = 0.f;
#pragma unroll
      for (int e = 0; e < PER; ++e) oc[c][e] = 0.f;
      if (c < cg.n_parts) {
        const size_t pr = size_t(cg.part0 + c) * p.part_rows + lr;
        const float2 ml = *reinterpret_cast<const float2*>(p.part_ml + pr * 2);
        mc[c] = ml.x;
        lc[c] = ml.y;
        load_part<PER>(p.part_o, pr * D + d0, oc[c]);
      }
    }
#pragma unroll
    for (int c = 0; c < kFewParts; ++c) m = fmaxf(m, mc[c]);
#pragma unroll
    for (int c = 0; c < kFewParts; ++c) {
      const float w = c < cg.n_parts ? exp2f(mc[c] - m) : 0.f;
      L += w * lc[c];
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] += w * oc[c][e];
    }
  } else {
    // many partials: each slice takes its partials kFewParts at a time, all of
    // a group's loads issued before the group is merged into the running state
    for (int c0 = slice; active && c0 < cg.n_parts; c0 += kFewParts * SLICES) {
      float mc[kFewParts], lc[kFewParts], oc[kFewParts][PER];
#pragma unroll
      for (int k = 0; k < kFewParts; ++k) {
        const int c = c0 + k * SLICES;
        mc[k] = -INFINITY;
        lc[k] = 0.f;
#pragma unroll
        for (int e = 0; e < PER; ++e) oc[k][e] = 0.f;
        if (c < cg.n_parts) {
          const size_t pr = size_t(cg.part0 + c) * p.part_rows + lr;
          const float2 ml = *reinterpret_cast<const float2*>(p.part_ml + pr * 2);
          mc[k] = ml.x;
          lc[k] = ml.y;
          load_part<PER>(p.part_o, pr * D + d0, oc[k]);
        }
      }
      float m_new = m;
#pragma unroll
      for (int k = 0; k < kFewParts; ++k) m_new = fmaxf(m_new, mc[k]);
      const float a = exp2f(m - m_new);
      L *= a;
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] *= a;
#pragma unroll
      for (int k = 0; k < kFewParts; ++k) {
        const float w = c0 + k * SLICES < cg.n_parts ? exp2f(mc[k] - m_new) : 0.f;
        L += w * lc[k];
#pragma unroll
        for (int e = 0; e < PER; ++e) acc[e] += w * oc[k][e];
      }
      m = m_new;
    }
  }
  if (SLICES > 1) {
#pragma unroll
    for (int e = 0; e < PER; ++e) sh_o[rsub][slice][d0 + e] = acc[e];
    if (threadIdx.x % 32 == 0) {
      sh_m[rsub][slice] = m;
      sh_l[rsub][slice] = L;
    }
    __syncthreads();
  }
  if (slice != 0 || !active) return;
  float mstar = -INFINITY;
  if (SLICES == 1) {
    mstar = m;
  } else {
#pragma unroll
    for (int s = 0; s < SLICES; ++s) mstar = fmaxf(mstar, sh_m[rsub][s]);
  }
  float Lt = 0.f, out[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) out[e] = 0.f;
  if (SLICES == 1) {
    Lt = L;
#pragma unroll
    for (int e = 0; e < PER; ++e) out[e] = acc[e];
  } else {
#pragma unroll
    for (int s = 0; s < SLICES; ++s) {
      const float w = sh_m[rsub][s] == -INFINITY ? 0.f : exp2f(sh_m[rsub][s] - mstar);
      Lt += w * sh_l[rsub][s];
#pragma unroll
      for (int e = 0; e < PER; ++e) out[e] += w * sh_o[rsub][s][d0 + e];
    }
  }
  const SeqInfo sq = plan_ptr<AP>(ap, p.ap_seqs, p.seqs)[cg.seq];
  const int G = p.gqa_group, hq = p.num_kv_heads * G;
  const int r = cg.q_row0 + lr;
  const int t = r / G, g = r - t * G;
  const float inv = 1.f / Lt;
  uint16_t* orow = static_cast<uint16_t*>(p.out) + (size_t(sq.cu + t) * hq + size_t(cg.kvh) * G + g) * D + d0;
#pragma unroll
  for (int e = 0; e < PER; ++e) orow[e] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(out[e] * inv));
  if (p.lse != nullptr && threadIdx.x % 32 == 0)
    p.lse[size_t(sq.cu + t) * hq + size_t(cg.kvh) * G + g] = (mstar + log2f(Lt)) * kLn2;
}

}  // namespace

hipError_t launch_combine(const ExtendParams& p, int head_dim, int max_parts, hipStream_t stream,
                          const ArgPlan* ap) {
  if (p.n_groups <= 0) return hipSuccess;
  const bool many = max_parts > 4;
  const int rows_per_wg = many ? 1 : 8;
  const dim3 grid(p.n_groups * ((p.part_rows + rows_per_wg - 1) / rows_per_wg));
#define CW_COMBINE(D_, S_)                                                                           \
  do {                                                                                               \
    if (ap) hipLaunchKernelGGL((combine_kernel<D_, S_, true>), grid, dim3(256), 0, stream, p, *ap); \
    else hipLaunchKernelGGL((combine_kernel<D_, S_, false>), grid, dim3(256), 0, stream, p, NoArgPlan{}); \
  } while (0)
  if (head_dim == 64) {
    if (many) CW_COMBINE(64, 8);
    else CW_COMBINE(64, 1);
  } else if (head_dim == 128) {
    if (many) CW_COMBINE(128, 8);
    else CW_COMBINE(128, 1);
  } else {
    return hipErrorInvalidValue;
  }
#undef CW_COMBINE
  return hipGetLastError();
}

}  // namespace cw
