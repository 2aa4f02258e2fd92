// Prefix-cached paged extend attention, bf16 MFMA on gfx950.
//
// One workgroup = four wave64s = BLOCK_M (128) packed query rows of one
// (sequence, kv head); packed row r is token r / G, query head kvh * G + r % G,
// so one staged key/value tile serves the whole GQA group.  Keys are walked
// BLOCK_N (64) at a time over [kv_begin, kv_end); key j < Lp comes from the page
// pool through the block table, key j >= Lp from k_new / v_new.
//
// Per tile, each wave computes S^T = K Q^T (keys x its 32 rows) with
// v_mfma_f32_32x32x16_bf16, so that a lane owns one query row: the row max is a
// max over the lane's 32 values plus one exchange with the other half-wave, and
// the softmax statistics and the O rescale stay in the lane.  Then
// O^T += V^T P^T with P rounded to bf16; V is stored transposed in LDS so that
// the contraction (key) dimension is contiguous for the MFMA operand.
//
// MFMA 32x32x16 operand layouts (wave64, lane l, half h = l / 32):
//   A[m][k]: lane m + 32 * (k / 8), element k % 8
//   B[k][n]: lane n + 32 * (k / 8), element k % 8
//   C[m][n]: lane n + 32 * ((m / 4) % 2), element (m % 4) + 4 * (m / 8)
// Row m of the S^T output held in element i of half h is m = 8(i/4) + 4h + i%4.
// Reading A row m from key swap_bits_2_3(m) makes element i of half h hold key
// 16(i/8) + 8h + i%8 (within a 32-key block), which is exactly the B-operand
// order the P^T V product needs: P values feed the second MFMA without any
// data movement across lanes.  K rows are stored in LDS at row swap(j) so the
// A-operand reads stay linear.
//
// Softmax runs in base 2 with scale * log2(e) folded into one FMA; the running
// max starts at a large negative finite value so that fully masked rows give
// exp2(-inf) = 0 instead of NaN.  Masked keys are excluded by setting their
// score to -inf; K/V rows past the sequence are staged as zeros, so stale or
// NaN pool slots are never multiplied in.
//
// fp8-e4m3fn pools: codes are widened exactly to bf16 while staging (every
// e4m3fn value is a bf16 value); the page's K scale multiplies the scores of
// its keys and the V scale multiplies P before the bf16 rounding.
#include <hip/hip_runtime.h>

#include "../cw_internal.h"

namespace cw {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr float kNegBig = -1.0e30f;
constexpr float kLn2 = 0.69314718055994531f;

__device__ __forceinline__ int swap_bits_2_3(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Two e4m3fn codes (bytes 0,1 or 2,3 of `w`) -> two bf16 in one dword, exact.
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  f32x2 f = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w), HI);
  const uint32_t a = __float_as_uint(f.x), b = __float_as_uint(f.y);
  return (a >> 16) | (b & 0xFFFF0000u);  // the low 16 bits of an e4m3fn value are zero
}

__device__ __forceinline__ u32x4 fp8x8_to_bf16x8(u32x2 c) {
  u32x4 r;
  r.x = fp8x2_to_bf16x2<false>(c.x);
  r.y = fp8x2_to_bf16x2<true>(c.x);
  r.z = fp8x2_to_bf16x2<false>(c.y);
  r.w = fp8x2_to_bf16x2<true>(c.y);
  return r;
}

template <int D, int P, bool FP8>
struct Geo {
  static constexpr int KROW = D + 8;        // K tile row stride (elements): 16 B pad
  static constexpr int VROW = BLOCK_N + 8;  // V^T tile row stride (elements)
  static constexpr int CPR = D / 8;         // 16-byte chunks per K/V row
  static constexpr int KCH = BLOCK_N * CPR / THREADS;  // K chunks per thread
  static constexpr int RSTEP = THREADS / CPR;          // rows between a thread's K chunks
  static constexpr int VUNITS = 16 * CPR;              // (4 keys x 8 dims) V units per tile
  static constexpr int NPG = BLOCK_N / P;              // pages per tile
  static constexpr int KT = D / 16;                    // k-steps of K Q^T
  static constexpr int DB = D / 32;                    // 32-row blocks of O^T
};

template <int N>
struct Pages {
  int id[N];
};
template <int N>
struct Scales {
  float k[N], v[N];
};

// Tile modes (uniform across the workgroup): every key in the cached prefix,
// every key in the new suffix, or anything else (prefix/suffix boundary or the
// end of the sequence inside the tile).
enum : int { MODE_PREFIX = 0, MODE_SUFFIX = 1, MODE_MIXED = 2 };

template <int D, int P, bool FP8>
__global__ __launch_bounds__(THREADS) void extend_kernel(ExtendParams p) {
  using T = Geo<D, P, FP8>;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[BLOCK_N * T::KROW];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[D * T::VROW];

  const WorkItem it = p.items[blockIdx.x];
  if (it.seq < 0) return;  // idle padding item (uniform across the workgroup)
  const SeqInfo sq = p.seqs[it.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int G = p.gqa_group, hkv = p.num_kv_heads, hq = hkv * G;
  const int kvh = it.kvh;
  const int lp = sq.lp, total_len = sq.lp + sq.ls;
  const int32_t* bt = p.block_table + size_t(it.seq) * p.bt_stride;
  const uint16_t* k_new = static_cast<const uint16_t*>(p.k_new);
  const uint16_t* v_new = static_cast<const uint16_t*>(p.v_new);

  // this lane's query row and its causal limit (number of visible keys)
  const int r_local = wave * 32 + col;
  const bool row_ok = r_local < it.rows;
  const int r = it.q_row0 + r_local;
  const int t = r / G, g = r - t * G;
  const int lim = row_ok ? lp + t + 1 : 0x7FFFFFFF;
  const bool wave_active = wave * 32 < it.rows;
  const int wave_min_lim = lp + (it.q_row0 + wave * 32) / G + 1;
  const int wave_last_row = it.q_row0 + min(wave * 32 + 31, it.rows - 1);
  const int wave_max_lim = lp + wave_last_row / G + 1;

  // Q^T as the B operand: k-step kk holds dims 16 kk + 8 h + [0, 8) of this row
  bf16x8 qf[T::KT];
  {
    const uint16_t* qrow =
        static_cast<const uint16_t*>(p.q) + (size_t(sq.cu + t) * hq + size_t(kvh) * G + g) * D;
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row_ok) v = *reinterpret_cast<const u32x4*>(qrow + 16 * kk + 8 * h);
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  f32x16 o[T::DB];
#pragma unroll
  for (int b = 0; b < T::DB; ++b) o[b] = f32x16{};
  float m_run = kNegBig, l_run = 0.f;
  const float c = p.scale_log2;

  // staging geometry: K chunk i = row kr0 + RSTEP i, dims 8 kc .. +7 (eight
  // consecutive lanes fill one 128-byte stretch of a K row in LDS);
  // V unit = keys 4 vkg .. +3, dims 8 vdg .. +7 (threads below VUNITS).  The 16
  // lanes of a V store group have 16 different key groups: V^T rows 8 apart are
  // 288 dwords apart (a multiple of the 32 banks), so distinct key columns are
  // what keeps the 8-byte transposed stores conflict-free.
  const int kr0 = tid / T::CPR, kc = tid % T::CPR;
  const int vkg = tid & 15, vdg = tid >> 4;
  const bool v_unit = tid < T::VUNITS;

  auto mode_of = [&](int j0) {
    if (j0 + BLOCK_N <= lp) return int(MODE_PREFIX);
    if (j0 >= lp && j0 + BLOCK_N <= total_len) return int(MODE_SUFFIX);
    return int(MODE_MIXED);
  };
  // physical pages of the prefix part of the tile at j0 (same address in every lane)
  auto load_pages = [&](int j0) {
    Pages<T::NPG> pg;
#pragma unroll
    for (int q = 0; q < T::NPG; ++q) pg.id[q] = (j0 + q * P < lp) ? bt[j0 / P + q] : 0;
    return pg;
  };
  auto load_scales = [&](int j0, Pages<T::NPG> pg) {
    Scales<T::NPG> sc;
#pragma unroll
    for (int q = 0; q < T::NPG; ++q) {
      sc.k[q] = 1.f;
      sc.v[q] = 1.f;
      if (j0 + q * P < lp) {
        const size_t si = size_t(pg.id[q]) * hkv + kvh;
        sc.k[q] = p.k_scale[si];
        sc.v[q] = p.v_scale[si];
      }
    }
    return sc;
  };
  // element offset of tile row `row` (j0 page aligned) in the pool
  auto pool_off = [&](Pages<T::NPG> pg, int row) -> size_t {
    int pgid = pg.id[0];
#pragma unroll
    for (int q = 1; q < T::NPG; ++q) pgid = (row / P == q) ? pg.id[q] : pgid;
    return ((size_t(pgid) * hkv + kvh) * P + (row % P)) * D;
  };
  // element offset of key j >= lp in k_new / v_new
  auto fresh_off = [&](int j) -> size_t { return (size_t(sq.cu + j - lp) * hkv + kvh) * D; };
  auto load_pool = [&](const void* pool, size_t off) -> u32x4 {
    u32x4 v = {0u, 0u, 0u, 0u};
    if constexpr (FP8) {
      const u32x2 w = *reinterpret_cast<const u32x2*>(static_cast<const uint8_t*>(pool) + off);
      v.x = w.x;
      v.y = w.y;
    } else {
      v = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(pool) + off);
    }
    return v;
  };
  // One 8-element piece of tile row `row`: pool (prefix), k_new/v_new (suffix)
  // or zero past the sequence.  Branches depend only on the tile mode (uniform);
  // a mixed tile loads both candidates from valid addresses and selects.
  auto load_piece = [&](int mode, int j0, int row, int d0, Pages<T::NPG> pg, const void* pool,
                        const uint16_t* fresh) -> u32x4 {
    const int j = j0 + row;
    if (mode == MODE_PREFIX) return load_pool(pool, pool_off(pg, row) + d0);
    if (mode == MODE_SUFFIX) return *reinterpret_cast<const u32x4*>(fresh + fresh_off(j) + d0);
    const bool pre = j < lp, fr = !pre && j < total_len;
    u32x4 a = {0u, 0u, 0u, 0u};
    if (j0 < lp) a = load_pool(pool, pool_off(pg, pre ? row : 0) + d0);
    const u32x4 b = *reinterpret_cast<const u32x4*>(fresh + fresh_off(fr ? j : lp) + d0);
    const u32x4 z = {0u, 0u, 0u, 0u};
    return pre ? a : (fr ? b : z);
  };

  // raw tile registers: bf16 rows, or fp8 prefix rows in .xy (widened when stored)
  u32x4 kraw[T::KCH], vraw[4];
  auto load_data = [&](int j0, Pages<T::NPG> pg) {
    const int mode = mode_of(j0);
#pragma unroll
    for (int i = 0; i < T::KCH; ++i)
      kraw[i] = load_piece(mode, j0, kr0 + T::RSTEP * i, kc * 8, pg, p.k_pool, k_new);
    if (v_unit) {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        vraw[k] = load_piece(mode, j0, 4 * vkg + k, vdg * 8, pg, p.v_pool, v_new);
    }
  };
  auto widen = [&](int mode, int j, u32x4 v) -> u32x4 {
    if constexpr (FP8) {
      const u32x4 w = fp8x8_to_bf16x8(u32x2{v.x, v.y});
      if (mode == MODE_PREFIX) return w;
      if (mode == MODE_MIXED) return j < lp ? w : v;
    }
    return v;
  };
  auto store_tile = [&](int j0) {
    const int mode = mode_of(j0);
#pragma unroll
    for (int i = 0; i < T::KCH; ++i) {
      const int row = kr0 + T::RSTEP * i;
      *reinterpret_cast<u32x4*>(k_lds + swap_bits_2_3(row) * T::KROW + kc * 8) =
          widen(mode, j0 + row, kraw[i]);
    }
    if (v_unit) {
      u32x4 x[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) x[k] = widen(mode, j0 + 4 * vkg + k, vraw[k]);
      // transpose 4 keys x 8 dims: dword w of row k holds dims 2w (low) and 2w+1 (high)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t a0 = x[0][w], a1 = x[1][w], a2 = x[2][w], a3 = x[3][w];
        u32x2 lo, hi;
        lo.x = (a0 & 0xFFFFu) | (a1 << 16);
        lo.y = (a2 & 0xFFFFu) | (a3 << 16);
        hi.x = (a0 >> 16) | (a1 & 0xFFFF0000u);
        hi.y = (a2 >> 16) | (a3 & 0xFFFF0000u);
        *reinterpret_cast<u32x2*>(v_lds + (vdg * 8 + 2 * w) * T::VROW + 4 * vkg) = lo;
        *reinterpret_cast<u32x2*>(v_lds + (vdg * 8 + 2 * w + 1) * T::VROW + 4 * vkg) = hi;
      }
    }
  };

  // three-stage pipeline: page ids two tiles ahead, scales and data one ahead
  Pages<T::NPG> pg_next{};
  Scales<T::NPG> sc_cur, sc_next;
#pragma unroll
  for (int q = 0; q < T::NPG; ++q) sc_cur.k[q] = sc_cur.v[q] = sc_next.k[q] = sc_next.v[q] = 1.f;
  if (it.kv_begin < it.kv_end) {
    const Pages<T::NPG> pg0 = load_pages(it.kv_begin);
    load_data(it.kv_begin, pg0);
    if constexpr (FP8) sc_next = load_scales(it.kv_begin, pg0);
    if (it.kv_begin + BLOCK_N < it.kv_end) pg_next = load_pages(it.kv_begin + BLOCK_N);
  }

  for (int j0 = it.kv_begin; j0 < it.kv_end; j0 += BLOCK_N) {
    const int mode = mode_of(j0);
    __syncthreads();  // every wave is done reading the previous tile
    store_tile(j0);
    sc_cur = sc_next;
    __syncthreads();
    const int jn = j0 + BLOCK_N;
    if (jn < it.kv_end) {  // next tile's data and scales, the one after's page ids
      const Pages<T::NPG> pg1 = pg_next;
      load_data(jn, pg1);
      if constexpr (FP8) sc_next = load_scales(jn, pg1);
      if (jn + BLOCK_N < it.kv_end) pg_next = load_pages(jn + BLOCK_N);
    }

    if (!wave_active || j0 >= wave_max_lim) continue;  // nothing visible for this wave

    // S^T = K Q^T for two 32-key blocks; the two accumulators alternate so that
    // consecutive MFMAs are independent
    f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      bf16x8 kf[2];
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
        kf[blk] = *reinterpret_cast<const bf16x8*>(k_lds + (32 * blk + col) * T::KROW + 16 * kk + 8 * h);
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
        s[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[blk], qf[kk], s[blk], 0, 0, 0);
    }

    // element i of block blk holds key j0 + 32 blk + 16 (i / 8) + 8 h + i % 8;
    // the eight keys of group gi = 2 blk + i / 8 (for either half) lie in one page
    if (j0 + BLOCK_N > wave_min_lim) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (j0 + 32 * blk + 16 * (i >> 3) + 8 * h + (i & 7) >= lim) s[blk][i] = -INFINITY;
    }
    // per-group factor from raw score to log2 units.  fp8: times the K scale of
    // the key's page; a tile that crosses the prefix end scales per key instead.
    float cg[4];
#pragma unroll
    for (int gi = 0; gi < 4; ++gi) cg[gi] = c;
    if constexpr (FP8) {
      if (mode == MODE_PREFIX) {
#pragma unroll
        for (int gi = 0; gi < 4; ++gi) cg[gi] = c * sc_cur.k[(16 * gi + 8 * h) / P];
      } else if (mode == MODE_MIXED) {
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int kl = 32 * blk + 16 * (i >> 3) + 8 * h + (i & 7);
            if (j0 + kl < lp) s[blk][i] *= sc_cur.k[kl / P];
          }
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int gi = 0; gi < 4; ++gi) {
      float gm = -INFINITY;
#pragma unroll
      for (int e = 0; e < 8; ++e) gm = fmaxf(gm, s[gi >> 1][8 * (gi & 1) + e]);
      mx = fmaxf(mx, gm * cg[gi]);
    }
    {
      // lanes l and l + 32 hold the two halves of one row's keys
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                       false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    // lazy rescale: keep a stale running max until some row's max exceeds it
    // by more than 8 (log2 units); the weights then stay below 2^8
    if (__any(mx > m_run + 8.f)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int b = 0; b < T::DB; ++b) o[b] *= alpha;
    }

    bf16x8 pf[4];
#pragma unroll
    for (int gi = 0; gi < 4; ++gi) {
      float pv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pv[e] = __builtin_amdgcn_exp2f(fmaf(s[gi >> 1][8 * (gi & 1) + e], cg[gi], -m_run));
      if constexpr (FP8) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int kl = 16 * gi + 8 * h + e;
          const float vsc = (mode == MODE_PREFIX || (mode == MODE_MIXED && j0 + kl < lp))
                                ? sc_cur.v[kl / P] : 1.f;
          l_run += pv[e];
          pf[gi][e] = static_cast<__bf16>(pv[e] * vsc);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[gi][e] = static_cast<__bf16>(pv[e]);
        // row sum of the rounded weights, so numerator and denominator agree
        const bf16x2 one = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
#pragma unroll
        for (int e = 0; e < 8; e += 2)
          l_run = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pf[gi][e], pf[gi][e + 1]}, one, l_run, false);
      }
    }

    // O^T += V^T P^T over four 16-key slices (the DB accumulators alternate)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      bf16x8 vf[T::DB];
#pragma unroll
      for (int b = 0; b < T::DB; ++b)
        vf[b] = *reinterpret_cast<const bf16x8*>(v_lds + (32 * b + col) * T::VROW + 16 * u + 8 * h);
#pragma unroll
      for (int b = 0; b < T::DB; ++b)
        o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[b], pf[u], o[b], 0, 0, 0);
    }
  }

  if (!wave_active) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (it.part < 0) {
    if (!row_ok) return;
    const float inv = 1.f / l_tot;
    uint16_t* orow = static_cast<uint16_t*>(p.out) + (size_t(sq.cu + t) * hq + size_t(kvh) * G + g) * D;
#pragma unroll
    for (int b = 0; b < T::DB; ++b) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = 32 * b + 8 * q4 + 4 * h;
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = static_cast<__bf16>(o[b][4 * q4 + e] * inv);
        *reinterpret_cast<u32x2*>(orow + d) = __builtin_bit_cast(u32x2, v4);
      }
    }
    if (p.lse != nullptr && h == 0)
      p.lse[size_t(sq.cu + t) * hq + size_t(kvh) * G + g] = (m_run + __log2f(l_tot)) * kLn2;
  } else {
    float* po = p.part_o + (size_t(it.part) * p.part_rows + r_local) * D;
#pragma unroll
    for (int b = 0; b < T::DB; ++b) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = 32 * b + 8 * q4 + 4 * h;
        float4 v = make_float4(o[b][4 * q4], o[b][4 * q4 + 1], o[b][4 * q4 + 2], o[b][4 * q4 + 3]);
        *reinterpret_cast<float4*>(po + d) = v;
      }
    }
    if (h == 0) {
      float* ml = p.part_ml + (size_t(it.part) * p.part_rows + r_local) * 2;
      ml[0] = m_run;
      ml[1] = l_tot;
    }
  }
}

// Merges the split-K partials of query rows: weights 2^(m_c - max m),
// O = sum w_c O_c / sum w_c l_c.  A workgroup of 256 lanes covers ROWS rows;
// each row's SLICES slices of 32 lanes fold every SLICES-th partial with an
// online merge, then the slices are merged through LDS (SLICES = 1 for a few
// partials per row, 8 for many).  Fixed order, no atomics.
template <int D, int SLICES>
__global__ __launch_bounds__(256) void combine_kernel(ExtendParams p) {
  constexpr int ROWS = 8 / SLICES;
  constexpr int PER = D / 32;  // dims per lane
  __shared__ float sh_o[ROWS][SLICES][D];
  __shared__ float sh_m[ROWS][SLICES], sh_l[ROWS][SLICES];
  const int wg_per_group = (p.part_rows + ROWS - 1) / ROWS;
  const int grp = blockIdx.x / wg_per_group;
  const int rsub = threadIdx.x / (32 * SLICES);
  const int lr = (blockIdx.x % wg_per_group) * ROWS + rsub;
  const CombineGroup cg = p.groups[grp];
  const bool active = lr < cg.rows;
  const int slice = (threadIdx.x / 32) % SLICES, d0 = (threadIdx.x % 32) * PER;

  float m = -INFINITY, L = 0.f, acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  for (int c = slice; active && c < cg.n_parts; c += SLICES) {
    const size_t pr = size_t(cg.part0 + c) * p.part_rows + lr;
    const float mc = p.part_ml[pr * 2], lc = p.part_ml[pr * 2 + 1];
    const float m_new = fmaxf(m, mc);
    const float a = exp2f(m - m_new), w = exp2f(mc - m_new);
    const float* po = p.part_o + pr * D + d0;
    L = L * a + w * lc;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] = acc[e] * a + w * po[e];
    m = m_new;
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
  const SeqInfo sq = p.seqs[cg.seq];
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

template <int D, int P, bool FP8>
hipError_t launch_extend_t(const ExtendParams& p, hipStream_t stream) {
  hipLaunchKernelGGL((extend_kernel<D, P, FP8>), dim3(p.n_items), dim3(THREADS), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_extend(const ExtendParams& p, int head_dim, int page_size, bool fp8,
                         hipStream_t stream) {
  if (p.n_items <= 0) return hipSuccess;
#define CW_CASE(D_, P_)                                                       \
  if (head_dim == D_ && page_size == P_)                                      \
    return fp8 ? launch_extend_t<D_, P_, true>(p, stream)                     \
               : launch_extend_t<D_, P_, false>(p, stream);
  CW_CASE(64, 16)
  CW_CASE(64, 64)
  CW_CASE(128, 16)
  CW_CASE(128, 64)
#undef CW_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_combine(const ExtendParams& p, int head_dim, int max_parts, hipStream_t stream) {
  if (p.n_groups <= 0) return hipSuccess;
  const bool many = max_parts > 4;
  const int rows_per_wg = many ? 1 : 8;
  const dim3 grid(p.n_groups * ((p.part_rows + rows_per_wg - 1) / rows_per_wg));
  if (head_dim == 64) {
    if (many) hipLaunchKernelGGL((combine_kernel<64, 8>), grid, dim3(256), 0, stream, p);
    else hipLaunchKernelGGL((combine_kernel<64, 1>), grid, dim3(256), 0, stream, p);
  } else if (head_dim == 128) {
    if (many) hipLaunchKernelGGL((combine_kernel<128, 8>), grid, dim3(256), 0, stream, p);
    else hipLaunchKernelGGL((combine_kernel<128, 1>), grid, dim3(256), 0, stream, p);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace cw
