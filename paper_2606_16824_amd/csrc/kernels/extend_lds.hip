// Prefix-cached paged extend attention, bf16 pools: direct-to-LDS staging with
// a software-pipelined tile loop.
//
// The math follows the register-staged kernel (each wave64 owns 32 packed
// query rows of one (sequence, kv head); S^T = K Q^T and O^T += V^T P^T with
// v_mfma_f32_32x32x16_bf16), but a workgroup is eight waves = 256 rows, one
// per CU, so every K/V tile brought into LDS serves twice the rows (the
// tile DMA's share of the LDS and vector-memory pipes halves per FLOP).  Three
// more changes aim at the CDNA4 issue model, where every MFMA holds the vector
// issue port for half its duration and the exponentials of the softmax cost as
// much port time as the matrix products:
//
//  * Pipelining.  While the MFMAs of tile j+1's scores run, the same wave
//    computes tile j's weights (exp2, bf16 pack, row sums); while tile j's
//    P V MFMAs run, it scales and masks tile j+1's scores.  K tiles and V tiles
//    rotate through separate two-stage rings: in iteration j the wave reads
//    K_{j+1} and V_j while K_{j+2} and V_{j+1} land, one barrier per tile.
//
//  * A max-free fast path.  The running max m is only raised when it has to
//    be: the weights exp2(s c - m) of a tile are computed against the current
//    m, and only if some half-row's weight sum exceeds 2^16 (or is not finite)
//    is the tile's row max taken, m raised and the tile's weights recomputed
//    (the final O / l and the log-sum-exp do not depend on which m was used).
//    The first tile of an item sets m to its exact row max.
//
//  * Buffer-addressed DMA.  K and V tiles travel from HBM straight into LDS
//    with buffer_load_dwordx4 ... lds: the page base sits in the scalar buffer
//    descriptor and each lane's offset within the page is a constant register,
//    so issuing a tile costs no vector instructions.
//
// LDS holds K and V rows in their natural [key][dim] order, 16-byte chunks
// XOR-swizzled per row so that every fragment read is bank-conflict free:
//   K row R, chunk c at position c ^ k_swz(R);  V row R, chunk c at c ^ v_swz(R)
// The DMA writes lane l's 16 bytes at base + 16 l, so each lane fetches the
// global chunk that belongs at its position.  Each wave fetches 8 consecutive
// rows of a tile, which lie in one page (P = 16 or 64).
//
// V^T operand: ds_read_b64_tr_b16 hands lane i of each 16-lane group element
// in[4k + i/4][i % 4] of the 4-element rows its group's lanes point at.  Lanes
// (k, a) = (i / 4, i % 4) point at key 4k-offset rows and dims 4a .. 4a+3, so
// lane L receives V[keys 4e .. 4e+3 of its 8-key slot][dim 32b + L % 32]: half of
// the A operand of V^T P^T; two reads give all eight keys.
#include <hip/hip_runtime.h>

#include "../cw_internal.h"

namespace cw {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr float kNegBig = -1.0e30f;
constexpr float kLn2 = 0.69314718055994531f;
// A half-row weight sum above this (or not finite) makes the tile raise the
// running max: weights then stay below 2^16 and fp32 accumulators far from
// overflow.
constexpr float kSumLimit = 65536.f;

// Raw buffer descriptor for `base` (no stride, no range limit in practice).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_at(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, -1, 0x00020000);
}

// 16 bytes per lane from base + voff + soff straight into LDS (lane l's bytes
// land at dst + 16 l).  Kept in a non-template function: referenced directly
// from the kernel template, the builtin keeps the host pass from emitting the
// kernel's launch stub.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, lds_void* dst, uint32_t voff,
                                      uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, soff, 0, 0);
}

__device__ __forceinline__ int swap_bits_2_3(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Chunk swizzles.  The LDS serves 256 bytes per clock (64 banks of 4 bytes), so a
// fragment read is conflict free when the lanes served together hit distinct
// 16-byte positions modulo 256 bytes.
//  K (ds_read_b128, 16 lanes per clock): lane m reads row swap_bits_2_3(m);
//    XOR-ing the chunk with swap_bits_2_3(row) & 15 (D=128, 256-byte rows) or
//    (swap_bits_2_3(row) >> 1) & 7 (D=64, two rows per 256 bytes) spreads them.
//  V (ds_read_b64_tr_b16, 32 lanes per clock): four consecutive key rows x
//    four chunks per clock; XOR-ing with 4 (row & 3) (D=128) or 4 ((row >> 1) & 1)
//    (D=64) spreads them.
template <int D>
__device__ __forceinline__ int k_swz(int row) {
  return D == 128 ? (swap_bits_2_3(row) & 15) : ((swap_bits_2_3(row) >> 1) & 7);
}
template <int D>
__device__ __forceinline__ int v_swz(int row) {
  return D == 128 ? 4 * (row & 3) : 4 * ((row >> 1) & 1);
}

template <int D, int P>
struct LGeo {
  static constexpr int RB = 2 * D;                    // bytes per K/V row
  static constexpr int CPR = D / 8;                   // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;                // rows per wave DMA instruction
  static constexpr int NI = BLOCK_N / RPI / LDS_WAVES;  // DMA instructions per wave per matrix
  static constexpr int TILE = BLOCK_N * RB;           // bytes of one K (or V) tile
  static constexpr int KT = D / 16;                   // k-steps of K Q^T
  static constexpr int DB = D / 32;                   // 32-row blocks of O^T
  static_assert(NI * RPI == 8, "each wave fetches 8 rows of a tile");
};

template <int D, int P>
__global__ __launch_bounds__(LDS_THREADS) __attribute__((amdgpu_waves_per_eu(2)))
void extend_lds_kernel(ExtendParams p) {
  using T = LGeo<D, P>;
  // two-stage rings of K and V tiles, each stage its own array so the compiler
  // can tell that reads of one stage never alias the DMA in flight into another
  __shared__ __attribute__((aligned(1024))) uint8_t lds_k0[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_k1[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_v0[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_v1[T::TILE];

  const WorkItem it = p.items[blockIdx.x];
  if (it.seq < 0) return;  // idle padding item (uniform across the workgroup)
  const SeqInfo sq = p.seqs[it.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  const int h = lane >> 5, col = lane & 31;
  const int G = p.gqa_group, hkv = p.num_kv_heads, hq = hkv * G;
  const int kvh = it.kvh;
  const int lp = sq.lp, total_len = sq.lp + sq.ls;
  const int32_t* bt = p.block_table + size_t(it.seq) * p.bt_stride;
  const uint8_t* k_pool = static_cast<const uint8_t*>(p.k_pool);
  const uint8_t* v_pool = static_cast<const uint8_t*>(p.v_pool);
  const uint8_t* k_new = static_cast<const uint8_t*>(p.k_new);
  const uint8_t* v_new = static_cast<const uint8_t*>(p.v_new);

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

  // stale LDS must be finite: rows past the sequence are never fetched
  for (int i = tid; i < T::TILE / 16; i += LDS_THREADS) {
    reinterpret_cast<u32x4*>(lds_k0)[i] = u32x4{0u, 0u, 0u, 0u};
    reinterpret_cast<u32x4*>(lds_k1)[i] = u32x4{0u, 0u, 0u, 0u};
    reinterpret_cast<u32x4*>(lds_v0)[i] = u32x4{0u, 0u, 0u, 0u};
    reinterpret_cast<u32x4*>(lds_v1)[i] = u32x4{0u, 0u, 0u, 0u};
  }

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

  // ---- DMA geometry.  Wave w fetches tile rows [8 w, 8 w + 8); its
  // instruction j covers rows R0_j = 8 w + RPI j .. + RPI - 1 and lane l fetches
  // row R0_j + l / CPR into position l % CPR.  Within a page block the lane's
  // source offset is (R % P) RB + 16 chunk; a suffix row lives at R hkv RB +
  // 16 chunk from the tile's first new row, which is the same offset plus
  // sfx_lane (per lane) plus sfx_uniform(j) (per instruction).
  const int dma_row = lane / T::CPR, dma_pos = lane % T::CPR;
  const int wrow0 = 8 * wave;
  uint32_t k_off[T::NI], v_off[T::NI];
#pragma unroll
  for (int j = 0; j < T::NI; ++j) {
    const int R = wrow0 + T::RPI * j + dma_row;
    k_off[j] = (R % P) * T::RB + 16 * (dma_pos ^ k_swz<D>(R));
    v_off[j] = (R % P) * T::RB + 16 * (dma_pos ^ v_swz<D>(R));
  }
  const uint32_t sfx_lane = uint32_t(dma_row * (hkv - 1) * T::RB);
  auto sfx_uniform = [&](int j) -> uint32_t {
    const int R0 = wrow0 + T::RPI * j;
    return uint32_t((R0 * hkv - R0 % P) * T::RB);
  };
  const size_t page_bytes = size_t(P) * T::RB;  // one (page, kv head) block

  // physical page of this wave's rows of the tile at j0 (0 if they hold no
  // prefix key).  The load stays a vector register until the tile is issued an
  // iteration later, so waiting for it never waits for the DMA issued meanwhile.
  // Read through the constant address space so the load is a scalar one: it
  // counts against lgkmcnt instead of vmcnt, so waiting for it never waits for
  // tile DMA issued before it.
  typedef __attribute__((address_space(4))) const int32_t const_i32;
  const_i32* bt_s = (const_i32*)bt;
  auto load_page = [&](int j0) -> int { return (j0 + wrow0 < lp) ? bt_s[(j0 + wrow0) / P] : 0; };

  // DMA of one matrix (K or V) of the tile at j0 into dst.  Rows of the cached
  // prefix come from the pool page `pg`, rows of the suffix from the new
  // tokens; rows past the sequence are left as they are (their scores are
  // masked).  Wave-uniform branches except where the wave's rows straddle the
  // prefix end or the sequence end.
  auto issue = [&](int j0, uint8_t* dst, int pg, const uint8_t* pool, const uint8_t* fresh,
                   const uint32_t(&off)[T::NI]) __attribute__((always_inline)) {
    const int k_first = j0 + wrow0, k_last = k_first + 7;
    if (k_first < lp) {
      const auto rs = rsrc_at(pool + (size_t(pg) * hkv + kvh) * page_bytes);
      if (k_last < lp) {
#pragma unroll
        for (int j = 0; j < T::NI; ++j)
          dma16(rs, (lds_void*)(dst + (wrow0 + T::RPI * j) * T::RB), off[j], 0);
      } else {
#pragma unroll
        for (int j = 0; j < T::NI; ++j)
          if (k_first + T::RPI * j + dma_row < lp)
            dma16(rs, (lds_void*)(dst + (wrow0 + T::RPI * j) * T::RB), off[j], 0);
      }
    }
    if (k_last >= lp && k_first < total_len) {
      // base of the tile's first key as if it were a new token (it may lie
      // before the buffer when the tile straddles the prefix end; only rows
      // at or past the prefix end are fetched from it)
      const ptrdiff_t row0 = ptrdiff_t(sq.cu) + j0 - lp;
      const auto rs = rsrc_at(fresh + (row0 * hkv + kvh) * T::RB);
      if (k_first >= lp && k_last < total_len) {
#pragma unroll
        for (int j = 0; j < T::NI; ++j)
          dma16(rs, (lds_void*)(dst + (wrow0 + T::RPI * j) * T::RB), off[j] + sfx_lane,
                sfx_uniform(j));
      } else {
#pragma unroll
        for (int j = 0; j < T::NI; ++j) {
          const int key = k_first + T::RPI * j + dma_row;
          if (key >= lp && key < total_len)
            dma16(rs, (lds_void*)(dst + (wrow0 + T::RPI * j) * T::RB), off[j] + sfx_lane,
                  sfx_uniform(j));
        }
      }
    }
  };

  // ---- LDS fragment addresses (relative to a stage's base).
  // K: k-step kk of block blk reads row swap_bits_2_3(col) + 32 blk, position
  //    (2 kk + h) ^ k_swz(row); the swizzle of row + 32 equals that of row.
  uint32_t k_addr[T::KT];
  {
    const int R = swap_bits_2_3(col);
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) k_addr[kk] = R * T::RB + 16 * ((2 * kk + h) ^ k_swz<D>(R));
  }
  // V: slice u, block b, half e4 reads row 16 u + 8 h + 4 e4 + kq at chunk
  //    (4 b + 2 (grp & 1) + (a >> 1)) ^ v_swz(row); v_swz depends on kq only,
  //    so (u, e4) become immediate offsets.
  uint32_t v_addr[T::DB];
  {
    const int grp = lane >> 4, ri = lane & 15;
    const int kq = ri >> 2, a = ri & 3;
#pragma unroll
    for (int b = 0; b < T::DB; ++b) {
      const int chunk = 4 * b + 2 * (grp & 1) + (a >> 1);
      v_addr[b] = (8 * h + kq) * T::RB + 16 * (chunk ^ v_swz<D>(kq)) + 8 * (a & 1);
    }
  }

  const float c = p.scale_log2;
  f32x16 o[T::DB];
#pragma unroll
  for (int b = 0; b < T::DB; ++b) o[b] = f32x16{};
  float m_run = 0.f, l_run = 0.f;

  // raw scores S^T = K Q^T of the tile in `ks`, two 32-key blocks
  auto scores = [&](const uint8_t* ks, f32x16(&s)[2]) __attribute__((always_inline)) {
    s[0] = f32x16{};
    s[1] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(ks + k_addr[kk]);
      const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(ks + k_addr[kk] + 32 * T::RB);
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qf[kk], s[0], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qf[kk], s[1], 0, 0, 0);
    }
  };
  // causal mask (only tiles that cross some row's limit).  Element i of block
  // blk holds key j0 + 32 blk + 16 (i / 8) + 8 h + i % 8.
  auto mask = [&](int j0, f32x16(&s)[2]) __attribute__((always_inline)) {
    if (j0 + BLOCK_N > wave_min_lim) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (j0 + 32 * blk + 16 * (i >> 3) + 8 * h + (i & 7) >= lim) s[blk][i] = -INFINITY;
    }
  };
  // log2 units relative to the running max
  auto to_log2 = [&](f32x16(&s)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 16; ++i) s[blk][i] = fmaf(s[blk][i], c, -m_run);
  };
  // bf16 weights of 16-key slice gi in B-operand order, and their half-row sum
  // (of the rounded weights, so numerator and denominator agree)
  auto weights = [&](const f32x16(&x)[2], bf16x8(&pf)[4], float& lsum) __attribute__((always_inline)) {
    const bf16x2 one = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
    float la = 0.f, lb = 0.f;
#pragma unroll
    for (int gi = 0; gi < 4; ++gi) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pf[gi][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(x[gi >> 1][8 * (gi & 1) + e]));
#pragma unroll
      for (int e = 0; e < 8; e += 4) {
        la = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pf[gi][e], pf[gi][e + 1]}, one, la, false);
        lb = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pf[gi][e + 2], pf[gi][e + 3]}, one, lb, false);
      }
    }
    lsum = la + lb;
  };
  // row max of x over both halves of the row (lanes l and l + 32)
  auto row_max = [&](const f32x16(&x)[2]) -> float {
    float mx = -INFINITY;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, x[blk][i]);
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                     false, false);
    return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
  };
  // O^T += V^T P^T over four 16-key slices of the V tile in `vs`
  auto accumulate = [&](const uint8_t* vs, const bf16x8(&pf)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      bf16x8 vf[T::DB];
#pragma unroll
      for (int b = 0; b < T::DB; ++b) {
        i16x4 half[2];
#pragma unroll
        for (int e4 = 0; e4 < 2; ++e4)
          half[e4] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4*)(vs + v_addr[b] + (16 * u + 4 * e4) * T::RB));
        vf[b] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(half[0], half[1], 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int b = 0; b < T::DB; ++b)
        o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[b], pf[u], o[b], 0, 0, 0);
    }
  };

  // Instruction interleaving for the scheduler (masks: 0x8 MFMA, 0x2 VALU,
  // 0x400 transcendental, 0x100 LDS read).  Scores of the next tile: four K
  // fragment reads ahead, then per MFMA two exponentials, two other vector ops
  // and one more read.
  auto interleave_scores_weights = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int i = 0; i < 2 * T::KT; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x400, 32 / (2 * T::KT), 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 32 / (2 * T::KT), 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
  };
  // P V: one slice of V fragments ahead, then per MFMA two scaling FMAs and
  // two more reads
  auto interleave_pv_scale = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * T::DB, 0);
#pragma unroll
    for (int i = 0; i < 4 * T::DB; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 32 / (4 * T::DB), 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
  };

  const int n_tiles = (it.kv_end - it.kv_begin + BLOCK_N - 1) / BLOCK_N;
  auto tile0 = [&](int j) { return it.kv_begin + j * BLOCK_N; };
  auto visible = [&](int j) { return wave_active && tile0(j) < wave_max_lim; };

  // ---- prologue: K_0, V_0 and K_1 in flight, tile 0's scores against its exact max
  f32x16 x[2] = {f32x16{}, f32x16{}};
  int pg_v = 0;      // page of V_{j+1} (uniform)
  int pg_k_raw = 0;  // page of K_{j+2}, still a vector register
  __syncthreads();   // zero fill done before any DMA lands
  if (n_tiles > 0) {
    const int pg0 = __builtin_amdgcn_readfirstlane(load_page(tile0(0)));
    const int pg1 = n_tiles > 1 ? __builtin_amdgcn_readfirstlane(load_page(tile0(1))) : 0;
    issue(tile0(0), lds_k0, pg0, k_pool, k_new, k_off);
    issue(tile0(0), lds_v0, pg0, v_pool, v_new, v_off);
    if (n_tiles > 1) issue(tile0(1), lds_k1, pg1, k_pool, k_new, k_off);
    pg_v = pg1;
    if (n_tiles > 2) pg_k_raw = load_page(tile0(2));
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (visible(0)) {
      scores(lds_k0, x);
      mask(tile0(0), x);
      to_log2(x);  // m_run = 0 here
      const float mx = row_max(x);
      // a row with no visible key in the first tile sees none in the item
      const float d = mx == -INFINITY ? 0.f : mx;
      m_run = mx == -INFINITY ? kNegBig : mx;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) x[blk] -= d;
    }
  }

  // the work of iteration j after its DMA is issued: tile j+1's scores
  // (discarded after the last visible tile: the stage then holds finite stale
  // data) while tile j's weights are formed, then tile j's P V while tile j+1's
  // scores are scaled
  auto compute = [&](int j, const uint8_t* k_nxt, const uint8_t* v_cur,
                     bool may_mask) __attribute__((always_inline)) {
    f32x16 s[2];
    bf16x8 pf[4];
    float lsum;
    scores(k_nxt, s);
    weights(x, pf, lsum);
    interleave_scores_weights();
    if (__any(!(lsum <= kSumLimit))) {
      // raise the running max to this tile's row max and redo its weights
      const float d = fmaxf(row_max(x), 0.f);
      m_run += d;
      const float alpha = __builtin_amdgcn_exp2f(-d);
      l_run *= alpha;
#pragma unroll
      for (int b = 0; b < T::DB; ++b) o[b] *= alpha;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) x[blk] -= d;
      weights(x, pf, lsum);
    }
    l_run += lsum;
    if (may_mask) mask(tile0(j + 1), s);
    accumulate(v_cur, pf);
    to_log2(s);
    interleave_pv_scale();
    x[0] = s[0];
    x[1] = s[1];
  };

  // iteration j: K_{j+1} and V_j are resident; K_{j+2} goes to K_j's stage,
  // V_{j+1} to V_{j-1}'s
  auto iteration = [&](int j, uint8_t* k_cur, uint8_t* k_nxt, uint8_t* v_cur,
                       uint8_t* v_nxt) __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's DMA of K_{j+1} and V_j has landed
    __syncthreads();                // everyone's has; K_j and V_{j-1} are no longer read
    const int pg_k = __builtin_amdgcn_readfirstlane(pg_k_raw);
    if (j + 2 < n_tiles) issue(tile0(j + 2), k_cur, pg_k, k_pool, k_new, k_off);
    if (j + 1 < n_tiles) issue(tile0(j + 1), v_nxt, pg_v, v_pool, v_new, v_off);
    pg_v = pg_k;
    if (j + 3 < n_tiles) pg_k_raw = load_page(tile0(j + 3));
    if (!visible(j)) return;  // nothing visible for this wave from here on
    compute(j, k_nxt, v_cur, true);
  };

  // Iterations whose tiles j .. j+2 lie wholly in the cached prefix: every row
  // sees all their keys (no mask) and their DMA comes from one pool page per
  // wave, so the loop carries no per-tile mode decisions.
  const uint8_t* k_pool_kvh = k_pool + size_t(kvh) * page_bytes;
  const uint8_t* v_pool_kvh = v_pool + size_t(kvh) * page_bytes;
  const size_t page_stride = size_t(hkv) * page_bytes;
  auto issue_prefix = [&](uint8_t* dst, int pg, const uint8_t* pool_kvh,
                          const uint32_t(&off)[T::NI]) __attribute__((always_inline)) {
    const auto rs = rsrc_at(pool_kvh + size_t(pg) * page_stride);
#pragma unroll
    for (int j = 0; j < T::NI; ++j)
      dma16(rs, (lds_void*)(dst + (wrow0 + T::RPI * j) * T::RB), off[j], 0);
  };
  auto steady = [&](int j, uint8_t* k_cur, uint8_t* k_nxt, uint8_t* v_cur,
                    uint8_t* v_nxt) __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    const int pg_k = __builtin_amdgcn_readfirstlane(pg_k_raw);
    issue_prefix(k_cur, pg_k, k_pool_kvh, k_off);
    issue_prefix(v_nxt, pg_v, v_pool_kvh, v_off);
    pg_v = pg_k;
    pg_k_raw = load_page(tile0(j + 3));  // an in-range entry whenever it is a prefix page
    if (wave_active) compute(j, k_nxt, v_cur, false);
  };

  const int n_prefix = lp > it.kv_begin ? min(n_tiles, (lp - it.kv_begin) / BLOCK_N) : 0;
  const int n_steady = max(0, n_prefix - 2);
  int j = 0;
  for (; j + 1 < n_steady; j += 2) {
    steady(j, lds_k0, lds_k1, lds_v0, lds_v1);
    steady(j + 1, lds_k1, lds_k0, lds_v1, lds_v0);
  }
  if (j < n_steady) {
    steady(j, lds_k0, lds_k1, lds_v0, lds_v1);
    ++j;
  }
  if ((j & 1) && j < n_tiles) {
    iteration(j, lds_k1, lds_k0, lds_v1, lds_v0);
    ++j;
  }
  for (; j < n_tiles; j += 2) {
    iteration(j, lds_k0, lds_k1, lds_v0, lds_v1);
    if (j + 1 < n_tiles) iteration(j + 1, lds_k1, lds_k0, lds_v1, lds_v0);
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

template <int D, int P>
hipError_t launch_t(const ExtendParams& p, hipStream_t stream) {
  hipLaunchKernelGGL((extend_lds_kernel<D, P>), dim3(p.n_items), dim3(LDS_THREADS), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_extend_lds(const ExtendParams& p, int head_dim, int page_size,
                             hipStream_t stream) {
  if (p.n_items <= 0) return hipSuccess;
  if (head_dim == 64 && page_size == 16) return launch_t<64, 16>(p, stream);
  if (head_dim == 64 && page_size == 64) return launch_t<64, 64>(p, stream);
  if (head_dim == 128 && page_size == 16) return launch_t<128, 16>(p, stream);
  if (head_dim == 128 && page_size == 64) return launch_t<128, 64>(p, stream);
  return hipErrorInvalidValue;
}

}  // namespace cw
