// Prefix-cached paged extend attention on LDS-staged tiles, software-pipelined.
//
// The math follows the register-staged kernel (each wave64 owns 32 packed
// query rows of one (sequence, kv head); S^T = K Q^T and O^T += V^T P^T with
// v_mfma_f32_32x32x16_bf16), but a workgroup is eight waves = 256 rows, one
// per CU, so every K/V tile brought into LDS serves twice the rows (the tile
// staging's share of the LDS and vector-memory pipes halves per FLOP).  Three
// more changes aim at the CDNA4 issue model, where every MFMA holds the vector
// issue port for half its duration and the exponentials of the softmax cost as
// much port time as the matrix products:
//
//  * Pipelining.  While the MFMAs of tile j+1's scores run, the same wave
//    computes tile j's weights (exp2, bf16 pack, row sums); while tile j's
//    P V MFMAs run, it scales and masks tile j+1's scores.  K tiles and V tiles
//    rotate through separate two-stage rings: in iteration j the wave reads
//    K_{j+1} and V_j while K_{j+2} and V_{j+1} are staged, one barrier per tile.
//
//  * A max-free fast path.  The running max m is only raised when it has to
//    be: the weights exp2(s c - m) of a tile are computed against the current
//    m, and only if some half-row's weight sum exceeds 2^16 (or is not finite)
//    is the tile's row max taken, m raised and the tile's weights recomputed
//    (the final O / l and the log-sum-exp do not depend on which m was used).
//    The first tile of an item sets m to its exact row max.
//
//  * Buffer-addressed staging.  The page base sits in a scalar buffer
//    descriptor and each lane's offset within the page is a constant register.
//    bf16 rows travel from HBM straight into LDS (buffer_load_dwordx4 ... lds).
//
// fp8-e4m3fn pools run the same loop in fp16 (v_mfma_f32_32x32x16_f16): pool
// rows are loaded into registers one iteration ahead and dequantised while they
// are widened into LDS, code x page scale rounded to fp16 once (the scale's
// power of two is applied exactly by the conversion, its significand by one
// packed fp16 multiply per two values), so the loop itself never sees a scale.
// The new tokens' bf16 rows arrive by DMA like bf16 pool rows, and the wave
// that staged them converts them to fp16 in place before the barrier that
// publishes the tile.  Q is scaled into fp16 the same way as into bf16 for bf16
// pools, and P is rounded to fp16.  fp16 keeps 11 significant bits against
// bf16's 8, so every rounding of this path is finer than the bf16 path's; the
// values must lie within the fp16 range (|x| < 65504), which holds for the
// scaled e4m3fn codes of any page scale below 146 and for the new K/V rows the
// path is used with.
//
// LDS holds K and V rows in their natural [key][dim] order, 16-byte chunks
// XOR-swizzled per row so that every fragment read is bank-conflict free:
//   K row R, chunk c at position c ^ k_swz(R);  V row R, chunk c at c ^ v_swz(R)
// The DMA writes lane l's 16 bytes at base + 16 l, so each lane fetches the
// global chunk that belongs at its position.  Each wave stages 8 consecutive
// rows of a tile, which lie in one page (P = 16 or 64).
//
// V^T operand: ds_read_b64_tr_b16 hands lane i of each 16-lane group element
// in[4k + i/4][i % 4] of the 4-element rows its group's lanes point at.  Lanes
// (k, a) = (i / 4, i % 4) point at key 4k-offset rows and dims 4a .. 4a+3, so
// lane L receives V[keys 4e .. 4e+3 of its 8-key slot][dim 32b + L % 32]: half of
// the A operand of V^T P^T; two reads give all eight keys.
#include <hip/hip_runtime.h>

#include "../cw_internal.h"
#include "page_write.h"

namespace cw {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
// Read through the constant address space so that loads with a uniform
// address are scalar loads: they count against lgkmcnt instead of vmcnt, so
// waiting for them never waits for tile staging issued before them.
typedef __attribute__((address_space(4))) const int32_t const_i32;
typedef __attribute__((address_space(4))) const float const_f32;
constexpr uint32_t kOnePairF16 = 0x3C003C00u;  // fp16 pair (1, 1)

constexpr float kNegBig = -1.0e30f;
constexpr float kLn2 = 0.69314718055994531f;
// A half-row weight sum above this (or not finite) makes the tile raise the
// running max: weights then stay below 2^16 and fp32 accumulators far from
// overflow.
constexpr float kSumLimit = 65536.f;
constexpr uint32_t kOnePair = 0x3F803F80u;  // bf16 pair (1, 1)

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

// Page scale s = p2 x fm with p2 a positive power of two and |fm| in [1, 2):
// the conversion applies p2 exactly, fm is rounded to fp16 for the packed
// multiply (s finite and normal; 0 dequantises to 0).
struct PageScale {
  float p2;
  f16x2 fm;
};
__device__ __forceinline__ PageScale page_scale(float s) {
  const uint32_t b = __float_as_uint(s);
  const float p2 = __uint_as_float(b & 0x7F800000u);                   // exponent
  const float f = __uint_as_float((b & 0x807FFFFFu) | 0x3F800000u);    // sign, significand in [1, 2)
  const _Float16 m = static_cast<_Float16>(f);
  return PageScale{p2, f16x2{m, m}};
}
// Two e4m3fn codes (bytes 0,1 or 2,3 of `w`) -> two fp16 code x s in one dword.
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_f16x2(uint32_t w, PageScale sc) {
  const f16x2 v = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(static_cast<int>(w), sc.p2, HI);
  return __builtin_bit_cast(uint32_t, v * sc.fm);
}
__device__ __forceinline__ u32x4 fp8x8_f16x8(uint32_t lo, uint32_t hi, PageScale sc) {
  return u32x4{fp8x2_f16x2<false>(lo, sc), fp8x2_f16x2<true>(lo, sc), fp8x2_f16x2<false>(hi, sc),
               fp8x2_f16x2<true>(hi, sc)};
}
// Eight bf16 -> eight fp16 (exact within the fp16 range: bf16 keeps 8
// significant bits, fp16 11).
__device__ __forceinline__ u32x4 bf16x8_f16x8(u32x4 x) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float lo = __uint_as_float(x[i] << 16), hi = __uint_as_float(x[i] & 0xFFFF0000u);
    r[i] = __builtin_bit_cast(uint32_t, f16x2{static_cast<_Float16>(lo), static_cast<_Float16>(hi)});
  }
  return r;
}
// 32x32x16 MFMA on 16-bit operands held as raw bits: fp16 for fp8 pools, bf16
// otherwise.
template <bool F16>
__device__ __forceinline__ f32x16 mfma16(u32x4 a, u32x4 b, f32x16 c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
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

template <int D, int P, bool FP8>
struct LGeo {
  static constexpr int RB = 2 * D;                    // bytes per bf16 K/V row in LDS
  static constexpr int CPR = D / 8;                   // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;                // rows per wave DMA instruction
  static constexpr int NI = BLOCK_N / RPI / LDS_WAVES;  // DMA instructions per wave per matrix
  static constexpr int TILE = BLOCK_N * RB;           // bytes of one K (or V) tile
  static constexpr int KT = D / 16;                   // k-steps of K Q^T
  static constexpr int DB = D / 32;                   // 32-row blocks of O^T
  static constexpr int PRB = FP8 ? D : RB;            // bytes per pool row
  static constexpr int B8 = D / 8;                    // fp8 bytes each lane stages per matrix
  static_assert(NI * RPI == 8, "each wave stages 8 rows of a tile");
};

template <int D, int P, bool FP8, bool AP>
__global__ __launch_bounds__(LDS_THREADS) __attribute__((amdgpu_waves_per_eu(2)))
void extend_lds_kernel(ExtendParams p, PlanArg<AP> ap) {
  using T = LGeo<D, P, FP8>;
  // two-stage rings of K and V tiles, each stage its own array so the compiler
  // can tell that reads of one stage never alias the DMA in flight into another
  __shared__ __attribute__((aligned(1024))) uint8_t lds_k0[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_k1[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_v0[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_v1[T::TILE];

  // Fused page write: this workgroup's share of the new rows' 16-byte pieces
  // goes to the pools.  The extend never reads a slot at or past a sequence's
  // prefix end from the pool, so the writes and the attention are independent.
  auto fused_write = [&]() __attribute__((always_inline)) {
    WriteParams w = p.w;
    w.seqs = plan_ptr<AP>(ap, p.ap_wseqs, p.w.seqs);
    const int64_t total = int64_t(w.total_tokens) * w.num_kv_heads * (D / 8);
    const int64_t per = (total + gridDim.x - 1) / gridDim.x;
    const int64_t end = min(total, int64_t(blockIdx.x + 1) * per);
    for (int64_t idx = int64_t(blockIdx.x) * per + threadIdx.x; idx < end; idx += LDS_THREADS)
      pw::write_piece<D, P, FP8>(w, idx);
  };

  const WorkItem it = plan_ptr<AP>(ap, p.ap_items, p.items)[blockIdx.x];
  if (it.seq < 0) {  // idle padding item (uniform across the workgroup)
    if (p.w.total_tokens > 0) fused_write();
    return;
  }
  const SeqInfo sq = plan_ptr<AP>(ap, p.ap_seqs, p.seqs)[it.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  const int h = lane >> 5, col = lane & 31;
  const int G = p.gqa_group, hkv = p.num_kv_heads, hq = hkv * G;
  const int kvh = it.kvh;
  const int lp = sq.lp, total_len = sq.lp + sq.ls;
  const int32_t* bt = p.block_table + size_t(sq.bt_row) * p.bt_stride;
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

  // stale LDS must be finite: rows past the sequence are never staged
  for (int i = tid; i < T::TILE / 16; i += LDS_THREADS) {
    reinterpret_cast<u32x4*>(lds_k0)[i] = u32x4{0u, 0u, 0u, 0u};
    reinterpret_cast<u32x4*>(lds_k1)[i] = u32x4{0u, 0u, 0u, 0u};
    reinterpret_cast<u32x4*>(lds_v0)[i] = u32x4{0u, 0u, 0u, 0u};
    reinterpret_cast<u32x4*>(lds_v1)[i] = u32x4{0u, 0u, 0u, 0u};
  }

  // Q^T as the B operand: k-step kk holds dims 16 kk + 8 h + [0, 8) of this row.
  // Q carries the softmax scale in log2 units (q c rounded to bf16, or to fp16
  // for fp8 pools), so the score MFMAs, started from -m, leave s c - m with no
  // vector work.
  const float c = p.scale_log2;
  u32x4 qf[T::KT];
  {
    const uint16_t* qrow =
        static_cast<const uint16_t*>(p.q) + (size_t(sq.cu + t) * hq + size_t(kvh) * G + g) * D;
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row_ok) v = *reinterpret_cast<const u32x4*>(qrow + 16 * kk + 8 * h);
      const bf16x8 qb = __builtin_bit_cast(bf16x8, v);
      if constexpr (FP8) {
        f16x8 qh;
#pragma unroll
        for (int e = 0; e < 8; ++e) qh[e] = static_cast<_Float16>(static_cast<float>(qb[e]) * c);
        qf[kk] = __builtin_bit_cast(u32x4, qh);
      } else {
        bf16x8 qs;
#pragma unroll
        for (int e = 0; e < 8; ++e) qs[e] = static_cast<__bf16>(static_cast<float>(qb[e]) * c);
        qf[kk] = __builtin_bit_cast(u32x4, qs);
      }
    }
  }

  // ---- staging geometry.  Wave w stages tile rows [8 w, 8 w + 8).
  // bf16 rows: DMA instruction j covers rows R0_j = 8 w + RPI j .. + RPI - 1 and
  // lane l fetches row R0_j + l / CPR into position l % CPR.  Within a page
  // block the lane's source offset is (R % P) RB + 16 chunk; a suffix row lives
  // at R hkv RB + 16 chunk from the tile's first new row, which is the same
  // offset plus sfx_lane (per lane) plus sfx_uniform(j) (per instruction).
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
  const size_t page_bytes = size_t(P) * T::PRB;  // one (page, kv head) block
  // fp8 rows.  D = 64: lane l stages the 8 bytes [8 (l % 8), 8 (l % 8) + 8) of row
  // 8 w + l / 8 (one widened chunk, stored at its swizzled position).  D = 128:
  // like the bf16 DMA, load u of lane l fetches what belongs at LDS position
  // l % 16 of row 8 w + 4 u + l / 16, i.e. the 8 codes of global chunk
  // (l % 16) ^ swz(row), so that each widened store fills 1 KiB of contiguous LDS
  // (conflict-free) instead of scattering two chunks over a row.
  const int r8 = wrow0 + (lane >> 3), q8 = lane & 7;
  const uint32_t off8 = uint32_t((r8 % P) * D + q8 * T::B8);
  int r8u[2];
  uint32_t koff8[2], voff8[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int R = wrow0 + 4 * u + (lane >> 4), pos = lane & 15;
    r8u[u] = R;
    koff8[u] = uint32_t((R % P) * D + 8 * (pos ^ k_swz<D>(R)));
    voff8[u] = uint32_t((R % P) * D + 8 * (pos ^ v_swz<D>(R)));
  }

  const_i32* bt_s = (const_i32*)bt;
  // physical page of this wave's rows of the tile at j0 (0 if they hold no prefix key)
  auto load_page = [&](int j0) -> int { return (j0 + wrow0 < lp) ? bt_s[(j0 + wrow0) / P] : 0; };

  // DMA of one matrix (K or V) of the tile at j0 into dst.  Rows of the cached
  // prefix come from the pool page `pg` (bf16 pools only: fp8 rows are widened
  // through registers), rows of the suffix from the new tokens; rows past the
  // sequence are left as they are (their scores are masked).  Wave-uniform
  // branches except where the wave's rows straddle the prefix end or the
  // sequence end.
  auto issue = [&](int j0, uint8_t* dst, int pg, const uint8_t* pool, const uint8_t* fresh,
                   const uint32_t(&off)[T::NI]) __attribute__((always_inline)) {
    const int k_first = j0 + wrow0, k_last = k_first + 7;
    if (!FP8 && k_first < lp) {
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

  // fp8 pool rows of the tile at j0 into registers (nothing when this wave's
  // rows hold no prefix key; rows of the page past the prefix end are loaded
  // but never stored)
  // (`in_prefix`: the tile lies wholly in the cached prefix, so every row check
  // below is known to pass)
  auto load8 = [&](int j0, int pg, const uint8_t* pool, bool is_k,
                   bool in_prefix) __attribute__((always_inline)) -> u32x4 {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (in_prefix || j0 + wrow0 < lp) {
      const auto rs = rsrc_at(pool + (size_t(pg) * hkv + kvh) * page_bytes);
      if constexpr (T::B8 == 16) {
        const u32x2 a = __builtin_amdgcn_raw_buffer_load_b64(rs, is_k ? koff8[0] : voff8[0], 0, 0);
        const u32x2 b = __builtin_amdgcn_raw_buffer_load_b64(rs, is_k ? koff8[1] : voff8[1], 0, 0);
        v = u32x4{a.x, a.y, b.x, b.y};
      } else {
        const u32x2 w = __builtin_amdgcn_raw_buffer_load_b64(rs, off8, 0, 0);
        v = u32x4{w.x, w.y, 0u, 0u};
      }
    }
    return v;
  };
  // ... dequantised to fp16 with the page's scale and stored at the swizzled
  // positions of their rows
  auto store8 = [&](int j0, u32x4 v, uint8_t* dst, bool is_k, float scale,
                    bool in_prefix) __attribute__((always_inline)) {
    if (!in_prefix && j0 + wrow0 >= lp) return;
    const PageScale sc = page_scale(scale);
    if constexpr (T::B8 == 16) {
      if (in_prefix || j0 + r8u[0] < lp)
        *reinterpret_cast<u32x4*>(dst + wrow0 * T::RB + 16 * lane) = fp8x8_f16x8(v.x, v.y, sc);
      if (in_prefix || j0 + r8u[1] < lp)
        *reinterpret_cast<u32x4*>(dst + (wrow0 + 4) * T::RB + 16 * lane) = fp8x8_f16x8(v.z, v.w, sc);
    } else if (in_prefix || j0 + r8 < lp) {
      const int swz = is_k ? k_swz<D>(r8) : v_swz<D>(r8);
      *reinterpret_cast<u32x4*>(dst + r8 * T::RB + 16 * (q8 ^ swz)) = fp8x8_f16x8(v.x, v.y, sc);
    }
  };
  // fp8 pools: the new tokens' rows of the tile at j0 that this wave staged by
  // DMA into dst (bf16) are converted to fp16 in place, each lane its own 16
  // bytes (before the barrier that publishes the tile)
  auto convert_new = [&](int j0, uint8_t* dst) __attribute__((always_inline)) {
    const int k_first = j0 + wrow0, k_last = k_first + 7;
    if (k_last < lp || k_first >= total_len) return;
#pragma unroll
    for (int j = 0; j < T::NI; ++j) {
      const int key = k_first + T::RPI * j + dma_row;
      if (key >= lp && key < total_len) {
        u32x4* ptr = reinterpret_cast<u32x4*>(dst + (wrow0 + T::RPI * j) * T::RB + 16 * lane);
        *ptr = bf16x8_f16x8(*ptr);
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

  f32x16 o[T::DB];
#pragma unroll
  for (int b = 0; b < T::DB; ++b) o[b] = f32x16{};
  // A wave that sees no key of this item (a split-K chunk past its rows' causal
  // limits) keeps m = kNegBig and l = 0, so its partial gets weight 0 in the
  // merge whatever the other chunks' maxima are.
  float m_run = kNegBig, l_run = 0.f;
  f32x16 negm = f32x16{};  // -m_run in every element (the score MFMAs' start)

  const int n_tiles = (it.kv_end - it.kv_begin + BLOCK_N - 1) / BLOCK_N;
  auto tile0 = [&](int j) { return it.kv_begin + j * BLOCK_N; };
  auto visible = [&](int j) { return wave_active && tile0(j) < wave_max_lim; };

  // ---- fp8 page scales: the wave's rows of a tile lie in one page, so one K
  // and one V scale per wave and tile (1 where its rows hold no prefix key)
  const_f32* ks_s = (const_f32*)p.k_scale;
  const_f32* vs_s = (const_f32*)p.v_scale;
  auto load_scale = [&](const_f32* tbl, int j0, int pg) -> float {
    return j0 + wrow0 < lp ? tbl[size_t(pg) * hkv + kvh] : 1.f;
  };

  // scores S^T = K Q^T of the tile in `ks`, two 32-key blocks: s c - m_run
  // (scaled Q, accumulation started at -m_run)
  auto scores = [&](const uint8_t* ks, f32x16(&s)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      const u32x4 k0 = *reinterpret_cast<const u32x4*>(ks + k_addr[kk]);
      const u32x4 k1 = *reinterpret_cast<const u32x4*>(ks + k_addr[kk] + 32 * T::RB);
      s[0] = mfma16<FP8>(k0, qf[kk], kk > 0 ? s[0] : negm);
      s[1] = mfma16<FP8>(k1, qf[kk], kk > 0 ? s[1] : negm);
    }
  };
  // causal mask (only tiles that cross some row's limit).  Element i of block
  // blk holds key j0 + 32 blk + 16 (i / 8) + 8 h + i % 8, which is in group
  // 2 blk + i / 8.
  auto mask = [&](int j0, f32x16(&s)[2]) __attribute__((always_inline)) {
    if (j0 + BLOCK_N > wave_min_lim) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (j0 + 32 * blk + 16 * (i >> 3) + 8 * h + (i & 7) >= lim) s[blk][i] = -INFINITY;
    }
  };
  // weights of 16-key slice gi in B-operand order (bf16, fp16 for fp8 pools)
  // and their half-row sum (of the rounded weights, so numerator and
  // denominator agree)
  auto weights = [&](const f32x16(&x)[2], u32x4(&pf)[4], float& lsum) __attribute__((always_inline)) {
    float la = 0.f, lb = 0.f;
    if constexpr (FP8) {
      const f16x2 one = __builtin_bit_cast(f16x2, kOnePairF16);
#pragma unroll
      for (int gi = 0; gi < 4; ++gi) {
        f16x8 w;
#pragma unroll
        for (int e = 0; e < 8; ++e) w[e] = static_cast<_Float16>(__builtin_amdgcn_exp2f(x[gi >> 1][8 * (gi & 1) + e]));
#pragma unroll
        for (int e = 0; e < 8; e += 4) {
          la = __builtin_amdgcn_fdot2(f16x2{w[e], w[e + 1]}, one, la, false);
          lb = __builtin_amdgcn_fdot2(f16x2{w[e + 2], w[e + 3]}, one, lb, false);
        }
        pf[gi] = __builtin_bit_cast(u32x4, w);
      }
    } else {
      const bf16x2 one = __builtin_bit_cast(bf16x2, kOnePair);
#pragma unroll
      for (int gi = 0; gi < 4; ++gi) {
        bf16x8 w;
#pragma unroll
        for (int e = 0; e < 8; ++e) w[e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(x[gi >> 1][8 * (gi & 1) + e]));
#pragma unroll
        for (int e = 0; e < 8; e += 4) {
          la = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{w[e], w[e + 1]}, one, la, false);
          lb = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{w[e + 2], w[e + 3]}, one, lb, false);
        }
        pf[gi] = __builtin_bit_cast(u32x4, w);
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
  auto accumulate = [&](const uint8_t* vs, const u32x4(&pf)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      u32x4 vf[T::DB];
#pragma unroll
      for (int b = 0; b < T::DB; ++b) {
        i16x4 half[2];
#pragma unroll
        for (int e4 = 0; e4 < 2; ++e4)
          half[e4] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4*)(vs + v_addr[b] + (16 * u + 4 * e4) * T::RB));
        vf[b] = __builtin_bit_cast(u32x4, __builtin_shufflevector(half[0], half[1], 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int b = 0; b < T::DB; ++b) o[b] = mfma16<FP8>(vf[b], pf[u], o[b]);
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
  // P V: one slice of V fragments ahead, then per MFMA two more reads
  auto interleave_pv = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * T::DB, 0);
#pragma unroll
    for (int i = 0; i < 4 * T::DB; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
  };

  // ---- prologue: tiles 0 and 1 of K and tile 0 of V staged, tile 0's scores
  // against its exact max.  bf16: K_0, V_0, K_1 by DMA, the loop then stages
  // K_{j+2} and V_{j+1} in iteration j.  fp8: the same tiles dequantised here
  // (new tokens' rows by DMA, converted in place), and the loop's first
  // iteration finds K_2 and V_1 already in registers.
  // scores of tile j in log2 units: xa for even j, xb for odd j (the stage
  // parity), so tile j+1's scores land in place with no copy
  f32x16 xa[2] = {f32x16{}, f32x16{}}, xb[2] = {f32x16{}, f32x16{}};
  int pg_v = 0;    // bf16: page of V_{j+1};  fp8: page of V_{j+2} (uniform)
  int pg_raw = 0;  // bf16: page of K_{j+2};  fp8: page of K_{j+3} (scalar load in flight)
  u32x4 k8 = {0u, 0u, 0u, 0u}, v8 = {0u, 0u, 0u, 0u};  // fp8: K_{j+2}, V_{j+1} rows
  float sk8 = 1.f, sv8 = 1.f;  // fp8: the page scales of the rows in k8 and v8
  __syncthreads();  // zero fill done before any tile lands
  if (n_tiles > 0) {
    const int pg0 = load_page(tile0(0));
    const int pg1 = n_tiles > 1 ? load_page(tile0(1)) : 0;
    issue(tile0(0), lds_k0, pg0, k_pool, k_new, k_off);
    issue(tile0(0), lds_v0, pg0, v_pool, v_new, v_off);
    if (n_tiles > 1) issue(tile0(1), lds_k1, pg1, k_pool, k_new, k_off);
    if constexpr (!FP8) {
      pg_v = pg1;
      if (n_tiles > 2) pg_raw = load_page(tile0(2));
    } else {
      const u32x4 a = load8(tile0(0), pg0, k_pool, true, false), b = load8(tile0(0), pg0, v_pool, false, false);
      u32x4 k1 = {0u, 0u, 0u, 0u};
      if (n_tiles > 1) k1 = load8(tile0(1), pg1, k_pool, true, false);
      const float sk0 = load_scale(ks_s, tile0(0), pg0), sv0 = load_scale(vs_s, tile0(0), pg0);
      const float sk1 = n_tiles > 1 ? load_scale(ks_s, tile0(1), pg1) : 1.f;
      const int pg2 = n_tiles > 2 ? load_page(tile0(2)) : 0;
      __builtin_amdgcn_s_waitcnt(0);
      store8(tile0(0), a, lds_k0, true, sk0, false);
      store8(tile0(0), b, lds_v0, false, sv0, false);
      if (n_tiles > 1) store8(tile0(1), k1, lds_k1, true, sk1, false);
      if (n_tiles > 2) {
        k8 = load8(tile0(2), pg2, k_pool, true, false);
        sk8 = load_scale(ks_s, tile0(2), pg2);
      }
      if (n_tiles > 1) {
        v8 = load8(tile0(1), pg1, v_pool, false, false);
        sv8 = load_scale(vs_s, tile0(1), pg1);
      }
      pg_v = pg2;
      if (n_tiles > 3) pg_raw = load_page(tile0(3));
    }
    if (p.w.total_tokens > 0) fused_write();  // under the first tiles' latency
    __builtin_amdgcn_s_waitcnt(0);
    // K_0's DMA'd new-token rows become fp16 here; K_1 and V_0 before the barrier
    // of iteration 0, which reads them first (every tile is converted once)
    if constexpr (FP8) convert_new(tile0(0), lds_k0);
    __syncthreads();
    if (visible(0)) {
      m_run = 0.f;  // the scores below are taken relative to 0 (negm is 0 too)
      scores(lds_k0, xa);
      mask(tile0(0), xa);
      const float mx = row_max(xa);
      // a row with no visible key in the first tile sees none in the item
      const float d = mx == -INFINITY ? 0.f : mx;
      m_run = mx == -INFINITY ? kNegBig : mx;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) xa[blk] -= d;
      negm = -m_run;
    }
  } else if (p.w.total_tokens > 0) {
    fused_write();
  }

  // the work of iteration j after its staging is issued: tile j+1's scores
  // (discarded after the last visible tile: the stage then holds finite stale
  // data) while tile j's weights are formed, then tile j's P V.  `edge` false:
  // tiles j and j+1 lie wholly in the prefix (no mask).
  auto compute = [&](int j, const uint8_t* k_nxt, const uint8_t* v_cur, bool edge,
                     f32x16(&x)[2], f32x16(&s)[2]) __attribute__((always_inline)) {
    u32x4 pf[4];
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
      // tile j+1's scores were started from the old -m_run
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) s[blk] -= d;
      negm = -m_run;
    }
    l_run += lsum;
    if (edge) mask(tile0(j + 1), s);
    accumulate(v_cur, pf);
    interleave_pv();
  };

  // fp8 staging of iteration j (after the barrier): dequantise K_{j+2} (into
  // K_j's stage) and V_{j+1} (into V_{j-1}'s) from registers, then load the
  // codes and page scales of K_{j+3} and V_{j+2}
  auto stage8 = [&](int j, uint8_t* k_cur, uint8_t* v_nxt,
                    bool all_prefix) __attribute__((always_inline)) {
    // all_prefix: tiles j .. j+3 lie wholly in the cached prefix
    if (all_prefix || j + 2 < n_tiles) store8(tile0(j + 2), k8, k_cur, true, sk8, all_prefix);
    if (all_prefix || j + 1 < n_tiles) store8(tile0(j + 1), v8, v_nxt, false, sv8, all_prefix);
    const int pg3 = pg_raw;
    if (all_prefix || j + 3 < n_tiles) {
      k8 = load8(tile0(j + 3), pg3, k_pool, true, all_prefix);
      sk8 = load_scale(ks_s, tile0(j + 3), pg3);
    }
    if (all_prefix || j + 2 < n_tiles) {
      v8 = load8(tile0(j + 2), pg_v, v_pool, false, all_prefix);
      sv8 = load_scale(vs_s, tile0(j + 2), pg_v);
    }
    pg_v = pg3;
    pg_raw = load_page(tile0(j + 4));  // an in-range entry whenever it is a prefix page
  };

  // iteration j: K_{j+1} and V_j are resident; K_{j+2} goes to K_j's stage,
  // V_{j+1} to V_{j-1}'s
  auto iteration = [&](int j, uint8_t* k_cur, uint8_t* k_nxt, uint8_t* v_cur, uint8_t* v_nxt,
                       f32x16(&x)[2], f32x16(&xn)[2]) __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's staging of K_{j+1} and V_j has landed
    if constexpr (FP8) {
      // its DMA'd new-token rows of K_{j+1} and V_j become fp16 before the barrier
      if (j + 1 < n_tiles) convert_new(tile0(j + 1), k_nxt);
      convert_new(tile0(j), v_cur);
    }
    __syncthreads();                // everyone's has; K_j and V_{j-1} are no longer read
    if constexpr (!FP8) {
      const int pg_k = pg_raw;
      if (j + 2 < n_tiles) issue(tile0(j + 2), k_cur, pg_k, k_pool, k_new, k_off);
      if (j + 1 < n_tiles) issue(tile0(j + 1), v_nxt, pg_v, v_pool, v_new, v_off);
      pg_v = pg_k;
      if (j + 3 < n_tiles) pg_raw = load_page(tile0(j + 3));
    } else {
      if (j + 2 < n_tiles) issue(tile0(j + 2), k_cur, 0, k_pool, k_new, k_off);
      if (j + 1 < n_tiles) issue(tile0(j + 1), v_nxt, 0, v_pool, v_new, v_off);
      stage8(j, k_cur, v_nxt, false);
    }
    if (!visible(j)) return;  // nothing visible for this wave from here on
    compute(j, k_nxt, v_cur, true, x, xn);
  };

  // Iterations whose staged tiles lie wholly in the cached prefix (bf16: tiles
  // j .. j+2; fp8: j .. j+3): every row sees all their keys (no mask) and
  // their rows come from one pool page per wave, so the loop carries no
  // per-tile mode decisions.
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
  auto steady = [&](int j, uint8_t* k_cur, uint8_t* k_nxt, uint8_t* v_cur, uint8_t* v_nxt,
                    f32x16(&x)[2], f32x16(&xn)[2]) __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if constexpr (!FP8) {
      const int pg_k = pg_raw;
      issue_prefix(k_cur, pg_k, k_pool_kvh, k_off);
      issue_prefix(v_nxt, pg_v, v_pool_kvh, v_off);
      pg_v = pg_k;
      pg_raw = load_page(tile0(j + 3));  // an in-range entry whenever it is a prefix page
    } else {
      stage8(j, k_cur, v_nxt, true);
    }
    if (wave_active) compute(j, k_nxt, v_cur, false, x, xn);
  };

  const int n_prefix = lp > it.kv_begin ? min(n_tiles, (lp - it.kv_begin) / BLOCK_N) : 0;
  const int n_steady = max(0, n_prefix - (FP8 ? 3 : 2));
  int j = 0;
  for (; j + 1 < n_steady; j += 2) {
    steady(j, lds_k0, lds_k1, lds_v0, lds_v1, xa, xb);
    steady(j + 1, lds_k1, lds_k0, lds_v1, lds_v0, xb, xa);
  }
  if (j < n_steady) {
    steady(j, lds_k0, lds_k1, lds_v0, lds_v1, xa, xb);
    ++j;
  }
  if ((j & 1) && j < n_tiles) {
    iteration(j, lds_k1, lds_k0, lds_v1, lds_v0, xb, xa);
    ++j;
  }
  for (; j < n_tiles; j += 2) {
    iteration(j, lds_k0, lds_k1, lds_v0, lds_v1, xa, xb);
    if (j + 1 < n_tiles) iteration(j + 1, lds_k1, lds_k0, lds_v1, lds_v0, xb, xa);
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
    // the unnormalised partial O in bf16 (relative rounding 2^-9, the range of fp32)
    uint16_t* po = p.part_o + (size_t(it.part) * p.part_rows + r_local) * D;
#pragma unroll
    for (int b = 0; b < T::DB; ++b) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = 32 * b + 8 * q4 + 4 * h;
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = static_cast<__bf16>(o[b][4 * q4 + e]);
        *reinterpret_cast<u32x2*>(po + d) = __builtin_bit_cast(u32x2, v4);
      }
    }
    if (h == 0) {
      float* ml = p.part_ml + (size_t(it.part) * p.part_rows + r_local) * 2;
      ml[0] = m_run;
      ml[1] = l_tot;
    }
  }
}

template <int D, int P, bool FP8>
hipError_t launch_t(const ExtendParams& p, hipStream_t stream, const ArgPlan* ap) {
  if (ap != nullptr)
    hipLaunchKernelGGL((extend_lds_kernel<D, P, FP8, true>), dim3(p.n_items), dim3(LDS_THREADS), 0, stream, p, *ap);
  else
    hipLaunchKernelGGL((extend_lds_kernel<D, P, FP8, false>), dim3(p.n_items), dim3(LDS_THREADS), 0, stream, p,
                       NoArgPlan{});
  return hipGetLastError();
}

}  // namespace

hipError_t launch_extend_lds(const ExtendParams& p, int head_dim, int page_size, bool fp8,
                             hipStream_t stream, const ArgPlan* ap) {
  if (p.n_items <= 0) return hipSuccess;
#define CW_LDS_CASE(D_, P_)                                                        \
  if (head_dim == D_ && page_size == P_)                                           \
    return fp8 ? launch_t<D_, P_, true>(p, stream, ap) : launch_t<D_, P_, false>(p, stream, ap);
  CW_LDS_CASE(64, 16)
  CW_LDS_CASE(64, 64)
  CW_LDS_CASE(128, 16)
  CW_LDS_CASE(128, 64)
#undef CW_LDS_CASE
  return hipErrorInvalidValue;
}

}  // namespace cw
