// Prefix-cached paged extend attention, bf16 pools: direct-to-LDS staging.
//
// Same work decomposition and math as the register-staged kernel (one
// workgroup = four wave64s = 128 packed query rows of one (sequence, kv head);
// S^T = K Q^T and O^T += V^T P^T with v_mfma_f32_32x32x16_bf16; base-2 online
// softmax with lazy rescaling), but K and V tiles travel from HBM straight into
// LDS with global_load_lds_dwordx4, two stages deep, so staging costs no VGPRs
// and no VALU, and each 64-key tile needs a single barrier.
//
// LDS holds K and V rows in their natural [key][dim] order, 16-byte chunks
// XOR-swizzled per row so that every fragment read is bank-conflict free:
//   K row R, chunk c at position c ^ k_swz(R);  V row R, chunk c at c ^ v_swz(R)
// The DMA writes lane l's 16 bytes at base + 16 l, so each lane simply fetches
// the global chunk that belongs at its position.
//
// V^T operand: ds_read_b64_tr_b16 hands lane i of each 16-lane group element
// in[4k + i/4][i % 4] of the 4-element rows its group's lanes point at.  Lanes
// (k, a) = (i / 4, i % 4) point at key 4k-offset rows and dims 4a .. 4a+3, so
// lane L receives V[keys 4e .. 4e+3 of its 8-key slot][dim 32b + L % 32]: half of
// the A operand of V^T P^T; two reads give all eight keys.
//
// Pages: each wave fetches 16 consecutive key rows of a tile, which lie in one
// page (P = 16 or 64), so a wave needs one page id per tile (a uniform value,
// loaded a tile ahead) and each lane adds an offset that is the same for every
// tile.
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

// 16 bytes per lane from global memory straight into LDS (lane l's bytes land
// at dst + 16 l).  Kept in a non-template function: referenced directly from
// the kernel template, the builtin keeps the host pass from emitting the
// kernel's launch stub.
__device__ __forceinline__ void dma16(const void* src, lds_void* dst) {
  __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
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
  static constexpr int NI = BLOCK_N / RPI / WAVES;    // DMA instructions per wave per matrix
  static constexpr int TILE = BLOCK_N * RB;           // bytes of one K (or V) tile
  static constexpr int NPG = BLOCK_N / P;             // pages per tile
  static constexpr int KT = D / 16;                   // k-steps of K Q^T
  static constexpr int DB = D / 32;                   // 32-row blocks of O^T
};

enum : int { MODE_PREFIX = 0, MODE_SUFFIX = 1, MODE_MIXED = 2 };


template <int D, int P>
__global__ __launch_bounds__(THREADS) void extend_lds_kernel(ExtendParams p) {
  using T = LGeo<D, P>;
  // [stage][K | V][tile]
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * 2 * T::TILE];

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
  for (int i = tid; i < 2 * 2 * T::TILE / 16; i += THREADS)
    reinterpret_cast<u32x4*>(lds)[i] = u32x4{0u, 0u, 0u, 0u};

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

  // DMA geometry: wave w covers tile rows [16 w, 16 w + 16), which lie in one page
  // (its page index in the tile is wq); its instruction j covers rows r0_j ..
  // r0_j + RPI - 1 and lane l fetches row r0_j + l / CPR into position l % CPR
  const int dma_row = lane / T::CPR, dma_pos = lane % T::CPR;
  uint32_t k_lane_off[T::NI], v_lane_off[T::NI];  // within a page (pool) block
  uint32_t kf_lane_off[T::NI], vf_lane_off[T::NI];  // relative to the tile's first new row
#pragma unroll
  for (int j = 0; j < T::NI; ++j) {
    const int R = (wave * T::NI + j) * T::RPI + dma_row;
    const int kc = dma_pos ^ k_swz<D>(R);
    const int vc = dma_pos ^ v_swz<D>(R);
    k_lane_off[j] = (R % P) * T::RB + 16 * kc;
    v_lane_off[j] = (R % P) * T::RB + 16 * vc;
    kf_lane_off[j] = R * hkv * T::RB + 16 * kc;
    vf_lane_off[j] = R * hkv * T::RB + 16 * vc;
  }
  const size_t page_bytes = size_t(P) * T::RB;  // one (page, kv head) block
  const int wq = (wave * T::NI * T::RPI) / P;

  auto mode_of = [&](int j0) {
    if (j0 + BLOCK_N <= lp) return int(MODE_PREFIX);
    if (j0 >= lp && j0 + BLOCK_N <= total_len) return int(MODE_SUFFIX);
    return int(MODE_MIXED);
  };
  // physical page of this wave's rows of the tile at j0 (0 if they hold no prefix key)
  auto load_page = [&](int j0) -> int {
    return (j0 + wq * P < lp) ? __builtin_amdgcn_readfirstlane(bt[j0 / P + wq]) : 0;
  };
  // issue the K and V DMA of the tile at j0 into stage `st`.  Whole-prefix and
  // whole-suffix tiles use a wave-uniform base plus the per-lane offsets;
  // a tile that crosses the prefix end or the sequence end picks per lane.
  auto issue_tile = [&](int j0, int st, int pg) __attribute__((always_inline)) {
    uint8_t* kdst = lds + (2 * st) * T::TILE;
    uint8_t* vdst = lds + (2 * st + 1) * T::TILE;
    const int mode = mode_of(j0);
    if (mode != MODE_MIXED) {
      if (mode == MODE_PREFIX) {
        const size_t base = (size_t(pg) * hkv + kvh) * page_bytes;
#pragma unroll
        for (int j = 0; j < T::NI; ++j) {
          const int r0 = (wave * T::NI + j) * T::RPI;
          dma16(k_pool + base + k_lane_off[j], (lds_void*)(kdst + r0 * T::RB));
          dma16(v_pool + base + v_lane_off[j], (lds_void*)(vdst + r0 * T::RB));
        }
      } else {
        const size_t base = (size_t(sq.cu + j0 - lp) * hkv + kvh) * T::RB;
#pragma unroll
        for (int j = 0; j < T::NI; ++j) {
          const int r0 = (wave * T::NI + j) * T::RPI;
          dma16(k_new + base + kf_lane_off[j], (lds_void*)(kdst + r0 * T::RB));
          dma16(v_new + base + vf_lane_off[j], (lds_void*)(vdst + r0 * T::RB));
        }
      }
      return;
    }
#pragma unroll
    for (int j = 0; j < T::NI; ++j) {
      const int r0 = (wave * T::NI + j) * T::RPI;
      const int key = j0 + r0 + dma_row;
      const uint8_t* ksrc = nullptr;
      const uint8_t* vsrc = nullptr;
      if (key < lp) {
        const size_t base = (size_t(pg) * hkv + kvh) * page_bytes;
        ksrc = k_pool + base + k_lane_off[j];
        vsrc = v_pool + base + v_lane_off[j];
      } else if (key < total_len) {
        // kf/vf offsets hold R * hkv * RB + 16 c; the row is in the base here
        const size_t base = (size_t(sq.cu + key - lp) * hkv + kvh) * T::RB;
        ksrc = k_new + base + (kf_lane_off[j] - (r0 + dma_row) * hkv * T::RB);
        vsrc = v_new + base + (vf_lane_off[j] - (r0 + dma_row) * hkv * T::RB);
      }
      if (ksrc != nullptr) {
        dma16(ksrc, (lds_void*)(kdst + r0 * T::RB));
        dma16(vsrc, (lds_void*)(vdst + r0 * T::RB));
      }
    }
  };

  f32x16 o[T::DB];
#pragma unroll
  for (int b = 0; b < T::DB; ++b) o[b] = f32x16{};
  float m_run = kNegBig, l_run = 0.f;
  const float c = p.scale_log2;

  // page ids of the next tile (prefix keys only), loaded a tile ahead
  int pg_next = 0;

  __syncthreads();  // zero fill done before any DMA lands
  if (it.kv_begin < it.kv_end) {
    issue_tile(it.kv_begin, 0, load_page(it.kv_begin));
    if (it.kv_begin + BLOCK_N < it.kv_end) pg_next = load_page(it.kv_begin + BLOCK_N);
  }

  int st = 0;
  for (int j0 = it.kv_begin; j0 < it.kv_end; j0 += BLOCK_N, st ^= 1) {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's DMA of tile j0 has landed
    __syncthreads();                // everyone's has; stage st^1 is free again
    const int jn = j0 + BLOCK_N;
    if (jn < it.kv_end) {
      issue_tile(jn, st ^ 1, pg_next);
      if (jn + BLOCK_N < it.kv_end) pg_next = load_page(jn + BLOCK_N);
    }

    if (!wave_active || j0 >= wave_max_lim) continue;  // nothing visible for this wave
    const uint8_t* ks = lds + (2 * st) * T::TILE;
    const uint8_t* vs = lds + (2 * st + 1) * T::TILE;

    // S^T = K Q^T for two 32-key blocks (row m of block blk reads key swap(m))
    f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      bf16x8 kf[2];
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) {
        const int R = swap_bits_2_3(col) + 32 * blk;
        const int pos = (2 * kk + h) ^ k_swz<D>(R);
        kf[blk] = *reinterpret_cast<const bf16x8*>(ks + R * T::RB + 16 * pos);
      }
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
        s[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[blk], qf[kk], s[blk], 0, 0, 0);
    }

    // element i of block blk holds key j0 + 32 blk + 16 (i / 8) + 8 h + i % 8
    if (j0 + BLOCK_N > wave_min_lim) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (j0 + 32 * blk + 16 * (i >> 3) + 8 * h + (i & 7) >= lim) s[blk][i] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[blk][i]);
    mx *= c;
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
    const bf16x2 one = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
#pragma unroll
    for (int gi = 0; gi < 4; ++gi) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pf[gi][e] = static_cast<__bf16>(
            __builtin_amdgcn_exp2f(fmaf(s[gi >> 1][8 * (gi & 1) + e], c, -m_run)));
      // row sum of the rounded weights, so numerator and denominator agree
#pragma unroll
      for (int e = 0; e < 8; e += 2)
        l_run = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pf[gi][e], pf[gi][e + 1]}, one, l_run, false);
    }

    // O^T += V^T P^T over four 16-key slices; V^T fragments by transposing reads
    {
      const int grp = lane >> 4, ri = lane & 15;
      const int kq = ri >> 2, a = ri & 3;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        bf16x8 vf[T::DB];
#pragma unroll
        for (int b = 0; b < T::DB; ++b) {
          const int chunk = 4 * b + 2 * (grp & 1) + (a >> 1);
          i16x4 half[2];
#pragma unroll
          for (int e4 = 0; e4 < 2; ++e4) {
            const int R = 16 * u + 8 * h + 4 * e4 + kq;
            const int off = R * T::RB + 16 * (chunk ^ v_swz<D>(R)) + 8 * (a & 1);
            half[e4] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vs + off));
          }
          vf[b] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(half[0], half[1], 0, 1, 2, 3, 4, 5, 6, 7));
        }
#pragma unroll
        for (int b = 0; b < T::DB; ++b)
          o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[b], pf[u], o[b], 0, 0, 0);
      }
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

template <int D, int P>
hipError_t launch_t(const ExtendParams& p, hipStream_t stream) {
  hipLaunchKernelGGL((extend_lds_kernel<D, P>), dim3(p.n_items), dim3(THREADS), 0, stream, p);
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
