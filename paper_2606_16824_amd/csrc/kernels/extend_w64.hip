// Prefix-cached paged extend attention, 64 query rows per wave.
//
// A workgroup is four wave64s, one per SIMD, owning the same 256 packed query
// rows (row = token * G + group member) of one (sequence, kv head) as the
// eight-wave kernel, but each wave holds 64 rows as two 32-row blocks.  Every
// K fragment read from LDS feeds the score MFMAs of both row blocks, and every
// V^T fragment the P V MFMAs of both, so LDS read bytes per MFMA are half those
// of a 32-row wave: per 32 keys a wave issues 8 ds_read_b128 (K) and 16
// ds_read_b64_tr_b16 (V^T) for 32 MFMAs.
//
// Registers (D = 128): O^T is 2 x 4 accumulators of 16 fp32 (128 per lane),
// Q 2 x 8 bf16x8 (64), scores of two 32-key steps 2 x 32, P 16, the -m splats
// of the score MFMAs' start 32.  One wave per SIMD leaves 512 registers per
// lane; the P V accumulators live in the accumulation registers.
//
// Keys are staged through LDS 32 at a time and consumed 32 at a time, one
// barrier per step.  Step n computes the scores of keys 32 (n + 1) .. + 31 with
// the MFMAs while the same wave forms the weights of step n's keys (exp2, bf16
// pack, row sums), then accumulates step n's P V.  K and V rotate through
// three LDS stages each (48 KiB at D = 128, so every fragment address is a
// register plus an immediate offset): at the start of step n a wave issues the
// DMA of K_{n+3} and V_{n+2}, two steps before their first use.
//
// The softmax keeps the running max lazily as the eight-wave kernel does: Q
// carries the softmax scale in log2 units, the first score MFMA of a step
// starts from -m, and m is raised only when a half-row weight sum of a step
// passes 2^16 or is not finite.
//
// LDS layout, DMA staging and the fragment swizzles are those of the
// eight-wave kernel: K row R, chunk c at position c ^ k_swz(R); V row R, chunk c
// at c ^ v_swz(R); the DMA writes lane l's 16 bytes at base + 16 l.  Each wave
// stages 8 consecutive rows of a tile, which lie in one page.
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

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(4))) const int32_t const_i32;

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
static_assert(kWaves * 64 == LDS_BLOCK_M, "four waves of 64 rows cover a work item");
constexpr float kNegBig = -1.0e30f;
constexpr float kLn2 = 0.69314718055994531f;
constexpr float kSumLimit = 65536.f;
constexpr uint32_t kOnePair = 0x3F803F80u;  // bf16 pair (1, 1)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_at(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, -1, 0x00020000);
}

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, lds_void* dst, uint32_t voff,
                                      uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, soff, 0, 0);
}

// O^T += V^T P^T with the accumulator in accumulation registers.  Written as
// inline assembly so that the register allocator keeps the 64-row O^T (128
// registers at D = 128) out of the architectural VGPRs.  The compiler does not
// see an MFMA here, so the wait states it would insert are the kernel's job: a
// vector instruction that writes an operand needs two wait states before the
// MFMA (mfma_guard, at the start of every P V phase: inside one, no vector
// instruction writes an operand of these MFMAs), and reads of O^T wait in
// drain_acc after the last accumulation.
__device__ __forceinline__ void mfma_acc(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
__device__ __forceinline__ void mfma_guard() { asm volatile("s_nop 1"); }
template <int DB>
__device__ __forceinline__ void drain_acc(f32x16 (&o)[2][DB]) {
  if constexpr (DB == 4)
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+a"(o[0][0]), "+a"(o[0][1]), "+a"(o[0][2]), "+a"(o[0][3]), "+a"(o[1][0]),
                   "+a"(o[1][1]), "+a"(o[1][2]), "+a"(o[1][3]));
  else
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+a"(o[0][0]), "+a"(o[0][1]), "+a"(o[1][0]), "+a"(o[1][1]));
}

__device__ __forceinline__ int swap_bits_2_3(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

template <int D>
__device__ __forceinline__ int k_swz(int row) {
  return D == 128 ? (swap_bits_2_3(row) & 15) : ((swap_bits_2_3(row) >> 1) & 7);
}
template <int D>
__device__ __forceinline__ int v_swz(int row) {
  return D == 128 ? 4 * (row & 3) : 4 * ((row >> 1) & 1);
}

constexpr int kTileN = 32;  // keys per LDS tile and per step

template <int D, int P>
struct WGeo {
  static constexpr int RB = 2 * D;                   // bytes per bf16 row in LDS
  static constexpr int CPR = D / 8;                  // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;               // rows per wave DMA instruction
  static constexpr int WROWS = kTileN / kWaves;      // rows each wave stages per tile
  static constexpr int NI = WROWS / RPI;             // DMA instructions per wave per matrix
  static constexpr int TILE = kTileN * RB;           // bytes of one K (or V) tile
  static constexpr int KT = D / 16;                  // k-steps of K Q^T
  static constexpr int DB = D / 32;                  // 32-row blocks of O^T
  static_assert(NI * RPI == WROWS, "each wave stages 8 rows of a tile");
  static_assert(P % WROWS == 0, "a wave's rows of a tile lie in one page");
  static_assert(BLOCK_N % kTileN == 0, "work items start on a tile");
};

template <int D, int P, bool AP>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void extend_w64_kernel(ExtendParams p, PlanArg<AP> ap) {
  using T = WGeo<D, P>;
  // each stage its own array, so the compiler can tell that fragment reads of
  // one stage never alias the DMA in flight into another
  __shared__ __attribute__((aligned(1024))) uint8_t lds_k0[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_k1[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_k2[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_v0[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_v1[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_v2[T::TILE];

  auto fused_write = [&]() __attribute__((always_inline)) {
    WriteParams w = p.w;
    w.seqs = plan_ptr<AP>(ap, p.ap_wseqs, p.w.seqs);
    const int64_t total = int64_t(w.total_tokens) * w.num_kv_heads * (D / 8);
    const int64_t per = (total + gridDim.x - 1) / gridDim.x;
    const int64_t end = min(total, int64_t(blockIdx.x + 1) * per);
    for (int64_t idx = int64_t(blockIdx.x) * per + threadIdx.x; idx < end; idx += kThreads)
      pw::write_piece<D, P, false>(w, idx);
  };

  const WorkItem it = plan_ptr<AP>(ap, p.ap_items, p.items)[blockIdx.x];
  if (it.seq < 0) {
    if (p.w.total_tokens > 0) fused_write();
    return;
  }
  const SeqInfo sq = plan_ptr<AP>(ap, p.ap_seqs, p.seqs)[it.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, col = lane & 31;
  const int G = p.gqa_group, hkv = p.num_kv_heads, hq = hkv * G;
  const int kvh = it.kvh;
  const int lp = sq.lp, total_len = sq.lp + sq.ls;
  const int32_t* bt = p.block_table + size_t(sq.bt_row) * p.bt_stride;
  const uint8_t* k_pool = static_cast<const uint8_t*>(p.k_pool);
  const uint8_t* v_pool = static_cast<const uint8_t*>(p.v_pool);
  const uint8_t* k_new = static_cast<const uint8_t*>(p.k_new);
  const uint8_t* v_new = static_cast<const uint8_t*>(p.v_new);

  // this lane's two query rows (row block rb = 0, 1) and their causal limits
  int r_local[2], tok[2], grp[2], lim[2];
  bool row_ok[2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    r_local[rb] = wave * 64 + rb * 32 + col;
    row_ok[rb] = r_local[rb] < it.rows;
    const int r = it.q_row0 + r_local[rb];
    tok[rb] = r / G;
    grp[rb] = r - tok[rb] * G;
    lim[rb] = row_ok[rb] ? lp + tok[rb] + 1 : 0x7FFFFFFF;
  }
  const bool wave_active = wave * 64 < it.rows;
  const int wave_min_lim = lp + (it.q_row0 + wave * 64) / G + 1;
  const int wave_last_row = it.q_row0 + min(wave * 64 + 63, it.rows - 1);
  const int wave_max_lim = lp + wave_last_row / G + 1;

  for (int i = tid; i < T::TILE / 16; i += kThreads) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    reinterpret_cast<u32x4*>(lds_k0)[i] = z;
    reinterpret_cast<u32x4*>(lds_k1)[i] = z;
    reinterpret_cast<u32x4*>(lds_k2)[i] = z;
    reinterpret_cast<u32x4*>(lds_v0)[i] = z;
    reinterpret_cast<u32x4*>(lds_v1)[i] = z;
    reinterpret_cast<u32x4*>(lds_v2)[i] = z;
  }

  // Q^T (B operand), scaled by the softmax scale in log2 units and rounded to
  // bf16: k-step kk of row block rb holds dims 16 kk + 8 h + [0, 8).
  const float c = p.scale_log2;
  bf16x8 qf[2][T::KT];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const uint16_t* qrow = static_cast<const uint16_t*>(p.q) +
                           (size_t(sq.cu + tok[rb]) * hq + size_t(kvh) * G + grp[rb]) * D;
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row_ok[rb]) v = *reinterpret_cast<const u32x4*>(qrow + 16 * kk + 8 * h);
      qf[rb][kk] = __builtin_bit_cast(bf16x8, v);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        qf[rb][kk][e] = static_cast<__bf16>(static_cast<float>(qf[rb][kk][e]) * c);
      // Q^T lives in accumulation registers (the score MFMAs read it there)
      asm volatile("" : "+a"(qf[rb][kk]));
    }
  }

  // ---- staging geometry: wave w stages tile rows [8 w, 8 w + 8); DMA
  // instruction j covers rows 8 w + RPI j .. + RPI - 1, lane l fetches row
  // + l / CPR into position l % CPR.
  const int dma_row = lane / T::CPR, dma_pos = lane % T::CPR;
  const int wrow0 = T::WROWS * wave;
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
  const size_t page_bytes = size_t(P) * T::RB;

  // k_off / v_off hold row R's slot as R % P; a tile whose first key is not on
  // a page boundary (P = 64: every other tile) adds its first key's slot
  auto page_slot_bytes = [&](int j0) -> uint32_t { return uint32_t((j0 % P) * T::RB); };
  const_i32* bt_s = (const_i32*)bt;
  auto load_page = [&](int j0) -> int { return (j0 + wrow0 < lp) ? bt_s[(j0 + wrow0) / P] : 0; };

  // DMA of one matrix of the tile at j0: prefix rows from pool page `pg`,
  // suffix rows from the new tokens, rows past the sequence left as they are.
  auto issue = [&](int j0, uint8_t* dst, int pg, const uint8_t* pool, const uint8_t* fresh,
                   const uint32_t(&off)[T::NI]) __attribute__((always_inline)) {
    const int k_first = j0 + wrow0, k_last = k_first + T::WROWS - 1;
    if (k_first < lp) {
      const auto rs = rsrc_at(pool + (size_t(pg) * hkv + kvh) * page_bytes);
      const uint32_t slot0 = page_slot_bytes(j0);
      if (k_last < lp) {
#pragma unroll
        for (int j = 0; j < T::NI; ++j)
          dma16(rs, (lds_void*)(dst + (wrow0 + T::RPI * j) * T::RB), off[j], slot0);
      } else {
#pragma unroll
        for (int j = 0; j < T::NI; ++j)
          if (k_first + T::RPI * j + dma_row < lp)
            dma16(rs, (lds_void*)(dst + (wrow0 + T::RPI * j) * T::RB), off[j], slot0);
      }
    }
    if (k_last >= lp && k_first < total_len) {
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

  // ---- fragment addresses within a stage
  uint32_t k_addr[T::KT];
  {
    const int R = swap_bits_2_3(col);
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) k_addr[kk] = R * T::RB + 16 * ((2 * kk + h) ^ k_swz<D>(R));
  }
  uint32_t v_addr[T::DB];
  {
    const int g4 = lane >> 4, ri = lane & 15;
    const int kq = ri >> 2, a = ri & 3;
#pragma unroll
    for (int b = 0; b < T::DB; ++b) {
      const int chunk = 4 * b + 2 * (g4 & 1) + (a >> 1);
      v_addr[b] = (8 * h + kq) * T::RB + 16 * (chunk ^ v_swz<D>(kq)) + 8 * (a & 1);
    }
  }

  f32x16 o[2][T::DB];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int b = 0; b < T::DB; ++b) o[rb][b] = f32x16{};
  float m_run[2] = {kNegBig, kNegBig}, l_run[2] = {0.f, 0.f};
  f32x16 negm[2] = {f32x16{}, f32x16{}};

  const int n_keys = it.kv_end - it.kv_begin;
  const int n_tiles = (n_keys + kTileN - 1) / kTileN;
  auto key0 = [&](int n) { return it.kv_begin + kTileN * n; };
  auto visible = [&](int n) { return wave_active && n < n_tiles && key0(n) < wave_max_lim; };

  auto read_k = [&](const uint8_t* ks, int kk) -> bf16x8 {
    return *reinterpret_cast<const bf16x8*>(ks + k_addr[kk]);
  };
  // V^T fragment of 16-key slice u, 32-dim block b
  auto read_v = [&](const uint8_t* vs, int u, int b) -> bf16x8 {
    i16x4 half[2];
#pragma unroll
    for (int e4 = 0; e4 < 2; ++e4)
      half[e4] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vs + v_addr[b] + (16 * u + 4 * e4) * T::RB));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(half[0], half[1], 0, 1, 2, 3, 4, 5, 6, 7));
  };
  // scores S^T = K Q^T - m of the 32 keys at `ks`, both row blocks
  auto scores = [&](const uint8_t* ks, f32x16(&s)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      const bf16x8 kf = read_k(ks, kk);
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[0][kk], kk > 0 ? s[0] : negm[0], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[1][kk], kk > 0 ? s[1] : negm[1], 0, 0, 0);
    }
  };
  // causal mask of the 32 keys at k0: element i holds key k0 + 16 (i / 8) + 8 h + i % 8
  auto mask = [&](int k0, f32x16(&s)[2]) __attribute__((always_inline)) {
    if (k0 + kTileN > wave_min_lim) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (k0 + 16 * (i >> 3) + 8 * h + (i & 7) >= lim[rb]) s[rb][i] = -INFINITY;
    }
  };
  // bf16 weights of 16-key slice u of row block rb (B-operand order) and the
  // half-row sums of the rounded weights
  auto weights = [&](const f32x16(&x)[2], bf16x8(&pf)[2][2], float(&lsum)[2]) __attribute__((always_inline)) {
    const bf16x2 one = __builtin_bit_cast(bf16x2, kOnePair);
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pf[rb][u][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(x[rb][8 * u + e]));
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      float la = 0.f, lb = 0.f;
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 8; e += 4) {
          la = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pf[rb][u][e], pf[rb][u][e + 1]}, one, la, false);
          lb = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pf[rb][u][e + 2], pf[rb][u][e + 3]}, one, lb, false);
        }
      lsum[rb] = la + lb;
    }
  };
  auto row_max = [&](const f32x16& x) -> float {
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, x[i]);
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                     false, false);
    return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
  };

  // A tile's 32 weights per lane are formed in two halves so that both phases
  // of a step carry vector work (one wave per SIMD: nothing else fills the
  // issue slots the MFMAs leave): the first 16-key slice of each row block
  // during the previous step's P V MFMAs, the second slice during the step's
  // own score MFMAs.  pf holds the weights of the current tile, la / lb the
  // partial row sums of its first slice.
  bf16x8 pf[2][2];  // [row block][16-key slice]
  float la[2] = {0.f, 0.f}, lb[2] = {0.f, 0.f};
  const bf16x2 one = __builtin_bit_cast(bf16x2, kOnePair);
  // weights 2 q, 2 q + 1 of slice u of row block rb from scores x (q < 4),
  // added to the partial sums
  auto weight_pair = [&](const f32x16(&x)[2], int rb, int u, int q, bf16x8(&w)[2][2], float(&sa)[2],
                         float(&sb)[2]) __attribute__((always_inline)) {
    const int e = 2 * q, i = 8 * u + e;
    bf16x2 pr = bf16x2{static_cast<__bf16>(__builtin_amdgcn_exp2f(x[rb][i])),
                       static_cast<__bf16>(__builtin_amdgcn_exp2f(x[rb][i + 1]))};
    // pins the pair here: IR passes would otherwise sink it to its first use,
    // past the scheduling barriers that place it between MFMAs
    asm volatile("" : "+v"(pr));
    w[rb][u][e] = pr[0];
    w[rb][u][e + 1] = pr[1];
    if (q & 1) sb[rb] = __builtin_amdgcn_fdot2_f32_bf16(pr, one, sb[rb], false);
    else sa[rb] = __builtin_amdgcn_fdot2_f32_bf16(pr, one, sa[rb], false);
  };
  // pair index t in [0, 8): row block t / 4, weights 2 (t % 4), + 1 of slice u
  auto weight_pair_t = [&](const f32x16(&x)[2], int u, int t, bf16x8(&w)[2][2], float(&sa)[2],
                           float(&sb)[2]) __attribute__((always_inline)) {
    weight_pair(x, t >> 2, u, t & 3, w, sa, sb);
  };

  // step n: scores of tile n + 1 (keys at k_next) while the second half of
  // tile n's weights is formed, then tile n's P V (values at v_cur) while the
  // first half of tile n + 1's weights is formed.  x holds tile n's scores, s
  // receives tile n + 1's.
  //
  // Both phases are written as chunks separated by scheduling barriers, one
  // MFMA each, so the instruction order is the one below.  Score phase: first
  // the reads of the first kLead K fragments with kLeadPairs weight pairs
  // (which need no fresh LDS data and cover the reads' latency), then per chunk
  // one MFMA, its share of weight pairs and a fragment read (the remaining K
  // k-steps, then the first V^T slice, which the P V MFMAs need first).  P V
  // phase: per chunk one MFMA (inline assembly), its share of tile n + 1's
  // first-half weight pairs and, for the first slice, the reads of the second.
  constexpr int kLead = 3;
  constexpr int kLeadPairs = 2;
  constexpr int kChunks = 2 * T::KT;                      // score MFMAs per step
  constexpr int kPvChunks = 4 * T::DB;                    // P V MFMAs per step
  constexpr int kVReadChunk0 = kChunks - 2 * T::DB;       // first chunk reading the V^T slice
  auto step = [&](int n, const uint8_t* k_next, const uint8_t* v_cur, bool edge, f32x16(&x)[2],
                  f32x16(&s)[2]) __attribute__((always_inline)) {
    bf16x8 kf[T::KT];
    bf16x8 v0[T::DB], v1[T::DB];
    i16x4 v0h[T::DB][2];
#pragma unroll
    for (int kk = 0; kk < kLead; ++kk) kf[kk] = read_k(k_next, kk);
    // second-slice pairs t = 0 .. 7 of tile n, spread over the lead and the chunks
#pragma unroll
    for (int t = 0; t < kLeadPairs; ++t) weight_pair_t(x, 1, t, pf, la, lb);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const int kk = c >> 1, rb = c & 1;
      s[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[rb][kk], kk > 0 ? s[rb] : negm[rb], 0, 0, 0);
      // pairs kLeadPairs .. 7 over the chunks, evenly
      const int t0 = kLeadPairs + (c * (8 - kLeadPairs)) / kChunks;
      const int t1 = kLeadPairs + ((c + 1) * (8 - kLeadPairs)) / kChunks;
#pragma unroll
      for (int t = t0; t < t1; ++t) weight_pair_t(x, 1, t, pf, la, lb);
      if (rb == 0 && kk + kLead < T::KT) kf[kk + kLead] = read_k(k_next, kk + kLead);
      if (c >= kVReadChunk0) {
        const int r = c - kVReadChunk0, b = r >> 1, e4 = r & 1;
        v0h[b][e4] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4*)(v_cur + v_addr[b] + (4 * e4) * T::RB));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int b = 0; b < T::DB; ++b)
      v0[b] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0h[b][0], v0h[b][1], 0, 1, 2, 3, 4, 5, 6, 7));
    float lsum[2] = {la[0] + lb[0], la[1] + lb[1]};
    if (__any(!(lsum[0] <= kSumLimit) || !(lsum[1] <= kSumLimit))) {
      drain_acc<T::DB>(o);
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const float d = fmaxf(row_max(x[rb]), 0.f);
        m_run[rb] += d;
        const float alpha = __builtin_amdgcn_exp2f(-d);
        l_run[rb] *= alpha;
        // one accumulator at a time, so that the copies through the
        // architectural registers never hold more than 16 of them
#pragma unroll
        for (int b = 0; b < T::DB; ++b) {
          __builtin_amdgcn_sched_barrier(0);
          o[rb][b] *= alpha;
        }
        __builtin_amdgcn_sched_barrier(0);
        x[rb] -= d;
        s[rb] -= d;
        negm[rb] = -m_run[rb];
      }
      weights(x, pf, lsum);
    }
    l_run[0] += lsum[0];
    l_run[1] += lsum[1];
    // tile n + 1's scores are complete: mask them, then form their first slice
    // during the P V MFMAs
    if (edge) mask(key0(n + 1), s);
    bf16x8 pn[2][2];
    float na[2] = {0.f, 0.f}, nb[2] = {0.f, 0.f};
    __builtin_amdgcn_sched_barrier(0);
    mfma_guard();
#pragma unroll
    for (int c = 0; c < kPvChunks; ++c) {
      const int u = c / (2 * T::DB), b = (c >> 1) % T::DB, rb = c & 1;
      mfma_acc(o[rb][b], u == 0 ? v0[b] : v1[b], pf[rb][u]);
      const int t0 = (c * 8) / kPvChunks, t1 = ((c + 1) * 8) / kPvChunks;
#pragma unroll
      for (int t = t0; t < t1; ++t) weight_pair_t(s, 0, t, pn, na, nb);
      if (u == 0 && rb == 1) v1[b] = read_v(v_cur, 1, b);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      pf[rb][0] = pn[rb][0];
      la[rb] = na[rb];
      lb[rb] = nb[rb];
    }
  };
  // the first slice of a tile's weights from its scores x (before its step)
  auto first_slice = [&](const f32x16(&x)[2]) __attribute__((always_inline)) {
    la[0] = la[1] = lb[0] = lb[1] = 0.f;
#pragma unroll
    for (int t = 0; t < 8; ++t) weight_pair_t(x, 0, t, pf, la, lb);
  };

  f32x16 xa[2] = {f32x16{}, f32x16{}}, xb[2] = {f32x16{}, f32x16{}};
  int pg_k = 0;  // page of K_{n+3}
  int pg_v = 0;  // page of V_{n+2}
  __syncthreads();
  if (n_tiles > 0) {
    // K_0, K_1, K_2 and V_0, V_1 ahead of the first step
    const int pg0 = load_page(key0(0));
    const int pg1 = n_tiles > 1 ? load_page(key0(1)) : 0;
    const int pg2 = n_tiles > 2 ? load_page(key0(2)) : 0;
    issue(key0(0), lds_k0, pg0, k_pool, k_new, k_off);
    issue(key0(0), lds_v0, pg0, v_pool, v_new, v_off);
    if (n_tiles > 1) issue(key0(1), lds_k1, pg1, k_pool, k_new, k_off);
    if (n_tiles > 1) issue(key0(1), lds_v1, pg1, v_pool, v_new, v_off);
    if (n_tiles > 2) issue(key0(2), lds_k2, pg2, k_pool, k_new, k_off);
    pg_v = pg2;
    if (n_tiles > 3) pg_k = load_page(key0(3));
    if (p.w.total_tokens > 0) fused_write();
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (visible(0)) {
      scores(lds_k0, xa);  // negm is 0: raw scores in log2 units
      mask(key0(0), xa);
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const float mx = row_max(xa[rb]);
        // a row with no visible key among the item's first 32 sees none in the item
        const float d = mx == -INFINITY ? 0.f : mx;
        m_run[rb] = mx == -INFINITY ? kNegBig : mx;
        xa[rb] -= d;
        negm[rb] = -m_run[rb];
      }
      first_slice(xa);
    }
  } else if (p.w.total_tokens > 0) {
    fused_write();
  }

  // Step n: K_{n+1} (in kn1) and V_n (in vn) are resident; K_{n+3} goes to kn3
  // (K_n's stage) and V_{n+2} to vn2 (V_{n-1}'s).  Steady: tiles n .. n + 3 lie
  // wholly in the cached prefix (one page per wave, every row sees every key,
  // no mask) and each step issues exactly 2 NI DMA instructions, so the wait
  // before the barrier leaves the previous step's DMA in flight.
  auto iteration = [&](int n, const uint8_t* kn1, uint8_t* kn3, const uint8_t* vn, uint8_t* vn2,
                       bool steady, f32x16(&x)[2], f32x16(&s)[2]) __attribute__((always_inline)) {
    if (steady) {
      // vmcnt <= 2 NI: everything but the previous step's DMA has landed;
      // lgkmcnt 0: the page id loaded at the end of the last step has arrived
      // (nothing else is outstanding there)
      __builtin_amdgcn_s_waitcnt((2 * T::NI) | (0x7 << 4));
    } else {
      __builtin_amdgcn_s_waitcnt(0);
    }
    // everyone's K_{n+1} and V_n have landed; K_n and V_{n-1} are free.  The
    // empty asm statements keep the compiler from moving memory accesses across
    // the barrier (a fence here would also wait for the DMA still in flight).
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    const int pk = pg_k, pv = pg_v;
    if (steady) {
      const auto rk = rsrc_at(k_pool + (size_t(pk) * hkv + kvh) * page_bytes);
      const auto rv = rsrc_at(v_pool + (size_t(pv) * hkv + kvh) * page_bytes);
      const uint32_t sk = page_slot_bytes(key0(n + 3)), sv = page_slot_bytes(key0(n + 2));
#pragma unroll
      for (int i = 0; i < T::NI; ++i) dma16(rk, (lds_void*)(kn3 + (wrow0 + T::RPI * i) * T::RB), k_off[i], sk);
#pragma unroll
      for (int i = 0; i < T::NI; ++i) dma16(rv, (lds_void*)(vn2 + (wrow0 + T::RPI * i) * T::RB), v_off[i], sv);
      pg_v = pk;
      // the next page id is loaded after the step's fragment reads, so that no
      // scalar load (whose counter shares lgkmcnt with LDS reads and completes
      // out of order) makes the step's LDS waits conservative
      if (wave_active) step(n, kn1, vn, false, x, s);
      pg_k = load_page(key0(n + 4));  // an in-range entry whenever it is a prefix page
    } else {
      if (n + 3 < n_tiles) issue(key0(n + 3), kn3, pk, k_pool, k_new, k_off);
      if (n + 2 < n_tiles) issue(key0(n + 2), vn2, pv, v_pool, v_new, v_off);
      pg_v = pk;
      if (visible(n)) step(n, kn1, vn, true, x, s);
      if (n + 4 < n_tiles) pg_k = load_page(key0(n + 4));
    }
  };

  // Stage indices have period 3 and the score registers alternate with period
  // 2, so the loops run six steps per trip.
  const int n_prefix = lp > it.kv_begin ? min(n_tiles, (lp - it.kv_begin) / kTileN) : 0;
  const int n_steady = max(0, n_prefix - 3);
  int n = 0;
  for (; n + 6 <= n_steady; n += 6) {
    iteration(n, lds_k1, lds_k0, lds_v0, lds_v2, true, xa, xb);
    iteration(n + 1, lds_k2, lds_k1, lds_v1, lds_v0, true, xb, xa);
    iteration(n + 2, lds_k0, lds_k2, lds_v2, lds_v1, true, xa, xb);
    iteration(n + 3, lds_k1, lds_k0, lds_v0, lds_v2, true, xb, xa);
    iteration(n + 4, lds_k2, lds_k1, lds_v1, lds_v0, true, xa, xb);
    iteration(n + 5, lds_k0, lds_k2, lds_v2, lds_v1, true, xb, xa);
  }
  // the steady loop leaves n a multiple of six, so stage indices stay compile-time
  for (; n < n_tiles; n += 6) {
    iteration(n, lds_k1, lds_k0, lds_v0, lds_v2, false, xa, xb);
    if (n + 1 < n_tiles) iteration(n + 1, lds_k2, lds_k1, lds_v1, lds_v0, false, xb, xa);
    if (n + 2 < n_tiles) iteration(n + 2, lds_k0, lds_k2, lds_v2, lds_v1, false, xa, xb);
    if (n + 3 < n_tiles) iteration(n + 3, lds_k1, lds_k0, lds_v0, lds_v2, false, xb, xa);
    if (n + 4 < n_tiles) iteration(n + 4, lds_k2, lds_k1, lds_v1, lds_v0, false, xa, xb);
    if (n + 5 < n_tiles) iteration(n + 5, lds_k0, lds_k2, lds_v2, lds_v1, false, xb, xa);
  }

  if (!wave_active) return;
  drain_acc<T::DB>(o);
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const float l_tot = l_run[rb] + __shfl_xor(l_run[rb], 32);
    if (it.part < 0) {
      if (!row_ok[rb]) continue;
      const float inv = 1.f / l_tot;
      const size_t orow_idx = size_t(sq.cu + tok[rb]) * hq + size_t(kvh) * G + grp[rb];
      uint16_t* orow = static_cast<uint16_t*>(p.out) + orow_idx * D;
#pragma unroll
      for (int b = 0; b < T::DB; ++b) {
        __builtin_amdgcn_sched_barrier(0);  // one accumulator at a time
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int d = 32 * b + 8 * q4 + 4 * h;
          bf16x4 v4;
#pragma unroll
          for (int e = 0; e < 4; ++e) v4[e] = static_cast<__bf16>(o[rb][b][4 * q4 + e] * inv);
          *reinterpret_cast<u32x2*>(orow + d) = __builtin_bit_cast(u32x2, v4);
        }
      }
      if (p.lse != nullptr && h == 0) p.lse[orow_idx] = (m_run[rb] + __log2f(l_tot)) * kLn2;
    } else {
      // the unnormalised partial O in bf16
      uint16_t* po = p.part_o + (size_t(it.part) * p.part_rows + r_local[rb]) * D;
#pragma unroll
      for (int b = 0; b < T::DB; ++b) {
        __builtin_amdgcn_sched_barrier(0);  // one accumulator at a time
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int d = 32 * b + 8 * q4 + 4 * h;
          bf16x4 v4;
#pragma unroll
          for (int e = 0; e < 4; ++e) v4[e] = static_cast<__bf16>(o[rb][b][4 * q4 + e]);
          *reinterpret_cast<u32x2*>(po + d) = __builtin_bit_cast(u32x2, v4);
        }
      }
      if (h == 0) {
        float* ml = p.part_ml + (size_t(it.part) * p.part_rows + r_local[rb]) * 2;
        ml[0] = m_run[rb];
        ml[1] = l_tot;
      }
    }
  }
}

template <int D, int P>
hipError_t launch_t(const ExtendParams& p, hipStream_t stream, const ArgPlan* ap) {
  if (ap != nullptr)
    hipLaunchKernelGGL((extend_w64_kernel<D, P, true>), dim3(p.n_items), dim3(kThreads), 0, stream, p, *ap);
  else
    hipLaunchKernelGGL((extend_w64_kernel<D, P, false>), dim3(p.n_items), dim3(kThreads), 0, stream, p,
                       NoArgPlan{});
  return hipGetLastError();
}

}  // namespace

hipError_t launch_extend_w64(const ExtendParams& p, int head_dim, int page_size, hipStream_t stream,
                             const ArgPlan* ap) {
  if (p.n_items <= 0) return hipSuccess;
  if (head_dim == 64 && page_size == 16) return launch_t<64, 16>(p, stream, ap);
  if (head_dim == 64 && page_size == 64) return launch_t<64, 64>(p, stream, ap);
  if (head_dim == 128 && page_size == 16) return launch_t<128, 16>(p, stream, ap);
  if (head_dim == 128 && page_size == 64) return launch_t<128, 64>(p, stream, ap);
  return hipErrorInvalidValue;
}

}  // namespace cw
