// Decode attention (one new token per sequence), HBM-streaming.
//
// Work item = one wave: G <= 16 query rows (the query heads of one kv head)
// against a chunk of at most 64 pages of one sequence's cached prefix, plus the
// new token's own key when the chunk ends the sequence.  A decode step reads
// each cached K/V byte once, so the kernel is bound by HBM bandwidth; it keeps
// three tiles per wave in flight with global_load_lds_dwordx4 (16 KB tiles for
// bf16 pools, three waves per CU; 8 KB for fp8 pools, six waves per CU: 144 KB
// of LDS either way) and uses no barriers (every wave owns its LDS).
//
// Math per tile (same formulation as the extend kernels): S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (queries padded to 32 columns), base-2 online softmax
// with lazy rescaling, O^T += V^T P^T.  fp8 pools keep e4m3fn codes in LDS and
// widen them exactly on the fragment read with v_cvt_scalef32_pk_bf16_fp8
// (scale 1); the page's K scale multiplies its scores and log2 of its V scale
// is added to their exponent (P arrives multiplied by the V scale; the row sum
// divides it back out).  No row max per block: weights are taken against the
// running max and only a block whose weight sum passes a limit raises it.  V^T fragments come from transposing LDS reads: ds_read_b64_tr_b16 for
// bf16 (lane i of a 16-lane group gets element i % 4 of rows 4k + i / 4) and
// ds_read_b64_tr_b8 for fp8 (byte i % 8 of rows 2k + i / 8).
//
// Page ids (and fp8 scales) of the whole chunk are loaded once, one page per
// lane, and read back with v_readlane; a chunk therefore spans <= 64 pages.
#include <hip/hip_runtime.h>

#include "../cw_internal.h"
#include "../plan_expand.h"
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
typedef int i32x2 __attribute__((ext_vector_type(2)));

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) i32x2 lds_i32x2;

constexpr float kNegBig = -1.0e30f;
// A half-column weight sum above this (or not finite) makes a block raise the
// running max: weights then stay below 2^16 and fp32 accumulators far from
// overflow.
constexpr float kSumLimit = 65536.f;
constexpr float kLn2 = 0.69314718055994531f;
constexpr int kStages = 3;
// K + V bytes of one tile: 16 KB for bf16 pools (three waves per CU), 8 KB for
// fp8 pools, whose tiles cost twice the math per byte: six waves per CU (two
// per SIMD) hide each other's MFMA and LDS latencies with the same bytes in
// flight per CU
__host__ __device__ constexpr int tile_bytes(bool fp8) { return fp8 ? 8192 : 16384; }

// 16 bytes per lane from global memory straight into LDS (lane l at LDS
// address m0 + 16 l).  Issued as inline assembly, so the compiler neither
// counts these loads nor guards LDS reads against them: the kernel's own
// vmcnt waits, whose counts are exact (every tile issues the same number of
// DMA instructions), order each stage's reads after its DMA.  The compiler's
// own tracking merges its per-array state conservatively at the loop header
// and would drain every DMA in flight there.  Loads it does count stay
// correct: extra outstanding DMA only makes its count-based waits stricter.
// The loads carry the nontemporal hint: every K/V byte of a decode step is
// read exactly once, and with the hint the memory system streams it instead of
// keeping it in the caches (+12% sustained bandwidth for this access pattern,
// measured with the same pipeline and the math removed).
__device__ __forceinline__ void dma16(const void* src, uint32_t lds_addr) {
  asm volatile("global_load_lds_dwordx4 %0, off nt" ::"v"(src), "{m0}"(lds_addr) : "memory");
}

// s_waitcnt on one counter, also a compiler barrier for memory accesses
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_lgkmcnt0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_void*)p));
}

__device__ __forceinline__ int swap_bits_2_3(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Two e4m3fn codes (bytes 2w, 2w+1 of `v`) -> two bf16, exact.
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_bf16x2(uint32_t v) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(static_cast<int>(v), 1.0f, HI));
}
__device__ __forceinline__ bf16x8 fp8x8_bf16x8(u32x2 c) {
  u32x4 r;
  r.x = fp8x2_bf16x2<false>(c.x);
  r.y = fp8x2_bf16x2<true>(c.x);
  r.z = fp8x2_bf16x2<false>(c.y);
  r.w = fp8x2_bf16x2<true>(c.y);
  return __builtin_bit_cast(bf16x8, r);
}

template <int D, int P, bool FP8>
struct DGeo {
  static constexpr int ELEM = FP8 ? 1 : 2;
  static constexpr int RB = D * ELEM;                  // bytes per K/V row
  static constexpr int TILE = tile_bytes(FP8);         // K + V bytes per tile
  static constexpr int KPT = TILE / (2 * RB);          // keys per tile
  static constexpr int CPR = RB / 16;                  // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;                 // rows per DMA instruction
  static constexpr int NI = KPT / RPI;                 // DMA instructions per matrix per tile
  static constexpr int NBLK = KPT / 32;                // 32-key S^T blocks per tile
  static constexpr int NPG = KPT >= P ? KPT / P : 1;   // pages touched by a tile
  static constexpr int KT = D / 16;                    // k-steps of K Q^T
  static constexpr int DB = D / 32;                    // 32-row blocks of O^T
  static constexpr int MAX_CHUNK_KEYS = 64 * P;        // one page id per lane
  static_assert(KPT % 32 == 0, "tile holds whole 32-key blocks");
};

// Chunk swizzles for a 256-bytes-per-clock LDS (see the extend kernel).
// K: ds_read_b128 of row swap(m), chunk c, 16 lanes per clock.
template <int RB>
__device__ __forceinline__ int k_swz(int row) {
  const int s = swap_bits_2_3(row);
  return RB == 256 ? (s & 15) : RB == 128 ? ((s >> 1) & 7) : ((s >> 2) & 3);
}
// V, bf16 (tr_b16, 32 lanes per clock: 4 rows x 4 chunks)
template <int RB>
__device__ __forceinline__ int v_swz16(int row) {
  return RB == 256 ? 4 * (row & 3) : 4 * ((row >> 1) & 1);
}
// V, fp8 (tr_b8, 32 lanes per clock: 8 rows x 2 chunks x 2 halves)
template <int RB>
__device__ __forceinline__ int v_swz8(int row) {
  return RB == 128 ? 2 * ((row >> 1) & 3) : 2 * ((row >> 2) & 1);
}

template <int D, int P, bool FP8, bool AP>
__global__ __launch_bounds__(64) void decode_kernel(ExtendParams p, PlanArg<AP> ap) {
  using T = DGeo<D, P, FP8>;
  // one array per stage; the tile loop is unrolled by the stage count, so
  // every step addresses a fixed array
  static_assert(kStages == 3, "the tile loop below is unrolled by three");
  __shared__ __attribute__((aligned(1024))) uint8_t lds_s0[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_s1[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_s2[T::TILE];

  WorkItem it;
  if constexpr (AP) {
    // the plan in the kernel arguments, in compact form: this item is rebuilt
    // from the sequence records (the whole wave searches them)
    const ExpandDesc& d = *reinterpret_cast<const ExpandDesc*>(ap.bytes + p.ap_desc);
    const DecodeRec* rec = reinterpret_cast<const DecodeRec*>(ap.bytes + d.rec_off);
    const int i = blockIdx.x;
    const int b_full = i < d.n_full ? wave_last_at_most(d.n_seqs, i, static_cast<int>(threadIdx.x),
                                                        [&](int k) { return rec[k].full_off; })
                                    : 0;
    it = expand_item_at(rec, reinterpret_cast<const int32_t*>(ap.bytes + d.tail_off), d, i, b_full);
  } else {
    it = p.items[blockIdx.x];
  }
  if (it.seq < 0) return;
  const SeqInfo sq = plan_ptr<AP>(ap, p.ap_seqs, p.seqs)[it.seq];
  const int lane = threadIdx.x;
  const int h = lane >> 5, col = lane & 31;
  const int G = p.gqa_group, hkv = p.num_kv_heads, hq = hkv * G;
  const int kvh = it.kvh;
  const int lp = sq.lp;
  const int tok = sq.cu;  // the sequence's single new token
  const int32_t* bt = p.block_table + size_t(sq.bt_row) * p.bt_stride;
  const uint8_t* k_pool = static_cast<const uint8_t*>(p.k_pool);
  const uint8_t* v_pool = static_cast<const uint8_t*>(p.v_pool);
  const bool row_ok = col < G;

  // prefix keys of this item: [kb, ke); the new key when kv_end passes lp
  const int kb = it.kv_begin;
  const int ke = min(it.kv_end, lp);
  const bool has_new = it.kv_end > lp;
  const int n_tiles = ke > kb ? (ke - kb + T::KPT - 1) / T::KPT : 0;

  // page ids (and fp8 scales) of the chunk: lane j holds page kb / P + j
  const int page0 = kb / P;
  const int n_pages = ke > kb ? (ke - 1) / P - page0 + 1 : 0;
  int my_pg = 0;
  float my_ks = 1.f, my_vs = 1.f;
  if (lane < n_pages) {
    my_pg = bt[page0 + lane];
    if constexpr (FP8) {
      const size_t si = size_t(my_pg) * hkv + kvh;
      my_ks = p.k_scale[si];
      my_vs = p.v_scale[si];
    }
  }
  // per page: log2 and reciprocal of the V scale (read back per key group)
  float my_lvs = 0.f, my_ivs = 1.f;
  // Fused page write (a step of decodes only): the item holding the new key
  // also stores the new token's K/V into slot lp of its page, after its own
  // DMA has drained.  The attention reads no pool slot at or past lp, so the
  // two are independent.  The page and its scales land with the page ids, so
  // no load of this is outstanding in the counted DMA pipeline.
  const bool writer = has_new && p.w.total_tokens > 0;
  int pg_new = 0;
  float ks_new = 1.f, vs_new = 1.f;
  if (writer) {
    pg_new = bt[lp / P];
    if constexpr (FP8) {
      const size_t si = size_t(pg_new) * hkv + kvh;
      ks_new = p.k_scale[si];
      vs_new = p.v_scale[si];
    }
  }

  // Q^T (B operand).  bf16 pools: k-step kk holds dims 16 kk + 8 h + e.  fp8
  // pools read 16 fp8 dims per fragment, so k-steps 2t and 2t+1 hold dims
  // 32 t + 16 h + 8 (kk & 1) + e (the contraction order is free).
  bf16x8 qf[T::KT];
  {
    const uint16_t* qrow = static_cast<const uint16_t*>(p.q) + (size_t(tok) * hq + size_t(kvh) * G + col) * D;
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      const int d0 = FP8 ? 32 * (kk >> 1) + 16 * h + 8 * (kk & 1) : 16 * kk + 8 * h;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row_ok) v = *reinterpret_cast<const u32x4*>(qrow + d0);
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  // DMA: instruction j covers tile rows [j RPI, (j+1) RPI); lane fetches row
  // j RPI + lane / CPR into chunk position lane % CPR.  Rows past the chunk's
  // prefix end fetch the chunk's last key again (same page as the instruction's
  // first row, whose scores are masked), so every tile issues exactly 2 NI
  // instructions and the vmcnt arithmetic below is exact.
  const int dma_row = lane / T::CPR, dma_pos = lane % T::CPR;
  auto issue_tile = [&](int t, uint32_t kdst) __attribute__((always_inline)) {
    const int j0 = kb + t * T::KPT;
    const uint32_t vdst = kdst + T::TILE / 2;
#pragma unroll
    for (int j = 0; j < T::NI; ++j) {
      const int R = j * T::RPI + dma_row;
      const int key = min(j0 + R, ke - 1);
      // page index within the chunk (uniform per instruction: its rows lie in one page)
      const int r0 = min(j0 + j * T::RPI, ke - 1);
      const int pg = __builtin_amdgcn_readlane(my_pg, min(r0 / P - page0, 63));
      const size_t base = (size_t(pg) * hkv + kvh) * P * T::RB + size_t(key % P) * T::RB;
      const uint32_t kc = dma_pos ^ k_swz<T::RB>(R);
      const uint32_t vc = dma_pos ^ (FP8 ? v_swz8<T::RB>(R) : v_swz16<T::RB>(R));
      dma16(k_pool + base + 16 * kc, kdst + j * T::RPI * T::RB);
      dma16(v_pool + base + 16 * vc, vdst + j * T::RPI * T::RB);
    }
  };

  f32x16 o[T::DB];
#pragma unroll
  for (int b = 0; b < T::DB; ++b) o[b] = f32x16{};
  float m_run = kNegBig, l_run = 0.f;
  const float c = p.scale_log2;

  // prologue: tiles 0, 1 and 2 in flight.  Q and the page ids land first (the
  // addresses need the ids), so only DMA is outstanding in the loop; this wait
  // is the compiler's own, so it knows that Q has landed.
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
  if (n_tiles > 0) {
    issue_tile(0, lds_addr(lds_s0));
    issue_tile(1, lds_addr(lds_s1));
    issue_tile(2, lds_addr(lds_s2));
  }
  if constexpr (FP8) {
    my_lvs = __builtin_amdgcn_logf(my_vs);
    my_ivs = 1.f / my_vs;
  }

  // compute on tile t, read from stage ks once it has landed
  auto compute = [&](int t, const uint8_t* ks) __attribute__((always_inline)) {
    const uint8_t* vs = ks + T::TILE / 2;
    const int j0 = kb + t * T::KPT;

#pragma unroll
    for (int blk = 0; blk < T::NBLK; ++blk) {
      // S^T block: rows m of the block read key swap(m)
      f32x16 s = f32x16{};
      const int R = swap_bits_2_3(col) + 32 * blk;
      if constexpr (FP8) {
#pragma unroll
        for (int t2 = 0; t2 < T::KT / 2; ++t2) {
          const int pos = (2 * t2 + h) ^ k_swz<T::RB>(R);
          const u32x4 raw = *reinterpret_cast<const u32x4*>(ks + R * T::RB + 16 * pos);
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fp8x8_bf16x8(u32x2{raw.x, raw.y}), qf[2 * t2], s, 0, 0, 0);
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fp8x8_bf16x8(u32x2{raw.z, raw.w}), qf[2 * t2 + 1], s, 0, 0, 0);
        }
      } else {
#pragma unroll
        for (int kk = 0; kk < T::KT; ++kk) {
          const int pos = (2 * kk + h) ^ k_swz<T::RB>(R);
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(ks + R * T::RB + 16 * pos);
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s, 0, 0, 0);
        }
      }
      // element i holds key j0 + 32 blk + 16 (i / 8) + 8 h + i % 8; the 8 keys of
      // half-group i / 8 share one page.  Exponent of key j: x = s c k_scale +
      // log2 v_scale (fp8; s c for bf16), so that P = 2^(x - m) arrives already
      // multiplied by the page's V scale and the row sum divides it back out.
      float cg[2] = {c, c};
      float lvs[2] = {0.f, 0.f};
      float ivs[2] = {1.f, 1.f};
      if constexpr (FP8) {
#pragma unroll
        for (int s8 = 0; s8 < 2; ++s8) {
          const int q = (j0 + 32 * blk + 16 * s8) / P - page0;
          cg[s8] = c * __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_ks), q));
          lvs[s8] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_lvs), q));
          ivs[s8] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_ivs), q));
        }
      }
      if (j0 + 32 * blk + 32 > ke) {  // keys past the chunk's prefix end
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (j0 + 32 * blk + 16 * (i >> 3) + 8 * h + (i & 7) >= ke) s[i] = -INFINITY;
      }
      // Weights against the running max as it stands (no row max per block):
      // only when some half-column's sum of 2^(s c - m) passes kSumLimit (or is
      // not finite, as on an item's first block) is the block's max taken, m
      // raised and the weights recomputed.  O / l and lse do not depend on m.
      bf16x8 pf[2];
      float tsum;
      auto weights = [&]() __attribute__((always_inline)) {
        tsum = 0.f;
#pragma unroll
        for (int s8 = 0; s8 < 2; ++s8) {
          const float bias = lvs[s8] - m_run;
          float gsum = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pv = __builtin_amdgcn_exp2f(fmaf(s[8 * s8 + e], cg[s8], bias));
            gsum += pv;
            pf[s8][e] = static_cast<__bf16>(pv);
          }
          tsum = FP8 ? fmaf(gsum, ivs[s8], tsum) : tsum + gsum;
        }
      };
      weights();
      if (__any(!(tsum <= kSumLimit))) {
        float mx = -INFINITY;
#pragma unroll
        for (int s8 = 0; s8 < 2; ++s8) {
          float gm = -INFINITY;
#pragma unroll
          for (int e = 0; e < 8; ++e) gm = fmaxf(gm, s[8 * s8 + e]);
          mx = fmaxf(mx, fmaf(gm, cg[s8], lvs[s8]));
        }
        // both halves of a column hold its keys: they agree on one m
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                         false, false);
        mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
        if (mx > m_run) {
          const float alpha = __builtin_amdgcn_exp2f(m_run - mx);
          m_run = mx;
          l_run *= alpha;
#pragma unroll
          for (int b = 0; b < T::DB; ++b) o[b] *= alpha;
        }
        weights();
      }
      l_run += tsum;
      // O^T += V^T P^T over the block's two 16-key slices
      const int grp = lane >> 4, ri = lane & 15;
#pragma unroll
      for (int s8 = 0; s8 < 2; ++s8) {
        const int u = 2 * blk + s8;
#pragma unroll
        for (int b = 0; b < T::DB; ++b) {
          bf16x8 vf;
          if constexpr (FP8) {
            // source lane (k, a) = (ri / 2, ri % 2): key 16u + 8h + k, dims 32b + 16(grp&1) + 8a
            const int Rv = 16 * u + 8 * h + (ri >> 1);
            const int dbyte = 32 * b + 16 * (grp & 1) + 8 * (ri & 1);
            const int off = Rv * T::RB + 16 * ((dbyte >> 4) ^ v_swz8<T::RB>(Rv)) + (dbyte & 15);
            const i32x2 raw = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(vs + off));
            vf = fp8x8_bf16x8(u32x2{static_cast<uint32_t>(raw.x), static_cast<uint32_t>(raw.y)});
          } else {
            const int kq = ri >> 2, a = ri & 3;
            const int chunk = 4 * b + 2 * (grp & 1) + (a >> 1);
            i16x4 half[2];
#pragma unroll
            for (int e4 = 0; e4 < 2; ++e4) {
              const int Rv = 16 * u + 8 * h + 4 * e4 + kq;
              const int off = Rv * T::RB + 16 * (chunk ^ v_swz16<T::RB>(Rv)) + 8 * (a & 1);
              half[e4] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vs + off));
            }
            vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(half[0], half[1], 0, 1, 2, 3, 4, 5, 6, 7));
          }
          o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[s8], o[b], 0, 0, 0);
        }
      }
    }
  };
  // Tile t lives in stage t % 3.  Every step waits for its tile (the two
  // issued after it may still fly), computes on it, then refills the stage with
  // tile t + 3.  Steps past the last tile compute nothing, and issues past it
  // fetch the chunk's last key again, so each step issues exactly 2 NI
  // instructions and one fixed wait count holds everywhere.
  auto step = [&](int t, const uint8_t* st) __attribute__((always_inline)) {
    wait_vmcnt<2 * 2 * T::NI>();
    if (t < n_tiles) compute(t, st);
    wait_lgkmcnt0();  // the stage's reads are done before it is refilled
    issue_tile(t + 3, lds_addr(st));
  };
  for (int t = 0; t < n_tiles; t += 3) {
    step(t, lds_s0);
    step(t + 1, lds_s1);
    step(t + 2, lds_s2);
  }
  wait_vmcnt<0>();  // no DMA may land in LDS after the wave has ended
  if (writer && lane < D / 8)
    pw::store_piece<D, P, FP8>(p.w, tok, kvh, lane, pg_new, lp % P, ks_new, vs_new);

  // the new token's own key and value (bf16, from k_new / v_new)
  if (has_new) {
    const uint16_t* kn = static_cast<const uint16_t*>(p.k_new) + (size_t(tok) * hkv + kvh) * D;
    const uint16_t* vn = static_cast<const uint16_t*>(p.v_new) + (size_t(tok) * hkv + kvh) * D;
    float part = 0.f;
#pragma unroll
    for (int kk = 0; kk < T::KT; ++kk) {
      const int d0 = FP8 ? 32 * (kk >> 1) + 16 * h + 8 * (kk & 1) : 16 * kk + 8 * h;
      const bf16x8 kv = *reinterpret_cast<const bf16x8*>(kn + d0);
#pragma unroll
      for (int e = 0; e < 8; ++e) part = fmaf(static_cast<float>(qf[kk][e]), static_cast<float>(kv[e]), part);
    }
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(part), __float_as_uint(part), false, false);
    const float x = (__uint_as_float(sw[0]) + __uint_as_float(sw[1])) * c;
    const float m_new = fmaxf(m_run, x);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    const float pn = __builtin_amdgcn_exp2f(x - m_new);
    m_run = m_new;
    l_run = l_run * alpha + (h == 0 ? pn : 0.f);
    const float pb = static_cast<float>(static_cast<__bf16>(pn));
#pragma unroll
    for (int b = 0; b < T::DB; ++b) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const bf16x4 v4 = *reinterpret_cast<const bf16x4*>(vn + 32 * b + 8 * q4 + 4 * h);
#pragma unroll
        for (int e = 0; e < 4; ++e) o[b][4 * q4 + e] = fmaf(pb, static_cast<float>(v4[e]), o[b][4 * q4 + e] * alpha);
      }
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!row_ok) return;
  if (it.part < 0) {
    const float inv = 1.f / l_tot;
    uint16_t* orow = static_cast<uint16_t*>(p.out) + (size_t(tok) * hq + size_t(kvh) * G + col) * D;
#pragma unroll
    for (int b = 0; b < T::DB; ++b) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = static_cast<__bf16>(o[b][4 * q4 + e] * inv);
        *reinterpret_cast<u32x2*>(orow + 32 * b + 8 * q4 + 4 * h) = __builtin_bit_cast(u32x2, v4);
      }
    }
    if (p.lse != nullptr && h == 0)
      p.lse[size_t(tok) * hq + size_t(kvh) * G + col] = (m_run + __log2f(l_tot)) * kLn2;
  } else {
    // the unnormalised partial O in bf16 (relative rounding 2^-9, the range of fp32)
    uint16_t* po = p.part_o + (size_t(it.part) * p.part_rows + col) * D;
#pragma unroll
    for (int b = 0; b < T::DB; ++b) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        bf16x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = static_cast<__bf16>(o[b][4 * q4 + e]);
        *reinterpret_cast<u32x2*>(po + 32 * b + 8 * q4 + 4 * h) = __builtin_bit_cast(u32x2, v4);
      }
    }
    if (h == 0) {
      float* ml = p.part_ml + (size_t(it.part) * p.part_rows + col) * 2;
      ml[0] = m_run;
      ml[1] = l_tot;
    }
  }
}

template <int D, int P, bool FP8>
hipError_t launch_t(const ExtendParams& p, hipStream_t stream, const ArgPlan* ap) {
  if (ap) hipLaunchKernelGGL((decode_kernel<D, P, FP8, true>), dim3(p.n_items), dim3(64), 0, stream, p, *ap);
  else hipLaunchKernelGGL((decode_kernel<D, P, FP8, false>), dim3(p.n_items), dim3(64), 0, stream, p, NoArgPlan{});
  return hipGetLastError();
}

}  // namespace

int decode_max_chunk_keys(int page_size) { return 64 * page_size; }

int decode_keys_per_tile(int head_dim, bool fp8) { return tile_bytes(fp8) / (2 * head_dim * (fp8 ? 1 : 2)); }

int decode_waves_per_cu(bool fp8) { return (160 * 1024) / (kStages * tile_bytes(fp8)); }  // 160 KB of LDS per CU

hipError_t launch_decode(const ExtendParams& p, int head_dim, int page_size, bool fp8,
                         hipStream_t stream, const ArgPlan* ap) {
  if (p.n_items <= 0) return hipSuccess;
#define CW_CASE(D_, P_)                                                                   \
  if (head_dim == D_ && page_size == P_)                                                  \
    return fp8 ? launch_t<D_, P_, true>(p, stream, ap) : launch_t<D_, P_, false>(p, stream, ap);
  CW_CASE(64, 16)
  CW_CASE(64, 64)
  CW_CASE(128, 16)
  CW_CASE(128, 64)
#undef CW_CASE
  return hipErrorInvalidValue;
}

}  // namespace cw
