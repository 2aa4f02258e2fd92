// Scatter of one 16-byte piece of a new K/V row into its page-pool slot (bf16
// copy, or fp8 quantise-on-write with the page's scale), shared by the
// stand-alone page-write kernel and the fused writes of the extend and decode
// kernels.
#pragma once
#include <hip/hip_runtime.h>

#include "../cw_internal.h"

namespace cw {
namespace pw {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Eight bf16 -> eight e4m3fn codes of clamp(x / s, -448, 448), nearest-even.
__device__ __forceinline__ u32x2 quantise8(u32x4 x, float s) {
  u32x2 out;
#pragma unroll
  for (int w = 0; w < 2; ++w) {
    float f[4];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const uint32_t d = x[2 * w + e];
      f[2 * e] = __uint_as_float(d << 16);
      f[2 * e + 1] = __uint_as_float(d & 0xFFFF0000u);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = fminf(fmaxf(__fdiv_rn(f[e], s), -448.f), 448.f);
    int packed = __builtin_amdgcn_cvt_pk_fp8_f32(f[0], f[1], 0, false);
    packed = __builtin_amdgcn_cvt_pk_fp8_f32(f[2], f[3], packed, true);
    out[w] = static_cast<uint32_t>(packed);
  }
  return out;
}

// Elements c8 * 8 .. c8 * 8 + 7 of K and V of new row (tok, kv head h) into slot
// `slot` of physical page `pg`; fp8 pools quantise with the page's scales ks, vs.
template <int D, int P, bool FP8>
__device__ __forceinline__ void store_piece(const WriteParams& p, int tok, int h, int c8, int pg,
                                            int slot, float ks, float vs) {
  const int hkv = p.num_kv_heads;
  const size_t src = (size_t(tok) * hkv + h) * D + c8 * 8;
  const size_t dst = ((size_t(pg) * hkv + h) * P + slot) * D + c8 * 8;
  const u32x4 kx = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.k_new) + src);
  const u32x4 vx = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.v_new) + src);
  if constexpr (FP8) {
    *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(p.k_pool) + dst) = quantise8(kx, ks);
    *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(p.v_pool) + dst) = quantise8(vx, vs);
  } else {
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.k_pool) + dst) = kx;
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.v_pool) + dst) = vx;
  }
}

// Piece `idx` of the flat [token, kv head, D / 8] order: the 8 elements
// c8 * 8 .. c8 * 8 + 7 of K and of V for (token, kv head) go to slot
// (Lp + i) % P of page block_table[b][(Lp + i) / P], where token = cu_b + i.
template <int D, int P, bool FP8>
__device__ __forceinline__ void write_piece(const WriteParams& p, int64_t idx) {
  constexpr int CH = D / 8;  // 8-element pieces per row
  const int hkv = p.num_kv_heads;
  const int c8 = static_cast<int>(idx % CH);
  const int64_t rest = idx / CH;
  const int h = static_cast<int>(rest % hkv);
  const int tok = static_cast<int>(rest / hkv);
  // sequence owning this token: the last one whose first row is <= tok
  int lo = 0, hi = p.num_seqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.seqs[mid].cu <= tok) lo = mid;
    else hi = mid - 1;
  }
  const SeqInfo sq = p.seqs[lo];
  const int pos = sq.lp + (tok - sq.cu);
  const int pg = p.block_table[size_t(sq.bt_row) * p.bt_stride + pos / P];
  if constexpr (FP8) {
    const size_t si = size_t(pg) * hkv + h;
    store_piece<D, P, FP8>(p, tok, h, c8, pg, pos % P, p.k_scale[si], p.v_scale[si]);
  } else {
    store_piece<D, P, FP8>(p, tok, h, c8, pg, pos % P, 1.f, 1.f);
  }
}

}  // namespace pw
}  // namespace cw
