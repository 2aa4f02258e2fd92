// Scatter of new K/V rows into their page-pool slots (bf16 copy or fp8
// quantise-on-write).  One thread moves 8 elements (16 bytes of bf16) of one
// (token, kv head) row of K and of V; consecutive threads take consecutive
// 16-byte pieces of a row, so both the reads of k_new/v_new and the writes of a
// pool row are contiguous.
#include <hip/hip_runtime.h>

#include "../cw_internal.h"

namespace cw {
namespace {

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

template <int D, int P, bool FP8>
__global__ __launch_bounds__(256) void write_pages_kernel(WriteParams p) {
  constexpr int CH = D / 8;  // 8-element pieces per row
  const int hkv = p.num_kv_heads;
  const int64_t total = int64_t(p.total_tokens) * hkv * CH;
  for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
       idx += int64_t(gridDim.x) * blockDim.x) {
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
    const int pg = p.block_table[size_t(lo) * p.bt_stride + pos / P];
    const int slot = pos % P;
    const size_t src = (size_t(tok) * hkv + h) * D + c8 * 8;
    const size_t dst = ((size_t(pg) * hkv + h) * P + slot) * D + c8 * 8;
    const u32x4 kx = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.k_new) + src);
    const u32x4 vx = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.v_new) + src);
    if constexpr (FP8) {
      const size_t si = size_t(pg) * hkv + h;
      *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(p.k_pool) + dst) = quantise8(kx, p.k_scale[si]);
      *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(p.v_pool) + dst) = quantise8(vx, p.v_scale[si]);
    } else {
      *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.k_pool) + dst) = kx;
      *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.v_pool) + dst) = vx;
    }
  }
}

template <int D, int P, bool FP8>
hipError_t launch_t(const WriteParams& p, hipStream_t stream) {
  const int64_t total = int64_t(p.total_tokens) * p.num_kv_heads * (D / 8);
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL((write_pages_kernel<D, P, FP8>), dim3(static_cast<unsigned>(blocks)), dim3(256),
                     0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_write_pages(const WriteParams& p, int head_dim, int page_size, bool fp8,
                              hipStream_t stream) {
  if (p.total_tokens <= 0) return hipSuccess;
#define CW_CASE(D_, P_)                                                                  \
  if (head_dim == D_ && page_size == P_)                                                 \
    return fp8 ? launch_t<D_, P_, true>(p, stream) : launch_t<D_, P_, false>(p, stream);
  CW_CASE(64, 16)
  CW_CASE(64, 64)
  CW_CASE(128, 16)
  CW_CASE(128, 64)
#undef CW_CASE
  return hipErrorInvalidValue;
}

}  // namespace cw
