// Scatter of new K/V rows into their page-pool slots (bf16 copy or fp8
// quantise-on-write).  One thread moves 8 elements (16 bytes of bf16) of one
// (token, kv head) row of K and of V; consecutive threads take consecutive
// 16-byte pieces of a row, so both the reads of k_new/v_new and the writes of a
// pool row are contiguous.
#include <hip/hip_runtime.h>

#include "../cw_internal.h"
#include "page_write.h"

namespace cw {
namespace {

template <int D, int P, bool FP8>
__global__ __launch_bounds__(256) void write_pages_kernel(WriteParams p) {
  constexpr int CH = D / 8;  // 8-element pieces per row
  const int hkv = p.num_kv_heads;
  const int64_t total = int64_t(p.total_tokens) * hkv * CH;
  for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
       idx += int64_t(gridDim.x) * blockDim.x)
    pw::write_piece<D, P, FP8>(p, idx);
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
