// Whole-page copies between the device page pool and a host block pool (the
// offloading configuration of CacheWise Sec. 6.4: evicted KV blocks go to CPU
// DRAM and come back when their session resumes).  Entry i of a swap copies
// block src_ids[i] of the source pool to block dst_ids[i] of the destination
// pool: every kv head of the page, K and V, and for fp8 pools the page's
// per-(page, kv head) scales.  A page of all kv heads is one contiguous
// Hkv * P * D-element block in the [pages, Hkv, P, D] layout, so the copy is a
// list of contiguous blocks: consecutive lanes move consecutive 16-byte pieces
// of a block, and the host side of the copy is read or written straight over
// the host link (pinned, device-mapped memory), with no staging buffer.
#include <hip/hip_runtime.h>

#include "../cw_internal.h"

namespace cw {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void swap_kernel(SwapParams p) {
  const int64_t pieces = p.block_bytes / 16;  // 16-byte pieces per block and matrix
  const int64_t total = int64_t(p.n) * 2 * pieces;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total; idx += stride) {
    const int64_t e = idx / pieces;  // entry * 2 + matrix
    const int64_t off = (idx - e * pieces) * 16;
    const int i = static_cast<int>(e >> 1);
    const bool v = e & 1;
    const size_t s = size_t(p.src_ids[i]) * p.block_bytes + off;
    const size_t d = size_t(p.dst_ids[i]) * p.block_bytes + off;
    const u32x4 x = *reinterpret_cast<const u32x4*>((v ? p.src_v : p.src_k) + s);
    *reinterpret_cast<u32x4*>((v ? p.dst_v : p.dst_k) + d) = x;
  }
  if (p.src_ks == nullptr) return;
  const int64_t n_sc = int64_t(p.n) * p.scales_per_block;
  for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < n_sc; idx += stride) {
    const int i = static_cast<int>(idx / p.scales_per_block);
    const int h = static_cast<int>(idx - int64_t(i) * p.scales_per_block);
    const size_t s = size_t(p.src_ids[i]) * p.scales_per_block + h;
    const size_t d = size_t(p.dst_ids[i]) * p.scales_per_block + h;
    p.dst_ks[d] = p.src_ks[s];
    p.dst_vs[d] = p.src_vs[s];
  }
}

}  // namespace

hipError_t launch_swap(const SwapParams& p, hipStream_t stream) {
  if (p.n <= 0) return hipSuccess;
  const int64_t total = int64_t(p.n) * 2 * (p.block_bytes / 16);
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 65536));
  hipLaunchKernelGGL(swap_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace cw
