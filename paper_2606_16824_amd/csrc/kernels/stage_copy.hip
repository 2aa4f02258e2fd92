// Plan upload: copies a call's plan (per-sequence info, work items, merge
// groups) from the library's pinned staging slot to the caller's workspace.
// The device reads the pinned host memory directly over the host link, on the
// call's stream, so the upload is one small kernel in the same queue as the
// attention kernels (a copy engine would cost a hand-off between queues).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "../cw_internal.h"
#include "../plan_expand.h"

namespace cw {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

// Once a workgroup has read its share of the slot it writes `seq` into its
// word of `done` (pinned host memory, a system-scope store), so the host knows
// when the slot may be refilled without an event in the stream.
__device__ __forceinline__ void report_read(uint32_t* done, uint32_t seq) {
  __syncthreads();  // every lane's reads of the slot have returned
  if (done != nullptr && threadIdx.x == 0)
    __hip_atomic_store(done + blockIdx.x, seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__global__ __launch_bounds__(kThreads) void stage_copy_kernel(const uint8_t* src, uint8_t* dst,
                                                              int64_t bytes, uint32_t* done,
                                                              uint32_t seq) {
  const int64_t n16 = bytes / 16;
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  const int64_t first = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  for (int64_t i = first; i < n16; i += stride)
    reinterpret_cast<u32x4*>(dst)[i] = reinterpret_cast<const u32x4*>(src)[i];
  if (first < bytes - n16 * 16) dst[n16 * 16 + first] = src[n16 * 16 + first];
  report_read(done, seq);
}

// Plan upload under stream capture: the bytes travel in the kernel's own
// arguments, which a captured launch keeps by value, so every replay of the
// graph writes the plan the call was captured with (a staging slot would be
// read at replay time, after later calls may have refilled it).
struct ArgChunk {
  uint32_t* dst;
  uint32_t words;
  uint32_t data[kArgChunkBytes / 4];
};

__global__ __launch_bounds__(kThreads) void arg_copy_kernel(ArgChunk a) {
  for (uint32_t i = threadIdx.x; i < a.words; i += kThreads) a.dst[i] = a.data[i];
}

// Upload of a compact plan blob: the first `verbatim` bytes are copied as they
// are (16 bytes per lane), then every workgroup reads the decode records and
// the tail order into LDS and rebuilds its share of the work items and merge
// groups (expand_item / expand_group, the functions the host checks them with).
__global__ __launch_bounds__(kThreads) void plan_expand_kernel(const uint8_t* src, uint8_t* dst,
                                                              int64_t verbatim, ExpandDesc d,
                                                              uint32_t* done, uint32_t seq) {
  __shared__ DecodeRec rec[kMaxExpandSeqs];
  __shared__ int32_t tails[kMaxExpandSeqs];
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  const int64_t first = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  const int64_t n16 = verbatim / 16;
  for (int64_t i = first; i < n16; i += stride)
    reinterpret_cast<u32x4*>(dst)[i] = reinterpret_cast<const u32x4*>(src)[i];
  const DecodeRec* rs = reinterpret_cast<const DecodeRec*>(src + d.rec_off);
  const int32_t* ts = reinterpret_cast<const int32_t*>(src + d.tail_off);
  for (int32_t i = threadIdx.x; i < d.n_seqs; i += kThreads) rec[i] = rs[i];
  for (int32_t i = threadIdx.x; i < d.n_tails; i += kThreads) tails[i] = ts[i];
  report_read(done, seq);  // the slot is read; the rest works from LDS
  WorkItem* items = reinterpret_cast<WorkItem*>(dst + d.items_off);
  CombineGroup* groups = reinterpret_cast<CombineGroup*>(dst + d.groups_off);
  for (int64_t i = first; i < d.n_items + d.n_groups; i += stride) {
    if (i < d.n_items) items[i] = expand_item(rec, tails, d, static_cast<int32_t>(i));
    else groups[i - d.n_items] = expand_group(rec, d, static_cast<int32_t>(i - d.n_items));
  }
}

}  // namespace

hipError_t launch_plan_expand(const void* src, void* dst, size_t verbatim, const ExpandDesc& d,
                              hipStream_t stream, uint32_t* done, uint32_t seq, int32_t* workgroups) {
  if (d.n_seqs < 1 || d.n_seqs > kMaxExpandSeqs || d.n_tails > d.n_seqs || verbatim % 16 != 0)
    return hipErrorInvalidValue;
  const int64_t work = std::max<int64_t>(int64_t(verbatim / 16), int64_t(d.n_items) + d.n_groups);
  const int64_t blocks =
      std::max<int64_t>(1, std::min<int64_t>((work + kThreads - 1) / kThreads, kMaxUploadWorkgroups));
  *workgroups = static_cast<int32_t>(blocks);
  hipLaunchKernelGGL(plan_expand_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream,
                     static_cast<const uint8_t*>(src), static_cast<uint8_t*>(dst), int64_t(verbatim), d,
                     done, seq);
  return hipGetLastError();
}

hipError_t launch_arg_copy(const void* src, void* dst, size_t bytes, hipStream_t stream) {
  const uint8_t* s = static_cast<const uint8_t*>(src);
  uint8_t* d = static_cast<uint8_t*>(dst);
  for (size_t off = 0; off < bytes; off += kArgChunkBytes) {
    ArgChunk a;
    const size_t n = std::min(bytes - off, kArgChunkBytes);
    a.dst = reinterpret_cast<uint32_t*>(d + off);
    a.words = static_cast<uint32_t>(n / 4);
    std::memcpy(a.data, s + off, n);
    hipLaunchKernelGGL(arg_copy_kernel, dim3(1), dim3(kThreads), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_stage_copy(const void* src, void* dst, size_t bytes, hipStream_t stream, uint32_t* done,
                             uint32_t seq, int32_t* workgroups) {
  const int64_t n16 = int64_t(bytes / 16);
  const int64_t blocks =
      std::max<int64_t>(1, std::min<int64_t>((n16 + kThreads - 1) / kThreads, kMaxUploadWorkgroups));
  if (workgroups) *workgroups = static_cast<int32_t>(blocks);
  hipLaunchKernelGGL(stage_copy_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream,
                     static_cast<const uint8_t*>(src), static_cast<uint8_t*>(dst), int64_t(bytes), done, seq);
  return hipGetLastError();
}

}  // namespace cw
