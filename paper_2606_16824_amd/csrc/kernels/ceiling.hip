// Measured ceilings for the two rooflines of the attention kernels: a
// matrix-core loop with no memory traffic (dense bf16 MFMA) and streaming
// read / copy kernels (HBM).  Not part of the attention path; a benchmark
// places each attention kernel against these next to the published peaks.
#include <hip/hip_runtime.h>

#include <cstdio>

#include "../../include/cw_ceiling.h"
#include "../cw_internal.h"

namespace cw {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kStreamGrid = 16384;
constexpr int kStreamThreads = 256;
constexpr int kUnroll = 4;  // 16-byte loads in flight per lane per round

// Eight waves (two per SIMD), four independent accumulator chains per wave:
// an MFMA's result is needed again only four issues later, so the matrix pipe
// never waits on a dependency.  Operands come from the lane id, so nothing is
// known at compile time; the values stay small (no overflow over 2^24 rounds).
__global__ __launch_bounds__(512) void mfma_loop_kernel(int iters, float* sink) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = static_cast<__bf16>(float((lane + e) & 7) * (1.f / 1024.f));
    b[e] = static_cast<__bf16>(float((lane * 3 + e) & 7) * (1.f / 1024.f));
  }
  f32x16 c0 = f32x16{}, c1 = f32x16{}, c2 = f32x16{}, c3 = f32x16{};
  for (int i = 0; i < iters; ++i) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  if (lane == 0) sink[blockIdx.x * 8 + (threadIdx.x >> 6)] = c0[0] + c1[1] + c2[2] + c3[3];
}

// Grid-stride streaming read: each lane keeps kUnroll 16-byte loads in flight
// per round; the XOR of everything read leaves as one word per workgroup.
__global__ __launch_bounds__(kStreamThreads) void stream_read_kernel(const u32x4* src, int64_t n16,
                                                                     uint32_t* sink) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u];
  }
  for (; i < n16; i += stride) acc ^= src[i];
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x ^= __shfl_xor(x, o);
  __shared__ uint32_t part[kStreamThreads / 64];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0;
    for (int w = 0; w < kStreamThreads / 64; ++w) r ^= part[w];
    sink[blockIdx.x] = r;
  }
}

__global__ __launch_bounds__(kStreamThreads) void stream_copy_kernel(const u32x4* src, u32x4* dst,
                                                                     int64_t n16) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) __builtin_nontemporal_store(v[u], dst + i + u * stride);
  }
  for (; i < n16; i += stride) dst[i] = src[i];
}

cw_status_t fail_msg(cw_status_t s, const char* msg) {
  set_last_error(msg);
  return s;
}

cw_status_t launched(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return CW_OK;
  char buf[256];
  snprintf(buf, sizeof(buf), "%s: %s", what, hipGetErrorString(e));
  return fail_msg(CW_ERR_HIP, buf);
}

cw_status_t check_stream_args(const void* src, const void* dst, size_t bytes) {
  if (src == nullptr || dst == nullptr) return fail_msg(CW_ERR_NULL, "a buffer pointer is NULL");
  if (bytes == 0) return fail_msg(CW_ERR_UNSUPPORTED, "bytes must be > 0");
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst) | bytes) & 15u)
    return fail_msg(CW_ERR_ALIGN, "pointers and size must be multiples of 16 bytes");
  return CW_OK;
}

}  // namespace
}  // namespace cw

extern "C" {

cw_status_t cw_ceiling_mfma_bf16(int32_t workgroups, int32_t iters, float* sink,
                                 hipStream_t stream) {
  using namespace cw;
  if (sink == nullptr) return fail_msg(CW_ERR_NULL, "sink is NULL");
  if (workgroups < 1 || workgroups > 65536 || iters < 1 || iters > (1 << 24))
    return fail_msg(CW_ERR_UNSUPPORTED, "workgroups must be in [1, 65536], iters in [1, 2^24]");
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(workgroups), dim3(512), 0, stream, iters, sink);
  return launched("mfma_loop_kernel");
}

cw_status_t cw_ceiling_stream_read(const void* src, size_t bytes, uint32_t* sink,
                                   hipStream_t stream) {
  using namespace cw;
  const cw_status_t s = check_stream_args(src, sink, bytes);
  if (s != CW_OK) return s;
  hipLaunchKernelGGL(stream_read_kernel, dim3(kStreamGrid), dim3(kStreamThreads), 0, stream,
                     static_cast<const u32x4*>(src), int64_t(bytes / 16), sink);
  return launched("stream_read_kernel");
}

cw_status_t cw_ceiling_stream_copy(const void* src, void* dst, size_t bytes, hipStream_t stream) {
  using namespace cw;
  const cw_status_t s = check_stream_args(src, dst, bytes);
  if (s != CW_OK) return s;
  const char* a = static_cast<const char*>(src);
  const char* b = static_cast<const char*>(dst);
  if (a < b + bytes && b < a + bytes) return fail_msg(CW_ERR_UNSUPPORTED, "src and dst overlap");
  hipLaunchKernelGGL(stream_copy_kernel, dim3(kStreamGrid), dim3(kStreamThreads), 0, stream,
                     static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), int64_t(bytes / 16));
  return launched("stream_copy_kernel");
}

}  // extern "C"
