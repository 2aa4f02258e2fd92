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

// 32-bit integer hash (the two-multiply avalanche mix); all arithmetic mod 2^32.
__device__ inline uint32_t mix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// A bf16 with a random sign and mantissa and a magnitude in [2^-4, 4).
__device__ inline __bf16 random_bf16(uint32_t u) {
  const uint32_t bits = ((u >> 31) << 15) | ((123u + (u >> 8) % 6u) << 7) | (u & 127u);
  return __builtin_bit_cast(__bf16, static_cast<uint16_t>(bits));
}

// Eight waves (two per SIMD), four independent accumulator chains per wave:
// an MFMA's result is needed again only four issues later, so the matrix pipe
// never waits on a dependency.  Operands come from the lane id (never known at
// compile time), either as eight repeated small patterns or as random bits per
// chain; the accumulators stay finite over 2^24 rounds either way.
__global__ __launch_bounds__(512) void mfma_loop_kernel(int iters, int random, float* sink) {
  const int lane = threadIdx.x & 63;
  const uint32_t g = blockIdx.x * 512u + threadIdx.x;
  bf16x8 a[4], b[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (random) {
        const uint32_t ha = mix32(64u * g + 8u * c + e);
        a[c][e] = random_bf16(ha);
        b[c][e] = random_bf16(mix32(ha ^ 0x9e3779b9u));
      } else {
        a[c][e] = static_cast<__bf16>(float((lane + e) & 7) * (1.f / 1024.f));
        b[c][e] = static_cast<__bf16>(float((lane * 3 + e) & 7) * (1.f / 1024.f));
      }
    }
  }
  f32x16 c0 = f32x16{}, c1 = f32x16{}, c2 = f32x16{}, c3 = f32x16{};
  for (int i = 0; i < iters; ++i) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1], b[1], c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[2], b[2], c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[3], b[3], c3, 0, 0, 0);
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

cw_status_t cw_ceiling_mfma_bf16(int32_t workgroups, int32_t iters, cw_ceiling_operands_t operands,
                                 float* sink, hipStream_t stream) {
  using namespace cw;
  if (sink == nullptr) return fail_msg(CW_ERR_NULL, "sink is NULL");
  if (workgroups < 1 || workgroups > 65536 || iters < 1 || iters > (1 << 24))
    return fail_msg(CW_ERR_UNSUPPORTED, "workgroups must be in [1, 65536], iters in [1, 2^24]");
  int random = 0;
  switch (operands) {
    case CW_CEILING_LOW_ENTROPY: random = 0; break;
    case CW_CEILING_RANDOM: random = 1; break;
    default: return fail_msg(CW_ERR_UNSUPPORTED, "operands must be CW_CEILING_LOW_ENTROPY or CW_CEILING_RANDOM");
  }
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(workgroups), dim3(512), 0, stream, iters, random, sink);
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
