// Debug check of the block table: per sequence, the number of entries that an
// attention or page-write call would read (pages 0 .. ceil((Lp + Ls) / P) - 1)
// and that lie outside [0, num_pages).  One workgroup per sequence (grid-stride
// over sequences), a fixed-order reduction, one count written per sequence.
#include <hip/hip_runtime.h>

#include "../cw_internal.h"

namespace cw {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void check_table_kernel(const int32_t* bt, int32_t bt_stride,
                                                               int32_t num_pages,
                                                               const SeqInfo* seqs,
                                                               int32_t num_seqs, int32_t page_size,
                                                               int32_t* bad) {
  __shared__ int32_t part[kThreads / 64];
  for (int b = blockIdx.x; b < num_seqs; b += gridDim.x) {
    const SeqInfo sq = seqs[b];
    const int64_t n = (int64_t(sq.lp) + sq.ls + page_size - 1) / page_size;
    const int32_t* row = bt + size_t(sq.bt_row) * bt_stride;
    int32_t c = 0;
    for (int64_t j = threadIdx.x; j < n; j += kThreads) {
      const int32_t id = row[j];
      c += (id < 0 || id >= num_pages) ? 1 : 0;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
      int32_t t = 0;
      for (int w = 0; w < kThreads / 64; ++w) t += part[w];
      bad[b] = t;
    }
    __syncthreads();  // part[] is reused by the next sequence
  }
}

}  // namespace

hipError_t launch_check_table(const int32_t* bt, int32_t bt_stride, int32_t num_pages,
                              const SeqInfo* seqs, int32_t num_seqs, int32_t page_size,
                              int32_t* bad, hipStream_t stream) {
  if (num_seqs <= 0) return hipSuccess;
  const int grid = num_seqs < 65535 ? num_seqs : 65535;
  hipLaunchKernelGGL(check_table_kernel, dim3(grid), dim3(kThreads), 0, stream, bt, bt_stride,
                     num_pages, seqs, num_seqs, page_size, bad);
  return hipGetLastError();
}

}  // namespace cw
