// Internal types shared by the host front end, the planner and the kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

#include <type_traits>

namespace cw {

// Tile shape of the extend kernel: a workgroup of LDS_WAVES wave64s owns
// LDS_BLOCK_M packed query rows (row = token * G + group member, 32 per wave)
// of one (sequence, kv head) and walks keys BLOCK_N at a time; one workgroup
// is resident per CU.
constexpr int BLOCK_N = 64;
constexpr int LDS_WAVES = 8;
constexpr int LDS_THREADS = LDS_WAVES * 64;
constexpr int LDS_BLOCK_M = LDS_WAVES * 32;

// Per-sequence metadata on the device.
struct SeqInfo {
  int32_t lp;      // cached prefix length
  int32_t ls;      // suffix length
  int32_t cu;      // first packed token row of the sequence
  int32_t bt_row;  // its row of the block table
};

// One workgroup's share of the extend: packed query rows
// [q_row0, q_row0 + rows) of sequence `seq`, kv head `kvh`, keys
// [kv_begin, kv_end).  part >= 0 writes an unnormalised split-K partial.
struct WorkItem {
  int32_t seq;  // -1: idle padding item
  int32_t kvh;
  int32_t q_row0;
  int32_t kv_begin;
  int32_t kv_end;
  int32_t part;
  int32_t rows;
  int32_t pad;
};

// A query tile whose key range was split: `n_parts` partial slots starting at
// `part0` are merged into the output.
struct CombineGroup {
  int32_t seq;
  int32_t kvh;
  int32_t q_row0;
  int32_t rows;
  int32_t part0;
  int32_t n_parts;
  int32_t pad0;
  int32_t pad1;
};

struct WriteParams {
  const void* k_new;
  const void* v_new;
  void* k_pool;
  void* v_pool;
  const float* k_scale;
  const float* v_scale;
  const int32_t* block_table;
  const SeqInfo* seqs;
  int32_t bt_stride;
  int32_t num_seqs;
  int32_t num_kv_heads;
  int32_t total_tokens;
};

// A work plan small enough to travel in the kernel arguments: the extend and
// merge kernels then read it from there, and no upload kernel runs before them
// (an upload kernel costs ~4 us of the stream's time however small the plan).
constexpr size_t kArgPlanBytes = 16384;
struct ArgPlan {
  uint8_t bytes[kArgPlanBytes];
};
struct NoArgPlan {
  uint8_t unused;
};
template <bool AP>
using PlanArg = typename std::conditional<AP, ArgPlan, NoArgPlan>::type;
// Pointer to a plan array: at byte `off` of the argument plan, or `dev`.
template <bool AP, class T>
__device__ __forceinline__ const T* plan_ptr(const PlanArg<AP>& ap, int32_t off, const T* dev) {
  if constexpr (AP) return reinterpret_cast<const T*>(ap.bytes + off);
  else return dev;
}

struct ExtendParams {
  const void* q;
  const void* k_new;
  const void* v_new;
  const void* k_pool;
  const void* v_pool;
  const float* k_scale;
  const float* v_scale;
  const int32_t* block_table;
  void* out;
  float* lse;
  const SeqInfo* seqs;
  const WorkItem* items;
  const CombineGroup* groups;
  uint16_t* part_o;  // [n_parts, part_rows, D] bf16: the unnormalised partial O
  float* part_ml;  // [n_parts, part_rows, 2]  (running max in log2 units, sum)
  int32_t bt_stride;
  int32_t num_kv_heads;
  int32_t gqa_group;
  int32_t num_seqs;
  float scale_log2;  // softmax_scale * log2(e)
  int32_t n_items;
  int32_t n_groups;
  int32_t part_rows;  // rows per split-K partial slot (the row block for extend, G for decode)
  // with an argument plan: byte offsets in it of seqs, items, groups and the
  // page write's seqs (the device pointers above are then unused); a decode
  // plan in compact form (plan_expand.h) has its ExpandDesc at ap_desc (> 0),
  // and its items and groups are rebuilt from the records where they are read
  int32_t ap_seqs, ap_items, ap_groups, ap_wseqs, ap_desc;
  WriteParams w;      // extend: also scatter the new K/V into the pools when w.total_tokens > 0
};


// Whole-block copies between two block pools (device page pool <-> host block
// pool): block src_ids[i] of (src_k, src_v) goes to block dst_ids[i] of
// (dst_k, dst_v); scales (fp8 pools) likewise, `scales_per_block` floats each.
struct SwapParams {
  const uint8_t* src_k;
  const uint8_t* src_v;
  uint8_t* dst_k;
  uint8_t* dst_v;
  const float* src_ks;  // nullptr: no scales to copy
  const float* src_vs;
  float* dst_ks;
  float* dst_vs;
  const int32_t* src_ids;  // [n], device-visible
  const int32_t* dst_ids;  // [n]
  int32_t n;
  int32_t block_bytes;  // Hkv * P * D * element bytes, a multiple of 16
  int32_t scales_per_block;  // Hkv
};

// Sets the thread-local message returned by cw_last_error_message.
void set_last_error(const char* msg);

// Kernel launchers (each defined in the translation unit of its kernel).
// `ap`: the plan in the kernel arguments (nullptr: read through p's pointers).
hipError_t launch_extend_lds(const ExtendParams& p, int head_dim, int page_size, bool fp8,
                             hipStream_t stream, const ArgPlan* ap = nullptr);
hipError_t launch_extend_w64(const ExtendParams& p, int head_dim, int page_size, hipStream_t stream,
                             const ArgPlan* ap = nullptr);
hipError_t launch_combine(const ExtendParams& p, int head_dim, int max_parts, hipStream_t stream,
                          const ArgPlan* ap = nullptr);
hipError_t launch_decode(const ExtendParams& p, int head_dim, int page_size, bool fp8,
                         hipStream_t stream, const ArgPlan* ap = nullptr);
int decode_keys_per_tile(int head_dim, bool fp8);
int decode_waves_per_cu(bool fp8);  // resident decode waves per CU (LDS-bound)
hipError_t launch_write_pages(const WriteParams& p, int head_dim, int page_size, bool fp8,
                              hipStream_t stream);
hipError_t launch_swap(const SwapParams& p, hipStream_t stream);
// Copies `bytes` from device-visible pinned host memory to device memory on
// `stream` with a kernel (the plan upload).  With `done` (device address of
// pinned host words), each of its *workgroups (at most kMaxUploadWorkgroups)
// writes `seq` into done[its index] once it has read its share.
constexpr int32_t kMaxUploadWorkgroups = 1024;
hipError_t launch_stage_copy(const void* src, void* dst, size_t bytes, hipStream_t stream,
                             uint32_t* done = nullptr, uint32_t seq = 0, int32_t* workgroups = nullptr);
// Plan bytes carried in kernel arguments, kArgChunkBytes per launch (bytes a
// multiple of 4; for calls captured into a graph).
constexpr size_t kArgChunkBytes = 2048;
hipError_t launch_arg_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);
hipError_t launch_check_table(const int32_t* bt, int32_t bt_stride, int32_t num_pages,
                              const SeqInfo* seqs, int32_t num_seqs, int32_t page_size,
                              int32_t* bad, hipStream_t stream);

}  // namespace cw
