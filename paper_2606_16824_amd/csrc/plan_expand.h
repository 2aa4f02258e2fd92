// Decode plans in compact form.  A decode plan is regular: every (sequence,
// kv head) cuts its keys (prefix plus the new token) into chunks of one length,
// the full-length chunks run first in (sequence, head, chunk) order, then the
// shorter last chunks, longest first.  So instead of the work items and merge
// groups themselves, the plan upload can carry one record per sequence and the
// order of the sequences' last chunks, and the upload kernel rebuilds the items
// and groups on the device (a few KB over the host link instead of 32 bytes per
// item); a compact plan small enough for the kernel arguments goes there, and
// the decode and merge kernels rebuild their own item or group.  The same
// functions rebuild them on the host, where the planner's own items check them.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cw_internal.h"

namespace cw {

// One sequence of a decode plan.
struct DecodeRec {
  int32_t full_off;   // items before this sequence's full-length chunks
  int32_t full;       // full-length chunks per kv head
  int32_t nc;         // chunks per kv head (full plus a shorter last one, if any)
  int32_t n;          // keys: the prefix and the new token
  int32_t part_off;   // partial slots before this sequence's (0 if nc == 1)
  int32_t group_off;  // merge groups before this sequence's
};

// What the upload kernel rebuilds, and where.
struct ExpandDesc {
  int32_t n_seqs;
  int32_t n_full;       // full-length chunk items (they come first)
  int32_t n_items;      // all items
  int32_t n_groups;
  int32_t n_tails;      // sequences with a shorter last chunk
  int32_t chunk;        // keys per chunk
  int32_t hkv;
  int32_t rows;         // the GQA group: query rows per item
  uint32_t rec_off;     // source bytes: DecodeRec[n_seqs] at rec_off, then int32 tails[n_tails]
  uint32_t tail_off;
  uint32_t items_off;   // destination bytes of the WorkItem and CombineGroup arrays
  uint32_t groups_off;
};

// Largest b in [0, n) with key(b) <= x (key non-decreasing, key(0) <= x).
template <class Key>
__host__ __device__ inline int32_t last_at_most(int32_t n, int32_t x, Key key) {
  int32_t lo = 0, hi = n - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) / 2;
    if (key(mid) <= x) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// The same search by one whole wave (every lane active, `lane` its index):
// the keys are non-decreasing, so the b with key(b) <= x are a prefix, and
// their count less one is the result; 64 keys per load and ballot instead of
// a chain of dependent loads.
template <class Key>
__device__ inline int32_t wave_last_at_most(int32_t n, int32_t x, int32_t lane, Key key) {
  int32_t count = 0;
  for (int32_t k0 = 0; k0 < n; k0 += 64) {
    const int32_t k = k0 + lane;
    count += __popcll(__ballot(k < n && key(k < n ? k : 0) <= x));
  }
  return __builtin_amdgcn_readfirstlane(count) - 1;
}

// Item i of the plan.  Full-length chunks: the sequence whose range holds i
// (sequences without full chunks have empty ranges, so the last sequence that
// starts at or before i is it), found by the caller as `b_full`; last chunks:
// the i-th of the tail order.
__host__ __device__ inline WorkItem expand_item_at(const DecodeRec* rec, const int32_t* tails,
                                                   const ExpandDesc& d, int32_t i, int32_t b_full) {
  int32_t b, h, c;
  if (i < d.n_full) {
    b = b_full;
    const int32_t r = i - rec[b].full_off;
    h = r / rec[b].full;
    c = r - h * rec[b].full;
  } else {
    const int32_t t = (i - d.n_full) / d.hkv;
    h = (i - d.n_full) - t * d.hkv;
    b = tails[t];
    c = rec[b].nc - 1;
  }
  const DecodeRec& s = rec[b];
  const int64_t begin = int64_t(c) * d.chunk;
  const int64_t end = begin + d.chunk < s.n ? begin + d.chunk : s.n;
  WorkItem w;
  w.seq = b;
  w.kvh = h;
  w.q_row0 = 0;
  w.kv_begin = static_cast<int32_t>(begin);
  w.kv_end = static_cast<int32_t>(end);
  w.part = s.nc > 1 ? s.part_off + h * s.nc + c : -1;
  w.rows = d.rows;
  w.pad = 0;
  return w;
}

// The sequence of full-length chunk item i (i < d.n_full).
__host__ __device__ inline int32_t full_item_seq(const DecodeRec* rec, const ExpandDesc& d, int32_t i) {
  return last_at_most(d.n_seqs, i, [&](int32_t k) { return rec[k].full_off; });
}

__host__ __device__ inline WorkItem expand_item(const DecodeRec* rec, const int32_t* tails,
                                                const ExpandDesc& d, int32_t i) {
  return expand_item_at(rec, tails, d, i, i < d.n_full ? full_item_seq(rec, d, i) : 0);
}

// Merge group g: kv head h of a sequence cut into several chunks, the b-th
// (the last sequence whose groups start at or before g).
__host__ __device__ inline CombineGroup expand_group_at(const DecodeRec* rec, int32_t g, int32_t b, int32_t rows) {
  const DecodeRec& s = rec[b];
  const int32_t h = g - s.group_off;
  CombineGroup cg;
  cg.seq = b;
  cg.kvh = h;
  cg.q_row0 = 0;
  cg.rows = rows;
  cg.part0 = s.part_off + h * s.nc;
  cg.n_parts = s.nc;
  cg.pad0 = 0;
  cg.pad1 = 0;
  return cg;
}

__host__ __device__ inline CombineGroup expand_group(const DecodeRec* rec, const ExpandDesc& d, int32_t g) {
  return expand_group_at(rec, g, last_at_most(d.n_seqs, g, [&](int32_t k) { return rec[k].group_off; }), d.rows);
}

// Upload of a plan blob: its first `verbatim` bytes are copied as they are,
// then the decode plan of `d` is rebuilt into dst (d.n_seqs <= kMaxExpandSeqs).
constexpr int32_t kMaxExpandSeqs = 2048;
// Its workgroups report their reads as launch_stage_copy's do.
hipError_t launch_plan_expand(const void* src, void* dst, size_t verbatim, const ExpandDesc& d,
                              hipStream_t stream, uint32_t* done, uint32_t seq, int32_t* workgroups);

}  // namespace cw
