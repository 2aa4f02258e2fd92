// KV block manager of the CacheWise host policy (CacheWise Sec. 4 and 5.3).
//
// A node's M physical KV blocks of B tokens.  Every block is free, or resident
// and owned by one session (private) or by a shared-prefix group (the whole
// blocks of a prefix common to the group's members, one copy).  A resident
// block carries a reference count: the running requests that use it.  When a
// request is released its blocks' counts drop, and blocks left unreferenced
// enter the eviction heap keyed by their owner's eviction value (larger evicts
// first); the heap is rebuilt from the current values on request (the periodic
// rebuild every N_rebuild engine iterations).
//
// Keys: a private block of session s at logical position p has key
// (value_s, -s, p); a shared block's value is the smallest value among the
// sessions attached to its group (the sharer that needs it soonest), with the
// largest id among the sharers that have it.  So a session's blocks leave tail
// first and every sharer's private blocks leave before the shared blocks they
// follow: resident blocks always form a leading run of every context, and an
// evicted block is always the tail of its owner's run.  The blocks of one run
// share their value and id and are ordered by position, and a run is
// referenced as a whole (a running request references all of it), so the heap
// holds one entry per run, for its tail block: the block order above at
// O(log runs) per eviction.
//
// Offload (a host pool of host_blocks > 0 blocks; CacheWise Sec. 6.4): an
// evicted block is copied to a free host block (a swap out) and joins its
// owner's host-held run, which follows the resident run; with no free host
// block it is dropped, and with it the owner's host-held run (past it, so no
// longer part of a leading run; for a shared block also the sharers' host-held
// private runs).  An admission swaps the requesting context's host-held run
// back in (shared blocks, then private ones once the shared run is complete)
// after the evictions that make room.  Each admission records its swaps, outs
// before ins: a caller copies them in that order before the request's kernels.
#pragma once

#include <stdint.h>

#include <queue>
#include <vector>

namespace cw {

class BlockManager {
 public:
  struct Admission {
    int32_t resident_before = 0;  // leading resident blocks found (k)
    int32_t blocks = 0;           // blocks of the request (d)
    int64_t cached_tokens = 0;    // prompt tokens whose K/V were resident or swapped in
    int64_t evicted = 0;          // blocks evicted to make room
    int32_t swapped_out = 0;      // of them, copied to the host pool
    int32_t swapped_in = 0;       // blocks of the request brought back from the host pool
  };
  struct Swap {
    int32_t device;  // page of the device pool
    int32_t host;    // block of the host pool
  };

  BlockManager(int32_t capacity_blocks, int32_t block_tokens, int32_t host_blocks = 0);

  // Registers session s (ids 0, 1, ...) in shared-prefix group g (-1: none)
  // whose members share their first shared_tokens tokens.  Sessions are
  // registered before their first admission; a group's shared token count is
  // fixed by its first member.
  void add_session(int32_t s, int32_t group, int32_t shared_tokens);

  // Leading resident blocks of session s's context (shared blocks count even
  // before its first request).
  int32_t resident_run(int32_t s) const;
  int32_t shared_blocks(int32_t s) const { return sess_[s].shared; }
  int64_t free_blocks() const { return static_cast<int64_t>(free_.size()); }
  int64_t resident_blocks() const { return capacity_ - free_blocks(); }
  int64_t referenced_blocks() const;
  // Blocks of a request of `tokens` context + input + output tokens.
  int64_t blocks_for(int64_t tokens) const { return (tokens + block_tokens_ - 1) / block_tokens_; }
  // The fewest blocks a request of session s may have: its group's shared
  // blocks and every private block it holds, resident or on the host (a
  // context only grows).
  int64_t min_blocks(int32_t s) const {
    const Session& x = sess_[s];
    return int64_t(x.shared) + int64_t(x.priv.size()) + int64_t(x.hpriv.size());
  }

  // Admits a request of session s: its context holds context_tokens tokens,
  // the request adds input_tokens and output_tokens.  References the resident
  // leading run, evicts unreferenced blocks of others (largest key first)
  // until the missing blocks fit, allocates and references them.  Returns
  // false (nothing changed) when the request cannot fit even after evicting
  // every unreferenced block.
  bool admit(int32_t s, int64_t context_tokens, int64_t input_tokens, int64_t output_tokens,
             Admission* out);
  // Physical ids of session s's resident blocks in logical order.
  void table(int32_t s, std::vector<int32_t>* ids) const;
  // Releases session s's running request: its blocks lose one reference and
  // those left unreferenced become evictable with the session's eviction value.
  void release(int32_t s, double value);
  // Sets session s's eviction value without touching the heap (see rebuild).
  void set_value(int32_t s, double value) { sess_[s].value = value; }
  // Rebuilds the eviction heap from the current values.
  void rebuild();
  bool is_running(int32_t s) const { return sess_[s].running; }
  // Swaps of the last admission: device -> host (before the ins), host -> device.
  const std::vector<Swap>& swaps_out() const { return swap_out_; }
  const std::vector<Swap>& swaps_in() const { return swap_in_; }
  int32_t host_capacity() const { return host_capacity_; }
  int64_t free_host_blocks() const { return static_cast<int64_t>(host_free_.size()); }

 private:
  enum Kind : uint8_t { kFree = 0, kPrivate = 1, kShared = 2 };
  struct Block {
    Kind kind = kFree;
    int32_t owner = -1;  // session (private) or group (shared)
    int32_t pos = 0;     // logical position in its context
    int32_t ref = 0;
  };
  struct Session {
    int32_t group = -1;
    int32_t shared = 0;            // whole shared blocks (G)
    std::vector<int32_t> priv;     // resident private blocks, positions shared ..
    std::vector<int32_t> hpriv;    // host-held private blocks after them (back(): lowest position)
    double value = 0.0;
    bool attached = false;         // has run at least one request
    bool running = false;
    int32_t run_blocks = 0;        // blocks referenced by its running request
    uint32_t version = 0;          // of its heap entry
  };
  struct Group {
    int32_t shared = 0;
    std::vector<int32_t> blocks;   // resident shared blocks, positions 0 ..
    std::vector<int32_t> hblocks;  // host-held shared blocks after them (back(): lowest position)
    std::vector<int32_t> members;  // attached sessions
    uint32_t version = 0;
  };
  // heap entry of a run: owner s >= 0 is session s's private run, -1 - g group g's
  struct Entry {
    double v;
    int32_t neg_s;
    int32_t pos;
    int32_t owner;
    uint32_t version;
    bool operator<(const Entry& o) const {
      if (v != o.v) return v < o.v;
      if (neg_s != o.neg_s) return neg_s < o.neg_s;
      return pos < o.pos;
    }
  };

  void push(int32_t owner);
  std::vector<int32_t>& run_of(int32_t owner);
  std::vector<int32_t>& host_run_of(int32_t owner);
  void drop_host_run(int32_t owner);
  void swap_in_run(std::vector<int32_t>& host_run, std::vector<int32_t>& run, Kind kind, int32_t owner,
                   int32_t* pos);
  void ref(int32_t b);
  void unref(int32_t b);
  bool group_key(int32_t g, double* v, int32_t* s) const;
  bool evict_one();
  int32_t block_at(int32_t s, int32_t pos) const;

  int32_t capacity_, block_tokens_;
  std::vector<Block> blocks_;
  std::vector<int32_t> free_;  // stack of free block ids
  std::vector<Session> sess_;
  std::vector<Group> groups_;
  std::priority_queue<Entry> heap_;
  int64_t referenced_ = 0;  // resident blocks with a reference
  int32_t host_capacity_;
  std::vector<int32_t> host_free_;  // stack of free host block ids
  std::vector<Swap> swap_out_, swap_in_;
  // per host block: its entry in swap_out_ while the admission that wrote it
  // runs its evictions (-1 otherwise); a drop cancels that copy
  std::vector<int32_t> host_out_;
};

}  // namespace cw
