// KV block manager of the CacheWise host policy; see block_manager.h.
#include "block_manager.h"

#include <algorithm>
#include <limits>

namespace cw {

BlockManager::BlockManager(int32_t capacity_blocks, int32_t block_tokens, int32_t host_blocks)
    : capacity_(capacity_blocks), block_tokens_(block_tokens), blocks_(capacity_blocks),
      host_capacity_(host_blocks), host_out_(host_blocks, -1) {
  free_.reserve(capacity_blocks);
  for (int32_t b = capacity_blocks - 1; b >= 0; --b) free_.push_back(b);  // hands out 0, 1, 2, ...
  host_free_.reserve(host_blocks);
  for (int32_t b = host_blocks - 1; b >= 0; --b) host_free_.push_back(b);
}

void BlockManager::add_session(int32_t s, int32_t group, int32_t shared_tokens) {
  if (s >= static_cast<int32_t>(sess_.size())) sess_.resize(s + 1);
  Session& x = sess_[s];
  x.group = group;
  x.shared = 0;
  if (group >= 0) {
    if (group >= static_cast<int32_t>(groups_.size())) {
      const size_t old = groups_.size();
      groups_.resize(group + 1);
      for (size_t g = old; g < groups_.size(); ++g) groups_[g].shared = -1;
    }
    Group& g = groups_[group];
    if (g.shared < 0) g.shared = shared_tokens / block_tokens_;
    x.shared = g.shared;
  }
}

int32_t BlockManager::resident_run(int32_t s) const {
  const Session& x = sess_[s];
  if (x.group < 0) return static_cast<int32_t>(x.priv.size());
  const Group& g = groups_[x.group];
  const int32_t rs = static_cast<int32_t>(g.blocks.size());
  if (rs < x.shared) return rs;
  return x.shared + static_cast<int32_t>(x.priv.size());
}

int32_t BlockManager::block_at(int32_t s, int32_t pos) const {
  const Session& x = sess_[s];
  return pos < x.shared ? groups_[x.group].blocks[pos] : x.priv[pos - x.shared];
}

int64_t BlockManager::referenced_blocks() const { return referenced_; }

void BlockManager::ref(int32_t b) {
  if (blocks_[b].ref++ == 0) ++referenced_;
}
void BlockManager::unref(int32_t b) {
  if (--blocks_[b].ref == 0) --referenced_;
}

void BlockManager::table(int32_t s, std::vector<int32_t>* ids) const {
  const int32_t k = resident_run(s);
  ids->resize(k);
  for (int32_t p = 0; p < k; ++p) (*ids)[p] = block_at(s, p);
}

// A shared block's value: the smallest value among the group's attached
// sessions, and the largest id among those that have it.
bool BlockManager::group_key(int32_t g, double* v, int32_t* s) const {
  bool any = false;
  for (int32_t m : groups_[g].members) {
    const double x = sess_[m].value;
    if (!any || x < *v || (x == *v && m > *s)) {
      *v = x;
      *s = m;
      any = true;
    }
  }
  return any;
}

std::vector<int32_t>& BlockManager::run_of(int32_t owner) {
  return owner >= 0 ? sess_[owner].priv : groups_[-1 - owner].blocks;
}

std::vector<int32_t>& BlockManager::host_run_of(int32_t owner) {
  return owner >= 0 ? sess_[owner].hpriv : groups_[-1 - owner].hblocks;
}

// Frees the owner's host-held run (and, for a group, its sharers' host-held
// private runs): they no longer follow a leading run.  Copies into them that
// the current admission listed are cancelled: their data is never read.
void BlockManager::drop_host_run(int32_t owner) {
  auto release = [&](std::vector<int32_t>& run) {
    for (auto it = run.rbegin(); it != run.rend(); ++it) {
      const int32_t hb = *it;
      if (host_out_[hb] >= 0) {
        swap_out_[host_out_[hb]].host = -1;
        host_out_[hb] = -1;
      }
      host_free_.push_back(hb);
    }
    run.clear();
  };
  release(host_run_of(owner));
  if (owner < 0)
    for (int32_t m : groups_[-1 - owner].members) release(sess_[m].hpriv);
}

// Moves the whole host-held run back to device blocks (lowest position first),
// referenced by the admitting request, recording the swaps.
void BlockManager::swap_in_run(std::vector<int32_t>& host_run, std::vector<int32_t>& run, Kind kind,
                               int32_t owner, int32_t* pos) {
  while (!host_run.empty()) {
    const int32_t hb = host_run.back();
    host_run.pop_back();
    const int32_t b = free_.back();
    free_.pop_back();
    Block& bl = blocks_[b];
    bl.kind = kind;
    bl.owner = owner;
    bl.pos = (*pos)++;
    bl.ref = 1;
    ++referenced_;
    run.push_back(b);
    host_free_.push_back(hb);
    swap_in_.push_back(Swap{b, hb});
  }
}

// (Re)enters the run's tail block into the heap; older entries of the run are
// stale from now on.  A referenced run has no entry.
void BlockManager::push(int32_t owner) {
  uint32_t& version = owner >= 0 ? sess_[owner].version : groups_[-1 - owner].version;
  ++version;
  const std::vector<int32_t>& run = run_of(owner);
  if (run.empty() || blocks_[run.back()].ref != 0) return;
  double v = 0.0;
  int32_t s = 0;
  if (owner >= 0) {
    v = sess_[owner].value;
    s = owner;
  } else if (!group_key(-1 - owner, &v, &s)) {
    return;  // a group with resident blocks always has an attached member
  }
  heap_.push(Entry{v, -s, blocks_[run.back()].pos, owner, version});
}

void BlockManager::rebuild() {
  heap_ = std::priority_queue<Entry>();
  for (int32_t s = 0; s < static_cast<int32_t>(sess_.size()); ++s) push(s);
  for (int32_t g = 0; g < static_cast<int32_t>(groups_.size()); ++g) push(-1 - g);
}

bool BlockManager::evict_one() {
  while (!heap_.empty()) {
    const Entry e = heap_.top();
    heap_.pop();
    const uint32_t version = e.owner >= 0 ? sess_[e.owner].version : groups_[-1 - e.owner].version;
    std::vector<int32_t>& run = run_of(e.owner);
    if (e.version != version || run.empty() || blocks_[run.back()].ref != 0) continue;  // stale
    const int32_t b = run.back();
    run.pop_back();
    blocks_[b].kind = kFree;
    blocks_[b].owner = -1;
    free_.push_back(b);
    if (host_capacity_ > 0) {
      // to the host pool while it has room, unless no one will use the block
      // again (value +inf): it then leads the owner's host-held run
      if (!host_free_.empty() && e.v != std::numeric_limits<double>::infinity()) {
        const int32_t hb = host_free_.back();
        host_free_.pop_back();
        host_run_of(e.owner).push_back(hb);
        host_out_[hb] = static_cast<int32_t>(swap_out_.size());
        swap_out_.push_back(Swap{b, hb});
      } else {
        drop_host_run(e.owner);
      }
    }
    push(e.owner);  // the run's new tail
    return true;
  }
  return false;
}

bool BlockManager::admit(int32_t s, int64_t context_tokens, int64_t input_tokens,
                         int64_t output_tokens, Admission* out) {
  Session& x = sess_[s];
  const int64_t B = block_tokens_;
  const int64_t d = (context_tokens + input_tokens + output_tokens + B - 1) / B;
  const int32_t k = resident_run(s);
  const int64_t a = d - k;
  // feasible: free blocks plus every unreferenced resident block outside the run
  for (int32_t p = 0; p < k; ++p) ref(block_at(s, p));
  if (d > capacity_ || static_cast<int64_t>(free_.size()) + (resident_blocks() - referenced_) < a) {
    for (int32_t p = 0; p < k; ++p) unref(block_at(s, p));  // their heap entries are still valid
    return false;
  }
  int64_t evicted = 0;
  swap_out_.clear();
  swap_in_.clear();
  while (static_cast<int64_t>(free_.size()) < a) {
    if (!evict_one()) {  // unreachable: the heap holds every evictable block
      for (const Swap& w : swap_out_)
        if (w.host >= 0) host_out_[w.host] = -1;
      return false;
    }
    ++evicted;
  }
  // the copies that still matter (each host block written at most once)
  size_t kept = 0;
  for (const Swap& w : swap_out_) {
    if (w.host < 0) continue;
    host_out_[w.host] = -1;
    swap_out_[kept++] = w;
  }
  swap_out_.resize(kept);
  // the host-held run comes back first, in position order
  int32_t pos = k;
  if (host_capacity_ > 0) {
    if (x.group >= 0 && static_cast<int32_t>(groups_[x.group].blocks.size()) < x.shared) {
      Group& g = groups_[x.group];
      swap_in_run(g.hblocks, g.blocks, kShared, x.group, &pos);
    }
    if (x.group < 0 || static_cast<int32_t>(groups_[x.group].blocks.size()) >= x.shared)
      swap_in_run(x.hpriv, x.priv, kPrivate, s, &pos);
  }
  for (int64_t p = pos; p < d; ++p) {
    const int32_t b = free_.back();
    free_.pop_back();
    Block& bl = blocks_[b];
    bl.ref = 1;
    ++referenced_;
    bl.pos = static_cast<int32_t>(p);
    if (p < x.shared) {
      bl.kind = kShared;
      bl.owner = x.group;
      groups_[x.group].blocks.push_back(b);
    } else {
      bl.kind = kPrivate;
      bl.owner = s;
      x.priv.push_back(b);
    }
  }
  if (x.group >= 0 && !x.attached) groups_[x.group].members.push_back(s);
  x.attached = true;
  x.running = true;
  x.run_blocks = static_cast<int32_t>(d);
  out->resident_before = k;
  out->blocks = static_cast<int32_t>(d);
  out->cached_tokens = std::min<int64_t>(int64_t(pos) * B, std::max<int64_t>(context_tokens, int64_t(x.shared) * B));
  out->evicted = evicted;
  out->swapped_out = static_cast<int32_t>(swap_out_.size());
  out->swapped_in = static_cast<int32_t>(swap_in_.size());
  return true;
}

void BlockManager::release(int32_t s, double value) {
  Session& x = sess_[s];
  x.value = value;
  if (!x.running) return;
  x.running = false;
  for (int32_t p = 0; p < x.run_blocks; ++p) unref(block_at(s, p));
  x.run_blocks = 0;
  push(s);
  if (x.group >= 0) push(-1 - x.group);  // the group's value may have changed
}

}  // namespace cw
