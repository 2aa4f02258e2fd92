// CacheWise host policy: prefix-aware scheduling and predictive eviction over
// the KV block manager (block_manager.h), simulated over closed-loop agent
// sessions (see cw_policy.h for the model), and the block manager's C ABI.
// Paper anchors: Sec. 4 (formal model: capacity M, resident prefix
// k_i, new blocks a_i = d_i - k_i, eviction when the working set exceeds M),
// Sec. 5.1 (dispatch the request with the fewest a_i), Sec. 5.2 (evict in
// decreasing order of the predicted time to next reuse, from tool-duration
// histories conditioned on the time already elapsed), Sec. 5.3 (one priority
// per session, set when its blocks become unreferenced, recomputed for every
// unreferenced session every N_rebuild engine iterations).
#include <cmath>
#include <cstdarg>
#include <exception>
#include <new>
#include <cstdio>
#include <limits>
#include <vector>

#include <memory>

#include "../../../include/cw_policy.h"
#include "../cw_internal.h"
#include "block_manager.h"

namespace cw {
namespace {

constexpr double kInf = std::numeric_limits<double>::infinity();
constexpr int32_t kMaxBlocks = int32_t(1) << 26;  // capacity_blocks (1 GiB of block records)
constexpr int32_t kMaxIds = int32_t(1) << 24;     // block manager session and group ids
constexpr int64_t kMaxTokens = int64_t(1) << 40;  // token counts of one request

cw_status_t policy_fail(cw_status_t s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  set_last_error(buf);
  return s;
}

// Expected remaining duration of a call of tool type y that has run for e
// seconds: mean of (x - e) over the history samples x > e; e when there is none.
double predict_remaining(const cw_sim_trace_t& tr, int32_t y, double e) {
  double sum = 0.0;
  int64_t n = 0;
  for (int32_t k = tr.hist_off[y]; k < tr.hist_off[y + 1]; ++k) {
    if (tr.hist_s[k] > e) {
      sum += tr.hist_s[k] - e;
      ++n;
    }
  }
  return n > 0 ? sum / double(n) : e;
}

cw_status_t check_trace(const cw_sim_trace_t& tr, const cw_sim_config_t* cfg) {
  if (tr.num_sessions < 0) return policy_fail(CW_ERR_BAD_LENS, "num_sessions = %d", tr.num_sessions);
  if (tr.num_tools < 0) return policy_fail(CW_ERR_BAD_LENS, "num_tools = %d", tr.num_tools);
  if (!tr.turn_off || !tr.hist_off) return policy_fail(CW_ERR_NULL, "turn_off and hist_off are required");
  if (tr.turn_off[0] != 0 || tr.hist_off[0] != 0)
    return policy_fail(CW_ERR_BAD_LENS, "offset arrays must start at 0");
  for (int32_t s = 0; s < tr.num_sessions; ++s)
    if (tr.turn_off[s + 1] < tr.turn_off[s]) return policy_fail(CW_ERR_BAD_LENS, "turn_off decreases at %d", s);
  for (int32_t y = 0; y < tr.num_tools; ++y)
    if (tr.hist_off[y + 1] < tr.hist_off[y]) return policy_fail(CW_ERR_BAD_LENS, "hist_off decreases at %d", y);
  const int32_t turns = tr.turn_off[tr.num_sessions];
  if (tr.num_sessions > 0 && !tr.session_start) return policy_fail(CW_ERR_NULL, "session_start is required");
  if (turns > 0 && (!tr.in_tokens || !tr.out_tokens || !tr.tool || !tr.tool_s))
    return policy_fail(CW_ERR_NULL, "per-turn arrays are required");
  if (tr.hist_off[tr.num_tools] > 0 && !tr.hist_s) return policy_fail(CW_ERR_NULL, "hist_s is required");
  for (int32_t k = 0; k < tr.hist_off[tr.num_tools]; ++k)
    if (!(tr.hist_s[k] >= 0.0) || !std::isfinite(tr.hist_s[k]))
      return policy_fail(CW_ERR_BAD_LENS, "history sample %d = %g", k, tr.hist_s[k]);
  if (tr.num_groups < 0) return policy_fail(CW_ERR_BAD_LENS, "num_groups = %d", tr.num_groups);
  if (tr.num_groups > 0 && (!tr.session_group || !tr.group_shared_tokens))
    return policy_fail(CW_ERR_NULL, "session_group and group_shared_tokens are required with groups");
  for (int32_t g = 0; g < tr.num_groups; ++g)
    if (tr.group_shared_tokens[g] < 0)
      return policy_fail(CW_ERR_BAD_LENS, "group %d shares %d tokens", g, tr.group_shared_tokens[g]);
  for (int32_t s = 0; s < tr.num_sessions; ++s) {
    if (!(tr.session_start[s] >= 0.0) || !std::isfinite(tr.session_start[s]))
      return policy_fail(CW_ERR_BAD_LENS, "session %d starts at %g", s, tr.session_start[s]);
    const int32_t g = tr.num_groups > 0 ? tr.session_group[s] : -1;
    if (g < -1 || g >= tr.num_groups)
      return policy_fail(CW_ERR_BAD_LENS, "session %d: group %d of %d", s, g, tr.num_groups);
    if (g >= 0 && tr.turn_off[s + 1] > tr.turn_off[s] && tr.in_tokens[tr.turn_off[s]] < tr.group_shared_tokens[g])
      return policy_fail(CW_ERR_BAD_LENS, "session %d: first input shorter than its group's shared prefix", s);
    int64_t ctx = 0;
    for (int32_t j = tr.turn_off[s]; j < tr.turn_off[s + 1]; ++j) {
      if (tr.in_tokens[j] < 0 || tr.out_tokens[j] < 0)
        return policy_fail(CW_ERR_BAD_LENS, "turn %d has negative token counts", j);
      const bool last = j + 1 == tr.turn_off[s + 1];
      if (!last && (tr.tool[j] < 0 || tr.tool[j] >= tr.num_tools))
        return policy_fail(CW_ERR_BAD_LENS, "turn %d: tool type %d of %d", j, tr.tool[j], tr.num_tools);
      if (!last && (!(tr.tool_s[j] >= 0.0) || !std::isfinite(tr.tool_s[j])))
        return policy_fail(CW_ERR_BAD_LENS, "turn %d: tool duration %g", j, tr.tool_s[j]);
      ctx += int64_t(tr.in_tokens[j]) + tr.out_tokens[j];
      if (cfg && (ctx + cfg->block_tokens - 1) / cfg->block_tokens > cfg->capacity_blocks)
        return policy_fail(CW_ERR_BAD_LENS, "session %d needs more than %d blocks at turn %d", s,
                           cfg->capacity_blocks, j);
    }
  }
  return CW_OK;
}

enum State { kWaiting, kQueued, kRunning, kDone };

struct Session {
  int32_t first = 0, n = 0;  // turns [first, first + n)
  int32_t next = 0;          // next turn (index within the session)
  int64_t ctx = 0;           // context tokens
  State state = kWaiting;
  double arrival = 0.0;      // arrival of the pending request
  double last_use = 0.0;     // end of its last request
  double tool_start = 0.0;   // start of its current tool call
  int32_t tool = 0;          // type of its current tool call
  double priority = 0.0;     // predictive eviction priority (stale between rebuilds)
  double done_at = 0.0;
};

}  // namespace
}  // namespace cw

using namespace cw;

extern "C" {

cw_status_t cw_policy_predict(const cw_sim_trace_t* trace, int32_t tool, double elapsed_s,
                              double* remaining_s) {
  if (!trace || !remaining_s) return policy_fail(CW_ERR_NULL, "trace and remaining_s are required");
  cw_status_t st = check_trace(*trace, nullptr);
  if (st != CW_OK) return st;
  if (tool < 0 || tool >= trace->num_tools) return policy_fail(CW_ERR_BAD_LENS, "tool type %d", tool);
  if (!(elapsed_s >= 0.0) || !std::isfinite(elapsed_s))
    return policy_fail(CW_ERR_BAD_LENS, "elapsed_s = %g", elapsed_s);
  *remaining_s = predict_remaining(*trace, tool, elapsed_s);
  return CW_OK;
}

}  // extern "C"

namespace {

// Runs `f` and turns a failed host allocation (or any other C++ exception)
// into a status: nothing is thrown across the C ABI.
template <class F>
cw_status_t guarded(F&& f) {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    return policy_fail(CW_ERR_UNSUPPORTED, "out of host memory");
  } catch (const std::exception& e) {
    return policy_fail(CW_ERR_UNSUPPORTED, "%s", e.what());
  }
}

cw_status_t check_config(const cw_sim_config_t& c) {
  if (c.capacity_blocks < 1 || c.capacity_blocks > kMaxBlocks || c.block_tokens < 1 || !(c.prefill_s_per_token >= 0.0) ||
      !(c.decode_s_per_token >= 0.0) || !std::isfinite(c.prefill_s_per_token) ||
      !std::isfinite(c.decode_s_per_token) || c.rebuild_every < 1 ||
      (c.sched != CW_SCHED_FCFS && c.sched != CW_SCHED_PREFIX_AWARE) ||
      (c.evict != CW_EVICT_LRU && c.evict != CW_EVICT_PREDICTIVE && c.evict != CW_EVICT_BELADY) ||
      c.host_blocks < 0 || c.host_blocks > kMaxBlocks || !(c.swap_s_per_block >= 0.0) ||
      !std::isfinite(c.swap_s_per_block))
    return policy_fail(CW_ERR_UNSUPPORTED, "invalid simulation configuration");
  return CW_OK;
}

// The simulation proper; `log` may be null.
cw_status_t simulate(const cw_sim_config_t& c, const cw_sim_trace_t& tr, cw_sim_result_t* result,
                     int32_t* dispatch, int64_t dispatch_capacity, cw_sim_log_t* log) {
  const int32_t S = tr.num_sessions;
  const int64_t B = c.block_tokens;
  std::vector<Session> ss(S);
  BlockManager bm(c.capacity_blocks, c.block_tokens, c.host_blocks);
  int64_t total_tokens = 0;
  for (int32_t s = 0; s < S; ++s) {
    ss[s].first = tr.turn_off[s];
    ss[s].n = tr.turn_off[s + 1] - tr.turn_off[s];
    ss[s].arrival = tr.session_start[s];
    const int32_t g = tr.num_groups > 0 ? tr.session_group[s] : -1;
    bm.add_session(s, g, g >= 0 ? tr.group_shared_tokens[g] : 0);
    if (ss[s].n == 0) {
      ss[s].state = kDone;
      ss[s].done_at = tr.session_start[s];
      ss[s].priority = kInf;
      bm.set_value(s, c.evict == CW_EVICT_LRU ? -0.0 : kInf);
    }
    for (int32_t j = ss[s].first; j < ss[s].first + ss[s].n; ++j)
      total_tokens += int64_t(tr.in_tokens[j]) + tr.out_tokens[j];
  }
  if (log) log->written = 0;

  cw_sim_result_t r{};
  int64_t dispatches = 0, table_used = 0;
  int32_t running = -1;
  double run_end = 0.0, t = 0.0;
  std::vector<int32_t> ids;

  // time to next use of session k's blocks as Belady's rule sees it
  auto true_next_use = [&](const Session& k) {
    if (k.state == kDone) return kInf;
    if (k.state == kQueued) return 0.0;
    return std::max(0.0, k.arrival - t);
  };
  // the periodic rebuild: every unreferenced session's priority re-estimated
  auto rebuild = [&]() {
    for (int32_t s = 0; s < S; ++s) {
      Session& k = ss[s];
      if (k.state == kDone) k.priority = kInf;
      else if (k.state == kQueued) k.priority = 0.0;
      else if (k.state == kWaiting) k.priority = predict_remaining(tr, k.tool, t - k.tool_start);
      bm.set_value(s, k.priority);
    }
    bm.rebuild();
    ++r.heap_rebuilds;
  };
  auto dispatch_one = [&](int32_t i) -> cw_status_t {
    Session& s = ss[i];
    const int32_t j = s.first + s.next;
    ++dispatches;
    if (c.evict == CW_EVICT_PREDICTIVE && dispatches % c.rebuild_every == 0) rebuild();
    if (c.evict == CW_EVICT_BELADY) {  // Belady's values change with time: fresh keys
      for (int32_t k = 0; k < S; ++k) bm.set_value(k, true_next_use(ss[k]));
      bm.rebuild();
    }
    if (bm.resident_run(i) < (s.ctx + B - 1) / B) ++r.faults;  // part of its context was evicted
    BlockManager::Admission adm;
    if (!bm.admit(i, s.ctx, tr.in_tokens[j], tr.out_tokens[j], &adm))
      return policy_fail(CW_ERR_HIP, "block manager: request of session %d did not fit", i);
    r.evicted_blocks += adm.evicted;
    r.swapped_out_blocks += adm.swapped_out;
    r.swapped_in_blocks += adm.swapped_in;
    const int64_t hit = adm.cached_tokens;
    const int64_t prefill = s.ctx + tr.in_tokens[j] - hit;
    r.recomputed_tokens += std::max<int64_t>(0, s.ctx - hit);
    r.prefilled_tokens += prefill;
    if (log && r.requests < log->capacity) {
      bm.table(i, &ids);
      const int64_t w = r.requests;
      if (w == 0) log->table_off[0] = 0;
      log->session[w] = i;
      log->cached_tokens[w] = static_cast<int32_t>(hit);
      log->new_tokens[w] = static_cast<int32_t>(prefill);
      if (log->swapped_in) log->swapped_in[w] = adm.swapped_in;
      if (log->swapped_out) log->swapped_out[w] = adm.swapped_out;
      const int64_t n = std::min<int64_t>(int64_t(ids.size()), std::max<int64_t>(0, log->table_capacity - table_used));
      for (int64_t q = 0; q < n; ++q) log->tables[table_used + q] = ids[q];
      table_used += n;
      log->table_off[w + 1] = table_used;
      log->written = w + 1;
    }
    s.state = kRunning;
    running = i;
    run_end = t + (c.prefill_s_per_token * double(prefill) + c.decode_s_per_token * double(tr.out_tokens[j]) +
                   c.swap_s_per_block * double(adm.swapped_out + adm.swapped_in));
    if (dispatch && r.requests < dispatch_capacity) dispatch[r.requests] = i;
    ++r.requests;
    return CW_OK;
  };
  auto complete = [&](int32_t i) {
    Session& s = ss[i];
    const int32_t j = s.first + s.next;
    s.ctx += int64_t(tr.in_tokens[j]) + tr.out_tokens[j];
    s.last_use = t;
    ++s.next;
    if (s.next == s.n) {
      s.state = kDone;
      s.done_at = t;
      s.priority = kInf;  // its blocks are never used again
    } else {
      s.state = kWaiting;
      s.tool = tr.tool[j];
      s.tool_start = t;
      s.arrival = t + tr.tool_s[j];
      s.priority = predict_remaining(tr, s.tool, 0.0);  // unreferenced now: fresh estimate
    }
    // its blocks lose their reference and enter the eviction heap
    bm.release(i, c.evict == CW_EVICT_LRU ? -s.last_use : s.priority);
  };

  while (true) {
    for (Session& k : ss)
      if (k.state == kWaiting && k.arrival <= t) k.state = kQueued;
    if (running < 0) {
      int32_t pick = -1;
      int64_t pick_a = 0;
      for (int32_t k = 0; k < S; ++k) {
        if (ss[k].state != kQueued) continue;
        const Session& a = ss[k];
        const int32_t ja = a.first + a.next;
        const int64_t aa = (a.ctx + tr.in_tokens[ja] + tr.out_tokens[ja] + B - 1) / B - bm.resident_run(k);
        bool better = pick < 0;
        if (!better) {
          const Session& b = ss[pick];
          if (c.sched == CW_SCHED_PREFIX_AWARE) better = aa < pick_a || (aa == pick_a && a.arrival < b.arrival);
          else better = a.arrival < b.arrival;
        }
        if (better) {
          pick = k;
          pick_a = aa;
        }
      }
      if (pick >= 0) {
        const cw_status_t st = dispatch_one(pick);
        if (st != CW_OK) return st;
        continue;
      }
    }
    double next = kInf;
    if (running >= 0) next = run_end;
    for (const Session& k : ss)
      if (k.state == kWaiting) next = std::min(next, k.arrival);
    if (next == kInf) break;
    t = std::max(t, next);
    if (running >= 0 && run_end <= t) {
      complete(running);
      running = -1;
    }
  }

  double sum_sessions = 0.0;
  int32_t counted = 0;
  for (int32_t s = 0; s < S; ++s) {
    r.makespan_s = std::max(r.makespan_s, ss[s].done_at);
    if (ss[s].n > 0) {
      sum_sessions += ss[s].done_at - tr.session_start[s];
      ++counted;
    }
  }
  r.mean_session_s = counted > 0 ? sum_sessions / counted : 0.0;
  r.goodput_tok_s = r.makespan_s > 0.0 ? double(total_tokens) / r.makespan_s : 0.0;
  *result = r;
  return CW_OK;
}

}  // namespace

extern "C" {

cw_status_t cw_policy_simulate(const cw_sim_config_t* config, const cw_sim_trace_t* trace,
                               cw_sim_result_t* result, int32_t* dispatch,
                               int64_t dispatch_capacity) {
  if (!config || !trace || !result) return policy_fail(CW_ERR_NULL, "config, trace and result are required");
  cw_status_t st = check_config(*config);
  if (st != CW_OK) return st;
  st = check_trace(*trace, config);
  if (st != CW_OK) return st;
  if (dispatch_capacity < 0) return policy_fail(CW_ERR_BAD_LENS, "dispatch_capacity < 0");
  return guarded([&] { return simulate(*config, *trace, result, dispatch, dispatch_capacity, nullptr); });
}

cw_status_t cw_policy_simulate_log(const cw_sim_config_t* config, const cw_sim_trace_t* trace,
                                   cw_sim_result_t* result, cw_sim_log_t* log) {
  if (!config || !trace || !result || !log) return policy_fail(CW_ERR_NULL, "config, trace, result and log are required");
  cw_status_t st = check_config(*config);
  if (st != CW_OK) return st;
  st = check_trace(*trace, config);
  if (st != CW_OK) return st;
  if (log->capacity < 0 || log->table_capacity < 0)
    return policy_fail(CW_ERR_BAD_LENS, "negative log capacity");
  if (log->capacity > 0 && (!log->session || !log->cached_tokens || !log->new_tokens || !log->table_off))
    return policy_fail(CW_ERR_NULL, "log arrays are required");
  if (log->table_capacity > 0 && !log->tables) return policy_fail(CW_ERR_NULL, "log tables are required");
  return guarded([&] { return simulate(*config, *trace, result, nullptr, 0, log); });
}

struct cw_block_manager {
  std::unique_ptr<BlockManager> bm;
  int32_t sessions = 0;  // registered ids are [0, sessions)
  std::vector<uint8_t> known;
};

static cw_status_t bm_create(int32_t capacity_blocks, int32_t block_tokens, int32_t host_blocks,
                             cw_block_manager_t** out) {
  if (!out) return policy_fail(CW_ERR_NULL, "out is required");
  *out = nullptr;
  if (capacity_blocks < 1 || capacity_blocks > kMaxBlocks || block_tokens < 1 || host_blocks < 0 ||
      host_blocks > kMaxBlocks)
    return policy_fail(CW_ERR_UNSUPPORTED, "capacity_blocks = %d (1 .. %d), block_tokens = %d, host_blocks = %d",
                       capacity_blocks, kMaxBlocks, block_tokens, host_blocks);
  return guarded([&] {
    auto m = std::make_unique<cw_block_manager>();
    m->bm = std::make_unique<BlockManager>(capacity_blocks, block_tokens, host_blocks);
    *out = m.release();
    return CW_OK;
  });
}

cw_status_t cw_bm_create(int32_t capacity_blocks, int32_t block_tokens, cw_block_manager_t** out) {
  return bm_create(capacity_blocks, block_tokens, 0, out);
}

cw_status_t cw_bm_create_with_host_pool(int32_t capacity_blocks, int32_t block_tokens, int32_t host_blocks,
                                        cw_block_manager_t** out) {
  if (host_blocks < 1) {
    if (out) *out = nullptr;
    return policy_fail(CW_ERR_UNSUPPORTED, "host_blocks = %d: a host pool holds at least one block", host_blocks);
  }
  return bm_create(capacity_blocks, block_tokens, host_blocks, out);
}

cw_status_t cw_bm_destroy(cw_block_manager_t* m) {
  delete m;
  return CW_OK;
}

cw_status_t cw_bm_add_session(cw_block_manager_t* m, int32_t session, int32_t group, int32_t shared_tokens) {
  if (!m) return policy_fail(CW_ERR_NULL, "block manager is NULL");
  if (session < 0 || group < -1 || shared_tokens < 0)
    return policy_fail(CW_ERR_BAD_LENS, "session %d, group %d, shared_tokens %d", session, group, shared_tokens);
  if (session >= kMaxIds || group >= kMaxIds)
    return policy_fail(CW_ERR_UNSUPPORTED, "session %d, group %d: ids must be below %d", session, group, kMaxIds);
  if (session < m->sessions && m->known[session])
    return policy_fail(CW_ERR_BAD_LENS, "session %d is already registered", session);
  return guarded([&] {
    if (session >= m->sessions) {
      m->known.resize(session + 1, 0);
      m->sessions = session + 1;
    }
    m->bm->add_session(session, group, shared_tokens);
    m->known[session] = 1;
    return CW_OK;
  });
}

static cw_status_t bm_admit(cw_block_manager_t* m, int32_t session, int64_t context_tokens, int64_t input_tokens,
                            int64_t output_tokens, int32_t* table, int32_t table_capacity, int32_t* blocks,
                            int64_t* cached_tokens, int64_t* evicted_blocks, cw_bm_swaps_t* swaps) {
  if (!blocks || !cached_tokens) return policy_fail(CW_ERR_NULL, "blocks and cached_tokens are required");
  if (session < 0 || session >= m->sessions || !m->known[session])
    return policy_fail(CW_ERR_BAD_LENS, "session %d is not registered", session);
  if (context_tokens < 0 || input_tokens < 0 || output_tokens < 0 || context_tokens > kMaxTokens ||
      input_tokens > kMaxTokens || output_tokens > kMaxTokens)
    return policy_fail(CW_ERR_BAD_LENS, "token counts must lie in [0, 2^40]");
  if (m->bm->is_running(session)) return policy_fail(CW_ERR_BAD_LENS, "session %d already has a request running", session);
  if (table_capacity < 0) return policy_fail(CW_ERR_BAD_LENS, "table_capacity < 0");
  if (m->bm->blocks_for(context_tokens + input_tokens + output_tokens) < m->bm->min_blocks(session))
    return policy_fail(CW_ERR_BAD_LENS,
                       "session %d: the request's %lld blocks do not cover its shared prefix and held blocks (%lld)",
                       session, static_cast<long long>(m->bm->blocks_for(context_tokens + input_tokens + output_tokens)),
                       static_cast<long long>(m->bm->min_blocks(session)));
  if (swaps) {
    if (swaps->capacity < 0) return policy_fail(CW_ERR_BAD_LENS, "swap capacity < 0");
    if (swaps->capacity > 0 && (!swaps->out_device || !swaps->out_host || !swaps->in_host || !swaps->in_device))
      return policy_fail(CW_ERR_NULL, "the four swap arrays are required");
    // every swap of the admission is one of the request's blocks: its block count bounds both lists
    const int64_t need = m->bm->blocks_for(context_tokens + input_tokens + output_tokens);
    if (need > swaps->capacity)
      return policy_fail(CW_ERR_WORKSPACE, "swap lists hold %d entries; the request has %lld blocks", swaps->capacity,
                         static_cast<long long>(need));
  }
  return guarded([&] {
    BlockManager::Admission adm;
    if (!m->bm->admit(session, context_tokens, input_tokens, output_tokens, &adm))
      return policy_fail(CW_ERR_WORKSPACE,
                         "request of session %d does not fit: the referenced blocks would exceed the capacity", session);
    *blocks = adm.blocks;
    *cached_tokens = adm.cached_tokens;
    if (evicted_blocks) *evicted_blocks = adm.evicted;
    if (table) {
      std::vector<int32_t> ids;
      m->bm->table(session, &ids);
      const int32_t n = std::min<int32_t>(table_capacity, static_cast<int32_t>(ids.size()));
      for (int32_t q = 0; q < n; ++q) table[q] = ids[q];
    }
    if (swaps) {
      const auto& so = m->bm->swaps_out();
      const auto& si = m->bm->swaps_in();
      for (size_t q = 0; q < so.size(); ++q) {
        swaps->out_device[q] = so[q].device;
        swaps->out_host[q] = so[q].host;
      }
      for (size_t q = 0; q < si.size(); ++q) {
        swaps->in_host[q] = si[q].host;
        swaps->in_device[q] = si[q].device;
      }
      swaps->n_out = static_cast<int32_t>(so.size());
      swaps->n_in = static_cast<int32_t>(si.size());
    }
    return CW_OK;
  });
}

cw_status_t cw_bm_admit(cw_block_manager_t* m, int32_t session, int64_t context_tokens, int64_t input_tokens,
                        int64_t output_tokens, int32_t* table, int32_t table_capacity, int32_t* blocks,
                        int64_t* cached_tokens, int64_t* evicted_blocks) {
  if (!m) return policy_fail(CW_ERR_NULL, "block manager is NULL");
  if (m->bm->host_capacity() > 0)
    return policy_fail(CW_ERR_UNSUPPORTED, "a manager with a host pool admits through cw_bm_admit_swaps");
  return bm_admit(m, session, context_tokens, input_tokens, output_tokens, table, table_capacity, blocks,
                  cached_tokens, evicted_blocks, nullptr);
}

cw_status_t cw_bm_admit_swaps(cw_block_manager_t* m, int32_t session, int64_t context_tokens, int64_t input_tokens,
                              int64_t output_tokens, int32_t* table, int32_t table_capacity, int32_t* blocks,
                              int64_t* cached_tokens, int64_t* evicted_blocks, cw_bm_swaps_t* swaps) {
  if (!m || !swaps) return policy_fail(CW_ERR_NULL, "block manager and swaps are required");
  swaps->n_out = 0;
  swaps->n_in = 0;
  return bm_admit(m, session, context_tokens, input_tokens, output_tokens, table, table_capacity, blocks,
                  cached_tokens, evicted_blocks, swaps);
}

cw_status_t cw_bm_release(cw_block_manager_t* m, int32_t session, double value) {
  if (!m) return policy_fail(CW_ERR_NULL, "block manager is NULL");
  if (session < 0 || session >= m->sessions || !m->known[session])
    return policy_fail(CW_ERR_BAD_LENS, "session %d is not registered", session);
  if (!m->bm->is_running(session)) return policy_fail(CW_ERR_BAD_LENS, "session %d has no request running", session);
  if (std::isnan(value)) return policy_fail(CW_ERR_BAD_LENS, "eviction value is NaN");
  return guarded([&] {
    m->bm->release(session, value);
    return CW_OK;
  });
}

cw_status_t cw_bm_rebuild(cw_block_manager_t* m, const int32_t* sessions, const double* values, int32_t n) {
  if (!m) return policy_fail(CW_ERR_NULL, "block manager is NULL");
  if (n < 0 || (n > 0 && (!sessions || !values))) return policy_fail(CW_ERR_NULL, "sessions and values are required");
  for (int32_t q = 0; q < n; ++q) {
    if (sessions[q] < 0 || sessions[q] >= m->sessions || !m->known[sessions[q]])
      return policy_fail(CW_ERR_BAD_LENS, "session %d is not registered", sessions[q]);
    if (std::isnan(values[q])) return policy_fail(CW_ERR_BAD_LENS, "eviction value is NaN");
  }
  for (int32_t q = 0; q < n; ++q) m->bm->set_value(sessions[q], values[q]);
  return guarded([&] {
    m->bm->rebuild();
    return CW_OK;
  });
}

cw_status_t cw_bm_stats(cw_block_manager_t* m, int64_t* free_blocks, int64_t* referenced_blocks) {
  if (!m || !free_blocks || !referenced_blocks) return policy_fail(CW_ERR_NULL, "arguments are required");
  *free_blocks = m->bm->free_blocks();
  *referenced_blocks = m->bm->referenced_blocks();
  return CW_OK;
}

cw_status_t cw_bm_host_stats(cw_block_manager_t* m, int64_t* free_host_blocks, int64_t* held_host_blocks) {
  if (!m || !free_host_blocks || !held_host_blocks) return policy_fail(CW_ERR_NULL, "arguments are required");
  *free_host_blocks = m->bm->free_host_blocks();
  *held_host_blocks = m->bm->host_capacity() - m->bm->free_host_blocks();
  return CW_OK;
}

}  // extern "C"
