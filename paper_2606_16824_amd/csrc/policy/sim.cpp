// CacheWise host policy: block manager, prefix-aware scheduling and predictive
// eviction, simulated over closed-loop agent sessions (see cw_policy.h for the
// model).  Paper anchors: Sec. 4 (formal model: capacity M, resident prefix
// k_i, new blocks a_i = d_i - k_i, eviction when the working set exceeds M),
// Sec. 5.1 (dispatch the request with the fewest a_i), Sec. 5.2 (evict in
// decreasing order of the predicted time to next reuse, from tool-duration
// histories conditioned on the time already elapsed), Sec. 5.3 (one priority
// per session, set when its blocks become unreferenced, recomputed for every
// unreferenced session every N_rebuild engine iterations).
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <limits>
#include <vector>

#include "../../../include/cw_policy.h"
#include "../cw_internal.h"

namespace cw {
namespace {

constexpr double kInf = std::numeric_limits<double>::infinity();

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
  for (int32_t s = 0; s < tr.num_sessions; ++s) {
    if (!(tr.session_start[s] >= 0.0) || !std::isfinite(tr.session_start[s]))
      return policy_fail(CW_ERR_BAD_LENS, "session %d starts at %g", s, tr.session_start[s]);
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
  int64_t resident = 0;      // k_i: leading resident blocks
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

cw_status_t cw_policy_simulate(const cw_sim_config_t* config, const cw_sim_trace_t* trace,
                               cw_sim_result_t* result, int32_t* dispatch,
                               int64_t dispatch_capacity) {
  if (!config || !trace || !result) return policy_fail(CW_ERR_NULL, "config, trace and result are required");
  const cw_sim_config_t& c = *config;
  if (c.capacity_blocks < 1 || c.block_tokens < 1 || !(c.prefill_s_per_token >= 0.0) ||
      !(c.decode_s_per_token >= 0.0) || !std::isfinite(c.prefill_s_per_token) ||
      !std::isfinite(c.decode_s_per_token) || c.rebuild_every < 1 ||
      (c.sched != CW_SCHED_FCFS && c.sched != CW_SCHED_PREFIX_AWARE) ||
      (c.evict != CW_EVICT_LRU && c.evict != CW_EVICT_PREDICTIVE && c.evict != CW_EVICT_BELADY))
    return policy_fail(CW_ERR_UNSUPPORTED, "invalid simulation configuration");
  const cw_sim_trace_t& tr = *trace;
  cw_status_t st = check_trace(tr, &c);
  if (st != CW_OK) return st;
  if (dispatch_capacity < 0) return policy_fail(CW_ERR_BAD_LENS, "dispatch_capacity < 0");

  const int32_t S = tr.num_sessions;
  const int64_t B = c.block_tokens, M = c.capacity_blocks;
  std::vector<Session> ss(S);
  int64_t total_tokens = 0;
  for (int32_t s = 0; s < S; ++s) {
    ss[s].first = tr.turn_off[s];
    ss[s].n = tr.turn_off[s + 1] - tr.turn_off[s];
    ss[s].arrival = tr.session_start[s];
    if (ss[s].n == 0) {
      ss[s].state = kDone;
      ss[s].done_at = tr.session_start[s];
      ss[s].priority = kInf;
    }
    for (int32_t j = ss[s].first; j < ss[s].first + ss[s].n; ++j)
      total_tokens += int64_t(tr.in_tokens[j]) + tr.out_tokens[j];
  }

  cw_sim_result_t r{};
  int64_t used = 0;  // resident blocks over all sessions
  int64_t dispatches = 0;
  int32_t running = -1;
  double run_end = 0.0, t = 0.0;

  // time to next use of session k's blocks as Belady's rule sees it
  auto true_next_use = [&](const Session& k) {
    if (k.state == kDone) return kInf;
    if (k.state == kQueued) return 0.0;
    return std::max(0.0, k.arrival - t);
  };
  auto rebuild = [&]() {
    for (Session& k : ss) {
      if (k.state == kDone) k.priority = kInf;
      else if (k.state == kQueued) k.priority = 0.0;
      else if (k.state == kWaiting) k.priority = predict_remaining(tr, k.tool, t - k.tool_start);
    }
    ++r.heap_rebuilds;
  };
  // next victim among the other sessions' resident blocks
  auto victim = [&](int32_t self) {
    int32_t best = -1;
    double best_key = 0.0;
    for (int32_t k = 0; k < S; ++k) {
      if (k == self || ss[k].resident == 0) continue;
      double key;  // larger evicts first
      if (c.evict == CW_EVICT_LRU) key = -ss[k].last_use;
      else if (c.evict == CW_EVICT_PREDICTIVE) key = ss[k].priority;
      else key = true_next_use(ss[k]);
      if (best < 0 || key > best_key) {
        best = k;
        best_key = key;
      }
    }
    return best;
  };
  auto dispatch_one = [&](int32_t i) {
    Session& s = ss[i];
    const int32_t j = s.first + s.next;
    ++dispatches;
    if (c.evict == CW_EVICT_PREDICTIVE && dispatches % c.rebuild_every == 0) rebuild();
    const int64_t need = (s.ctx + tr.in_tokens[j] + tr.out_tokens[j] + B - 1) / B;
    const int64_t a = need - s.resident;
    if (s.resident < (s.ctx + B - 1) / B) ++r.faults;  // part of its context was evicted
    while (M - used < a) {
      const int32_t v = victim(i);  // exists: need <= M
      const int64_t take = std::min(ss[v].resident, a - (M - used));
      ss[v].resident -= take;  // from the tail of its context
      used -= take;
      r.evicted_blocks += take;
    }
    const int64_t recompute = std::max<int64_t>(0, s.ctx - s.resident * B);
    r.recomputed_tokens += recompute;
    r.prefilled_tokens += recompute + tr.in_tokens[j];
    used += need - s.resident;
    s.resident = need;
    s.state = kRunning;
    running = i;
    run_end = t + c.prefill_s_per_token * double(recompute + tr.in_tokens[j]) +
              c.decode_s_per_token * double(tr.out_tokens[j]);
    if (dispatch && r.requests < dispatch_capacity) dispatch[r.requests] = i;
    ++r.requests;
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
  };

  while (true) {
    for (Session& k : ss)
      if (k.state == kWaiting && k.arrival <= t) k.state = kQueued;
    if (running < 0) {
      int32_t pick = -1;
      for (int32_t k = 0; k < S; ++k) {
        if (ss[k].state != kQueued) continue;
        if (pick < 0) {
          pick = k;
          continue;
        }
        const Session &a = ss[k], &b = ss[pick];
        bool better;
        if (c.sched == CW_SCHED_PREFIX_AWARE) {
          const int32_t ja = a.first + a.next, jb = b.first + b.next;
          const int64_t aa = (a.ctx + tr.in_tokens[ja] + tr.out_tokens[ja] + B - 1) / B - a.resident;
          const int64_t ab = (b.ctx + tr.in_tokens[jb] + tr.out_tokens[jb] + B - 1) / B - b.resident;
          better = aa < ab || (aa == ab && a.arrival < b.arrival);
        } else {
          better = a.arrival < b.arrival;
        }
        if (better) pick = k;
      }
      if (pick >= 0) {
        dispatch_one(pick);
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

}  // extern "C"
