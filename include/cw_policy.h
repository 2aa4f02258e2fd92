/* CacheWise host policy: a KV block manager with prefix-aware request
 * scheduling and predictive eviction, run as a discrete-event simulation of
 * closed-loop agent sessions on one inference node (CacheWise Sec. 4 formal
 * model, Sec. 5.1 prefix-aware scheduling, Sec. 5.2 predictive eviction and
 * Sec. 5.3 the eviction heap with periodic rebuilds), with the baselines the
 * paper compares against (FCFS scheduling, LRU eviction) and Belady's rule.
 *
 * Host-only C ABI: no HIP call, no allocation visible to the caller; every
 * argument is validated before any work, errors are cw_status_t codes with a
 * thread-local message (cw_last_error_message in cw.h).
 *
 * Model (the readings the paper leaves open are stated in the design notes):
 *  - Session s arrives at session_start[s] and runs its turns in order.  Turn
 *    j appends in_tokens[j] to the session's context and generates
 *    out_tokens[j]; unless it is the session's last turn, a tool call of type
 *    tool[j] then runs for tool_s[j] seconds, after which the next turn arrives.
 *  - The node holds capacity_blocks KV blocks of block_tokens tokens.  A
 *    session's resident blocks are always a leading run of its context (k_i
 *    blocks); a turn needs d_i = ceil((context + in + out) / block_tokens)
 *    blocks, a_i = d_i - k_i of them newly allocated.
 *  - One engine runs one request at a time, without preemption.  When idle it
 *    takes a queued request: FCFS = earliest arrival; prefix-aware = fewest
 *    a_i (then earliest arrival).  If fewer than a_i blocks are free, blocks
 *    of other sessions are evicted, a victim session at a time, from the tail
 *    of its context: LRU = least recently used session; predictive = largest
 *    priority in the eviction heap, where a session's priority is the
 *    predicted remaining tool time E[tau | tau > elapsed] (0 once its next
 *    request is queued, +inf after its last turn), computed when its blocks
 *    become unreferenced and recomputed for every session each rebuild_every
 *    engine iterations (dispatches); Belady = largest true time to next use.
 *  - A request takes prefill_s_per_token x (context tokens not resident +
 *    in_tokens) + decode_s_per_token x out_tokens seconds.
 *  - The predictor estimates E[tau | tau > e] of a tool type as the mean of
 *    (x - e) over its history samples x > e, and e when no sample exceeds e. */
#ifndef CW_POLICY_H_
#define CW_POLICY_H_

#include <stdint.h>

#include "cw.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { CW_SCHED_FCFS = 0, CW_SCHED_PREFIX_AWARE = 1 } cw_sched_policy_t;
typedef enum { CW_EVICT_LRU = 0, CW_EVICT_PREDICTIVE = 1, CW_EVICT_BELADY = 2 } cw_evict_policy_t;

typedef struct {
  int32_t capacity_blocks;     /* M >= 1 */
  int32_t block_tokens;        /* >= 1 */
  double prefill_s_per_token;  /* >= 0 */
  double decode_s_per_token;   /* >= 0 */
  int32_t sched;               /* cw_sched_policy_t */
  int32_t evict;               /* cw_evict_policy_t */
  int32_t rebuild_every;       /* >= 1; predictive eviction only */
} cw_sim_config_t;

/* Sessions and their turns, flattened (host arrays, read during the call):
 * session s owns turns [turn_off[s], turn_off[s+1]); turn_off[0] = 0 and the
 * offsets do not decrease.  Tool types index the predictor history: type y
 * owns samples hist_s[hist_off[y] .. hist_off[y+1]). */
typedef struct {
  int32_t num_sessions;
  const int32_t* turn_off;      /* [num_sessions + 1] */
  const double* session_start;  /* [num_sessions], >= 0 */
  const int32_t* in_tokens;     /* [turns], >= 0 */
  const int32_t* out_tokens;    /* [turns], >= 0 */
  const int32_t* tool;          /* [turns], in [0, num_tools) (the last turn's is ignored) */
  const double* tool_s;         /* [turns], >= 0 */
  int32_t num_tools;
  const int32_t* hist_off;      /* [num_tools + 1] */
  const double* hist_s;         /* [hist_off[num_tools]], >= 0 */
} cw_sim_trace_t;

typedef struct {
  double makespan_s;           /* last completion time */
  double mean_session_s;       /* mean of (last completion - session start) */
  double goodput_tok_s;        /* sum of in + out tokens / makespan */
  int64_t requests;
  int64_t faults;              /* requests that found part of their existing context evicted */
  int64_t evicted_blocks;
  int64_t recomputed_tokens;   /* context tokens prefilled again because their blocks were evicted */
  int64_t prefilled_tokens;    /* all prefilled tokens (recomputed + new input) */
  int64_t heap_rebuilds;
} cw_sim_result_t;

/* Runs the simulation.  `dispatch` (optional, NULL to skip) receives the
 * session of each dispatched request in order, up to `dispatch_capacity`
 * entries.  CW_ERR_NULL for a missing required pointer, CW_ERR_UNSUPPORTED for
 * an out-of-range configuration, CW_ERR_BAD_LENS for an invalid trace
 * (negative values, bad offsets or tool ids, or a turn needing more than
 * capacity_blocks blocks). */
cw_status_t cw_policy_simulate(const cw_sim_config_t* config, const cw_sim_trace_t* trace,
                               cw_sim_result_t* result, int32_t* dispatch,
                               int64_t dispatch_capacity);

/* The predictor alone: the expected remaining time of a tool call of type
 * `tool` that has run for elapsed_s seconds, from the trace's history samples
 * (see the model above). */
cw_status_t cw_policy_predict(const cw_sim_trace_t* trace, int32_t tool, double elapsed_s,
                              double* remaining_s);

#ifdef __cplusplus
}
#endif

#endif  // CW_POLICY_H_
