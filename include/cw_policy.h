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
 *    in_tokens) + decode_s_per_token x out_tokens seconds (+ swap_s_per_block
 *    per block swapped out or in for it, with offload).
 *  - Offload (host_blocks > 0; CacheWise Sec. 6.4): an evicted block is copied
 *    to the host pool while it has a free block, else dropped together with the
 *    owner's host-held blocks past it (and, for a shared block, the sharers'
 *    host-held private blocks); a block of value +inf (no one uses it again:
 *    a finished session under predictive or Belady eviction) is dropped the
 *    same way.  A copy that a drop in the same admission discards is not made
 *    nor charged.  A request first swaps its context's host-held blocks back
 *    in, after the evictions that make room for them.
 *  - The predictor estimates E[tau | tau > e] of a tool type as the mean of
 *    (x - e) over its history samples x > e, and e when no sample exceeds e.
 *
 * Blocks (the KV block manager below, on which the simulation runs): every
 * resident block is private to a session or shared by a prefix group (the
 * whole blocks of the first shared_tokens tokens its members' contexts have in
 * common, one copy; a member's first input starts with them) and carries a
 * reference count of the running requests that use it.  Blocks left
 * unreferenced when a request is released enter an eviction heap keyed by
 * their owner's eviction value (predictive: priority; LRU: minus last use;
 * Belady: true time to next use; larger evicts first), then the session id,
 * then the block's position (tail first); a shared block takes the smallest
 * value among its group's attached sessions (ties: the largest session id),
 * so the sharers' private blocks leave before it.  The heap is rebuilt from
 * current values every rebuild_every dispatches (predictive) and before every
 * dispatch (Belady).  A request's resident run is its leading resident
 * blocks (shared ones count before its first request), and the prompt tokens
 * it finds resident are min(run x block_tokens, max(context, shared whole
 * blocks x block_tokens)).  Without groups this is the session model above. */
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
  int32_t capacity_blocks;     /* M, 1 .. 2^26 */
  int32_t block_tokens;        /* >= 1 */
  double prefill_s_per_token;  /* >= 0 */
  double decode_s_per_token;   /* >= 0 */
  int32_t sched;               /* cw_sched_policy_t */
  int32_t evict;               /* cw_evict_policy_t */
  int32_t rebuild_every;       /* >= 1; predictive eviction only */
  int32_t host_blocks;         /* 0 .. 2^26: offload host pool (0: evicted blocks are dropped) */
  double swap_s_per_block;     /* >= 0: engine time of one block swapped out or in */
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
  int32_t num_groups;           /* shared-prefix groups (0: none) */
  const int32_t* session_group; /* [num_sessions], in [-1, num_groups) (-1: none); NULL if no groups */
  const int32_t* group_shared_tokens; /* [num_groups], >= 0, <= each member's first input */
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
  int64_t swapped_out_blocks;  /* evicted blocks copied to the host pool */
  int64_t swapped_in_blocks;   /* blocks brought back from it */
} cw_sim_result_t;

/* Runs the simulation.  `dispatch` (optional, NULL to skip) receives the
 * session of each dispatched request in order, up to `dispatch_capacity`
 * entries.  CW_ERR_NULL for a missing required pointer, CW_ERR_UNSUPPORTED for
 * an out-of-range configuration or exhausted host memory, CW_ERR_BAD_LENS for an
 * invalid trace
 * (negative values, bad offsets or tool ids, or a turn needing more than
 * capacity_blocks blocks). */
cw_status_t cw_policy_simulate(const cw_sim_config_t* config, const cw_sim_trace_t* trace,
                               cw_sim_result_t* result, int32_t* dispatch,
                               int64_t dispatch_capacity);

/* Per-dispatch log of a simulation (caller-owned host arrays): session,
 * cached_tokens (prompt tokens whose K/V the request found resident: the
 * attention prefix of its prefill), new_tokens (prompt tokens it prefilled:
 * context + input - cached), and its block table (physical ids of its blocks
 * for context + input + output tokens, logical order) at
 * tables[table_off[i] .. table_off[i + 1]).  At most `capacity` dispatches and
 * `table_capacity` table entries are written (tables are cut at the end);
 * `written` returns the dispatches written. */
typedef struct {
  int64_t capacity;
  int32_t* session;        /* [capacity] */
  int32_t* cached_tokens;  /* [capacity] */
  int32_t* new_tokens;     /* [capacity] */
  int64_t* table_off;      /* [capacity + 1] */
  int32_t* tables;         /* [table_capacity] */
  int64_t table_capacity;
  int64_t written;         /* out */
  int32_t* swapped_in;     /* [capacity] or NULL: blocks of the request swapped in */
  int32_t* swapped_out;    /* [capacity] or NULL: blocks of others swapped out for it */
} cw_sim_log_t;

/* cw_policy_simulate with the per-dispatch log instead of the dispatch order. */
cw_status_t cw_policy_simulate_log(const cw_sim_config_t* config, const cw_sim_trace_t* trace,
                                   cw_sim_result_t* result, cw_sim_log_t* log);

/* The KV block manager on its own, for a serving loop (host-only; one
 * manager is not safe to use from several threads at once).  Sessions are
 * registered with their prefix group (-1: none) before their first request.
 * cw_bm_admit admits a session's next request (its context holds
 * context_tokens, the request adds input_tokens and will generate
 * output_tokens): references its resident leading blocks, evicts unreferenced
 * blocks of others in heap order until the missing blocks fit, allocates and
 * references them, and returns its block table (physical ids of all `blocks`
 * = ceil((context + input + output) / block_tokens) blocks, logical order;
 * at most table_capacity written), the prompt tokens found resident and the
 * blocks evicted.  CW_ERR_WORKSPACE (nothing changed) when the blocks it needs
 * exceed the capacity left by referenced blocks.  cw_bm_release drops the
 * request's references; blocks left unreferenced enter the eviction heap with
 * `value` (larger evicts first).  cw_bm_rebuild sets the values of the listed
 * sessions and rebuilds the heap from every session's value (the periodic
 * rebuild).  Several requests may be admitted before any runs (one serving
 * step), with one restriction: while a group's shared blocks are not all
 * resident, admit at most one of its members per step, since the blocks that
 * member allocates are reported as the next member's resident prefix before
 * they hold its K/V.  Limits: capacity_blocks <= 2^26, session and group ids
 * below 2^24 (ids index dense tables: use small consecutive integers), token
 * counts of a request <= 2^40.  Errors: CW_ERR_NULL, CW_ERR_BAD_LENS (unknown or
 * running session, negative or oversized counts, NaN values, a request whose
 * blocks do not cover its group's shared blocks and the private blocks its
 * session already holds: a context only grows),
 * CW_ERR_UNSUPPORTED (sizes beyond the limits, or host memory exhausted; after
 * the latter from cw_bm_admit, cw_bm_release or cw_bm_rebuild the manager's
 * state is undefined and it should only be destroyed).  No call throws. */
typedef struct cw_block_manager cw_block_manager_t;
cw_status_t cw_bm_create(int32_t capacity_blocks, int32_t block_tokens, cw_block_manager_t** out);
cw_status_t cw_bm_destroy(cw_block_manager_t* bm);
cw_status_t cw_bm_add_session(cw_block_manager_t* bm, int32_t session, int32_t group,
                              int32_t shared_tokens);
cw_status_t cw_bm_admit(cw_block_manager_t* bm, int32_t session, int64_t context_tokens,
                        int64_t input_tokens, int64_t output_tokens, int32_t* table,
                        int32_t table_capacity, int32_t* blocks, int64_t* cached_tokens,
                        int64_t* evicted_blocks);
cw_status_t cw_bm_release(cw_block_manager_t* bm, int32_t session, double value);
cw_status_t cw_bm_rebuild(cw_block_manager_t* bm, const int32_t* sessions, const double* values,
                          int32_t n);
cw_status_t cw_bm_stats(cw_block_manager_t* bm, int64_t* free_blocks, int64_t* referenced_blocks);

/* The block manager with offload (CacheWise Sec. 6.4): evicted blocks move to a
 * host pool of host_blocks blocks (1 .. 2^26) while it has room, else they are
 * dropped with the owner's host-held blocks past them (for a shared block, also
 * the sharers' host-held private blocks), and a request's host-held context
 * blocks are swapped back in when it is admitted (a block released with value
 * +inf is never copied out, and copies a later drop of the same admission
 * discards are not listed).  The manager decides; the
 * caller moves the data (cw_kv_swap_out / cw_kv_swap_in of cw.h).  Admissions of
 * such a manager go through cw_bm_admit_swaps, which also returns the swaps:
 * out_device[i] -> out_host[i] (copy device page to host block) for the blocks
 * evicted to the host pool, then in_host[i] -> in_device[i] for the blocks of
 * the request brought back.  Apply every admission's swaps in admission order,
 * its swap-outs before its swap-ins (a swap-in may fill a page just swapped out,
 * and a later admission may reuse a host block just swapped in), all before the
 * step that reads the pages.  The four arrays hold `capacity` entries each;
 * capacity must be at least the request's blocks (both counts are bounded by
 * it), else CW_ERR_WORKSPACE with nothing changed.  cw_bm_admit on such a
 * manager is CW_ERR_UNSUPPORTED (it would lose the swap lists).
 * cw_bm_host_stats reports the free and held host blocks. */
typedef struct {
  int32_t* out_device;  /* [capacity] */
  int32_t* out_host;    /* [capacity] */
  int32_t* in_host;     /* [capacity] */
  int32_t* in_device;   /* [capacity] */
  int32_t capacity;
  int32_t n_out;        /* out: swap-outs written */
  int32_t n_in;         /* out: swap-ins written */
} cw_bm_swaps_t;
cw_status_t cw_bm_create_with_host_pool(int32_t capacity_blocks, int32_t block_tokens,
                                        int32_t host_blocks, cw_block_manager_t** out);
cw_status_t cw_bm_admit_swaps(cw_block_manager_t* bm, int32_t session, int64_t context_tokens,
                              int64_t input_tokens, int64_t output_tokens, int32_t* table,
                              int32_t table_capacity, int32_t* blocks, int64_t* cached_tokens,
                              int64_t* evicted_blocks, cw_bm_swaps_t* swaps);
cw_status_t cw_bm_host_stats(cw_block_manager_t* bm, int64_t* free_host_blocks,
                             int64_t* held_host_blocks);

/* The predictor alone: the expected remaining time of a tool call of type
 * `tool` that has run for elapsed_s seconds, from the trace's history samples
 * (see the model above). */
cw_status_t cw_policy_predict(const cw_sim_trace_t* trace, int32_t tool, double elapsed_s,
                              double* remaining_s);

#ifdef __cplusplus
}
#endif

#endif  // CW_POLICY_H_
