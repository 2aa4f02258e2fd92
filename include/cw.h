/*
 * cw.h -- prefix-cached paged extend attention on MI355X (gfx950).
 *
 * The computation behind the CacheWise KV-cache policy (CacheWise, Sec. 2:
 * KV prefixes persist in fixed-size blocks and later requests that extend a
 * prefix reuse them; Sec. 3: each agent turn reuses and extends a growing
 * prefix; Sec. 6.1: GQA/MQA models served with chunked prefill).  A new turn's
 * suffix tokens attend causally to themselves and to the cached prefix whose
 * K/V sit in a paged pool reached through a per-sequence block table.
 *
 * Semantics (sequence b, prefix length Lp, suffix length Ls, GQA group G):
 *   suffix row i of b is packed row cu_b + i, cu = exclusive prefix sum of
 *   suffix_lens; it sits at absolute position Lp + i and attends to keys
 *   0 .. Lp + i (bottom-right causal alignment).  Query head h uses kv head
 *   h / G.  Key j < Lp is slot j % P of physical page block_table[b][j / P]
 *   of the pool; key Lp + i is row cu_b + i of k_new / v_new.
 *   out = softmax(scale * q K^T) V per row, lse = natural log of the softmax
 *   denominator including the row maximum (m + ln sum exp(s - m)).
 *
 * Layouts (row-major, last dimension contiguous):
 *   q, out          bf16 [T, Hq, D]         T = sum of suffix_lens, Hq = Hkv * G
 *   k_new, v_new    bf16 [T, Hkv, D]
 *   k_pool, v_pool  bf16 or fp8-e4m3fn [num_pages, Hkv, P, D]
 *                   one (page, kv head) is P*D contiguous elements
 *   k_scale,v_scale fp32 [num_pages, Hkv]   fp8 pools only (NULL for bf16):
 *                   stored value = code * scale of its (page, kv head)
 *   block_table     int32 [num_seqs, bt_stride]; entries at or past
 *                   ceil((Lp+Ls)/P) are never read
 *   lse             fp32 [T, Hq] or NULL
 *   prefix_lens_h, suffix_lens_h   HOST int32 [num_seqs], read during the call
 *
 * Supported: head_dim 64 or 128; page_size 16 or 64; 1 <= gqa_group <= 16;
 * softmax_scale finite and > 0.  In an fp8 pool only the cached prefix is fp8:
 * the suffix keys/values come from the bf16 k_new / v_new.  With an fp8 pool
 * the extend kernel computes in fp16 on the dequantised values, so every
 * |code * scale| must lie below 65504 (scales below 146 for codes up to 448)
 * and so must every k_new / v_new value (beyond it the result is inf or NaN;
 * the scales are device data, which the calls do not inspect).  The decode
 * kernel has no such limit.
 *
 * Ownership and ordering: the caller owns every buffer, including the
 * workspace.  Per device the library keeps a cache of device properties, a
 * pinned host staging ring for the per-call plan (8 slots of 4 MiB, allocated
 * once by cw_init or by the first call that needs it, never grown or freed;
 * a call whose plan exceeds a slot fails with CW_ERR_UNSUPPORTED) and the
 * static scratch array of cw_extend_attention_noalloc.  No call allocates
 * device or pinned memory after that one-time set-up.  All work is
 * enqueued on `stream`; returning CW_OK means enqueued, not finished; buffers
 * must stay valid until the stream has passed the work.  Calls on one stream
 * may share one workspace; calls that may run concurrently need separate ones.
 *
 * Graph capture: every call that runs kernels may be captured into a HIP graph
 * (hipStreamBeginCapture on `stream`).  A captured call carries its plan in
 * kernel arguments, never in the staging ring: in those of its attention and
 * merge kernels when the plan fits there (CW_TUNE_ARG_PLANS), else in those
 * of small copy kernels (2 KiB each) that write it into the workspace at every
 * replay; either way a replay runs with the plan it was captured with, and
 * the lengths are those of capture time.  cw_init() must have been called on
 * the device first (CW_ERR_INIT), and a plan that goes through the copy
 * kernels may take at most 256 KiB (CW_ERR_UNSUPPORTED beyond).  The buffers of a captured
 * call must stay valid while the graph may be replayed, and a replay shares
 * its workspace (or the no-alloc scratch) with every other call using it, as
 * any call on the graph's stream would.
 *
 * Errors: every argument is checked before anything is enqueued, so a call
 * that returns an error has enqueued nothing.  A HIP failure while enqueuing
 * returns CW_ERR_HIP; faults inside kernels surface, as usual with HIP, at a
 * later synchronisation.  cw_last_error_message() returns a thread-local
 * description of the last error.  No call throws or aborts.
 *
 * Aliasing: the attention calls reject (CW_ERR_ALIAS) an out or lse range that
 * overlaps q, k_new, v_new, the pools, the fp8 scales, the block table, the
 * workspace or each other (ranges from the shapes and lengths of the call).
 *
 * Preconditions the library does not check (checking would need device reads;
 * cw_check_block_table checks the first on request): page ids < num_pages;
 * write slots of different sequences are disjoint; pages shared between
 * sequences lie inside every sharer's prefix.
 */
#ifndef CW_H_
#define CW_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CW_OK = 0,
  CW_ERR_NULL = 1,        /* a required pointer is NULL */
  CW_ERR_UNSUPPORTED = 2, /* head_dim, page_size, gqa_group, dtype or scale not supported */
  CW_ERR_BAD_LENS = 3,    /* negative length, Lp+Ls > bt_stride*P, or sizes overflow */
  CW_ERR_ALIGN = 4,       /* a tensor or workspace pointer not 16-byte aligned */
  CW_ERR_WORKSPACE = 5,   /* workspace_bytes smaller than the matching *_workspace_bytes() */
  CW_ERR_HIP = 6,         /* a HIP runtime call failed while enqueuing */
  CW_ERR_ALIAS = 7,       /* out or lse overlaps an input, the workspace or each other */
  CW_ERR_INIT = 8,        /* cw_extend_attention_noalloc before cw_init on this device */
  CW_STATUS_RANGE_MIN_ = -2147483647 - 1,
  CW_STATUS_RANGE_MAX_ = 2147483647
} cw_status_t;

/* Every enum of this ABI carries two range markers (never valid arguments):
 * they make every int32 value a value of the type, so an out-of-range argument
 * reaches the library's checks as a plain integer and is rejected with
 * CW_ERR_UNSUPPORTED instead of being undefined in the C++ implementation. */
typedef enum {
  CW_KV_BF16 = 0,
  CW_KV_FP8_E4M3FN = 1,
  CW_KV_DTYPE_RANGE_MIN_ = -2147483647 - 1,
  CW_KV_DTYPE_RANGE_MAX_ = 2147483647
} cw_kv_dtype_t;

/* Scatter the new K/V rows into their pool slots (CacheWise Sec. 2: the KV of a
 * request is kept in fixed-size blocks so a later turn can reuse it).
 * For i < Ls_b: pos = Lp_b + i, page = block_table[b][pos / P], slot = pos % P;
 * k_pool[page][h][slot][:] = k_new[cu_b + i][h][:] for every kv head h (and V).
 * bf16 pool: a bit copy.  fp8 pool: code = nearest e4m3fn value (ties to even)
 * of clamp(x / scale[page][h], -448, 448), x the bf16 value and the quotient an
 * IEEE fp32 division; k_scale/v_scale are then required.  No other byte of the
 * pools changes.  Workspace: cw_write_pages_workspace_bytes(num_seqs) bytes. */
size_t cw_write_pages_workspace_bytes(int32_t num_seqs);
cw_status_t cw_kv_write_pages(const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                              const float* k_scale, const float* v_scale,
                              const int32_t* block_table, int32_t bt_stride, int32_t num_pages,
                              const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                              int32_t num_seqs, int32_t num_kv_heads, int32_t head_dim,
                              int32_t page_size, cw_kv_dtype_t kv_dtype, void* workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes cw_extend_attention needs for these lengths on the current
 * device (work list plus split-K partials; the same for both pool dtypes).
 * 0 if the arguments are invalid. */
size_t cw_extend_workspace_bytes(const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                                 int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                                 int32_t head_dim, int32_t page_size);

/* Prefix-cached paged extend attention (CacheWise Sec. 2-3: a request that
 * extends a cached prefix computes attention only for its new tokens, over the
 * reused prefix blocks plus itself; Sec. 6.1: GQA).  See the file comment for
 * the exact semantics and layouts.  Sequences with Ls = 0 own no rows; Lp = 0
 * is plain causal self-attention.  Does not write the new K/V into the pool:
 * cw_kv_write_pages does, and the two calls commute. */
cw_status_t cw_extend_attention(const void* q, const void* k_new, const void* v_new,
                                const void* k_pool, const void* v_pool, const float* k_scale,
                                const float* v_scale, const int32_t* block_table,
                                int32_t bt_stride, int32_t num_pages,
                                const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                                int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                                int32_t head_dim, int32_t page_size, float softmax_scale,
                                cw_kv_dtype_t kv_dtype, void* out, float* lse, void* workspace,
                                size_t workspace_bytes, hipStream_t stream);

/* For callers that cannot allocate (code under HIP graph capture, serving
 * loops or harnesses that forbid hipMalloc): cw_extend_attention without a
 * workspace argument.  The work list and split-K partials live in a static
 * device array of CW_NOALLOC_SCRATCH_BYTES per GPU, held until the process
 * ends; the call allocates nothing (no hipMalloc, hipFree or pinned memory),
 * so cw_init() must have been called on the current device first, else
 * CW_ERR_INIT.  A call whose plan needs more scratch than the array holds
 * (cw_extend_workspace_bytes of its lengths > CW_NOALLOC_SCRATCH_BYTES) fails
 * with CW_ERR_WORKSPACE before anything is enqueued.  Every call on one GPU
 * shares that GPU's array: calls that may overlap on one GPU (different
 * streams, or different host threads) race and give wrong results; calls
 * ordered on one stream are safe.  Nothing in the array needs to start at
 * zero (each call writes its plan there, unless it travels in the kernel
 * arguments, and writes every partial it reads).
 * Results are bit-identical to cw_extend_attention with the same arguments. */
#define CW_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
cw_status_t cw_extend_attention_noalloc(const void* q, const void* k_new, const void* v_new,
                                        const void* k_pool, const void* v_pool,
                                        const float* k_scale, const float* v_scale,
                                        const int32_t* block_table, int32_t bt_stride,
                                        int32_t num_pages, const int32_t* prefix_lens_h,
                                        const int32_t* suffix_lens_h, int32_t num_seqs,
                                        int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                                        int32_t page_size, float softmax_scale,
                                        cw_kv_dtype_t kv_dtype, void* out, float* lse,
                                        hipStream_t stream);

/* cw_kv_write_pages and cw_extend_attention of the same arguments in one
 * launch (the extend kernel's workgroups scatter the new K/V into the pools
 * under their first tiles' latency).  The attention never reads a pool slot
 * at or past a sequence's prefix end, so the result is that of the two calls
 * in either order: `out`/`lse` bit-identical to cw_extend_attention, the pools
 * byte-identical to cw_kv_write_pages.  k_pool and v_pool are required (they
 * are written) and get the preconditions of cw_kv_write_pages; the workspace
 * is that of cw_extend_attention (cw_extend_workspace_bytes).  Errors as for
 * the two calls; nothing is enqueued on an error. */
cw_status_t cw_write_extend_attention(const void* q, const void* k_new, const void* v_new,
                                      void* k_pool, void* v_pool, const float* k_scale,
                                      const float* v_scale, const int32_t* block_table,
                                      int32_t bt_stride, int32_t num_pages,
                                      const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                                      int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                                      int32_t head_dim, int32_t page_size, float softmax_scale,
                                      cw_kv_dtype_t kv_dtype, void* out, float* lse,
                                      void* workspace, size_t workspace_bytes, hipStream_t stream);

/* One serving step (a chunked-prefill batch: sequences extending their
 * cached prefix by a chunk of new tokens, mixed with decodes of one token;
 * CacheWise Sec. 6.1 serves with chunked prefill): writes every sequence's
 * new K/V into the pools and computes the attention of every new token, like
 * cw_kv_write_pages + cw_extend_attention over the whole batch.  Sequences
 * with exactly one new token run on the HBM-streaming decode kernel, the
 * others on the extend kernel (which also performs the batch's page write),
 * each sub-batch with the plan it would get alone: the rows of the decode
 * sequences are bit-identical to cw_decode_attention of those sequences, the
 * other rows to cw_extend_attention of the others, and the pools to
 * cw_kv_write_pages.  Arguments, layouts and errors as for
 * cw_write_extend_attention; the workspace is cw_step_workspace_bytes.  With
 * timing events set, `start` is recorded before the step's first attention
 * kernel and `stop` after its extend kernel (after the decode part and the
 * page write when no sequence extends by more than one token). */
size_t cw_step_workspace_bytes(const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                               int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                               int32_t head_dim, int32_t page_size, cw_kv_dtype_t kv_dtype);
cw_status_t cw_step_attention(const void* q, const void* k_new, const void* v_new, void* k_pool,
                              void* v_pool, const float* k_scale, const float* v_scale,
                              const int32_t* block_table, int32_t bt_stride, int32_t num_pages,
                              const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                              int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                              int32_t head_dim, int32_t page_size, float softmax_scale,
                              cw_kv_dtype_t kv_dtype, void* out, float* lse, void* workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* Page swaps between the device page pool and a host block pool (CacheWise
 * Sec. 6.4: in the offloading configuration, evicted KV blocks move to CPU DRAM
 * and are swapped back when their session resumes).  The host pools have the
 * device pools' layout with their own block count: k_host, v_host
 * [num_host_blocks, Hkv, P, D] of the pool dtype and, for fp8 pools,
 * k_scale_host, v_scale_host fp32 [num_host_blocks, Hkv]; they must be
 * device-accessible host memory (hipHostMalloc / pinned) or device memory, and
 * 16-byte aligned.  Entry i of cw_kv_swap_out copies pool page pages_h[i]
 * (every kv head, K and V, and for fp8 its scales) to host block
 * host_blocks_h[i]; cw_kv_swap_in copies host block host_blocks_h[i] to pool
 * page pages_h[i].  Bytes are copied unchanged.  The two lists are *host*
 * int32 arrays of n entries, read during the call; ids must be in range and
 * destinations distinct (sources may repeat), else CW_ERR_BAD_LENS before
 * anything is enqueued; a pool pointer that is neither device memory nor
 * device-mapped host memory gives CW_ERR_UNSUPPORTED.  The copy runs on `stream`; the host side is read or
 * written by the kernel over the host link, so the host buffers must stay
 * valid and untouched until the stream passes the call.  Workspace:
 * cw_swap_workspace_bytes(n) bytes of device memory (the lists). */
size_t cw_swap_workspace_bytes(int32_t n);
cw_status_t cw_kv_swap_out(const void* k_pool, const void* v_pool, const float* k_scale,
                           const float* v_scale, int32_t num_pages, void* k_host, void* v_host,
                           float* k_scale_host, float* v_scale_host, int32_t num_host_blocks,
                           const int32_t* pages_h, const int32_t* host_blocks_h, int32_t n,
                           int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                           cw_kv_dtype_t kv_dtype, void* workspace, size_t workspace_bytes,
                           hipStream_t stream);
cw_status_t cw_kv_swap_in(const void* k_host, const void* v_host, const float* k_scale_host,
                          const float* v_scale_host, int32_t num_host_blocks, void* k_pool,
                          void* v_pool, float* k_scale, float* v_scale, int32_t num_pages,
                          const int32_t* host_blocks_h, const int32_t* pages_h, int32_t n,
                          int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                          cw_kv_dtype_t kv_dtype, void* workspace, size_t workspace_bytes,
                          hipStream_t stream);

/* Decode: every sequence has exactly one new token (CacheWise Sec. 2:
 * continuous batching of decode steps).  Same as cw_extend_attention with all
 * suffix lengths 1: q/out are [num_seqs, Hq, D], k_new/v_new [num_seqs, Hkv, D],
 * and the new token sits at position prefix_lens_h[b]. */
size_t cw_decode_workspace_bytes(const int32_t* prefix_lens_h, int32_t num_seqs,
                                 int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                                 int32_t page_size, cw_kv_dtype_t kv_dtype);
cw_status_t cw_decode_attention(const void* q, const void* k_new, const void* v_new,
                                const void* k_pool, const void* v_pool, const float* k_scale,
                                const float* v_scale, const int32_t* block_table,
                                int32_t bt_stride, int32_t num_pages,
                                const int32_t* prefix_lens_h, int32_t num_seqs,
                                int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                                int32_t page_size, float softmax_scale, cw_kv_dtype_t kv_dtype,
                                void* out, float* lse, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* Debug check of the block-table precondition (page ids < num_pages), which the
 * attention and page-write calls cannot check without reading device memory.
 * For each sequence b, counts the entries block_table[b][j], j <
 * ceil((Lp_b + Ls_b) / page_size) (exactly the entries those calls read), that
 * lie outside [0, num_pages), and writes the count to bad_per_seq[b] (device
 * int32 [num_seqs], overwritten; no atomics, so the counts are exact and
 * repeatable).  Entries past a sequence's length are not read.  Lens and
 * block_table as for cw_kv_write_pages; workspace: cw_write_pages_workspace_bytes
 * (num_seqs) bytes, 16-byte aligned.  Errors: CW_ERR_NULL, CW_ERR_UNSUPPORTED
 * (page_size), CW_ERR_BAD_LENS (as cw_kv_write_pages), CW_ERR_ALIGN,
 * CW_ERR_WORKSPACE; all checked before anything is enqueued. */
cw_status_t cw_check_block_table(const int32_t* block_table, int32_t bt_stride, int32_t num_pages,
                                 const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                                 int32_t num_seqs, int32_t page_size, int32_t* bad_per_seq,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Tuning knobs for tests and benchmarks; every value gives the same results
 * within floating-point tolerance.  Process-wide; set them before querying a
 * workspace size, since they change the plan.
 *   CW_TUNE_KV_CHUNK_TILES  0 = automatic split-K; n > 0 = split every key
 *                           range into chunks of n 64-key tiles.
 *   CW_TUNE_TARGET_WGS      0 = automatic; n > 0 = split-K until at least n
 *                           workgroups are launched.
 *   CW_TUNE_EXTEND_KERNEL   0 or 1 = eight waves of 32 query rows per work
 *                           item (the default), 2 = four waves of 64 rows
 *                           (bf16 pools only; fp8 pools always run the
 *                           eight-wave kernel).
 *   CW_TUNE_DEAL_ROUNDS     1 = the work of a (sequence, kv head) that fills
 *                           whole rounds of the GPU (a work item per resident
 *                           workgroup on every XCD) is dealt across all XCDs a
 *                           round at a time (the default); 0 = it stays on one
 *                           XCD.  Larger values act as 1.
 *   CW_TUNE_PLAN_DIRECT     0 = the attention calls copy their plan from the
 *                           pinned staging slot into the workspace with a
 *                           small kernel before the attention kernels; 1 = the
 *                           kernels read it from the staging slot over the
 *                           host link (no copy kernel; cw_extend_attention_noalloc
 *                           always copies).  Larger values act as 1.
 *   CW_TUNE_SUFFIX_WEIGHT   split-K chunk boundaries divide a tile's keys into
 *                           equal shares of cost, where a 64-key tile that
 *                           reaches past the cached prefix costs value / 100
 *                           of a prefix tile (1 .. 10000; default 125, the
 *                           measured cost of the masked tiles; 100: equal
 *                           key counts).
 *   CW_TUNE_COMPACT_DECODE  1 = a decode plan (of cw_decode_attention or of a
 *                           step's decodes) is uploaded in compact form, one
 *                           record per sequence, and rebuilt on the device by
 *                           the upload kernel (the default; up to 2048
 *                           sequences, beyond that as 0); 0 = its work items
 *                           are uploaded as they are.  Larger values act as 1.
 *   CW_TUNE_ARG_PLANS       1 = an extend plan of up to 16 KB (of an extend
 *                           call, or of a step without decodes), and a decode
 *                           plan whose compact form fits in 16 KB (of a decode
 *                           call, or of a step without extends; about 250
 *                           sequences), travel in the kernel arguments of the
 *                           attention and merge kernels, with no upload kernel
 *                           (the default; the kernels rebuild a compact plan's
 *                           items and merge groups themselves); 0 = they are
 *                           uploaded like larger plans.  Larger values act as 1.
 * Returns CW_ERR_UNSUPPORTED for an unknown key or a negative value. */
typedef enum {
  CW_TUNE_KV_CHUNK_TILES = 0,
  CW_TUNE_TARGET_WGS = 1,
  CW_TUNE_EXTEND_KERNEL = 2,
  CW_TUNE_DEAL_ROUNDS = 3,
  CW_TUNE_PLAN_DIRECT = 4,
  CW_TUNE_SUFFIX_WEIGHT = 5,
  CW_TUNE_COMPACT_DECODE = 6,
  CW_TUNE_ARG_PLANS = 7,
  CW_TUNE_RANGE_MIN_ = -2147483647 - 1,
  CW_TUNE_RANGE_MAX_ = 2147483647
} cw_tune_key_t;
cw_status_t cw_set_tuning(cw_tune_key_t key, int32_t value);

/* Benchmark hook: when `start` and `stop` are non-NULL, every later
 * cw_extend_attention / cw_decode_attention / cw_step_attention call records
 * `start` on its stream right before the main attention kernel and `stop` right
 * after it (before any split-K merge), so hipEventElapsedTime gives that
 * kernel's duration alone.  For cw_step_attention the main kernel is the
 * extend kernel when the step has extends, else the decode kernel.
 * Pass NULL, NULL to stop.  Process-wide; the events stay owned by the caller. */
cw_status_t cw_set_timing_events(hipEvent_t start, hipEvent_t stop);

/* Host-only view of the extend work plan, for tests of the planner: writes up
 * to `capacity` work items of 8 int32 each, in launch order
 * {seq, kv_head, first packed row, key begin, key end, partial slot or -1,
 *  rows in tile, 0}; a seq of -1 marks an idle padding item.  Returns the
 * number of items, or -1 if the arguments are invalid.  The plan is the one
 * cw_extend_attention uses (for either pool dtype).  Makes no HIP call
 * other than a cached device-property query, and works without a GPU. */
int64_t cw_extend_plan_items(const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                             int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                             int32_t head_dim, int32_t page_size, int32_t* items_out,
                             int64_t capacity);

/* Host-only view of the decode plan (cw_decode_attention's), for tests: its
 * work items (8 int32 each, as cw_extend_plan_items) and merge groups (8 int32
 * each: {seq, kv_head, first row, rows, first partial slot, partial slots, 0,
 * 0}), as the planner builds them (rebuilt = 0) or as the plan-upload kernel
 * rebuilds them from the compact form (rebuilt = 1, the same function run on
 * the host).  Writes up to items_capacity items and groups_capacity groups;
 * returns the number of items and sets *num_groups, or returns -1 if the
 * arguments are invalid or (rebuilt = 1) the plan has no compact form.  Works
 * without a GPU. */
int64_t cw_decode_plan_items(const int32_t* prefix_lens_h, int32_t num_seqs, int32_t num_kv_heads,
                             int32_t gqa_group, int32_t head_dim, int32_t page_size,
                             cw_kv_dtype_t kv_dtype, int32_t rebuilt, int32_t* items_out,
                             int64_t items_capacity, int32_t* groups_out, int64_t groups_capacity,
                             int64_t* num_groups);

/* One-time set-up of the current device: allocates the pinned plan staging
 * ring (which every other call otherwise does on first use) and resolves this
 * device's copy of the static scratch array of cw_extend_attention_noalloc
 * (which requires this call).  Idempotent.  CW_ERR_HIP on failure
 * (nothing stays allocated then, and the call can be repeated). */
cw_status_t cw_init(void);

/* Number of pinned host allocations the library has made in this process
 * (kStagingSlots per initialised device; for tests that no call allocates). */
int64_t cw_pinned_allocations(void);

/* Number of calls in this process whose plan travelled in the kernel
 * arguments (CW_TUNE_ARG_PLANS) rather than through the staging ring or the
 * copy kernels of a captured call; for tests that a call took that path. */
int64_t cw_arg_plan_calls(void);

const char* cw_status_string(cw_status_t status);
const char* cw_last_error_message(void);
/* Library version, major * 10000 + minor * 100 + patch. */
int32_t cw_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CW_H_ */
