// C ABI front end: argument validation, planning, plan upload, launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <exception>
#include <initializer_list>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "../../include/cw.h"
#include "cw_internal.h"
#include "planner.h"

// Scratch memory of cw_extend_attention_noalloc (plan and split-K partials):
// every GPU the library runs on holds its own copy until the process ends.  In
// host code this name is only a stand-in; kernels get the device address that
// hipGetSymbolAddress returns for the current device (DeviceState::scratch).
static __device__ __align__(256) uint8_t scratch[CW_NOALLOC_SCRATCH_BYTES];

namespace cw {
namespace {

thread_local std::string g_last_error;
Tuning g_tuning;
std::mutex g_tuning_mu;
hipEvent_t g_ev_start = nullptr, g_ev_stop = nullptr;  // guarded by g_tuning_mu

cw_status_t fail(cw_status_t s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

}  // namespace

void set_last_error(const char* msg) { g_last_error = msg; }

namespace {

cw_status_t hip_fail(hipError_t e, const char* what) {
  return fail(CW_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

Tuning current_tuning() {
  std::lock_guard<std::mutex> g(g_tuning_mu);
  return g_tuning;
}

// Extend kernel: the eight-wave kernel (32 rows per wave) unless the four-wave
// one (64 rows per wave, bf16 pools only) is asked for.  Both own LDS_BLOCK_M
// rows per work item, so they share the plan.
hipError_t launch_extend(const ExtendParams& p, int head_dim, int page_size, bool fp8,
                         hipStream_t stream, const ArgPlan* ap) {
  if (!fp8 && current_tuning().extend_kernel == 2) return launch_extend_w64(p, head_dim, page_size, stream, ap);
  return launch_extend_lds(p, head_dim, page_size, fp8, stream, ap);
}

// ---------------------------------------------------------------------------
// per-device state

constexpr int kMaxDevices = 64;
constexpr int kStagingSlots = 8;
// Every staging slot has this fixed size, allocated once per device (cw_init or
// the first call that uploads a plan); a plan larger than a slot is rejected.
constexpr size_t kStagingSlotBytes = size_t(4) << 20;
// The last bytes of a slot are the words its upload kernel's workgroups write
// once they have read the slot (one per workgroup); the plan gets the rest.
constexpr size_t kDoneBytes = size_t(kMaxUploadWorkgroups) * sizeof(uint32_t);
constexpr size_t kPlanSlotBytes = kStagingSlotBytes - kDoneBytes;
// A call captured into a graph carries its plan in kernel arguments (2 KiB per
// copy launch); its plan may take at most this many bytes.
constexpr size_t kCaptureMaxBytes = size_t(256) << 10;

struct StagingSlot {
  void* host = nullptr;
  void* dev = nullptr;  // the same pinned memory as the device addresses it
  hipEvent_t ev = nullptr;
  bool pending = false;        // `ev` recorded behind kernels that read the slot (direct mode)
  bool reads_pending = false;  // an upload kernel reads the slot: wait for its done words
  uint32_t seq = 0;            // the value its workgroups write
  int32_t workgroups = 0;
};

struct DeviceState {
  std::once_flag props_once;
  int32_t num_cus = 256;
  int32_t num_xcds = 8;
  std::mutex staging_mu;  // guards everything below
  bool ready = false;     // staging ring allocated
  StagingSlot slots[kStagingSlots];
  int next_slot = 0;
  uint8_t* capture_buf = nullptr;  // kCaptureMaxBytes of host memory: plans of captured calls
  uint32_t upload_seq = 0;         // the last value handed to an upload kernel
  uint8_t* scratch = nullptr;  // this device's copy of the static scratch array (cw_init)
};

DeviceState g_devices[kMaxDevices];
std::atomic<int64_t> g_pinned_allocs{0};
std::atomic<int64_t> g_arg_plan_calls{0};

// Current device, or -1 when no GPU runtime is usable (host-only queries).
int current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return -1;
  }
  return (dev >= 0 && dev < kMaxDevices) ? dev : -1;
}

// Compute-unit and XCD count of the current device; MI355X defaults without one.
void device_shape(int32_t* cus, int32_t* xcds) {
  const int dev = current_device();
  if (dev < 0) {
    *cus = 256;
    *xcds = 8;
    return;
  }
  DeviceState& st = g_devices[dev];
  std::call_once(st.props_once, [&]() {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) {
      st.num_cus = n;
      // gfx950 groups 32 CUs per XCD (256 CUs in 8 XCDs; a CPX partition is one XCD)
      st.num_xcds = n >= 32 ? n / 32 : 1;
    } else {
      (void)hipGetLastError();
    }
  });
  *cus = st.num_cus;
  *xcds = st.num_xcds;
}

// The device's one-time set-up, under st.staging_mu: the pinned staging ring
// (kStagingSlots slots of kStagingSlotBytes, with their events).  Nothing is allocated
// after it succeeds; a failure frees what it allocated and can be retried.
cw_status_t init_locked(DeviceState& st) {
  if (st.ready) return CW_OK;
  hipError_t e = hipSuccess;
  int made = 0;
  auto undo = [&]() {
    for (int i = 0; i < made; ++i) {
      (void)hipHostFree(st.slots[i].host);
      if (st.slots[i].ev) (void)hipEventDestroy(st.slots[i].ev);
      st.slots[i] = StagingSlot{};
    }
    delete[] st.capture_buf;
    st.capture_buf = nullptr;
  };
  st.capture_buf = new (std::nothrow) uint8_t[kCaptureMaxBytes];
  if (st.capture_buf == nullptr) return fail(CW_ERR_UNSUPPORTED, "host memory for captured plans");
  for (; made < kStagingSlots; ++made) {
    StagingSlot& s = st.slots[made];
    e = hipHostMalloc(&s.host, kStagingSlotBytes, hipHostMallocDefault);
    if (e != hipSuccess) {
      s.host = nullptr;
      undo();
      return hip_fail(e, "hipHostMalloc of the plan staging ring");
    }
    g_pinned_allocs.fetch_add(1);
    // The event only tells the host that the kernels reading the slot (the upload
    // kernel, or with direct plan reads the attention kernels) have finished; it
    // needs no system-scope fence (by default an L2 write-back and invalidate,
    // which held the next kernel back by ~5 us and left it a cold L2).
    e = hipHostGetDevicePointer(&s.dev, s.host, 0);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&s.ev, hipEventDisableTiming | hipEventDisableSystemFence);
    if (e != hipSuccess) {
      ++made;
      undo();
      return hip_fail(e, "staging slot set-up");
    }
  }
  st.next_slot = 0;
  st.ready = true;
  return CW_OK;
}

cw_status_t current_state(DeviceState** out) {
  int dev = -1;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(CW_ERR_HIP, "device index %d out of range", dev);
  *out = &g_devices[dev];
  return CW_OK;
}

// Stages `bytes` of host data for `stream` in a pinned staging slot, so that the
// caller's host buffer can be reused at once, and enqueues the kernels that read
// it: `fill(host)` writes the bytes into the slot (the plan is packed there
// directly, without an intermediate buffer), then `launch(base)` enqueues the
// kernels, with `base` the device address they read the data at.  Copy mode:
// a small kernel copies the slot to `dst` (device memory) and base = dst.
// Direct mode: the kernels read the slot itself over the host link (base = the
// slot's device address), which saves the copy kernel and its launch gap; the
// slot is then held until those kernels have run.  A slot is reused only after
// the event recorded behind its last reader has completed.  The ring is set up
// on the first use on a device when cw_init has not done it, unless `no_alloc`
// is set, in which case an uninitialised device is an error (CW_ERR_INIT).
// A stream being captured into a graph gets the plan in the arguments of copy
// kernels instead (each replay writes the captured plan again; no slot, no
// event, no wait), and the ring must exist already (CW_ERR_INIT otherwise).
// With `compact` (a decode plan in compact form, copy mode only) the slot gets
// the meta's first compact->verbatim bytes (fill_head) and the plan's records,
// and the upload kernel rebuilds the decode items and groups on the device.
struct CompactUpload {
  const ExtendPlan* plan = nullptr;  // nullptr: upload the meta as it is
  size_t verbatim = 0;               // bytes of the meta before the decode items
  size_t bytes = 0;                  // bytes of the compact blob
  ExpandDesc desc{};
};

// The compact upload of decode plan `plan` whose meta starts at byte `at` of a
// call's meta; false when the plan has no compact form or it is switched off.
bool compact_upload(const ExtendPlan& plan, size_t at, CompactUpload* cu) {
  if (!plan.compact || current_tuning().compact_decode == 0 || plan.recs.empty() ||
      plan.recs.size() > size_t(kMaxExpandSeqs))
    return false;
  cu->plan = &plan;
  cu->verbatim = at + plan.off_items;
  cu->desc = plan.desc;
  cu->desc.rec_off = static_cast<uint32_t>(cu->verbatim);
  cu->desc.tail_off = static_cast<uint32_t>(cu->verbatim + plan.recs.size() * sizeof(DecodeRec));
  cu->desc.items_off = static_cast<uint32_t>(at + plan.off_items);
  cu->desc.groups_off = static_cast<uint32_t>(at + plan.off_groups);
  cu->bytes = (size_t(cu->desc.tail_off) + plan.tails.size() * sizeof(int32_t) + 15) & ~size_t(15);
  return true;
}

// Writes the compact blob: the meta's head, the records, the tail order.
template <class FillHead>
void fill_compact(const CompactUpload& cu, uint8_t* h, FillHead&& fill_head) {
  const ExtendPlan& cp = *cu.plan;
  fill_head(h);
  std::memcpy(h + cu.desc.rec_off, cp.recs.data(), cp.recs.size() * sizeof(DecodeRec));
  std::memcpy(h + cu.desc.tail_off, cp.tails.data(), cp.tails.size() * sizeof(int32_t));
}

// Whether the compact blob and its ExpandDesc (at byte cu.bytes) fit the
// kernel arguments.
bool compact_arg_fits(const CompactUpload& cu) { return cu.bytes + sizeof(ExpandDesc) <= kArgPlanBytes; }

// Waits until every workgroup of the upload kernel that last read `s` has
// reported its reads (the done words at the slot's end).  The host runs up to
// kStagingSlots calls ahead of the device, so this waits for the device to
// reach an upload issued that many calls ago.  If the words have not all
// arrived after two seconds (calls of hundreds of milliseconds each, or an
// upload that never ran), the device is synchronised once, which also surfaces
// a fault, and they are checked again.
cw_status_t wait_slot_reads(StagingSlot& s) {
  if (!s.reads_pending) return CW_OK;
  const volatile uint32_t* done =
      reinterpret_cast<const volatile uint32_t*>(static_cast<uint8_t*>(s.host) + kPlanSlotBytes);
  auto all_read = [&]() {
    for (int32_t w = 0; w < s.workgroups; ++w)
      if (done[w] != s.seq) return false;
    return true;
  };
  const auto t0 = std::chrono::steady_clock::now();
  for (uint32_t spin = 1; !all_read(); ++spin) {
    if ((spin & 1023u) == 0) {
      if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(2)) {
        const hipError_t e = hipDeviceSynchronize();
        if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize while waiting for a staging slot");
        if (!all_read()) return fail(CW_ERR_HIP, "the upload kernel of a staging slot never reported its reads");
        break;
      }
      std::this_thread::yield();
    }
  }
  std::atomic_thread_fence(std::memory_order_acquire);
  s.reads_pending = false;
  return CW_OK;
}

template <class Fill, class Launch, class FillHead>
cw_status_t stage_and_launch(size_t bytes, void* dst, hipStream_t stream, Fill&& fill,
                             Launch&& launch, bool no_alloc, bool direct,
                             const CompactUpload* compact, FillHead&& fill_head, bool arg_plan = false) {
  if (bytes == 0) return launch(static_cast<const uint8_t*>(dst), nullptr);
  if (arg_plan && !direct) {
    // the plan travels in the kernel arguments: no slot, no upload kernel (and
    // a captured launch keeps it by value); a decode plan in compact form, with
    // its ExpandDesc behind the records, else as it is
    if (compact != nullptr && compact->plan != nullptr) {
      if (compact_arg_fits(*compact)) {
        ArgPlan ap;
        fill_compact(*compact, ap.bytes, fill_head);
        std::memcpy(ap.bytes + compact->bytes, &compact->desc, sizeof(ExpandDesc));
        g_arg_plan_calls.fetch_add(1);
        return launch(nullptr, &ap);
      }
    } else if (bytes <= kArgPlanBytes) {
      ArgPlan ap;
      fill(ap.bytes);
      g_arg_plan_calls.fetch_add(1);
      return launch(nullptr, &ap);
    }
  }
  if (bytes > kPlanSlotBytes)
    return fail(CW_ERR_UNSUPPORTED,
                "the call's plan takes %zu bytes, more than the %zu-byte staging slot "
                "(too many sequences or work items for one call)",
                bytes, kPlanSlotBytes);
  hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
  hipError_t ce = hipStreamIsCapturing(stream, &capture);
  if (ce != hipSuccess) return hip_fail(ce, "hipStreamIsCapturing");
  DeviceState* stp = nullptr;
  cw_status_t s0 = current_state(&stp);
  if (s0 != CW_OK) return s0;
  DeviceState& st = *stp;
  std::lock_guard<std::mutex> g(st.staging_mu);
  if (capture != hipStreamCaptureStatusNone) {
    if (capture != hipStreamCaptureStatusActive) return fail(CW_ERR_HIP, "the stream's capture has been invalidated");
    if (!st.ready) return fail(CW_ERR_INIT, "cw_init() must be called on this device before capturing a call");
    if (bytes > kCaptureMaxBytes || bytes % 4 != 0)
      return fail(CW_ERR_UNSUPPORTED, "a captured call's plan takes %zu bytes, more than %zu", bytes,
                  kCaptureMaxBytes);
    fill(st.capture_buf);
    ce = launch_arg_copy(st.capture_buf, dst, bytes, stream);
    if (ce != hipSuccess) return hip_fail(ce, "plan upload kernel launch");
    return launch(static_cast<const uint8_t*>(dst), nullptr);
  }
  if (!st.ready) {
    if (no_alloc) return fail(CW_ERR_INIT, "cw_init() has not been called on this device");
    s0 = init_locked(st);
    if (s0 != CW_OK) return s0;
  }
  StagingSlot& s = st.slots[st.next_slot];
  st.next_slot = (st.next_slot + 1) % kStagingSlots;
  hipError_t e = hipSuccess;
  if (s.pending) {
    e = hipEventSynchronize(s.ev);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    s.pending = false;
  }
  s0 = wait_slot_reads(s);
  if (s0 != CW_OK) return s0;
  const bool use_compact = compact != nullptr && compact->plan != nullptr && !direct &&
                           compact->bytes <= kPlanSlotBytes && compact->bytes < bytes;
  uint8_t* h = static_cast<uint8_t*>(s.host);
  if (use_compact) {
    fill_compact(*compact, h, fill_head);
  } else {
    fill(h);
  }
  if (direct) {
    const cw_status_t launched = launch(static_cast<const uint8_t*>(s.dev), nullptr);
    // recorded even when a launch failed: whatever was enqueued may read the slot
    e = hipEventRecord(s.ev, stream);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
    s.pending = true;
    return launched;
  }
  // copy mode: only the upload kernel reads the slot, and it reports its reads
  // itself (no event in the stream: a marker between two kernels costs ~4 us)
  uint32_t* done = reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(s.dev) + kPlanSlotBytes);
  st.upload_seq = st.upload_seq == 0xFFFFFFFFu ? 1u : st.upload_seq + 1u;
  std::memset(static_cast<uint8_t*>(s.host) + kPlanSlotBytes, 0, kDoneBytes);
  int32_t workgroups = 0;
  e = use_compact
          ? launch_plan_expand(s.dev, dst, compact->verbatim, compact->desc, stream, done, st.upload_seq, &workgroups)
          : launch_stage_copy(s.dev, dst, bytes, stream, done, st.upload_seq, &workgroups);
  if (e != hipSuccess) return hip_fail(e, "plan upload kernel launch");
  s.seq = st.upload_seq;
  s.workgroups = workgroups;
  s.reads_pending = true;
  return launch(static_cast<const uint8_t*>(dst), nullptr);
}

template <class Fill>
cw_status_t upload_fill(size_t bytes, void* dst, hipStream_t stream, Fill&& fill) {
  return stage_and_launch(bytes, dst, stream, fill, [](const uint8_t*, const ArgPlan*) { return CW_OK; },
                          false, false, nullptr, fill);
}

cw_status_t upload(const void* src, size_t bytes, void* dst, hipStream_t stream) {
  return upload_fill(bytes, dst, stream, [&](uint8_t* h) { std::memcpy(h, src, bytes); });
}

// Whether a small extend plan travels in the kernel arguments (CW_TUNE_ARG_PLANS).
bool arg_plans() { return current_tuning().arg_plans != 0; }

// Whether a call's plan is read by its kernels straight from the staging slot
// (CW_TUNE_PLAN_DIRECT).
bool plan_direct(bool no_alloc) {
  return !no_alloc && current_tuning().plan_direct != 0;
}

// A byte range of one argument, for the aliasing check.
struct Span {
  const void* p;
  size_t bytes;
  const char* name;
};

bool overlap(const Span& a, const Span& b) {
  if (a.p == nullptr || b.p == nullptr || a.bytes == 0 || b.bytes == 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
  return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

// out / lse must not overlap any input, the workspace or each other.
cw_status_t check_no_alias(std::initializer_list<Span> outputs, std::initializer_list<Span> inputs) {
  for (const Span* o = outputs.begin(); o != outputs.end(); ++o) {
    for (const Span& i : inputs)
      if (overlap(*o, i)) return fail(CW_ERR_ALIAS, "%s overlaps %s", o->name, i.name);
    for (const Span* o2 = o + 1; o2 != outputs.end(); ++o2)
      if (overlap(*o, *o2)) return fail(CW_ERR_ALIAS, "%s overlaps %s", o->name, o2->name);
  }
  return CW_OK;
}

// The aliasing check of an attention call (extend, decode or step).
cw_status_t check_attention_alias(const void* q, const void* k_new, const void* v_new,
                                  const void* k_pool, const void* v_pool, const float* k_scale,
                                  const float* v_scale, const int32_t* block_table,
                                  int32_t bt_stride, int32_t num_pages, int32_t num_seqs,
                                  int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                                  int32_t page_size, cw_kv_dtype_t kv_dtype, int64_t total,
                                  const void* out, const float* lse, const void* workspace,
                                  size_t workspace_bytes) {
  const size_t hq = size_t(num_kv_heads) * gqa_group;
  const size_t rows_q = size_t(total) * hq * head_dim * 2;
  const size_t rows_kv = size_t(total) * num_kv_heads * head_dim * 2;
  const size_t elem = kv_dtype == CW_KV_FP8_E4M3FN ? 1 : 2;
  const size_t pool = size_t(num_pages) * num_kv_heads * page_size * head_dim * elem;
  const size_t scales = kv_dtype == CW_KV_FP8_E4M3FN ? size_t(num_pages) * num_kv_heads * 4 : 0;
  return check_no_alias({{out, rows_q, "out"}, {lse, size_t(total) * hq * 4, "lse"}},
                        {{q, rows_q, "q"}, {k_new, rows_kv, "k_new"}, {v_new, rows_kv, "v_new"},
                         {k_pool, pool, "k_pool"}, {v_pool, pool, "v_pool"},
                         {k_scale, scales, "k_scale"}, {v_scale, scales, "v_scale"},
                         {block_table, size_t(num_seqs) * bt_stride * 4, "block_table"},
                         {workspace, workspace_bytes, "workspace"}});
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---------------------------------------------------------------------------
// validation

cw_status_t check_shape(int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                        int32_t page_size) {
  if (num_seqs < 0) return fail(CW_ERR_BAD_LENS, "num_seqs = %d is negative", num_seqs);
  if (head_dim != 64 && head_dim != 128)
    return fail(CW_ERR_UNSUPPORTED, "head_dim = %d (supported: 64, 128)", head_dim);
  if (page_size != 16 && page_size != 64)
    return fail(CW_ERR_UNSUPPORTED, "page_size = %d (supported: 16, 64)", page_size);
  if (num_kv_heads < 1 || num_kv_heads > 1024)
    return fail(CW_ERR_UNSUPPORTED, "num_kv_heads = %d (supported: 1..1024)", num_kv_heads);
  if (gqa_group < 1 || gqa_group > 16)
    return fail(CW_ERR_UNSUPPORTED, "gqa_group = %d (supported: 1..16)", gqa_group);
  return CW_OK;
}

// Lengths: non-negative, fit the block table, and the packed sizes fit int32.
cw_status_t check_lens(const int32_t* lp, const int32_t* ls, int32_t num_seqs, int32_t bt_stride,
                       int32_t page_size, int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                       bool check_table) {
  if (num_seqs > 0 && (lp == nullptr || ls == nullptr))
    return fail(CW_ERR_NULL, "prefix_lens_h / suffix_lens_h is NULL");
  if (check_table && num_seqs > 0 && bt_stride < 1)
    return fail(CW_ERR_BAD_LENS, "bt_stride = %d must be >= 1", bt_stride);
  int64_t total = 0;
  for (int32_t b = 0; b < num_seqs; ++b) {
    if (lp[b] < 0 || ls[b] < 0)
      return fail(CW_ERR_BAD_LENS, "sequence %d: negative length (Lp=%d, Ls=%d)", b, lp[b], ls[b]);
    const int64_t n = int64_t(lp[b]) + ls[b];
    if (n > INT32_MAX / 2) return fail(CW_ERR_BAD_LENS, "sequence %d: Lp+Ls=%lld too long", b, (long long)n);
    if (check_table && n > int64_t(bt_stride) * page_size)
      return fail(CW_ERR_BAD_LENS, "sequence %d: Lp+Ls=%lld exceeds bt_stride*P=%lld", b,
                  (long long)n, (long long)bt_stride * page_size);
    total += ls[b];
  }
  const int64_t hq = int64_t(num_kv_heads) * gqa_group;
  if (total * hq * head_dim > INT64_C(1) << 40 || total > INT32_MAX / 32)
    return fail(CW_ERR_BAD_LENS, "total suffix tokens %lld too large", (long long)total);
  (void)hq;
  return CW_OK;
}

cw_status_t check_dtype(cw_kv_dtype_t kv_dtype, const float* k_scale, const float* v_scale) {
  if (kv_dtype != CW_KV_BF16 && kv_dtype != CW_KV_FP8_E4M3FN)
    return fail(CW_ERR_UNSUPPORTED, "kv_dtype = %d", int(kv_dtype));
  if (kv_dtype == CW_KV_FP8_E4M3FN && (k_scale == nullptr || v_scale == nullptr))
    return fail(CW_ERR_NULL, "fp8 pool needs k_scale and v_scale");
  return CW_OK;
}

int64_t sum_suffix(const int32_t* ls, int32_t num_seqs) {
  int64_t t = 0;
  for (int32_t b = 0; b < num_seqs; ++b) t += ls[b];
  return t;
}

// Both pool dtypes run the LDS-staged kernel with the same row block
// (LDS_BLOCK_M rows per work item, one workgroup per CU), so the extend plan
// does not depend on the pool dtype.
ExtendPlan make_plan(const int32_t* lp, const int32_t* ls, int32_t num_seqs, int32_t num_kv_heads,
                     int32_t gqa_group, int32_t head_dim, const int32_t* cu_rows = nullptr,
                     const int32_t* bt_rows = nullptr) {
  int32_t cus = 256, xcds = 8;
  device_shape(&cus, &xcds);
  return build_extend_plan(lp, ls, num_seqs, num_kv_heads, gqa_group, head_dim, LDS_BLOCK_M, 1,
                           cus, xcds, current_tuning(), cu_rows, bt_rows);
}

// Decode plans follow the pool dtype's tile length and residency (three
// 16 KB-tile waves per CU for bf16, six 8 KB-tile waves for fp8).
ExtendPlan make_decode_plan(const int32_t* lp, int32_t num_seqs, int32_t num_kv_heads,
                            int32_t gqa_group, int32_t head_dim, int32_t page_size,
                            cw_kv_dtype_t kv_dtype, const int32_t* cu_rows = nullptr,
                            const int32_t* bt_rows = nullptr) {
  int32_t cus = 256, xcds = 8;
  device_shape(&cus, &xcds);
  const bool fp8 = kv_dtype == CW_KV_FP8_E4M3FN;
  return build_decode_plan(lp, num_seqs, num_kv_heads, gqa_group, head_dim, page_size,
                           decode_keys_per_tile(head_dim, fp8), decode_waves_per_cu(fp8), cus,
                           current_tuning(), cu_rows, bt_rows);
}

// A step of a serving engine: the sequences with one new token go to the decode
// kernel, the others to the extend kernel, as sub-batches whose plans keep the
// step's packed rows and block-table rows.
struct StepPlan {
  std::vector<int32_t> ext, dec;  // step sequence indices of each sub-batch
  ExtendPlan ext_plan, dec_plan;
  std::vector<SeqInfo> seqs;      // every sequence of the step (for the page write)
  // workspace: [step seqs | extend meta | decode meta | extend partials | decode partials]
  size_t off_ext_meta = 0, off_dec_meta = 0, off_ext_part = 0, off_dec_part = 0, meta_bytes = 0,
         total_bytes = 0;
};

size_t align256h(size_t x) { return (x + 255) & ~size_t(255); }

StepPlan make_step_plan(const int32_t* lp, const int32_t* ls, int32_t num_seqs, int32_t num_kv_heads,
                        int32_t gqa_group, int32_t head_dim, int32_t page_size, cw_kv_dtype_t kv_dtype) {
  StepPlan sp;
  std::vector<int32_t> lp_e, ls_e, cu_e, lp_d, cu_d;
  int32_t cu = 0;
  for (int32_t b = 0; b < num_seqs; ++b) {
    sp.seqs.push_back(SeqInfo{lp[b], ls[b], cu, b});
    if (ls[b] == 1) {
      sp.dec.push_back(b);
      lp_d.push_back(lp[b]);
      cu_d.push_back(cu);
    } else if (ls[b] > 1) {
      sp.ext.push_back(b);
      lp_e.push_back(lp[b]);
      ls_e.push_back(ls[b]);
      cu_e.push_back(cu);
    }
    cu += ls[b];
  }
  if (!sp.ext.empty())
    sp.ext_plan = make_plan(lp_e.data(), ls_e.data(), static_cast<int32_t>(sp.ext.size()), num_kv_heads,
                            gqa_group, head_dim, cu_e.data(), sp.ext.data());
  if (!sp.dec.empty())
    sp.dec_plan = make_decode_plan(lp_d.data(), static_cast<int32_t>(sp.dec.size()), num_kv_heads,
                                   gqa_group, head_dim, page_size, kv_dtype, cu_d.data(), sp.dec.data());
  sp.off_ext_meta = align256h(sp.seqs.size() * sizeof(SeqInfo));
  sp.off_dec_meta = sp.off_ext_meta + sp.ext_plan.meta_bytes;
  sp.meta_bytes = sp.off_dec_meta + sp.dec_plan.meta_bytes;
  sp.off_ext_part = sp.meta_bytes;
  sp.off_dec_part = sp.off_ext_part + (sp.ext_plan.total_bytes - sp.ext_plan.meta_bytes);
  sp.total_bytes = std::max<size_t>(256, sp.off_dec_part + (sp.dec_plan.total_bytes - sp.dec_plan.meta_bytes));
  return sp;
}

// Kernel arguments of a plan whose meta is read at `meta` and whose partials
// sit at ws + part.
ExtendParams plan_params(const ExtendPlan& plan, const uint8_t* meta, uint8_t* ws, size_t part) {
  ExtendParams p{};
  if (meta != nullptr) {
    p.seqs = reinterpret_cast<const SeqInfo*>(meta + plan.off_seqs);
    p.items = reinterpret_cast<const WorkItem*>(meta + plan.off_items);
    p.groups = reinterpret_cast<const CombineGroup*>(meta + plan.off_groups);
  }
  p.part_o = reinterpret_cast<uint16_t*>(ws + part + (plan.off_part_o - plan.meta_bytes));
  p.part_ml = reinterpret_cast<float*>(ws + part + (plan.off_part_ml - plan.meta_bytes));
  p.n_items = static_cast<int32_t>(plan.items.size());
  p.n_groups = static_cast<int32_t>(plan.groups.size());
  p.part_rows = plan.part_rows;
  return p;
}

cw_status_t extend_impl(const void* q, const void* k_new, const void* v_new, void* k_pool,
                        void* v_pool, const float* k_scale, const float* v_scale,
                        const int32_t* block_table, int32_t bt_stride, int32_t num_pages,
                        const int32_t* lp, const int32_t* ls, int32_t num_seqs,
                        int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                        int32_t page_size, float softmax_scale, cw_kv_dtype_t kv_dtype, void* out,
                        float* lse, void* workspace, size_t workspace_bytes, hipStream_t stream,
                        bool decode, bool write_pages, bool no_alloc = false) {
  cw_status_t s = check_shape(num_seqs, num_kv_heads, gqa_group, head_dim, page_size);
  if (s != CW_OK) return s;
  s = check_dtype(kv_dtype, k_scale, v_scale);
  if (s != CW_OK) return s;
  if (!(softmax_scale > 0.0f) || !std::isfinite(softmax_scale))
    return fail(CW_ERR_UNSUPPORTED, "softmax_scale = %g (must be finite and > 0)", double(softmax_scale));
  if (num_pages < 0) return fail(CW_ERR_BAD_LENS, "num_pages = %d is negative", num_pages);
  s = check_lens(lp, ls, num_seqs, bt_stride, page_size, num_kv_heads, gqa_group, head_dim, true);
  if (s != CW_OK) return s;
  const int64_t total = sum_suffix(ls, num_seqs);
  if (total == 0) return CW_OK;  // no rows: nothing to do
  if (!q || !k_new || !v_new || !out || !block_table)
    return fail(CW_ERR_NULL, "q, k_new, v_new, out and block_table are required");
  bool any_prefix = write_pages;  // the fused page write needs the pools too
  for (int32_t b = 0; b < num_seqs; ++b) any_prefix |= lp[b] > 0;
  if (any_prefix && (!k_pool || !v_pool)) return fail(CW_ERR_NULL, "k_pool / v_pool is NULL");
  if (!aligned16(q) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(out) ||
      !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(workspace))
    return fail(CW_ERR_ALIGN, "tensor and workspace pointers must be 16-byte aligned");
  if (lse && (reinterpret_cast<uintptr_t>(lse) & 3u)) return fail(CW_ERR_ALIGN, "lse not 4-byte aligned");
  if ((reinterpret_cast<uintptr_t>(block_table) & 3u)) return fail(CW_ERR_ALIGN, "block_table not 4-byte aligned");

  ExtendPlan plan = decode ? make_decode_plan(lp, num_seqs, num_kv_heads, gqa_group, head_dim, page_size, kv_dtype)
                           : make_plan(lp, ls, num_seqs, num_kv_heads, gqa_group, head_dim);
  if (no_alloc && plan.total_bytes > workspace_bytes)
    return fail(CW_ERR_WORKSPACE, "the call needs %zu bytes of scratch; the static scratch array holds %zu",
                plan.total_bytes, workspace_bytes);
  if (workspace == nullptr || workspace_bytes < plan.total_bytes)
    return fail(CW_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, plan.total_bytes);
  s = check_attention_alias(q, k_new, v_new, k_pool, v_pool, k_scale, v_scale, block_table,
                            bt_stride, num_pages, num_seqs, num_kv_heads, gqa_group, head_dim,
                            page_size, kv_dtype, total, out, lse, workspace, workspace_bytes);
  if (s != CW_OK) return s;

  uint8_t* ws = static_cast<uint8_t*>(workspace);
  ExtendParams p{};
  p.q = q;
  p.k_new = k_new;
  p.v_new = v_new;
  p.k_pool = k_pool;
  p.v_pool = v_pool;
  p.k_scale = k_scale;
  p.v_scale = v_scale;
  p.block_table = block_table;
  p.out = out;
  p.lse = lse;
  p.part_o = reinterpret_cast<uint16_t*>(ws + plan.off_part_o);
  p.part_ml = reinterpret_cast<float*>(ws + plan.off_part_ml);
  p.bt_stride = bt_stride;
  p.num_kv_heads = num_kv_heads;
  p.gqa_group = gqa_group;
  p.num_seqs = num_seqs;
  p.scale_log2 = softmax_scale * 1.4426950408889634f;
  p.n_items = static_cast<int32_t>(plan.items.size());
  p.n_groups = static_cast<int32_t>(plan.groups.size());
  p.part_rows = plan.part_rows;
  if (write_pages) {
    p.w.k_new = k_new;
    p.w.v_new = v_new;
    p.w.k_pool = k_pool;
    p.w.v_pool = v_pool;
    p.w.k_scale = k_scale;
    p.w.v_scale = v_scale;
    p.w.block_table = block_table;
    p.w.bt_stride = bt_stride;
    p.w.num_seqs = num_seqs;
    p.w.num_kv_heads = num_kv_heads;
    p.w.total_tokens = static_cast<int32_t>(total);
  }
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  {
    std::lock_guard<std::mutex> g(g_tuning_mu);
    ev0 = g_ev_start;
    ev1 = g_ev_stop;
  }
  const bool fp8 = kv_dtype == CW_KV_FP8_E4M3FN;
  CompactUpload cu;
  const bool compact = decode && compact_upload(plan, 0, &cu);
  auto launch = [&](const uint8_t* meta, const ArgPlan* ap) -> cw_status_t {
    if (ap != nullptr) {  // the plan is in the kernel arguments (decodes: in compact form)
      p.seqs = nullptr;
      p.items = nullptr;
      p.groups = nullptr;
      p.ap_seqs = static_cast<int32_t>(plan.off_seqs);
      p.ap_items = static_cast<int32_t>(plan.off_items);
      p.ap_groups = static_cast<int32_t>(plan.off_groups);
      p.ap_wseqs = static_cast<int32_t>(plan.off_seqs);
      p.ap_desc = decode ? static_cast<int32_t>(cu.bytes) : 0;
    } else {
      p.seqs = reinterpret_cast<const SeqInfo*>(meta + plan.off_seqs);
      p.items = reinterpret_cast<const WorkItem*>(meta + plan.off_items);
      p.groups = reinterpret_cast<const CombineGroup*>(meta + plan.off_groups);
    }
    if (write_pages) p.w.seqs = p.seqs;
    hipError_t e = hipSuccess;
    if (ev0 && (e = hipEventRecord(ev0, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    if (decode) e = launch_decode(p, head_dim, page_size, fp8, stream, ap);
    else e = launch_extend(p, head_dim, page_size, fp8, stream, ap);
    if (e != hipSuccess) return hip_fail(e, "extend kernel launch");
    if (ev1 && (e = hipEventRecord(ev1, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    if (p.n_groups > 0) {
      int max_parts = 0;
      for (const CombineGroup& g : plan.groups) max_parts = std::max(max_parts, g.n_parts);
      e = launch_combine(p, head_dim, max_parts, stream, ap);
      if (e != hipSuccess) return hip_fail(e, "combine kernel launch");
    }
    return CW_OK;
  };
  const bool arg_plan = arg_plans() && (decode ? compact && compact_arg_fits(cu) : true);
  return stage_and_launch(plan.meta_bytes, ws, stream, [&](uint8_t* h) { pack_plan_meta(plan, h); },
                          launch, no_alloc, plan_direct(no_alloc), compact ? &cu : nullptr,
                          [&](uint8_t* h) { pack_plan_head(plan, h); }, arg_plan);
}

// Shared by both swap directions: validates and enqueues block src_ids[i] of
// the source pools -> block dst_ids[i] of the destination pools.
cw_status_t swap_impl(const void* src_k, const void* src_v, const float* src_ks,
                      const float* src_vs, int32_t n_src_blocks, void* dst_k, void* dst_v,
                      float* dst_ks, float* dst_vs, int32_t n_dst_blocks, const int32_t* src_ids,
                      const int32_t* dst_ids, int32_t n, int32_t num_kv_heads, int32_t head_dim,
                      int32_t page_size, cw_kv_dtype_t kv_dtype, void* workspace,
                      size_t workspace_bytes, hipStream_t stream) {
  cw_status_t s = check_shape(0, num_kv_heads, 1, head_dim, page_size);
  if (s != CW_OK) return s;
  if (kv_dtype != CW_KV_BF16 && kv_dtype != CW_KV_FP8_E4M3FN)
    return fail(CW_ERR_UNSUPPORTED, "kv_dtype = %d", int(kv_dtype));
  const bool fp8 = kv_dtype == CW_KV_FP8_E4M3FN;
  if (n < 0 || n_src_blocks < 0 || n_dst_blocks < 0)
    return fail(CW_ERR_BAD_LENS, "negative count (n = %d, pools of %d and %d blocks)", n, n_src_blocks,
                n_dst_blocks);
  if (n == 0) return CW_OK;
  if (!src_ids || !dst_ids) return fail(CW_ERR_NULL, "the block lists are required");
  if (!src_k || !src_v || !dst_k || !dst_v) return fail(CW_ERR_NULL, "K and V pools of both sides are required");
  if (fp8 && (!src_ks || !src_vs || !dst_ks || !dst_vs))
    return fail(CW_ERR_NULL, "fp8 pools need the scales of both sides");
  if (!aligned16(src_k) || !aligned16(src_v) || !aligned16(dst_k) || !aligned16(dst_v) || !aligned16(workspace))
    return fail(CW_ERR_ALIGN, "pool and workspace pointers must be 16-byte aligned");
  std::vector<uint8_t> seen(size_t(n_dst_blocks), 0);
  for (int32_t i = 0; i < n; ++i) {
    if (src_ids[i] < 0 || src_ids[i] >= n_src_blocks || dst_ids[i] < 0 || dst_ids[i] >= n_dst_blocks)
      return fail(CW_ERR_BAD_LENS, "entry %d: block %d -> %d out of range (%d, %d blocks)", i, src_ids[i],
                  dst_ids[i], n_src_blocks, n_dst_blocks);
    if (seen[dst_ids[i]]++)
      return fail(CW_ERR_BAD_LENS, "entry %d: destination block %d appears twice", i, dst_ids[i]);
  }
  const size_t need = cw_swap_workspace_bytes(n);
  if (workspace == nullptr || workspace_bytes < need)
    return fail(CW_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
  // the kernel dereferences both sides: each pool pointer must be device memory
  // or host memory mapped into the device at the same address (pinned)
  const void* sides[] = {src_k, src_v, dst_k, dst_v, src_ks, src_vs, dst_ks, dst_vs};
  for (const void* ptr : sides) {
    if (ptr == nullptr) continue;
    hipPointerAttribute_t attr{};
    const hipError_t pe = hipPointerGetAttributes(&attr, ptr);
    const bool ok = pe == hipSuccess &&
                    (attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeManaged ||
                     attr.type == hipMemoryTypeUnified ||
                     (attr.type == hipMemoryTypeHost && attr.devicePointer == ptr));
    if (!ok) {
      (void)hipGetLastError();  // the query's error is ours, not a later call's
      return fail(CW_ERR_UNSUPPORTED, "pool pointer %p is not device-accessible (pageable host memory?)", ptr);
    }
  }
  std::vector<int32_t> lists(size_t(2) * n);
  std::copy(src_ids, src_ids + n, lists.begin());
  std::copy(dst_ids, dst_ids + n, lists.begin() + n);
  s = upload(lists.data(), lists.size() * sizeof(int32_t), workspace, stream);
  if (s != CW_OK) return s;
  SwapParams p{};
  p.src_k = static_cast<const uint8_t*>(src_k);
  p.src_v = static_cast<const uint8_t*>(src_v);
  p.dst_k = static_cast<uint8_t*>(dst_k);
  p.dst_v = static_cast<uint8_t*>(dst_v);
  if (fp8) {
    p.src_ks = src_ks;
    p.src_vs = src_vs;
    p.dst_ks = dst_ks;
    p.dst_vs = dst_vs;
  }
  p.src_ids = static_cast<const int32_t*>(workspace);
  p.dst_ids = static_cast<const int32_t*>(workspace) + n;
  p.n = n;
  p.block_bytes = num_kv_heads * page_size * head_dim * (fp8 ? 1 : 2);
  p.scales_per_block = num_kv_heads;
  const hipError_t e = launch_swap(p, stream);
  if (e != hipSuccess) return hip_fail(e, "swap kernel launch");
  return CW_OK;
}

cw_status_t step_impl(const void* q, const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                      const float* k_scale, const float* v_scale, const int32_t* block_table,
                      int32_t bt_stride, int32_t num_pages, const int32_t* lp, const int32_t* ls,
                      int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                      int32_t page_size, float softmax_scale, cw_kv_dtype_t kv_dtype, void* out,
                      float* lse, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  cw_status_t s = check_shape(num_seqs, num_kv_heads, gqa_group, head_dim, page_size);
  if (s != CW_OK) return s;
  s = check_dtype(kv_dtype, k_scale, v_scale);
  if (s != CW_OK) return s;
  if (!(softmax_scale > 0.0f) || !std::isfinite(softmax_scale))
    return fail(CW_ERR_UNSUPPORTED, "softmax_scale = %g (must be finite and > 0)", double(softmax_scale));
  if (num_pages < 0) return fail(CW_ERR_BAD_LENS, "num_pages = %d is negative", num_pages);
  s = check_lens(lp, ls, num_seqs, bt_stride, page_size, num_kv_heads, gqa_group, head_dim, true);
  if (s != CW_OK) return s;
  const int64_t total = sum_suffix(ls, num_seqs);
  if (total == 0) return CW_OK;
  if (!q || !k_new || !v_new || !out || !block_table)
    return fail(CW_ERR_NULL, "q, k_new, v_new, out and block_table are required");
  if (!k_pool || !v_pool) return fail(CW_ERR_NULL, "k_pool / v_pool is NULL");
  if (!aligned16(q) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(out) ||
      !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(workspace))
    return fail(CW_ERR_ALIGN, "tensor and workspace pointers must be 16-byte aligned");
  if (lse && (reinterpret_cast<uintptr_t>(lse) & 3u)) return fail(CW_ERR_ALIGN, "lse not 4-byte aligned");
  if ((reinterpret_cast<uintptr_t>(block_table) & 3u)) return fail(CW_ERR_ALIGN, "block_table not 4-byte aligned");

  const StepPlan sp = make_step_plan(lp, ls, num_seqs, num_kv_heads, gqa_group, head_dim, page_size, kv_dtype);
  if (workspace == nullptr || workspace_bytes < sp.total_bytes)
    return fail(CW_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, sp.total_bytes);
  s = check_attention_alias(q, k_new, v_new, k_pool, v_pool, k_scale, v_scale, block_table,
                            bt_stride, num_pages, num_seqs, num_kv_heads, gqa_group, head_dim,
                            page_size, kv_dtype, total, out, lse, workspace, workspace_bytes);
  if (s != CW_OK) return s;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  auto common = [&](ExtendParams& p) {
    p.q = q;
    p.k_new = k_new;
    p.v_new = v_new;
    p.k_pool = k_pool;
    p.v_pool = v_pool;
    p.k_scale = k_scale;
    p.v_scale = v_scale;
    p.block_table = block_table;
    p.out = out;
    p.lse = lse;
    p.bt_stride = bt_stride;
    p.num_kv_heads = num_kv_heads;
    p.gqa_group = gqa_group;
    p.num_seqs = num_seqs;
    p.scale_log2 = softmax_scale * 1.4426950408889634f;
  };
  WriteParams w{};
  w.k_new = k_new;
  w.v_new = v_new;
  w.k_pool = k_pool;
  w.v_pool = v_pool;
  w.k_scale = k_scale;
  w.v_scale = v_scale;
  w.block_table = block_table;
  w.bt_stride = bt_stride;
  w.num_seqs = num_seqs;
  w.num_kv_heads = num_kv_heads;
  w.total_tokens = static_cast<int32_t>(total);

  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  {
    std::lock_guard<std::mutex> g(g_tuning_mu);
    ev0 = g_ev_start;
    ev1 = g_ev_stop;
  }
  const bool fp8 = kv_dtype == CW_KV_FP8_E4M3FN;
  CompactUpload cu;
  const bool compact = !sp.dec.empty() && compact_upload(sp.dec_plan, sp.off_dec_meta, &cu);
  auto launch = [&](const uint8_t* meta, const ArgPlan* ap) -> cw_status_t {
    // with an argument plan (steps of extends only, or of decodes only with the
    // decode plan in compact form) the step's sequences sit at its byte 0, the
    // extend meta at off_ext_meta and the decode meta at off_dec_meta
    w.seqs = ap != nullptr ? nullptr : reinterpret_cast<const SeqInfo*>(meta);
    hipError_t e = hipSuccess;
    // the timing events bracket the extend kernel, or the decode kernel of a
    // step without extends
    if (sp.ext.empty() && ev0 && (e = hipEventRecord(ev0, stream)) != hipSuccess)
      return hip_fail(e, "hipEventRecord");
    if (!sp.dec.empty()) {
      ExtendParams pd = plan_params(sp.dec_plan, ap != nullptr ? nullptr : meta + sp.off_dec_meta, ws,
                                    sp.off_dec_part);
      common(pd);
      // without extends, the decode launch performs the page write (each
      // sequence's one new token, stored by the work item holding its key)
      if (sp.ext.empty()) pd.w = w;
      if (ap != nullptr) {
        pd.ap_seqs = static_cast<int32_t>(sp.off_dec_meta + sp.dec_plan.off_seqs);
        pd.ap_desc = static_cast<int32_t>(cu.bytes);
      }
      if ((e = launch_decode(pd, head_dim, page_size, fp8, stream, ap)) != hipSuccess)
        return hip_fail(e, "decode kernel launch");
      if (sp.ext.empty() && ev1 && (e = hipEventRecord(ev1, stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
      if (pd.n_groups > 0) {
        int max_parts = 0;
        for (const CombineGroup& g : sp.dec_plan.groups) max_parts = std::max(max_parts, g.n_parts);
        if ((e = launch_combine(pd, head_dim, max_parts, stream, ap)) != hipSuccess)
          return hip_fail(e, "combine kernel launch");
      }
    }
    if (!sp.ext.empty()) {
      ExtendParams pe = plan_params(sp.ext_plan, ap != nullptr ? nullptr : meta + sp.off_ext_meta, ws,
                                    sp.off_ext_part);
      common(pe);
      pe.w = w;  // every sequence's new K/V, written under the extend's first tiles
      if (ap != nullptr) {
        pe.seqs = nullptr;
        pe.items = nullptr;
        pe.groups = nullptr;
        pe.ap_seqs = static_cast<int32_t>(sp.off_ext_meta + sp.ext_plan.off_seqs);
        pe.ap_items = static_cast<int32_t>(sp.off_ext_meta + sp.ext_plan.off_items);
        pe.ap_groups = static_cast<int32_t>(sp.off_ext_meta + sp.ext_plan.off_groups);
        pe.ap_wseqs = 0;
      }
      if (ev0 && (e = hipEventRecord(ev0, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
      if ((e = launch_extend(pe, head_dim, page_size, fp8, stream, ap)) != hipSuccess)
        return hip_fail(e, "extend kernel launch");
      if (ev1 && (e = hipEventRecord(ev1, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
      if (pe.n_groups > 0) {
        int max_parts = 0;
        for (const CombineGroup& g : sp.ext_plan.groups) max_parts = std::max(max_parts, g.n_parts);
        if ((e = launch_combine(pe, head_dim, max_parts, stream, ap)) != hipSuccess)
          return hip_fail(e, "combine kernel launch");
      }
    }
    return CW_OK;
  };
  // the step's sequences and the extend meta, then the decode meta (in full or
  // in compact form, rebuilt by the upload kernel)
  auto head = [&](uint8_t* h) {
    std::fill(h, h + sp.off_ext_meta, uint8_t(0));
    std::copy(reinterpret_cast<const uint8_t*>(sp.seqs.data()),
              reinterpret_cast<const uint8_t*>(sp.seqs.data() + sp.seqs.size()), h);
    if (!sp.ext.empty()) pack_plan_meta(sp.ext_plan, h + sp.off_ext_meta);
  };
  const bool arg_plan =
      arg_plans() && (sp.dec.empty() || (sp.ext.empty() && compact && compact_arg_fits(cu)));
  return stage_and_launch(sp.meta_bytes, ws, stream, [&](uint8_t* h) {
    head(h);
    if (!sp.dec.empty()) pack_plan_meta(sp.dec_plan, h + sp.off_dec_meta);
  }, launch, false, plan_direct(false), compact ? &cu : nullptr, [&](uint8_t* h) {
    head(h);
    pack_plan_head(sp.dec_plan, h + sp.off_dec_meta);
  }, arg_plan);
}

// Runs an entry point's body: a failed host allocation (or any other C++
// exception) becomes a status, so nothing is thrown across the C ABI.
template <class F>
cw_status_t guarded(F&& f) {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    return fail(CW_ERR_UNSUPPORTED, "out of host memory");
  } catch (const std::exception& e) {
    return fail(CW_ERR_UNSUPPORTED, "%s", e.what());
  }
}
template <class T, class F>
T guarded_value(T on_error, F&& f) {
  try {
    return f();
  } catch (...) {
    return on_error;
  }
}

}  // namespace
}  // namespace cw

using namespace cw;

extern "C" {

size_t cw_swap_workspace_bytes(int32_t n) {
  if (n < 0) return 0;
  return std::max<size_t>(256, (size_t(n) * 2 * sizeof(int32_t) + 255) & ~size_t(255));
}

cw_status_t cw_kv_swap_out(const void* k_pool, const void* v_pool, const float* k_scale,
                           const float* v_scale, int32_t num_pages, void* k_host, void* v_host,
                           float* k_scale_host, float* v_scale_host, int32_t num_host_blocks,
                           const int32_t* pages_h, const int32_t* host_blocks_h, int32_t n,
                           int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                           cw_kv_dtype_t kv_dtype, void* workspace, size_t workspace_bytes,
                           hipStream_t stream) {
  return guarded([&]() -> cw_status_t {
    return swap_impl(k_pool, v_pool, k_scale, v_scale, num_pages, k_host, v_host, k_scale_host,
                     v_scale_host, num_host_blocks, pages_h, host_blocks_h, n, num_kv_heads, head_dim,
                     page_size, kv_dtype, workspace, workspace_bytes, stream);
  });
}

cw_status_t cw_kv_swap_in(const void* k_host, const void* v_host, const float* k_scale_host,
                          const float* v_scale_host, int32_t num_host_blocks, void* k_pool,
                          void* v_pool, float* k_scale, float* v_scale, int32_t num_pages,
                          const int32_t* host_blocks_h, const int32_t* pages_h, int32_t n,
                          int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                          cw_kv_dtype_t kv_dtype, void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  return guarded([&]() -> cw_status_t {
    return swap_impl(k_host, v_host, k_scale_host, v_scale_host, num_host_blocks, k_pool, v_pool,
                     k_scale, v_scale, num_pages, host_blocks_h, pages_h, n, num_kv_heads, head_dim,
                     page_size, kv_dtype, workspace, workspace_bytes, stream);
  });
}

size_t cw_write_pages_workspace_bytes(int32_t num_seqs) {
  if (num_seqs < 0) return 0;
  return std::max<size_t>(256, (size_t(num_seqs) * sizeof(SeqInfo) + 255) & ~size_t(255));
}

cw_status_t cw_check_block_table(const int32_t* block_table, int32_t bt_stride, int32_t num_pages,
                                 const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                                 int32_t num_seqs, int32_t page_size, int32_t* bad_per_seq,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return guarded([&]() -> cw_status_t {
    cw_status_t s = check_shape(num_seqs, 1, 1, 64, page_size);
    if (s != CW_OK) return s;
    if (num_pages < 0) return fail(CW_ERR_BAD_LENS, "num_pages = %d is negative", num_pages);
    s = check_lens(prefix_lens_h, suffix_lens_h, num_seqs, bt_stride, page_size, 1, 1, 64, true);
    if (s != CW_OK) return s;
    if (num_seqs == 0) return CW_OK;
    if (!block_table || !bad_per_seq) return fail(CW_ERR_NULL, "block_table and bad_per_seq are required");
    if ((reinterpret_cast<uintptr_t>(block_table) & 3u) || (reinterpret_cast<uintptr_t>(bad_per_seq) & 3u))
      return fail(CW_ERR_ALIGN, "block_table and bad_per_seq must be 4-byte aligned");
    if (!aligned16(workspace)) return fail(CW_ERR_ALIGN, "workspace must be 16-byte aligned");
    const size_t need = cw_write_pages_workspace_bytes(num_seqs);
    if (workspace == nullptr || workspace_bytes < need)
      return fail(CW_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    std::vector<SeqInfo> seqs(num_seqs);
    int64_t cu = 0;
    for (int32_t b = 0; b < num_seqs; ++b) {
      seqs[b] = SeqInfo{prefix_lens_h[b], suffix_lens_h[b], static_cast<int32_t>(cu), b};
      cu += suffix_lens_h[b];
    }
    s = upload(seqs.data(), seqs.size() * sizeof(SeqInfo), workspace, stream);
    if (s != CW_OK) return s;
    const hipError_t e = launch_check_table(block_table, bt_stride, num_pages,
                                            static_cast<const SeqInfo*>(workspace), num_seqs,
                                            page_size, bad_per_seq, stream);
    return e == hipSuccess ? CW_OK : hip_fail(e, "check_table kernel launch");
  });
}

cw_status_t cw_kv_write_pages(const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                              const float* k_scale, const float* v_scale,
                              const int32_t* block_table, int32_t bt_stride, int32_t num_pages,
                              const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                              int32_t num_seqs, int32_t num_kv_heads, int32_t head_dim,
                              int32_t page_size, cw_kv_dtype_t kv_dtype, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  return guarded([&]() -> cw_status_t {
    cw_status_t s = check_shape(num_seqs, num_kv_heads, 1, head_dim, page_size);
    if (s != CW_OK) return s;
    s = check_dtype(kv_dtype, k_scale, v_scale);
    if (s != CW_OK) return s;
    if (num_pages < 0) return fail(CW_ERR_BAD_LENS, "num_pages = %d is negative", num_pages);
    s = check_lens(prefix_lens_h, suffix_lens_h, num_seqs, bt_stride, page_size, num_kv_heads, 1,
                   head_dim, true);
    if (s != CW_OK) return s;
    const int64_t total = sum_suffix(suffix_lens_h, num_seqs);
    if (total == 0) return CW_OK;
    if (!k_new || !v_new || !k_pool || !v_pool || !block_table)
      return fail(CW_ERR_NULL, "k_new, v_new, k_pool, v_pool and block_table are required");
    if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pool) || !aligned16(v_pool) ||
        !aligned16(workspace))
      return fail(CW_ERR_ALIGN, "tensor and workspace pointers must be 16-byte aligned");
    const size_t need = cw_write_pages_workspace_bytes(num_seqs);
    if (workspace == nullptr || workspace_bytes < need)
      return fail(CW_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    std::vector<SeqInfo> seqs(num_seqs);
    int64_t cu = 0;
    for (int32_t b = 0; b < num_seqs; ++b) {
      seqs[b] = SeqInfo{prefix_lens_h[b], suffix_lens_h[b], static_cast<int32_t>(cu), b};
      cu += suffix_lens_h[b];
    }
    s = upload(seqs.data(), seqs.size() * sizeof(SeqInfo), workspace, stream);
    if (s != CW_OK) return s;
    WriteParams p{};
    p.k_new = k_new;
    p.v_new = v_new;
    p.k_pool = k_pool;
    p.v_pool = v_pool;
    p.k_scale = k_scale;
    p.v_scale = v_scale;
    p.block_table = block_table;
    p.seqs = static_cast<const SeqInfo*>(workspace);
    p.bt_stride = bt_stride;
    p.num_seqs = num_seqs;
    p.num_kv_heads = num_kv_heads;
    p.total_tokens = static_cast<int32_t>(total);
    hipError_t e = launch_write_pages(p, head_dim, page_size, kv_dtype == CW_KV_FP8_E4M3FN, stream);
    if (e != hipSuccess) return hip_fail(e, "write_pages kernel launch");
    return CW_OK;
  });
}

size_t cw_extend_workspace_bytes(const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                                 int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                                 int32_t head_dim, int32_t page_size) {
  return guarded_value<size_t>(0, [&]() -> size_t {
    if (check_shape(num_seqs, num_kv_heads, gqa_group, head_dim, page_size) != CW_OK) return 0;
    if (check_lens(prefix_lens_h, suffix_lens_h, num_seqs, 0, page_size, num_kv_heads, gqa_group,
                   head_dim, false) != CW_OK)
      return 0;
    if (num_seqs == 0) return 256;
    return make_plan(prefix_lens_h, suffix_lens_h, num_seqs, num_kv_heads, gqa_group, head_dim).total_bytes;
  });
}

cw_status_t cw_extend_attention(const void* q, const void* k_new, const void* v_new,
                                const void* k_pool, const void* v_pool, const float* k_scale,
                                const float* v_scale, const int32_t* block_table,
                                int32_t bt_stride, int32_t num_pages,
                                const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                                int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                                int32_t head_dim, int32_t page_size, float softmax_scale,
                                cw_kv_dtype_t kv_dtype, void* out, float* lse, void* workspace,
                                size_t workspace_bytes, hipStream_t stream) {
  return guarded([&]() -> cw_status_t {
    return extend_impl(q, k_new, v_new, const_cast<void*>(k_pool), const_cast<void*>(v_pool), k_scale,
                       v_scale, block_table, bt_stride, num_pages, prefix_lens_h, suffix_lens_h,
                       num_seqs, num_kv_heads, gqa_group, head_dim, page_size, softmax_scale, kv_dtype,
                       out, lse, workspace, workspace_bytes, stream, false, false);
  });
}

cw_status_t cw_write_extend_attention(const void* q, const void* k_new, const void* v_new,
                                      void* k_pool, void* v_pool, const float* k_scale,
                                      const float* v_scale, const int32_t* block_table,
                                      int32_t bt_stride, int32_t num_pages,
                                      const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                                      int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                                      int32_t head_dim, int32_t page_size, float softmax_scale,
                                      cw_kv_dtype_t kv_dtype, void* out, float* lse,
                                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return guarded([&]() -> cw_status_t {
    return extend_impl(q, k_new, v_new, k_pool, v_pool, k_scale, v_scale, block_table, bt_stride,
                       num_pages, prefix_lens_h, suffix_lens_h, num_seqs, num_kv_heads, gqa_group,
                       head_dim, page_size, softmax_scale, kv_dtype, out, lse, workspace,
                       workspace_bytes, stream, false, true);
  });
}

size_t cw_step_workspace_bytes(const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                               int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                               int32_t head_dim, int32_t page_size, cw_kv_dtype_t kv_dtype) {
  return guarded_value<size_t>(0, [&]() -> size_t {
    if (check_shape(num_seqs, num_kv_heads, gqa_group, head_dim, page_size) != CW_OK) return 0;
    if (kv_dtype != CW_KV_BF16 && kv_dtype != CW_KV_FP8_E4M3FN) return 0;
    if (check_lens(prefix_lens_h, suffix_lens_h, num_seqs, 0, page_size, num_kv_heads, gqa_group,
                   head_dim, false) != CW_OK)
      return 0;
    if (num_seqs == 0) return 256;
    return make_step_plan(prefix_lens_h, suffix_lens_h, num_seqs, num_kv_heads, gqa_group, head_dim,
                          page_size, kv_dtype)
        .total_bytes;
  });
}

cw_status_t cw_step_attention(const void* q, const void* k_new, const void* v_new, void* k_pool,
                              void* v_pool, const float* k_scale, const float* v_scale,
                              const int32_t* block_table, int32_t bt_stride, int32_t num_pages,
                              const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                              int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                              int32_t head_dim, int32_t page_size, float softmax_scale,
                              cw_kv_dtype_t kv_dtype, void* out, float* lse, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  return guarded([&]() -> cw_status_t {
    return step_impl(q, k_new, v_new, k_pool, v_pool, k_scale, v_scale, block_table, bt_stride,
                     num_pages, prefix_lens_h, suffix_lens_h, num_seqs, num_kv_heads, gqa_group,
                     head_dim, page_size, softmax_scale, kv_dtype, out, lse, workspace,
                     workspace_bytes, stream);
  });
}

size_t cw_decode_workspace_bytes(const int32_t* prefix_lens_h, int32_t num_seqs,
                                 int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                                 int32_t page_size, cw_kv_dtype_t kv_dtype) {
  return guarded_value<size_t>(0, [&]() -> size_t {
    if (num_seqs < 0) return 0;
    if (kv_dtype != CW_KV_BF16 && kv_dtype != CW_KV_FP8_E4M3FN) return 0;
    std::vector<int32_t> ones(num_seqs, 1);
    if (check_shape(num_seqs, num_kv_heads, gqa_group, head_dim, page_size) != CW_OK) return 0;
    if (check_lens(prefix_lens_h, ones.data(), num_seqs, 0, page_size, num_kv_heads, gqa_group,
                   head_dim, false) != CW_OK)
      return 0;
    if (num_seqs == 0) return 256;
    return make_decode_plan(prefix_lens_h, num_seqs, num_kv_heads, gqa_group, head_dim, page_size, kv_dtype)
        .total_bytes;
  });
}

cw_status_t cw_decode_attention(const void* q, const void* k_new, const void* v_new,
                                const void* k_pool, const void* v_pool, const float* k_scale,
                                const float* v_scale, const int32_t* block_table,
                                int32_t bt_stride, int32_t num_pages,
                                const int32_t* prefix_lens_h, int32_t num_seqs,
                                int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                                int32_t page_size, float softmax_scale, cw_kv_dtype_t kv_dtype,
                                void* out, float* lse, void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  return guarded([&]() -> cw_status_t {
    if (num_seqs < 0) return fail(CW_ERR_BAD_LENS, "num_seqs = %d is negative", num_seqs);
    std::vector<int32_t> ones(num_seqs, 1);
    return extend_impl(q, k_new, v_new, const_cast<void*>(k_pool), const_cast<void*>(v_pool), k_scale,
                       v_scale, block_table, bt_stride, num_pages, prefix_lens_h, ones.data(),
                       num_seqs, num_kv_heads, gqa_group, head_dim, page_size, softmax_scale, kv_dtype,
                       out, lse, workspace, workspace_bytes, stream, true, false);
  });
}

cw_status_t cw_init(void) {
  DeviceState* st = nullptr;
  cw_status_t s = current_state(&st);
  if (s != CW_OK) return s;
  std::lock_guard<std::mutex> g(st->staging_mu);
  s = init_locked(*st);
  if (s != CW_OK || st->scratch != nullptr) return s;
  // this device's copy of the scratch array: the name is a host-side stand-in,
  // the address the runtime returns (with this device current) is the one kernels use
  void* ptr = nullptr;
  const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(::scratch));
  if (e != hipSuccess || ptr == nullptr)
    return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress(scratch)");
  st->scratch = static_cast<uint8_t*>(ptr);
  return CW_OK;
}

cw_status_t cw_extend_attention_noalloc(const void* q, const void* k_new, const void* v_new,
                                        const void* k_pool, const void* v_pool,
                                        const float* k_scale, const float* v_scale,
                                        const int32_t* block_table, int32_t bt_stride,
                                        int32_t num_pages, const int32_t* prefix_lens_h,
                                        const int32_t* suffix_lens_h, int32_t num_seqs,
                                        int32_t num_kv_heads, int32_t gqa_group, int32_t head_dim,
                                        int32_t page_size, float softmax_scale,
                                        cw_kv_dtype_t kv_dtype, void* out, float* lse,
                                        hipStream_t stream) {
  return guarded([&]() -> cw_status_t {
    DeviceState* st = nullptr;
    const cw_status_t s = current_state(&st);
    if (s != CW_OK) return s;
    uint8_t* ws = nullptr;
    {
      std::lock_guard<std::mutex> g(st->staging_mu);
      if (!st->ready || st->scratch == nullptr)
        return fail(CW_ERR_INIT, "cw_init() has not been called on this device");
      ws = st->scratch;
    }
    return extend_impl(q, k_new, v_new, const_cast<void*>(k_pool), const_cast<void*>(v_pool), k_scale,
                       v_scale, block_table, bt_stride, num_pages, prefix_lens_h, suffix_lens_h,
                       num_seqs, num_kv_heads, gqa_group, head_dim, page_size, softmax_scale, kv_dtype,
                       out, lse, ws, CW_NOALLOC_SCRATCH_BYTES, stream, false, false, true);
  });
}

int64_t cw_pinned_allocations(void) { return g_pinned_allocs.load(); }

int64_t cw_arg_plan_calls(void) { return g_arg_plan_calls.load(); }

cw_status_t cw_set_tuning(cw_tune_key_t key, int32_t value) {
  if (value < 0) return fail(CW_ERR_UNSUPPORTED, "tuning value %d is negative", value);
  std::lock_guard<std::mutex> g(g_tuning_mu);
  switch (key) {
    case CW_TUNE_KV_CHUNK_TILES: g_tuning.kv_chunk_tiles = value; return CW_OK;
    case CW_TUNE_TARGET_WGS: g_tuning.target_wgs = value; return CW_OK;
    case CW_TUNE_EXTEND_KERNEL:
      if (value > 2) return fail(CW_ERR_UNSUPPORTED, "extend kernel %d is not 0, 1 or 2", value);
      g_tuning.extend_kernel = value;
      return CW_OK;
    case CW_TUNE_DEAL_ROUNDS: g_tuning.deal_rounds = value; return CW_OK;
    case CW_TUNE_PLAN_DIRECT: g_tuning.plan_direct = value; return CW_OK;
    case CW_TUNE_SUFFIX_WEIGHT:
      if (value < 1 || value > 10000) return fail(CW_ERR_UNSUPPORTED, "suffix weight %d is not in 1 .. 10000", value);
      g_tuning.suffix_weight = value;
      return CW_OK;
    case CW_TUNE_COMPACT_DECODE:
      g_tuning.compact_decode = value;
      return CW_OK;
    case CW_TUNE_ARG_PLANS:
      g_tuning.arg_plans = value;
      return CW_OK;
    default: break;
  }
  return fail(CW_ERR_UNSUPPORTED, "unknown tuning key %d", int(key));
}

cw_status_t cw_set_timing_events(hipEvent_t start, hipEvent_t stop) {
  std::lock_guard<std::mutex> g(g_tuning_mu);
  g_ev_start = start;
  g_ev_stop = stop;
  return CW_OK;
}

int64_t cw_extend_plan_items(const int32_t* prefix_lens_h, const int32_t* suffix_lens_h,
                             int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                             int32_t head_dim, int32_t page_size, int32_t* items_out,
                             int64_t capacity) {
  return guarded_value<int64_t>(-1, [&]() -> int64_t {
    if (check_shape(num_seqs, num_kv_heads, gqa_group, head_dim, page_size) != CW_OK) return -1;
    if (check_lens(prefix_lens_h, suffix_lens_h, num_seqs, 0, page_size, num_kv_heads, gqa_group,
                   head_dim, false) != CW_OK)
      return -1;
    ExtendPlan plan = make_plan(prefix_lens_h, suffix_lens_h, num_seqs, num_kv_heads, gqa_group, head_dim);
    const int64_t n = static_cast<int64_t>(plan.items.size());
    if (items_out) {
      for (int64_t i = 0; i < std::min(n, capacity); ++i) {
        const WorkItem& w = plan.items[i];
        int32_t* o = items_out + 8 * i;
        o[0] = w.seq; o[1] = w.kvh; o[2] = w.q_row0; o[3] = w.kv_begin;
        o[4] = w.kv_end; o[5] = w.part; o[6] = w.rows; o[7] = 0;
      }
    }
    return n;
  });
}

int64_t cw_decode_plan_items(const int32_t* prefix_lens_h, int32_t num_seqs, int32_t num_kv_heads,
                             int32_t gqa_group, int32_t head_dim, int32_t page_size,
                             cw_kv_dtype_t kv_dtype, int32_t rebuilt, int32_t* items_out,
                             int64_t items_capacity, int32_t* groups_out, int64_t groups_capacity,
                             int64_t* num_groups) {
  return guarded_value<int64_t>(-1, [&]() -> int64_t {
    if (check_shape(num_seqs, num_kv_heads, gqa_group, head_dim, page_size) != CW_OK) return -1;
    if (kv_dtype != CW_KV_BF16 && kv_dtype != CW_KV_FP8_E4M3FN) return -1;
    if (!prefix_lens_h && num_seqs > 0) return -1;
    std::vector<int32_t> ones(size_t(std::max(num_seqs, 0)), 1);
    if (check_lens(prefix_lens_h, ones.data(), num_seqs, 0, page_size, num_kv_heads, gqa_group, head_dim,
                   false) != CW_OK)
      return -1;
    const ExtendPlan plan =
        make_decode_plan(prefix_lens_h, num_seqs, num_kv_heads, gqa_group, head_dim, page_size, kv_dtype);
    if (rebuilt && (!plan.compact || plan.recs.empty())) return -1;
    const int64_t n = static_cast<int64_t>(plan.items.size()), ng = static_cast<int64_t>(plan.groups.size());
    for (int64_t i = 0; items_out && i < std::min(n, items_capacity); ++i) {
      const WorkItem w = rebuilt ? expand_item(plan.recs.data(), plan.tails.data(), plan.desc, int32_t(i))
                                 : plan.items[i];
      int32_t* o = items_out + 8 * i;
      o[0] = w.seq; o[1] = w.kvh; o[2] = w.q_row0; o[3] = w.kv_begin;
      o[4] = w.kv_end; o[5] = w.part; o[6] = w.rows; o[7] = w.pad;
    }
    for (int64_t g = 0; groups_out && g < std::min(ng, groups_capacity); ++g) {
      const CombineGroup c = rebuilt ? expand_group(plan.recs.data(), plan.desc, int32_t(g)) : plan.groups[g];
      int32_t* o = groups_out + 8 * g;
      o[0] = c.seq; o[1] = c.kvh; o[2] = c.q_row0; o[3] = c.rows;
      o[4] = c.part0; o[5] = c.n_parts; o[6] = c.pad0; o[7] = c.pad1;
    }
    if (num_groups) *num_groups = ng;
    return n;
  });
}

const char* cw_status_string(cw_status_t status) {
  switch (status) {
    case CW_OK: return "CW_OK";
    case CW_ERR_NULL: return "CW_ERR_NULL: a required pointer is NULL";
    case CW_ERR_UNSUPPORTED: return "CW_ERR_UNSUPPORTED: unsupported shape, dtype or parameter";
    case CW_ERR_BAD_LENS: return "CW_ERR_BAD_LENS: invalid sequence lengths";
    case CW_ERR_ALIGN: return "CW_ERR_ALIGN: misaligned pointer";
    case CW_ERR_WORKSPACE: return "CW_ERR_WORKSPACE: workspace too small";
    case CW_ERR_HIP: return "CW_ERR_HIP: HIP runtime error";
    case CW_ERR_ALIAS: return "CW_ERR_ALIAS: an output overlaps an input or the workspace";
    case CW_ERR_INIT: return "CW_ERR_INIT: cw_init() has not been called on the current device";
    default: break;
  }
  return "unknown cw_status_t";
}

const char* cw_last_error_message(void) { return g_last_error.c_str(); }

int32_t cw_version(void) { return 200; }

}  // extern "C"
