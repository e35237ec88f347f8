// C-ABI of libhvdx: argument checks, the Tensor Fusion plan (host), and the ring
// step sequence.  Every check runs before the first HIP call, so invalid requests
// return an error without touching the GPU.

#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <initializer_list>
#include <mutex>
#include <utility>
#include <vector>

#include "internal.hpp"

namespace {

thread_local char g_last_error[512] = "";

// ---- timeline state ----------------------------------------------------------------
struct TimelineEntry {
  hvdx_trace_record rec;
  hipEvent_t start, end;
};

struct Timeline {
  std::recursive_mutex mu;  // a phase record wraps the launches it covers
  bool on = false;
  bool per_phase = false;
  int capacity = 0;
  int dropped = 0;
  std::vector<hipEvent_t> pool;  // 2 * capacity events, created at begin
  std::vector<TimelineEntry> entries;
};

Timeline& timeline() {
  static Timeline t;
  return t;
}

}  // namespace

hvdx::LaunchEvents& hvdx::pending_launch_events() {
  thread_local LaunchEvents ev;
  return ev;
}

namespace {

// Times kernel launches for the timeline when it records at this granularity.  A
// launch record (per-launch mode) hands its events to the one launch in its scope,
// which stamps them with the kernel's own start and end; a phase record (per-phase
// mode) covers several launches with event records in the stream before and after.
class TimedLaunch {
 public:
  TimedLaunch(int kind, int step, int nranks, int dtype, int compress, int64_t count, hipStream_t st, int root = -1,
              bool phase = false, int launches = 1)
      : st_(st), lock_(timeline().mu) {
    Timeline& t = timeline();
    if (!t.on || t.per_phase != phase) return;
    // Launches recorded into a HIP graph run later, at each replay: they get no record.
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st_, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return;
    if ((int)t.entries.size() >= t.capacity) {
      ++t.dropped;
      return;
    }
    TimelineEntry e{};
    e.rec.kind = kind;
    e.rec.step = step;
    e.rec.launches = launches;
    e.rec.nranks = nranks;
    e.rec.dtype = dtype;
    e.rec.compress = compress;
    e.rec.root = root;
    e.rec.count = count;
    e.start = t.pool[2 * t.entries.size()];
    e.end = t.pool[2 * t.entries.size() + 1];
    if (!phase) {
      t.entries.push_back(e);
      hvdx::pending_launch_events() = {e.start, e.end};
      start_ = e.start;
      end_ = e.end;
    } else if (hipEventRecord(e.start, st_) == hipSuccess) {
      t.entries.push_back(e);
      end_ = e.end;
    }
  }
  // The lock is still held here: no other thread's launch lands inside the record.
  ~TimedLaunch() {
    if (start_) {
      hvdx::LaunchEvents& ev = hvdx::pending_launch_events();
      if (ev.start == start_) {  // nothing was launched (an error): a zero-length record
        ev = hvdx::LaunchEvents{};
        (void)hipEventRecord(start_, st_);
        (void)hipEventRecord(end_, st_);
      }
      return;
    }
    if (end_) (void)hipEventRecord(end_, st_);
  }

 private:
  hipStream_t st_;
  std::unique_lock<std::recursive_mutex> lock_;
  hipEvent_t start_ = nullptr, end_ = nullptr;
};

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(HVDX_ERR_HIP, "%s: %s (%s)", what, hipGetErrorName(e), hipGetErrorString(e));
}

int elem_size(int dtype) {
  switch (dtype) {
    case HVDX_FLOAT32: return 4;
    case HVDX_FLOAT16: return 2;
    default: return 0;
  }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Pairwise disjointness of [base, base + bytes) over all ranges (sorted sweep).
bool overlapping(std::vector<std::pair<uintptr_t, uintptr_t>> ranges) {
  std::sort(ranges.begin(), ranges.end());
  for (size_t i = 1; i < ranges.size(); ++i)
    if (ranges[i].first < ranges[i - 1].second) return true;
  return false;
}

int check_rank_buffers(void* const* bufs, int nranks, int64_t count, int esize, const char* what) {
  if (!bufs) return fail(HVDX_ERR_INVALID, "%s: rank pointer array is NULL", what);
  if (nranks < 1 || nranks > HVDX_MAX_RANKS)
    return fail(HVDX_ERR_INVALID, "%s: nranks=%d outside 1..%d", what, nranks, HVDX_MAX_RANKS);
  if (count < 0) return fail(HVDX_ERR_INVALID, "%s: negative element count %lld", what, (long long)count);
  if (count > (INT64_MAX >> 4))  // byte extents below must not overflow
    return fail(HVDX_ERR_INVALID, "%s: element count %lld too large", what, (long long)count);
  for (int r = 0; r < nranks; ++r) {
    if (!bufs[r] && count > 0) return fail(HVDX_ERR_INVALID, "%s: buffer of rank %d is NULL", what, r);
    if (reinterpret_cast<uintptr_t>(bufs[r]) % esize)
      return fail(HVDX_ERR_INVALID, "%s: buffer of rank %d is not aligned to its element size", what, r);
  }
  if (count > 0) {
    std::vector<std::pair<uintptr_t, uintptr_t>> rg;
    for (int r = 0; r < nranks; ++r) {
      const uintptr_t b = reinterpret_cast<uintptr_t>(bufs[r]);
      rg.emplace_back(b, b + (uintptr_t)count * esize);
    }
    if (overlapping(rg)) return fail(HVDX_ERR_ALIAS, "%s: rank buffers overlap", what);
  }
  return HVDX_OK;
}

hvdx::RankPtrs rank_ptrs(void* const* bufs, int nranks) {
  hvdx::RankPtrs p{};
  for (int r = 0; r < nranks; ++r) p.p[r] = bufs[r];
  return p;
}

int64_t wire_stride(int64_t count) { return (count + 127) / 128 * 128; }

// Arguments shared by hvdx_ring_allreduce and hvdx_ring_step.
int check_ring(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress, void* workspace,
               size_t workspace_bytes, const char* what) {
  const int es = elem_size(dtype);
  if (!es) return fail(HVDX_ERR_INVALID, "%s: unknown dtype %d", what, dtype);
  if (op != HVDX_SUM && op != HVDX_AVERAGE) return fail(HVDX_ERR_INVALID, "%s: unknown op %d", what, op);
  if (compress != HVDX_COMPRESS_NONE && compress != HVDX_COMPRESS_FP16)
    return fail(HVDX_ERR_INVALID, "%s: unknown compression %d", what, compress);
  if (compress == HVDX_COMPRESS_FP16 && dtype != HVDX_FLOAT32)
    return fail(HVDX_ERR_INVALID, "%s: fp16 compression needs float32 buffers", what);
  int rc = check_rank_buffers(bufs, nranks, count, es, what);
  if (rc) return rc;
  if (compress == HVDX_COMPRESS_FP16 && nranks > 1 && count > 0) {
    const size_t need = hvdx_ring_workspace_bytes(nranks, count, dtype, compress);
    if (!workspace || workspace_bytes < need)
      return fail(HVDX_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", what,
                  workspace ? workspace_bytes : (size_t)0, need);
    if (reinterpret_cast<uintptr_t>(workspace) & 255)
      return fail(HVDX_ERR_WORKSPACE, "%s: workspace is not 256-byte aligned", what);
    std::vector<std::pair<uintptr_t, uintptr_t>> rg;
    const uintptr_t w = reinterpret_cast<uintptr_t>(workspace);
    rg.emplace_back(w, w + need);
    for (int r = 0; r < nranks; ++r) {
      const uintptr_t b = reinterpret_cast<uintptr_t>(bufs[r]);
      rg.emplace_back(b, b + (uintptr_t)count * es);
    }
    if (overlapping(rg)) return fail(HVDX_ERR_ALIAS, "%s: workspace overlaps a rank buffer", what);
  }
  return HVDX_OK;
}

hvdx::RingArgs ring_args(int nranks, int64_t count, int step) {
  hvdx::RingArgs a{};
  a.n = nranks;
  a.step = step;
  a.q = count / nranks;
  a.rem = count % nranks;
  a.nf = (float)nranks;
  a.inv = 1.0f / (float)nranks;
  a.wire_stride = wire_stride(count);
  return a;
}

int div_mode(int op, int nranks) {
  if (op != HVDX_AVERAGE || nranks == 1) return hvdx::DIV_NONE;
  return (nranks & (nranks - 1)) == 0 ? hvdx::DIV_POW2 : hvdx::DIV_TRUE;
}

bool vectors_ok(void* const* bufs, int nranks, const void* workspace) {
  for (int r = 0; r < nranks; ++r)
    if (!aligned16(bufs[r])) return false;
  return aligned16(workspace);
}

// One step, arguments already checked, nranks >= 2, count > 0.  `fused` runs adding
// step N-2 together with replacing step 0.
int run_step(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress, int phase, int step,
             void* workspace, hipStream_t st, bool fused = false) {
  const hvdx::RingArgs a = ring_args(nranks, count, step);
  const hvdx::RankPtrs p = rank_ptrs(bufs, nranks);
  const bool vok = vectors_ok(bufs, nranks, workspace);
  const int dm = (fused || step == nranks - 2) && phase == HVDX_PHASE_REDUCE_SCATTER ? div_mode(op, nranks)
                                                                                  : hvdx::DIV_NONE;
  const int kind = fused ? HVDX_KERNEL_RS_AG
                         : (phase == HVDX_PHASE_REDUCE_SCATTER ? HVDX_KERNEL_REDUCE_SCATTER : HVDX_KERNEL_ALLGATHER);
  TimedLaunch timed(kind, step, nranks, dtype, compress, count, st);
  hipError_t e;
  if (fused) {
    e = compress == HVDX_COMPRESS_FP16 ? hvdx::launch_rs_ag_step_c16(p, workspace, a, dm, vok, st)
                                       : hvdx::launch_rs_ag_step(p, a, dtype, dm, vok, st);
  } else if (compress == HVDX_COMPRESS_FP16) {
    e = phase == HVDX_PHASE_REDUCE_SCATTER ? hvdx::launch_rs_step_c16(p, workspace, a, dm, vok, st)
                                           : hvdx::launch_ag_step_c16(p, workspace, a, vok, st);
  } else {
    e = phase == HVDX_PHASE_REDUCE_SCATTER ? hvdx::launch_rs_step(p, a, dtype, dm, vok, st)
                                           : hvdx::launch_ag_step(p, a, dtype, vok, st);
  }
  if (e != hipSuccess)
    return hip_fail(e, fused ? "fused step launch"
                             : (phase == HVDX_PHASE_REDUCE_SCATTER ? "reduce-scatter step launch"
                                                                   : "allgather step launch"));
  return HVDX_OK;
}

// Steps [s0, s1) of one phase, as one timeline phase record.
int run_steps(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress, int phase, int s0,
              int s1, void* workspace, hipStream_t st) {
  if (s1 <= s0) return HVDX_OK;
  TimedLaunch timed(phase == HVDX_PHASE_REDUCE_SCATTER ? HVDX_KERNEL_REDUCE_SCATTER : HVDX_KERNEL_ALLGATHER, s0,
                    nranks, dtype, compress, count, st, -1, true, s1 - s0);
  for (int s = s0; s < s1; ++s) {
    const int rc = run_step(bufs, nranks, count, dtype, op, compress, phase, s, workspace, st);
    if (rc) return rc;
  }
  return HVDX_OK;
}

int check_fusion(const void* const* tensors, const int64_t* numel, const int64_t* offset, int ntensors,
                 int tensor_dtype, const void* const* bufs, int64_t buf_count, int buf_dtype, int nranks,
                 const char* what) {
  if (ntensors < 0) return fail(HVDX_ERR_INVALID, "%s: negative tensor count", what);
  if (ntensors > 0 && (!tensors || !numel || !offset))
    return fail(HVDX_ERR_INVALID, "%s: a descriptor array is NULL", what);
  const int es = elem_size(buf_dtype);
  if (!es || !elem_size(tensor_dtype)) return fail(HVDX_ERR_INVALID, "%s: unknown dtype", what);
  if (tensor_dtype == HVDX_FLOAT16 && buf_dtype == HVDX_FLOAT32)
    return fail(HVDX_ERR_UNSUPPORTED, "%s: float16 tensors with a float32 buffer", what);
  int rc = check_rank_buffers(const_cast<void* const*>(bufs), nranks, buf_count, es, what);
  if (rc) return rc;
  for (int r = 0; r < nranks; ++r)
    if (buf_count > 0 && !aligned16(bufs[r]))
      return fail(HVDX_ERR_INVALID, "%s: fusion buffer of rank %d is not 16-byte aligned", what, r);
  return HVDX_OK;
}

}  // namespace

// ---- the ring without a caller-provided workspace --------------------------------------
//
// The compressed ring's binary16 wire copies live in `scratch`, a static device array
// that the code object carries (one copy per GPU the library runs on, held until the
// process ends).  Its device address is looked up once per device, with that device
// current, and kept; host code never passes the array's own name to a kernel (on the
// host that name is only a stand-in for the device symbol).
namespace {
constexpr size_t kScratchBytes = (size_t)64 << 20;
__attribute__((used)) static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices] = {};

int scratch_for(hipStream_t st, void** out, const char* what) {
  int dev = -1;
  hipError_t e = st ? hipStreamGetDevice(st, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "static workspace: the stream's device");
  if (dev < 0 || dev >= kScratchDevices)
    return fail(HVDX_ERR_UNSUPPORTED, "%s: device %d beyond the %d this build serves", what, dev, kScratchDevices);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = -1;
    e = hipGetDevice(&cur);
    if (e != hipSuccess) return hip_fail(e, "static workspace: hipGetDevice");
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return hip_fail(e, "static workspace: hipSetDevice");
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess) return hip_fail(e, "static workspace: hipGetSymbolAddress");
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255))
      return fail(HVDX_ERR_HIP, "%s: static workspace address %p is not 256-byte aligned", what, p);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return HVDX_OK;
}
}  // namespace

extern "C" {

int hvdx_version(void) { return HVDX_VERSION; }

int hvdx_timeline_begin(int capacity, int per_phase) {
  if (capacity < 1 || capacity > (1 << 24)) return fail(HVDX_ERR_INVALID, "hvdx_timeline_begin: bad capacity %d", capacity);
  Timeline& t = timeline();
  std::lock_guard<std::recursive_mutex> g(t.mu);
  if (t.on) return fail(HVDX_ERR_INVALID, "hvdx_timeline_begin: a timeline is already recording");
  t.pool.assign(2 * (size_t)capacity, nullptr);
  for (auto& ev : t.pool) {
    const hipError_t e = hipEventCreate(&ev);
    if (e != hipSuccess) {
      for (auto& x : t.pool)
        if (x) (void)hipEventDestroy(x);
      t.pool.clear();
      return hip_fail(e, "hvdx_timeline_begin: hipEventCreate");
    }
  }
  t.entries.clear();
  t.entries.reserve(capacity);
  t.capacity = capacity;
  t.dropped = 0;
  t.per_phase = per_phase != 0;
  t.on = true;
  return HVDX_OK;
}

int hvdx_timeline_end(hvdx_trace_record* out, int capacity, int* nrecords, int* ndropped) {
  if (!nrecords || !ndropped || capacity < 0 || (capacity > 0 && !out))
    return fail(HVDX_ERR_INVALID, "hvdx_timeline_end: bad arguments");
  Timeline& t = timeline();
  std::lock_guard<std::recursive_mutex> g(t.mu);
  if (!t.on) return fail(HVDX_ERR_INVALID, "hvdx_timeline_end: no timeline is recording");
  t.on = false;
  int rc = HVDX_OK;
  const int n = (int)t.entries.size();
  hipError_t e = hipSuccess;
  for (int i = 0; i < n && e == hipSuccess; ++i) e = hipEventSynchronize(t.entries[i].end);
  if (e != hipSuccess) rc = hip_fail(e, "hvdx_timeline_end: hipEventSynchronize");
  int written = 0;
  for (int i = 0; i < n && written < capacity && rc == HVDX_OK; ++i) {
    float t0 = 0.f, dur = 0.f;
    e = hipEventElapsedTime(&t0, t.entries[0].start, t.entries[i].start);
    if (e == hipSuccess) e = hipEventElapsedTime(&dur, t.entries[i].start, t.entries[i].end);
    if (e != hipSuccess) {
      rc = hip_fail(e, "hvdx_timeline_end: hipEventElapsedTime");
      break;
    }
    out[written] = t.entries[i].rec;
    out[written].start_us = 1000.0 * t0;
    out[written].duration_us = 1000.0 * dur;
    ++written;
  }
  *nrecords = written;
  *ndropped = t.dropped + (n - written);
  for (auto& ev : t.pool) (void)hipEventDestroy(ev);
  t.pool.clear();
  t.entries.clear();
  return rc;
}

const char* hvdx_last_error(void) { return g_last_error; }

const char* hvdx_strerror(int status) {
  switch (status) {
    case HVDX_OK: return "success";
    case HVDX_ERR_INVALID: return "invalid argument";
    case HVDX_ERR_ALIAS: return "overlapping buffers";
    case HVDX_ERR_WORKSPACE: return "workspace missing or too small";
    case HVDX_ERR_HIP: return "HIP runtime error";
    case HVDX_ERR_UNSUPPORTED: return "unsupported combination";
    default: return "unknown status";
  }
}

int hvdx_ring_chunk(int64_t count, int nranks, int c, int64_t* start, int64_t* len) {
  if (count < 0 || nranks < 1 || c < 0 || c >= nranks || !start || !len)
    return fail(HVDX_ERR_INVALID, "hvdx_ring_chunk: bad arguments");
  const int64_t q = count / nranks, r = count % nranks;
  *start = (int64_t)c * q + std::min<int64_t>(c, r);
  *len = q + (c < r ? 1 : 0);
  return HVDX_OK;
}

size_t hvdx_ring_workspace_bytes(int nranks, int64_t count, int dtype, int compress) {
  if (compress != HVDX_COMPRESS_FP16 || dtype != HVDX_FLOAT32 || nranks < 2 || count <= 0) return 0;
  return (size_t)nranks * (size_t)wire_stride(count) * 2;
}

int hvdx_fuse_plan(const int64_t* numel, int ntensors, int buf_dtype, int64_t threshold_bytes, int64_t align_bytes,
                   int32_t* bucket_of, int64_t* offset, int64_t* bucket_count, int32_t* bucket_direct,
                   int32_t* nbuckets) {
  const char* what = "hvdx_fuse_plan";
  if (ntensors < 0) return fail(HVDX_ERR_INVALID, "%s: negative tensor count", what);
  if (!nbuckets || (ntensors > 0 && (!numel || !bucket_of || !offset || !bucket_count || !bucket_direct)))
    return fail(HVDX_ERR_INVALID, "%s: NULL array", what);
  const int64_t es = elem_size(buf_dtype);
  if (!es) return fail(HVDX_ERR_INVALID, "%s: unknown dtype %d", what, buf_dtype);
  if (threshold_bytes < 0) return fail(HVDX_ERR_INVALID, "%s: negative threshold", what);
  if (align_bytes < es || (align_bytes & (align_bytes - 1)))
    return fail(HVDX_ERR_INVALID, "%s: alignment %lld is not a power of two >= the element size", what,
                (long long)align_bytes);
  for (int t = 0; t < ntensors; ++t)
    if (numel[t] < 0 || numel[t] > (INT64_MAX / 4) / es)
      return fail(HVDX_ERR_INVALID, "%s: bad element count for tensor %d", what, t);

  // Walk the ready list once.  `open` is the buffer being filled, `used` its length in
  // elements; a tensor joins it when its aligned start plus its bytes stay within the
  // threshold, else the buffer is closed and the tensor starts a new one.  A tensor
  // larger than the threshold closes the open buffer and forms a direct one.
  int nb = 0;
  int open = -1;
  int64_t used = 0;
  for (int t = 0; t < ntensors; ++t) {
    const int64_t bytes = numel[t] * es;
    if (bytes > threshold_bytes) {
      open = -1;
      bucket_of[t] = nb;
      offset[t] = 0;
      bucket_count[nb] = numel[t];
      bucket_direct[nb] = 1;
      ++nb;
      continue;
    }
    int64_t start_bytes = 0;
    if (open >= 0) {
      start_bytes = (used * es + align_bytes - 1) / align_bytes * align_bytes;
      if (start_bytes + bytes > threshold_bytes) open = -1;
    }
    if (open < 0) {
      open = nb++;
      bucket_direct[open] = 0;
      start_bytes = 0;
    }
    bucket_of[t] = open;
    offset[t] = start_bytes / es;
    used = offset[t] + numel[t];
    bucket_count[open] = used;
  }
  *nbuckets = nb;
  return HVDX_OK;
}

int hvdx_fuse_pack(const void* const* srcs, const int64_t* numel, const int64_t* offset, int ntensors, int src_dtype,
                   void* const* bufs, int64_t buf_count, int buf_dtype, int nranks, void* stream) {
  int rc = check_fusion(srcs, numel, offset, ntensors, src_dtype, bufs, buf_count, buf_dtype, nranks,
                        "hvdx_fuse_pack");
  if (rc) return rc;
  if (buf_count == 0) return HVDX_OK;
  TimedLaunch timed(HVDX_KERNEL_PACK, -1, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count,
                    static_cast<hipStream_t>(stream));
  TimedLaunch timed_phase(HVDX_KERNEL_PACK, -1, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count,
                          static_cast<hipStream_t>(stream), -1, true);
  const hipError_t e = hvdx::launch_pack(srcs, numel, offset, ntensors, src_dtype, rank_ptrs(bufs, nranks),
                                         buf_count, buf_dtype, nranks, false, false,
                                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "pack launch");
}

// The copy-in fused with adding step 0, or the copy-out fused with replacing step N-2
// (arguments already checked, nranks >= 3, buf_count > 0).  Inside a whole cycle the
// copy-in leaves out each chunk's sender's copy of its own chunk: the sender's value
// goes straight from its tensor into the receiver's sum, and replacing step 0
// overwrites that copy before anything reads it.
static int run_pack_rs(const void* const* srcs, const int64_t* numel, const int64_t* offset, int ntensors,
                       int src_dtype, void* const* bufs, int64_t buf_count, int buf_dtype, int nranks,
                       bool in_cycle, hipStream_t st) {
  TimedLaunch timed(HVDX_KERNEL_PACK_RS, 0, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count, st);
  TimedLaunch timed_phase(HVDX_KERNEL_PACK_RS, 0, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count, st, -1, true);
  const hipError_t e = hvdx::launch_pack(srcs, numel, offset, ntensors, src_dtype, rank_ptrs(bufs, nranks), buf_count,
                                         buf_dtype, nranks, true, in_cycle, st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "fused copy-in launch");
}

static int run_ag_unpack(const void* const* bufs, int64_t buf_count, int buf_dtype, void* const* dsts,
                         const int64_t* numel, const int64_t* offset, int ntensors, int dst_dtype, int nranks,
                         hipStream_t st) {
  TimedLaunch timed(HVDX_KERNEL_AG_UNPACK, nranks - 2, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count, st);
  TimedLaunch timed_phase(HVDX_KERNEL_AG_UNPACK, nranks - 2, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count, st,
                          -1, true);
  const hipError_t e = hvdx::launch_unpack(rank_ptrs(const_cast<void* const*>(bufs), nranks), buf_count, buf_dtype,
                                           dsts, numel, offset, ntensors, dst_dtype, nranks, true, st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "fused copy-out launch");
}

int hvdx_fuse_pack_rs(const void* const* srcs, const int64_t* numel, const int64_t* offset, int ntensors,
                      int src_dtype, void* const* bufs, int64_t buf_count, int buf_dtype, int nranks, void* stream) {
  int rc = check_fusion(srcs, numel, offset, ntensors, src_dtype, bufs, buf_count, buf_dtype, nranks,
                        "hvdx_fuse_pack_rs");
  if (rc) return rc;
  if (nranks < 3)
    return fail(HVDX_ERR_UNSUPPORTED, "hvdx_fuse_pack_rs: needs 3 or more ranks (adding step 0 is the last one)");
  if (buf_count == 0) return HVDX_OK;
  return run_pack_rs(srcs, numel, offset, ntensors, src_dtype, bufs, buf_count, buf_dtype, nranks, false,
                     static_cast<hipStream_t>(stream));
}

int hvdx_fuse_ag_unpack(const void* const* bufs, int64_t buf_count, int buf_dtype, void* const* dsts,
                        const int64_t* numel, const int64_t* offset, int ntensors, int dst_dtype, int nranks,
                        void* stream) {
  int rc = check_fusion(dsts, numel, offset, ntensors, dst_dtype, bufs, buf_count, buf_dtype, nranks,
                        "hvdx_fuse_ag_unpack");
  if (rc) return rc;
  if (nranks < 3)
    return fail(HVDX_ERR_UNSUPPORTED, "hvdx_fuse_ag_unpack: needs 3 or more ranks (replacing step N-2 is step 0)");
  if (buf_count == 0) return HVDX_OK;
  return run_ag_unpack(bufs, buf_count, buf_dtype, dsts, numel, offset, ntensors, dst_dtype, nranks,
                       static_cast<hipStream_t>(stream));
}

int hvdx_fuse_unpack(const void* const* bufs, int64_t buf_count, int buf_dtype, void* const* dsts,
                     const int64_t* numel, const int64_t* offset, int ntensors, int dst_dtype, int nranks,
                     void* stream) {
  int rc = check_fusion(dsts, numel, offset, ntensors, dst_dtype, bufs, buf_count, buf_dtype, nranks,
                        "hvdx_fuse_unpack");
  if (rc) return rc;
  if (buf_count == 0) return HVDX_OK;
  TimedLaunch timed(HVDX_KERNEL_UNPACK, -1, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count,
                    static_cast<hipStream_t>(stream));
  TimedLaunch timed_phase(HVDX_KERNEL_UNPACK, -1, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count,
                          static_cast<hipStream_t>(stream), -1, true);
  const hipError_t e =
      hvdx::launch_unpack(rank_ptrs(const_cast<void* const*>(bufs), nranks), buf_count, buf_dtype, dsts, numel,
                          offset, ntensors, dst_dtype, nranks, false, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "unpack launch");
}

int hvdx_ring_step(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress, int phase,
                   int step, void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_ring(bufs, nranks, count, dtype, op, compress, workspace, workspace_bytes, "hvdx_ring_step");
  if (rc) return rc;
  if (phase != HVDX_PHASE_REDUCE_SCATTER && phase != HVDX_PHASE_ALLGATHER)
    return fail(HVDX_ERR_INVALID, "hvdx_ring_step: unknown phase %d", phase);
  if (step < 0 || step > nranks - 2)
    return fail(HVDX_ERR_INVALID, "hvdx_ring_step: step %d outside 0..%d", step, nranks - 2);
  if (count == 0) return HVDX_OK;
  return run_step(bufs, nranks, count, dtype, op, compress, phase, step, workspace,
                  static_cast<hipStream_t>(stream));
}

// The N-1 steps of one phase; the one-rank compressed ring rounds in the adding phase.
static int run_phase(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress, int phase,
                     void* workspace, size_t workspace_bytes, void* stream, const char* what) {
  int rc = check_ring(bufs, nranks, count, dtype, op, compress, workspace, workspace_bytes, what);
  if (rc) return rc;
  if (count == 0) return HVDX_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (nranks == 1) {  // no messages; AVERAGE divides by 1; compression still rounds
    if (compress != HVDX_COMPRESS_FP16 || phase != HVDX_PHASE_REDUCE_SCATTER) return HVDX_OK;
    TimedLaunch timed(HVDX_KERNEL_ROUNDTRIP, -1, 1, dtype, compress, count, st);
    TimedLaunch timed_phase(HVDX_KERNEL_ROUNDTRIP, -1, 1, dtype, compress, count, st, -1, true);
    const hipError_t e = hvdx::launch_roundtrip_c16(bufs[0], count, st);
    return e == hipSuccess ? HVDX_OK : hip_fail(e, "fp16 round-trip launch");
  }
  return run_steps(bufs, nranks, count, dtype, op, compress, phase, 0, nranks - 1, workspace, st);
}

int hvdx_ring_reduce_scatter(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress,
                             void* workspace, size_t workspace_bytes, void* stream) {
  return run_phase(bufs, nranks, count, dtype, op, compress, HVDX_PHASE_REDUCE_SCATTER, workspace,
                   workspace_bytes, stream, "hvdx_ring_reduce_scatter");
}

int hvdx_ring_allgather(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress,
                        void* workspace, size_t workspace_bytes, void* stream) {
  return run_phase(bufs, nranks, count, dtype, op, compress, HVDX_PHASE_ALLGATHER, workspace, workspace_bytes,
                   stream, "hvdx_ring_allgather");
}

int hvdx_ring_allreduce(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress,
                        void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_ring(bufs, nranks, count, dtype, op, compress, workspace, workspace_bytes, "hvdx_ring_allreduce");
  if (rc) return rc;
  if (count == 0) return HVDX_OK;
  if (nranks == 1)
    return run_phase(bufs, nranks, count, dtype, op, compress, HVDX_PHASE_REDUCE_SCATTER, workspace,
                     workspace_bytes, stream, "hvdx_ring_allreduce");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int last = nranks - 2;
  rc = run_steps(bufs, nranks, count, dtype, op, compress, HVDX_PHASE_REDUCE_SCATTER, 0, last, workspace, st);
  if (rc) return rc;
  {
    TimedLaunch timed_phase(HVDX_KERNEL_RS_AG, last, nranks, dtype, compress, count, st, -1, true);
    rc = run_step(bufs, nranks, count, dtype, op, compress, HVDX_PHASE_REDUCE_SCATTER, last, workspace, st, true);
    if (rc) return rc;
  }
  return run_steps(bufs, nranks, count, dtype, op, compress, HVDX_PHASE_ALLGATHER, 1, nranks - 1, workspace, st);
}

int hvdx_fuse_allreduce(void* const* tensors, const int64_t* numel, const int64_t* offset, int ntensors,
                        int tensor_dtype, void* const* bufs, int64_t buf_count, int buf_dtype, int nranks, int op,
                        void* stream) {
  int rc = check_fusion(tensors, numel, offset, ntensors, tensor_dtype, bufs, buf_count, buf_dtype, nranks,
                        "hvdx_fuse_allreduce");
  if (rc) return rc;
  if (op != HVDX_SUM && op != HVDX_AVERAGE) return fail(HVDX_ERR_INVALID, "hvdx_fuse_allreduce: unknown op %d", op);
  if (buf_count == 0) return HVDX_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const void* const* srcs = const_cast<const void* const*>(tensors);
  if (nranks < 3) {  // no adding step before the last, no replacing step after the first
    rc = hvdx_fuse_pack(srcs, numel, offset, ntensors, tensor_dtype, bufs, buf_count, buf_dtype, nranks, stream);
    if (!rc && nranks == 2) {
      TimedLaunch timed_phase(HVDX_KERNEL_RS_AG, 0, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count, st, -1, true);
      rc = run_step(bufs, nranks, buf_count, buf_dtype, op, HVDX_COMPRESS_NONE, HVDX_PHASE_REDUCE_SCATTER, 0,
                    nullptr, st, true);
    }
    if (rc) return rc;
    return hvdx_fuse_unpack(bufs, buf_count, buf_dtype, tensors, numel, offset, ntensors, tensor_dtype, nranks,
                            stream);
  }
  const int last = nranks - 2;
  rc = run_pack_rs(srcs, numel, offset, ntensors, tensor_dtype, bufs, buf_count, buf_dtype, nranks, true, st);
  if (!rc)
    rc = run_steps(bufs, nranks, buf_count, buf_dtype, op, HVDX_COMPRESS_NONE, HVDX_PHASE_REDUCE_SCATTER, 1, last,
                   nullptr, st);
  if (rc) return rc;
  {
    TimedLaunch timed_phase(HVDX_KERNEL_RS_AG, last, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count, st, -1, true);
    rc = run_step(bufs, nranks, buf_count, buf_dtype, op, HVDX_COMPRESS_NONE, HVDX_PHASE_REDUCE_SCATTER, last,
                  nullptr, st, true);
    if (rc) return rc;
  }
  rc = run_steps(bufs, nranks, buf_count, buf_dtype, op, HVDX_COMPRESS_NONE, HVDX_PHASE_ALLGATHER, 1, last, nullptr,
                 st);
  if (rc) return rc;
  return run_ag_unpack(bufs, buf_count, buf_dtype, tensors, numel, offset, ntensors, tensor_dtype, nranks, st);
}

// One step of two rings in one launch (arguments already checked, nranks >= 3).
static int run_pair_step(const hvdx_bucket* b0, const hvdx_bucket* b1, int dtype, int op, int kind, int step,
                         int nranks, hipStream_t st) {
  hvdx::RingPair m{};
  m.bufs[0] = rank_ptrs(b0->bufs, nranks);
  m.bufs[1] = rank_ptrs(b1->bufs, nranks);
  m.a[0] = ring_args(nranks, b0->buf_count, step);
  m.a[1] = ring_args(nranks, b1->buf_count, step);
  TimedLaunch timed(kind, step, nranks, dtype, HVDX_COMPRESS_NONE, b0->buf_count + b1->buf_count, st);
  hipError_t e;
  if (kind == HVDX_KERNEL_RS_AG) e = hvdx::launch_rs_ag_step_pair(m, dtype, div_mode(op, nranks), st);
  else if (kind == HVDX_KERNEL_REDUCE_SCATTER) e = hvdx::launch_rs_step_pair(m, dtype, hvdx::DIV_NONE, st);
  else e = hvdx::launch_ag_step_pair(m, dtype, st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "two-ring step launch");
}

// Steps [s0, s1) of one phase for two rings, as one timeline phase record.
static int run_pair_steps(const hvdx_bucket* b0, const hvdx_bucket* b1, int dtype, int op, int kind, int s0, int s1,
                          int nranks, hipStream_t st) {
  if (s1 <= s0) return HVDX_OK;
  TimedLaunch timed(kind, s0, nranks, dtype, HVDX_COMPRESS_NONE, b0->buf_count + b1->buf_count, st, -1, true,
                    s1 - s0);
  for (int s = s0; s < s1; ++s) {
    const int rc = run_pair_step(b0, b1, dtype, op, kind, s, nranks, st);
    if (rc) return rc;
  }
  return HVDX_OK;
}

int hvdx_fuse_allreduce_pair(const hvdx_bucket* b0, const hvdx_bucket* b1, int tensor_dtype, int buf_dtype,
                             int nranks, int op, void* stream) {
  static const char* what = "hvdx_fuse_allreduce_pair";
  if (!b0 || !b1) return fail(HVDX_ERR_INVALID, "%s: a bucket descriptor is NULL", what);
  for (const hvdx_bucket* b : {b0, b1}) {
    const int rc = check_fusion(b->tensors, b->numel, b->offset, b->ntensors, tensor_dtype, b->bufs, b->buf_count,
                                buf_dtype, nranks, what);
    if (rc) return rc;
  }
  if (op != HVDX_SUM && op != HVDX_AVERAGE) return fail(HVDX_ERR_INVALID, "%s: unknown op %d", what, op);
  if (nranks < 3) return fail(HVDX_ERR_UNSUPPORTED, "%s: needs 3 or more ranks", what);
  const int es = elem_size(buf_dtype);
  if (b0->buf_count > 0 && b1->buf_count > 0) {  // both rings run at once: all 2N buffers disjoint
    std::vector<std::pair<uintptr_t, uintptr_t>> rg;
    for (const hvdx_bucket* b : {b0, b1})
      for (int r = 0; r < nranks; ++r) {
        const uintptr_t x = reinterpret_cast<uintptr_t>(b->bufs[r]);
        rg.emplace_back(x, x + (uintptr_t)b->buf_count * es);
      }
    if (overlapping(rg)) return fail(HVDX_ERR_ALIAS, "%s: fusion buffers of the two buckets overlap", what);
  }
  if (b0->buf_count == 0 || b1->buf_count == 0) {
    const hvdx_bucket* b = b0->buf_count ? b0 : b1;
    return hvdx_fuse_allreduce(b->tensors, b->numel, b->offset, b->ntensors, tensor_dtype, b->bufs, b->buf_count,
                               buf_dtype, nranks, op, stream);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int last = nranks - 2;
  const int64_t both = b0->buf_count + b1->buf_count;
  hvdx::CopyPair cp{};
  const hvdx_bucket* bk[2] = {b0, b1};
  for (int i = 0; i < 2; ++i) {
    cp.t[i] = bk[i]->tensors;
    cp.numel[i] = bk[i]->numel;
    cp.offset[i] = bk[i]->offset;
    cp.ntensors[i] = bk[i]->ntensors;
    cp.bufs[i] = rank_ptrs(bk[i]->bufs, nranks);
    cp.count[i] = bk[i]->buf_count;
    cp.q[i] = bk[i]->buf_count / nranks;
    cp.rem[i] = bk[i]->buf_count % nranks;
  }
  int rc = HVDX_OK;
  {
    TimedLaunch timed(HVDX_KERNEL_PACK_RS, 0, nranks, buf_dtype, HVDX_COMPRESS_NONE, both, st);
    TimedLaunch timed_phase(HVDX_KERNEL_PACK_RS, 0, nranks, buf_dtype, HVDX_COMPRESS_NONE, both, st, -1, true);
    const hipError_t e = hvdx::launch_pack_pair(cp, tensor_dtype, buf_dtype, nranks, st);
    if (e != hipSuccess) return hip_fail(e, "two-buffer copy-in launch");
  }
  rc = run_pair_steps(b0, b1, buf_dtype, op, HVDX_KERNEL_REDUCE_SCATTER, 1, last, nranks, st);
  if (rc) return rc;
  {
    TimedLaunch timed_phase(HVDX_KERNEL_RS_AG, last, nranks, buf_dtype, HVDX_COMPRESS_NONE,
                            b0->buf_count + b1->buf_count, st, -1, true);
    rc = run_pair_step(b0, b1, buf_dtype, op, HVDX_KERNEL_RS_AG, last, nranks, st);
    if (rc) return rc;
  }
  rc = run_pair_steps(b0, b1, buf_dtype, op, HVDX_KERNEL_ALLGATHER, 1, last, nranks, st);
  if (rc) return rc;
  TimedLaunch timed(HVDX_KERNEL_AG_UNPACK, last, nranks, buf_dtype, HVDX_COMPRESS_NONE, both, st);
  TimedLaunch timed_phase(HVDX_KERNEL_AG_UNPACK, last, nranks, buf_dtype, HVDX_COMPRESS_NONE, both, st, -1, true);
  const hipError_t e = hvdx::launch_unpack_pair(cp, buf_dtype, tensor_dtype, nranks, st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "two-buffer copy-out launch");
}

int64_t hvdx_fuse_tile_elems(int tensor_dtype, int buf_dtype) {
  if (!elem_size(tensor_dtype) || !elem_size(buf_dtype) || (tensor_dtype == HVDX_FLOAT16 && buf_dtype == HVDX_FLOAT32))
    return 0;
  return (int64_t)hvdx::kTileLanes * hvdx::tile_vectors(tensor_dtype, buf_dtype) *
         hvdx::tile_vec_elems(tensor_dtype, buf_dtype);
}

int64_t hvdx_fuse_copy_tiles(const int64_t* numel, const int64_t* offset, int ntensors, int64_t buf_count,
                             int tensor_dtype, int buf_dtype, int nranks, int direction, hvdx_copy_tile* tiles,
                             int64_t capacity) {
  static const char* what = "hvdx_fuse_copy_tiles";
  if (ntensors < 0 || (ntensors > 0 && (!numel || !offset)))
    return fail(HVDX_ERR_INVALID, "%s: bad tensor table", what);
  if (!elem_size(tensor_dtype) || !elem_size(buf_dtype)) return fail(HVDX_ERR_INVALID, "%s: unknown dtype", what);
  if (tensor_dtype == HVDX_FLOAT16 && buf_dtype == HVDX_FLOAT32)
    return fail(HVDX_ERR_UNSUPPORTED, "%s: float16 tensors with a float32 buffer", what);
  if (nranks < 1 || nranks > HVDX_MAX_RANKS)
    return fail(HVDX_ERR_INVALID, "%s: nranks=%d outside 1..%d", what, nranks, HVDX_MAX_RANKS);
  if (buf_count < 0 || buf_count > (INT64_MAX >> 4)) return fail(HVDX_ERR_INVALID, "%s: bad buffer length", what);
  if (direction != HVDX_COPY_IN && direction != HVDX_COPY_OUT)
    return fail(HVDX_ERR_INVALID, "%s: unknown direction %d", what, direction);
  if (capacity < 0 || (capacity > 0 && !tiles)) return fail(HVDX_ERR_INVALID, "%s: bad capacity", what);
  int64_t prev_end = 0;
  for (int t = 0; t < ntensors; ++t) {  // tensors in order, disjoint, inside the buffer
    if (numel[t] < 0 || offset[t] < prev_end || offset[t] > buf_count || numel[t] > buf_count - offset[t])
      return fail(HVDX_ERR_INVALID, "%s: tensor %d does not fit the buffer after the previous one", what, t);
    if (numel[t] > 0) prev_end = offset[t] + numel[t];
  }
  const int64_t vec = hvdx::tile_vec_elems(tensor_dtype, buf_dtype);
  const int64_t tile = hvdx_fuse_tile_elems(tensor_dtype, buf_dtype);
  const int64_t q = buf_count / nranks, rem = buf_count % nranks, big = rem * (q + 1);
  auto chunk_of = [&](int64_t p) { return p < big ? p / (q + 1) : rem + (p - big) / q; };
  auto chunk_end = [&](int64_t c) { return (c + 1) * q + std::min<int64_t>(c + 1, rem); };
  int64_t n = 0;
  // Cut [a, b) (tensor t, or padding for t < 0) at chunk ends and at the tile grid that starts
  // at `base`; a piece that starts off the vector grid ends at the next vector boundary.
  auto cut = [&](int64_t a, int64_t b, int t, int64_t base) {
    for (int64_t p = a; p < b;) {
      const int64_t c = chunk_of(p);
      int64_t stop = std::min(b, chunk_end(c));
      stop = std::min(stop, base + ((p - base) / tile + 1) * tile);
      if ((p - base) % vec) stop = std::min(stop, base + ((p - base) / vec + 1) * vec);
      if (tiles && n < capacity) {
        hvdx_copy_tile& x = tiles[n];
        x.pos = p;
        x.li = t >= 0 ? p - offset[t] : 0;
        x.tensor = t;
        x.len = (int32_t)(stop - p);
        x.chunk = (int32_t)c;
        x.reserved = 0;
      }
      ++n;
      p = stop;
    }
  };
  if (direction == HVDX_COPY_IN) {  // every buffer position, on the buffer's tile grid
    int64_t at = 0;
    for (int t = 0; t < ntensors; ++t) {
      if (numel[t] == 0) continue;
      cut(at, offset[t], -1, 0);
      cut(offset[t], offset[t] + numel[t], t, 0);
      at = offset[t] + numel[t];
    }
    cut(at, buf_count, -1, 0);
  } else {  // every tensor element, on each tensor's own tile grid
    for (int t = 0; t < ntensors; ++t)
      if (numel[t] > 0) cut(offset[t], offset[t] + numel[t], t, offset[t]);
  }
  if (tiles && n > capacity)
    return fail(HVDX_ERR_WORKSPACE, "%s: %lld tiles, room for %lld", what, (long long)n, (long long)capacity);
  return n;
}

static_assert(hvdx::kRingBuckets == HVDX_TILED_MAX_BUCKETS, "one launch descriptor slot per bucket");

int hvdx_fuse_allreduce_tiled(const hvdx_tiled_bucket* buckets, int nbuckets, int tensor_dtype, int buf_dtype,
                              int nranks, int op, int flags, void* stream) {
  static const char* what = "hvdx_fuse_allreduce_tiled";
  if (!buckets || nbuckets < 1 || nbuckets > HVDX_TILED_MAX_BUCKETS)
    return fail(HVDX_ERR_INVALID, "%s: need 1 to %d buckets", what, HVDX_TILED_MAX_BUCKETS);
  if (flags & ~(HVDX_TILED_REPLACE_IN_TENSORS | HVDX_TILED_ADD_FROM_TENSORS))
    return fail(HVDX_ERR_INVALID, "%s: unknown flags 0x%x", what, flags);
  const bool replace_t = flags & HVDX_TILED_REPLACE_IN_TENSORS;
  const bool add_t = flags & HVDX_TILED_ADD_FROM_TENSORS;
  for (int i = 0; i < nbuckets; ++i) {
    const hvdx_tiled_bucket* t = &buckets[i];
    const int rc = check_fusion(t->b.tensors, t->b.numel, t->b.offset, t->b.ntensors, tensor_dtype, t->b.bufs,
                                t->b.buf_count, buf_dtype, nranks, what);
    if (rc) return rc;
    if (t->n_in < 0 || t->n_out < 0 || (t->n_in > 0 && !t->in_tiles) || (t->n_out > 0 && !t->out_tiles) ||
        (t->b.buf_count > 0 && t->n_in == 0))
      return fail(HVDX_ERR_INVALID, "%s: a tile table is missing", what);
  }
  if (op != HVDX_SUM && op != HVDX_AVERAGE) return fail(HVDX_ERR_INVALID, "%s: unknown op %d", what, op);
  if (nranks < 3) return fail(HVDX_ERR_UNSUPPORTED, "%s: needs 3 or more ranks", what);
  if (replace_t && tensor_dtype == HVDX_FLOAT16 && buf_dtype == HVDX_FLOAT32)
    return fail(HVDX_ERR_UNSUPPORTED, "%s: binary16 tensors with binary32 buffers", what);
  if (add_t && !replace_t)
    return fail(HVDX_ERR_UNSUPPORTED, "%s: adding from the tensors needs replacing in the tensors", what);
  // the buckets with something to reduce
  const hvdx_tiled_bucket* run[HVDX_TILED_MAX_BUCKETS];
  int nrun = 0;
  for (int i = 0; i < nbuckets; ++i)
    if (buckets[i].b.buf_count > 0) run[nrun++] = &buckets[i];
  if (nrun > 2 && !add_t)
    return fail(HVDX_ERR_UNSUPPORTED, "%s: more than two buckets need both tensor flags", what);
  if (replace_t && (int64_t)nrun * nranks > hvdx::kRingBufPtrs)
    return fail(HVDX_ERR_UNSUPPORTED, "%s: %d buckets of %d ranks: at most %d buffers per launch", what, nrun, nranks,
                hvdx::kRingBufPtrs);
  const int es = elem_size(buf_dtype);
  if (nrun > 1) {  // they run at once: all their buffers disjoint
    std::vector<std::pair<uintptr_t, uintptr_t>> rg;
    for (int i = 0; i < nrun; ++i)
      for (int r = 0; r < nranks; ++r) {
        const uintptr_t x = reinterpret_cast<uintptr_t>(run[i]->b.bufs[r]);
        rg.emplace_back(x, x + (uintptr_t)run[i]->b.buf_count * es);
      }
    if (overlapping(rg)) return fail(HVDX_ERR_ALIAS, "%s: fusion buffers of two buckets overlap", what);
  }
  if (nrun == 0) return HVDX_OK;
  int64_t n_in = 0, n_out = 0, all = 0;
  for (int i = 0; i < nrun; ++i) {
    n_in += run[i]->n_in;
    n_out += run[i]->n_out;
    all += run[i]->b.buf_count;
  }
  if (n_in > 0x7fffffff || n_out > 0x7fffffff) return fail(HVDX_ERR_UNSUPPORTED, "%s: too many tiles", what);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int last = nranks - 2;
  // the ring on the tensors: one descriptor for all buckets, its tile tables set per step kind
  hvdx::TiledRing ring{};
  ring.nbuckets = nrun;
  ring.nranks = nranks;
  for (int i = 0; i < nrun; ++i) {
    ring.t[i] = run[i]->b.tensors;
    ring.ntensors[i] = run[i]->b.ntensors;
    for (int r = 0; r < nranks && replace_t; ++r) ring.bufs[i * nranks + r] = run[i]->b.bufs[r];
  }
  auto use_tiles = [&](bool out) {
    int64_t at = 0;
    for (int i = 0; i < nrun; ++i) {
      ring.tiles[i] = out ? run[i]->out_tiles : run[i]->in_tiles;
      at += out ? run[i]->n_out : run[i]->n_in;
      ring.end[i] = at;
    }
  };
  // the copies of one or two buckets (the paper's buffers)
  hvdx::TiledCopy k{};
  for (int i = 0; i < nrun && i < 2; ++i) {
    k.m.t[i] = run[i]->b.tensors;
    k.m.numel[i] = run[i]->b.numel;
    k.m.offset[i] = run[i]->b.offset;
    k.m.ntensors[i] = run[i]->b.ntensors;
    k.m.bufs[i] = rank_ptrs(run[i]->b.bufs, nranks);
    k.m.count[i] = run[i]->b.buf_count;
  }
  k.tiles[0] = run[0]->in_tiles;
  k.tiles[1] = nrun > 1 ? run[1]->in_tiles : nullptr;
  k.x0 = run[0]->n_in;
  int rc;
  if (add_t) {  // adding steps 0 .. N-3 with every rank's own values read from its tensors
    use_tiles(false);
    TimedLaunch timed_phase(HVDX_KERNEL_REDUCE_SCATTER, 0, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st, -1, true,
                            last);
    for (int s = 0; s < last; ++s) {
      TimedLaunch timed(HVDX_KERNEL_REDUCE_SCATTER, s, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st);
      const hipError_t e = hvdx::launch_add_tiles(ring, tensor_dtype, buf_dtype, s, st);
      if (e != hipSuccess) return hip_fail(e, "adding step from the tensors");
    }
  } else {
    {
      TimedLaunch timed(HVDX_KERNEL_PACK_RS, 0, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st);
      TimedLaunch timed_phase(HVDX_KERNEL_PACK_RS, 0, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st, -1, true);
      const hipError_t e = hvdx::launch_pack_tiles(k, tensor_dtype, buf_dtype, nranks, n_in, st);
      if (e != hipSuccess) return hip_fail(e, "tiled copy-in launch");
    }
    if (replace_t) {
      if (nrun == 2) rc = run_pair_steps(&run[0]->b, &run[1]->b, buf_dtype, op, HVDX_KERNEL_REDUCE_SCATTER, 1, last,
                                         nranks, st);
      else rc = run_steps(run[0]->b.bufs, nranks, run[0]->b.buf_count, buf_dtype, op, HVDX_COMPRESS_NONE,
                          HVDX_PHASE_REDUCE_SCATTER, 1, last, nullptr, st);
      if (rc) return rc;
    }
  }
  if (replace_t) {
    if (n_out == 0) return HVDX_OK;  // every tensor empty: nothing to deliver
    use_tiles(true);
    {
      TimedLaunch timed(HVDX_KERNEL_RS_AG, last, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st);
      TimedLaunch timed_phase(HVDX_KERNEL_RS_AG, last, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st, -1, true);
      const hipError_t e = hvdx::launch_rs_ag_tiles(ring, ring_args(nranks, run[0]->b.buf_count, last), tensor_dtype,
                                                    buf_dtype, div_mode(op, nranks), add_t, st);
      if (e != hipSuccess) return hip_fail(e, "replacing step 0 into the tensors");
    }
    TimedLaunch timed_phase(HVDX_KERNEL_ALLGATHER, 1, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st, -1, true,
                            last);
    for (int s = 1; s <= last; ++s) {
      TimedLaunch timed(HVDX_KERNEL_ALLGATHER, s, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st);
      const hipError_t e = hvdx::launch_ag_tiles(ring, tensor_dtype, buf_dtype, s, st);
      if (e != hipSuccess) return hip_fail(e, "replacing step into the tensors");
    }
    return HVDX_OK;
  }
  if (nrun == 2) {
    rc = run_pair_steps(&run[0]->b, &run[1]->b, buf_dtype, op, HVDX_KERNEL_REDUCE_SCATTER, 1, last, nranks, st);
    if (rc) return rc;
    {
      TimedLaunch timed_phase(HVDX_KERNEL_RS_AG, last, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st, -1, true);
      rc = run_pair_step(&run[0]->b, &run[1]->b, buf_dtype, op, HVDX_KERNEL_RS_AG, last, nranks, st);
      if (rc) return rc;
    }
    rc = run_pair_steps(&run[0]->b, &run[1]->b, buf_dtype, op, HVDX_KERNEL_ALLGATHER, 1, last, nranks, st);
  } else {
    void* const* bufs = run[0]->b.bufs;
    const int64_t count = run[0]->b.buf_count;
    rc = run_steps(bufs, nranks, count, buf_dtype, op, HVDX_COMPRESS_NONE, HVDX_PHASE_REDUCE_SCATTER, 1, last, nullptr,
                   st);
    if (rc) return rc;
    {
      TimedLaunch timed_phase(HVDX_KERNEL_RS_AG, last, nranks, buf_dtype, HVDX_COMPRESS_NONE, count, st, -1, true);
      rc = run_step(bufs, nranks, count, buf_dtype, op, HVDX_COMPRESS_NONE, HVDX_PHASE_REDUCE_SCATTER, last, nullptr,
                    st, true);
      if (rc) return rc;
    }
    rc = run_steps(bufs, nranks, count, buf_dtype, op, HVDX_COMPRESS_NONE, HVDX_PHASE_ALLGATHER, 1, last, nullptr, st);
  }
  if (rc) return rc;
  if (n_out == 0) return HVDX_OK;  // every tensor empty: nothing to copy out
  TimedLaunch timed(HVDX_KERNEL_AG_UNPACK, last, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st);
  TimedLaunch timed_phase(HVDX_KERNEL_AG_UNPACK, last, nranks, buf_dtype, HVDX_COMPRESS_NONE, all, st, -1, true);
  k.tiles[0] = run[0]->out_tiles;
  k.tiles[1] = nrun > 1 ? run[1]->out_tiles : nullptr;
  k.x0 = run[0]->n_out;
  const hipError_t e = hvdx::launch_unpack_tiles(k, buf_dtype, tensor_dtype, nranks, n_out, st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "tiled copy-out launch");
}

int hvdx_fuse_allreduce_small(void* const* tensors, const int64_t* numel, const int64_t* offset, int ntensors,
                              int tensor_dtype, void* const* bufs, int64_t buf_count, int buf_dtype, int nranks,
                              int op, void* stream) {
  int rc = check_fusion(tensors, numel, offset, ntensors, tensor_dtype, bufs, buf_count, buf_dtype, nranks,
                        "hvdx_fuse_allreduce_small");
  if (rc) return rc;
  if (op != HVDX_SUM && op != HVDX_AVERAGE)
    return fail(HVDX_ERR_INVALID, "hvdx_fuse_allreduce_small: unknown op %d", op);
  if (buf_count == 0) return HVDX_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  TimedLaunch timed(HVDX_KERNEL_CYCLE_SMALL, -1, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count, st);
  TimedLaunch timed_phase(HVDX_KERNEL_CYCLE_SMALL, -1, nranks, buf_dtype, HVDX_COMPRESS_NONE, buf_count, st, -1,
                          true);
  const hipError_t e =
      hvdx::launch_small_cycle(const_cast<const void* const*>(tensors), numel, offset, ntensors, tensor_dtype,
                               rank_ptrs(bufs, nranks), ring_args(nranks, buf_count, 0), buf_count, buf_dtype,
                               div_mode(op, nranks), st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "small cycle launch");
}

int hvdx_ring_allreduce_small(void* const* bufs, int nranks, int64_t count, int dtype, int op, void* stream) {
  int rc = check_ring(bufs, nranks, count, dtype, op, HVDX_COMPRESS_NONE, nullptr, 0, "hvdx_ring_allreduce_small");
  if (rc) return rc;
  if (count == 0 || nranks == 1) return HVDX_OK;  // no messages; AVERAGE divides by 1
  hipStream_t st = static_cast<hipStream_t>(stream);
  TimedLaunch timed(HVDX_KERNEL_RING_SMALL, -1, nranks, dtype, HVDX_COMPRESS_NONE, count, st);
  TimedLaunch timed_phase(HVDX_KERNEL_RING_SMALL, -1, nranks, dtype, HVDX_COMPRESS_NONE, count, st, -1, true);
  const hipError_t e = hvdx::launch_chain(rank_ptrs(bufs, nranks), ring_args(nranks, count, 0), count, dtype,
                                          div_mode(op, nranks), vectors_ok(bufs, nranks, nullptr), st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "small ring launch");
}

int hvdx_fold_allreduce(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress,
                        void* stream) {
  int rc = check_ring(bufs, nranks, count, dtype, op, HVDX_COMPRESS_NONE, nullptr, 0, "hvdx_fold_allreduce");
  if (rc) return rc;
  if (compress != HVDX_COMPRESS_NONE && compress != HVDX_COMPRESS_FP16)
    return fail(HVDX_ERR_INVALID, "hvdx_fold_allreduce: unknown compression %d", compress);
  if (compress == HVDX_COMPRESS_FP16 && dtype != HVDX_FLOAT32)
    return fail(HVDX_ERR_INVALID, "hvdx_fold_allreduce: fp16 compression needs float32 buffers");
  if (count == 0) return HVDX_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const hvdx::RingArgs a = ring_args(nranks, count, 0);
  TimedLaunch timed(HVDX_KERNEL_FOLD, -1, nranks, dtype, compress, count, st);
  TimedLaunch timed_phase(HVDX_KERNEL_FOLD, -1, nranks, dtype, compress, count, st, -1, true);
  const hipError_t e = hvdx::launch_fold(rank_ptrs(bufs, nranks), a, count, dtype, compress, div_mode(op, nranks),
                                         vectors_ok(bufs, nranks, nullptr), st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "fold launch");
}

size_t hvdx_ring_noalloc_max_bytes(void) { return kScratchBytes; }

int hvdx_ring_allreduce_noalloc(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress,
                                void* stream) {
  static const char* what = "hvdx_ring_allreduce_noalloc";
  // every argument check first (no HIP call before them), the workspace's size included
  int rc = check_ring(bufs, nranks, count, dtype, op, HVDX_COMPRESS_NONE, nullptr, 0, what);
  if (rc) return rc;
  if (compress != HVDX_COMPRESS_NONE && compress != HVDX_COMPRESS_FP16)
    return fail(HVDX_ERR_INVALID, "%s: unknown compression %d", what, compress);
  if (compress == HVDX_COMPRESS_FP16 && dtype != HVDX_FLOAT32)
    return fail(HVDX_ERR_INVALID, "%s: fp16 compression needs float32 buffers", what);
  const size_t need = hvdx_ring_workspace_bytes(nranks, count, dtype, compress);
  if (need > kScratchBytes)
    return fail(HVDX_ERR_WORKSPACE, "%s: %d ranks of %lld elements need %zu bytes of wire workspace; the static one "
                "holds %zu (use hvdx_ring_allreduce with a workspace)", what, nranks, (long long)count, need,
                kScratchBytes);
  if (need == 0)  // nothing compressed: no workspace at all
    return hvdx_ring_allreduce(bufs, nranks, count, dtype, op, compress, nullptr, 0, stream);
  void* ws = nullptr;
  rc = scratch_for(static_cast<hipStream_t>(stream), &ws, what);
  if (rc) return rc;
  return hvdx_ring_allreduce(bufs, nranks, count, dtype, op, compress, ws, kScratchBytes, stream);
}

static int check_bcast(void* const* bufs, int nranks, int64_t nbytes, int root, const char* what) {
  int rc = check_rank_buffers(bufs, nranks, nbytes, 1, what);
  if (rc) return rc;
  if (root < 0 || root >= nranks) return fail(HVDX_ERR_INVALID, "%s: root %d outside 0..%d", what, root, nranks - 1);
  return HVDX_OK;
}

static int bcast_step(void* const* bufs, int nranks, int64_t nbytes, int root, int step, hipStream_t st) {
  hvdx::BcastArgs a{};
  a.n = nranks;
  a.root = root;
  a.step = step;
  a.nbytes = nbytes;
  const int64_t units = (nbytes + 15) / 16;
  a.q = units / nranks;
  a.rem = units % nranks;
  bool vok = true;
  for (int r = 0; r < nranks; ++r) vok = vok && aligned16(bufs[r]);
  TimedLaunch timed(HVDX_KERNEL_BROADCAST, step, nranks, -1, HVDX_COMPRESS_NONE, nbytes, st, root);
  TimedLaunch timed_phase(HVDX_KERNEL_BROADCAST, step, nranks, -1, HVDX_COMPRESS_NONE, nbytes, st, root, true);
  const hipError_t e = hvdx::launch_bcast_step(rank_ptrs(bufs, nranks), a, vok, st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "broadcast step launch");
}

int hvdx_broadcast_step(void* const* bufs, int nranks, int64_t nbytes, int root, int step, void* stream) {
  int rc = check_bcast(bufs, nranks, nbytes, root, "hvdx_broadcast_step");
  if (rc) return rc;
  if (step < 0 || step > 2 * nranks - 3)
    return fail(HVDX_ERR_INVALID, "hvdx_broadcast_step: step %d outside 0..%d", step, 2 * nranks - 3);
  if (nbytes == 0) return HVDX_OK;
  return bcast_step(bufs, nranks, nbytes, root, step, static_cast<hipStream_t>(stream));
}

int hvdx_broadcast_layout(const int64_t* nbytes, int ntensors, int64_t* voffset, int64_t* total_bytes) {
  if (ntensors < 0 || !total_bytes || (ntensors > 0 && (!nbytes || !voffset)))
    return fail(HVDX_ERR_INVALID, "hvdx_broadcast_layout: bad arguments");
  int64_t end = 0;
  for (int t = 0; t < ntensors; ++t) {
    if (nbytes[t] < 0 || nbytes[t] > (INT64_MAX >> 2) - end)
      return fail(HVDX_ERR_INVALID, "hvdx_broadcast_layout: bad byte count for tensor %d", t);
    voffset[t] = (end + 15) / 16 * 16;
    end = voffset[t] + nbytes[t];
  }
  *total_bytes = end;
  return HVDX_OK;
}

static int check_bcast_tensors(const void* const* ptrs, const int64_t* nbytes, const int64_t* voffset, int ntensors,
                               int64_t total_bytes, int nranks, int root, const char* what) {
  if (ntensors < 0) return fail(HVDX_ERR_INVALID, "%s: negative tensor count", what);
  if (ntensors > 0 && (!ptrs || !nbytes || !voffset))
    return fail(HVDX_ERR_INVALID, "%s: a descriptor array is NULL", what);
  if (nranks < 1 || nranks > HVDX_MAX_RANKS)
    return fail(HVDX_ERR_INVALID, "%s: nranks=%d outside 1..%d", what, nranks, HVDX_MAX_RANKS);
  if (root < 0 || root >= nranks) return fail(HVDX_ERR_INVALID, "%s: root %d outside 0..%d", what, root, nranks - 1);
  if (total_bytes < 0 || total_bytes > (INT64_MAX >> 2))
    return fail(HVDX_ERR_INVALID, "%s: bad virtual length %lld", what, (long long)total_bytes);
  return HVDX_OK;
}

static int bcast_tensors_step(const void* const* ptrs, const int64_t* nbytes, const int64_t* voffset, int ntensors,
                              int64_t total_bytes, int nranks, int root, int step, hipStream_t st) {
  hvdx::BcastTensorsArgs a{};
  a.ptrs = ptrs;
  a.nbytes = nbytes;
  a.voff = voffset;
  a.ntensors = ntensors;
  a.n = nranks;
  a.root = root;
  a.step = step;
  a.total = total_bytes;
  const int64_t units = (total_bytes + 15) / 16;
  a.q = units / nranks;
  a.rem = units % nranks;
  TimedLaunch timed(HVDX_KERNEL_BROADCAST, step, nranks, -1, HVDX_COMPRESS_NONE, total_bytes, st, root);
  TimedLaunch timed_phase(HVDX_KERNEL_BROADCAST, step, nranks, -1, HVDX_COMPRESS_NONE, total_bytes, st, root, true);
  const hipError_t e = hvdx::launch_bcast_tensors_step(a, st);
  return e == hipSuccess ? HVDX_OK : hip_fail(e, "tensor broadcast step launch");
}

int hvdx_broadcast_tensors_step(const void* const* ptrs, const int64_t* nbytes, const int64_t* voffset, int ntensors,
                                int64_t total_bytes, int nranks, int root, int step, void* stream) {
  int rc = check_bcast_tensors(ptrs, nbytes, voffset, ntensors, total_bytes, nranks, root,
                               "hvdx_broadcast_tensors_step");
  if (rc) return rc;
  if (step < 0 || step > 2 * nranks - 3)
    return fail(HVDX_ERR_INVALID, "hvdx_broadcast_tensors_step: step %d outside 0..%d", step, 2 * nranks - 3);
  if (total_bytes == 0 || ntensors == 0) return HVDX_OK;
  return bcast_tensors_step(ptrs, nbytes, voffset, ntensors, total_bytes, nranks, root, step,
                            static_cast<hipStream_t>(stream));
}

int hvdx_broadcast_tensors(const void* const* ptrs, const int64_t* nbytes, const int64_t* voffset, int ntensors,
                           int64_t total_bytes, int nranks, int root, void* stream) {
  int rc = check_bcast_tensors(ptrs, nbytes, voffset, ntensors, total_bytes, nranks, root, "hvdx_broadcast_tensors");
  if (rc) return rc;
  if (total_bytes == 0 || ntensors == 0) return HVDX_OK;
  for (int s = 0; s < 2 * nranks - 2; ++s) {
    rc = bcast_tensors_step(ptrs, nbytes, voffset, ntensors, total_bytes, nranks, root, s,
                            static_cast<hipStream_t>(stream));
    if (rc) return rc;
  }
  return HVDX_OK;
}

int hvdx_broadcast(void* const* bufs, int nranks, int64_t nbytes, int root, void* stream) {
  int rc = check_bcast(bufs, nranks, nbytes, root, "hvdx_broadcast");
  if (rc) return rc;
  for (int s = 0; nbytes > 0 && s < 2 * nranks - 2; ++s) {
    rc = bcast_step(bufs, nranks, nbytes, root, s, static_cast<hipStream_t>(stream));
    if (rc) return rc;
  }
  return HVDX_OK;
}

}  // extern "C"
