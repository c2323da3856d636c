// Host-side plumbing of the planner library: argument validation and shape
// arithmetic, error reporting, the per-stream scratch blocks, per-kernel
// event timing, and the calibration copy kernel.
#include <functional>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "common.hpp"

namespace nopfs {

static thread_local std::string g_last_error;

void set_last_error(const std::string& msg) { g_last_error = msg; }

int fail(int code, const std::string& msg) {
  set_last_error(msg);
  return code;
}

int hip_fail(hipError_t err, const char* what) {
  set_last_error(std::string(what) + ": " + hipGetErrorString(err));
  return NOPFS_EDEVICE;
}

int make_shape(const nopfs_job* job, Shape* s) {
  if (!job) return fail(NOPFS_EINVAL, "job is NULL");
  if (job->F < 1 || job->E < 1 || job->N < 1 || job->B < 1)
    return fail(NOPFS_EINVAL, "F, E, N and B must be >= 1");
  if (job->drop_last != 0 && job->drop_last != 1)
    return fail(NOPFS_EINVAL, "drop_last must be 0 or 1");
  if (job->F >= (int64_t(1) << 31)) return fail(NOPFS_ERANGE, "F must be < 2^31");
  if (job->E > 255) return fail(NOPFS_ERANGE, "E must be <= 255 (uint8 counts)");
  s->F = job->F;
  s->E = job->E;
  s->N = job->N;
  s->B = job->B;
  s->drop_last = job->drop_last;
  s->seed = job->seed;
  const int64_t G = s->N * s->B;
  s->T = s->drop_last ? s->F / G : (s->F + G - 1) / G;
  s->L = epoch_len(s->F, s->N, s->B, s->drop_last, 0);
  s->M_max = s->E * s->L;
  s->P = s->drop_last ? s->T * G : s->F;
  if (s->M_max >= (int64_t(1) << 31)) return fail(NOPFS_ERANGE, "M_max must be < 2^31");
  return NOPFS_OK;
}

// ---------------------------------------------------------------- scratch --
// Test overrides (nopfs_debug_set): per host thread, so a test that forces a
// slow path affects only the calls it makes itself.
static thread_local int64_t g_debug[6] = {0, 0, 0, 0, 0, 0};

int64_t debug_value(int which) { return (which >= 0 && which < 6) ? g_debug[which] : 0; }

bool take_alloc_failure() {
  if (g_debug[3]) {
    g_debug[3] = 0;
    return true;
  }
  return false;
}

// Scratch of one (device, stream): one block of device memory reused by
// every call on that stream, handed out as a stack (the Scratch objects of a
// call nest, and a buffer's space is taken back once every buffer above it
// is released). A call that needs more than the block gets extra blocks; at
// its end the stream is synchronised and the block is replaced by one of the
// call's peak size, so later calls of that size allocate nothing. Per-call
// stream-ordered allocations of gigabytes stalled the host for hundreds of
// milliseconds per call after ~100 calls (the allocator returned and mapped
// memory again); the arena keeps its memory until nopfs_scratch_release or
// the end of the process.
struct Arena {
  std::recursive_mutex mu;
  bool fixed = false;       // a fixed block that never grows (no allocation)
  int depth = 0;            // live Scratch objects
  char* block = nullptr;    // the reused block
  size_t cap = 0;
  size_t top = 0;           // bytes of the block in use
  size_t extent = 0;        // top plus live extra blocks
  size_t peak = 0;          // largest extent of the current call
  size_t peak_total = 0;    // largest extent of any call (sizing passes)
  bool failed = false;      // an allocation of the current call failed
  std::vector<void*> extra; // blocks beyond `block`, freed at the call's end
  struct Rec {
    size_t off, bytes;
    bool in_block, live;
  };
  std::vector<Rec> stack;
};

static std::mutex g_arenas_mu;
static std::map<std::pair<int, hipStream_t>, Arena*> g_arenas;  // kept until exit

// The arena of (current device, s); created on first use unless `create` is
// false (then nullptr when there is none).
static Arena* arena_of(hipStream_t s, bool create = true) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> g(g_arenas_mu);
  auto it = g_arenas.find({dev, s});
  if (it != g_arenas.end()) return it->second;
  if (!create) return nullptr;
  Arena* a = new (std::nothrow) Arena;
  if (a) g_arenas[{dev, s}] = a;
  return a;
}

// A fixed arena installed for the calls of this thread (sizing passes and
// the allocation-free entry point), and whether launches are only counted.
static thread_local Arena* t_fixed_arena = nullptr;
static thread_local bool t_sizing = false;

bool sizing_only() { return t_sizing; }

int run_sizing(const std::function<int()>& call, size_t* peak) {
  // The call runs its host logic with every scratch buffer carved from a
  // block that is never dereferenced and no kernel launched. No decision of
  // the library depends on where its scratch lies (only on the job and the
  // caller's pointers), so the sizes are those of a real call.
  Arena a;
  a.fixed = true;
  a.block = reinterpret_cast<char*>(uintptr_t(1) << 46);
  a.cap = size_t(1) << 45;
  Arena* prev = t_fixed_arena;
  const bool prev_sizing = t_sizing;
  t_fixed_arena = &a;
  t_sizing = true;
  int rc;
  try {
    rc = call();
  } catch (...) {
    rc = fail(NOPFS_EDEVICE, "unexpected host exception");
  }
  t_fixed_arena = prev;
  t_sizing = prev_sizing;
  *peak = a.peak_total;
  return rc;
}

int run_in_fixed_block(char* block, size_t cap, const std::function<int()>& call) {
  static std::mutex mu;
  static std::map<char*, Arena*> arenas;  // one per block (per device), kept until exit
  Arena* a;
  {
    std::lock_guard<std::mutex> g(mu);
    Arena*& r = arenas[block];
    if (!r) {
      r = new (std::nothrow) Arena;
      if (!r) return fail(NOPFS_ENOMEM, "host allocation failed");
      r->fixed = true;
      r->block = block;
      r->cap = cap;
    }
    a = r;
  }
  std::lock_guard<std::recursive_mutex> g(a->mu);  // one call per block at a time
  Arena* prev = t_fixed_arena;
  t_fixed_arena = a;
  int rc;
  try {
    rc = call();
  } catch (...) {
    rc = fail(NOPFS_EDEVICE, "unexpected host exception");
  }
  t_fixed_arena = prev;
  return rc;
}

Scratch::Scratch(hipStream_t s) : stream_(s), arena_(t_fixed_arena ? t_fixed_arena : arena_of(s)) {
  if (!arena_) return;
  arena_->mu.lock();
  ++arena_->depth;
}

Scratch::~Scratch() {
  Arena* a = arena_;
  if (!a) return;
  for (int i = 0; i < n_; ++i) a->stack[recs_[i]].live = false;
  while (!a->stack.empty() && !a->stack.back().live) {
    const Arena::Rec& r = a->stack.back();
    if (r.in_block) a->top = r.off;
    a->extent -= r.bytes;
    a->stack.pop_back();
  }
  if (--a->depth == 0) {
    if (a->peak > a->peak_total) a->peak_total = a->peak;
    if (!a->fixed && !a->extra.empty()) {
      // the call outgrew the block: after its work, one block of its peak
      // (a call that ran out of memory keeps the old block)
      (void)hipStreamSynchronize(stream_);
      for (void* q : a->extra) (void)hipFree(q);
      a->extra.clear();
      if (!a->failed) {
        if (a->block) (void)hipFree(a->block);
        a->block = nullptr;
        a->cap = 0;
        void* q = nullptr;
        if (hipMalloc(&q, a->peak) == hipSuccess && q) {
          a->block = static_cast<char*>(q);
          a->cap = a->peak;
        }
      }
      (void)hipGetLastError();
    }
    a->peak = 0;
    a->failed = false;
  }
  a->mu.unlock();
}

int Scratch::alloc(void** p, size_t bytes) {
  *p = nullptr;
  if (n_ >= 32) return fail(NOPFS_ENOMEM, "too many scratch buffers");
  if (take_alloc_failure()) return fail(NOPFS_ENOMEM, "scratch allocation failed (test hook)");
  Arena* a = arena_;
  if (!a) return fail(NOPFS_ENOMEM, "no device memory for scratch (no current device)");
  bytes = (bytes + 255) & ~size_t(255);
  if (bytes == 0) bytes = 256;
  Arena::Rec r{0, bytes, false, true};
  if (a->top + bytes <= a->cap) {
    r.off = a->top;
    r.in_block = true;
    a->top += bytes;
    *p = a->block + r.off;
  } else if (a->fixed) {
    return fail(NOPFS_ENOMEM, std::string("scratch of ") + std::to_string(a->top + bytes) +
                                  " bytes exceeds the fixed block of " + std::to_string(a->cap));
  } else {
    void* q = nullptr;
    const hipError_t e = hipMalloc(&q, bytes);
    if (e != hipSuccess || !q) {
      (void)hipGetLastError();
      a->failed = true;
      return fail(NOPFS_ENOMEM, std::string("scratch allocation of ") + std::to_string(bytes) +
                                    " bytes failed");
    }
    a->extra.push_back(q);
    *p = q;
  }
  a->extent += bytes;
  if (a->extent > a->peak) a->peak = a->extent;
  recs_[n_++] = a->stack.size();
  a->stack.push_back(r);
  return NOPFS_OK;
}

// -------------------------------------------------------------- profiling --
namespace {
struct ProfRec {
  const char* name;
  hipEvent_t start, stop;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRec> g_prof;
thread_local size_t t_open_idx = 0;
}  // namespace

void prof_begin(const char* name, hipStream_t s) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  if (!g_prof_on) return;
  ProfRec r{name, nullptr, nullptr};
  if (hipEventCreate(&r.start) != hipSuccess || hipEventCreate(&r.stop) != hipSuccess) {
    (void)hipGetLastError();
    return;
  }
  (void)hipEventRecord(r.start, s);
  g_prof.push_back(r);
  t_open_idx = g_prof.size();
}

void prof_end(hipStream_t s) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  if (!g_prof_on || t_open_idx == 0 || t_open_idx > g_prof.size()) return;
  (void)hipEventRecord(g_prof[t_open_idx - 1].stop, s);
  t_open_idx = 0;
}

static void prof_clear() {
  for (auto& r : g_prof) {
    if (r.start) (void)hipEventDestroy(r.start);
    if (r.stop) (void)hipEventDestroy(r.stop);
  }
  g_prof.clear();
}

// -------------------------------------------------------- calibration copy --
__global__ void __launch_bounds__(256) calibration_copy_kernel(const uint4* __restrict__ src,
                                                               uint4* __restrict__ dst,
                                                               int64_t n) {
  int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (; i < n; i += stride) dst[i] = src[i];
}

}  // namespace nopfs

using namespace nopfs;

extern "C" {

int nopfs_stream_shape(const nopfs_job* job, int64_t* T, int64_t* M_max,
                       int64_t* M_per_worker) {
  try {
    Shape s;
    int rc = make_shape(job, &s);
    if (rc) return rc;
    if (T) *T = s.T;
    if (M_max) *M_max = s.M_max;
    if (M_per_worker)
      for (int64_t i = 0; i < s.N; ++i)
        M_per_worker[i] = s.E * epoch_len(s.F, s.N, s.B, s.drop_last, i);
    return NOPFS_OK;
  } catch (...) {
    return fail(NOPFS_EINVAL, "unexpected host exception");
  }
}

const char* nopfs_strerror(int code) {
  switch (code) {
    case NOPFS_OK: return "ok";
    case NOPFS_EINVAL: return "invalid argument";
    case NOPFS_ERANGE: return "argument out of supported range";
    case NOPFS_ENOMEM: return "scratch allocation failed";
    case NOPFS_EDEVICE: return "HIP runtime or launch error";
    default: return "unknown status code";
  }
}

const char* nopfs_last_error(void) { return g_last_error.c_str(); }

int nopfs_profile_enable(int enable) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  if (enable) {
    prof_clear();
    g_prof_on = true;
  } else {
    g_prof_on = false;
  }
  return NOPFS_OK;
}

int nopfs_profile_query(int idx, const char** name, int64_t* launches,
                        double* total_ms) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  std::vector<const char*> names;
  for (auto& r : g_prof) {
    bool seen = false;
    for (auto* n : names) seen |= (std::string(n) == r.name);
    if (!seen) names.push_back(r.name);
  }
  if (idx < 0 || idx >= int(names.size())) return NOPFS_EINVAL;
  double ms = 0;
  int64_t cnt = 0;
  for (auto& r : g_prof) {
    if (std::string(r.name) != names[idx]) continue;
    if (hipEventSynchronize(r.stop) != hipSuccess) return hip_fail(hipGetLastError(), "event sync");
    float t = 0;
    if (hipEventElapsedTime(&t, r.start, r.stop) != hipSuccess)
      return hip_fail(hipGetLastError(), "event elapsed");
    ms += t;
    cnt++;
  }
  if (name) *name = names[idx];
  if (launches) *launches = cnt;
  if (total_ms) *total_ms = ms;
  return NOPFS_OK;
}

int nopfs_calibration_copy(const void* src, void* dst, int64_t bytes, void* hip_stream) {
  if (!src || !dst || bytes < 0 || (bytes & 15) ||
      (reinterpret_cast<uintptr_t>(src) & 15) || (reinterpret_cast<uintptr_t>(dst) & 15))
    return fail(NOPFS_EINVAL, "calibration copy needs 16-byte aligned, 16-byte multiple buffers");
  const int64_t n = bytes / 16;
  if (n == 0) return NOPFS_OK;
  int64_t blocks = ceil_div(n, 256 * 8);
  if (blocks > 65536) blocks = 65536;
  return launch("calibration_copy", calibration_copy_kernel, dim3(uint32_t(blocks)), dim3(256), 0,
                static_cast<hipStream_t>(hip_stream), static_cast<const uint4*>(src),
                static_cast<uint4*>(dst), n);
}

int nopfs_scratch_release(void* hip_stream) {
  try {
    const hipStream_t s = static_cast<hipStream_t>(hip_stream);
    Arena* a = arena_of(s, false);
    if (!a) return NOPFS_OK;  // no block on this stream
    std::lock_guard<std::recursive_mutex> g(a->mu);  // waits for a call being enqueued
    if (a->depth != 0) return fail(NOPFS_EINVAL, "scratch release from inside a call");
    if (!a->block) return NOPFS_OK;
    NOPFS_HIP(hipStreamSynchronize(s));
    NOPFS_HIP(hipFree(a->block));
    a->block = nullptr;
    a->cap = 0;
    a->top = 0;
    return NOPFS_OK;
  } catch (...) {
    return fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}

int nopfs_debug_set(int which, int64_t value) {
  if (which < 1 || which > 5 || value < 0) return NOPFS_EINVAL;
  g_debug[which] = value;
  return NOPFS_OK;
}

}  // extern "C"
