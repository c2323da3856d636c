// Shared host and device helpers of the planner library (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <functional>
#include <string>

#include "nopfs.h"

namespace nopfs {

// ---------------------------------------------------------------- errors --
struct Status {
  int code = NOPFS_OK;
  bool ok() const { return code == NOPFS_OK; }
};

void set_last_error(const std::string& msg);
int fail(int code, const std::string& msg);  // records msg, returns code
int hip_fail(hipError_t err, const char* what);

#define NOPFS_HIP(call)                                   \
  do {                                                    \
    hipError_t _e = (call);                               \
    if (_e != hipSuccess) return ::nopfs::hip_fail(_e, #call); \
  } while (0)

// ----------------------------------------------------------------- shape --
struct Shape {
  int64_t F, E, N, B;
  int drop_last;
  int64_t T;       // iterations per epoch
  int64_t L;       // per-epoch reads of worker 0 (the longest row)
  int64_t M_max;   // E * L
  int64_t P;       // issued positions per epoch
  uint64_t seed;
};

// Validates the job and fills the shape. Returns a NOPFS_* code.
int make_shape(const nopfs_job* job, Shape* s);
// Validates the performance model's parameters (J in 1..32, every rate and
// thread count positive and finite).
int model_check(const nopfs_model* m);

// Per-epoch reads of worker i (same rule as the public header).
__host__ __device__ inline int64_t epoch_len(int64_t F, int64_t N, int64_t B,
                                             int drop_last, int64_t i) {
  if (drop_last) return (F / (N * B)) * B;
  if (i >= F) return 0;
  return (F - i + N - 1) / N;
}

// --------------------------------------------------------------- scratch --
// Device scratch of a call, from the block of (current device, stream).
class Scratch {
 public:
  // Takes the scratch arena of (current device, s): calls on one stream share
  // it and run one at a time (a Scratch holds the arena's lock while it lives;
  // Scratch objects of one call nest).
  explicit Scratch(hipStream_t s);
  ~Scratch();
  Scratch(const Scratch&) = delete;
  Scratch& operator=(const Scratch&) = delete;
  // Allocates `bytes` (rounded up to 256) and returns NOPFS_OK or ENOMEM.
  int alloc(void** p, size_t bytes);
  template <typename T>
  int alloc_n(T** p, size_t n) { return alloc(reinterpret_cast<void**>(p), n * sizeof(T)); }

 private:
  hipStream_t stream_;
  struct Arena* arena_ = nullptr;
  size_t recs_[32] = {};  // this object's entries on the arena's stack
  int n_ = 0;
};

// Runs `call` (an entry point's implementation) on this thread with every
// scratch buffer carved from a stand-in block that is never dereferenced and
// no kernel launched; *peak receives the most scratch the call held at once.
// Returns the call's status (argument errors as usual).
int run_sizing(const std::function<int()>& call, size_t* peak);
// Runs `call` on this thread with its scratch carved from the fixed device
// block [block, block + cap), which never grows: a call that needs more
// fails with ENOMEM. Calls on one block are enqueued one at a time.
int run_in_fixed_block(char* block, size_t cap, const std::function<int()>& call);
// True inside run_sizing on this thread.
bool sizing_only();

// ---------------------------------------------------------------- launch --
// Records HIP events around a launch when profiling is on.
void prof_begin(const char* name, hipStream_t s);
void prof_end(hipStream_t s);

template <typename Kernel, typename... Args>
int launch(const char* name, Kernel k, dim3 grid, dim3 block, size_t shmem,
           hipStream_t s, Args... args) {
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return NOPFS_OK;
  if (sizing_only()) return NOPFS_OK;
  prof_begin(name, s);
  hipLaunchKernelGGL(k, grid, block, shmem, s, args...);
  hipError_t e = hipGetLastError();
  prof_end(s);
  if (e != hipSuccess) return hip_fail(e, name);
  return NOPFS_OK;
}

// Debug overrides (nopfs_debug_set).
int64_t debug_value(int which);
bool take_alloc_failure();

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------- device --
// Workgroups are dispatched round-robin over the 8 XCDs (WG i -> XCD i % 8),
// and each XCD has its own L2. Remapping the flat block id so that XCD x
// receives a contiguous range of logical tiles keeps neighbouring tiles
// (which touch neighbouring cache lines) inside one L2. `padded` is the grid
// size rounded up to a multiple of 8; callers drop logical ids >= real count.
__device__ inline uint32_t xcd_logical(uint32_t bid, uint32_t padded) {
  const uint32_t per = padded >> 3;
  return (bid & 7u) * per + (bid >> 3);
}

inline uint32_t xcd_padded(uint32_t n) { return (n + 7u) & ~7u; }

// Non-temporal stores, for outputs written once in whole lines that the same
// pass does not read back: they stream to memory instead of being held in L2
// (the dense count and first-read rows: 7.1 -> 6.3 ms at ImageNet-22k).
// Scattered or partial-line stores must not use them: the read-cell list
// stored this way (4-byte stores a few per line) took 14.4 ms instead.
template <typename T>
__device__ __forceinline__ void stream_store(T* p, T v) {
  __builtin_nontemporal_store(v, p);
}
__device__ __forceinline__ void stream_store(int4* p, int4 v) {
  typedef int v4 __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(v4{v.x, v.y, v.z, v.w}, reinterpret_cast<v4*>(p));
}
__device__ __forceinline__ void stream_store(uint4* p, uint4 v) {
  typedef unsigned v4 __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(v4{v.x, v.y, v.z, v.w}, reinterpret_cast<v4*>(p));
}

__device__ inline uint64_t lanemask_lt() {
  const uint32_t lane = __lane_id();
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Inclusive scan of a 32-bit value across the 64 lanes of a wave (all lanes
// active), in registers: shifts by 1, 2, 4 and 8 lanes inside each row of
// 16 (lanes shifted in from outside the row add 0), then the last lane of
// row 0 is added to row 1 and that of row 2 to row 3, then the last lane of
// row 1 (the sum of rows 0 and 1) to rows 2 and 3.
__device__ inline uint32_t wave_inclusive_scan(uint32_t v) {
  v += __builtin_amdgcn_update_dpp(0u, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0u, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0u, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0u, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0u, v, 0x142, 0xa, 0xf, false);  // row_bcast:15, rows 1 and 3
  v += __builtin_amdgcn_update_dpp(0u, v, 0x143, 0xc, 0xf, false);  // row_bcast:31, rows 2 and 3
  return v;
}

// One DPP move of a 64-bit value (both halves with the same control); lanes
// with no source, or in rows outside RowMask, receive 0.
template <int Ctrl, int RowMask>
__device__ __forceinline__ uint64_t dpp_move64(uint64_t v) {
  const uint32_t lo = __builtin_amdgcn_update_dpp(0u, uint32_t(v), Ctrl, RowMask, 0xf, false);
  const uint32_t hi = __builtin_amdgcn_update_dpp(0u, uint32_t(v >> 32), Ctrl, RowMask, 0xf, false);
  return (uint64_t(hi) << 32) | lo;
}

// The 64-bit form of wave_inclusive_scan, same steps (all lanes active).
__device__ inline uint64_t wave_inclusive_scan64(uint64_t v) {
  v += dpp_move64<0x111, 0xf>(v);  // row_shr:1
  v += dpp_move64<0x112, 0xf>(v);  // row_shr:2
  v += dpp_move64<0x114, 0xf>(v);  // row_shr:4
  v += dpp_move64<0x118, 0xf>(v);  // row_shr:8
  v += dpp_move64<0x142, 0xa>(v);  // row_bcast:15, rows 1 and 3
  v += dpp_move64<0x143, 0xc>(v);  // row_bcast:31, rows 2 and 3
  return v;
}

// A lane's 64-bit value, read by every lane (the lane index is uniform).
__device__ __forceinline__ uint64_t read_lane64(uint64_t v, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane(int(uint32_t(v)), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(int(uint32_t(v >> 32)), lane);
  return (uint64_t(hi) << 32) | lo;
}

// Exclusive scan over the whole workgroup (blockDim.x a multiple of 64, at
// most 1024). `tmp` holds one slot per wave plus one. Returns the exclusive
// prefix of v; *total receives the sum over the block. kClose = false leaves
// out the closing barrier, for callers that pass another barrier before tmp
// is written again.
template <bool kClose = true>
__device__ inline uint32_t block_exclusive_scan(uint32_t v, uint32_t* tmp,
                                                uint32_t* total) {
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  uint32_t inc = wave_inclusive_scan(v);
  if (lane == 63) tmp[wave] = inc;
  __syncthreads();
  if (threadIdx.x < 64) {
    uint32_t w = threadIdx.x < (unsigned)nwaves ? tmp[threadIdx.x] : 0u;
    uint32_t wi = wave_inclusive_scan(w);
    if (threadIdx.x < (unsigned)nwaves) tmp[threadIdx.x] = wi - w;
    if (threadIdx.x == 63) tmp[64] = wi;
  }
  __syncthreads();
  uint32_t r = tmp[wave] + inc - v;
  *total = tmp[64];
  if (kClose) __syncthreads();
  return r;
}

__device__ inline uint64_t block_exclusive_scan64(uint64_t v, uint64_t* tmp,
                                                  uint64_t* total) {
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  uint64_t inc = wave_inclusive_scan64(v);
  if (lane == 63) tmp[wave] = inc;
  __syncthreads();
  if (threadIdx.x < 64) {
    uint64_t w = threadIdx.x < (unsigned)nwaves ? tmp[threadIdx.x] : 0ull;
    uint64_t wi = wave_inclusive_scan64(w);
    if (threadIdx.x < (unsigned)nwaves) tmp[threadIdx.x] = wi - w;
    if (threadIdx.x == 63) tmp[64] = wi;
  }
  __syncthreads();
  uint64_t r = tmp[wave] + inc - v;
  *total = tmp[64];
  __syncthreads();
  return r;
}

// In-place exclusive scan of the n-entry LDS array a by the whole workgroup:
// each thread sums a contiguous segment, one block scan combines the
// segments, and each thread writes its segment's prefixes. Returns the total.
// Ends with a barrier.
__device__ inline uint32_t block_scan_array(uint32_t* a, uint32_t n, uint32_t* tmp) {
  const uint32_t per = (n + blockDim.x - 1) / blockDim.x;
  const uint32_t b0 = threadIdx.x * per;
  const uint32_t b1 = b0 + per < n ? b0 + per : n;
  uint32_t sum = 0;
  for (uint32_t b = b0; b < b1; ++b) sum += a[b];
  uint32_t total;
  uint32_t run = block_exclusive_scan<false>(sum, tmp, &total);  // the barrier below closes it
  for (uint32_t b = b0; b < b1; ++b) {
    const uint32_t v = a[b];
    a[b] = run;
    run += v;
  }
  __syncthreads();
  return total;
}

}  // namespace nopfs
