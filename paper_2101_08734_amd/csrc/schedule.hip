// nopfs_prefetch_order and nopfs_staging_schedule: what the Design section
// derives from the streams and the placement for a worker's prefetchers.
//
// Both need R grouped by sample (a first read, a size) and then results in
// stream order, so both run on the per-worker partition of R by sample
// window (the one the counting pass uses, windows of 2^13 samples): a tile
// per window does the per-sample work in LDS and writes one value per read
// in partitioned order; a pass per sub-chunk of 2^14 reads puts the values
// back in stream order through LDS. No pass scatters into or gathers from
// HBM at random.
//
// Prefetch order. Each storage class is filled in the order the worker first
// needs its samples (the first rule of optimal prefetching, I/O Access
// Patterns section). Tier t's queue holds the samples placed in t that the
// worker reads, by first read; the queues are concatenated fastest tier first.
//   pf_tile   -- per (worker, window): first read of each sample of the
//                window (LDS atomic min over its reads) and the window's
//                tiers; each read gets code t + 1 if it is its sample's first
//                read and the sample sits in cache tier t < J, else 0
//                (one byte per read, partitioned order).
//   pf_count  -- per sub-chunk: codes per tier.
//   pf_scan   -- per worker and tier: exclusive scan over sub-chunks plus
//                the start of the tier's queue; the queue lengths.
//   pf_write  -- per sub-chunk: codes back in stream order in LDS; each wave
//                step of 64 positions splits its coded positions by tier
//                (one ballot per tier present) and writes R[i][f] to the
//                next queue slots; then its share of the -1 padding.
// Staging schedule. The staging buffer is filled in stream order and a
// sample is dropped once read (Design); it is filled circularly
// (Implementation). With S the prefix sum of the sizes along R_i (S(-1) = 0),
// the sample at h may be fetched once the worker has read position
// fill(h) - 1: fill(h) is the smallest f <= h with S(h) - S(f - 1) <= d0,
// or h when the sample alone is larger than d0. Equivalently fill(h) is one
// past the smallest g in [-1, h] with S(g) >= S(h) - d0, capped at h.
//   st_tile   -- per (window, group of workers): the window's sizes in LDS;
//                every read of the group's workers gets its sample's size
//                (partitioned order).
//   st_sum    -- per sub-chunk: sizes back in stream order in LDS, their
//                inclusive prefix sums inside the sub-chunk, its total.
//   st_base   -- per worker: exclusive scan of the sub-chunk totals.
//   st_bounds -- per quarter of a sub-chunk (4096 positions): the g of its
//                first and of its last position (binary search over S; g
//                never decreases along R).
//   st_fill   -- per quarter: S over that g range is staged in LDS (the few
//                sub-chunks it spans give the bases), each thread
//                binary-searches the g of its first position there and walks
//                its other positions with two pointers; -1 in padding.
#include <limits.h>

#include <new>

#include "partition.hpp"

namespace nopfs {
namespace {

// Tuning knob (identical results; only speed changes): workers per st_tile
// workgroup (each loads the window's sizes once for all of them).
#ifndef NOPFS_ST_GROUP
#define NOPFS_ST_GROUP 16
#endif


constexpr int kSchedWs = 13;             // partition windows: 2^13 samples
constexpr int kWin = 1 << kSchedWs;      // samples per LDS pass of a tile
constexpr int kTileThreads = 256;
constexpr int kPfMaxJ = 128;

// ------------------------------------------------------------- prefetch --
constexpr int kPfKeep = 8;  // reads per thread kept in registers between the passes

// Per read of the tile: first-read candidate for its sample (pass 1), then
// its code (pass 2). When the tile's runs fit one run table and its reads fit
// kPfKeep per thread, the reads are spread evenly over the threads through
// the run table and kept in registers between the passes (two dependent
// global loads per tile); otherwise each thread walks whole runs twice.
__global__ void __launch_bounds__(kTileThreads)
pf_tile(SegParams p, const uint32_t* __restrict__ Pk, const uint16_t* __restrict__ OT,
        const int8_t* __restrict__ tier, int32_t J, uint8_t* __restrict__ code,
        uint32_t ntiles) {
  __shared__ int32_t fi[kWin];  // first read of each sample of the pass
  __shared__ int8_t tw[kWin];   // its tier
  __shared__ RunTable<kTileThreads> rt;
  const uint32_t tile = xcd_logical(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int64_t i = tile / p.nbk;
  const uint32_t kb = tile - uint32_t(i) * p.nbk;
  const int64_t k0 = int64_t(kb) << p.ws;
  const int64_t kend = k0 + (int64_t(1) << p.ws) < p.F ? k0 + (int64_t(1) << p.ws) : p.F;
  const int8_t* trow = tier + i * p.F;
  uint8_t* crow = code + i * p.M_max;
  const uint32_t* prow = Pk + i * p.M_max;
  const int64_t runs = int64_t(p.E) * p.nsc;
  const bool one_table = runs <= kTileThreads && kend - k0 <= kWin;  // uniform
  if (one_table) {
    const uint32_t wl = uint32_t(kend - k0);
    constexpr int kTb = kWin / kTileThreads;  // tier bytes per thread
    int8_t tv[kTb];
#pragma unroll
    for (int u = 0; u < kTb; ++u) {
      const uint32_t x = threadIdx.x + u * kTileThreads;
      tv[u] = x < wl ? trow[k0 + x] : int8_t(-1);
    }
#pragma unroll
    for (int u = 0; u < kTb; ++u) {
      const uint32_t x = threadIdx.x + u * kTileThreads;
      if (x < wl) {
        fi[x] = INT_MAX;
        tw[x] = tv[u];
      }
    }
    // run table (its scan's barriers also publish fi and tw)
    const uint32_t total = load_runs(p, i, kb, OT, rt, 0, runs, 0);
    if (total <= uint32_t(kPfKeep * kTileThreads)) {
      uint32_t v[kPfKeep];
      int32_t pos[kPfKeep], fb[kPfKeep];
#pragma unroll
      for (int u = 0; u < kPfKeep; ++u) {
        const uint32_t t = threadIdx.x + u * kTileThreads;
        pos[u] = -1;
        fb[u] = 0;
        if (t < total) {
          int lo;
          if (total <= kRunMap) {
            lo = rt.run_of[t];
          } else {
            lo = 0;  // last run with pref <= t
            int hi = int(runs) - 1;
            while (lo < hi) {
              const int mid = (lo + hi + 1) >> 1;
              if (rt.pref[mid] <= t) lo = mid; else hi = mid - 1;
            }
          }
          pos[u] = rt.start[lo] + int32_t(t - rt.pref[lo]);
          fb[u] = rt.fbase[lo];
        }
      }
#pragma unroll
      for (int u = 0; u < kPfKeep; ++u) v[u] = pos[u] >= 0 ? prow[pos[u]] : 0u;
#pragma unroll
      for (int u = 0; u < kPfKeep; ++u)
        if (pos[u] >= 0) {
          const uint32_t x = v[u] >> kScShift;
          if (x < wl) atomicMin(&fi[x], fb[u] + int32_t(v[u] & kJMask));
        }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < kPfKeep; ++u)
        if (pos[u] >= 0) {
          const uint32_t x = v[u] >> kScShift;
          if (x < wl) {
            const int32_t t = tw[x];
            const bool queued = fi[x] == fb[u] + int32_t(v[u] & kJMask) && t >= 0 && t < J;
            crow[pos[u]] = queued ? uint8_t(t + 1) : uint8_t(0);
          }
        }
      return;
    }
    __syncthreads();  // the table is no longer read
  }
  for (int64_t w0 = k0; w0 < kend; w0 += kWin) {
    const uint32_t wl = uint32_t(kend - w0 < kWin ? kend - w0 : kWin);
    const uint32_t xoff = uint32_t(w0 - k0);
    for (uint32_t x = threadIdx.x; x < wl; x += kTileThreads) {
      fi[x] = INT_MAX;
      tw[x] = trow[w0 + x];
    }
    __syncthreads();
    walk_runs(p, i, kb, Pk, OT, threadIdx.x, kTileThreads, [&](int64_t fb, uint32_t, uint32_t v) {
      const uint32_t x = (v >> kScShift) - xoff;
      if (x < wl) atomicMin(&fi[x], int32_t(fb + (v & kJMask)));
    });
    __syncthreads();
    walk_runs(p, i, kb, Pk, OT, threadIdx.x, kTileThreads, [&](int64_t fb, uint32_t q, uint32_t v) {
      const uint32_t x = (v >> kScShift) - xoff;
      if (x < wl) {
        const int32_t t = tw[x];
        const bool queued = fi[x] == int32_t(fb + (v & kJMask)) && t >= 0 && t < J;
        crow[fb + q] = queued ? uint8_t(t + 1) : uint8_t(0);
      }
    });
    __syncthreads();
  }
}

// Code byte -> tier code in [0, J] (codes above J, which pf_tile never
// writes, are dropped so every queue slot stays inside the row).
__device__ __forceinline__ uint32_t clamp_code(uint32_t m, int32_t J) {
  return m <= uint32_t(J) ? m : 0u;
}

// cnt layout: [N][nch][J]. Order of positions does not matter for counting,
// so the codes are read in partitioned order.
__global__ void __launch_bounds__(256)
pf_count(SegParams p, int32_t J, const uint8_t* __restrict__ code, uint32_t nch,
         int32_t* __restrict__ cnt) {
  __shared__ uint32_t s_cnt[kPfMaxJ];
  const SubChunk s = sub_chunk(p, nch, blockIdx.x);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int x = threadIdx.x; x < J; x += 256) s_cnt[x] = 0;
  __syncthreads();
  const uint8_t* src = code + s.base;
  constexpr int kBatch = 8;
  for (int64_t j0 = int64_t(w) * 64 * kBatch; j0 < s.len; j0 += 256 * kBatch) {
    uint32_t m[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int64_t j = j0 + u * 64 + lane;
      m[u] = j < s.len ? clamp_code(src[j], J) : 0u;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      uint64_t act = __ballot(m[u] != 0);
      while (act) {
        const int lead = __builtin_ctzll(act);
        const uint32_t tc = __builtin_amdgcn_readlane(m[u], lead);
        const uint64_t same = __ballot(m[u] == tc);
        if (lane == lead) atomicAdd(&s_cnt[tc - 1], uint32_t(__popcll(same)));
        act &= ~same;
      }
    }
  }
  __syncthreads();
  int32_t* out = cnt + (s.i * nch + s.c) * J;
  for (int x = threadIdx.x; x < J; x += 256) out[x] = int32_t(s_cnt[x]);
}

// In place: cnt[i][c][j] becomes the queue slot (within row i of order) of
// sub-chunk c's first tier-j sample; qlen[i][j] the queue lengths; tot[i]
// their sum.
__global__ void __launch_bounds__(1024)
pf_scan(int32_t J, uint32_t nch, int32_t* __restrict__ cnt, int64_t* __restrict__ qlen,
        int64_t* __restrict__ tot) {
  __shared__ uint32_t tmp[65];
  const int64_t i = blockIdx.x;
  int32_t* row = cnt + i * int64_t(nch) * J;
  uint32_t start = 0;
  for (int32_t j = 0; j < J; ++j) {
    uint32_t carry = 0;
    for (uint32_t c0 = 0; c0 < nch; c0 += 1024) {
      const uint32_t c = c0 + threadIdx.x;
      const uint32_t v = c < nch ? uint32_t(row[int64_t(c) * J + j]) : 0u;
      uint32_t total;
      const uint32_t ex = block_exclusive_scan(v, tmp, &total);
      if (c < nch) row[int64_t(c) * J + j] = int32_t(start + carry + ex);
      carry += total;
    }
    if (threadIdx.x == 0) qlen[i * J + j] = int64_t(carry);
    start += carry;
  }
  if (threadIdx.x == 0) tot[i] = int64_t(start);
}

constexpr int kPfWaves = 4;
constexpr int kPfQuarter = kSC / kPfWaves;  // positions per wave: 4096
constexpr int kPfBatch = 8;                 // wave steps whose loads are issued together

__global__ void __launch_bounds__(64 * kPfWaves)
pf_write(SegParams p, int32_t J, const uint32_t* __restrict__ Pk, const uint8_t* __restrict__ code,
         const int32_t* __restrict__ R, uint32_t nch, const int32_t* __restrict__ slot0,
         const int64_t* __restrict__ tot, int32_t* __restrict__ order) {
  __shared__ uint8_t s_code[kSC];
  __shared__ uint32_t s_wcnt[kPfWaves][kPfMaxJ];
  __shared__ int32_t s_run[kPfWaves][kPfMaxJ];
  const SubChunk s = sub_chunk(p, nch, blockIdx.x);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  // codes to stream order (every position of the sub-chunk has one entry)
  for (int64_t q = threadIdx.x; q < s.len; q += 64 * kPfWaves)
    s_code[Pk[s.base + q] & kJMask] = code[s.base + q];
  for (int x = lane; x < J; x += 64) s_wcnt[w][x] = 0;
  __syncthreads();
  const int64_t j0 = int64_t(w) * kPfQuarter;
  // this wave's codes per tier
  for (int u = 0; u < kPfQuarter / 64; ++u) {
    const int64_t j = j0 + u * 64 + lane;
    const uint32_t m = j < s.len ? clamp_code(s_code[j], J) : 0u;
    uint64_t act = __ballot(m != 0);
    while (act) {
      const int lead = __builtin_ctzll(act);
      const uint32_t tc = __builtin_amdgcn_readlane(m, lead);
      const uint64_t same = __ballot(m == tc);
      if (lane == lead) s_wcnt[w][tc - 1] += uint32_t(__popcll(same));
      act &= ~same;
    }
  }
  __syncthreads();
  const int32_t* sl = slot0 + (s.i * nch + s.c) * J;
  for (int x = lane; x < J; x += 64) {
    int32_t run = sl[x];
    for (int v = 0; v < w; ++v) run += int32_t(s_wcnt[v][x]);
    s_run[w][x] = run;
  }
  // s_run[w] is this wave's own row: its writes above and the reads below
  // come from the same wave, in order
  const int32_t* Rsub = R + s.base;
  int32_t* orow = order + s.i * p.M_max;
  const uint64_t below = lanemask_lt();
  for (int u0 = 0; u0 < kPfQuarter / 64; u0 += kPfBatch) {
    uint32_t m[kPfBatch];
    int32_t k[kPfBatch];
#pragma unroll
    for (int u = 0; u < kPfBatch; ++u) {
      const int64_t j = j0 + (u0 + u) * 64 + lane;
      m[u] = j < s.len ? clamp_code(s_code[j], J) : 0u;
      k[u] = m[u] ? Rsub[j] : 0;
    }
#pragma unroll
    for (int u = 0; u < kPfBatch; ++u) {
      uint64_t act = __ballot(m[u] != 0);
      while (act) {
        const int lead = __builtin_ctzll(act);
        const uint32_t tc = __builtin_amdgcn_readlane(m[u], lead);
        const uint64_t same = __ballot(m[u] == tc);
        const int32_t run = s_run[w][tc - 1];
        if (m[u] == tc) orow[run + __popcll(same & below)] = k[u];
        if (lane == lead) s_run[w][tc - 1] = run + __popcll(same);
        act &= ~same;
      }
    }
  }
  // padding after the last queue: this sub-chunk's range of the row, and
  // the row's tail past its last read for the row's last sub-chunk
  const int64_t T = tot[s.i];
  const int64_t q0 = s.base - s.i * p.M_max;
  for (int64_t q = (T > q0 ? T : q0) + threadIdx.x; q < q0 + s.len; q += 64 * kPfWaves)
    orow[q] = -1;
  if (s.c == int64_t(nch) - 1) {
    const int64_t Mi = int64_t(p.E) * s.Li;
    for (int64_t q = (T > Mi ? T : Mi) + threadIdx.x; q < p.M_max; q += 64 * kPfWaves) orow[q] = -1;
  }
}

// -------------------------------------------------------------- staging --
constexpr int kStGroup = NOPFS_ST_GROUP;
constexpr int kSumThreads = 1024;
constexpr int kHalf = kSC / 2;                // positions per LDS pass of st_sum
constexpr int kSumPer = kHalf / kSumThreads;  // 8 positions per thread
constexpr int kSumEnt = kSC / kSumThreads;    // 16 entries per thread

static_assert(kSumPer * kSumThreads == kHalf && kSumEnt * kSumThreads == kSC, "st_sum shape");

__device__ __forceinline__ int sum_slot(int p) { return p + (p >> 3); }

constexpr int kStTileThreads = 1024;

__global__ void __launch_bounds__(kStTileThreads)
st_tile(SegParams p, const uint32_t* __restrict__ Pk, const uint16_t* __restrict__ OT,
        const int64_t* __restrict__ sizes, int64_t* __restrict__ zP,
        uint32_t ntiles) {
  __shared__ int64_t sz[kWin];
  // group-major tiles, like the other tile passes: a group's consecutive
  // windows run together on one XCD, so the partial lines their runs write
  // are completed there (window-major order, which shares a window's sizes
  // between groups instead, measured 1.7x slower)
  const uint32_t tile = xcd_logical(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int64_t g = tile / p.nbk;
  const uint32_t kb = tile - uint32_t(g) * p.nbk;
  const int64_t i0 = g * kStGroup;
  const int64_t gw = p.N - i0 < kStGroup ? p.N - i0 : kStGroup;  // workers in the group
  const int64_t k0 = int64_t(kb) << p.ws;
  const int64_t kend = k0 + (int64_t(1) << p.ws) < p.F ? k0 + (int64_t(1) << p.ws) : p.F;
  const int64_t runs = int64_t(p.E) * p.nsc;
  for (int64_t w0 = k0; w0 < kend; w0 += kWin) {
    const uint32_t wl = uint32_t(kend - w0 < kWin ? kend - w0 : kWin);
    const uint32_t xoff = uint32_t(w0 - k0);
    for (uint32_t x = threadIdx.x; x < wl; x += kStTileThreads) sz[x] = sizes[w0 + x];
    __syncthreads();
    // (worker, run) pairs of the group, spread over the threads
    for (int64_t pr = threadIdx.x; pr < gw * runs; pr += kStTileThreads) {
      const int64_t i = i0 + pr / runs;
      int64_t* zrow = zP + i * p.M_max;
      walk_runs(p, i, kb, Pk, OT, pr % runs, runs, [&](int64_t fb, uint32_t q, uint32_t v) {
        const uint32_t x = (v >> kScShift) - xoff;
        if (x < wl) zrow[fb + q] = sz[x];
      });
    }
    __syncthreads();
  }
}

// S[i*M_max + f] = sum of the sizes at the positions of f's sub-chunk up to
// and including f; ctot[i][c] = the sub-chunk's total.
__global__ void __launch_bounds__(kSumThreads)
st_sum(SegParams p, const uint32_t* __restrict__ Pk, const int64_t* __restrict__ zP, uint32_t nch,
       int64_t* __restrict__ S, int64_t* __restrict__ ctot) {
  __shared__ int64_t sv[kHalf + kHalf / kSumPer];
  __shared__ uint64_t tmp[65];
  const SubChunk s = sub_chunk(p, nch, blockIdx.x);
  uint32_t jj[kSumEnt];
  int64_t vv[kSumEnt];
#pragma unroll
  for (int u = 0; u < kSumEnt; ++u) {
    const int64_t q = int64_t(u) * kSumThreads + threadIdx.x;
    jj[u] = q < s.len ? (Pk[s.base + q] & kJMask) : 0xFFFFFFFFu;
    vv[u] = q < s.len ? zP[s.base + q] : 0;
  }
  uint64_t carry = 0;
  for (int64_t j0 = 0; j0 < s.len; j0 += kHalf) {
    const uint32_t hl = uint32_t(s.len - j0 < kHalf ? s.len - j0 : kHalf);
#pragma unroll
    for (int u = 0; u < kSumEnt; ++u) {
      const uint32_t x = jj[u] - uint32_t(j0);
      if (x < hl) sv[sum_slot(int(x))] = vv[u];
    }
    __syncthreads();
    uint64_t v[kSumPer];
    uint64_t run = 0;
#pragma unroll
    for (int u = 0; u < kSumPer; ++u) {
      const int x = int(threadIdx.x) * kSumPer + u;
      run += x < int(hl) ? uint64_t(sv[sum_slot(x)]) : 0ull;
      v[u] = run;
    }
    uint64_t total;
    const uint64_t ex = block_exclusive_scan64(run, tmp, &total);
#pragma unroll
    for (int u = 0; u < kSumPer; ++u) {
      const int x = int(threadIdx.x) * kSumPer + u;
      if (x < int(hl)) sv[sum_slot(x)] = int64_t(carry + ex + v[u]);
    }
    __syncthreads();
    int64_t* dst = S + s.base + j0;
#pragma unroll
    for (int u = 0; u < kSumPer; ++u) {
      const int x = u * kSumThreads + int(threadIdx.x);
      if (x < int(hl)) dst[x] = sv[sum_slot(x)];
    }
    carry += total;
    __syncthreads();
  }
  if (threadIdx.x == 0) ctot[s.i * nch + s.c] = int64_t(carry);
}

// In place: ctot[i][c] becomes the sum of the sizes in the sub-chunks before c.
__global__ void __launch_bounds__(1024)
st_base(uint32_t nch, int64_t* __restrict__ ctot) {
  __shared__ uint64_t tmp[65];
  int64_t* row = ctot + int64_t(blockIdx.x) * nch;
  uint64_t carry = 0;
  for (uint32_t c0 = 0; c0 < nch; c0 += 1024) {
    const uint32_t c = c0 + threadIdx.x;
    const uint64_t v = c < nch ? uint64_t(row[c]) : 0ull;
    uint64_t total;
    const uint64_t ex = block_exclusive_scan64(v, tmp, &total);
    if (c < nch) row[c] = int64_t(carry + ex);
    carry += total;
  }
}

// Prefix sums along row i of R: at(x) = sum of the sizes at positions 0..x.
struct Prefix {
  const int64_t* S;     // row i of S (prefix sums local to each sub-chunk)
  const int64_t* base;  // row i of the sub-chunk bases
  int64_t Li;           // reads per epoch of worker i (> 0 whenever at() is used)
  double rinv;          // 1 / Li
  int64_t nsc;
  // sub-chunk of position x >= 0
  __device__ __forceinline__ int64_t chunk_of(int64_t x) const {
    // epoch of x: the double quotient is off by at most one
    int64_t e = int64_t(double(x) * rinv);
    if (e * Li > x) --e;
    else if ((e + 1) * Li <= x) ++e;
    return e * nsc + ((x - e * Li) >> kScShift);
  }
  __device__ __forceinline__ int64_t at(int64_t x) const {
    if (x < 0) return 0;
    return int64_t(uint64_t(base[chunk_of(x)]) + uint64_t(S[x]));
  }
  // smallest g in [-1, h] with at(g) >= target (h qualifies when target <= at(h))
  __device__ int64_t lower_bound(int64_t h, int64_t target) const {
    int64_t lo = -1, hi = h;
    while (lo < hi) {
      const int64_t mid = lo + ((hi - lo) >> 1);
      if (at(mid) >= target) hi = mid;
      else lo = mid + 1;
    }
    return lo;
  }
};

__device__ __forceinline__ Prefix row_prefix(const SegParams& p, int64_t i, uint32_t nch,
                                             const int64_t* S, const int64_t* base) {
  Prefix P;
  P.S = S + i * p.M_max;
  P.base = base + i * int64_t(nch);
  P.Li = seg_len(p, i);
  P.rinv = P.Li > 0 ? 1.0 / double(P.Li) : 0.0;
  P.nsc = p.nsc;
  return P;
}

__device__ __forceinline__ int64_t sub_sat(int64_t a, int64_t b) {
  // a - b without overflow (b >= 0)
  return a < INT64_MIN + b ? INT64_MIN : a - b;
}

constexpr int kStThreads = 256;
constexpr int kStPer = 16;
constexpr int64_t kStChunk = int64_t(kStThreads) * kStPer;  // 4096 positions
constexpr int kStParts = int(kSC / kStChunk);                // quarters of a sub-chunk
constexpr int kStPad = kStChunk + kStChunk / kStPer;        // LDS slots with one pad per 16
constexpr int kGCap = 5120;                                  // g values staged in LDS
constexpr int kSegMax = 8;  // sub-chunks a staged g range may span

static_assert(kStParts * kStChunk == kSC, "staging quarters");

__device__ __forceinline__ int lds_slot(int p) { return p + (p >> 4); }

// Block b of the fill covers quarter `part` of sub-chunk c of worker i:
// positions [h0, h0 + hl) of row i (hl may be 0).
struct FillPart {
  int64_t i, c, part, Li, h0, hl;
};

__device__ __forceinline__ FillPart fill_part(const SegParams& p, uint32_t nch, int64_t b) {
  FillPart f;
  const int64_t per = int64_t(nch) * kStParts;
  f.i = b / per;
  const int64_t rem = b - f.i * per;
  f.c = rem / kStParts;
  f.part = rem - f.c * kStParts;
  f.Li = seg_len(p, f.i);
  const int64_t e = f.c / p.nsc, sc = f.c - e * p.nsc;
  const int64_t len = sub_len(f.Li, sc) - f.part * kStChunk;
  f.hl = len < 0 ? 0 : (len > kStChunk ? kStChunk : len);
  f.h0 = e * f.Li + sc * kSC + f.part * kStChunk;
  return f;
}

// bnd[b] = (g of the part's first position, g of its last position, the
// sub-chunk holding the first g (-1 when it is -1), 0).
__global__ void __launch_bounds__(256)
st_bounds(SegParams p, int64_t d0, uint32_t nch, int64_t nparts, const int64_t* __restrict__ S,
          const int64_t* __restrict__ base, int4* __restrict__ bnd) {
  const int64_t b = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (b >= nparts) return;
  const FillPart f = fill_part(p, nch, b);
  if (f.hl == 0) {
    bnd[b] = make_int4(0, -1, -1, 0);
    return;
  }
  const Prefix P = row_prefix(p, f.i, nch, S, base);
  const int64_t h1 = f.h0 + f.hl - 1;
  const int64_t glo = P.lower_bound(f.h0, sub_sat(P.at(f.h0), d0));
  const int64_t ghi = P.lower_bound(h1, sub_sat(P.at(h1), d0));
  bnd[b] = make_int4(int32_t(glo), int32_t(ghi), int32_t(glo >= 0 ? P.chunk_of(glo) : -1), 0);
}

__global__ void __launch_bounds__(kStThreads)
st_fill(SegParams p, int64_t d0, uint32_t nch, int64_t nparts, const int64_t* __restrict__ S,
        const int64_t* __restrict__ base, const int4* __restrict__ bnd, int32_t gcap,
        int32_t* __restrict__ fill) {
  // the staged g values, then (after a barrier) the results for the transpose
  __shared__ int64_t gS[kGCap];
  static_assert(kStPad * sizeof(int32_t) <= sizeof(gS), "result staging fits");
  int32_t* fo = reinterpret_cast<int32_t*>(gS);
  __shared__ int64_t seg_hi[kSegMax], seg_base[kSegMax];
  __shared__ int32_t s_staged;
  const int64_t b = xcd_logical(blockIdx.x, gridDim.x);
  if (b >= nparts) return;
  const FillPart f = fill_part(p, nch, b);
  int32_t* out = fill + f.i * p.M_max;
  if (f.c == int64_t(nch) - 1 && f.part == 0) {
    // the row's padding past its last read
    for (int64_t h = int64_t(p.E) * f.Li + threadIdx.x; h < p.M_max; h += kStThreads) out[h] = -1;
  }
  if (f.hl == 0) return;
  const int64_t* Srow = S + f.i * p.M_max;
  const int64_t* brow = base + f.i * int64_t(nch);
  // this thread's positions: prefix sums within sub-chunk c (loads first)
  const int64_t ht0 = int64_t(threadIdx.x) * kStPer;  // offset in the part
  int64_t sh[kStPer];
#pragma unroll
  for (int u = 0; u < kStPer; ++u) sh[u] = ht0 + u < f.hl ? Srow[f.h0 + ht0 + u] : 0;
  const int64_t hbase = brow[f.c];  // every position of the part is in sub-chunk c
  const int4 bb = bnd[b];
  const int64_t glo = bb.x, ghi = bb.y;
  const int64_t Lg = ghi - glo + 1;
  // sub-chunks c0, c0 + 1, ... spanned by [max(glo, 0), ghi], one per lane
  // of the first wave: the end position and base of each
  const int64_t c0 = bb.z >= 0 ? bb.z : 0;
  const bool fits = Lg >= 1 && Lg <= gcap;  // uniform
  if (threadIdx.x < 64) {
    bool need = false, covered = false;
    if (fits && threadIdx.x < kSegMax && ghi >= 0) {
      const int64_t c = c0 + threadIdx.x;
      if (c < int64_t(nch)) {
        const int64_t e = c / p.nsc, sc = c - e * p.nsc;
        const int64_t lo = e * f.Li + sc * kSC;
        const int64_t hi = lo + sub_len(f.Li, sc);
        need = lo <= ghi;
        covered = need && hi > ghi;
        seg_hi[threadIdx.x] = hi;
        seg_base[threadIdx.x] = need ? brow[c] : 0;
      }
    }
    const uint64_t cov = __ballot(covered);
    if (threadIdx.x == 0) s_staged = fits && (ghi < 0 || cov != 0);
  }
  __syncthreads();
  const bool staged = s_staged;  // uniform over the workgroup
  if (staged) {
    for (int64_t x = threadIdx.x; x < Lg; x += kStThreads) {
      const int64_t g = glo + x;
      int64_t v = 0;
      if (g >= 0) {
        int k = 0;
        while (g >= seg_hi[k]) ++k;  // the covering sub-chunk ends past ghi
        v = int64_t(uint64_t(seg_base[k]) + uint64_t(Srow[g]));
      }
      gS[x] = v;
    }
  }
  __syncthreads();
  const Prefix P = row_prefix(p, f.i, nch, S, base);
  int32_t res[kStPer];
  int64_t x = 0;
  bool started = false;
#pragma unroll
  for (int u = 0; u < kStPer; ++u) {
    const int64_t h = f.h0 + ht0 + u;
    res[u] = -1;
    if (ht0 + u < f.hl) {
      const int64_t target = sub_sat(int64_t(uint64_t(hbase) + uint64_t(sh[u])), d0);
      int64_t g;
      if (staged) {
        if (!started) {
          int64_t lo = 0, hi = Lg;
          while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (gS[mid] >= target) hi = mid;
            else lo = mid + 1;
          }
          x = lo < Lg ? lo : Lg - 1;
          started = true;
        }
        while (x < Lg - 1 && gS[x] < target) ++x;
        g = glo + x;
      } else {
        // g range too wide for LDS (or not monotone): search the row itself
        if (!started) {
          x = P.lower_bound(h, target);
          started = true;
        }
        while (x < h && P.at(x) < target) ++x;
        g = x;
      }
      const int64_t fv = g + 1 < h ? g + 1 : h;
      res[u] = int32_t(fv > 0 ? fv : 0);
    }
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kStPer; ++u) fo[lds_slot(threadIdx.x * kStPer + u)] = res[u];
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kStPer; ++u) {
    const int q = u * kStThreads + threadIdx.x;
    if (q < f.hl) out[f.h0 + q] = fo[lds_slot(q)];
  }
}

int prefetch_impl(const nopfs_job* job, const int32_t* R, const int8_t* tier, int32_t J,
                  int32_t* order, int64_t* qlen, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (!tier || !qlen) return fail(NOPFS_EINVAL, "tier and qlen must be non-NULL");
  if (s.M_max > 0 && (!R || !order)) return fail(NOPFS_EINVAL, "R and order must be non-NULL");
  if (J < 1) return fail(NOPFS_EINVAL, "J must be >= 1");
  if (J > 127) return fail(NOPFS_ERANGE, "J must be <= 127");
  const SegParams p = seg_params(s, kSchedWs);
  const uint32_t nch = uint32_t(s.E * p.nsc);  // sub-chunks per worker
  const int64_t nblk = s.N * int64_t(nch);
  const int64_t ntiles = s.N * int64_t(p.nbk);
  if (nblk >= (int64_t(1) << 31) || ntiles >= (int64_t(1) << 31))
    return fail(NOPFS_ERANGE, "job too large for one launch");
  Scratch scr(st);
  int64_t* tot;
  int32_t* cnt;
  if ((rc = scr.alloc_n(&tot, size_t(s.N)))) return rc;
  if ((rc = scr.alloc_n(&cnt, size_t(nblk) * size_t(J)))) return rc;
  if (s.M_max == 0)  // no reads at all: empty queues
    return launch("pf_scan", pf_scan, dim3(uint32_t(s.N)), dim3(1024), 0, st, J, 0u, cnt, qlen,
                  tot);
  uint32_t* Pk;
  uint16_t* OT;
  uint8_t* code;
  if ((rc = run_partition(p, R, scr, &Pk, &OT, st))) return rc;
  if ((rc = scr.alloc_n(&code, size_t(s.N * s.M_max)))) return rc;
  if ((rc = launch("pf_tile", pf_tile, dim3(xcd_padded(uint32_t(ntiles))), dim3(kTileThreads), 0,
                   st, p, (const uint32_t*)Pk, (const uint16_t*)OT, tier, J, code,
                   uint32_t(ntiles))))
    return rc;
  if ((rc = launch("pf_count", pf_count, dim3(uint32_t(nblk)), dim3(256), 0, st, p, J,
                   (const uint8_t*)code, nch, cnt)))
    return rc;
  if ((rc = launch("pf_scan", pf_scan, dim3(uint32_t(s.N)), dim3(1024), 0, st, J, nch, cnt, qlen,
                   tot)))
    return rc;
  return launch("pf_write", pf_write, dim3(uint32_t(nblk)), dim3(64 * kPfWaves), 0, st, p, J,
                (const uint32_t*)Pk, (const uint8_t*)code, R, nch, (const int32_t*)cnt,
                (const int64_t*)tot, order);
}

int staging_impl(const nopfs_job* job, const int32_t* R, const int64_t* sizes, int64_t d0,
                 int32_t* fill, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (!sizes) return fail(NOPFS_EINVAL, "sizes must be non-NULL");
  if (s.M_max > 0 && (!R || !fill)) return fail(NOPFS_EINVAL, "R and fill must be non-NULL");
  if (d0 < 0) return fail(NOPFS_EINVAL, "d0 must be >= 0");
  if (s.M_max == 0) return NOPFS_OK;
  const SegParams p = seg_params(s, kSchedWs);
  const uint32_t nch = uint32_t(s.E * p.nsc);  // sub-chunks per worker
  const uint32_t ngroups = uint32_t(ceil_div(s.N, kStGroup));
  const int64_t nblk = s.N * int64_t(nch);
  const int64_t nparts = nblk * kStParts;
  const int64_t ntiles = int64_t(p.nbk) * ngroups;
  if (nparts >= (int64_t(1) << 31) || ntiles >= (int64_t(1) << 31))
    return fail(NOPFS_ERANGE, "job too large for one launch");
  Scratch scr(st);
  uint32_t* Pk;
  uint16_t* OT;
  int64_t *zP, *S, *ctot;
  int4* bnd;
  if ((rc = run_partition(p, R, scr, &Pk, &OT, st))) return rc;
  if ((rc = scr.alloc_n(&zP, size_t(s.N * s.M_max)))) return rc;
  if ((rc = scr.alloc_n(&S, size_t(s.N * s.M_max)))) return rc;
  if ((rc = scr.alloc_n(&ctot, size_t(nblk)))) return rc;
  if ((rc = scr.alloc_n(&bnd, size_t(nparts)))) return rc;
  if ((rc = launch("st_tile", st_tile, dim3(xcd_padded(uint32_t(ntiles))), dim3(kStTileThreads), 0,
                   st, p, (const uint32_t*)Pk, (const uint16_t*)OT, sizes, zP,
                   uint32_t(ntiles))))
    return rc;
  if ((rc = launch("st_sum", st_sum, dim3(uint32_t(nblk)), dim3(kSumThreads), 0, st, p,
                   (const uint32_t*)Pk, (const int64_t*)zP, nch, S, ctot)))
    return rc;
  if ((rc = launch("st_base", st_base, dim3(uint32_t(s.N)), dim3(1024), 0, st, nch, ctot))) return rc;
  if ((rc = launch("st_bounds", st_bounds, dim3(uint32_t(ceil_div(nparts, 256))), dim3(256), 0, st,
                   p, d0, nch, nparts, (const int64_t*)S, (const int64_t*)ctot, bnd)))
    return rc;
  const int32_t gcap = (debug_value(4) > 0 && debug_value(4) < kGCap) ? int32_t(debug_value(4)) : kGCap;
  return launch("st_fill", st_fill, dim3(xcd_padded(uint32_t(nparts))), dim3(kStThreads), 0, st, p,
                d0, nch, nparts, (const int64_t*)S, (const int64_t*)ctot, (const int4*)bnd, gcap,
                fill);
}

}  // namespace
}  // namespace nopfs

extern "C" int nopfs_prefetch_order(const nopfs_job* job, const int32_t* R, const int8_t* tier,
                                    int32_t J, int32_t* order, int64_t* qlen, void* hip_stream) {
  try {
    return nopfs::prefetch_impl(job, R, tier, J, order, qlen, static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}

extern "C" int nopfs_staging_schedule(const nopfs_job* job, const int32_t* R, const int64_t* sizes,
                                      int64_t d0, int32_t* fill, void* hip_stream) {
  try {
    return nopfs::staging_impl(job, R, sizes, d0, fill, static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}
