// nopfs_access_stats and nopfs_reuse_next.
//
// Both read the stream R (worker-major, in stream order) and need it grouped
// by sample: the access frequency of section 3.1 is a per-(worker, sample)
// count, and the next use of section 3 (Belady) links reads of one sample.
// The grouping is a per-worker partition of R by sample range:
//
//   seg_partition -- for every sub-chunk of 2^14 consecutive reads of one
//                    (worker, epoch) segment, counting-sort the reads by
//                    sample window kb = k >> ws into LDS and write them back
//                    in place of order, packed as (k - kb*W) << 14 | j, with
//                    the window offsets of the sub-chunk (uint16).
//   stats_tile    -- one workgroup per (worker, window of W samples): count
//                    (bytes) and first read (int32) privatised in LDS,
//                    updated with LDS atomics, then written as dense row
//                    segments of count[N][F] and first[N][F].
//   next_tile     -- one workgroup per (worker, window): the window's reads
//                    are bucketed by sample in LDS, each bucket ordered by
//                    position, and every read gets the position of the next
//                    read of its bucket (the "segmented sort plus shift").
//                    The results go to a scratch array laid out like the
//                    partitioned reads.
//   next_unpartition -- per sub-chunk, scatter those results back to stream
//                    order through LDS and write next[N][M_max].
// A next_tile window whose reads do not fit in LDS takes an epoch-serial path
// (walk the epochs backwards, remembering the last position per sample).
#include <limits.h>

#include <new>

#include "common.hpp"

namespace nopfs {
namespace {

constexpr int kScShift = 14;
constexpr int kSC = 1 << kScShift;  // reads per sub-chunk
constexpr uint32_t kJMask = kSC - 1;
constexpr uint32_t kMaxWindows = 8192;  // sample windows per worker
constexpr int kThreads = 256;
constexpr int kStatsWin = 16384;        // samples held in LDS by stats_tile
constexpr int kNextWin = 4096;          // samples per next_tile window (fast path)
constexpr int kNextEnt = 4096;          // reads per next_tile window (fast path)
constexpr int kSlowWin = 16384;         // samples per pass of the epoch-serial path

struct SegParams {
  int64_t F, N, B, L, M_max;
  int32_t E, drop_last;
  int32_t ws;     // log2 of the window width W
  uint32_t nbk;   // windows per worker: ceil(F / W)
  int32_t nsc;    // sub-chunks per (worker, epoch) segment
  int32_t ent_cap;  // next_tile fast-path capacity (reads)
};

__device__ __forceinline__ int64_t seg_len(const SegParams& p, int64_t i) {
  return p.drop_last ? p.L : epoch_len(p.F, p.N, p.B, 0, i);
}

__device__ __forceinline__ int64_t orow(const SegParams& p, int64_t i, int64_t e, int64_t sc) {
  return ((i * p.E + e) * p.nsc + sc) * int64_t(p.nbk + 1);
}

// -- partition ----------------------------------------------------------------
__global__ void __launch_bounds__(kThreads)
seg_partition(SegParams p, const int32_t* __restrict__ R, uint32_t* __restrict__ Pk,
              uint16_t* __restrict__ O) {
  extern __shared__ uint32_t sm[];
  __shared__ uint32_t tmp[65];
  const uint32_t nbk = p.nbk;
  uint32_t* hist = sm;
  uint32_t* stage = sm + ((nbk + 4) & ~3u);
  const int64_t wg = blockIdx.x;
  const int64_t per_worker = int64_t(p.E) * p.nsc;
  const int64_t i = wg / per_worker;
  const int64_t rem = wg - i * per_worker;
  const int64_t e = rem / p.nsc, sc = rem - e * p.nsc;
  const int64_t Li = seg_len(p, i);
  int64_t len64 = Li - sc * kSC;
  len64 = len64 < 0 ? 0 : (len64 > kSC ? kSC : len64);
  const uint32_t len = uint32_t(len64);
  const int64_t base = i * p.M_max + e * Li + sc * kSC;
  const uint32_t W = 1u << p.ws;

  for (uint32_t b = threadIdx.x; b <= nbk; b += kThreads) hist[b] = 0;
  __syncthreads();
  constexpr int kPer = kSC / kThreads;
  int32_t kk[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const uint32_t q = uint32_t(r * kThreads) + threadIdx.x;
    kk[r] = q < len ? R[base + q] : -1;
    // entries outside [0, F) break the precondition; keep them in bounds
    if (q < len && uint64_t(uint32_t(kk[r])) >= uint64_t(p.F)) kk[r] = 0;
    if (q < len) atomicAdd(&hist[uint32_t(kk[r]) >> p.ws], 1u);
  }
  __syncthreads();
  uint16_t* o = O + orow(p, i, e, sc);
  uint32_t carry = 0;
  for (uint32_t b0 = 0; b0 < nbk; b0 += kThreads) {
    const uint32_t b = b0 + threadIdx.x;
    const uint32_t v = b < nbk ? hist[b] : 0u;
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(v, tmp, &total);
    if (b < nbk) {
      hist[b] = carry + ex;
      o[b] = uint16_t(carry + ex);
    }
    carry += total;
  }
  if (threadIdx.x == 0) o[nbk] = uint16_t(len);
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const uint32_t q = uint32_t(r * kThreads) + threadIdx.x;
    if (q < len) {
      const uint32_t k = uint32_t(kk[r]);
      const uint32_t slot = atomicAdd(&hist[k >> p.ws], 1u);
      stage[slot] = ((k & (W - 1)) << kScShift) | q;
    }
  }
  __syncthreads();
  for (uint32_t q = threadIdx.x; q < len; q += kThreads) Pk[base + q] = stage[q];
}

// Iterates over every read of window kb of worker i, in batches of runs (one
// run = the window's slice of one sub-chunk). fn(pos_in_row, f_base, v)
// receives the read's position in the partitioned row, the stream position
// of its sub-chunk start, and the packed read.
struct RunTable {
  uint32_t pref[kThreads + 1];
  int64_t start[kThreads];  // position in the row of the run's first read
  int64_t fbase[kThreads];  // stream position of the sub-chunk start
  uint32_t tmp[65];
};

template <typename Fn>
__device__ __forceinline__ void for_each_read(const SegParams& p, int64_t i, uint32_t kb,
                                              const uint16_t* __restrict__ O, RunTable& rt,
                                              int64_t e_lo, int64_t e_hi, Fn fn) {
  const int64_t Li = seg_len(p, i);
  const int64_t runs = (e_hi - e_lo) * p.nsc;
  for (int64_t r0 = 0; r0 < runs; r0 += kThreads) {
    const int64_t r = r0 + threadIdx.x;
    uint32_t len = 0;
    if (r < runs) {
      const int64_t e = e_lo + r / p.nsc, sc = r % p.nsc;
      const uint16_t* o = O + orow(p, i, e, sc);
      const uint32_t a = o[kb], b = o[kb + 1];
      len = b - a;
      rt.fbase[threadIdx.x] = e * Li + sc * kSC;
      rt.start[threadIdx.x] = e * Li + sc * kSC + a;
    }
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(len, rt.tmp, &total);
    rt.pref[threadIdx.x] = ex;
    if (threadIdx.x == 0) rt.pref[kThreads] = total;
    __syncthreads();
    const int nr = int(runs - r0 < kThreads ? runs - r0 : kThreads);
    for (uint32_t t = threadIdx.x; t < total; t += kThreads) {
      int lo = 0, hi = nr - 1;  // last run with pref <= t
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (rt.pref[mid] <= t) lo = mid; else hi = mid - 1;
      }
      const int64_t pos = rt.start[lo] + (t - rt.pref[lo]);
      fn(pos, rt.fbase[lo], t + 0u);
    }
    __syncthreads();
  }
}

// -- stats --------------------------------------------------------------------
__global__ void __launch_bounds__(kThreads)
stats_tile(SegParams p, const uint32_t* __restrict__ Pk, const uint16_t* __restrict__ O,
           uint8_t* __restrict__ count, int32_t* __restrict__ first, uint32_t ntiles) {
  extern __shared__ uint32_t sm[];
  __shared__ RunTable rt;
  uint32_t* cw = sm;                                   // kStatsWin / 4 words of byte counters
  int32_t* fi = reinterpret_cast<int32_t*>(sm + kStatsWin / 4);
  const uint32_t tile = xcd_logical(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int64_t i = tile / p.nbk;
  const uint32_t kb = tile - uint32_t(i) * p.nbk;
  const int64_t W = int64_t(1) << p.ws;
  const int64_t k0 = int64_t(kb) * W;
  const int64_t kend = k0 + W < p.F ? k0 + W : p.F;
  const uint32_t* prow = Pk + i * p.M_max;
  for (int64_t w0 = k0; w0 < kend; w0 += kStatsWin) {
    const uint32_t wlen = uint32_t(kend - w0 < kStatsWin ? kend - w0 : kStatsWin);
    for (uint32_t x = threadIdx.x; x < (wlen + 3) / 4; x += kThreads) cw[x] = 0;
    for (uint32_t x = threadIdx.x; x < wlen; x += kThreads) fi[x] = INT_MAX;
    __syncthreads();
    const uint32_t xoff = uint32_t(w0 - k0);
    for_each_read(p, i, kb, O, rt, 0, p.E, [&](int64_t pos, int64_t fbase, uint32_t) {
      const uint32_t v = prow[pos];
      const uint32_t x = (v >> kScShift) - xoff;
      if (x < wlen) {
        atomicAdd(&cw[x >> 2], 1u << ((x & 3u) * 8u));
        atomicMin(&fi[x], int32_t(fbase + (v & kJMask)));
      }
    });
    __syncthreads();
    uint8_t* crow = count + i * p.F + w0;
    int32_t* frow = first + i * p.F + w0;
    for (uint32_t x = threadIdx.x; x < wlen; x += kThreads) {
      const uint32_t c = (cw[x >> 2] >> ((x & 3u) * 8u)) & 0xFFu;
      crow[x] = uint8_t(c);
      frow[x] = c ? fi[x] : -1;
    }
    __syncthreads();
  }
}

// -- next ---------------------------------------------------------------------
struct NextSmem {
  uint32_t start[kNextWin];
  uint32_t cur[kNextWin];
  int32_t f[kNextEnt];
  int32_t pos[kNextEnt];
  uint16_t kl[kNextEnt];
  uint16_t ord[kNextEnt];
};

__device__ void next_tile_slow(const SegParams& p, int64_t i, uint32_t kb, const uint32_t* prow,
                               const uint16_t* O, int32_t* nrow, RunTable& rt, int32_t* last) {
  const int64_t W = int64_t(1) << p.ws;
  const int64_t k0 = int64_t(kb) * W;
  const int64_t kend = k0 + W < p.F ? k0 + W : p.F;
  for (int64_t w0 = k0; w0 < kend; w0 += kSlowWin) {
    const uint32_t wlen = uint32_t(kend - w0 < kSlowWin ? kend - w0 : kSlowWin);
    const uint32_t xoff = uint32_t(w0 - k0);
    for (uint32_t x = threadIdx.x; x < wlen; x += kThreads) last[x] = -1;
    __syncthreads();
    for (int64_t e = p.E - 1; e >= 0; --e) {
      // reads of one epoch are distinct samples: no two threads share a slot
      for_each_read(p, i, kb, O, rt, e, e + 1, [&](int64_t pos, int64_t fbase, uint32_t) {
        const uint32_t v = prow[pos];
        const uint32_t x = (v >> kScShift) - xoff;
        if (x < wlen) {
          nrow[pos] = last[x];
          last[x] = int32_t(fbase + (v & kJMask));
        }
      });
      __syncthreads();
    }
  }
}

__global__ void __launch_bounds__(kThreads)
next_tile(SegParams p, const uint32_t* __restrict__ Pk, const uint16_t* __restrict__ O,
          int32_t* __restrict__ nextP, uint32_t ntiles) {
  extern __shared__ uint32_t sm[];
  __shared__ RunTable rt;
  __shared__ uint32_t s_total;
  const uint32_t tile = xcd_logical(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int64_t i = tile / p.nbk;
  const uint32_t kb = tile - uint32_t(i) * p.nbk;
  const uint32_t* prow = Pk + i * p.M_max;
  int32_t* nrow = nextP + i * p.M_max;
  const uint32_t W = 1u << p.ws;

  // number of reads in the window
  if (threadIdx.x == 0) s_total = 0;
  __syncthreads();
  {
    uint32_t mine = 0;
    const int64_t runs = int64_t(p.E) * p.nsc;
    for (int64_t r = threadIdx.x; r < runs; r += kThreads) {
      const uint16_t* o = O + orow(p, i, r / p.nsc, r % p.nsc);
      mine += uint32_t(o[kb + 1] - o[kb]);
    }
    atomicAdd(&s_total, mine);
  }
  __syncthreads();
  const uint32_t total = s_total;
  if (total == 0) return;
  if (W > uint32_t(kNextWin) || total > uint32_t(p.ent_cap)) {
    next_tile_slow(p, i, kb, prow, O, nrow, rt, reinterpret_cast<int32_t*>(sm));
    return;
  }
  NextSmem& s = *reinterpret_cast<NextSmem*>(sm);
  for (uint32_t x = threadIdx.x; x < W; x += kThreads) s.start[x] = 0;
  __syncthreads();
  // gather the window's reads; the flat index runs over (epoch, sub-chunk)
  uint32_t base = 0;
  {
    const int64_t runs = int64_t(p.E) * p.nsc;
    const int64_t Li = seg_len(p, i);
    for (int64_t r0 = 0; r0 < runs; r0 += kThreads) {
      const int64_t r = r0 + threadIdx.x;
      uint32_t len = 0;
      if (r < runs) {
        const int64_t e = r / p.nsc, sc = r % p.nsc;
        const uint16_t* o = O + orow(p, i, e, sc);
        const uint32_t a = o[kb], b = o[kb + 1];
        len = b - a;
        rt.fbase[threadIdx.x] = e * Li + sc * kSC;
        rt.start[threadIdx.x] = e * Li + sc * kSC + a;
      }
      uint32_t tot;
      const uint32_t ex = block_exclusive_scan(len, rt.tmp, &tot);
      rt.pref[threadIdx.x] = ex;
      __syncthreads();
      const int nr = int(runs - r0 < kThreads ? runs - r0 : kThreads);
      for (uint32_t t = threadIdx.x; t < tot; t += kThreads) {
        int lo = 0, hi = nr - 1;
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (rt.pref[mid] <= t) lo = mid; else hi = mid - 1;
        }
        const int64_t pos = rt.start[lo] + (t - rt.pref[lo]);
        const uint32_t v = prow[pos];
        const uint32_t idx = base + t;
        const uint32_t x = v >> kScShift;
        s.kl[idx] = uint16_t(x);
        s.f[idx] = int32_t(rt.fbase[lo] + (v & kJMask));
        s.pos[idx] = int32_t(pos);
        atomicAdd(&s.start[x], 1u);
      }
      base += tot;
      __syncthreads();
    }
  }
  // bucket starts
  {
    uint32_t carry = 0;
    for (uint32_t x0 = 0; x0 < W; x0 += kThreads) {
      const uint32_t x = x0 + threadIdx.x;
      const uint32_t v = x < W ? s.start[x] : 0u;
      uint32_t tot;
      const uint32_t ex = block_exclusive_scan(v, rt.tmp, &tot);
      if (x < W) {
        s.start[x] = carry + ex;
        s.cur[x] = carry + ex;
      }
      carry += tot;
    }
  }
  __syncthreads();
  for (uint32_t idx = threadIdx.x; idx < total; idx += kThreads) {
    const uint32_t slot = atomicAdd(&s.cur[s.kl[idx]], 1u);
    s.ord[slot] = uint16_t(idx);
  }
  __syncthreads();
  // order each bucket by stream position (buckets are short)
  for (uint32_t x = threadIdx.x; x < W; x += kThreads) {
    const uint32_t a = s.start[x], b = s.cur[x];
    for (uint32_t u = a + 1; u < b; ++u) {
      const uint16_t v = s.ord[u];
      const int32_t fv = s.f[v];
      uint32_t c = u;
      while (c > a && s.f[s.ord[c - 1]] > fv) {
        s.ord[c] = s.ord[c - 1];
        --c;
      }
      s.ord[c] = v;
    }
  }
  __syncthreads();
  for (uint32_t u = threadIdx.x; u < total; u += kThreads) {
    const uint32_t idx = s.ord[u];
    const uint32_t end = s.cur[s.kl[idx]];
    nrow[s.pos[idx]] = (u + 1 < end) ? s.f[s.ord[u + 1]] : -1;
  }
}

__global__ void __launch_bounds__(kThreads)
next_unpartition(SegParams p, const uint32_t* __restrict__ Pk, const int32_t* __restrict__ nextP,
                 int32_t* __restrict__ next) {
  __shared__ int32_t stage[kSC];
  const int64_t wg = blockIdx.x;
  const int64_t per_worker = int64_t(p.E) * p.nsc;
  const int64_t i = wg / per_worker;
  const int64_t rem = wg - i * per_worker;
  const int64_t e = rem / p.nsc, sc = rem - e * p.nsc;
  const int64_t Li = seg_len(p, i);
  int64_t len64 = Li - sc * kSC;
  len64 = len64 < 0 ? 0 : (len64 > kSC ? kSC : len64);
  const uint32_t len = uint32_t(len64);
  if (len == 0) return;
  const int64_t base = i * p.M_max + e * Li + sc * kSC;
  for (uint32_t q = threadIdx.x; q < len; q += kThreads) stage[Pk[base + q] & kJMask] = nextP[base + q];
  __syncthreads();
  for (uint32_t q = threadIdx.x; q < len; q += kThreads) next[base + q] = stage[q];
}

__global__ void pad_rows(SegParams p, int32_t* __restrict__ out) {
  const int64_t i = blockIdx.x;
  const int64_t Mi = int64_t(p.E) * seg_len(p, i);
  for (int64_t f = Mi + threadIdx.x; f < p.M_max; f += blockDim.x) out[i * p.M_max + f] = -1;
}

__global__ void fill_stats_empty(int64_t n, uint8_t* __restrict__ count, int32_t* __restrict__ first) {
  int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (; t < n; t += stride) {
    count[t] = 0;
    first[t] = -1;
  }
}

int log2_ceil(int64_t v) {
  int b = 0;
  while ((int64_t(1) << b) < v) ++b;
  return b;
}

SegParams seg_params(const Shape& s, int ws) {
  SegParams p;
  p.F = s.F; p.N = s.N; p.B = s.B; p.L = s.L; p.M_max = s.M_max;
  p.E = int32_t(s.E);
  p.drop_last = s.drop_last;
  const int ws_min = log2_ceil(ceil_div(s.F, kMaxWindows));
  p.ws = ws < ws_min ? ws_min : ws;
  p.nbk = uint32_t(ceil_div(s.F, int64_t(1) << p.ws));
  p.nsc = int32_t(ceil_div(s.L, kSC));
  if (p.nsc < 1) p.nsc = 1;
  p.ent_cap = kNextEnt;
  return p;
}

size_t partition_smem(const SegParams& p) {
  return size_t(((p.nbk + 4) & ~3u) + kSC) * 4;
}

int run_partition(const SegParams& p, const int32_t* R, Scratch& scr, uint32_t** Pk,
                  uint16_t** O, hipStream_t st) {
  int rc;
  if ((rc = scr.alloc_n(Pk, size_t(p.N * p.M_max)))) return rc;
  if ((rc = scr.alloc_n(O, size_t(p.N * p.E * p.nsc) * (p.nbk + 1)))) return rc;
  const int64_t wgs = p.N * p.E * p.nsc;
  return launch("seg_partition", seg_partition, dim3(uint32_t(wgs)), dim3(kThreads),
                partition_smem(p), st, p, R, *Pk, *O);
}

}  // namespace

int stats_impl(const nopfs_job* job, const int32_t* R, uint8_t* count, int32_t* first,
               hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (!count || !first) return fail(NOPFS_EINVAL, "count and first must be non-NULL");
  if (!R && s.M_max > 0) return fail(NOPFS_EINVAL, "R is NULL");
  if (s.M_max == 0) {
    const int64_t n = s.N * s.F;
    int64_t blocks = ceil_div(n, 256 * 4);
    if (blocks > 65536) blocks = 65536;
    return launch("fill_stats_empty", fill_stats_empty, dim3(uint32_t(blocks)), dim3(256), 0, st, n,
                  count, first);
  }
  SegParams p = seg_params(s, 14);
  Scratch scr(st);
  uint32_t* Pk;
  uint16_t* O;
  if ((rc = run_partition(p, R, scr, &Pk, &O, st))) return rc;
  const uint32_t ntiles = uint32_t(s.N * p.nbk);
  const size_t smem = size_t(kStatsWin / 4 + kStatsWin) * 4;
  return launch("stats_tile", stats_tile, dim3(xcd_padded(ntiles)), dim3(kThreads), smem, st, p,
                (const uint32_t*)Pk, (const uint16_t*)O, count, first, ntiles);
}

int next_impl(const nopfs_job* job, const int32_t* R, int32_t* next, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (s.M_max == 0) return NOPFS_OK;  // R and next have no elements and may be NULL
  if (!R || !next) return fail(NOPFS_EINVAL, "R and next must be non-NULL");
  // window width: about half the fast-path capacity of reads per window
  const double reads_per_sample = double(s.M_max) / double(s.F);
  int ws = 0;
  while (ws < 12 && double(int64_t(1) << (ws + 1)) * reads_per_sample <= kNextEnt / 2) ++ws;
  SegParams p = seg_params(s, ws);
  if (debug_value(2) > 0 && debug_value(2) < kNextEnt) p.ent_cap = int32_t(debug_value(2));
  Scratch scr(st);
  uint32_t* Pk;
  uint16_t* O;
  int32_t* nextP;
  if ((rc = run_partition(p, R, scr, &Pk, &O, st))) return rc;
  if ((rc = scr.alloc_n(&nextP, size_t(s.N * s.M_max)))) return rc;
  const uint32_t ntiles = uint32_t(s.N * p.nbk);
  size_t smem = sizeof(NextSmem);
  if (smem < size_t(kSlowWin) * 4) smem = size_t(kSlowWin) * 4;
  if ((rc = launch("next_tile", next_tile, dim3(xcd_padded(ntiles)), dim3(kThreads), smem, st, p,
                   (const uint32_t*)Pk, (const uint16_t*)O, nextP, ntiles)))
    return rc;
  const int64_t wgs = s.N * s.E * p.nsc;
  if ((rc = launch("next_unpartition", next_unpartition, dim3(uint32_t(wgs)), dim3(kThreads), 0, st, p,
                   (const uint32_t*)Pk, (const int32_t*)nextP, next)))
    return rc;
  if (!s.drop_last && s.F % s.N != 0)
    if ((rc = launch("pad_rows", pad_rows, dim3(uint32_t(s.N)), dim3(64), 0, st, p, next))) return rc;
  return NOPFS_OK;
}

}  // namespace nopfs

extern "C" int nopfs_access_stats(const nopfs_job* job, const int32_t* R, uint8_t* count,
                                  int32_t* first, void* hip_stream) {
  try {
    return nopfs::stats_impl(job, R, count, first, static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}

extern "C" int nopfs_reuse_next(const nopfs_job* job, const int32_t* R, int32_t* next,
                                void* hip_stream) {
  try {
    return nopfs::next_impl(job, R, next, static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}
