// Per-worker partition of the stream R by sample window, shared by the
// passes that need R grouped by sample (access frequencies and first reads,
// next uses, prefetch marks, staging sizes).
//
// For every sub-chunk of 2^14 consecutive reads of one (worker, epoch)
// segment, seg_partition counting-sorts the reads by sample window
// kb = k >> ws and writes them back in place of order, packed as
// (k - kb*W) << 14 | j (j: the read's position in the sub-chunk), with the
// window offsets of the sub-chunk. A "run" is the reads of one window inside
// one sub-chunk; tile (i, kb) walks the runs of all sub-chunks of worker i.
#pragma once

#include "common.hpp"

namespace nopfs {

constexpr int kScShift = 14;
constexpr int kSC = 1 << kScShift;  // reads per sub-chunk
constexpr uint32_t kJMask = kSC - 1;
constexpr uint32_t kMaxWindows = 8192;  // sample windows per worker

struct SegParams {
  int64_t F, N, B, L, M_max;
  int32_t E, drop_last;
  int32_t ws;     // log2 of the window width W
  uint32_t nbk;   // windows per worker: ceil(F / W)
  int32_t nsc;    // sub-chunks per (worker, epoch) segment
  int32_t ent_cap;  // next_tile fast-path capacity (reads)
  int32_t emul;   // epochs per segment: 1, or E when a row is one segment (E = 1)
};

// Reads of one segment of worker i (an epoch, or the whole row when the
// epochs are folded into one segment).
__device__ __forceinline__ int64_t seg_len(const SegParams& p, int64_t i) {
  return int64_t(p.emul) * (p.drop_last ? p.L : epoch_len(p.F, p.N, p.B, 0, i));
}

__device__ __forceinline__ int64_t orow(const SegParams& p, int64_t i, int64_t e, int64_t sc) {
  return ((i * p.E + e) * p.nsc + sc) * int64_t(p.nbk + 1);
}

constexpr uint32_t kRunMap = 2048;  // reads whose run index is kept in LDS

template <int NT>
struct RunTable {
  uint32_t pref[NT + 1];
  int32_t start[NT];  // position in the row of the run's first read
  int32_t fbase[NT];  // stream position of the sub-chunk start
  uint32_t tmp[65];
  uint16_t run_of[kRunMap];  // run index of each read (when total <= kRunMap)
};

// Loads the run table of runs [r0, r0 + NT) of epochs [e_lo, e_hi)
// and returns the number of reads they hold. Leaves rt ready for lookups.
template <int NT>
__device__ __forceinline__ uint32_t load_runs(const SegParams& p, int64_t i, uint32_t kb,
                                              const uint16_t* __restrict__ OT, RunTable<NT>& rt,
                                              int64_t e_lo, int64_t runs, int64_t r0) {
  const int64_t Li = seg_len(p, i);
  const int64_t R = int64_t(p.E) * p.nsc;
  const uint16_t* oa = OT + (i * (p.nbk + 1) + kb) * R;  // window kb: run starts
  const uint16_t* ob = oa + R;                            // window kb+1: run ends
  const int64_t r = r0 + threadIdx.x;
  uint32_t len = 0;
  if (r < runs) {
    const int64_t run = e_lo * p.nsc + r;
    const uint32_t e = uint32_t(run) / uint32_t(p.nsc), sc = uint32_t(run) - e * uint32_t(p.nsc);
    const uint32_t a = oa[run], b = ob[run];
    len = b - a;
    rt.fbase[threadIdx.x] = int32_t(e * Li + sc * kSC);
    rt.start[threadIdx.x] = int32_t(e * Li + sc * kSC + a);
  }
  uint32_t total;
  const uint32_t ex = block_exclusive_scan<false>(len, rt.tmp, &total);  // closed below
  rt.pref[threadIdx.x] = ex;
  if (total <= kRunMap)
    for (uint32_t q = 0; q < len; ++q) rt.run_of[ex + q] = uint16_t(threadIdx.x);
  __syncthreads();
  return total;
}

// Calls fn(pos, f_base, v, idx) for the `total` reads of the loaded runs:
// pos is the read's position in the partitioned row, f_base the stream
// position of its sub-chunk start, v the packed read and idx its running
// index in (epoch, sub-chunk, position) order. Four loads per thread are in
// flight before any is consumed.
template <int NT, typename Fn>
__device__ __forceinline__ void consume_runs(const RunTable<NT>& rt, int nr, uint32_t total,
                                             const uint32_t* __restrict__ prow, uint32_t done,
                                             Fn fn) {
  for (uint32_t t0 = threadIdx.x; t0 < total; t0 += 4 * NT) {
    int64_t pos[4], fb[4];
    uint32_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t t = t0 + u * NT;
      pos[u] = -1;
      fb[u] = 0;
      if (t < total) {
        int lo;
        if (total <= kRunMap) {
          lo = rt.run_of[t];
        } else {
          lo = 0;  // last run with pref <= t
          int hi = nr - 1;
          while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (rt.pref[mid] <= t) lo = mid; else hi = mid - 1;
          }
        }
        pos[u] = rt.start[lo] + (t - rt.pref[lo]);
        fb[u] = rt.fbase[lo];
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = pos[u] >= 0 ? prow[pos[u]] : 0u;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (pos[u] >= 0) fn(pos[u], fb[u], v[u], done + t0 + u * NT);
  }
}

template <int NT, typename Fn>
__device__ __forceinline__ void for_each_read(const SegParams& p, int64_t i, uint32_t kb,
                                              const uint16_t* __restrict__ O,
                                              const uint32_t* __restrict__ prow, RunTable<NT>& rt,
                                              int64_t e_lo, int64_t e_hi, Fn fn) {
  const int64_t runs = (e_hi - e_lo) * p.nsc;
  uint32_t done = 0;
  for (int64_t r0 = 0; r0 < runs; r0 += NT) {
    const uint32_t total = load_runs(p, i, kb, O, rt, e_lo, runs, r0);
    const int nr = int(runs - r0 < NT ? runs - r0 : NT);
    consume_runs(rt, nr, total, prow, done, fn);
    done += total;
    __syncthreads();
  }
}

constexpr int kRunBatch = 8;  // loads in flight per run walk

// Reads of sub-chunk sc of an epoch segment of Li reads.
__device__ __forceinline__ int64_t sub_len(int64_t Li, int64_t sc) {
  const int64_t len = Li - sc * kSC;
  return len < 0 ? 0 : (len > kSC ? kSC : len);
}

// Calls fn(fb, q, v) for every read of runs r = r0, r0 + stride, ... of
// window kb of worker i: fb is the stream position of the run's sub-chunk,
// q the read's index in the sub-chunk's partitioned entries (its
// partitioned position is fb + q) and v the packed read.
template <typename Fn>
__device__ __forceinline__ void walk_runs(const SegParams& p, int64_t i, uint32_t kb,
                                          const uint32_t* __restrict__ Pk,
                                          const uint16_t* __restrict__ OT, int64_t r0,
                                          int64_t stride, Fn fn) {
  const int64_t Li = seg_len(p, i);
  const int64_t runs = int64_t(p.E) * p.nsc;
  const uint16_t* oa = OT + (i * (p.nbk + 1) + kb) * runs;  // run starts in window kb
  const uint16_t* ob = oa + runs;                            // run ends
  const uint32_t* prow = Pk + i * p.M_max;
  const uint32_t nsc = uint32_t(p.nsc);
  for (int64_t r = r0; r < runs; r += stride) {
    const uint32_t ra = oa[r], rb = ob[r];
    const uint32_t e = uint32_t(r) / nsc, sc = uint32_t(r) - e * nsc;
    const int64_t fb = int64_t(e) * Li + int64_t(sc) * kSC;
    const uint32_t* src = prow + fb;
    for (uint32_t q = ra; q < rb; q += kRunBatch) {
      uint32_t v[kRunBatch];
#pragma unroll
      for (int u = 0; u < kRunBatch; ++u) v[u] = q + u < rb ? src[q + u] : 0u;
#pragma unroll
      for (int u = 0; u < kRunBatch; ++u)
        if (q + u < rb) fn(fb, q + u, v[u]);
    }
  }
}

// Sub-chunk c = e * nsc + sc of worker i covers stream positions
// [e*Li + sc*kSC, + len).
struct SubChunk {
  int64_t i, c, Li, len, base;  // base: offset of its first position in [N][M_max]
};

__device__ __forceinline__ SubChunk sub_chunk(const SegParams& p, uint32_t nch, uint32_t blk) {
  SubChunk s;
  s.i = blk / nch;
  s.c = blk - s.i * nch;
  const int64_t e = s.c / p.nsc, sc = s.c - e * p.nsc;
  s.Li = seg_len(p, s.i);
  s.len = sub_len(s.Li, sc);
  s.base = s.i * p.M_max + e * s.Li + sc * kSC;
  return s;
}

// Partition parameters for windows of 2^ws samples (raised to keep at most
// kMaxWindows windows per worker).
SegParams seg_params(const Shape& s, int ws);

// Partitions R (device, [N][M_max]) into *Pk ([N][M_max], packed reads) and
// the window-major run offsets *OT, both allocated from scr.
int run_partition(const SegParams& p, const int32_t* R, Scratch& scr, uint32_t** Pk,
                  uint16_t** OT, hipStream_t st);

}  // namespace nopfs
