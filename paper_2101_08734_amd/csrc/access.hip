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

#include "partition.hpp"
#include "pipeline.hpp"

namespace nopfs {
namespace {

// Tuning knobs (measured on MI355X; see the benchmark notes). Every value
// gives identical results; only speed changes.
#ifndef NOPFS_STATS_THREADS
#define NOPFS_STATS_THREADS 512
#endif
#ifndef NOPFS_STATS_WS
#define NOPFS_STATS_WS 13
#endif
#ifndef NOPFS_NEXT_THREADS
#define NOPFS_NEXT_THREADS 512
#endif
#ifndef NOPFS_NEXT_ENT
#define NOPFS_NEXT_ENT 2048
#endif
#ifndef NOPFS_NEXT_WSMAX
#define NOPFS_NEXT_WSMAX 13
#endif

constexpr int kStatsThreads = NOPFS_STATS_THREADS;
constexpr int kNextThreads = NOPFS_NEXT_THREADS;
static_assert(kNextThreads >= 64 && kNextThreads % 64 == 0, "next_tile block size");
static_assert(kStatsThreads >= 64 && kStatsThreads % 64 == 0, "stats_tile block size");
static_assert((1 << NOPFS_STATS_WS) % (4 * NOPFS_STATS_THREADS) == 0, "stats_tile window per thread");
constexpr int kStatsWin = 1 << NOPFS_STATS_WS;  // samples held in LDS by stats_tile
constexpr int kNextEnt = NOPFS_NEXT_ENT;   // reads per next_tile window (fast path)
constexpr int kSlowWin = 8192;          // samples per pass of the epoch-serial path

// -- partition ----------------------------------------------------------------
constexpr int kPartThreads = 512;

__global__ void __launch_bounds__(kPartThreads)
seg_partition(SegParams p, const int32_t* __restrict__ R, uint32_t* __restrict__ Pk,
              uint16_t* __restrict__ O) {
  extern __shared__ uint32_t sm[];
  __shared__ uint32_t tmp[65];
  const uint32_t nbk = p.nbk;
  uint32_t* hist = sm;
  uint32_t* stage = sm + ((nbk + 4) & ~3u);
  const uint32_t wg = blockIdx.x;
  const uint32_t per_worker = uint32_t(p.E) * uint32_t(p.nsc);
  const uint32_t i = wg / per_worker;
  const uint32_t rem = wg - i * per_worker;
  const uint32_t e = rem / uint32_t(p.nsc), sc = rem - e * uint32_t(p.nsc);
  const int64_t Li = seg_len(p, i);
  int64_t len64 = Li - int64_t(sc) * kSC;
  len64 = len64 < 0 ? 0 : (len64 > kSC ? kSC : len64);
  const uint32_t len = uint32_t(len64);
  const int64_t base = int64_t(i) * p.M_max + int64_t(e) * Li + int64_t(sc) * kSC;
  const uint32_t W = 1u << p.ws;
  const uint32_t F = uint32_t(p.F);

  // the sub-chunk's reads are requested before the histogram is cleared
  // (unconditional loads; past the end they read the first entry)
  constexpr int kPer = kSC / kPartThreads;
  uint32_t kk[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const uint32_t q = uint32_t(r * kPartThreads) + threadIdx.x;
    kk[r] = uint32_t(R[base + (q < len ? q : 0u)]);
  }
  for (uint32_t b = threadIdx.x; b <= nbk; b += kPartThreads) hist[b] = 0;
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const uint32_t k = kk[r];
    kk[r] = k < F ? k : 0u;  // entries outside [0, F) break the precondition; keep them in bounds
  }
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const uint32_t q = uint32_t(r * kPartThreads) + threadIdx.x;
    if (q < len) atomicAdd(&hist[kk[r] >> p.ws], 1u);
  }
  __syncthreads();
  block_scan_array(hist, nbk, tmp);
  uint16_t* o = O + orow(p, i, e, sc);
  for (uint32_t b = threadIdx.x; b < nbk; b += kPartThreads) o[b] = uint16_t(hist[b]);
  if (threadIdx.x == 0) o[nbk] = uint16_t(len);
  __syncthreads();  // the offsets are read above before they become cursors below
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const uint32_t q = uint32_t(r * kPartThreads) + threadIdx.x;
    if (q < len) {
      const uint32_t k = kk[r];
      const uint32_t slot = atomicAdd(&hist[k >> p.ws], 1u);
      stage[slot] = ((k & (W - 1)) << kScShift) | q;
    }
  }
  __syncthreads();
  for (uint32_t q = threadIdx.x; q < len; q += kPartThreads) stream_store(Pk + base + q, stage[q]);
}

// Window-major copy of the partition offsets: OT[i][b][run] = O[i][run][b],
// so a tile reads the starts and ends of all its runs contiguously.
__global__ void __launch_bounds__(256)
offsets_transpose(SegParams p, const uint16_t* __restrict__ O, uint16_t* __restrict__ OT) {
  __shared__ uint16_t tile[64][65];
  const int64_t R = int64_t(p.E) * p.nsc;
  const int64_t C = int64_t(p.nbk) + 1;
  const int64_t i = blockIdx.z;
  const int64_t r0 = int64_t(blockIdx.x) * 64, c0 = int64_t(blockIdx.y) * 64;
  const uint16_t* src = O + i * R * C;
  uint16_t* dst = OT + i * R * C;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int y = ty; y < 64; y += 4) {
    const int64_t r = r0 + y, c = c0 + tx;
    if (r < R && c < C) tile[y][tx] = src[r * C + c];
  }
  __syncthreads();
  for (int y = ty; y < 64; y += 4) {
    const int64_t c = c0 + y, r = r0 + tx;
    if (r < R && c < C) dst[c * R + r] = tile[tx][y];
  }
}

// -- stats --------------------------------------------------------------------
// Every thread takes whole runs (one run = the window's reads inside one
// sub-chunk, a few reads for uniform shuffles): it loads the run's bounds and
// then up to kRunLoads of its reads at once, so a tile needs one dependent
// pair of loads and no workgroup-wide scan before the LDS updates.
#ifndef NOPFS_RUN_LOADS
#define NOPFS_RUN_LOADS 8
#endif
constexpr int kRunLoads = NOPFS_RUN_LOADS;
#ifndef NOPFS_STATS_SPLIT
#define NOPFS_STATS_SPLIT 4
#endif
constexpr int kStatsSplit = NOPFS_STATS_SPLIT;  // most threads per run
static_assert(kStatsSplit >= 1, "at least one thread per run");
static_assert(kRunLoads % 4 == 0, "whole 16-byte loads");

// kCompact (fused planning call): the tile also lists its read cells for the
// tier plan, entry = the cell's rank-ordered bin << kListOffBits | offset in
// window, at the worker's offset base = its reads in earlier windows (the
// sum of the run starts).
//
// The LDS tables are laid out so that cell x of a pass sits at position
// (x + sh) mod kStatsWin, sh = (flat index of the pass's first cell) mod 4: a
// 4-cell group of the output rows is then one aligned 32-bit count word and
// one aligned 128-bit first-read word in LDS. Only cells after the last
// group wrap around, so the tables take exactly kStatsWin cells (40 KB, four
// workgroups per CU) and the workgroup uses no other LDS: each wave sums the
// run starts itself, and holds the bin records of classes below 64 one per
// lane (looked up with a lane shuffle). Once every wave has read its cells
// into registers, the waves exchange their read-cell totals through the
// first words of the (then free) tables to place their list entries.
constexpr int kStatsCwWords = kStatsWin / 4;  // byte counters
// read cells of a pass binned through LDS (8 bytes each in the first-read
// table's space); passes with more take the per-lane path. One path that
// takes any pass in rounds of kStatsStage cells measured 6.04 ms against
// 5.84 for the two at ImageNet-22k.
constexpr uint32_t kStatsStage = kStatsWin / 2;
constexpr uint32_t kStatsPosMask = kStatsWin - 1;

template <bool kVec, bool kCompact>
__global__ void __launch_bounds__(kStatsThreads) __attribute__((amdgpu_waves_per_eu(8)))
stats_tile(SegParams p, const uint32_t* __restrict__ Pk, const uint16_t* __restrict__ OT,
           uint8_t* __restrict__ count, int32_t* __restrict__ first, uint32_t ntiles,
           uint32_t* __restrict__ cent, int32_t* __restrict__ cbase, uint32_t* __restrict__ cnum,
           const ClassTable* __restrict__ classes) {
  extern __shared__ uint32_t sm[];
  uint32_t* cw = sm;                                             // byte counters
  // first reads, kept as unsigned values from an initial 0xFFFFFFFF: the
  // unsigned minimum of a cell's reads (positions below 2^31), and -1 as an
  // int32 for a cell nobody reads, which is the table's own value for it
  uint32_t* fi = sm + kStatsCwWords;
  const uint32_t tile = xcd_logical(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int64_t i = tile / p.nbk;
  const uint32_t kb = tile - uint32_t(i) * p.nbk;
  const int64_t W = int64_t(1) << p.ws;
  const int64_t k0 = int64_t(kb) * W;
  const int64_t kend = k0 + W < p.F ? k0 + W : p.F;
  const uint32_t* prow = Pk + i * p.M_max;
  const uint32_t* pk_end = Pk + p.N * p.M_max;
  const int64_t Li = seg_len(p, i);
  const int64_t runs = int64_t(p.E) * p.nsc;
  const uint16_t* oa = OT + (i * (p.nbk + 1) + kb) * runs;  // run starts in window kb
  const uint16_t* ob = oa + runs;                            // run ends
  const uint32_t nsc = uint32_t(p.nsc);
  const uint32_t lane = __lane_id();
  // kCompact: the worker's reads in earlier windows (the run starts are
  // requested four per lane at once); unaligned rows (one list slot per
  // cell, claimed with an atomic) start from a zeroed entry count
  uint32_t base = 0, zold = 0, listed = 0;
  if (kCompact) {
    if (!kVec && threadIdx.x == 0) zold = atomicExch(&cnum[tile], 0u);
    for (int64_t r0 = lane; r0 < runs; r0 += 256) {
      uint32_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {  // clamped index: the loads are unconditional
        const int64_t r = r0 + 64 * u;
        v[u] = oa[r < runs ? r : runs - 1];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = r0 + 64 * u < runs ? v[u] : 0u;
      base += v[0] + v[1] + v[2] + v[3];
    }
    base = __builtin_amdgcn_readlane(wave_inclusive_scan(base), 63);
  }
  for (int64_t w0 = k0; w0 < kend; w0 += kStatsWin) {
    const uint32_t wlen = uint32_t(kend - w0 < kStatsWin ? kend - w0 : kStatsWin);
    const uint32_t xoff = uint32_t(w0 - k0);
    const uint32_t sh = kVec ? uint32_t((i * p.F + w0) & 3) : 0u;
    // addresses below are formed anew in each pass (the empty asm keeps
    // the compiler from holding them in registers across the pass)
    uint32_t tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    // With fewer runs than threads, ns = min(threads / runs, kStatsSplit)
    // threads share a run, taking turns at groups of kRunLoads reads (a run
    // of up to ns * kRunLoads reads then needs one round of loads).
    uint32_t ns = runs < kStatsThreads ? uint32_t(kStatsThreads / runs) : 1u;  // uniform
    ns = ns < uint32_t(kStatsSplit) ? ns : uint32_t(kStatsSplit);
    const uint32_t r_first = tid / ns;
    const uint32_t r_step = kStatsThreads / ns;
    const uint32_t q_off = (tid - r_first * ns) * kRunLoads;
    const uint32_t q_step = ns * kRunLoads;
    // bounds of this thread's first run, requested before the LDS is cleared
    uint32_t ra = 0, rb = 0;
    if (r_first < runs) {
      ra = oa[r_first];
      rb = ob[r_first];
    }
    const uint32_t ncl = wlen + sh < uint32_t(kStatsWin) ? wlen + sh : uint32_t(kStatsWin);
    for (uint32_t x = threadIdx.x; x < (ncl + 3) / 4; x += kStatsThreads) cw[x] = 0;
    for (uint32_t x = threadIdx.x; x < ncl; x += kStatsThreads) fi[x] = 0xFFFFFFFFu;
    // kCompact: the zeroing of the entry count has been performed (its old
    // value returned) before this barrier; every claim comes after it
    if (kCompact && !kVec && w0 == k0) asm volatile("" ::"v"(zold));
    __syncthreads();
    for (int64_t r = r_first; r < runs; r += r_step) {
      if (r != r_first) {
        ra = oa[r];
        rb = ob[r];
      }
      const uint32_t e = uint32_t(r) / nsc, sc = uint32_t(r) - e * nsc;
      const int64_t fb = int64_t(e) * Li + int64_t(sc) * kSC;
      const uint32_t* src = prow + fb;
      for (uint32_t q = ra + q_off; q < rb; q += q_step) {
        uint32_t v[kRunLoads];
        if (src + q + kRunLoads <= pk_end) {
          // 16-byte loads (4-byte aligned); the words past the run are
          // other windows' reads, in bounds, and not used
#pragma unroll
          for (int u = 0; u < kRunLoads; u += 4) {
            uint4 a;
            __builtin_memcpy(&a, src + q + u, 16);
            v[u] = a.x;
            v[u + 1] = a.y;
            v[u + 2] = a.z;
            v[u + 3] = a.w;
          }
        } else {
#pragma unroll
          for (int u = 0; u < kRunLoads; ++u) v[u] = q + u < rb ? src[q + u] : 0u;
        }
#pragma unroll
        for (int u = 0; u < kRunLoads; ++u) {
          const uint32_t x = (v[u] >> kScShift) - xoff;
          if (q + u < rb && x < wlen) {
            const uint32_t px = (x + sh) & kStatsPosMask;
            atomicAdd(&cw[px >> 2], 1u << ((px & 3u) * 8u));
            atomicMin(&fi[px], uint32_t(fb + (v[u] & kJMask)));
          }
        }
      }
    }
    __syncthreads();
    // kCompact: bin record of class `lane`, requested here so that it
    // arrives while the tables are read out
    float rec_s = 0.f;
    uint32_t rec_b = 0;
    if (kCompact && kVec) {
      const float2 r = classes->e[tid & 63u];
      rec_s = r.x;
      rec_b = __float_as_uint(r.y);
    }
    // bin of a read cell of class c < 64 (all lanes call it: the shuffle
    // reads other lanes), and of any class from the table in memory
    auto bin_lane = [&](uint32_t c, int32_t f) {
      return bin_of(__shfl(rec_s, int(c), 64), __shfl(rec_b, int(c), 64), f);
    };
    auto bin_mem = [&](uint32_t c, int32_t f) { return bin_read(*classes, c, f); };
    uint8_t* crow = count + i * p.F + w0;
    int32_t* frow = first + i * p.F + w0;
    // cells up to the first flat index divisible by 4 (head, at most 3) and
    // after the last group of 4 (at most 3) go one per thread; the rest as
    // 4-cell groups per lane
    uint32_t head = kVec ? uint32_t((4 - ((i * p.F + w0) & 3)) & 3) : wlen;
    if (head > wlen) head = wlen;
    const uint32_t nunits = (wlen - head) >> 2;
    const uint32_t tail0 = head + 4 * nunits;
    auto cell = [&](uint32_t x, uint32_t& c, int32_t& f) {
      const uint32_t px = (x + sh) & kStatsPosMask;
      c = (cw[px >> 2] >> ((px & 3u) * 8u)) & 0xFFu;
      f = int32_t(fi[px]);  // -1 exactly when c == 0
    };
    uint32_t c1 = 0, c2 = 0;
    int32_t f1 = -1, f2 = -1;
    if (kVec) {
      if (threadIdx.x < head) cell(threadIdx.x, c1, f1);
      if (tail0 + threadIdx.x < wlen) cell(tail0 + threadIdx.x, c2, f2);
    } else {
      for (uint32_t x = threadIdx.x; x < wlen; x += kStatsThreads) {
        uint32_t c;
        int32_t f;
        cell(x, c, f);
        stream_store(crow + x, uint8_t(c));
        stream_store(frow + x, f);
        if (kCompact && c) {  // unaligned rows: one list slot per cell
          const uint32_t b = bin_of(classes->e[c].x, __float_as_uint(classes->e[c].y), f);
          cent[i * p.M_max + base + atomicAdd(&cnum[tile], 1u)] = (b << kListOffBits) | (xoff + x);
        }
      }
    }
    // 4-cell groups: one count word and one first-read quad from LDS
    constexpr int kUnits = kStatsWin / 4 / kStatsThreads;
    uint32_t cwr[kUnits];
    int4 frr[kUnits];
    uint32_t nmine = (c1 != 0) + (c2 != 0);
#pragma unroll
    for (int m = 0; m < kUnits; ++m) {
      const uint32_t u = threadIdx.x + uint32_t(m) * kStatsThreads;
      const uint32_t x = head + 4 * u;  // x + sh is a multiple of 4
      cwr[m] = 0;
      frr[m] = make_int4(-1, -1, -1, -1);
      if (u < nunits) {
        const uint32_t px = (x + sh) & kStatsPosMask;  // no group wraps
        const uint32_t word = cw[px >> 2];
        cwr[m] = word;
        frr[m] = *reinterpret_cast<const int4*>(&fi[px]);  // -1 for unread cells already
        // nonzero counts among the word's four bytes: a byte's high bit in
        // ((w & 0x7F..) + 0x7F..) | w is set exactly when the byte is nonzero
        const uint32_t nz = ((word & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | word;
        nmine += __popc(nz & 0x80808080u);
      }
    }
    // list: the waves' read cells go in wave order, each wave's as one run
    // (the list's users do not depend on the order of a tile's entries).
    // The totals are exchanged through LDS with barriers that wait for LDS
    // work only (the row stores stay in flight).
    uint32_t incl = 0, wbase = 0, pass_base = 0, pass_all = 0;
    if (kCompact && kVec) {
      constexpr int kWaves = kStatsThreads / 64;
      const uint32_t wave = threadIdx.x >> 6;
      incl = wave_inclusive_scan(nmine);
      const uint32_t wtot = __builtin_amdgcn_readlane(incl, 63);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");  // tables read
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
      if (lane == 0) sm[wave] = wtot;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
      uint32_t before = 0, all = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const uint32_t t = sm[w];
        before += uint32_t(w) < wave ? t : 0u;
        all += t;
      }
      wbase = listed + before;
      pass_base = listed;
      pass_all = all;
      listed += all;
    }
    // kCompact: the class records arrive before the row stores go out: a
    // wait for them behind the stores would wait for the stores too (one
    // counter covers loads and stores, in order)
    if (kCompact && kVec) asm volatile("" ::"v"(rec_s), "v"(rec_b));
    if (kVec) {
      if (threadIdx.x < head) {
        crow[threadIdx.x] = uint8_t(c1);
        frow[threadIdx.x] = f1;
      }
      if (tail0 + threadIdx.x < wlen) {
        crow[tail0 + threadIdx.x] = uint8_t(c2);
        frow[tail0 + threadIdx.x] = f2;
      }
    }
#pragma unroll
    for (int m = 0; m < kUnits; ++m) {
      const uint32_t u = threadIdx.x + uint32_t(m) * kStatsThreads;
      const uint32_t x = head + 4 * u;
      if (u < nunits) {
        stream_store(reinterpret_cast<uint32_t*>(crow + x), cwr[m]);
        stream_store(reinterpret_cast<int4*>(frow + x), frr[m]);
      }
    }
    if (kCompact && kVec && pass_all <= kStatsStage) {
      // The pass's read cells go through LDS (the first-read table, now
      // read out) in list order, then the waves bin them densely: each
      // lane bins and stores only read cells, and the stores are coalesced.
      uint32_t* cdst = cent + i * p.M_max + base + pass_base;
      uint2* stg = reinterpret_cast<uint2*>(sm + kStatsCwWords);
      uint32_t slot = wbase - pass_base + incl - nmine;
      auto put = [&](uint32_t c, int32_t f, uint32_t x) {
        if (c) stg[slot++] = make_uint2(((xoff + x) << 8) | c, uint32_t(f));
      };
      put(c1, f1, threadIdx.x);
      put(c2, f2, tail0 + threadIdx.x);
#pragma unroll
      for (int m = 0; m < kUnits; ++m) {
        const uint32_t x = head + 4 * (threadIdx.x + uint32_t(m) * kStatsThreads);
        const int32_t fv[4] = {frr[m].x, frr[m].y, frr[m].z, frr[m].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) put((cwr[m] >> (8 * q)) & 0xFFu, fv[q], x + q);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
      // the list addresses are formed here: an address held from the
      // kernel's start was spilled, and its reload's wait would also have
      // waited for the row stores above
      uint32_t ltid = threadIdx.x;
      asm volatile("" : "+v"(ltid));
      for (uint32_t t0 = 0; t0 < pass_all; t0 += kStatsThreads) {  // uniform trip count
        const uint32_t t = t0 + ltid;
        const uint2 e = stg[t < pass_all ? t : 0u];
        const uint32_t c = e.x & 0xFFu;
        uint32_t b = bin_lane(c & 63u, int32_t(e.y));
        if (c >= 64u) b = bin_mem(c, int32_t(e.y));  // counts of 64 or more
        if (t < pass_all) stream_store(cdst + t, (b << kListOffBits) | (e.x >> 8));
      }
    } else if (kCompact && kVec) {
      uint32_t* cdst = cent + i * p.M_max + base;
      uint32_t slot = wbase + incl - nmine;
      auto emit = [&](auto bin) {
        const uint32_t b1 = bin(c1, f1), b2 = bin(c2, f2);
        if (c1) cdst[slot++] = (b1 << kListOffBits) | (xoff + threadIdx.x);
        if (c2) cdst[slot++] = (b2 << kListOffBits) | (xoff + tail0 + threadIdx.x);
#pragma unroll
        for (int m = 0; m < kUnits; ++m) {
          const uint32_t x = head + 4 * (threadIdx.x + uint32_t(m) * kStatsThreads);
          const int32_t fv[4] = {frr[m].x, frr[m].y, frr[m].z, frr[m].w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t c = (cwr[m] >> (8 * q)) & 0xFFu;
            const uint32_t b = bin(c, fv[q]);
            if (c) cdst[slot++] = (b << kListOffBits) | (xoff + x + q);
          }
        }
      };
      // counts of 64 or more (jobs of more epochs) take the table in memory
      uint32_t hi = (c1 | c2) & 0xC0u;
#pragma unroll
      for (int m = 0; m < kUnits; ++m) hi |= cwr[m] & 0xC0C0C0C0u;
      if (__any(hi != 0))
        emit(bin_mem);
      else
        emit(bin_lane);
    }
    if (w0 + kStatsWin < kend) __syncthreads();  // the tables are reused
  }
  if (kCompact && threadIdx.x == 0) {
    cbase[tile] = int32_t(base);
    if (kVec) cnum[tile] = listed;
  }
}

// -- next ---------------------------------------------------------------------
// Fast path: the window's reads are gathered into LDS and pushed onto short
// chains, one per hash slot of their sample offset (atomic exchange on the
// slot head). A read's next use is then the smallest later stream position
// among the reads of the same sample on its chain; chains hold about one
// read on average, so no sort is needed.
constexpr int kNextSlots = 4096;  // hash slots per window (power of two)
constexpr uint32_t kNoLink = 0xFFFFu;

struct NextSmem {
  uint32_t head[kNextSlots];
  int32_t f[kNextEnt];
  uint16_t kl[kNextEnt];
  uint16_t link[kNextEnt];
};

__device__ void next_tile_slow(const SegParams& p, int64_t i, uint32_t kb, const uint32_t* prow,
                               const uint16_t* O, int32_t* nrow, RunTable<kNextThreads>& rt, int32_t* last) {
  const int64_t W = int64_t(1) << p.ws;
  const int64_t k0 = int64_t(kb) * W;
  const int64_t kend = k0 + W < p.F ? k0 + W : p.F;
  for (int64_t w0 = k0; w0 < kend; w0 += kSlowWin) {
    const uint32_t wlen = uint32_t(kend - w0 < kSlowWin ? kend - w0 : kSlowWin);
    const uint32_t xoff = uint32_t(w0 - k0);
    for (uint32_t x = threadIdx.x; x < wlen; x += kNextThreads) last[x] = -1;
    __syncthreads();
    for (int64_t e = p.E - 1; e >= 0; --e) {
      // reads of one epoch are distinct samples: no two threads share a slot
      for_each_read(p, i, kb, O, prow, rt, e, e + 1,
                    [&](int64_t pos, int64_t fbase, uint32_t v, uint32_t) {
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

__global__ void __launch_bounds__(kNextThreads)
next_tile(SegParams p, const uint32_t* __restrict__ Pk, const uint16_t* __restrict__ OT,
          int32_t* __restrict__ nextP, uint32_t ntiles) {
  extern __shared__ uint32_t sm[];
  __shared__ RunTable<kNextThreads> rt;
  __shared__ uint32_t s_total;
  const uint32_t tile = xcd_logical(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int64_t i = tile / p.nbk;
  const uint32_t kb = tile - uint32_t(i) * p.nbk;
  const uint32_t* prow = Pk + i * p.M_max;
  int32_t* nrow = nextP + i * p.M_max;
  const int64_t runs = int64_t(p.E) * p.nsc;

  // number of reads in the window; with at most kNextThreads runs the run
  // table loaded here is reused for the gather below
  uint32_t total;
  if (runs <= kNextThreads) {
    total = load_runs(p, i, kb, OT, rt, 0, runs, 0);
  } else {
    if (threadIdx.x == 0) s_total = 0;
    __syncthreads();
    const int64_t R = runs;
    const uint16_t* oa = OT + (i * (p.nbk + 1) + kb) * R;
    uint32_t mine = 0;
    for (int64_t r = threadIdx.x; r < runs; r += kNextThreads) mine += uint32_t(oa[R + r] - oa[r]);
    atomicAdd(&s_total, mine);
    __syncthreads();
    total = s_total;
  }
  if (total == 0) return;
  if (p.ws > 16 || total > uint32_t(p.ent_cap)) {
    __syncthreads();
    next_tile_slow(p, i, kb, prow, OT, nrow, rt, reinterpret_cast<int32_t*>(sm));
    return;
  }
  NextSmem& s = *reinterpret_cast<NextSmem*>(sm);
  auto gather = [&](int64_t, int64_t fbase, uint32_t v, uint32_t idx) {
    const uint32_t x = v >> kScShift;
    s.kl[idx] = uint16_t(x);
    s.f[idx] = int32_t(fbase + (v & kJMask));
    s.link[idx] = uint16_t(atomicExch(&s.head[x & (kNextSlots - 1)], idx));
  };
  // With at most kNextThreads runs, read idx = threadIdx.x + q * kNextThreads
  // is this thread's in the gather and in the output: its position in the
  // partitioned row, found once through the run table, stays in a register,
  // and all of the thread's reads are requested at once, before the chain
  // heads are cleared (the clearing and its barrier overlap the loads).
  constexpr int kPerThread = (kNextEnt + kNextThreads - 1) / kNextThreads;
  static_assert(kNextEnt <= int(kRunMap), "the run table maps every read of a fast-path window");
  int32_t posq[kPerThread];
  if (runs <= kNextThreads) {
    uint32_t vq[kPerThread];
    int32_t fbq[kPerThread];
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
      const uint32_t idx = threadIdx.x + q * kNextThreads;
      posq[q] = -1;
      fbq[q] = 0;
      if (idx < total) {
        const int r = rt.run_of[idx];
        posq[q] = rt.start[r] + int32_t(idx - rt.pref[r]);
        fbq[q] = rt.fbase[r];
      }
    }
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) vq[q] = prow[posq[q] >= 0 ? posq[q] : 0];  // unconditional
    for (int d = threadIdx.x; d < kNextSlots; d += kNextThreads) s.head[d] = kNoLink;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kPerThread; ++q)
      if (posq[q] >= 0) gather(posq[q], fbq[q], vq[q], threadIdx.x + q * kNextThreads);
  } else {
    for (int d = threadIdx.x; d < kNextSlots; d += kNextThreads) s.head[d] = kNoLink;
    __syncthreads();
    for_each_read(p, i, kb, OT, prow, rt, 0, p.E, gather);
  }
  __syncthreads();
  // each read: smallest later position of the same sample on its chain
  int32_t res[kPerThread];
#pragma unroll
  for (int q = 0; q < kPerThread; ++q) {
    const uint32_t idx = threadIdx.x + q * kNextThreads;
    res[q] = -1;
    if (idx < total) {
      const uint32_t x = s.kl[idx];
      const int32_t f = s.f[idx];
      int32_t best = INT_MAX;
      for (uint32_t w = s.head[x & (kNextSlots - 1)]; w != kNoLink; w = s.link[w]) {
        const int32_t fw = s.f[w];
        if (s.kl[w] == x && fw > f && fw < best) best = fw;
      }
      res[q] = best == INT_MAX ? -1 : best;
    }
  }
  if (runs <= kNextThreads) {
#pragma unroll
    for (int q = 0; q < kPerThread; ++q)
      if (posq[q] >= 0) nrow[posq[q]] = res[q];
  } else {
    __syncthreads();  // every chain walk is done before f is overwritten
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
      const uint32_t idx = threadIdx.x + q * kNextThreads;
      if (idx < total) s.f[idx] = res[q];
    }
    __syncthreads();
    for_each_read(p, i, kb, OT, prow, rt, 0, p.E,
                  [&](int64_t pos, int64_t, uint32_t, uint32_t idx) { nrow[pos] = s.f[idx]; });
  }
}

constexpr int kUnpartThreads = 1024;

__global__ void __launch_bounds__(kUnpartThreads)
next_unpartition(SegParams p, const uint32_t* __restrict__ Pk, const int32_t* __restrict__ nextP,
                 int32_t* __restrict__ next) {
  __shared__ int32_t stage[kSC];
  const uint32_t wg = blockIdx.x;
  const uint32_t per_worker = uint32_t(p.E) * uint32_t(p.nsc);
  const uint32_t i = wg / per_worker;
  const uint32_t rem = wg - i * per_worker;
  const uint32_t e = rem / uint32_t(p.nsc), sc = rem - e * uint32_t(p.nsc);
  const int64_t Li = seg_len(p, i);
  int64_t len64 = Li - int64_t(sc) * kSC;
  len64 = len64 < 0 ? 0 : (len64 > kSC ? kSC : len64);
  const uint32_t len = uint32_t(len64);
  if (len == 0) return;
  const int64_t base = int64_t(i) * p.M_max + int64_t(e) * Li + int64_t(sc) * kSC;
  {
    // all of the thread's loads at once (clamped), then the LDS stores
    constexpr int kPer = kSC / kUnpartThreads;
    uint32_t j[kPer];
    int32_t v[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const uint32_t q = u * kUnpartThreads + threadIdx.x;
      j[u] = Pk[base + (q < len ? q : 0u)];
      v[u] = nextP[base + (q < len ? q : 0u)];
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u)
      if (u * kUnpartThreads + threadIdx.x < len) stage[j[u] & kJMask] = v[u];
  }
  __syncthreads();
  for (uint32_t q = threadIdx.x; q < len; q += kUnpartThreads) stream_store(next + base + q, stage[q]);
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

int launch_stats(const SegParams& p, const uint32_t* Pk, const uint16_t* OT, uint8_t* count,
                 int32_t* first, CompactCells* cc, const ClassTable* classes, hipStream_t st) {
  const uint32_t ntiles = uint32_t(p.N * p.nbk);
  const size_t smem = size_t(kStatsCwWords + kStatsWin) * 4;
  // vector stores need 4-byte aligned count rows and 16-byte aligned first rows
  const bool vec = (reinterpret_cast<uintptr_t>(count) & 3) == 0 &&
                   (reinterpret_cast<uintptr_t>(first) & 15) == 0;
  const dim3 grid(xcd_padded(ntiles)), block(kStatsThreads);
  uint32_t* ent = cc ? cc->ent : nullptr;
  int32_t* base = cc ? cc->base : nullptr;
  uint32_t* num = cc ? cc->num : nullptr;
  if (cc)
    return vec ? launch("stats_tile", stats_tile<true, true>, grid, block, smem, st, p, Pk, OT, count,
                        first, ntiles, ent, base, num, classes)
               : launch("stats_tile", stats_tile<false, true>, grid, block, smem, st, p, Pk, OT,
                        count, first, ntiles, ent, base, num, classes);
  return vec ? launch("stats_tile", stats_tile<true, false>, grid, block, smem, st, p, Pk, OT, count,
                      first, ntiles, ent, base, num, classes)
             : launch("stats_tile", stats_tile<false, false>, grid, block, smem, st, p, Pk, OT, count,
                      first, ntiles, ent, base, num, classes);
}

// Window width of the next-use pass: the widest whose expected reads stay
// within three quarters of the fast-path capacity (windows that overflow it
// take the epoch-serial path).
int next_ws(const Shape& s) {
  const double reads_per_sample = double(s.M_max) / double(s.F);
  int ws = 0;
  while (ws < NOPFS_NEXT_WSMAX && double(int64_t(1) << (ws + 1)) * reads_per_sample <= kNextEnt * 3 / 4)
    ++ws;
  return ws;
}

SegParams next_params(const Shape& s) {
  SegParams p = seg_params(s, next_ws(s));
  if (debug_value(2) > 0 && debug_value(2) < kNextEnt) p.ent_cap = int32_t(debug_value(2));
  return p;
}

// nextP: scratch laid out like the partitioned reads (N * M_max int32).
int launch_next(const SegParams& p, const uint32_t* Pk, const uint16_t* OT, int32_t* nextP,
                int32_t* next, hipStream_t st) {
  int rc;
  const uint32_t ntiles = uint32_t(p.N * p.nbk);
  size_t smem = sizeof(NextSmem);
  if (smem < size_t(kSlowWin) * 4) smem = size_t(kSlowWin) * 4;
  if ((rc = launch("next_tile", next_tile, dim3(xcd_padded(ntiles)), dim3(kNextThreads), smem, st, p,
                   Pk, OT, nextP, ntiles)))
    return rc;
  const int64_t wgs = p.N * p.E * p.nsc;
  if ((rc = launch("next_unpartition", next_unpartition, dim3(uint32_t(wgs)), dim3(kUnpartThreads), 0,
                   st, p, Pk, (const int32_t*)nextP, next)))
    return rc;
  if (!p.drop_last && p.F % p.N != 0)
    if ((rc = launch("pad_rows", pad_rows, dim3(uint32_t(p.N)), dim3(64), 0, st, p, next))) return rc;
  return NOPFS_OK;
}

}  // namespace

static int log2_ceil(int64_t v) {
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
  p.emul = 1;
  return p;
}

static size_t partition_smem(const SegParams& p) {
  return size_t(((p.nbk + 4) & ~3u) + kSC) * 4;
}

int run_partition(const SegParams& p, const int32_t* R, Scratch& scr, uint32_t** Pk,
                  uint16_t** OT, hipStream_t st) {
  int rc;
  uint16_t* O;
  const size_t on = size_t(p.N * p.E * p.nsc) * (p.nbk + 1);
  if ((rc = scr.alloc_n(Pk, size_t(p.N * p.M_max)))) return rc;
  if ((rc = scr.alloc_n(&O, on))) return rc;
  if ((rc = scr.alloc_n(OT, on))) return rc;
  const int64_t wgs = p.N * p.E * p.nsc;
  if ((rc = launch("seg_partition", seg_partition, dim3(uint32_t(wgs)), dim3(kPartThreads),
                   partition_smem(p), st, p, R, *Pk, O)))
    return rc;
  const int64_t runs = int64_t(p.E) * p.nsc;
  return launch("offsets_transpose", offsets_transpose,
                dim3(uint32_t(ceil_div(runs, 64)), uint32_t(ceil_div(p.nbk + 1, 64)), uint32_t(p.N)),
                dim3(256), 0, st, p, (const uint16_t*)O, *OT);
}

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
  SegParams p = seg_params(s, NOPFS_STATS_WS);
  Scratch scr(st);
  uint32_t* Pk;
  uint16_t* OT;
  if ((rc = run_partition(p, R, scr, &Pk, &OT, st))) return rc;
  return launch_stats(p, Pk, OT, count, first, nullptr, nullptr, st);
}

int next_impl(const nopfs_job* job, const int32_t* R, int32_t* next, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (s.M_max == 0) return NOPFS_OK;  // R and next have no elements and may be NULL
  if (!R || !next) return fail(NOPFS_EINVAL, "R and next must be non-NULL");
  const SegParams p = next_params(s);
  Scratch scr(st);
  uint32_t* Pk;
  uint16_t* OT;
  int32_t* nextP;
  if ((rc = run_partition(p, R, scr, &Pk, &OT, st))) return rc;
  if ((rc = scr.alloc_n(&nextP, size_t(s.N * s.M_max)))) return rc;
  return launch_next(p, Pk, OT, nextP, next, st);
}

int access_fused(const Shape& s, const int32_t* R, const ClassTable* classes, uint8_t* count,
                 int32_t* first, int32_t* next, CompactCells* cc, Scratch& keep, hipStream_t st) {
  int rc;
  const SegParams ps = seg_params(s, NOPFS_STATS_WS);
  const SegParams pn = next_params(s);
  uint32_t *Pk, *Pn;
  uint16_t *OT, *OTn;
  int32_t* nextP;
  if ((rc = run_partition(ps, R, keep, &Pk, &OT, st))) return rc;
  cc->ws = ps.ws;
  cc->nbk = ps.nbk;
  if ((rc = keep.alloc_n(&cc->ent, size_t(s.N * s.M_max)))) return rc;
  if ((rc = keep.alloc_n(&cc->base, size_t(s.N) * ps.nbk))) return rc;
  if ((rc = keep.alloc_n(&cc->num, size_t(s.N) * ps.nbk))) return rc;
  if ((rc = launch_stats(ps, Pk, OT, count, first, cc, classes, st))) return rc;
  // the next-use pass shares the partition when it uses the same windows
  Pn = Pk;
  OTn = OT;
  if (pn.ws != ps.ws)
    if ((rc = run_partition(pn, R, keep, &Pn, &OTn, st))) return rc;
  if ((rc = keep.alloc_n(&nextP, size_t(s.N * s.M_max)))) return rc;
  return launch_next(pn, Pn, OTn, nextP, next, st);
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
