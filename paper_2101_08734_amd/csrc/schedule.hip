// nopfs_prefetch_order and nopfs_staging_schedule: what the Design section
// derives from the streams and the placement for a worker's prefetchers.
//
// Both calls need a per-sample value for every read (a first read, a size)
// and then results in stream order, so both run on a partition of R by
// sample window (counting sort of each sub-chunk of 2^14 reads by window, as
// in the counting pass): a tile per window does the per-sample work in LDS
// and writes one value per read in partitioned order; a pass per sub-chunk
// puts the values back in stream order through LDS. No pass scatters into or
// gathers from HBM at random: gathering each read's size straight from the
// size table is bound by the rate of random cache-line requests (about 5e10
// per second on MI355X, 11 ms for ImageNet-22k's 5.7e8 reads, more than this
// whole pipeline).
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
// The staging passes fold each row's E epochs into one segment of E * L_i
// reads, cut into spans of 2^14 positions, and partition the spans by
// windows of 2^14 samples:
//   st_range  -- whether every size fits 32 bits (then the sizes travel as
//                4-byte values, else as 8-byte ones).
//   st_gather -- per (window, group of 32 workers): the window's sizes in
//                LDS (128 KB); every read of the group's spans gets its
//                sample's size, written in partitioned order.
//   st_unpart -- per span: the sizes back in stream order in LDS, their
//                inclusive prefix sums inside the span (a wave scan per 64
//                positions, in registers), the span's total.
//   st_base   -- per worker: exclusive scan of the span totals.
//   st_bounds -- per quarter of a span (4096 positions): the g of its first
//                and of its last position (binary search over S; g never
//                decreases along R).
//   st_fill   -- per quarter: S over that g range is staged in LDS, each
//                thread binary-searches the g of its first position there
//                and walks its other positions with two pointers; -1 in
//                padding.
#include <limits.h>

#include <new>

#include "gather.hpp"
#include "partition.hpp"

namespace nopfs {
namespace {


constexpr int kSchedWs = 13;             // partition windows: 2^13 samples
constexpr int kWin = 1 << kSchedWs;      // samples per LDS pass of a tile
constexpr int kTileThreads = 512;
constexpr int kPfMaxJ = 128;

// ------------------------------------------------------------- prefetch --
constexpr int kPfKeep = 4;  // reads per thread kept in registers between the passes
// 4-byte words of a window's tiers per thread (the aligned cover of kWin
// bytes spans at most kWin / 4 + 1 words)
constexpr int kPfTierWords = (kWin / 4 + 1 + kTileThreads - 1) / kTileThreads;

// Per read of the tile: first-read candidate for its sample (pass 1), then
// its code (pass 2). When the tile's runs fit one run table and its reads fit
// kPfKeep per thread, the reads are spread evenly over the threads through
// the run table and kept in registers between the passes. The window's tiers
// and the run bounds are requested together, the reads before the tables
// are initialised: two dependent rounds of global loads per tile. Otherwise
// each thread walks whole runs twice.
__global__ void __launch_bounds__(kTileThreads)
pf_tile(SegParams p, const uint32_t* __restrict__ Pk, const uint16_t* __restrict__ OT,
        const int8_t* __restrict__ tier, int32_t J, uint8_t* __restrict__ code,
        uint32_t ntiles) {
  __shared__ int32_t fi[kWin];        // first read of each sample of the pass
  __shared__ uint32_t tw4[kWin / 4 + 1];  // its tier: byte x + tsh (fast path), x (walk)
  __shared__ RunTable<kTileThreads> rt;
  int8_t* tw = reinterpret_cast<int8_t*>(tw4);
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
    // the window's tiers as the 4-byte words covering it, when the cover lies
    // inside the tier table (not at an unaligned table start or end: then
    // one byte per load)
    const int8_t* wbeg = trow + k0;
    const uint32_t tsh = uint32_t(reinterpret_cast<uintptr_t>(wbeg) & 3u);
    const int8_t* cbeg = wbeg - tsh;
    const uint32_t nw = (tsh + wl + 3) / 4;
    const bool words = cbeg >= tier && cbeg + 4 * int64_t(nw) <= tier + p.N * p.F;  // uniform
    const uint32_t* w4 = reinterpret_cast<const uint32_t*>(cbeg);
    uint32_t tv[kPfTierWords];
    if (words) {
#pragma unroll
      for (int u = 0; u < kPfTierWords; ++u) {
        const uint32_t x = threadIdx.x + u * kTileThreads;
        tv[u] = w4[x < nw ? x : 0u];  // unconditional
      }
    } else {
#pragma unroll
      for (int u = 0; u < kPfTierWords; ++u) {
        const uint32_t x = threadIdx.x + u * kTileThreads;
        uint32_t w = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) {  // bytes of word x, laid out from the window start
          const uint32_t y = 4 * x + c;
          w |= uint32_t(uint8_t(wbeg[y < wl ? y : 0u])) << (8 * c);
        }
        tv[u] = w;
      }
    }
    const uint32_t tshl = words ? tsh : 0u;
    // run table
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
      for (int u = 0; u < kPfKeep; ++u) v[u] = prow[pos[u] >= 0 ? pos[u] : 0];  // unconditional
      // the tables, while the reads are in flight
      for (uint32_t x = threadIdx.x; x < kWin / 4; x += kTileThreads)
        reinterpret_cast<int4*>(fi)[x] = make_int4(INT_MAX, INT_MAX, INT_MAX, INT_MAX);
#pragma unroll
      for (int u = 0; u < kPfTierWords; ++u) {
        const uint32_t x = threadIdx.x + u * kTileThreads;
        if (x < kWin / 4 + 1) tw4[x] = tv[u];
      }
      __syncthreads();
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
            const int32_t t = tw[x + tshl];
            const bool queued = fi[x] == fb[u] + int32_t(v[u] & kJMask) && t >= 0 && t < J;
            crow[pos[u]] = queued ? uint8_t(t + 1) : uint8_t(0);
          }
        }
      return;
    }
    __syncthreads();  // the run table is no longer read
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
// so the codes are read in partitioned order. Up to kPfWordJ tiers the codes
// are read and counted four to a word; more tiers take one code per lane.
constexpr int kPfWordJ = 8;
__global__ void __launch_bounds__(256)
pf_count(SegParams p, int32_t J, const uint8_t* __restrict__ code, uint32_t nch,
         int32_t* __restrict__ cnt) {
  __shared__ uint32_t s_cnt[kPfMaxJ];
  const SubChunk s = sub_chunk(p, nch, blockIdx.x);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int x = threadIdx.x; x < J; x += 256) s_cnt[x] = 0;
  __syncthreads();
  const uint8_t* src = code + s.base;
  if (J <= kPfWordJ) {
    // four codes per load: the 4-byte words covering the sub-chunk (the code
    // table is the library's own, 256-byte aligned and sized, so the cover
    // stays inside it), bytes outside the sub-chunk masked to code 0; per
    // tier, the bytes equal to t + 1 counted within the word
    const uint32_t sh = uint32_t(reinterpret_cast<uintptr_t>(src) & 3u);
    const uint32_t* w4 = reinterpret_cast<const uint32_t*>(src - sh);
    const uint32_t len = uint32_t(s.len);
    const uint32_t nw = (sh + len + 3) / 4;
    uint32_t c[kPfWordJ];
#pragma unroll
    for (int t = 0; t < kPfWordJ; ++t) c[t] = 0;
    constexpr int kBatch = 8;
    for (uint32_t x0 = threadIdx.x; x0 < nw; x0 += 256 * kBatch) {
      uint32_t m[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {  // unconditional loads, all in flight together
        const uint32_t x = x0 + u * 256;
        m[u] = w4[x < nw ? x : 0u];
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const uint32_t x = x0 + u * 256;
        // byte b of word x is position 4x + b - sh of the sub-chunk
        uint32_t keep = 0xFFFFFFFFu;
        if (x == 0) keep &= 0xFFFFFFFFu << (8 * sh);
        const uint32_t end = 4 * x + 4;  // one past the word's last byte, in cover bytes
        if (end > sh + len) keep &= 0xFFFFFFFFu >> (8 * (end - sh - len) < 32 ? 8 * (end - sh - len) : 31);
        if (x >= nw || end - 4 >= sh + len) keep = 0;
        m[u] &= keep;
#pragma unroll
        for (int t = 0; t < kPfWordJ; ++t) {
          if (t < J) {
            const uint32_t d = m[u] ^ (uint32_t(t + 1) * 0x01010101u);  // zero bytes: code t + 1
            const uint32_t nz = ((d & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | d;   // high bit: byte nonzero
            c[t] += 4u - uint32_t(__popc(nz & 0x80808080u));
          }
        }
      }
    }
#pragma unroll
    for (int t = 0; t < kPfWordJ; ++t)
      if (t < J) {
        const uint32_t tot = __builtin_amdgcn_readlane(wave_inclusive_scan(c[t]), 63);
        if (lane == 0 && tot) atomicAdd(&s_cnt[t], tot);
      }
    __syncthreads();
    int32_t* out = cnt + (s.i * nch + s.c) * J;
    for (int x = threadIdx.x; x < J; x += 256) out[x] = int32_t(s_cnt[x]);
    return;
  }
  constexpr int kBatch = 8;
  for (int64_t j0 = int64_t(w) * 64 * kBatch; j0 < s.len; j0 += 256 * kBatch) {
    uint32_t m[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {  // unconditional loads, all in flight together
      const int64_t j = j0 + u * 64 + lane;
      m[u] = src[j < s.len ? j : 0];
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      m[u] = j0 + u * 64 + lane < s.len ? clamp_code(uint8_t(m[u]), J) : 0u;
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
  // codes to stream order (every position of the sub-chunk has one entry),
  // sixteen entries per thread and step with their loads issued together
  for (int64_t q0 = 0; q0 < s.len; q0 += 16 * 64 * kPfWaves) {
    uint32_t j[16];
    uint8_t c[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int64_t q = q0 + u * 64 * kPfWaves + threadIdx.x;
      j[u] = Pk[s.base + (q < s.len ? q : 0)];
      c[u] = code[s.base + (q < s.len ? q : 0)];
    }
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (q0 + u * 64 * kPfWaves + threadIdx.x < s.len) s_code[j[u] & kJMask] = c[u];
  }
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
      k[u] = Rsub[j < s.len ? j : 0];  // unconditional
    }
    // every sample id is in a register before the first store: a wait for
    // a load inside the store loop would also wait for the stores before it
#pragma unroll
    for (int u = 0; u < kPfBatch; ++u) asm volatile("" : "+v"(k[u]));
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
// The staging passes see each row of R as one segment of E * L_i reads (the
// epochs folded together), cut into spans of kSC = 2^14 positions: position
// h lies in span h >> kScShift. The partition of R by sample window is taken
// over those spans.

// zP[x] = sizes[k] for every read of the tile's window and rows, x being the
// read's place in the partitioned row (so zP holds the sizes in partitioned
// order).
// With every size in [0, 2^32) (*wide == 0, found by st_range) the sizes go
// out as 4-byte values into zc, else as 8-byte values into zP. Eight reads
// per thread and inner pass (the run map then fills the LDS the window
// leaves): half the dependent load rounds of four, 2.09 -> 1.94 ms at
// ImageNet-22k.
constexpr int kStGChunk = 8 * kGThreads;
constexpr int kStGPer = kStGChunk / kGThreads;
__global__ void __launch_bounds__(kGThreads)
st_gather(SegParams p, const uint32_t* __restrict__ Pk, const uint16_t* __restrict__ OT,
          const int64_t* __restrict__ sizes, const uint32_t* __restrict__ wide,
          uint32_t* __restrict__ zc, int64_t* __restrict__ zP, uint32_t ngroups, uint32_t ntiles) {
  __shared__ GatherLds<kStGChunk> L;
  const uint32_t tile = xcd_logical(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  if (*wide != 0u) {  // uniform
    gather_tile<uint64_t, kStGChunk>(
        p, Pk, OT, tile, ngroups, L, [&](int64_t k) { return uint64_t(sizes[k]); },
        [&](const int64_t (&pos)[kStGPer], const int64_t (&)[kStGPer], const uint32_t (&x)[kStGPer],
            int64_t, uint32_t wl) {
#pragma unroll
          for (int u = 0; u < kStGPer; ++u)
            if (pos[u] >= 0 && x[u] < wl) zP[pos[u]] = int64_t(L.win[x[u]]);
        });
  } else {
    gather_tile<uint32_t, kStGChunk>(
        p, Pk, OT, tile, ngroups, L, [&](int64_t k) { return uint32_t(sizes[k]); },
        [&](const int64_t (&pos)[kStGPer], const int64_t (&)[kStGPer], const uint32_t (&x)[kStGPer],
            int64_t, uint32_t wl) {
#pragma unroll
          for (int u = 0; u < kStGPer; ++u)
            if (pos[u] >= 0 && x[u] < wl) zc[pos[u]] = L.win4[x[u]];
        });
  }
}

// *wide = 1 when some size lies outside [0, 2^32); st_flag clears it first.
__global__ void st_flag(uint32_t* __restrict__ wide) { *wide = 0u; }

__global__ void __launch_bounds__(256)
st_range(int64_t F, const int64_t* __restrict__ sizes, uint32_t* __restrict__ wide) {
  const int64_t k0 = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 4;
  bool out = false;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int64_t k = k0 + u;
    const uint64_t v = uint64_t(sizes[k < F ? k : 0]);
    out |= k < F && (v >> 32) != 0;
  }
  if (__any(out) && __lane_id() == 0) atomicOr(wide, 1u);
}

constexpr int kUThreads = 1024;
constexpr int kUWaves = kUThreads / 64;
constexpr int kURows = kSC / kUThreads;  // 64-lane rows per wave: 16

// The reads of one span as loaded by st_unpart: thread t holds entries
// t, t + 1024, ... of the span's partitioned order (packed entry, size).
// The loads are unconditional (entries past the span's end load its first
// entry and are skipped when consumed), so they stay in flight together.
struct SpanRegs {
  uint32_t j[kURows];
  int64_t z[kURows];
};

__device__ __forceinline__ int64_t span_len(const SegParams& p, int64_t i, int64_t c) {
  const int64_t len = seg_len(p, i) - (c << kScShift);
  return len < 0 ? 0 : (len > kSC ? kSC : len);
}

template <bool kWide>
__device__ __forceinline__ void span_load(const SegParams& p, const uint32_t* __restrict__ Pk,
                                          const int64_t* zS, const uint32_t* zc, int64_t b,
                                          int64_t nblk, SpanRegs& g) {
  int64_t len = 0, base = 0;
  if (b < nblk) {
    const int64_t i = b / p.nsc, c = b - i * p.nsc;
    len = span_len(p, i, c);
    base = i * p.M_max + (c << kScShift);  // inside the row table even when len == 0
  }
#pragma unroll
  for (int u = 0; u < kURows; ++u) {
    const int64_t q = int64_t(u) * kUThreads + threadIdx.x;
    const int64_t at = base + (q < len ? q : 0);
    g.j[u] = Pk[at];
    g.z[u] = kWide ? zS[at] : int64_t(zc[at]);
  }
}

// Per span c of row i: S[h] = sum of the sizes at positions
// (h >> 14 << 14) .. h, and ctot[i][c] = the span's total. The sizes come
// in partitioned order (zS, 8-byte, or zc, 4-byte); with 4-byte sizes, a
// span whose total is below 2^32 writes S as 4-byte values into zc (in
// place of its sizes, which the workgroup holds in registers by then) and
// marks sw[b] = 0; any other span writes S as 8-byte values into zS (in
// place for 8-byte sizes) and marks sw[b] = 1. The sizes go back to
// stream order in LDS (each read's partitioned entry carries its position),
// then wave w sums its 1024 consecutive positions, takes the totals of the
// waves before it as its carry and scans them as 16 rows of 64 lanes in
// registers (a wave scan per row plus the running carry); S is written in
// whole lines. The span needs all of
// the LDS a CU has for one workgroup, so each workgroup walks spans b,
// b + gridDim.x, ... and loads the next span's entries before it scans the
// current one.
// kWide: the sizes are 8-byte values in zS (and S overwrites them in place);
// otherwise 4-byte values in zc. Both forms are launched; the one that does
// not match *wide returns at once.
template <bool kWide>
__global__ void __launch_bounds__(kUThreads)
st_unpart(SegParams p, const uint32_t* __restrict__ Pk, const uint32_t* __restrict__ wide,
          uint32_t* zc, int64_t* zS, int64_t* __restrict__ ctot, uint8_t* __restrict__ sw,
          int64_t nblk) {
  __shared__ int64_t sv[kSC];
  __shared__ uint64_t wtot[kUWaves];
  const uint32_t lane = __lane_id(), wave = threadIdx.x >> 6;
  const int64_t q0 = int64_t(wave) * (kURows * 64) + lane;
  if ((*wide != 0u) != kWide) return;  // uniform
  SpanRegs g;
  span_load<kWide>(p, Pk, zS, zc, blockIdx.x, nblk, g);
  for (int64_t b = blockIdx.x; b < nblk; b += gridDim.x) {
    const int64_t i = b / p.nsc, c = b - i * p.nsc;
    const int64_t len = span_len(p, i, c);
#pragma unroll
    for (int u = 0; u < kURows; ++u)
      if (int64_t(u) * kUThreads + threadIdx.x < len) sv[g.j[u] & kJMask] = g.z[u];
    __syncthreads();
    // the next span's entries are in flight while this one is scanned
    span_load<kWide>(p, Pk, zS, zc, b + gridDim.x, nblk, g);
    // the wave's total first, so that each row is written as soon as it is scanned
    uint64_t lsum = 0;
#pragma unroll 4
    for (int u = 0; u < kURows; ++u)
      lsum += q0 + u * 64 < len ? uint64_t(sv[q0 + u * 64]) : 0ull;
    const uint64_t wsum = read_lane64(wave_inclusive_scan64(lsum), 63);
    if (lane == 0) wtot[wave] = wsum;
    __syncthreads();
    uint64_t carry = 0;
    for (uint32_t w = 0; w < wave; ++w) carry += wtot[w];
    auto span_total = [&]() {
      uint64_t t = 0;
      for (int w = 0; w < kUWaves; ++w) t += wtot[w];
      return read_lane64(t, 0);  // the same in every lane: held once per wave
    };
    bool s64 = true;  // uniform
    if constexpr (!kWide) s64 = span_total() >= (uint64_t(1) << 32);
    int64_t* row = zS + i * p.M_max + (c << kScShift);
    uint32_t* row32 = zc + i * p.M_max + (c << kScShift);
#pragma unroll 4
    for (int u = 0; u < kURows; ++u) {
      const bool in = q0 + u * 64 < len;
      const uint64_t v = wave_inclusive_scan64(in ? uint64_t(sv[q0 + u * 64]) : 0ull) + carry;
      if (in) {
        if (s64) stream_store(row + q0 + u * 64, int64_t(v));
        else stream_store(row32 + q0 + u * 64, uint32_t(v));
      }
      carry = read_lane64(v, 63);
    }
    if (threadIdx.x == 0) {
      ctot[b] = int64_t(span_total());
      sw[b] = s64 ? 1 : 0;
    }
    __syncthreads();  // sv and wtot are rewritten for the next span
  }
}

// In place: ctot[i][c] becomes the sum of the sizes in the spans before c.
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

// The span prefix sums (4-byte S32 or 8-byte S by span, as st_unpart
// marked them in sw).
struct SpanSums {
  const int64_t* S;
  const uint32_t* S32;
  const uint8_t* sw;  // per span of a row
};

// Prefix sums along row i of R: at(x) = sum of the sizes at positions 0..x.
struct Prefix {
  const int64_t* S;     // row i of S (prefix sums local to each span)
  const uint32_t* S32;  // row i of S32
  const uint8_t* sw;    // row i of the span marks
  const int64_t* base;  // row i of the span bases
  __device__ __forceinline__ int64_t at(int64_t x) const {
    if (x < 0) return 0;
    const int64_t c = x >> kScShift;
    const uint32_t lo = S32[x];  // requested with the mark; the 8-byte value only if marked
    const uint64_t v = sw[c] ? uint64_t(S[x]) : uint64_t(lo);
    return int64_t(uint64_t(base[c]) + v);
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
                                             const SpanSums& ss, const int64_t* base) {
  Prefix P;
  P.S = ss.S + i * p.M_max;
  P.S32 = ss.S32 + i * p.M_max;
  P.sw = ss.sw + i * int64_t(nch);
  P.base = base + i * int64_t(nch);
  return P;
}

__device__ __forceinline__ int64_t sub_sat(int64_t a, int64_t b) {
  // a - b without overflow (b >= 0)
  return a < INT64_MIN + b ? INT64_MIN : a - b;
}

constexpr int kStThreads = 512;
constexpr int kStPer = 8;
constexpr int64_t kStChunk = int64_t(kStThreads) * kStPer;  // 4096 positions
constexpr int kStParts = int(kSC / kStChunk);                // quarters of a span
constexpr int kStPad = kStChunk + kStChunk / kStPer;        // LDS slots with one pad per 8
constexpr int kGCap = 5120;                                  // g values staged in LDS
constexpr int kGPerT = (kGCap + kStThreads - 1) / kStThreads;  // staged g values per thread

static_assert(kStParts * kStChunk == kSC, "staging quarters");
static_assert(kGCap < kSC, "a staged g range spans at most two spans");

__device__ __forceinline__ int lds_slot(int p) { return p + (p >> 3); }

// Block b of the fill covers quarter `part` of span c of worker i:
// positions [h0, h0 + hl) of row i (hl may be 0).
struct FillPart {
  int64_t i, c, q, h0, hl;
};

__device__ __forceinline__ FillPart fill_part(const SegParams& p, uint32_t nch, int64_t b) {
  FillPart f;
  const int64_t per = int64_t(nch) * kStParts;
  f.i = b / per;
  f.q = b - f.i * per;
  f.c = f.q / kStParts;
  f.h0 = f.q * kStChunk;
  const int64_t len = seg_len(p, f.i) - f.h0;
  f.hl = len < 0 ? 0 : (len > kStChunk ? kStChunk : len);
  return f;
}

// bnd[b] = (g of the part's first position, g of its last position, 0, 0).
__global__ void __launch_bounds__(256)
st_bounds(SegParams p, int64_t d0, uint32_t nch, int64_t nparts, SpanSums S,
          const int64_t* __restrict__ base, int4* __restrict__ bnd) {
  const int64_t b = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (b >= nparts) return;
  const FillPart f = fill_part(p, nch, b);
  if (f.hl == 0) {
    bnd[b] = make_int4(0, -1, 0, 0);
    return;
  }
  const Prefix P = row_prefix(p, f.i, nch, S, base);
  const int64_t h1 = f.h0 + f.hl - 1;
  const int64_t glo = P.lower_bound(f.h0, sub_sat(P.at(f.h0), d0));
  const int64_t ghi = P.lower_bound(h1, sub_sat(P.at(h1), d0));
  bnd[b] = make_int4(int32_t(glo), int32_t(ghi), 0, 0);
}

__global__ void __launch_bounds__(kStThreads) __attribute__((amdgpu_waves_per_eu(8)))
st_fill(SegParams p, int64_t d0, uint32_t nch, int64_t nparts, SpanSums S,
        const int64_t* __restrict__ base, const int4* __restrict__ bnd, int32_t gcap,
        int32_t* __restrict__ fill) {
  // the staged g values, then (after a barrier) the results for the transpose
  __shared__ int64_t gS[kGCap];
  static_assert(kStPad * sizeof(int32_t) <= sizeof(gS), "result staging fits");
  int32_t* fo = reinterpret_cast<int32_t*>(gS);
  const int64_t b = xcd_logical(blockIdx.x, gridDim.x);
  if (b >= nparts) return;
  const FillPart f = fill_part(p, nch, b);
  int32_t* out = fill + f.i * p.M_max;
  if (f.q == 0) {
    // the row's padding past its last read
    for (int64_t h = seg_len(p, f.i) + threadIdx.x; h < p.M_max; h += kStThreads)
      out[h] = -1;
  }
  if (f.hl == 0) return;
  const int64_t* Srow = S.S + f.i * p.M_max;
  const uint32_t* S32row = S.S32 + f.i * p.M_max;
  const uint8_t* swrow = S.sw + f.i * int64_t(nch);
  const int64_t* brow = base + f.i * int64_t(nch);
  // the part's g range first: the staging loads below wait for it
  const int4 bb = bnd[b];
  const int64_t hbase = brow[f.c];  // every position of the part is in span c
  const bool wc = swrow[f.c] != 0;  // uniform
  // this thread's positions: prefix sums within span c (the 4-byte values
  // requested with the span's mark; the 8-byte ones only for a marked span)
  const int32_t ht0 = int32_t(threadIdx.x) * kStPer;  // offset in the part
  const int32_t hl = int32_t(f.hl);
  int64_t sh[kStPer];
  static_assert(kStPer % 4 == 0, "whole 16-byte loads");
  if (ht0 + kStPer <= hl) {  // 16-byte loads (4-byte aligned)
#pragma unroll
    for (int u = 0; u < kStPer; u += 4) {
      uint4 w;
      __builtin_memcpy(&w, S32row + f.h0 + ht0 + u, 16);
      sh[u] = w.x;
      sh[u + 1] = w.y;
      sh[u + 2] = w.z;
      sh[u + 3] = w.w;
    }
  } else {
#pragma unroll
    for (int u = 0; u < kStPer; ++u)  // unconditional: past the part's end, its last position
      sh[u] = int64_t(S32row[f.h0 + (ht0 + u < hl ? ht0 + u : hl - 1)]);
  }
  if (wc) {
#pragma unroll
    for (int u = 0; u < kStPer; ++u) sh[u] = Srow[f.h0 + (ht0 + u < hl ? ht0 + u : hl - 1)];
  }
  // S(h) - d0 = (hbase - d0) + sh: sizes are >= 1, so no term saturates
  // (other sizes only need in-bounds results, which the index bounds give)
  const uint64_t hd = uint64_t(hbase) - uint64_t(d0);
  const int64_t glo = bb.x, ghi = bb.y;
  const int64_t Lg = ghi - glo + 1;
  const bool staged = Lg >= 1 && Lg <= gcap;  // uniform over the workgroup
  if (staged) {
    // every load of the range at once (clamped to g >= 0); the range spans
    // at most two spans, whose bases are loaded once
    const int64_t sA = (glo > 0 ? glo : 0) >> kScShift;
    const int64_t sB = sA + 1 < int64_t(nch) ? sA + 1 : sA;
    const int64_t bA = brow[sA];
    const int64_t bB = brow[sB];
    const bool wA = swrow[sA] != 0, wB = swrow[sB] != 0;
    // positions and g values fit 32 bits (rows are int32-indexed)
    const int32_t g0 = int32_t(glo), lg = int32_t(Lg);
    uint32_t gv[kGPerT];
#pragma unroll
    for (int u = 0; u < kGPerT; ++u) {
      const int32_t x = u * kStThreads + int32_t(threadIdx.x);
      gv[u] = S32row[x < lg && g0 + x > 0 ? g0 + x : 0];
    }
#pragma unroll
    for (int u = 0; u < kGPerT; ++u) {
      const int32_t x = u * kStThreads + int32_t(threadIdx.x);
      const int32_t g = g0 + x;
      if (x < lg)
        gS[x] = g >= 0 ? int64_t(uint64_t((g >> kScShift) == sA ? bA : bB) + uint64_t(gv[u])) : 0;
    }
    if (wA || wB) {  // a span marked 8-byte (uniform; not at the workloads here)
#pragma unroll 1
      for (int u = 0; u < kGPerT; ++u) {
        const int32_t x = u * kStThreads + int32_t(threadIdx.x);
        const int32_t g = g0 + x;
        const bool inA = (g >> kScShift) == sA;
        if (x < lg && g >= 0 && (inA ? wA : wB))
          gS[x] = int64_t(uint64_t(inA ? bA : bB) + uint64_t(Srow[g]));
      }
    }
  }
  __syncthreads();
  int32_t res[kStPer];
  if (staged) {
    // the staged range is read by every thread: the results wait for the
    // barrier below before they overwrite it
    // 32-bit indices into the staged range; only the sums are 64-bit
    const int32_t g0 = int32_t(glo), lg = int32_t(Lg);
    const int32_t hb = int32_t(f.h0) + ht0;
    int32_t x = 0;
    bool started = false;
#pragma unroll
    for (int u = 0; u < kStPer; ++u) {
      res[u] = -1;
      if (ht0 + u < hl) {
        const int64_t target = int64_t(hd + uint64_t(sh[u]));
        if (!started) {
          int32_t lo = 0, hi = lg;
          while (lo < hi) {
            const int32_t mid = (lo + hi) >> 1;
            if (gS[mid] >= target) hi = mid;
            else lo = mid + 1;
          }
          x = lo < lg ? lo : lg - 1;
          started = true;
        }
        while (x < lg - 1 && gS[x] < target) ++x;
        const int32_t g = g0 + x, h = hb + u;
        const int32_t fv = g + 1 < h ? g + 1 : h;
        res[u] = fv > 0 ? fv : 0;
      }
    }
  } else {
    // g range too wide for LDS (or not monotone): search the row itself,
    // one position at a time (rare: a loop, not unrolled), the results
    // straight into the transpose (nothing reads the staged range here)
    const Prefix P = row_prefix(p, f.i, nch, S, base);
    int64_t x = 0;
#pragma unroll 1
    for (int u = 0; u < kStPer; ++u) {
      const int64_t h = f.h0 + ht0 + u;
      int32_t r = -1;
      if (ht0 + u < f.hl) {
        const int64_t target = sub_sat(P.at(h), d0);
        if (u == 0) x = P.lower_bound(h, target);
        while (x < h && P.at(x) < target) ++x;
        const int64_t fv = x + 1 < h ? x + 1 : h;
        r = int32_t(fv > 0 ? fv : 0);
      }
      fo[lds_slot(threadIdx.x * kStPer + u)] = r;
    }
  }
  __syncthreads();
  if (staged) {
#pragma unroll
    for (int u = 0; u < kStPer; ++u) fo[lds_slot(threadIdx.x * kStPer + u)] = res[u];
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kStPer; ++u) {
    const int q = u * kStThreads + threadIdx.x;
    if (q < f.hl) stream_store(out + f.h0 + q, fo[lds_slot(q)]);
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
  // one segment per row: the E epochs folded together, cut into spans
  // windows of 2^15 samples: one LDS pass of 4-byte sizes, two of 8-byte
  // ones (at most 2^18: the packed partition entries hold 18 bits of offset)
  SegParams p = seg_params(s, gather_ws() + 1 < 18 ? gather_ws() + 1 : 18);
  const uint32_t nch = uint32_t(ceil_div(s.M_max, kSC));  // spans per row
  p.emul = int32_t(s.E);
  p.E = 1;
  p.nsc = int32_t(nch);
  const int64_t nblk = s.N * int64_t(nch);
  const int64_t nparts = nblk * kStParts;
  const uint32_t ngroups = gather_ngroups(s.N);
  const int64_t ntiles = int64_t(p.nbk) * ngroups;
  if (nparts >= (int64_t(1) << 31) || ntiles >= (int64_t(1) << 31))
    return fail(NOPFS_ERANGE, "job too large for one launch");
  Scratch scr(st);
  uint32_t *Pk, *zc, *wide;
  uint16_t* OT;
  int64_t *S, *ctot;
  uint8_t* sw;
  int4* bnd;
  if ((rc = scr.alloc_n(&wide, 1))) return rc;
  if ((rc = launch("st_flag", st_flag, dim3(1), dim3(1), 0, st, wide))) return rc;
  if ((rc = launch("st_range", st_range, dim3(uint32_t(ceil_div(s.F, 1024))), dim3(256), 0, st, s.F,
                   sizes, wide)))
    return rc;
  if ((rc = run_partition(p, R, scr, &Pk, &OT, st))) return rc;
  if ((rc = scr.alloc_n(&S, size_t(s.N * s.M_max)))) return rc;
  if ((rc = scr.alloc_n(&zc, size_t(s.N * s.M_max)))) return rc;
  if ((rc = scr.alloc_n(&ctot, size_t(nblk)))) return rc;
  if ((rc = scr.alloc_n(&sw, size_t(nblk)))) return rc;
  if ((rc = scr.alloc_n(&bnd, size_t(nparts)))) return rc;
  if ((rc = launch("st_gather", st_gather, dim3(xcd_padded(uint32_t(ntiles))), dim3(kGThreads), 0,
                   st, p, (const uint32_t*)Pk, (const uint16_t*)OT, sizes, (const uint32_t*)wide, zc,
                   S, ngroups, uint32_t(ntiles))))
    return rc;
  const int64_t ugrid = nblk < 1024 ? nblk : 1024;
  if ((rc = launch("st_unpart", st_unpart<false>, dim3(uint32_t(ugrid)), dim3(kUThreads), 0, st, p,
                   (const uint32_t*)Pk, (const uint32_t*)wide, zc, S, ctot, sw, nblk)))
    return rc;
  if ((rc = launch("st_unpart8", st_unpart<true>, dim3(uint32_t(ugrid)), dim3(kUThreads), 0, st, p,
                   (const uint32_t*)Pk, (const uint32_t*)wide, zc, S, ctot, sw, nblk)))
    return rc;
  if ((rc = launch("st_base", st_base, dim3(uint32_t(s.N)), dim3(1024), 0, st, nch, ctot))) return rc;
  const SpanSums ss{S, zc, sw};
  if ((rc = launch("st_bounds", st_bounds, dim3(uint32_t(ceil_div(nparts, 256))), dim3(256), 0, st,
                   p, d0, nch, nparts, ss, (const int64_t*)ctot, bnd)))
    return rc;
  const int32_t gcap = (debug_value(4) > 0 && debug_value(4) < kGCap) ? int32_t(debug_value(4)) : kGCap;
  return launch("st_fill", st_fill, dim3(xcd_padded(uint32_t(nparts))), dim3(kStThreads), 0, st, p,
                d0, nch, nparts, ss, (const int64_t*)ctot, (const int4*)bnd, gcap, fill);
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
