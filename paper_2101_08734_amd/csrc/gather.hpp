// Window-major pass over the partition of R for per-sample values: for every
// read, a value taken from its sample's window (held in LDS) is written at
// the read's place in the partitioned row. Used by the staging schedule
// (each read's size) and by the fetch model (each read's size and source).
//
// The rows are folded into one segment (E = 1 in SegParams, the epochs
// counted by emul), so run c of a row is the window's reads inside span c
// of 2^14 positions. A tile is (window of 2^14 samples, group of kGRows
// rows); tiles are window-major, so the groups of one window and the tiles
// of neighbouring windows (whose runs adjoin in memory) run together on one
// XCD. Consecutive threads take consecutive reads of the tile's runs, so
// loads and stores go out in run-long pieces (19 reads on average at
// ImageNet-22k) instead of one store per lane into 64 different runs.
#pragma once

#include "partition.hpp"

namespace nopfs {

constexpr int kGatherWs = 14;                 // window: 2^14 samples of 8-byte values
constexpr int kGatherWin = 1 << kGatherWs;    // 8-byte values held in LDS (128 KB)
constexpr int kGThreads = 1024;
constexpr int kGRows = 32;                    // rows per tile
constexpr int kGRuns = 1024;                  // runs per pass of a tile
static_assert(kGRuns % kGThreads == 0, "gather tile shape");

// kChunk: reads per inner pass (the run index map); each thread requests
// kChunk / kGThreads reads of the pass at once.
template <int kChunk>
struct GatherLds {
  static_assert(kChunk % kGThreads == 0, "gather tile shape");
  union {
    uint64_t win[kGatherWin];        // the window's 8-byte values
    uint32_t win4[2 * kGatherWin];   // or 4-byte values, twice as many
  };
  uint32_t pref[kGRuns + 1];  // reads before each run of the pass
  int32_t rpos[kGRuns];       // span start + run start, in the row
  uint8_t rrow[kGRuns];       // row - first row of the tile
  uint16_t run_of[kChunk];    // run of each read of the inner pass
  uint32_t tmp[65];
};

inline uint32_t gather_ngroups(int64_t N) { return uint32_t(ceil_div(N, kGRows)); }

// Window width (log2) of a gather pass: kGatherWs, or wider by the test
// hook's doublings (at most 4: the packed partition entries hold 18 bits of
// offset), so that small jobs take the several-pass path of larger ones.
inline int gather_ws() {
  const int64_t x = debug_value(5);
  return kGatherWs + int(x > 0 ? (x < 4 ? x : 4) : 0);
}

// Tile `tile` of the pass. value(k) gives sample k's value of type V (8 or
// 4 bytes; it is called for k in [0, F) only); emit(pos, row, x, w0, wl)
// receives kChunk / kGThreads reads of this thread at once: pos[u] the read's index in the
// row table ([N][M_max], -1 for none), row[u] its row, x[u] its sample's
// offset in the window pass starting at sample w0 (valid when x[u] < wl),
// with the window's values in L.win (V = uint64_t) or L.win4 (uint32_t).
template <typename V, int kChunk, typename Value, typename Emit>
__device__ __forceinline__ void gather_tile(const SegParams& p, const uint32_t* __restrict__ Pk,
                                            const uint16_t* __restrict__ OT, uint32_t tile,
                                            uint32_t ngroups, GatherLds<kChunk>& L, Value value,
                                            Emit emit) {
  constexpr int kPer = kChunk / kGThreads;
  const uint32_t kb = tile / ngroups;
  const int64_t i0 = int64_t(tile - kb * ngroups) * kGRows;
  const int64_t rows = p.N - i0 < kGRows ? p.N - i0 : kGRows;
  const int64_t nch = p.nsc;
  const int64_t nruns = rows * nch;  // < 2^31
  const int64_t k0 = int64_t(kb) << p.ws;
  const int64_t kend = k0 + (int64_t(1) << p.ws) < p.F ? k0 + (int64_t(1) << p.ws) : p.F;
  constexpr int kWin = int(kGatherWin * sizeof(uint64_t) / sizeof(V));  // values per pass
  V* win = sizeof(V) == 8 ? reinterpret_cast<V*>(L.win) : reinterpret_cast<V*>(L.win4);
  for (int64_t w0 = k0; w0 < kend; w0 += kWin) {  // one pass unless windows are wider
    const uint32_t wl = uint32_t(kend - w0 < kWin ? kend - w0 : kWin);
    const uint32_t xoff = uint32_t(w0 - k0);
    // the window's values, sixteen loads per thread in flight at once
    for (uint32_t x0 = 0; x0 < wl; x0 += 16 * kGThreads) {
      V v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const uint32_t x = x0 + u * kGThreads + threadIdx.x;
        v[u] = value(w0 + (x < wl ? x : 0));
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const uint32_t x = x0 + u * kGThreads + threadIdx.x;
        if (x < wl) win[x] = v[u];
      }
    }
    for (int64_t r0 = 0; r0 < nruns; r0 += kGRuns) {
      const uint32_t nr = uint32_t(nruns - r0 < kGRuns ? nruns - r0 : kGRuns);
      uint32_t len[kGRuns / kGThreads];
      uint32_t sum = 0;
#pragma unroll
      for (int m = 0; m < kGRuns / kGThreads; ++m) {
        const uint32_t r = threadIdx.x * (kGRuns / kGThreads) + m;
        // loads for runs past nr read run r0's bounds and are dropped
        const uint32_t rr = uint32_t(r0) + (r < nr ? r : 0u);
        const uint32_t il = rr / uint32_t(nch), c = rr - il * uint32_t(nch);
        const uint16_t* o = OT + ((i0 + il) * (p.nbk + 1) + kb) * nch + c;
        const uint32_t a = o[0], b = o[nch];
        len[m] = r < nr ? b - a : 0u;
        if (r < nr) {
          L.rpos[r] = int32_t((int64_t(c) << kScShift) + a);
          L.rrow[r] = uint8_t(il);
        }
        sum += len[m];
      }
      uint32_t total;
      uint32_t run = block_exclusive_scan<false>(sum, L.tmp, &total);  // closed below
#pragma unroll
      for (int m = 0; m < kGRuns / kGThreads; ++m) {
        L.pref[threadIdx.x * (kGRuns / kGThreads) + m] = run;
        run += len[m];
      }
      if (threadIdx.x == 0) L.pref[nr] = total;
      __syncthreads();
      for (uint32_t x0 = 0; x0 < total; x0 += kChunk) {
        const uint32_t xl = total - x0 < kChunk ? total - x0 : kChunk;
        // run index of every read of the inner pass, written by the runs' owners
#pragma unroll
        for (int m = 0; m < kGRuns / kGThreads; ++m) {
          const uint32_t r = threadIdx.x * (kGRuns / kGThreads) + m;
          if (r < nr) {
            const uint32_t a = L.pref[r] > x0 ? L.pref[r] - x0 : 0u;
            const uint32_t e = L.pref[r + 1] - x0 < xl ? L.pref[r + 1] - x0 : xl;
            for (uint32_t y = a; y < e && L.pref[r + 1] > x0; ++y) L.run_of[y] = uint16_t(r);
          }
        }
        __syncthreads();
        int64_t pos[kPer], row[kPer];
        uint32_t x[kPer];
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
          const uint32_t t = u * kGThreads + threadIdx.x;
          pos[u] = -1;
          row[u] = i0;
          if (t < xl) {
            const uint32_t r = L.run_of[t];
            row[u] = i0 + L.rrow[r];
            pos[u] = row[u] * p.M_max + L.rpos[r] + (x0 + t - L.pref[r]);
          }
        }
#pragma unroll
        for (int u = 0; u < kPer; ++u) x[u] = Pk[pos[u] >= 0 ? pos[u] : 0];  // unconditional
#pragma unroll
        for (int u = 0; u < kPer; ++u) x[u] = pos[u] >= 0 ? (x[u] >> kScShift) - xoff : 0xFFFFFFFFu;
        emit(pos, row, x, w0, wl);
        __syncthreads();
      }
    }
    __syncthreads();
  }
}

}  // namespace nopfs
