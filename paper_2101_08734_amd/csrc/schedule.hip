// nopfs_prefetch_order and nopfs_staging_schedule: what the Design section
// derives from the streams and the placement for a worker's prefetchers.
//
// Prefetch order. Each storage class is filled in the order the worker first
// needs its samples (the first rule of optimal prefetching, I/O Access
// Patterns section). Tier t's queue holds the samples placed in t that the
// worker reads, by first read; the queues are concatenated fastest tier first.
//   pf_mark   -- every cell (i, k) with a first read f and a cache tier t
//                marks its stream position: mark[i][f] = t + 1 (one byte per
//                position). Tiles are worker-major and grouped per XCD, so a
//                worker's mark row (one byte per read) stays in one L2 while
//                its cells are visited.
//   pf_count  -- per (worker, chunk of 2048 positions, one wave each): marks
//                per tier.
//   pf_scan   -- per worker and tier: exclusive scan over chunks plus the
//                start of the tier's queue; the queue lengths.
//   pf_write  -- per chunk, in stream order: each wave step of 64 positions
//                splits its marked positions by tier (one ballot per tier
//                present) and writes R[i][f] to the next queue slots; then
//                the chunk's share of the -1 padding after the queues.
// Staging schedule. The staging buffer is filled in stream order and a
// sample is dropped once read (Design); it is filled circularly
// (Implementation). With S the prefix sum of the sizes along R_i (S(-1) = 0),
// the sample at h may be fetched once the worker has read position
// fill(h) - 1: fill(h) is the smallest f <= h with S(h) - S(f - 1) <= d0,
// or h when the sample alone is larger than d0. Equivalently fill(h) is one
// past the smallest g in [-1, h] with S(g) >= S(h) - d0, capped at h.
//   st_sum    -- per (worker, chunk of 4096 positions): the sizes of the
//                samples read, their inclusive prefix sums inside the chunk
//                and the chunk total.
//   st_base   -- per worker: exclusive scan of the chunk totals.
//   st_bounds -- per chunk: the g of its first and of its last position
//                (binary search over S; g never decreases along R).
//   st_fill   -- per chunk: S over that g range is staged in LDS, each thread
//                binary-searches the g of its first position there and walks
//                its other positions with two pointers; -1 in padding.
#include <new>

#include "common.hpp"

namespace nopfs {
namespace {

struct RowShape {
  int64_t F, N, B, M_max, E;
  int32_t drop_last;
};

__device__ __forceinline__ int64_t row_len(const RowShape& r, int64_t i) {
  return r.E * epoch_len(r.F, r.N, r.B, r.drop_last, i);
}

// ------------------------------------------------------------- prefetch --
constexpr int kPfWaves = 4;                              // waves per workgroup
constexpr int kPfSteps = 32;                             // steps of 64 positions per wave
constexpr int64_t kPfChunk = int64_t(64) * kPfSteps;     // 2048 positions per chunk
constexpr int kPfMaxJ = 128;
constexpr int kMarkGroupsPerThread = 16;                 // 4-cell groups
constexpr int64_t kMarkTile = int64_t(256) * 4 * kMarkGroupsPerThread;  // 16384 cells

__global__ void __launch_bounds__(256) pf_zero(uint4* __restrict__ p, int64_t n16) {
  int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (; t < n16; t += stride) p[t] = make_uint4(0u, 0u, 0u, 0u);
}

// Mark rows have a pitch of mp bytes (a multiple of 16). Marks are plain
// byte stores: atomic ORs on the 4-byte words (executed in L2) measured
// twice as slow.
__device__ __forceinline__ void mark_cell(int32_t f, int32_t t, int64_t M_max, int32_t J,
                                          uint8_t* __restrict__ mr) {
  // first reads outside the row or tiers outside [0, J) are not queued
  if (f >= 0 && f < M_max && t >= 0 && t < J) mr[f] = uint8_t(t + 1);
}

// Mark byte -> tier code in [0, J] (codes above J, which no valid mark
// holds, are dropped so every queue slot stays inside the row).
__device__ __forceinline__ uint32_t mark_code(uint32_t m, int32_t J) {
  return m <= uint32_t(J) ? m : 0u;
}

// Tile (i, sl) covers the flat cells [i*F + sl*kMarkTile, ...) of row i. The
// vector form reads first as int4 and tier as 4-byte words over 4-cell groups
// aligned to the flat index (first 16-byte and tier 4-byte aligned), masking
// the cells of neighbouring rows; the last partial group of the table is read
// cell by cell.
template <bool kVec>
__global__ void __launch_bounds__(256)
pf_mark(RowShape r, int32_t J, const int32_t* __restrict__ first, const int8_t* __restrict__ tier,
        uint8_t* __restrict__ mark, int64_t mp, uint32_t nslices, uint32_t ntiles) {
  const uint32_t t = xcd_logical(blockIdx.x, gridDim.x);
  if (t >= ntiles) return;
  const int64_t i = t / nslices;
  const int64_t sl = t - i * nslices;
  const int64_t row0 = i * r.F;
  const int64_t lo = row0 + sl * kMarkTile;
  const int64_t hi = lo + kMarkTile < row0 + r.F ? lo + kMarkTile : row0 + r.F;
  uint8_t* mr = mark + i * mp;
  if (!kVec) {
    for (int64_t x = lo + threadIdx.x; x < hi; x += 256)
      mark_cell(first[x], tier[x], r.M_max, J, mr);
    return;
  }
  const int64_t NF = r.N * r.F;
  const int64_t gfull = NF >> 2;  // groups lying wholly inside the table
  const int64_t g0 = lo >> 2, g1 = (hi + 3) >> 2;
  const int4* f4 = reinterpret_cast<const int4*>(first);
  const uint32_t* t4 = reinterpret_cast<const uint32_t*>(tier);
  constexpr int kBatch = 4;
  for (int64_t gb = g0 + threadIdx.x; gb < g1; gb += int64_t(256) * kBatch) {
    int32_t fv[kBatch][4];
    uint32_t tv[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int64_t g = gb + int64_t(b) * 256;
      if (g < g1 && g < gfull) {
        const int4 a = f4[g];
        fv[b][0] = a.x;
        fv[b][1] = a.y;
        fv[b][2] = a.z;
        fv[b][3] = a.w;
        tv[b] = t4[g];
      } else {
        tv[b] = 0xFFFFFFFFu;  // tier -1: nothing queued
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int64_t x = g * 4 + q;
          const bool in = g < g1 && x < NF;
          fv[b][q] = in ? first[x] : -1;
          if (in) tv[b] = (tv[b] & ~(0xFFu << (8 * q))) | (uint32_t(uint8_t(tier[x])) << (8 * q));
        }
      }
    }
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int64_t g = gb + int64_t(b) * 256;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t x = g * 4 + q;
        if (x >= lo && x < hi)
          mark_cell(fv[b][q], int32_t(int8_t(uint8_t(tv[b] >> (8 * q)))), r.M_max, J, mr);
      }
    }
  }
}

// Logical block id -> (worker, block of kPfWaves chunks), worker-major per XCD.
__device__ __forceinline__ bool pf_block(uint32_t nbw, uint32_t nblocks, int64_t* i, uint32_t* cb) {
  const uint32_t t = xcd_logical(blockIdx.x, gridDim.x);
  if (t >= nblocks) return false;
  *i = t / nbw;
  *cb = t - uint32_t(*i) * nbw;
  return true;
}

// cnt layout: [N][nch][J]. Each wave counts one chunk; no workgroup barrier.
__global__ void __launch_bounds__(256)
pf_count(RowShape r, int32_t J, const uint8_t* __restrict__ mark, int64_t mp, uint32_t nch,
         uint32_t nbw, uint32_t nblocks, int32_t* __restrict__ cnt) {
  __shared__ uint32_t s_cnt[kPfWaves][kPfMaxJ];
  int64_t i;
  uint32_t cb;
  if (!pf_block(nbw, nblocks, &i, &cb)) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint32_t c = cb * kPfWaves + w;
  if (c >= nch) return;
  for (int x = lane; x < J; x += 64) s_cnt[w][x] = 0;
  const int64_t Mi = row_len(r, i);
  const uint8_t* mr = mark + i * mp;
  const int64_t f0 = int64_t(c) * kPfChunk + lane;
  uint32_t code[kPfSteps];
#pragma unroll
  for (int u = 0; u < kPfSteps; ++u) {
    const int64_t f = f0 + int64_t(u) * 64;
    code[u] = f < Mi ? mark_code(mr[f], J) : 0u;
  }
#pragma unroll
  for (int u = 0; u < kPfSteps; ++u) {
    uint64_t act = __ballot(code[u] != 0);
    while (act) {
      const int lead = __builtin_ctzll(act);
      const uint32_t tc = __builtin_amdgcn_readlane(code[u], lead);
      const uint64_t same = __ballot(code[u] == tc);
      if (lane == lead) s_cnt[w][tc - 1] += uint32_t(__popcll(same));
      act &= ~same;
    }
  }
  int32_t* out = cnt + (i * nch + c) * J;
  for (int x = lane; x < J; x += 64) out[x] = int32_t(s_cnt[w][x]);
}

// In place: cnt[i][c][j] becomes the queue slot (within row i of order) of
// chunk c's first tier-j sample; qlen[i][j] the queue lengths; tot[i] their sum.
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

__global__ void __launch_bounds__(256)
pf_write(RowShape r, int32_t J, const uint8_t* __restrict__ mark, int64_t mp,
         const int32_t* __restrict__ R, uint32_t nch, uint32_t nbw, uint32_t nblocks,
         const int32_t* __restrict__ slot0, const int64_t* __restrict__ tot,
         int32_t* __restrict__ order) {
  __shared__ int32_t s_run[kPfWaves][kPfMaxJ];
  int64_t i;
  uint32_t cb;
  if (!pf_block(nbw, nblocks, &i, &cb)) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint32_t c = cb * kPfWaves + w;
  if (c >= nch) return;
  const int32_t* sl = slot0 + (i * nch + c) * J;
  for (int x = lane; x < J; x += 64) s_run[w][x] = sl[x];
  const int64_t Mi = row_len(r, i);
  const uint8_t* mr = mark + i * mp;
  const int32_t* Rr = R + i * r.M_max;
  int32_t* orow = order + i * r.M_max;
  const int64_t f0 = int64_t(c) * kPfChunk + lane;
  uint32_t code[kPfSteps];
#pragma unroll
  for (int u = 0; u < kPfSteps; ++u) {
    const int64_t f = f0 + int64_t(u) * 64;
    code[u] = f < Mi ? mark_code(mr[f], J) : 0u;
  }
  int32_t k[kPfSteps];
#pragma unroll
  for (int u = 0; u < kPfSteps; ++u) k[u] = code[u] ? Rr[f0 + int64_t(u) * 64] : 0;
  const uint64_t below = lanemask_lt();
#pragma unroll
  for (int u = 0; u < kPfSteps; ++u) {
    uint64_t act = __ballot(code[u] != 0);
    while (act) {
      const int lead = __builtin_ctzll(act);
      const uint32_t tc = __builtin_amdgcn_readlane(code[u], lead);
      const uint64_t same = __ballot(code[u] == tc);
      const int32_t run = s_run[w][tc - 1];
      if (code[u] == tc) orow[run + __popcll(same & below)] = k[u];
      if (lane == lead) s_run[w][tc - 1] = run + __popcll(same);
      act &= ~same;
    }
  }
  // padding after the last queue, within this chunk's range of the row
  const int64_t q0 = int64_t(c) * kPfChunk;
  const int64_t q1 = q0 + kPfChunk < r.M_max ? q0 + kPfChunk : r.M_max;
  const int64_t T = tot[i];
  for (int64_t q = (T > q0 ? T : q0) + lane; q < q1; q += 64) orow[q] = -1;
}

// -------------------------------------------------------------- staging --
constexpr int kStThreads = 256;
constexpr int kStPer = 16;
constexpr int kStShift = 12;
constexpr int64_t kStChunk = int64_t(1) << kStShift;  // 4096 positions = 256 * 16
constexpr int kStPad = kStChunk + kStChunk / kStPer;  // LDS slots with one pad per 16
constexpr int kGCap = 6144;                            // g values staged in LDS

static_assert(kStThreads * kStPer == kStChunk, "staging chunk");

__device__ __forceinline__ int lds_slot(int p) { return p + (p >> 4); }

// S is chunk-local: S[i*Sp + f] = sum of the sizes at the positions of f's
// chunk up to and including f. Sp is a multiple of kStChunk.
__global__ void __launch_bounds__(kStThreads)
st_sum(RowShape r, const int32_t* __restrict__ R, const int64_t* __restrict__ sizes,
       uint32_t nch, int64_t Sp, int64_t* __restrict__ S, int64_t* __restrict__ ctot) {
  __shared__ int64_t sv[kStPad];
  __shared__ uint64_t tmp[65];
  const uint32_t t = xcd_logical(blockIdx.x, gridDim.x);
  if (t >= uint32_t(r.N) * nch) return;
  const int64_t i = t / nch;
  const int64_t c = t - i * nch;
  const int64_t Mi = row_len(r, i);
  const int64_t f0 = c * kStChunk;
  const int32_t* Rr = R + i * r.M_max;
  int32_t k[kStPer];
#pragma unroll
  for (int u = 0; u < kStPer; ++u) {
    const int64_t f = f0 + u * kStThreads + threadIdx.x;
    k[u] = f < Mi ? Rr[f] : -1;
  }
#pragma unroll
  for (int u = 0; u < kStPer; ++u) {
    // entries outside [0, F) break the precondition; they weigh nothing
    const int64_t s = (k[u] >= 0 && k[u] < r.F) ? sizes[k[u]] : 0;
    sv[lds_slot(u * kStThreads + threadIdx.x)] = s;
  }
  __syncthreads();
  uint64_t v[kStPer];
  uint64_t run = 0;
#pragma unroll
  for (int u = 0; u < kStPer; ++u) {
    run += uint64_t(sv[lds_slot(threadIdx.x * kStPer + u)]);
    v[u] = run;
  }
  uint64_t total;
  const uint64_t ex = block_exclusive_scan64(run, tmp, &total);
#pragma unroll
  for (int u = 0; u < kStPer; ++u) sv[lds_slot(threadIdx.x * kStPer + u)] = int64_t(ex + v[u]);
  __syncthreads();
  int64_t* Sr = S + i * Sp;
#pragma unroll
  for (int u = 0; u < kStPer; ++u) {
    const int p = u * kStThreads + threadIdx.x;
    if (f0 + p < Mi) Sr[f0 + p] = sv[lds_slot(p)];
  }
  if (threadIdx.x == 0) ctot[i * nch + c] = int64_t(total);
}

// In place: ctot[i][c] becomes the sum of the sizes in the chunks before c.
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

struct Prefix {
  const int64_t* S;     // row i of S
  const int64_t* base;  // row i of the chunk bases
  // sum of the sizes at positions 0..x of the row; 0 at x = -1
  __device__ __forceinline__ int64_t at(int64_t x) const {
    return x < 0 ? 0 : int64_t(uint64_t(base[x >> kStShift]) + uint64_t(S[x]));
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

__device__ __forceinline__ int64_t sub_sat(int64_t a, int64_t b) {
  // a - b without overflow (b >= 0)
  return a < INT64_MIN + b ? INT64_MIN : a - b;
}

// bnd[i][c] = (g of the chunk's first position, g of its last position).
__global__ void __launch_bounds__(256)
st_bounds(RowShape r, int64_t d0, uint32_t nch, int64_t Sp, const int64_t* __restrict__ S,
          const int64_t* __restrict__ base, int2* __restrict__ bnd) {
  const int64_t id = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= r.N * int64_t(nch)) return;
  const int64_t i = id / nch;
  const int64_t c = id - i * nch;
  const int64_t Mi = row_len(r, i);
  const int64_t h0 = c * kStChunk;
  if (h0 >= Mi) {
    bnd[id] = make_int2(0, -1);
    return;
  }
  const int64_t h1 = (h0 + kStChunk < Mi ? h0 + kStChunk : Mi) - 1;
  const Prefix P{S + i * Sp, base + i * int64_t(nch)};
  const int64_t glo = P.lower_bound(h0, sub_sat(P.at(h0), d0));
  const int64_t ghi = P.lower_bound(h1, sub_sat(P.at(h1), d0));
  bnd[id] = make_int2(int32_t(glo), int32_t(ghi));
}

__global__ void __launch_bounds__(kStThreads)
st_fill(RowShape r, int64_t d0, uint32_t nch, int64_t Sp, const int64_t* __restrict__ S,
        const int64_t* __restrict__ base, const int2* __restrict__ bnd, int32_t gcap,
        int32_t* __restrict__ fill) {
  // the staged g values, then (after a barrier) the results for the transpose
  __shared__ int64_t gS[kGCap];
  static_assert(kStPad * sizeof(int32_t) <= sizeof(gS), "result staging fits");
  int32_t* fo = reinterpret_cast<int32_t*>(gS);
  const uint32_t t = xcd_logical(blockIdx.x, gridDim.x);
  if (t >= uint32_t(r.N) * nch) return;
  const int64_t i = t / nch;
  const int64_t c = t - i * nch;
  const int64_t Mi = row_len(r, i);
  const int64_t h0c = c * kStChunk;
  const int64_t hend = h0c + kStChunk < r.M_max ? h0c + kStChunk : r.M_max;
  int32_t* out = fill + i * r.M_max;
  if (h0c >= Mi) {
    for (int64_t h = h0c + threadIdx.x; h < hend; h += kStThreads) out[h] = -1;
    return;
  }
  const int64_t h1c = h0c + kStChunk < Mi ? h0c + kStChunk : Mi;
  const Prefix P{S + i * Sp, base + i * int64_t(nch)};
  const int2 b = bnd[t];
  const int64_t glo = b.x;
  const int64_t Lg = int64_t(b.y) - glo + 1;
  const bool staged = Lg >= 1 && Lg <= gcap;  // uniform over the workgroup (gcap <= kGCap)
  if (staged)
    for (int64_t x = threadIdx.x; x < Lg; x += kStThreads) gS[x] = P.at(glo + x);
  __syncthreads();
  const int64_t ht0 = h0c + int64_t(threadIdx.x) * kStPer;
  const int64_t cb = P.base[c];
  int32_t res[kStPer];
  int64_t x = 0;
  bool started = false;
#pragma unroll
  for (int u = 0; u < kStPer; ++u) {
    const int64_t h = ht0 + u;
    res[u] = -1;
    if (h < h1c) {
      const int64_t target = sub_sat(int64_t(uint64_t(cb) + uint64_t(P.S[h])), d0);
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
      const int64_t f = g + 1 < h ? g + 1 : h;
      res[u] = int32_t(f > 0 ? f : 0);
    }
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kStPer; ++u) fo[lds_slot(threadIdx.x * kStPer + u)] = res[u];
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kStPer; ++u) {
    const int p = u * kStThreads + threadIdx.x;
    const int64_t h = h0c + p;
    if (h < hend) out[h] = h < h1c ? fo[lds_slot(p)] : -1;
  }
}

RowShape row_shape(const Shape& s) {
  RowShape r;
  r.F = s.F;
  r.N = s.N;
  r.B = s.B;
  r.M_max = s.M_max;
  r.E = s.E;
  r.drop_last = s.drop_last;
  return r;
}

int prefetch_impl(const nopfs_job* job, const int32_t* R, const int32_t* first,
                  const int8_t* tier, int32_t J, int32_t* order, int64_t* qlen, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (!first || !tier || !qlen) return fail(NOPFS_EINVAL, "first, tier and qlen must be non-NULL");
  if (s.M_max > 0 && (!R || !order)) return fail(NOPFS_EINVAL, "R and order must be non-NULL");
  if (J < 1) return fail(NOPFS_EINVAL, "J must be >= 1");
  if (J > 127) return fail(NOPFS_ERANGE, "J must be <= 127");
  const RowShape r = row_shape(s);
  const uint32_t nch = uint32_t(ceil_div(s.M_max, kPfChunk));
  const uint32_t nbw = uint32_t(ceil_div(nch, kPfWaves));
  const int64_t nblocks = s.N * int64_t(nbw);
  const int64_t nslices = ceil_div(s.F, kMarkTile);
  if (nblocks >= (int64_t(1) << 31) || s.N * nslices >= (int64_t(1) << 31))
    return fail(NOPFS_ERANGE, "job too large for one launch");
  Scratch scr(st);
  int64_t* tot;
  int32_t* cnt;
  uint8_t* mark;
  const int64_t mp = ceil_div(s.M_max, 16) * 16;  // mark row pitch
  const int64_t nm16 = s.N * mp / 16;
  if ((rc = scr.alloc_n(&tot, size_t(s.N)))) return rc;
  if ((rc = scr.alloc_n(&cnt, size_t(s.N) * nch * size_t(J)))) return rc;
  if ((rc = scr.alloc_n(&mark, size_t(nm16) * 16))) return rc;
  if (nm16 > 0) {
    const int64_t zb = ceil_div(nm16, 256 * 4) < 65536 ? ceil_div(nm16, 256 * 4) : 65536;
    if ((rc = launch("pf_zero", pf_zero, dim3(uint32_t(zb)), dim3(256), 0, st,
                     reinterpret_cast<uint4*>(mark), nm16)))
      return rc;
    const uint32_t ntiles = uint32_t(s.N * nslices);
    const bool vec = (reinterpret_cast<uintptr_t>(first) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(tier) & 3) == 0;
    rc = vec ? launch("pf_mark", pf_mark<true>, dim3(xcd_padded(ntiles)), dim3(256), 0, st, r, J,
                      first, tier, mark, mp, uint32_t(nslices), ntiles)
             : launch("pf_mark", pf_mark<false>, dim3(xcd_padded(ntiles)), dim3(256), 0, st, r, J,
                      first, tier, mark, mp, uint32_t(nslices), ntiles);
    if (rc) return rc;
    if ((rc = launch("pf_count", pf_count, dim3(xcd_padded(uint32_t(nblocks))), dim3(256), 0, st,
                     r, J, (const uint8_t*)mark, mp, nch, nbw, uint32_t(nblocks), cnt)))
      return rc;
  }
  if ((rc = launch("pf_scan", pf_scan, dim3(uint32_t(s.N)), dim3(1024), 0, st, J, nch, cnt, qlen,
                   tot)))
    return rc;
  if (nm16 > 0 &&
      (rc = launch("pf_write", pf_write, dim3(xcd_padded(uint32_t(nblocks))), dim3(256), 0, st, r,
                   J, (const uint8_t*)mark, mp, R, nch, nbw, uint32_t(nblocks),
                   (const int32_t*)cnt, (const int64_t*)tot, order)))
    return rc;
  return NOPFS_OK;
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
  const RowShape r = row_shape(s);
  const uint32_t nch = uint32_t(ceil_div(s.M_max, kStChunk));
  const int64_t nblocks = s.N * int64_t(nch);
  if (nblocks >= (int64_t(1) << 31)) return fail(NOPFS_ERANGE, "job too large for one launch");
  const int64_t Sp = int64_t(nch) * kStChunk;
  Scratch scr(st);
  int64_t *S, *ctot;
  int2* bnd;
  if ((rc = scr.alloc_n(&S, size_t(s.N) * size_t(Sp)))) return rc;
  if ((rc = scr.alloc_n(&ctot, size_t(nblocks)))) return rc;
  if ((rc = scr.alloc_n(&bnd, size_t(nblocks)))) return rc;
  const dim3 grid(xcd_padded(uint32_t(nblocks)));
  if ((rc = launch("st_sum", st_sum, grid, dim3(kStThreads), 0, st, r, R, sizes, nch, Sp, S, ctot)))
    return rc;
  if ((rc = launch("st_base", st_base, dim3(uint32_t(s.N)), dim3(1024), 0, st, nch, ctot))) return rc;
  if ((rc = launch("st_bounds", st_bounds, dim3(uint32_t(ceil_div(nblocks, 256))), dim3(256), 0, st,
                   r, d0, nch, Sp, (const int64_t*)S, (const int64_t*)ctot, bnd)))
    return rc;
  const int32_t gcap = (debug_value(4) > 0 && debug_value(4) < kGCap) ? int32_t(debug_value(4)) : kGCap;
  return launch("st_fill", st_fill, grid, dim3(kStThreads), 0, st, r, d0, nch, Sp,
                (const int64_t*)S, (const int64_t*)ctot, (const int2*)bnd, gcap, fill);
}

}  // namespace
}  // namespace nopfs

extern "C" int nopfs_prefetch_order(const nopfs_job* job, const int32_t* R, const int32_t* first,
                                    const int8_t* tier, int32_t J, int32_t* order, int64_t* qlen,
                                    void* hip_stream) {
  try {
    return nopfs::prefetch_impl(job, R, first, tier, J, order, qlen,
                                static_cast<hipStream_t>(hip_stream));
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
