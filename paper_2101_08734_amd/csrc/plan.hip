// nopfs_tier_plan: frequency-ordered, capacity-limited placement (section 5.1:
// the largest access frequencies go to the fastest storage class, then the
// next class, until the dataset is cached or local storage is full).
//
// Per worker the ranking is (count desc, first asc, id asc), which is the
// order of the 40-bit key  (E - count) << 32 | (count ? first : id)  because
// first reads are distinct stream positions. Tier j ends at the first sample
// that no longer fits ("first misfit"), so the plan is fixed by J cut points
// along the ranking. They are found without sorting the N*F cells:
//
//   plan_binsum  -- bytes of every run of 256 consecutive ids.
//   plan_hist    -- weighted histogram of sizes over rank-ordered bins of the
//                   key, LDS-privatised per (worker, slice of 2^19 samples)
//                   and flushed once per slice. Bins of class count>=1 split
//                   the first-read range; their number per class follows the
//                   expected Binomial(E, L/F) population so crowded classes
//                   get fine bins. Class 0 is binned by id, 256 ids a bin;
//                   the bytes read per class-0 bin are summed per wave and
//                   added to a global array, and plan_cut takes the bin's
//                   total minus those bytes.
//   Both passes over the [N][F] tables read four cells per lane with one
//   32-bit load of counts and one 128-bit load of first reads.
//   plan_cut     -- per worker: prefix sums over bins, then for each tier the
//                   range of bins that can contain its cut (interval
//                   arithmetic: the cut of tier j depends on where tier j-1
//                   ended, known only up to one bin at this point).
//   plan_write   -- every cell's tier from its bin; cells in a candidate bin
//                   get a placeholder and are appended to a per-worker list.
//   plan_resolve -- per worker: the candidates sorted by key in LDS and the
//                   greedy fill replayed over them exactly; writes their
//                   tiers and the bytes used per tier.
//   plan_exact   -- per worker whose candidate list overflowed: an exact
//                   weighted radix select over the full row for every cut,
//                   then a full rewrite of the row (slow, rarely taken).
#include <limits.h>
#include <math.h>

#include <new>
#include <vector>

#include "pipeline.hpp"

namespace nopfs {
namespace {

constexpr int kThreads = 512;
constexpr int64_t kSliceCells = int64_t(1) << 19;  // samples per (worker, slice) tile
constexpr int kClass0Shift = 8;           // 256 ids per class-0 bin
constexpr int kSliceBins0 = int(kSliceCells >> kClass0Shift);
constexpr uint32_t kBins1Budget = 4096;   // bins for classes count >= 1
constexpr int kCandMax = 4096;            // candidate records per worker (LDS sort)
constexpr int kResolveThreads = 1024;
// Tuning knobs of the histogram pass (every value gives identical results).
#ifndef NOPFS_HIST_UNITS
#define NOPFS_HIST_UNITS 4
#endif
#ifndef NOPFS_HIST_SIZES_AHEAD
#define NOPFS_HIST_SIZES_AHEAD 1
#endif
constexpr int kHistU = NOPFS_HIST_UNITS;        // 4-cell units per thread per iteration
constexpr bool kHistSizesAhead = NOPFS_HIST_SIZES_AHEAD != 0;

typedef long long I64x2 __attribute__((ext_vector_type(2)));

struct PlanArgs {
  int64_t F, N, M_max;
  int32_t E, J;
  uint32_t nbin1, nb0, nbin;
  uint32_t btp;  // row pitch of the per-bin tier table (nbin rounded up to 16)
  int32_t cmax;
  uint16_t nbc[256];   // bins of class c (1 <= c <= E)
  int64_t caps[128];
};

__device__ void build_class_table(const PlanArgs& a, ClassTable& t) {
  if (threadIdx.x == 0) {
    uint32_t b = 0;
    for (int c = a.E; c >= 1; --c) {
      const float scale = float(a.nbc[c]) / float(a.M_max > 0 ? a.M_max : 1);
      t.e[c] = make_float2(scale, __uint_as_float((b << 16) | (a.nbc[c] - 1u)));
      b += a.nbc[c];
    }
    t.e[0] = make_float2(0.f, __uint_as_float(b << 16));
    // counts above E break the precondition; they bin like class E
    for (int c = a.E + 1; c < 256; ++c) t.e[c] = t.e[a.E];
  }
  __syncthreads();
}

// The same table computed once into global memory (the fused call's
// counting pass bins the read cells with it).
__global__ void plan_classes(PlanArgs a, ClassTable* g) { build_class_table(a, *g); }


// Rank-ordered bin of a cell; identical in every kernel that uses it.
__device__ __forceinline__ uint32_t bin_of(const PlanArgs& a, const ClassTable& t, uint32_t c,
                                           int32_t f, int64_t k) {
  if (c == 0) return a.nbin1 + uint32_t(k >> kClass0Shift);
  return bin_read(t, c, f);
}

__device__ __forceinline__ uint64_t rank_key(const PlanArgs& a, uint32_t c, int32_t f, int64_t k) {
  if (c > uint32_t(a.E)) c = uint32_t(a.E);
  const uint64_t hi = uint64_t(uint32_t(a.E) - c) << 32;
  return hi | (c ? uint64_t(uint32_t(f)) : uint64_t(k));
}

__global__ void fill_u64(uint64_t* p, int64_t n) {
  int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (; i < n; i += stride) p[i] = 0;
}

__global__ void fill_i32(int32_t* p, int64_t n) {
  int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (; i < n; i += stride) p[i] = 0;
}

// -- histogram -----------------------------------------------------------------
__global__ void __launch_bounds__(256)
plan_binsum(int64_t F, uint32_t nb0, const int64_t* __restrict__ sizes, uint64_t* __restrict__ binsum) {
  const uint32_t b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= nb0) return;
  const int64_t k0 = int64_t(b) << kClass0Shift;
  uint64_t v = 0;
  for (int x = __lane_id(); x < (1 << kClass0Shift); x += 64)
    if (k0 + x < F) v += uint64_t(sizes[k0 + x]);
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  if (__lane_id() == 0) binsum[b] = v;
}

// Cells of row i in [ks, ke): cells before the first flat index that is a
// multiple of 4 ("head") and after the last whole group of 4 ("tail") go
// one per thread; the groups in between go one group per lane. kVec=false
// (unaligned caller buffers) visits every cell one per thread.
struct RowSplit {
  int64_t body0, nunits, tail0;
};

__device__ __forceinline__ RowSplit split_row(int64_t flat0, int64_t ks, int64_t ke, bool vec) {
  RowSplit r;
  if (!vec) {
    r.body0 = ke; r.nunits = 0; r.tail0 = ke;
    return r;
  }
  int64_t head = (4 - (flat0 & 3)) & 3;
  if (head > ke - ks) head = ke - ks;
  r.body0 = ks + head;
  r.nunits = (ke - r.body0) >> 2;
  r.tail0 = r.body0 + 4 * r.nunits;
  return r;
}

template <bool kVec>
__global__ void __launch_bounds__(kThreads)
plan_hist(PlanArgs a, const uint8_t* __restrict__ count, const int32_t* __restrict__ first,
          const int64_t* __restrict__ sizes, uint64_t* __restrict__ Z,
          uint64_t* __restrict__ H, uint32_t nslices) {
  extern __shared__ uint64_t sm[];
  uint64_t* h1 = sm;                              // nbin1 weighted bins
  unsigned long long* zs =                        // read bytes of this slice's class-0 bins
      reinterpret_cast<unsigned long long*>(sm + a.nbin1);
  __shared__ ClassTable ct;
  const uint32_t t = xcd_logical(blockIdx.x, gridDim.x);
  if (t >= uint32_t(a.N) * nslices) return;
  const int64_t sl = t / a.N, i = t - sl * a.N;
  build_class_table(a, ct);
  const int64_t ks = sl * kSliceCells;
  const int64_t ke = ks + kSliceCells < a.F ? ks + kSliceCells : a.F;
  const uint32_t zb0 = uint32_t(ks >> kClass0Shift);
  const uint32_t nz = uint32_t((ke - ks + (1 << kClass0Shift) - 1) >> kClass0Shift);
  for (uint32_t b = threadIdx.x; b < a.nbin1; b += kThreads) h1[b] = 0;
  for (uint32_t b = threadIdx.x; b < nz; b += kThreads) zs[b] = 0;
  __syncthreads();
  const uint8_t* crow = count + i * a.F;
  const int32_t* frow = first + i * a.F;
  auto cell = [&](int64_t k, uint32_t c, int32_t f) {
    if (c != 0) {
      const unsigned long long sz = static_cast<unsigned long long>(sizes[k]);
      atomicAdd(reinterpret_cast<unsigned long long*>(&h1[bin_read(ct, c, f)]), sz);
      atomicAdd(&zs[uint32_t(k >> kClass0Shift) - zb0], sz);
    }
  };
  const RowSplit rs = split_row(i * a.F + ks, ks, ke, kVec);
  for (int64_t k = ks + threadIdx.x; k < rs.body0; k += kThreads) cell(k, crow[k], frow[k]);
  for (int64_t k = rs.tail0 + threadIdx.x; k < ke; k += kThreads) cell(k, crow[k], frow[k]);
  // Body: 4 cells per lane, kHistU units per thread per iteration. The next
  // iteration's count, first and size words are requested before this
  // iteration's are used, so their memory round trip overlaps the work.
  // Sizes are fetched for every cell (two 16-byte loads per unit): a line of
  // sizes almost always holds some read cell, and waiting for the counts
  // before asking for sizes would put a second round trip on the path.
  constexpr int kU = kHistU;
  uint32_t cw[kU];
  int4 fw[kU];
  I64x2 sw[kU][2];
  auto load = [&](int64_t u0) {
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const int64_t u = u0 + j * kThreads + threadIdx.x;
      const int64_t k = rs.body0 + 4 * u;
      cw[j] = 0;
      if (u < rs.nunits) {
        cw[j] = *reinterpret_cast<const uint32_t*>(crow + k);
        fw[j] = *reinterpret_cast<const int4*>(frow + k);
        if (kHistSizesAhead) {
          __builtin_memcpy(&sw[j][0], sizes + k, 16);
          __builtin_memcpy(&sw[j][1], sizes + k + 2, 16);
        }
      }
    }
  };
  if (rs.nunits > 0) load(0);
  for (int64_t u0 = 0; u0 < rs.nunits; u0 += kU * kThreads) {
    uint32_t c[kU];
    int4 f[kU];
    uint64_t sz[kU][4];
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      c[j] = cw[j];
      f[j] = fw[j];
      if (kHistSizesAhead) {
        sz[j][0] = uint64_t(sw[j][0].x);
        sz[j][1] = uint64_t(sw[j][0].y);
        sz[j][2] = uint64_t(sw[j][1].x);
        sz[j][3] = uint64_t(sw[j][1].y);
      }
    }
    if (u0 + kU * kThreads < rs.nunits) load(u0 + kU * kThreads);
    if (!kHistSizesAhead) {
#pragma unroll
      for (int j = 0; j < kU; ++j) {
        const int64_t k = rs.body0 + 4 * (u0 + j * kThreads + threadIdx.x);
#pragma unroll
        for (int q = 0; q < 4; ++q)
          sz[j][q] = ((c[j] >> (8 * q)) & 0xFFu) ? uint64_t(sizes[k + q]) : 0ull;
      }
    }
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const int64_t k = rs.body0 + 4 * (u0 + j * kThreads + threadIdx.x);
      if (c[j] == 0) continue;
      const int32_t fv[4] = {f[j].x, f[j].y, f[j].z, f[j].w};
      // the unit's read bytes, split where its 4 cells cross into the
      // next class-0 bin (at most once)
      const uint32_t z = uint32_t(k >> kClass0Shift) - zb0;
      const uint32_t qcut = uint32_t(((k >> kClass0Shift) + 1) << kClass0Shift) - uint32_t(k);
      uint64_t lo = 0, hi = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t cq = (c[j] >> (8 * q)) & 0xFFu;
        if (cq != 0) {
          atomicAdd(reinterpret_cast<unsigned long long*>(&h1[bin_read(ct, cq, fv[q])]),
                    static_cast<unsigned long long>(sz[j][q]));
          if (uint32_t(q) < qcut) lo += sz[j][q]; else hi += sz[j][q];
        }
      }
      if (lo) atomicAdd(&zs[z], static_cast<unsigned long long>(lo));
      if (hi) atomicAdd(&zs[z + 1], static_cast<unsigned long long>(hi));
    }
  }
  __syncthreads();
  // every class-0 bin lies in exactly one slice (slices are whole bins)
  uint64_t* Zi = Z + i * int64_t(a.nb0) + zb0;
  for (uint32_t b = threadIdx.x; b < nz; b += kThreads) Zi[b] = zs[b];
  uint64_t* Hi = H + i * int64_t(a.nbin + 1);
  for (uint32_t b = threadIdx.x; b < a.nbin1; b += kThreads)
    if (h1[b]) atomicAdd(reinterpret_cast<unsigned long long*>(&Hi[b]),
                         static_cast<unsigned long long>(h1[b]));
}

// -- cut ranges ------------------------------------------------------------------
// H[i] becomes cum_before (nbin + 1 entries, the last is the row total).
// Class-0 bin b holds every byte of its 256 ids (binsum) minus the bytes of
// the ids this worker reads (Z).
__global__ void __launch_bounds__(1024)
plan_cut(PlanArgs a, const uint64_t* __restrict__ binsum, const uint64_t* __restrict__ Z,
         uint64_t* __restrict__ H, int32_t* __restrict__ ranges) {
  __shared__ uint64_t tmp[65];
  const int64_t i = blockIdx.x;
  uint64_t* Hi = H + i * int64_t(a.nbin + 1);
  const uint64_t* Zi = Z + i * int64_t(a.nb0);
  uint64_t carry = 0;
  for (uint32_t b0 = 0; b0 < a.nbin; b0 += 1024) {
    const uint32_t b = b0 + threadIdx.x;
    uint64_t v = 0;
    if (b < a.nbin1) v = Hi[b];
    else if (b < a.nbin) v = binsum[b - a.nbin1] - Zi[b - a.nbin1];
    uint64_t total;
    const uint64_t ex = block_exclusive_scan64(v, tmp, &total);
    if (b < a.nbin) Hi[b] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) Hi[a.nbin] = carry;
  __syncthreads();
  if (threadIdx.x != 0) return;
  const uint64_t total = carry;
  const int32_t nbin = int32_t(a.nbin);
  uint64_t s_lo = 0, s_hi = 0;
  int32_t* rg = ranges + i * 2 * a.J;
  for (int j = 0; j < a.J; ++j) {
    const uint64_t cap = uint64_t(a.caps[j]);
    const uint64_t t_lo = s_lo + cap < s_lo ? ~0ull : s_lo + cap;
    const uint64_t t_hi = s_hi + cap < s_hi ? ~0ull : s_hi + cap;
    if (t_lo >= total) {
      for (int jj = j; jj < a.J; ++jj) {
        rg[2 * jj] = nbin;
        rg[2 * jj + 1] = nbin;
      }
      return;
    }
    // lo: first bin b with cum_after(b) = Hi[b+1] > t_lo
    int32_t lo = 1, hi = nbin;  // search x in [1, nbin] for the first Hi[x] > t_lo
    while (lo < hi) {
      const int32_t mid = (lo + hi) >> 1;
      if (Hi[mid] > t_lo) hi = mid; else lo = mid + 1;
    }
    const int32_t blo = lo - 1;
    // hi: last bin b < nbin with cum_before(b) = Hi[b] <= t_hi
    lo = 0;
    hi = nbin - 1;
    while (lo < hi) {
      const int32_t mid = (lo + hi + 1) >> 1;
      if (Hi[mid] <= t_hi) lo = mid; else hi = mid - 1;
    }
    const int32_t bhi = lo;
    rg[2 * j] = blo;
    rg[2 * j + 1] = bhi;
    s_lo = Hi[blo];
    s_hi = t_hi < total ? t_hi : total;
  }
}

// -- tier write with candidate capture ----------------------------------------------
struct CandRec {
  uint64_t key;
  uint32_t k;
  uint32_t pad;
};

template <bool kVec>
__global__ void __launch_bounds__(kThreads)
plan_write(PlanArgs a, const uint8_t* __restrict__ count, const int32_t* __restrict__ first,
           const int32_t* __restrict__ ranges, int8_t* __restrict__ tier,
           CandRec* __restrict__ cand, int32_t* __restrict__ ccount, uint32_t nslices) {
  __shared__ ClassTable ct;
  __shared__ int32_t rg[256];
  // tier of every bin this workgroup can meet (all bins of classes >= 1,
  // then this slice's class-0 bins); kCand marks candidate bins
  __shared__ int8_t btier[kBins1Budget + 256 + kSliceBins0];
  constexpr int kCand = 127;
  const uint32_t t = xcd_logical(blockIdx.x, gridDim.x);
  if (t >= uint32_t(a.N) * nslices) return;
  const int64_t sl = t / a.N, i = t - sl * a.N;
  build_class_table(a, ct);
  for (int x = threadIdx.x; x < 2 * a.J; x += kThreads) rg[x] = ranges[i * 2 * a.J + x];
  __syncthreads();
  const int64_t ks = sl * kSliceCells;
  const int64_t ke = ks + kSliceCells < a.F ? ks + kSliceCells : a.F;
  const uint32_t b0_slice = a.nbin1 + uint32_t(ks >> kClass0Shift);
  const uint32_t nb_slice = uint32_t((ke - ks + (1 << kClass0Shift) - 1) >> kClass0Shift);
  for (uint32_t x = threadIdx.x; x < a.nbin1 + nb_slice; x += kThreads) {
    const int32_t b = int32_t(x < a.nbin1 ? x : b0_slice + (x - a.nbin1));
    bool cand = false;
    int tv = 0;
    for (int j = 0; j < a.J; ++j) {
      cand |= b >= rg[2 * j] && b <= rg[2 * j + 1];
      tv += rg[2 * j + 1] < b;
    }
    btier[x] = cand ? int8_t(kCand) : (tv >= a.J ? int8_t(-1) : int8_t(tv));
  }
  __syncthreads();
  const uint8_t* crow = count + i * a.F;
  const int32_t* frow = first + i * a.F;
  int8_t* trow = tier + i * a.F;
  CandRec* ci = cand + i * int64_t(a.cmax);
  // tier of one cell, or 256 for a candidate (its record key in *key)
  auto classify = [&](int64_t k, uint32_t c, int32_t f, uint64_t* key) -> int {
    if (c == 0) f = -1;
    const uint32_t b = bin_of(a, ct, c, f, k);
    const int tv = btier[b < a.nbin1 ? b : a.nbin1 + (b - b0_slice)];
    if (tv == kCand) {
      *key = (uint64_t(b) << 32) | (c ? uint64_t(uint32_t(f)) : uint64_t(k));
      return 256;
    }
    return tv;
  };
  auto single = [&](int64_t k) {
    uint64_t key = 0;
    const int tv = classify(k, crow[k], frow[k], &key);
    trow[k] = tv == 256 ? int8_t(0) : int8_t(tv);
    if (tv == 256) {
      const int32_t slot = atomicAdd(&ccount[i], 1);
      if (slot < a.cmax) ci[slot] = CandRec{key, uint32_t(k), 0u};
    }
  };
  const RowSplit rs = split_row(i * a.F + ks, ks, ke, kVec);
  for (int64_t k = ks + threadIdx.x; k < rs.body0; k += kThreads) single(k);
  for (int64_t k = rs.tail0 + threadIdx.x; k < ke; k += kThreads) single(k);
  constexpr int kU = 4;
  uint32_t cw[kU];
  int4 fw[kU];
  auto load = [&](int64_t u0) {
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const int64_t u = u0 + j * kThreads + threadIdx.x;
      const int64_t k = rs.body0 + 4 * u;
      if (u < rs.nunits) {
        cw[j] = *reinterpret_cast<const uint32_t*>(crow + k);
        fw[j] = *reinterpret_cast<const int4*>(frow + k);
      }
    }
  };
  if (rs.nunits > 0) load(0);
  for (int64_t u0 = 0; u0 < rs.nunits; u0 += kU * kThreads) {
    uint32_t cc[kU];
    int4 ff[kU];
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      cc[j] = cw[j];
      ff[j] = fw[j];
    }
    // the next iteration's words are in flight while this one is classified
    if (u0 + kU * kThreads < rs.nunits) load(u0 + kU * kThreads);
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const int64_t u = u0 + j * kThreads + threadIdx.x;
      const int64_t k = rs.body0 + 4 * u;
      const bool ok = u < rs.nunits;
      uint64_t key[4] = {0, 0, 0, 0};
      int tv[4] = {0, 0, 0, 0};
      int nc = 0;
      if (ok) {
        const int32_t fv[4] = {ff[j].x, ff[j].y, ff[j].z, ff[j].w};
        uint32_t packed = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          tv[q] = classify(k + q, (cc[j] >> (8 * q)) & 0xFFu, fv[q], &key[q]);
          nc += tv[q] == 256;
          packed |= uint32_t(uint8_t(int8_t(tv[q] == 256 ? 0 : tv[q]))) << (8 * q);
        }
        stream_store(reinterpret_cast<uint32_t*>(trow + k), packed);
      }
      if (__ballot(nc > 0)) {
        const uint32_t inc = wave_inclusive_scan(uint32_t(nc));
        const uint32_t tot = __builtin_amdgcn_readlane(inc, 63);
        int32_t basev = 0;
        if (__lane_id() == 63) basev = atomicAdd(&ccount[i], int32_t(tot));
        basev = __builtin_amdgcn_readlane(basev, 63);
        int32_t slot = basev + int32_t(inc) - nc;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (tv[q] == 256) {
            if (slot < a.cmax) ci[slot] = CandRec{key[q], uint32_t(k + q), 0u};
            ++slot;
          }
        }
      }
    }
  }
}

// -- exact resolution of the candidates --------------------------------------------------
struct ResolveSmem {
  uint64_t key[kCandMax];  // rank keys; after the sort, the bytes of the whole bins before each
  uint32_t k[kCandMax];
  uint64_t sz[kCandMax];   // each candidate's size
};

__global__ void __launch_bounds__(kResolveThreads)
plan_resolve(PlanArgs a, const uint64_t* __restrict__ H, const CandRec* __restrict__ cand,
             const int32_t* __restrict__ ccount, const int64_t* __restrict__ sizes,
             int8_t* __restrict__ tier, int64_t* __restrict__ used, int32_t* __restrict__ overflow) {
  __shared__ ResolveSmem s;
  const int64_t i = blockIdx.x;
  const int32_t n = ccount[i];
  if (threadIdx.x == 0) overflow[i] = n > a.cmax ? 1 : 0;
  if (n > a.cmax) return;
  const uint64_t* Hi = H + i * int64_t(a.nbin + 1);
  const CandRec* ci = cand + i * int64_t(a.cmax);
  int32_t P2 = 1;
  while (P2 < n) P2 <<= 1;
  for (int32_t x = threadIdx.x; x < P2; x += kResolveThreads) {
    if (x < n) {
      s.key[x] = ci[x].key;
      s.k[x] = ci[x].k;
    } else {
      s.key[x] = ~0ull;
      s.k[x] = 0xFFFFFFFFu;
    }
  }
  __syncthreads();
  // bitonic sort by key (keys are unique)
  for (int32_t kk = 2; kk <= P2; kk <<= 1) {
    for (int32_t j = kk >> 1; j > 0; j >>= 1) {
      for (int32_t x = threadIdx.x; x < P2; x += kResolveThreads) {
        const int32_t y = x ^ j;
        if (y > x) {
          const bool up = (x & kk) == 0;
          const uint64_t kx = s.key[x], ky = s.key[y];
          if ((kx > ky) == up) {
            s.key[x] = ky; s.key[y] = kx;
            const uint32_t t = s.k[x]; s.k[x] = s.k[y]; s.k[y] = t;
          }
        }
      }
      __syncthreads();
    }
  }
  // every thread gathers, for its candidates in sorted order, the size and
  // the bytes of the whole bins between the previous candidate's bin and
  // this one's (zero within a bin), so the serial fill below reads LDS only
  constexpr int kPerT = kCandMax / kResolveThreads;
  static_assert(kCandMax % kResolveThreads == 0, "candidates per thread");
  const int64_t last_bin = n > 0 ? int64_t(s.key[n - 1] >> 32) : -1;
  uint64_t gap[kPerT], hb[kPerT], hp[kPerT], sk[kPerT];
  // loads first, unconditional (clamped to entry 0), so they are in flight together
#pragma unroll
  for (int q = 0; q < kPerT; ++q) {
    const int32_t x = int32_t(threadIdx.x) + q * kResolveThreads;
    const bool in = x < n;
    const int64_t b = in ? int64_t(s.key[x] >> 32) : 0;
    const int64_t pb = in && x > 0 ? int64_t(s.key[x - 1] >> 32) : -1;
    hb[q] = Hi[b];
    hp[q] = Hi[pb + 1];
    sk[q] = uint64_t(sizes[in ? s.k[x] : 0u]);
  }
#pragma unroll
  for (int q = 0; q < kPerT; ++q) {
    const int32_t x = int32_t(threadIdx.x) + q * kResolveThreads;
    gap[q] = 0;
    if (x < n) {
      const int64_t b = int64_t(s.key[x] >> 32);
      const int64_t pb = x > 0 ? int64_t(s.key[x - 1] >> 32) : -1;
      if (b != pb) gap[q] = hb[q] - (pb < 0 ? 0ull : hp[q]);
      s.sz[x] = sk[q];
    }
  }
  __syncthreads();  // every key is read before any is replaced
#pragma unroll
  for (int q = 0; q < kPerT; ++q) {
    const int32_t x = int32_t(threadIdx.x) + q * kResolveThreads;
    if (x < n) s.key[x] = gap[q];
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  // replay the greedy fill: definite bins between candidates are added whole
  int64_t* ui = used + i * a.J;
  int8_t* trow = tier + i * a.F;
  int j = 0;
  uint64_t u = 0;
  for (int32_t x = 0; x < n; ++x) {
    u += s.key[x];
    const uint64_t sz = s.sz[x];
    while (j < a.J && u + sz > uint64_t(a.caps[j])) {
      ui[j] = int64_t(u);
      ++j;
      u = 0;
    }
    if (j < a.J) {
      trow[s.k[x]] = int8_t(j);
      u += sz;
    } else {
      trow[s.k[x]] = int8_t(-1);
    }
  }
  if (j < a.J) {
    const uint64_t gap_start = last_bin < 0 ? 0ull : Hi[last_bin + 1];
    u += Hi[a.nbin] - gap_start;
    ui[j] = int64_t(u);
    for (int jj = j + 1; jj < a.J; ++jj) ui[jj] = 0;
  }
}

// -- exact fallback: weighted radix select over the whole row ------------------------------
__global__ void __launch_bounds__(1024)
plan_exact(PlanArgs a, const uint8_t* __restrict__ count, const int32_t* __restrict__ first,
           const int64_t* __restrict__ sizes, const int32_t* __restrict__ overflow,
           int8_t* __restrict__ tier, int64_t* __restrict__ used) {
  __shared__ uint64_t hist[256];
  __shared__ uint64_t cuts[128];
  __shared__ uint64_t sh_prefix, sh_acc, sh_total;
  const int64_t i = blockIdx.x;
  if (!overflow[i]) return;
  const uint8_t* crow = count + i * a.F;
  const int32_t* frow = first + i * a.F;
  int8_t* trow = tier + i * a.F;
  uint64_t base = 0;        // bytes ranked before the start of tier j
  uint64_t total = 0;
  bool at_end = false;
  for (int j = 0; j < a.J; ++j) {
    if (at_end) {
      if (threadIdx.x == 0) {
        cuts[j] = ~0ull;
        used[i * a.J + j] = 0;
      }
      continue;
    }
    const uint64_t target = base + uint64_t(a.caps[j]) < base ? ~0ull : base + uint64_t(a.caps[j]);
    uint64_t prefix = 0, acc = 0;
    // 40-bit key, five 8-bit digits from the top
    for (int level = 0; level < 5; ++level) {
      const int shift = 32 - 8 * level;
      for (int d = threadIdx.x; d < 256; d += blockDim.x) hist[d] = 0;
      __syncthreads();
      for (int64_t k = threadIdx.x; k < a.F; k += blockDim.x) {
        const uint32_t c = crow[k];
        const uint64_t key = rank_key(a, c, c ? frow[k] : -1, k);
        if (level > 0 && (key >> (shift + 8)) != prefix) continue;
        atomicAdd(reinterpret_cast<unsigned long long*>(&hist[(key >> shift) & 0xFF]),
                  static_cast<unsigned long long>(sizes[k]));
      }
      __syncthreads();
      if (threadIdx.x == 0) {
        if (level == 0) {
          uint64_t t = 0;
          for (int d = 0; d < 256; ++d) t += hist[d];
          sh_total = t;
        }
        uint64_t run = acc;
        int d = 0;
        for (; d < 256; ++d) {
          if (run + hist[d] > target) break;
          run += hist[d];
        }
        sh_prefix = (prefix << 8) | uint64_t(d < 256 ? d : 255);
        sh_acc = run;
      }
      __syncthreads();
      if (level == 0) total = sh_total;
      if (total <= target) break;  // everything left fits
      prefix = sh_prefix;
      acc = sh_acc;
      __syncthreads();
    }
    if (total <= target) {
      if (threadIdx.x == 0) {
        cuts[j] = ~0ull;
        used[i * a.J + j] = int64_t(total - base);
      }
      at_end = true;
    } else {
      if (threadIdx.x == 0) {
        cuts[j] = prefix;
        used[i * a.J + j] = int64_t(acc - base);
      }
      base = acc;
    }
    __syncthreads();
  }
  __syncthreads();
  for (int64_t k = threadIdx.x; k < a.F; k += blockDim.x) {
    const uint32_t c = crow[k];
    const uint64_t key = rank_key(a, c, c ? frow[k] : -1, k);
    int tv = 0;
    for (int j = 0; j < a.J; ++j) tv += key >= cuts[j];
    trow[k] = tv >= a.J ? int8_t(-1) : int8_t(tv);
  }
}

// -- passes over the compact read-cell list (fused planning call) -----------------
// The counting pass lists, per (worker, window of 2^ws samples), the cells the
// worker reads: bin << kListOffBits | offset in window. Cells missing from the
// list are unread (class 0).
struct CompactArgs {
  const uint32_t* ent;
  const int32_t* base;
  const uint32_t* num;
  int32_t ws;
  uint32_t nbk;
  uint32_t wps;  // windows per slice of kSliceCells samples
};
#ifndef NOPFS_HIST_CU
#define NOPFS_HIST_CU 6
#endif
constexpr int kHistCU = NOPFS_HIST_CU;  // list entries per lane in flight

// Histogram of one (worker, slice): each wave takes whole windows of the
// slice; class-0 read bytes and class >= 1 bins as in plan_hist. The list
// bounds of up to kHistWins windows are staged in LDS at once, and a wave
// requests the next window's entries before waiting for this window's sizes.
constexpr uint32_t kHistWins = 1024;

__global__ void __launch_bounds__(kThreads)
plan_hist_c(PlanArgs a, CompactArgs c, const int64_t* __restrict__ sizes, uint64_t* __restrict__ Z,
            uint64_t* __restrict__ H, uint32_t nslices) {
  extern __shared__ uint64_t sm[];
  uint64_t* h1 = sm;
  unsigned long long* zs = reinterpret_cast<unsigned long long*>(sm + a.nbin1);
  __shared__ uint32_t wnum[kHistWins];
  __shared__ int32_t wbase[kHistWins];
  const uint32_t t = xcd_logical(blockIdx.x, gridDim.x);
  if (t >= uint32_t(a.N) * nslices) return;
  const int64_t sl = t / a.N, i = t - sl * a.N;
  const int64_t ks = sl * kSliceCells;
  const int64_t ke = ks + kSliceCells < a.F ? ks + kSliceCells : a.F;
  const uint32_t zb0 = uint32_t(ks >> kClass0Shift);
  const uint32_t nz = uint32_t((ke - ks + (1 << kClass0Shift) - 1) >> kClass0Shift);
  for (uint32_t b = threadIdx.x; b < a.nbin1; b += kThreads) h1[b] = 0;
  for (uint32_t b = threadIdx.x; b < nz; b += kThreads) zs[b] = 0;
  const uint32_t kb0 = uint32_t(sl) * c.wps;
  const uint32_t kb1 = kb0 + c.wps < c.nbk ? kb0 + c.wps : c.nbk;
  const uint32_t lane = __lane_id(), wave = threadIdx.x >> 6;
  constexpr uint32_t kWaves = kThreads / 64;
  const uint32_t* erow = c.ent + i * a.M_max;
  for (uint32_t g0 = kb0; g0 < kb1; g0 += kHistWins) {
    const uint32_t g1 = g0 + kHistWins < kb1 ? g0 + kHistWins : kb1;
    for (uint32_t kb = g0 + threadIdx.x; kb < g1; kb += kThreads) {
      wnum[kb - g0] = c.num[i * int64_t(c.nbk) + kb];
      wbase[kb - g0] = c.base[i * int64_t(c.nbk) + kb];
    }
    __syncthreads();
    // Each wave walks its windows kb = g0 + wave, + kWaves, ... in steps of
    // kHistCU * 64 entries, as one pipeline: a step requests its entries'
    // sizes, then the next step's entries, and adds its bins while those are
    // in flight. Loads are unconditional (clamped indices), so waiting for the
    // sizes leaves the later entry loads outstanding.
    constexpr uint32_t kStep = kHistCU * 64;
    auto add = [&](uint32_t e, uint64_t sz, int64_t kw) {
      const int64_t k = kw + (e & kListOffMask);
      atomicAdd(reinterpret_cast<unsigned long long*>(&h1[e >> kListOffBits]),
                static_cast<unsigned long long>(sz));
      atomicAdd(&zs[uint32_t(k >> kClass0Shift) - zb0], static_cast<unsigned long long>(sz));
    };
    auto window = [&](uint32_t kb, uint32_t& n, const uint32_t*& e) {
      n = kb < g1 ? wnum[kb - g0] : 0u;
      e = erow + (kb < g1 ? wbase[kb - g0] : 0);
    };
    auto next_window = [&](uint32_t& kb, uint32_t& n, const uint32_t*& e) {
      do {
        kb += kWaves;
        window(kb, n, e);
      } while (kb < g1 && n == 0u);
    };
    auto load = [&](uint32_t (&dst)[kHistCU], const uint32_t* e, uint32_t q0, uint32_t n) {
      const uint32_t last = n ? n - 1 : 0u;  // entry 0 of the row exists (M_max >= 1)
#pragma unroll
      for (int u = 0; u < kHistCU; ++u) {
        const uint32_t q = q0 + u * 64 + lane;
        dst[u] = e[q < last ? q : last];
      }
    };
    uint32_t kb = g0 + wave, q0 = 0, n;
    const uint32_t* e;
    window(kb, n, e);
    if (kb < g1 && n == 0u) next_window(kb, n, e);
    uint32_t cur[kHistCU];
    load(cur, e, 0, n);
    while (kb < g1) {
      const int64_t kw = int64_t(kb) << c.ws;
      uint64_t sz[kHistCU];
#pragma unroll
      for (int u = 0; u < kHistCU; ++u) sz[u] = uint64_t(sizes[kw + (cur[u] & kListOffMask)]);
      uint32_t nkb = kb, nq0 = q0 + kStep, nn = n;
      const uint32_t* ne = e;
      if (nq0 >= n) {
        nq0 = 0;
        next_window(nkb, nn, ne);
      }
      uint32_t nxt[kHistCU];
      load(nxt, ne, nq0, nn);
#pragma unroll
      for (int u = 0; u < kHistCU; ++u)
        if (q0 + u * 64 + lane < n) add(cur[u], sz[u], kw);
#pragma unroll
      for (int u = 0; u < kHistCU; ++u) cur[u] = nxt[u];
      kb = nkb;
      q0 = nq0;
      n = nn;
      e = ne;
    }
    __syncthreads();
  }
  uint64_t* Zi = Z + i * int64_t(a.nb0) + zb0;
  for (uint32_t b = threadIdx.x; b < nz; b += kThreads) Zi[b] = zs[b];
  uint64_t* Hi = H + i * int64_t(a.nbin + 1);
  for (uint32_t b = threadIdx.x; b < a.nbin1; b += kThreads)
    if (h1[b]) atomicAdd(reinterpret_cast<unsigned long long*>(&Hi[b]),
                         static_cast<unsigned long long>(h1[b]));
}

// Tier (or the candidate mark) of every bin of every worker, from the cut ranges.
constexpr int8_t kCandMark = 127;

__global__ void __launch_bounds__(256)
plan_btier(PlanArgs a, const int32_t* __restrict__ ranges, int8_t* __restrict__ btier) {
  const int64_t i = blockIdx.y;
  const int32_t b = int32_t(blockIdx.x) * 256 + int32_t(threadIdx.x);
  if (b >= int32_t(a.nbin)) return;
  const int32_t* rg = ranges + i * 2 * a.J;
  bool cand = false;
  int tv = 0;
  for (int j = 0; j < a.J; ++j) {
    const int32_t lo = rg[2 * j], hi = rg[2 * j + 1];
    cand |= b >= lo && b <= hi;
    tv += hi < b;
  }
  btier[i * a.btp + b] = cand ? kCandMark : (tv >= a.J ? int8_t(-1) : int8_t(tv));
}

// Tier row of one (worker, window): every cell starts with its class-0 bin's
// tier, the listed read cells take their own bin's, and the cells of
// candidate bins are appended to the worker's candidate list as in plan_write.
// All loads a tile needs go out in two rounds: the class table, the bin
// tiers of classes >= 1 (into LDS), the tile's list bounds and class-0 tiers,
// then the list entries. Cell x of the row sits at LDS byte x + sh, sh = (flat
// index of the window's first cell) mod 16, so the row is filled a 32-bit
// word (4 cells) at a time and written out as 16-byte stores.
constexpr int kWriteThreads = 256;
constexpr int kWriteWin = 8192;  // cells held in LDS at once
#ifndef NOPFS_WRITE_ENT
#define NOPFS_WRITE_ENT 6
#endif
constexpr int kWriteEnt = NOPFS_WRITE_ENT;  // list entries per thread loaded up front

constexpr uint32_t kBt1Max = ((kBins1Budget + 256 + 15) / 16) * 16;  // class >= 1 bins, padded

template <bool kVec>
__global__ void __launch_bounds__(kWriteThreads) __attribute__((amdgpu_waves_per_eu(8)))
plan_write_c(PlanArgs a, CompactArgs c, const int32_t* __restrict__ first,
             const int8_t* __restrict__ btier, int8_t* __restrict__ tier,
             CandRec* __restrict__ cand, int32_t* __restrict__ ccount, uint32_t ntiles) {
  __shared__ __align__(16) int8_t bt1[kBt1Max];
  __shared__ __align__(16) uint32_t tbw[kWriteWin / 4 + 8];  // the row's tiers, shifted by sh
  __shared__ int8_t t0[kWriteWin / (1 << kClass0Shift) + 1];
  int8_t* tb = reinterpret_cast<int8_t*>(tbw);
  __shared__ int s_c0cand;
  const uint32_t tile = xcd_logical(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int64_t i = tile / c.nbk;
  const uint32_t kb = tile - uint32_t(i) * c.nbk;
  const int8_t* bt = btier + i * int64_t(a.btp);  // 16-byte aligned rows
  const int64_t k0 = int64_t(kb) << c.ws;
  const int64_t kend = k0 + (int64_t(1) << c.ws) < a.F ? k0 + (int64_t(1) << c.ws) : a.F;
  const int64_t tix = i * int64_t(c.nbk) + kb;
  // round one: bin tiers, list bounds, class-0 tiers of the first piece
  const uint32_t nb1w = (a.nbin1 + 15) / 16;
  uint4 btw[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t w = threadIdx.x + uint32_t(h) * kWriteThreads;
    btw[h] = make_uint4(0, 0, 0, 0);
    if (w < nb1w) btw[h] = *reinterpret_cast<const uint4*>(bt + 16 * w);  // inside the padded row
  }
  // class-0 tiers of the first window pass (clamped index: unconditional)
  auto zbins = [&](int64_t w0) {
    const int64_t wl = kend - w0 < kWriteWin ? kend - w0 : kWriteWin;
    return uint32_t((w0 + wl - 1) >> kClass0Shift) - uint32_t(w0 >> kClass0Shift) + 1;
  };
  const uint32_t nzb_first = zbins(k0);
  const int8_t zt_first =
      bt[a.nbin1 + uint32_t(k0 >> kClass0Shift) + (threadIdx.x < nzb_first ? threadIdx.x : 0u)];
  const uint32_t n = c.num[tix];
  const uint32_t* ent = c.ent + i * a.M_max + c.base[tix];
  // round two: the list entries
  uint32_t ev[kWriteEnt];
#pragma unroll
  for (int u = 0; u < kWriteEnt; ++u) {
    const uint32_t q = threadIdx.x + uint32_t(u) * kWriteThreads;
    ev[u] = q < n ? ent[q] : 0u;
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t w = threadIdx.x + uint32_t(h) * kWriteThreads;
    if (w < nb1w) *reinterpret_cast<uint4*>(bt1 + 16 * w) = btw[h];
  }
  CandRec* ci = cand + i * int64_t(a.cmax);
  int8_t* trow = tier + i * a.F;
  auto append = [&](uint64_t key, int64_t k) {
    const int32_t slot = atomicAdd(&ccount[i], 1);
    if (slot < a.cmax) ci[slot] = CandRec{key, uint32_t(k), 0u};
  };
  const int32_t* frow = first + i * a.F;
  auto apply = [&](uint32_t v, uint32_t xoff, uint32_t wlen, int64_t w0, uint32_t sh) {
    const uint32_t x = (v & kListOffMask) - xoff;
    if (x < wlen) {
      const uint32_t b = v >> kListOffBits;
      const int8_t tv = bt1[b];
      if (tv == kCandMark) {
        // the rank key needs the first read itself (few cells per worker)
        append((uint64_t(b) << 32) | uint64_t(uint32_t(frow[w0 + x])), w0 + x);
        tb[x + sh] = 0;
      } else {
        tb[x + sh] = tv;
      }
    }
  };
  for (int64_t w0 = k0; w0 < kend; w0 += kWriteWin) {
    const uint32_t wlen = uint32_t(kend - w0 < kWriteWin ? kend - w0 : kWriteWin);
    const uint32_t xoff = uint32_t(w0 - k0);
    const uint32_t zb0 = uint32_t(w0 >> kClass0Shift);
    const uint32_t nzb = uint32_t((w0 + wlen - 1) >> kClass0Shift) - zb0 + 1;
    const uint32_t sh = kVec ? uint32_t((i * a.F + w0) & 15) : 0u;
    if (threadIdx.x == 0) s_c0cand = 0;
    int8_t zt = zt_first;
    if (w0 != k0 && threadIdx.x < nzb) zt = bt[a.nbin1 + zb0 + threadIdx.x];
    __syncthreads();
    if (threadIdx.x < nzb) {
      t0[threadIdx.x] = zt;
      if (zt == kCandMark) s_c0cand = 1;
    }
    __syncthreads();
    {
      // word wd holds cells 4 wd - sh .. 4 wd - sh + 3; bytes of cells
      // outside the window are never written out
      const uint32_t lo8 = uint32_t(w0) & ((1u << kClass0Shift) - 1);  // w0 = zb0 * 256 + lo8
      auto zbin = [&](int32_t x) {
        x = x < 0 ? 0 : (x >= int32_t(wlen) ? int32_t(wlen) - 1 : x);
        return (lo8 + uint32_t(x)) >> kClass0Shift;
      };
      const uint32_t nw = (wlen + sh + 3) / 4;
      // eight consecutive words (32 cells) per thread: almost always inside
      // one class-0 bin (256 cells), then one lookup and two 16-byte stores
      // (words past nw fall in the table's slack and are never read)
      for (uint32_t wd0 = 8 * threadIdx.x; wd0 < nw; wd0 += 8 * kWriteThreads) {
        const int32_t xa = int32_t(4 * wd0) - int32_t(sh);
        const uint32_t za = zbin(xa), zd = zbin(xa + 31);
        uint4* dst = reinterpret_cast<uint4*>(tbw + wd0);
        if (za == zd) {
          const uint32_t word = uint32_t(uint8_t(t0[za])) * 0x01010101u;
          dst[0] = make_uint4(word, word, word, word);
          dst[1] = make_uint4(word, word, word, word);
        } else {
          uint32_t wv[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const int32_t xq = xa + 4 * q;
            const uint32_t a = zbin(xq), d = zbin(xq + 3);
            wv[q] = uint32_t(uint8_t(t0[a])) * 0x01010101u;
            if (a != d)  // the word spans two class-0 bins
              wv[q] = uint32_t(uint8_t(t0[a])) | (uint32_t(uint8_t(t0[zbin(xq + 1)])) << 8) |
                      (uint32_t(uint8_t(t0[zbin(xq + 2)])) << 16) | (uint32_t(uint8_t(t0[d])) << 24);
          }
          dst[0] = make_uint4(wv[0], wv[1], wv[2], wv[3]);
          dst[1] = make_uint4(wv[4], wv[5], wv[6], wv[7]);
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kWriteEnt; ++u)
      if (threadIdx.x + uint32_t(u) * kWriteThreads < n) apply(ev[u], xoff, wlen, w0, sh);
    for (uint32_t q = threadIdx.x + kWriteEnt * kWriteThreads; q < n; q += kWriteThreads)
      apply(ent[q], xoff, wlen, w0, sh);
    __syncthreads();
    if (s_c0cand) {
      // unread cells of candidate class-0 bins (read ones were overwritten)
      for (uint32_t x = threadIdx.x; x < wlen; x += kWriteThreads) {
        if (tb[x + sh] == kCandMark) {
          const int64_t k = w0 + x;
          append((uint64_t(a.nbin1 + uint32_t(k >> kClass0Shift)) << 32) | uint64_t(k), k);
          tb[x + sh] = 0;
        }
      }
      __syncthreads();
    }
    // cells before the first 16-byte aligned cell of the output row and
    // after the last whole group of 16 go one per thread, the rest as one
    // 16-byte LDS read and one 16-byte store per group (x + sh is a
    // multiple of 16 there)
    int8_t* dst = trow + w0;
    uint32_t head = kVec ? (16u - sh) & 15u : wlen;
    if (head > wlen) head = wlen;
    const uint32_t nunits = (wlen - head) >> 4;
    const uint32_t tail0 = head + 16 * nunits;
    for (uint32_t x = threadIdx.x; x < head; x += kWriteThreads) stream_store(dst + x, tb[x + sh]);
    for (uint32_t x = tail0 + threadIdx.x; x < wlen; x += kWriteThreads)
      stream_store(dst + x, tb[x + sh]);
    for (uint32_t u = threadIdx.x; u < nunits; u += kWriteThreads) {
      const uint32_t x = head + 16 * u;
      stream_store(reinterpret_cast<uint4*>(dst + x), *reinterpret_cast<const uint4*>(tb + x + sh));
    }
    __syncthreads();
  }
}

// Bins per class c >= 1, in proportion to the expected number of cells of
// class c (a worker reads a sample in each epoch with probability L/F, so
// counts follow Binomial(E, L/F)); at least one bin per class.
void class_bins(int64_t F, int64_t E, int64_t L, uint16_t* nbc, uint32_t* nbin1) {
  const double p = F > 0 ? double(L) / double(F) : 0.0;
  std::vector<double> pmf(size_t(E) + 1, 0.0);
  double acc = 0;
  for (int64_t c = 1; c <= E; ++c) {
    double lp = lgamma(double(E) + 1) - lgamma(double(c) + 1) - lgamma(double(E - c) + 1);
    lp += (p > 0 ? double(c) * log(p) : -INFINITY);
    lp += (p < 1 ? double(E - c) * log1p(-p) : (E - c == 0 ? 0.0 : -INFINITY));
    pmf[size_t(c)] = exp(lp);
    acc += pmf[size_t(c)];
  }
  uint32_t total = 0;
  for (int64_t c = 0; c < 256; ++c) nbc[c] = 0;
  for (int64_t c = 1; c <= E; ++c) {
    double share = acc > 0 ? pmf[size_t(c)] / acc : 1.0 / double(E);
    double want = floor(share * double(kBins1Budget));
    if (!(want >= 1.0)) want = 1.0;
    if (want > 4096.0) want = 4096.0;
    nbc[c] = uint16_t(want);
    total += nbc[c];
  }
  *nbin1 = total;
}

struct PlanBufs {
  uint64_t *H, *binsum, *Z;
  int32_t *ranges, *ccount, *overflow;
  CandRec* cand;
};

void plan_args(const Shape& s, const int64_t* caps, int32_t J, PlanArgs* a) {
  a->F = s.F;
  a->N = s.N;
  a->M_max = s.M_max;
  a->E = int32_t(s.E);
  a->J = J;
  class_bins(s.F, s.E, s.L, a->nbc, &a->nbin1);
  a->nb0 = uint32_t(ceil_div(s.F, int64_t(1) << kClass0Shift));
  a->nbin = a->nbin1 + a->nb0;
  a->btp = (a->nbin + 15u) & ~15u;
  a->cmax = kCandMax;
  if (debug_value(2) > 0 && debug_value(2) < kCandMax) a->cmax = int32_t(debug_value(2));
  for (int j = 0; j < 128; ++j) a->caps[j] = j < J ? caps[j] : 0;
}

// Scratch of both plan paths, the zeroed histogram and candidate counters,
// and the per-bin byte totals of the sizes.
int plan_begin(const Shape& s, const PlanArgs& a, const int64_t* sizes, Scratch& scr,
               PlanBufs* b, hipStream_t st) {
  int rc;
  const int64_t hn = s.N * int64_t(a.nbin + 1);
  if ((rc = scr.alloc_n(&b->H, size_t(hn)))) return rc;
  if ((rc = scr.alloc_n(&b->binsum, size_t(a.nb0)))) return rc;
  if ((rc = scr.alloc_n(&b->Z, size_t(s.N) * a.nb0))) return rc;
  if ((rc = scr.alloc_n(&b->ranges, size_t(s.N * 2 * a.J)))) return rc;
  if ((rc = scr.alloc_n(&b->ccount, size_t(s.N)))) return rc;
  if ((rc = scr.alloc_n(&b->overflow, size_t(s.N)))) return rc;
  if ((rc = scr.alloc_n(&b->cand, size_t(s.N * a.cmax)))) return rc;
  int64_t fb = ceil_div(hn, 1024);
  if (fb > 65536) fb = 65536;
  if ((rc = launch("fill_u64", fill_u64, dim3(uint32_t(fb)), dim3(256), 0, st, b->H, hn))) return rc;
  if ((rc = launch("fill_i32", fill_i32, dim3(uint32_t(ceil_div(s.N, 256))), dim3(256), 0, st,
                   b->ccount, s.N)))
    return rc;
  if (!sizes) return NOPFS_OK;  // the caller sums the bins later
  return launch("plan_binsum", plan_binsum, dim3(uint32_t(ceil_div(a.nb0, 4))), dim3(256), 0, st,
                s.F, a.nb0, sizes, b->binsum);
}

// Exact resolution of the candidates, and the full-row fallback for workers
// whose candidate list overflowed.
int plan_end(const Shape& s, const PlanArgs& a, const PlanBufs& b, const uint8_t* count,
             const int32_t* first, const int64_t* sizes, int8_t* tier, int64_t* used,
             hipStream_t st) {
  int rc;
  if ((rc = launch("plan_resolve", plan_resolve, dim3(uint32_t(s.N)), dim3(kResolveThreads), 0, st,
                   a, (const uint64_t*)b.H, (const CandRec*)b.cand, (const int32_t*)b.ccount, sizes,
                   tier, used, b.overflow)))
    return rc;
  return launch("plan_exact", plan_exact, dim3(uint32_t(s.N)), dim3(1024), 0, st, a, count, first,
                sizes, (const int32_t*)b.overflow, tier, used);
}

}  // namespace

int plan_check(const int64_t* caps, int32_t J) {
  if (J < 1) return fail(NOPFS_EINVAL, "J must be >= 1");
  if (J > 127) return fail(NOPFS_ERANGE, "J must be <= 127");
  for (int j = 0; j < J; ++j)
    if (caps[j] < 0) return fail(NOPFS_EINVAL, "capacities must be >= 0");
  return NOPFS_OK;
}

int plan_impl(const nopfs_job* job, const uint8_t* count, const int32_t* first,
              const int64_t* sizes, const int64_t* caps, int32_t J, int8_t* tier, int64_t* used,
              hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (!count || !first || !sizes || !caps || !tier || !used)
    return fail(NOPFS_EINVAL, "count, first, sizes, caps, tier and used must be non-NULL");
  if ((rc = plan_check(caps, J))) return rc;
  PlanArgs a;
  plan_args(s, caps, J, &a);
  Scratch scr(st);
  PlanBufs b;
  if ((rc = plan_begin(s, a, sizes, scr, &b, st))) return rc;
  // vector loads need 4-byte aligned count/tier rows and 16-byte aligned first rows
  const bool vec = (reinterpret_cast<uintptr_t>(count) & 3) == 0 &&
                   (reinterpret_cast<uintptr_t>(tier) & 3) == 0 &&
                   (reinterpret_cast<uintptr_t>(first) & 15) == 0;
  const uint32_t nslices = uint32_t(ceil_div(s.F, kSliceCells));
  const uint32_t ntiles = uint32_t(s.N) * nslices;
  const size_t hsmem = (size_t(a.nbin1) + kSliceBins0) * 8;
  if ((rc = vec ? launch("plan_hist", plan_hist<true>, dim3(xcd_padded(ntiles)), dim3(kThreads), hsmem,
                         st, a, count, first, sizes, b.Z, b.H, nslices)
                : launch("plan_hist", plan_hist<false>, dim3(xcd_padded(ntiles)), dim3(kThreads), hsmem,
                         st, a, count, first, sizes, b.Z, b.H, nslices)))
    return rc;
  if ((rc = launch("plan_cut", plan_cut, dim3(uint32_t(s.N)), dim3(1024), 0, st, a,
                   (const uint64_t*)b.binsum, (const uint64_t*)b.Z, b.H, b.ranges)))
    return rc;
  if ((rc = vec ? launch("plan_write", plan_write<true>, dim3(xcd_padded(ntiles)), dim3(kThreads), 0,
                         st, a, count, first, (const int32_t*)b.ranges, tier, b.cand, b.ccount, nslices)
                : launch("plan_write", plan_write<false>, dim3(xcd_padded(ntiles)), dim3(kThreads), 0,
                         st, a, count, first, (const int32_t*)b.ranges, tier, b.cand, b.ccount,
                         nslices)))
    return rc;
  return plan_end(s, a, b, count, first, sizes, tier, used, st);
}

struct CompactPlan {
  Shape s;
  PlanArgs a;
  PlanBufs b;
  ClassTable* gct;
  int8_t* btier;
};

int compact_plan_prepare(const Shape& s, const int64_t* caps, int32_t J, Scratch& keep,
                         hipStream_t st, CompactPlan** out, const ClassTable** classes) {
  int rc;
  if ((rc = plan_check(caps, J))) return rc;
  CompactPlan* cp = new CompactPlan;
  *out = cp;
  cp->s = s;
  plan_args(s, caps, J, &cp->a);
  if ((rc = keep.alloc_n(&cp->gct, 1))) return rc;
  if ((rc = keep.alloc_n(&cp->btier, size_t(s.N) * cp->a.btp))) return rc;
  if ((rc = plan_begin(s, cp->a, nullptr, keep, &cp->b, st))) return rc;
  *classes = cp->gct;
  return launch("plan_classes", plan_classes, dim3(1), dim3(64), 0, st, cp->a, cp->gct);
}

int compact_plan_run(CompactPlan* cp, const CompactCells& cc, const uint8_t* count,
                     const int32_t* first, const int64_t* sizes, int8_t* tier, int64_t* used,
                     hipStream_t st) {
  int rc;
  if (cc.ws > kListOffBits) return fail(NOPFS_EDEVICE, "sample windows wider than a list offset");
  const Shape& s = cp->s;
  const PlanArgs& a = cp->a;
  const PlanBufs& b = cp->b;
  if ((rc = launch("plan_binsum", plan_binsum, dim3(uint32_t(ceil_div(a.nb0, 4))), dim3(256), 0, st,
                   s.F, a.nb0, sizes, b.binsum)))
    return rc;
  const CompactArgs c{cc.ent, cc.base, cc.num, cc.ws, cc.nbk, uint32_t(kSliceCells >> cc.ws)};
  const uint32_t nslices = uint32_t(ceil_div(s.F, kSliceCells));
  const uint32_t nht = uint32_t(s.N) * nslices;
  const size_t hsmem = (size_t(a.nbin1) + kSliceBins0) * 8;
  if ((rc = launch("plan_hist", plan_hist_c, dim3(xcd_padded(nht)), dim3(kThreads), hsmem, st, a, c,
                   sizes, b.Z, b.H, nslices)))
    return rc;
  if ((rc = launch("plan_cut", plan_cut, dim3(uint32_t(s.N)), dim3(1024), 0, st, a,
                   (const uint64_t*)b.binsum, (const uint64_t*)b.Z, b.H, b.ranges)))
    return rc;
  if ((rc = launch("plan_btier", plan_btier, dim3(uint32_t(ceil_div(a.nbin, 256)), uint32_t(s.N)),
                   dim3(256), 0, st, a, (const int32_t*)b.ranges, cp->btier)))
    return rc;
  const uint32_t ntiles = uint32_t(s.N) * cc.nbk;
  const bool vec = (reinterpret_cast<uintptr_t>(tier) & 15) == 0;  // 16-byte row stores
  if ((rc = vec ? launch("plan_write", plan_write_c<true>, dim3(xcd_padded(ntiles)),
                         dim3(kWriteThreads), 0, st, a, c, first, (const int8_t*)cp->btier, tier,
                         b.cand, b.ccount, ntiles)
                : launch("plan_write", plan_write_c<false>, dim3(xcd_padded(ntiles)),
                         dim3(kWriteThreads), 0, st, a, c, first, (const int8_t*)cp->btier, tier,
                         b.cand, b.ccount, ntiles)))
    return rc;
  return plan_end(s, a, b, count, first, sizes, tier, used, st);
}

void compact_plan_free(CompactPlan* cp) { delete cp; }

}  // namespace nopfs

extern "C" int nopfs_tier_plan(const nopfs_job* job, const uint8_t* count, const int32_t* first,
                               const int64_t* sizes, const int64_t* caps, int32_t J, int8_t* tier,
                               int64_t* used, void* hip_stream) {
  try {
    return nopfs::plan_impl(job, count, first, sizes, caps, J, tier, used,
                            static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}
