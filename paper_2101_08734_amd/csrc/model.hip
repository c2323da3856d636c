// nopfs_fetch_model: the performance model of the Performance Modeling
// section evaluated for every read of every worker's stream, with the
// placement static (a sample is in tier j of worker i exactly when
// tier[i][k] == j).
//
// A read of sample k (s bytes) by worker i is fetched from the fastest of
// the PFS (t(gamma) / gamma per reader), another worker's tier j
// (min(b_c, r_j / p_j)) and its own tier j (r_j / p_j); on equal throughput
// its own tier wins over a remote one and a remote one over the PFS. It is
// then preprocessed and written to the staging buffer at min(beta, w0 / p0)
// per thread. With the p0 staging threads load-balanced, read f is in the
// buffer at avail(f) = (sum of the read times of reads 0..f) / p0, and the
// worker consumes it at
//   t(f) = max(avail(f), t(f-1) + s(f-1) / c) = U(f) + max over g <= f of (avail(g) - U(g)),
// U(f) = sum of s(m) / c over m < f (the recurrence unrolled): a prefix sum
// and a prefix maximum, evaluated per sub-chunk and combined per worker.
//
//   fm_holders -- per sample: the best remote class among all workers'
//                 copies (highest min(b_c, r_j / p_j), lower tier on ties),
//                 packed above the sample's size. A worker's own copy may be
//                 that class: a remote copy of class j is never faster than
//                 the local copy of j, so counting it never changes a choice.
//   fm_gather  -- per (16K-sample window, group of 32 workers) of the
//                 partition of R (rows folded into one segment of E * L_i
//                 reads, cut into spans of 2^14): each read's source from
//                 its own tier and the sample's best remote class; size and
//                 source in partitioned order.
//   fm_sum     -- per span of 2^14 reads: every entry loaded once into
//                 the LDS slot of its stream position (the whole sub-chunk,
//                 135 KB), then scanned in four parts of 4,096 positions:
//                 its read-time sum, compute-time sum and maximum of
//                 avail - U relative to its start.
//   fm_scan    -- per worker: what enters each span.
//   fm_final   -- per span: the same scans, combined with what enters
//                 it; source codes and consumption times in stream order.
#include <math.h>

#include <new>

#include "gather.hpp"
#include "partition.hpp"

namespace nopfs {
namespace {

#ifndef NOPFS_FM_THREADS
#define NOPFS_FM_THREADS 1024  // threads of the scan kernels (tuning only)
#endif

constexpr int kMaxClasses = 32;
constexpr uint32_t kNoClass = 255;
constexpr int kSizeBits = 56;
constexpr uint64_t kSizeMask = (uint64_t(1) << kSizeBits) - 1;
constexpr int kFmThreads = NOPFS_FM_THREADS;
constexpr int kFmPart = kSC / 4;                // positions per LDS pass
constexpr int kFmPer = kFmPart / kFmThreads;    // positions per thread and pass
constexpr int kFmEnt = kSC / kFmThreads;        // entries per thread
static_assert(kFmPer * kFmThreads == kFmPart && kFmEnt * kFmThreads == kSC, "fm shape");

// Source codes inside the library: 0 the PFS, 1 + j another worker's tier j,
// 1 + kMaxClasses + j the worker's own tier j.
constexpr uint32_t kOwn0 = 1 + kMaxClasses;

// Source rates, computed once on the host from the model's parameters.
struct Rates {
  double own[kMaxClasses];  // r_j / p_j
  double rem[kMaxClasses];  // min(b_c, r_j / p_j)
  double pfs;               // t(gamma) / gamma
  double wthr;              // min(beta, w0 / p0)
  double c, p0;
  // reciprocals for the per-read times (a product instead of a division:
  // within two units in the last place of the quotient)
  double inv_own[kMaxClasses], inv_rem[kMaxClasses];
  double inv_pfs, inv_wthr, inv_c;
  int32_t J;
  uint8_t rank_cls[kMaxClasses];  // classes by remote rate, best first, lower tier on ties
  uint8_t cls_rank[kMaxClasses];  // the inverse
};

struct SharedRates {
  double own[kMaxClasses], rem[kMaxClasses];
  double inv_own[kMaxClasses], inv_rem[kMaxClasses];
  uint8_t rank_cls[kMaxClasses], cls_rank[kMaxClasses];
};

__device__ __forceinline__ void load_rates(const Rates& r, SharedRates& s) {
  if (threadIdx.x < kMaxClasses) {
    s.own[threadIdx.x] = r.own[threadIdx.x];
    s.rem[threadIdx.x] = r.rem[threadIdx.x];
    s.inv_own[threadIdx.x] = r.inv_own[threadIdx.x];
    s.inv_rem[threadIdx.x] = r.inv_rem[threadIdx.x];
    s.rank_cls[threadIdx.x] = r.rank_cls[threadIdx.x];
    s.cls_rank[threadIdx.x] = r.cls_rank[threadIdx.x];
  }
}

// 1 / (the rate of a source code)
__device__ __forceinline__ double inv_rate_of(const Rates& r, const SharedRates& s, uint32_t code) {
  return code == 0 ? r.inv_pfs : (code < kOwn0 ? s.inv_rem[code - 1] : s.inv_own[code - kOwn0]);
}

// ---------------------------------------------------------------- holders --
__global__ void __launch_bounds__(256)
fm_holders(int64_t F, int64_t N, const int8_t* __restrict__ tier, const int64_t* __restrict__ sizes,
           Rates rt, uint64_t* __restrict__ szb) {
  __shared__ SharedRates sr;
  load_rates(rt, sr);
  __syncthreads();
  const int64_t k = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (k >= F) return;
  uint32_t best = kNoClass;  // as a rank: lower is better
  constexpr int kRows = 8;
  for (int64_t i0 = 0; i0 < N; i0 += kRows) {
    int32_t q[kRows];
#pragma unroll
    for (int u = 0; u < kRows; ++u) q[u] = i0 + u < N ? tier[(i0 + u) * F + k] : -1;
#pragma unroll
    for (int u = 0; u < kRows; ++u)
      if (q[u] >= 0 && q[u] < rt.J) {
        const uint32_t rk = sr.cls_rank[q[u]];
        best = rk < best ? rk : best;
      }
  }
  const uint64_t cls = best == kNoClass ? kNoClass : sr.rank_cls[best];
  szb[k] = (uint64_t(sizes[k]) & kSizeMask) | (cls << kSizeBits);
}

// ------------------------------------------------------------------ tiles --
__device__ __forceinline__ uint32_t choose(const Rates& rt, const SharedRates& sr, int32_t own,
                                           uint32_t b1) {
  double best = -1;
  uint32_t code = 0;
  if (own >= 0 && own < rt.J) {
    best = sr.own[own];
    code = kOwn0 + uint32_t(own);
  }
  if (b1 != kNoClass && sr.rem[b1] > best) {
    best = sr.rem[b1];
    code = 1 + b1;
  }
  if (rt.pfs > best) code = 0;
  return code;
}

// Each read of the tile's window and rows gets its source (choose) and its
// size, packed, at its place in the partitioned row. Four reads per thread
// and inner pass (eight, as in the staging gather, were no faster here).
constexpr int kFmGChunk = 4 * kGThreads;
constexpr int kFmGPer = kFmGChunk / kGThreads;
__global__ void __launch_bounds__(kGThreads)
fm_gather(SegParams p, const uint32_t* __restrict__ Pk, const uint16_t* __restrict__ OT,
          const int8_t* __restrict__ tier, const uint64_t* __restrict__ szb, Rates rt,
          uint64_t* __restrict__ zP, uint32_t ngroups, uint32_t ntiles) {
  __shared__ GatherLds<kFmGChunk> L;
  __shared__ SharedRates sr;
  const uint32_t tile = xcd_logical(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  load_rates(rt, sr);  // visible after the tile's first barrier
  gather_tile<uint64_t, kFmGChunk>(
      p, Pk, OT, tile, ngroups, L, [&](int64_t k) { return szb[k]; },
      [&](const int64_t (&pos)[kFmGPer], const int64_t (&row)[kFmGPer], const uint32_t (&x)[kFmGPer],
          int64_t w0, uint32_t wl) {
        // each read's own tier: a byte of its row's window slice (cached),
        // loads first, unconditional
        int32_t own[kFmGPer];
#pragma unroll
        for (int u = 0; u < kFmGPer; ++u) own[u] = tier[row[u] * p.F + w0 + (x[u] < wl ? x[u] : 0u)];
#pragma unroll
        for (int u = 0; u < kFmGPer; ++u)
          if (pos[u] >= 0 && x[u] < wl) {
            const uint64_t sb = L.win[x[u]];
            const uint32_t code = choose(rt, sr, own[u], uint32_t(sb >> kSizeBits));
            zP[pos[u]] = (sb & kSizeMask) | (uint64_t(code) << kSizeBits);
          }
      });
}

// ------------------------------------------------------------------ scans --
__device__ __forceinline__ double wave_incl_sum(double v) {
  const int lane = __lane_id();
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const double o = __shfl_up(v, d, 64);
    if (lane >= d) v += o;
  }
  return v;
}

__device__ __forceinline__ double wave_incl_max(double v) {
  const int lane = __lane_id();
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const double o = __shfl_up(v, d, 64);
    if (lane >= d) v = fmax(v, o);
  }
  return v;
}

// Exclusive prefix scans over the workgroup (blockDim.x a multiple of 64):
// two sums at once, or a maximum with -inf as identity; the totals go to
// *tot*. No closing barrier: the caller's next use of tmp comes after later
// barriers. tmp holds 65 entries.
__device__ __forceinline__ void block_excl_sum2(double a, double u, double2* tmp, double* exa,
                                                double* exu, double* tota, double* totu) {
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const double ia = wave_incl_sum(a), iu = wave_incl_sum(u);
  if (lane == 63) tmp[wave] = make_double2(ia, iu);
  __syncthreads();
  if (threadIdx.x < 64) {
    const double2 w = threadIdx.x < unsigned(nwaves) ? tmp[threadIdx.x] : make_double2(0.0, 0.0);
    const double wa = wave_incl_sum(w.x), wu = wave_incl_sum(w.y);
    const double pa = __shfl_up(wa, 1, 64), pu = __shfl_up(wu, 1, 64);
    if (threadIdx.x < unsigned(nwaves))
      tmp[threadIdx.x] = threadIdx.x == 0 ? make_double2(0.0, 0.0) : make_double2(pa, pu);
    if (threadIdx.x == 63) tmp[64] = make_double2(wa, wu);
  }
  __syncthreads();
  const double ba = __shfl_up(ia, 1, 64), bu = __shfl_up(iu, 1, 64);
  const double2 tw = tmp[wave];
  *exa = tw.x + (lane == 0 ? 0.0 : ba);
  *exu = tw.y + (lane == 0 ? 0.0 : bu);
  *tota = tmp[64].x;
  *totu = tmp[64].y;
}

__device__ __forceinline__ double block_excl_max(double v, double* tmp, double* total) {
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const double inc = wave_incl_max(v);
  if (lane == 63) tmp[wave] = inc;
  __syncthreads();
  if (threadIdx.x < 64) {
    const double w = threadIdx.x < unsigned(nwaves) ? tmp[threadIdx.x] : -INFINITY;
    const double wi = wave_incl_max(w);
    const double prev = __shfl_up(wi, 1, 64);
    if (threadIdx.x < unsigned(nwaves)) tmp[threadIdx.x] = threadIdx.x == 0 ? -INFINITY : prev;
    if (threadIdx.x == 63) tmp[64] = wi;
  }
  __syncthreads();
  const double before_lane = __shfl_up(inc, 1, 64);
  *total = tmp[64];
  return fmax(tmp[wave], lane == 0 ? -INFINITY : before_lane);
}

// LDS slot of position p: one pad per 32 positions, so the four
// consecutive positions each thread takes fall on distinct banks across a
// half-wave
__device__ __forceinline__ int fm_slot(int p) { return p + (p >> 5); }

struct FmLds {
  uint64_t sv[kSC + kSC / 32];  // the span's entries by position, then results
  double2 tmp2[65];             // the two sum scans
  double tmpm[65];              // the maximum scan
  uint16_t code[kFmPart + kFmPart / 32];  // a part's source codes for the transpose
  SharedRates sr;
};

// What enters sub-chunk c of worker i: read-time sum and compute-time sum
// of the reads before it, and the largest avail(g) - U(g) over them.
struct Enter {
  double a, u, m;
};

// One sub-chunk in stream order: per position, its code and the scans.
// kFinal: also the consumption times t and source codes, written out.
// A span's entries as loaded by one thread: entries t, t + kFmThreads, ...
// of its partitioned order (packed position, size and source). The loads
// are unconditional (past the span's end they read its first entry and are
// dropped when stored), so they are in flight together.
struct FmRegs {
  uint32_t j[kFmEnt];
  uint64_t v[kFmEnt];
};

__device__ __forceinline__ void fm_load(const SubChunk& s, const uint32_t* __restrict__ Pk,
                                        const uint64_t* __restrict__ zP, bool valid, FmRegs& g) {
  const int64_t base = valid ? s.base : 0, len = valid ? s.len : 0;
#pragma unroll
  for (int u = 0; u < kFmEnt; ++u) {
    const int64_t q = int64_t(u) * kFmThreads + threadIdx.x;
    g.j[u] = Pk[base + (q < len ? q : 0)];
    g.v[u] = zP[base + (q < len ? q : 0)];
  }
}

// Every entry of the span into the LDS slot of its stream position. Ends
// with a barrier.
__device__ __forceinline__ void fm_place(const SubChunk& s, const FmRegs& g, FmLds& L) {
#pragma unroll
  for (int u = 0; u < kFmEnt; ++u)
    if (int64_t(u) * kFmThreads + threadIdx.x < s.len) L.sv[fm_slot(int(g.j[u] & kJMask))] = g.v[u];
  __syncthreads();
}

// One span in stream order, its entries in L.sv: per position, its code
// and the scans. kFinal: also the consumption times t and source codes,
// written out. Ends with a barrier.
template <bool kFinal>
__device__ void fm_chunk(const SegParams& p, const SubChunk& s, const Rates& rt, FmLds& L,
                         Enter in, Enter* sum_out, int16_t* __restrict__ src,
                         double* __restrict__ tout) {
  const double inv_p0 = 1.0 / rt.p0;
  double ca = 0, cu = 0, cm = -INFINITY;  // running over the parts, relative to the chunk
  const double base_mu = in.a * inv_p0 - in.u;
  for (int64_t j0 = 0; j0 < s.len; j0 += kFmPart) {
    const uint32_t hl = uint32_t(s.len - j0 < kFmPart ? s.len - j0 : kFmPart);
    const int jb = int(j0);
    double rd[kFmPer], uu[kFmPer];
    uint32_t cd[kFmPer];
    double ta = 0, tu = 0;
#pragma unroll
    for (int u = 0; u < kFmPer; ++u) {
      const int x = int(threadIdx.x) * kFmPer + u;
      rd[u] = 0;
      uu[u] = 0;
      cd[u] = 0;
      if (x < int(hl)) {
        const uint64_t e = L.sv[fm_slot(jb + x)];
        const double sz = double(e & kSizeMask);
        cd[u] = uint32_t(e >> kSizeBits);
        rd[u] = sz * inv_rate_of(rt, L.sr, cd[u]) + sz * rt.inv_wthr;
        uu[u] = sz * rt.inv_c;
      }
      ta += rd[u];
      tu += uu[u];
    }
    double tota, totu, exa, exu;
    block_excl_sum2(ta, tu, L.tmp2, &exa, &exu, &tota, &totu);
    // avail - U at each position, relative to the chunk start
    double mv[kFmPer];
    double ra = ca + exa, ru = cu + exu, tm = -INFINITY;
#pragma unroll
    for (int u = 0; u < kFmPer; ++u) {
      const int x = int(threadIdx.x) * kFmPer + u;
      ra += rd[u];
      mv[u] = x < int(hl) ? ra * inv_p0 - ru : -INFINITY;
      ru += uu[u];
      tm = fmax(tm, mv[u]);
    }
    double totm;
    const double exm = block_excl_max(tm, L.tmpm, &totm);
    if (kFinal) {
      // t at each position: U(f) + max(what entered, base + best so far)
      double tv[kFmPer];
      double run = fmax(cm, exm);
      double uf = cu + exu;
#pragma unroll
      for (int u = 0; u < kFmPer; ++u) {
        run = fmax(run, mv[u]);
        tv[u] = (in.u + uf) + fmax(in.m, base_mu + run);
        uf += uu[u];
      }
      // t into the slots this thread read its entries from, codes into their
      // own table; one barrier, then both go out in stream order
#pragma unroll
      for (int u = 0; u < kFmPer; ++u) {
        const int x = int(threadIdx.x) * kFmPer + u;
        L.sv[fm_slot(jb + x)] = __double_as_longlong(tv[u]);
        const uint32_t c = cd[u];
        L.code[fm_slot(x)] = uint16_t(c == 0 ? 0u : (c < kOwn0 ? 128u + (c - 1) : 256u + (c - kOwn0)));
      }
      __syncthreads();
      double* td = tout + s.base + j0;
      int16_t* sd = src + s.base + j0;
#pragma unroll
      for (int u = 0; u < kFmPer; ++u) {
        const int x = u * kFmThreads + int(threadIdx.x);
        if (x < int(hl)) {
          stream_store(td + x, __longlong_as_double(L.sv[fm_slot(jb + x)]));
          stream_store(sd + x, int16_t(L.code[fm_slot(x)]));
        }
      }
    }
    ca += tota;
    cu += totu;
    cm = fmax(cm, totm);
    __syncthreads();
  }
  if (!kFinal && threadIdx.x == 0) *sum_out = Enter{ca, cu, cm};
}

// One workgroup per span and per CU (the span takes 135 KB of LDS).
// Walking several spans per workgroup with the next span's entries requested
// during the scan needs 48 more registers than the scan leaves: the spills
// made it slower (3.0 and 5.2 ms against 2.8 and 3.7).
__global__ void __launch_bounds__(kFmThreads)
fm_sum(SegParams p, const uint32_t* __restrict__ Pk, const uint64_t* __restrict__ zP, Rates rt,
       uint32_t nch, Enter* __restrict__ sums) {
  __shared__ FmLds L;
  load_rates(rt, L.sr);
  const SubChunk s = sub_chunk(p, nch, blockIdx.x);
  FmRegs g;
  fm_load(s, Pk, zP, true, g);
  fm_place(s, g, L);  // its barrier also publishes the rates
  fm_chunk<false>(p, s, rt, L, Enter{0, 0, 0}, &sums[s.i * nch + s.c], nullptr, nullptr);
}

// In place: sums[i][c] becomes what enters sub-chunk c.
__global__ void __launch_bounds__(256)
fm_scan(int64_t N, uint32_t nch, double p0, Enter* __restrict__ sums) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= N) return;
  Enter* row = sums + i * nch;
  const double inv_p0 = 1.0 / p0;
  double a = 0, u = 0, m = -INFINITY;
  for (uint32_t c = 0; c < nch; ++c) {
    const Enter x = row[c];
    row[c] = Enter{a, u, m};
    m = fmax(m, a * inv_p0 - u + x.m);
    a += x.a;
    u += x.u;
  }
}

__global__ void __launch_bounds__(kFmThreads)
fm_final(SegParams p, const uint32_t* __restrict__ Pk, const uint64_t* __restrict__ zP, Rates rt,
         uint32_t nch, const Enter* __restrict__ ins, int16_t* __restrict__ src,
         double* __restrict__ t) {
  __shared__ FmLds L;
  load_rates(rt, L.sr);
  const SubChunk s = sub_chunk(p, nch, blockIdx.x);
  FmRegs g;
  fm_load(s, Pk, zP, true, g);
  if (s.c == int64_t(nch) - 1) {
    // the row's padding past its last read
    for (int64_t f = int64_t(p.E) * s.Li + threadIdx.x; f < p.M_max; f += kFmThreads) {
      src[s.i * p.M_max + f] = -1;
      t[s.i * p.M_max + f] = -1.0;
    }
  }
  fm_place(s, g, L);
  fm_chunk<true>(p, s, rt, L, ins[s.i * nch + s.c], nullptr, src, t);
}

Rates make_rates(const nopfs_model* m) {
  Rates r{};
  r.J = m->J;
  for (int32_t j = 0; j < kMaxClasses; ++j) {
    r.own[j] = j < m->J ? m->r[j] / m->p[j] : 0;
    r.rem[j] = j < m->J ? (m->b_c < r.own[j] ? m->b_c : r.own[j]) : 0;
  }
  r.pfs = m->pfs_t / m->pfs_gamma;
  const double wb = m->w0 / m->p0;
  r.wthr = m->beta < wb ? m->beta : wb;
  r.c = m->c;
  r.p0 = m->p0;
  for (int32_t j = 0; j < kMaxClasses; ++j) {
    r.inv_own[j] = j < m->J ? 1.0 / r.own[j] : 0;
    r.inv_rem[j] = j < m->J ? 1.0 / r.rem[j] : 0;
  }
  r.inv_pfs = 1.0 / r.pfs;
  r.inv_wthr = 1.0 / r.wthr;
  r.inv_c = 1.0 / r.c;
  // classes ranked by remote rate (higher first), lower tier on ties
  int32_t order[kMaxClasses];
  for (int32_t j = 0; j < m->J; ++j) order[j] = j;
  for (int32_t a = 1; a < m->J; ++a)
    for (int32_t b = a; b > 0 && r.rem[order[b]] > r.rem[order[b - 1]]; --b) {
      const int32_t x = order[b];
      order[b] = order[b - 1];
      order[b - 1] = x;
    }
  for (int32_t q = 0; q < kMaxClasses; ++q) {
    r.rank_cls[q] = q < m->J ? uint8_t(order[q]) : uint8_t(kNoClass);
    r.cls_rank[q] = uint8_t(kNoClass);
  }
  for (int32_t q = 0; q < m->J; ++q) r.cls_rank[order[q]] = uint8_t(q);
  return r;
}

int model_impl(const nopfs_job* job, const int32_t* R, const int8_t* tier, const int64_t* sizes,
               const nopfs_model* model, int16_t* src, double* t, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if ((rc = model_check(model))) return rc;
  if (!tier || !sizes) return fail(NOPFS_EINVAL, "tier and sizes must be non-NULL");
  if (s.M_max == 0) return NOPFS_OK;
  if (!R || !src || !t) return fail(NOPFS_EINVAL, "R, src and t must be non-NULL");
  const Rates rt = make_rates(model);
  // one segment per row (the E epochs folded together), cut into spans of
  // 2^14 positions, partitioned by windows of 2^14 samples
  SegParams p = seg_params(s, gather_ws());
  const uint32_t nch = uint32_t(ceil_div(s.M_max, kSC));  // spans per row
  p.emul = int32_t(s.E);
  p.E = 1;
  p.nsc = int32_t(nch);
  const uint32_t ngroups = gather_ngroups(s.N);
  const int64_t nblk = s.N * int64_t(nch);
  const int64_t ntiles = int64_t(p.nbk) * ngroups;
  if (nblk >= (int64_t(1) << 31) || ntiles >= (int64_t(1) << 31))
    return fail(NOPFS_ERANGE, "job too large for one launch");
  Scratch scr(st);
  uint64_t *szb, *zP;
  uint32_t* Pk;
  uint16_t* OT;
  Enter* sums;
  if ((rc = scr.alloc_n(&szb, size_t(s.F)))) return rc;
  if ((rc = run_partition(p, R, scr, &Pk, &OT, st))) return rc;
  if ((rc = scr.alloc_n(&zP, size_t(s.N * s.M_max)))) return rc;
  if ((rc = scr.alloc_n(&sums, size_t(nblk)))) return rc;
  if ((rc = launch("fm_holders", fm_holders, dim3(uint32_t(ceil_div(s.F, 256))), dim3(256), 0, st,
                   s.F, s.N, tier, sizes, rt, szb)))
    return rc;
  if ((rc = launch("fm_gather", fm_gather, dim3(xcd_padded(uint32_t(ntiles))), dim3(kGThreads), 0,
                   st, p, (const uint32_t*)Pk, (const uint16_t*)OT, tier, (const uint64_t*)szb, rt,
                   zP, ngroups, uint32_t(ntiles))))
    return rc;
  if ((rc = launch("fm_sum", fm_sum, dim3(uint32_t(nblk)), dim3(kFmThreads), 0, st, p,
                   (const uint32_t*)Pk, (const uint64_t*)zP, rt, nch, sums)))
    return rc;
  if ((rc = launch("fm_scan", fm_scan, dim3(uint32_t(ceil_div(s.N, 256))), dim3(256), 0, st, s.N,
                   nch, rt.p0, sums)))
    return rc;
  return launch("fm_final", fm_final, dim3(uint32_t(nblk)), dim3(kFmThreads), 0, st, p,
                (const uint32_t*)Pk, (const uint64_t*)zP, rt, nch, (const Enter*)sums, src, t);
}

}  // namespace

int model_check(const nopfs_model* m) {
  if (!m) return fail(NOPFS_EINVAL, "model is NULL");
  if (m->J < 1) return fail(NOPFS_EINVAL, "model J must be >= 1");
  if (m->J > kMaxClasses) return fail(NOPFS_ERANGE, "model J must be <= 32");
  const double v[7] = {m->c, m->beta, m->b_c, m->pfs_t, m->pfs_gamma, m->w0, m->p0};
  for (double x : v)
    if (!(x > 0) || !isfinite(x)) return fail(NOPFS_EINVAL, "model rates and counts must be positive and finite");
  for (int32_t j = 0; j < m->J; ++j)
    if (!(m->r[j] > 0) || !(m->p[j] > 0) || !isfinite(m->r[j]) || !isfinite(m->p[j]))
      return fail(NOPFS_EINVAL, "model rates and counts must be positive and finite");
  return NOPFS_OK;
}

}  // namespace nopfs

extern "C" int nopfs_fetch_model(const nopfs_job* job, const int32_t* R, const int8_t* tier,
                                 const int64_t* sizes, const nopfs_model* model, int16_t* src,
                                 double* t, void* hip_stream) {
  try {
    return nopfs::model_impl(job, R, tier, sizes, model, src, t,
                             static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}
