// nopfs_policy_sim: the data-loading policies of the Performance Simulator
// section, evaluated on the Performance Modeling section's model, read by
// read for every worker.
//
// For read f of a worker with size s: u(f) = s / c is its compute time,
// read(f) = fetch(f) + write(f) the time to stage it, write(f) =
// s / min(beta, w0 / p0) (preprocessing and buffer writes pipelined), and
// fetch(f) = s over the throughput of its source (the PFS, t(gamma) / gamma;
// another worker's tier j, min(b_c, r_j / p_j); the own tier j, r_j / p_j).
//   Perfect        t(0) = 0, t(f) = t(f-1) + u(f-1): never stalls.
//   Naive          t(0) = read(0), t(f) = t(f-1) + u(f-1) + read(f): one
//                  PFS read at a time, after the previous compute.
//   StagingBuffer  p0 threads stage reads in stream order from the PFS into
//   NoPFS          a buffer of d0 bytes (NoPFS: from the source the fetch
//                  model chose). Q(f) is the thread-time spent staging reads
//                  0..f; read f starts only once the reads before fill(f),
//                  its staging-schedule window, are consumed:
//                    Q(f) = max(Q(f-1), p0 t(fill(f) - 1)) + read(f),
//                    t(0) = Q(0) / p0, t(f) = max(Q(f) / p0, t(f-1) + u(f-1)).
// finish = t(last) + u(last); io sums fetch times by source class.
//
// The recurrence is sequential within a worker (a read may wait for the
// consumption of any earlier read), so each worker is one workgroup on one
// CU, and the arithmetic is the same IEEE operations in the same order as
// the definition: results are bit-identical to a read-by-read evaluation.
// (The maxima are taken with fmax: every operand is finite and non-negative
// and never -0, where fmax and "the larger of the two" agree bit for bit.)
// Reads go in batches of 64, one per lane: the per-read terms (u, fetch,
// read) are lane-parallel, the chains step through the batch with lane reads
// (full batches unrolled, so later steps' operands are formed while earlier
// steps finish). The fetch-time sums by class depend on no t and run in a
// wave of their own.
//
//   ps_sim    -- Perfect and Naive: one wave for the t chain (Naive: a
//                second for the PFS sum). Ids two batches ahead, sizes one.
//   ps_staged -- StagingBuffer and NoPFS: a Q wave, a T wave and a sums wave.
//                In iteration k the Q wave forms batch k's terms and its Q
//                chain (waits p0 t(g) from an LDS ring of the last 8,192
//                positions, older ones loaded from global memory a batch
//                ahead), while the T wave runs batch k - 1's t chain from the
//                Q values left in LDS (one division Q / p0 across the lanes).
//                A batch waiting on batch k - 1 gets its Q chain after the
//                iteration's first barrier; one waiting inside itself is
//                stepped read by read, Q and t, by the T wave in the next
//                iteration. The sums wave gives each class a lane.

#include <new>

#include "common.hpp"

namespace nopfs {
namespace {

constexpr int kPsRingLog = 13;
constexpr int64_t kPsRing = int64_t(1) << kPsRingLog;  // positions of t kept in LDS
constexpr int kPsMaxJ = 32;
constexpr int kPsClasses = 1 + 2 * kPsMaxJ;           // PFS, remote j, own j

enum : int32_t { kPerfect = 0, kNaive = 1, kStaging = 2, kNoPFS = 3 };

struct PsShape {
  int64_t F, N, B, M_max, E;
  int32_t drop_last;
};

// Throughputs computed once on the host, in the model's own expressions.
struct PsRates {
  double thr[kPsClasses];  // by class: 0 the PFS, 1 + j remote tier j, 1 + J + j own tier j
  double wthr;             // min(beta, w0 / p0)
  double c, p0;
  int32_t J;
};

__device__ __forceinline__ int64_t ps_row_len(const PsShape& r, int64_t i) {
  return r.E * epoch_len(r.F, r.N, r.B, r.drop_last, i);
}

__device__ __forceinline__ double rl_d(double v, int lane) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = __builtin_amdgcn_readlane(uint32_t(b), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(uint32_t(b >> 32), lane);
  return __builtin_bit_cast(double, (uint64_t(hi) << 32) | lo);
}

// class of a source code (0 the PFS, 128 + j remote, 256 + j own); any
// other code, and every code outside NoPFS, reads from the PFS
__device__ __forceinline__ int ps_class(int32_t policy, int32_t code, int32_t J) {
  if (policy != kNoPFS) return 0;
  if (code >= 128 && code < 128 + J) return 1 + (code - 128);
  if (code >= 256 && code < 256 + J) return 1 + J + (code - 256);
  return 0;
}

// Perfect and Naive. Naive takes a second wave per worker for its PFS
// fetch-time sum: it depends on no t, so its sequential chain (stream order)
// runs beside the t chain instead of inside it.
template <int32_t kPolicy>
constexpr int ps_threads() {
  return kPolicy == kPerfect ? 64 : 128;
}

template <int32_t kPolicy>
__global__ void __launch_bounds__(ps_threads<kPolicy>())
ps_sim(PsShape r, const int32_t* __restrict__ R, const int64_t* __restrict__ sizes,
       const int16_t* __restrict__ src, const int32_t* __restrict__ fill, PsRates rt,
       double* __restrict__ t, double* __restrict__ finish, double* __restrict__ io) {
#pragma clang fp contract(off)
  static_assert(kPolicy == kPerfect || kPolicy == kNaive, "the staging policies: ps_staged");
  __shared__ double thr[kPsClasses];
  const int64_t i = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int64_t Mi = ps_row_len(r, i);
  const int64_t M = r.M_max;
  const int32_t* Rr = R + i * M;
  double* tr = t + i * M;
  for (int c = threadIdx.x; c < kPsClasses; c += ps_threads<kPolicy>()) thr[c] = rt.thr[c];
  __syncthreads();
  if (kPolicy != kPerfect && threadIdx.x >= 64) {
    // the second wave: the PFS fetch time (class 0), reads in stream order
    // (ids one batch ahead, sizes when they arrive)
    double a0 = 0.0, a1 = 0.0;  // class lane, class 64 + lane
    auto ids = [&](int64_t f0, int32_t& k, int32_t& code) {
      const int64_t f = f0 + lane;
      const int64_t fc = f < Mi ? f : 0;  // unconditional (Mi >= 1 inside the loop)
      k = Rr[fc];
      code = 0;
      if (f >= Mi) k = -1;
    };
    int32_t kN = -1, cN = 0;
    if (Mi > 0) ids(0, kN, cN);
    for (int64_t f0 = 0; f0 < Mi; f0 += 64) {
      const int32_t k = kN, code = cN;
      if (f0 + 64 < Mi) ids(f0 + 64, kN, cN);
      const double s = double((k >= 0 && k < r.F) ? sizes[k] : int64_t(0));
      const int cls = ps_class(kPolicy, code, rt.J);
      const double fetch = s / thr[cls];
      const int nb = Mi - f0 < 64 ? int(Mi - f0) : 64;
      if (nb == 64) {
        // one class (the PFS) and a full batch: straight-line adds
        double a = rl_d(a0, 0);
#pragma unroll
        for (int q = 0; q < 64; ++q) a = a + rl_d(fetch, q);
        a0 = lane == 0 ? a : a0;
        continue;
      }
      uint64_t rem = nb == 64 ? ~uint64_t(0) : (uint64_t(1) << nb) - 1;
      while (rem) {
        const int c = __builtin_amdgcn_readlane(cls, __builtin_ctzll(rem));
        const uint64_t m = __ballot(cls == c) & rem;
        rem &= ~m;
        double a = c < 64 ? rl_d(a0, c) : rl_d(a1, c - 64);
        for (uint64_t mm = m; mm; mm &= mm - 1) a = a + rl_d(fetch, __builtin_ctzll(mm));
        if (c < 64) {
          a0 = lane == c ? a : a0;
        } else {
          a1 = lane == c - 64 ? a : a1;
        }
      }
    }
    const int K = 1 + 2 * rt.J;
    double* ior = io + i * K;
    if (lane < K) ior[lane] = a0;
    if (64 + lane < K) ior[64 + lane] = a1;
    return;
  }

  // per-lane raw inputs of a batch: the id (only a load here, so nothing
  // waits for it until it is used)
  auto load_ids = [&](int64_t f0, int32_t& k, int32_t& code, int32_t& fl) {
    const int64_t f = f0 + lane;
    k = -1;
    code = 0;
    fl = 0;
    if (f < Mi) k = Rr[f];
  };
  auto size_of = [&](int32_t k) -> int64_t {
    return (k >= 0 && k < r.F) ? sizes[k] : int64_t(0);
  };

  double tprev = 0.0, uprev = 0.0;

  // pipeline: ids two batches ahead, sizes one
  int32_t kA, cA, fA, kB, cB, fB;
  load_ids(0, kB, cB, fB);
  int64_t sB = size_of(kB);
  load_ids(64, kA, cA, fA);
  for (int64_t f0 = 0; f0 < Mi; f0 += 64) {
    // this batch's inputs
    const double s = double(sB);
    const int cls = ps_class(kPolicy, cB, rt.J);
    // per-read terms, lane-parallel, in the definition's expressions
    const double u = s / rt.c;
    const double fetch = s / thr[cls];
    const double rd = fetch + s / rt.wthr;
    // the next batch's sizes, the one after's ids
    sB = size_of(kA);
    cB = cA;
    fB = fA;
    load_ids(f0 + 128, kA, cA, fA);

    const int nb = Mi - f0 < 64 ? int(Mi - f0) : 64;
    double tb = -1.0;  // lane q: t of read f0 + q
    // one read's step
    auto step = [&](int q) {
      const int64_t f = f0 + q;
      const double uq = rl_d(u, q);
      const double rq = rl_d(rd, q);
      double tf;
      if (kPolicy == kPerfect) {
        tf = f == 0 ? 0.0 : tprev + uprev;
      } else {
        tf = f == 0 ? rq : (tprev + uprev) + rq;
      }
      tb = lane == q ? tf : tb;
      tprev = tf;
      uprev = uq;
    };
    if (nb == 64) {
      // a full batch: straight-line steps, so the terms of later steps can
      // be formed while earlier ones finish
#pragma unroll
      for (int q = 0; q < 64; ++q) step(q);
    } else {
      for (int q = 0; q < nb; ++q) step(q);
    }
    const int64_t f = f0 + lane;
    if (f < Mi) tr[f] = tb;
  }
  for (int64_t f = Mi + lane; f < M; f += 64) tr[f] = -1.0;
  if (kPolicy == kPerfect) {  // no fetches (the other policies' second wave writes io)
    const int K = 1 + 2 * rt.J;
    double* ior = io + i * K;
    if (lane < K) ior[lane] = 0.0;
    if (64 + lane < K) ior[64 + lane] = 0.0;
  }
  if (lane == 0) finish[i] = Mi > 0 ? tprev + uprev : 0.0;
}

// The staging policies with the Q and t chains in two waves of the worker's
// workgroup (and the fetch-time sums in a third). Iteration k: the Q wave
// forms batch k's per-read terms and, when every lookback of the batch is
// already known, its Q chain; the T wave runs batch k - 1's t chain from the
// Q values the Q wave left in LDS. Waits of batch k on batch k - 1 are known
// only once the T wave has finished it, so such a batch's Q chain runs after
// the iteration's first barrier; a batch with a lookback inside itself is
// stepped read by read (Q and t) by the T wave in the next iteration. Every
// wave passes the same two barriers per iteration, and the operations are
// those of the single-wave evaluation, in the same order.
struct PsSlot {
  double Qb[64];   // Q(f0 + q)
  double u[64];    // compute time of read f0 + q
  double rd[64];   // its staging time
  double W[64];    // its wait p0 t(g), lookbacks before the batch (stepped batches)
  int32_t gq[64];  // its lookback g - f0 (lookbacks inside the batch)
  uint64_t inb;    // lanes whose lookback is inside the batch
  int32_t near;    // the T wave steps the batch read by read
};

template <int32_t kPolicy>
__global__ void __launch_bounds__(192)
ps_staged(PsShape r, const int32_t* __restrict__ R, const int64_t* __restrict__ sizes,
          const int16_t* __restrict__ src, const int32_t* __restrict__ fill, PsRates rt,
          double* __restrict__ t, double* __restrict__ finish, double* __restrict__ io) {
#pragma clang fp contract(off)
  __shared__ double ring[kPsRing];
  __shared__ double thr[kPsClasses];
  __shared__ PsSlot slot[2];
  __shared__ double s_Qend;  // Q after the last batch the T wave stepped
  const int64_t i = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t Mi = ps_row_len(r, i);
  const int64_t M = r.M_max;
  const int32_t* Rr = R + i * M;
  const int16_t* Sr = kPolicy == kNoPFS ? src + i * M : nullptr;
  const int32_t* Fr = fill + i * M;
  double* tr = t + i * M;
  for (int c = threadIdx.x; c < kPsClasses; c += 192) thr[c] = rt.thr[c];
  if (threadIdx.x == 0) s_Qend = 0.0;
  __syncthreads();
  const int64_t nbat = (Mi + 63) / 64;

  // -- Q wave: inputs two batches ahead (ids), one ahead (sizes, far lookbacks)
  auto load_ids = [&](int64_t f0, int32_t& k, int32_t& code, int32_t& fl) {
    const int64_t f = f0 + lane;
    k = -1;
    code = 0;
    fl = 0;
    if (f < Mi) {
      k = Rr[f];
      if (kPolicy == kNoPFS) code = Sr[f];
      fl = Fr[f];
    }
  };
  auto look = [&](int64_t f0, int32_t fl) -> int64_t {
    const int64_t f = f0 + lane;
    int64_t g = int64_t(fl) - 1;
    if (g > f - 1) g = f - 1;
    if (g < -1 || f >= Mi) g = -1;
    return g;
  };
  auto size_of = [&](int32_t k) -> int64_t {
    return (k >= 0 && k < r.F) ? sizes[k] : int64_t(0);
  };
  auto far_wait = [&](int64_t f0, int64_t g) -> double {
    return (g >= 0 && g < f0 - kPsRing) ? tr[g] : 0.0;
  };
  double Q = 0.0;
  int32_t kA = -1, cA = 0, fA = 0, kB = -1, cB = 0, fB = 0;
  int64_t sB = 0;
  double farB = 0.0;
  if (wave == 0) {
    load_ids(0, kB, cB, fB);
    sB = size_of(kB);
    load_ids(64, kA, cA, fA);
  }
  // -- T wave
  double tprev = 0.0, uprev = 0.0;
  // -- io wave: fetch time by class, ids and sources one batch ahead
  double a0 = 0.0, a1 = 0.0;
  const int K = 1 + 2 * rt.J;  // source classes
  int32_t kN = -1, cN = 0;
  auto io_ids = [&](int64_t f0, int32_t& k, int32_t& code) {
    const int64_t f = f0 + lane;
    const int64_t fc = f < Mi ? f : 0;
    k = Rr[fc];
    code = kPolicy == kNoPFS ? int32_t(Sr[fc]) : 0;
    if (f >= Mi) k = -1;
  };
  if (wave == 2 && Mi > 0) io_ids(0, kN, cN);

  for (int64_t k = 0; k <= nbat; ++k) {
    const int64_t f0 = k * 64;
    // Q wave registers kept across the iteration's first barrier
    double rd = 0.0, far = 0.0;
    int64_t g = -1;
    bool q_done = false;
    // ------------------------------------------------------------ phase 1
    if (wave == 0 && k < nbat) {
      const double s = double(sB);
      const int cls = ps_class(kPolicy, cB, rt.J);
      g = look(f0, fB);
      far = farB;
      const double u = s / rt.c;
      const double fetch = s / thr[cls];
      rd = fetch + s / rt.wthr;
      sB = size_of(kA);
      cB = cA;
      fB = fA;
      farB = far_wait(f0 + 64, look(f0 + 64, fA));
      load_ids(f0 + 128, kA, cA, fA);
      PsSlot& sl = slot[k & 1];
      sl.u[lane] = u;
      sl.rd[lane] = rd;
      const bool prev_near = k > 0 && slot[(k - 1) & 1].near != 0;
      // every lookback in a batch the T wave has finished (k - 2 or before)
      if (!prev_near && __ballot(g >= f0 - 64) == 0) {
        const double tg = g >= 0 ? (g >= f0 - kPsRing ? ring[g & (kPsRing - 1)] : far) : 0.0;
        const double W = g >= 0 ? rt.p0 * tg : 0.0;
        const int nb = Mi - f0 < 64 ? int(Mi - f0) : 64;
        double Qb = 0.0;
        if (nb == 64) {
#pragma unroll
          for (int q = 0; q < 64; ++q) {
            Q = __builtin_fmax(Q, rl_d(W, q));
            Q = Q + rl_d(rd, q);
            Qb = lane == q ? Q : Qb;
          }
        } else {
          for (int q = 0; q < nb; ++q) {
            Q = __builtin_fmax(Q, rl_d(W, q));
            Q = Q + rl_d(rd, q);
            Qb = lane == q ? Q : Qb;
          }
        }
        sl.Qb[lane] = Qb;
        if (lane == 0) sl.near = 0;
        q_done = true;
      }
    }
    if (wave == 1 && k >= 1) {
      const int64_t fb = f0 - 64;
      const PsSlot& sl = slot[(k - 1) & 1];
      const int nb = Mi - fb < 64 ? int(Mi - fb) : 64;
      const double u = sl.u[lane];
      double tb = -1.0;
      if (sl.near) {
        // read by read, from the Q after the batch before
        double Qs = s_Qend;
        const double rd_l = sl.rd[lane], W_l = sl.W[lane];
        const int32_t gq_l = sl.gq[lane];
        const uint64_t inb = sl.inb;
        for (int q = 0; q < nb; ++q) {
          const double Wq = ((inb >> q) & 1) ? rt.p0 * rl_d(tb, __builtin_amdgcn_readlane(gq_l, q) & 63)
                                             : rl_d(W_l, q);
          Qs = __builtin_fmax(Qs, Wq);
          Qs = Qs + rl_d(rd_l, q);
          double tf = Qs / rt.p0;
          if (fb + q > 0) tf = __builtin_fmax(tf, tprev + uprev);
          tb = lane == q ? tf : tb;
          tprev = tf;
          uprev = rl_d(u, q);
        }
        if (lane == 0) s_Qend = Qs;
      } else {
        const double av = sl.Qb[lane] / rt.p0;
        auto tstep = [&](int q) {
          double tf = rl_d(av, q);
          if (fb + q > 0) tf = __builtin_fmax(tf, tprev + uprev);
          tb = lane == q ? tf : tb;
          tprev = tf;
          uprev = rl_d(u, q);
        };
        if (nb == 64) {
#pragma unroll
          for (int q = 0; q < 64; ++q) tstep(q);
        } else {
          for (int q = 0; q < nb; ++q) tstep(q);
        }
      }
      const int64_t f = fb + lane;
      if (f < Mi) {
        tr[f] = tb;
        ring[f & (kPsRing - 1)] = tb;
      }
    }
    if (wave == 2 && k < nbat) {
      const int32_t kk = kN, code = cN;
      if (f0 + 64 < Mi) io_ids(f0 + 64, kN, cN);
      const double s = double((kk >= 0 && kk < r.F) ? sizes[kk] : int64_t(0));
      const int cls = ps_class(kPolicy, code, rt.J);
      const double fetch = s / thr[cls];
      const int nb = Mi - f0 < 64 ? int(Mi - f0) : 64;
      if (kPolicy != kNoPFS && nb == 64) {
        double a = rl_d(a0, 0);
#pragma unroll
        for (int q = 0; q < 64; ++q) a = a + rl_d(fetch, q);
        a0 = lane == 0 ? a : a0;
      } else {
        // lane c carries class c's sum (and class 64 + c's): every step adds
        // the read's fetch time in its class's lane and 0.0 in the others,
        // so each class's sum takes its reads in stream order (the sums are
        // never -0, so adding +0.0 leaves them bit for bit)
        auto cstep = [&](int q) {
          const int cq = __builtin_amdgcn_readlane(cls, q);
          const double fq = rl_d(fetch, q);
          a0 = a0 + (cq == lane ? fq : 0.0);
          if (K > 64) a1 = a1 + (cq == lane + 64 ? fq : 0.0);
        };
        if (nb == 64) {
#pragma unroll
          for (int q = 0; q < 64; ++q) cstep(q);
        } else {
          for (int q = 0; q < nb; ++q) cstep(q);
        }
      }
    }
    __syncthreads();  // A: batch k - 1's t, and a stepped batch's Q, are in
    // ------------------------------------------------------------ phase 2
    if (wave == 0 && k < nbat && !q_done) {
      PsSlot& sl = slot[k & 1];
      if (k > 0 && slot[(k - 1) & 1].near != 0) Q = s_Qend;
      const bool inb = g >= f0;
      const double tg = (g >= 0 && !inb) ? (g >= f0 - kPsRing ? ring[g & (kPsRing - 1)] : far) : 0.0;
      const double W = (g >= 0 && !inb) ? rt.p0 * tg : 0.0;
      const uint64_t inb_mask = __ballot(inb);
      if (inb_mask == 0) {
        const int nb = Mi - f0 < 64 ? int(Mi - f0) : 64;
        double Qb = 0.0;
        for (int q = 0; q < nb; ++q) {
          Q = __builtin_fmax(Q, rl_d(W, q));
          Q = Q + rl_d(rd, q);
          Qb = lane == q ? Q : Qb;
        }
        sl.Qb[lane] = Qb;
        if (lane == 0) sl.near = 0;
      } else {
        sl.W[lane] = W;
        sl.gq[lane] = int32_t(g - f0);
        if (lane == 0) {
          sl.inb = inb_mask;
          sl.near = 1;
        }
      }
    }
    __syncthreads();  // B: batch k's Q values or its stepping data are in
  }
  if (wave == 1) {
    for (int64_t f = Mi + lane; f < M; f += 64) tr[f] = -1.0;
    if (lane == 0) finish[i] = Mi > 0 ? tprev + uprev : 0.0;
  }
  if (wave == 2) {
    double* ior = io + i * K;
    if (lane < K) ior[lane] = a0;
    if (64 + lane < K) ior[64 + lane] = a1;
  }
}

int policy_impl(const nopfs_job* job, const int32_t* R, const int64_t* sizes, const int16_t* src,
                const int32_t* fill, const nopfs_model* model, int32_t policy, double* t,
                double* finish, double* io, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if ((rc = model_check(model))) return rc;
  if (policy < kPerfect || policy > kNoPFS) return fail(NOPFS_EINVAL, "policy must be 0..3");
  if (!sizes || !finish || !io) return fail(NOPFS_EINVAL, "sizes, finish and io must be non-NULL");
  if (s.M_max > 0) {
    if (!R || !t) return fail(NOPFS_EINVAL, "R and t must be non-NULL");
    if (policy >= kStaging && !fill) return fail(NOPFS_EINVAL, "fill must be non-NULL for the staging policies");
    if (policy == kNoPFS && !src) return fail(NOPFS_EINVAL, "src must be non-NULL for NoPFS");
  }
  if (s.N >= (int64_t(1) << 31)) return fail(NOPFS_ERANGE, "N too large for one launch");
  PsShape r{s.F, s.N, s.B, s.M_max, s.E, s.drop_last};
  PsRates rt{};
  rt.J = model->J;
  rt.thr[0] = model->pfs_t / model->pfs_gamma;
  for (int32_t j = 0; j < model->J; ++j) {
    const double own = model->r[j] / model->p[j];
    rt.thr[1 + j] = model->b_c < own ? model->b_c : own;
    rt.thr[1 + model->J + j] = own;
  }
  for (int c = 1 + 2 * model->J; c < kPsClasses; ++c) rt.thr[c] = rt.thr[0];
  const double wb = model->w0 / model->p0;
  rt.wthr = model->beta < wb ? model->beta : wb;
  rt.c = model->c;
  rt.p0 = model->p0;
  const dim3 grid(uint32_t(s.N));
  switch (policy) {
    case kPerfect:
      return launch("ps_sim_perfect", ps_sim<kPerfect>, grid, dim3(ps_threads<kPerfect>()), 0, st, r, R, sizes, src, fill, rt, t,
                    finish, io);
    case kNaive:
      return launch("ps_sim_naive", ps_sim<kNaive>, grid, dim3(ps_threads<kNaive>()), 0, st, r, R, sizes, src, fill, rt, t,
                    finish, io);
    case kStaging:
      return launch("ps_sim_staging", ps_staged<kStaging>, grid, dim3(192), 0, st, r, R, sizes, src, fill,
                    rt, t, finish, io);
    default:
      return launch("ps_sim_nopfs", ps_staged<kNoPFS>, grid, dim3(192), 0, st, r, R, sizes, src, fill,
                    rt, t, finish, io);
  }
}

}  // namespace
}  // namespace nopfs

extern "C" int nopfs_policy_sim(const nopfs_job* job, const int32_t* R, const int64_t* sizes,
                                const int16_t* src, const int32_t* fill, const nopfs_model* model,
                                int32_t policy, double* t, double* finish, double* io,
                                void* hip_stream) {
  try {
    return nopfs::policy_impl(job, R, sizes, src, fill, model, policy, t, finish, io,
                              static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}
