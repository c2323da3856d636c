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
// consumption of any earlier read), so each worker is one wave, and the
// arithmetic is the same IEEE operations in the same order as the
// definition: results are bit-identical to a read-by-read evaluation. (The
// maxima are taken with fmax: every operand is finite and non-negative and
// never -0, where fmax and "the larger of the two" agree bit for bit.)
//
//   ps_sim -- one wave per worker (two but for Perfect, the second summing
//             the fetch times by class), 64 reads per batch, one per lane. The
//             per-read terms (u, fetch, read) and the wait p0 t(g) of every
//             lane whose g = fill(f) - 1 lies before the batch are computed
//             lane-parallel. A batch whose waits are all known runs the Q
//             chain over its 64 steps, one division Q / p0 across the lanes,
//             then the t chain; a batch with a wait inside itself steps read
//             by read, taking that wait from the batch's t register. Full
//             batches are unrolled, so later steps' operands are fetched
//             while earlier steps finish. The batch's t goes to global memory
//             and to an LDS ring of the last 8,192 positions; waits older
//             than the ring are loaded from global memory a batch ahead. Ids,
//             sources and windows are loaded two batches ahead, sizes one.

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

// Every policy but Perfect takes a second wave per worker for the fetch-time
// sums by source class (Naive and StagingBuffer: the PFS only): they depend
// on no t, so their sequential chains (stream order within each class) run
// beside the t chain instead of inside or after each batch of it.
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
  constexpr bool kStaged = kPolicy >= kStaging;
  __shared__ double ring[kPsRing];
  __shared__ double thr[kPsClasses];
  const int64_t i = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int64_t Mi = ps_row_len(r, i);
  const int64_t M = r.M_max;
  const int32_t* Rr = R + i * M;
  const int16_t* Sr = src ? src + i * M : nullptr;
  const int32_t* Fr = fill ? fill + i * M : nullptr;
  double* tr = t + i * M;
  for (int c = threadIdx.x; c < kPsClasses; c += ps_threads<kPolicy>()) thr[c] = rt.thr[c];
  __syncthreads();
  if (kPolicy != kPerfect && threadIdx.x >= 64) {
    // the second wave: fetch time by class, each class's reads in stream
    // order (ids and sources one batch ahead, sizes when they arrive)
    double a0 = 0.0, a1 = 0.0;  // class lane, class 64 + lane
    auto ids = [&](int64_t f0, int32_t& k, int32_t& code) {
      const int64_t f = f0 + lane;
      const int64_t fc = f < Mi ? f : 0;  // unconditional (Mi >= 1 inside the loop)
      k = Rr[fc];
      code = kPolicy == kNoPFS ? int32_t(Sr[fc]) : 0;
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
      if (kPolicy != kNoPFS && nb == 64) {
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

  // per-lane raw inputs of a batch: id, source code, window start (only
  // loads here, so nothing waits for them until they are used)
  auto load_ids = [&](int64_t f0, int32_t& k, int32_t& code, int32_t& fl) {
    const int64_t f = f0 + lane;
    k = -1;
    code = 0;
    fl = 0;
    if (f < Mi) {
      k = Rr[f];
      if (kPolicy == kNoPFS) code = Sr[f];
      if (kStaged) fl = Fr[f];
    }
  };
  // the lookback position g = fill - 1 of read f, clamped to [-1, f - 1]
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
  // a lookback older than the ring, loaded from global memory a batch ahead
  auto far_wait = [&](int64_t f0, int64_t g) -> double {
    return (g >= 0 && g < f0 - kPsRing) ? tr[g] : 0.0;
  };

  double Q = 0.0, tprev = 0.0, uprev = 0.0;

  // pipeline: ids two batches ahead, sizes and far lookbacks one
  int32_t kA, cA, fA, kB, cB, fB;
  load_ids(0, kB, cB, fB);
  int64_t sB = size_of(kB);
  double farB = 0.0;  // nothing is older than the ring in the first batch
  load_ids(64, kA, cA, fA);
  for (int64_t f0 = 0; f0 < Mi; f0 += 64) {
    // this batch's inputs
    const double s = double(sB);
    const int cls = ps_class(kPolicy, cB, rt.J);
    const int64_t g = kStaged ? look(f0, fB) : -1;
    const double far = farB;
    // per-read terms, lane-parallel, in the definition's expressions
    const double u = s / rt.c;
    const double fetch = s / thr[cls];
    const double rd = fetch + s / rt.wthr;
    // waits resolvable now: before the batch (ring or the far load)
    double W = 0.0;
    bool inb = false;
    if (kStaged) {
      if (g >= f0) {
        inb = true;
      } else if (g >= 0) {
        const double tg = g >= f0 - kPsRing ? ring[g & (kPsRing - 1)] : far;
        W = rt.p0 * tg;
      }
    }
    // the next batch's sizes and far lookbacks, the one after's ids
    sB = size_of(kA);
    cB = cA;
    fB = fA;
    farB = kStaged ? far_wait(f0 + 64, look(f0 + 64, fA)) : 0.0;
    load_ids(f0 + 128, kA, cA, fA);

    const int nb = Mi - f0 < 64 ? int(Mi - f0) : 64;
    double tb = -1.0;  // lane q: t of read f0 + q
    const uint64_t inb_mask = __ballot(inb);
    // one read's step; Wq is its wait (staging policies)
    auto step = [&](int q, double Wq) {
      const int64_t f = f0 + q;
      const double uq = rl_d(u, q);
      const double rq = rl_d(rd, q);
      double tf;
      if (kPolicy == kPerfect) {
        tf = f == 0 ? 0.0 : tprev + uprev;
      } else if (kPolicy == kNaive) {
        tf = f == 0 ? rq : (tprev + uprev) + rq;
      } else {
        Q = __builtin_fmax(Q, Wq);
        Q = Q + rq;
        tf = Q / rt.p0;
        if (f > 0) {
          const double a = tprev + uprev;
          tf = __builtin_fmax(tf, a);
        }
      }
      tb = lane == q ? tf : tb;
      tprev = tf;
      uprev = uq;
    };
    if (kStaged && inb_mask == 0) {
      // every wait is known: Q does not depend on this batch's t, so its
      // chain runs first, the divisions Q(f) / p0 run once across the lanes,
      // and then the t chain (the same operations as step by step)
      double Qb = 0.0;  // lane q: Q(f0 + q)
      if (nb == 64) {
#pragma unroll
        for (int q = 0; q < 64; ++q) {
          const double Wq = rl_d(W, q);
          Q = __builtin_fmax(Q, Wq);
          Q = Q + rl_d(rd, q);
          Qb = lane == q ? Q : Qb;
        }
      } else {
        for (int q = 0; q < nb; ++q) {
          const double Wq = rl_d(W, q);
          Q = __builtin_fmax(Q, Wq);
          Q = Q + rl_d(rd, q);
          Qb = lane == q ? Q : Qb;
        }
      }
      const double av = Qb / rt.p0;
      auto tstep = [&](int q) {
        double tf = rl_d(av, q);
        if (f0 + q > 0) {
          const double a = tprev + uprev;
          tf = __builtin_fmax(tf, a);
        }
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
    } else if (!kStaged && nb == 64) {
      // a full batch: straight-line steps, so the terms of later steps can
      // be formed while earlier ones finish
#pragma unroll
      for (int q = 0; q < 64; ++q) step(q, 0.0);
    } else {
      for (int q = 0; q < nb; ++q) {
        double Wq = 0.0;
        if (kStaged) {
          if ((inb_mask >> q) & 1) {
            const int gq = __builtin_amdgcn_readlane(int(g - f0), q);
            Wq = rt.p0 * rl_d(tb, gq);
          } else {
            Wq = rl_d(W, q);
          }
        }
        step(q, Wq);
      }
    }
    const int64_t f = f0 + lane;
    if (f < Mi) {
      tr[f] = tb;
      if (kStaged) ring[f & (kPsRing - 1)] = tb;
    }
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
      return launch("ps_sim_staging", ps_sim<kStaging>, grid, dim3(ps_threads<kStaging>()), 0, st, r, R, sizes, src, fill, rt, t,
                    finish, io);
    default:
      return launch("ps_sim_nopfs", ps_sim<kNoPFS>, grid, dim3(ps_threads<kNoPFS>()), 0, st, r, R, sizes, src, fill, rt, t,
                    finish, io);
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
