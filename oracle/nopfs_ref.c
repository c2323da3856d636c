/*
 * nopfs_ref.c -- CPU oracle for the clairvoyant planning path of NoPFS
 * (Dryden, Boehringer, Ben-Nun, Hoefler, "Clairvoyant Prefetching for
 * Distributed Machine Learning I/O", SC'21).
 *
 * TEST INFRASTRUCTURE ONLY. Plain, slow, single-threaded C. It is called by
 * the test suite, the smoke check and the benchmark's CPU-baseline leg, and by
 * nothing in the product path. It shares no source with the GPU library.
 *
 * Every stage is written as the plain definition, in the paper's order:
 *   keys   -> one 32-bit Philox-4x32-10 word per (epoch, sample)
 *   perm   -> samples sorted by (key, id)        (Background: one shuffle per
 *             epoch, every sample exactly once, reproducible from the seed)
 *   shard  -> worker i reads global positions p = i (mod N) of each epoch, in
 *             order, giving its access stream R (Performance Modeling: the
 *             batches B^h, the worker batches B^{h,i} and the stream R)
 *   stats  -> per (worker, sample): number of reads and first read position
 *             (Distribution of Accesses: the access frequency X / r_k)
 *   next   -> per stream position: the next position reading the same sample
 *             (I/O Access Patterns: Belady's rule needs the next use)
 *   plan   -> per worker, samples ranked by frequency, then poured into the
 *             storage classes fastest first until full (Design, last steps)
 *
 * Readings where the paper is silent (each is stated where it is used):
 *   - keys are Philox-4x32-10 words: counter (k/4, e, 0, 0), key (seed lo,
 *     seed hi), word k%4; equal keys are ordered by the smaller sample id;
 *   - ids, epochs and positions are 0-based;
 *   - B is the per-worker batch; the global batch is N*B;
 *   - worker i takes global positions p with p % N == i (strided split);
 *   - drop_last=1 issues the first T*N*B positions of each epoch; with
 *     drop_last=0 every position is issued and rows are padded with -1;
 *   - "first" and "next" are positions in the worker's own stream, -1 = never;
 *   - the plan ranks by (count desc, first asc with never = +inf, id asc),
 *     fills tier 0, then tier 1, ..., stopping each tier at its first misfit;
 *     samples never read by a worker are ranked last, by id, and still placed.
 */
#include "nopfs_ref.h"

#include <stdlib.h>
#include <string.h>

#define REF_EINVAL (-1)
#define REF_ERANGE (-2)
#define REF_ENOMEM (-3)

/* ------------------------------------------------------------------------ */
/* Philox-4x32-10, from the description in Salmon et al., SC'11:             */
/* each round multiplies words 0 and 2 by two fixed 32-bit constants, takes  */
/* the high halves, XORs them with the other two words and the round key,    */
/* and the round key is bumped by two Weyl constants between rounds.         */
/* ------------------------------------------------------------------------ */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void nopfs_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                             uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    uint64_t p0 = (uint64_t)PHILOX_M0 * x0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * x2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t y0 = hi1 ^ x1 ^ k0;
    uint32_t y1 = lo1;
    uint32_t y2 = hi0 ^ x3 ^ k1;
    uint32_t y3 = lo0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    k0 += PHILOX_W0;
    k1 += PHILOX_W1;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* ------------------------------------------------------------------------ */
/* Shape (Performance Modeling: T iterations per epoch, floor or ceil of    */
/* F over the global batch; worker batches partition each global batch).    */
/* ------------------------------------------------------------------------ */
static int check_job(const nopfs_ref_job* job) {
  if (!job) return REF_EINVAL;
  if (job->F < 1 || job->E < 1 || job->N < 1 || job->B < 1) return REF_EINVAL;
  if (job->drop_last != 0 && job->drop_last != 1) return REF_EINVAL;
  if (job->F >= ((int64_t)1 << 31) || job->E > 255) return REF_ERANGE;
  return 0;
}

/* Length of worker i's stream in one epoch. */
static int64_t epoch_len(const nopfs_ref_job* job, int64_t i) {
  int64_t F = job->F, N = job->N, B = job->B;
  if (job->drop_last) {
    int64_t T = F / (N * B);
    return T * B;
  }
  if (i >= F) return 0;
  return (F - i + N - 1) / N; /* positions p < F with p % N == i */
}

/* Number of positions of each epoch that are actually read. */
static int64_t issued(const nopfs_ref_job* job) {
  int64_t F = job->F, N = job->N, B = job->B;
  if (job->drop_last) return (F / (N * B)) * N * B;
  return F;
}

int nopfs_ref_stream_shape(const nopfs_ref_job* job, int64_t* T, int64_t* M_max,
                           int64_t* M_per_worker) {
  int rc = check_job(job);
  if (rc) return rc;
  int64_t F = job->F, N = job->N, B = job->B, E = job->E;
  int64_t t = job->drop_last ? F / (N * B) : (F + N * B - 1) / (N * B);
  int64_t mmax = 0;
  for (int64_t i = 0; i < N; ++i) {
    int64_t m = E * epoch_len(job, i);
    if (m > mmax) mmax = m;
    if (M_per_worker) M_per_worker[i] = m;
  }
  if (mmax >= ((int64_t)1 << 31)) return REF_ERANGE;
  if (T) *T = t;
  if (M_max) *M_max = mmax;
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Keys and the epoch permutation (Background: each epoch is a random       */
/* shuffle of all sample indices, and knowing the seed reproduces it).      */
/* ------------------------------------------------------------------------ */
int nopfs_ref_epoch_keys(const nopfs_ref_job* job, int32_t e, uint32_t* keys) {
  int rc = check_job(job);
  if (rc) return rc;
  if (!keys || e < 0 || e >= job->E) return REF_EINVAL;
  uint32_t key[2] = {(uint32_t)job->seed, (uint32_t)(job->seed >> 32)};
  for (int64_t k = 0; k < job->F; ++k) {
    uint32_t ctr[4] = {(uint32_t)(k >> 2), (uint32_t)e, 0u, 0u};
    uint32_t out[4];
    nopfs_ref_philox4x32_10(ctr, key, out);
    keys[k] = out[k & 3];
  }
  return 0;
}

typedef struct { uint32_t key; int32_t id; } keyed_t;

static int cmp_keyed(const void* a, const void* b) {
  const keyed_t* x = (const keyed_t*)a;
  const keyed_t* y = (const keyed_t*)b;
  if (x->key != y->key) return x->key < y->key ? -1 : 1;
  if (x->id != y->id) return x->id < y->id ? -1 : 1;
  return 0;
}

int nopfs_ref_epoch_perm(const nopfs_ref_job* job, int32_t e, int32_t* perm) {
  int rc = check_job(job);
  if (rc) return rc;
  if (!perm || e < 0 || e >= job->E) return REF_EINVAL;
  int64_t F = job->F;
  uint32_t* keys = (uint32_t*)malloc((size_t)F * sizeof(uint32_t));
  keyed_t* rec = (keyed_t*)malloc((size_t)F * sizeof(keyed_t));
  if (!keys || !rec) { free(keys); free(rec); return REF_ENOMEM; }
  nopfs_ref_epoch_keys(job, e, keys);
  for (int64_t k = 0; k < F; ++k) { rec[k].key = keys[k]; rec[k].id = (int32_t)k; }
  qsort(rec, (size_t)F, sizeof(keyed_t), cmp_keyed);
  for (int64_t p = 0; p < F; ++p) perm[p] = rec[p].id;
  free(keys);
  free(rec);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Shard (Performance Modeling: B^{h,1..N} partition B^h, and worker i's    */
/* stream R is the concatenation of its local batches in iteration order).  */
/* With the strided split, the j-th read of worker i in epoch e is global    */
/* position p = j*N + i, and it lands at stream position e*L_i + j.          */
/* ------------------------------------------------------------------------ */
static void shard_epoch(const nopfs_ref_job* job, int32_t e, const int32_t* perm,
                        int64_t M_max, int32_t* R) {
  int64_t N = job->N, P = issued(job);
  for (int64_t p = 0; p < P; ++p) {
    int64_t i = p % N, j = p / N;
    int64_t L = epoch_len(job, i);
    R[i * M_max + (int64_t)e * L + j] = perm[p];
  }
}

static void pad_rows(const nopfs_ref_job* job, int64_t M_max, int32_t* R) {
  for (int64_t i = 0; i < job->N; ++i) {
    int64_t M = (int64_t)job->E * epoch_len(job, i);
    for (int64_t f = M; f < M_max; ++f) R[i * M_max + f] = -1;
  }
}

int nopfs_ref_streams_from_perms(const nopfs_ref_job* job, const int32_t* perms,
                                 int32_t* R) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if (!perms || !R) return REF_EINVAL;
  pad_rows(job, M_max, R);
  for (int32_t e = 0; e < job->E; ++e)
    shard_epoch(job, e, perms + (int64_t)e * job->F, M_max, R);
  return 0;
}

/* Rows [i0, i1) of the same streams, walked row by row: worker i's j-th read
 * of epoch e is global position j*N + i, for each of its L_i reads per epoch
 * (positions past the issued prefix belong to no worker's L_i reads). R
 * points at row i0; rows are padded with -1 like the full streams. */
int nopfs_ref_streams_rows(const nopfs_ref_job* job, const int32_t* perms, int64_t i0,
                           int64_t i1, int32_t* R) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if (!perms || !R || i0 < 0 || i1 > job->N || i0 > i1) return REF_EINVAL;
  int64_t N = job->N, F = job->F;
  for (int64_t i = i0; i < i1; ++i) {
    int32_t* row = R + (i - i0) * M_max;
    int64_t L = epoch_len(job, i);
    for (int32_t e = 0; e < job->E; ++e)
      for (int64_t j = 0; j < L; ++j) row[(int64_t)e * L + j] = perms[(int64_t)e * F + j * N + i];
    for (int64_t f = (int64_t)job->E * L; f < M_max; ++f) row[f] = -1;
  }
  return 0;
}

int nopfs_ref_access_streams(const nopfs_ref_job* job, int32_t* R) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if (!R) return REF_EINVAL;
  int32_t* perm = (int32_t*)malloc((size_t)job->F * sizeof(int32_t));
  if (!perm) return REF_ENOMEM;
  pad_rows(job, M_max, R);
  for (int32_t e = 0; e < job->E; ++e) {
    rc = nopfs_ref_epoch_perm(job, e, perm);
    if (rc) break;
    shard_epoch(job, e, perm, M_max, R);
  }
  free(perm);
  return rc;
}

/* ------------------------------------------------------------------------ */
/* Access statistics (Distribution of Accesses: the number of times a       */
/* worker reads a sample over all E epochs; the first read time is kept so  */
/* the plan can order equally frequent samples).                            */
/* ------------------------------------------------------------------------ */
int nopfs_ref_access_stats_rows(const nopfs_ref_job* job, const int32_t* R,
                                int64_t i0, int64_t i1, uint8_t* count,
                                int32_t* first) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if (!R || !count || !first || i0 < 0 || i1 > job->N || i0 > i1) return REF_EINVAL;
  int64_t F = job->F;
  for (int64_t i = i0; i < i1; ++i) {
    uint8_t* c = count + (i - i0) * F;
    int32_t* fi = first + (i - i0) * F;
    const int32_t* row = R + (i - i0) * M_max;
    for (int64_t k = 0; k < F; ++k) { c[k] = 0; fi[k] = -1; }
    int64_t M = (int64_t)job->E * epoch_len(job, i);
    for (int64_t f = 0; f < M; ++f) {
      int32_t k = row[f];
      if (k < 0 || k >= F) return REF_EINVAL;
      if (c[k] == 0) fi[k] = (int32_t)f;
      c[k] += 1;
    }
  }
  return 0;
}

int nopfs_ref_access_stats(const nopfs_ref_job* job, const int32_t* R,
                           uint8_t* count, int32_t* first) {
  int rc = check_job(job);
  if (rc) return rc;
  return nopfs_ref_access_stats_rows(job, R, 0, job->N, count, first);
}

/* ------------------------------------------------------------------------ */
/* Next use (I/O Access Patterns: the optimal replacement discards the      */
/* sample whose next use is furthest; the next use is found by walking the  */
/* stream backwards and remembering the last position seen per sample).     */
/* ------------------------------------------------------------------------ */
int nopfs_ref_reuse_next_rows(const nopfs_ref_job* job, const int32_t* R,
                              int64_t i0, int64_t i1, int32_t* next) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if (!R || !next || i0 < 0 || i1 > job->N || i0 > i1) return REF_EINVAL;
  int64_t F = job->F;
  int32_t* last = (int32_t*)malloc((size_t)F * sizeof(int32_t));
  if (!last) return REF_ENOMEM;
  for (int64_t i = i0; i < i1; ++i) {
    const int32_t* row = R + (i - i0) * M_max;
    int32_t* nrow = next + (i - i0) * M_max;
    for (int64_t k = 0; k < F; ++k) last[k] = -1;
    int64_t M = (int64_t)job->E * epoch_len(job, i);
    for (int64_t f = M; f < M_max; ++f) nrow[f] = -1;
    for (int64_t f = M - 1; f >= 0; --f) {
      int32_t k = row[f];
      if (k < 0 || k >= F) { free(last); return REF_EINVAL; }
      nrow[f] = last[k];
      last[k] = (int32_t)f;
    }
  }
  free(last);
  return 0;
}

int nopfs_ref_reuse_next(const nopfs_ref_job* job, const int32_t* R,
                         int32_t* next) {
  int rc = check_job(job);
  if (rc) return rc;
  return nopfs_ref_reuse_next_rows(job, R, 0, job->N, next);
}

/* ------------------------------------------------------------------------ */
/* Tier plan (Design: a worker caches the samples with the largest access    */
/* frequency r_k in its fastest storage class, then the next class, and so  */
/* on, until the dataset is cached or local storage is full).               */
/* ------------------------------------------------------------------------ */
typedef struct { int32_t count; int64_t first; int32_t id; } ranked_t;

static int cmp_ranked(const void* a, const void* b) {
  const ranked_t* x = (const ranked_t*)a;
  const ranked_t* y = (const ranked_t*)b;
  if (x->count != y->count) return x->count > y->count ? -1 : 1;  /* desc */
  if (x->first != y->first) return x->first < y->first ? -1 : 1;  /* asc  */
  if (x->id != y->id) return x->id < y->id ? -1 : 1;              /* asc  */
  return 0;
}

int nopfs_ref_tier_plan(const nopfs_ref_job* job, const uint8_t* count,
                        const int32_t* first, const int64_t* sizes,
                        const int64_t* caps, int32_t J, int8_t* tier,
                        int64_t* used) {
  int rc = check_job(job);
  if (rc) return rc;
  if (!count || !first || !sizes || !caps || !tier || !used) return REF_EINVAL;
  if (J < 1) return REF_EINVAL;
  if (J > 127) return REF_ERANGE;
  for (int32_t j = 0; j < J; ++j)
    if (caps[j] < 0) return REF_EINVAL;
  int64_t F = job->F;
  ranked_t* order = (ranked_t*)malloc((size_t)F * sizeof(ranked_t));
  if (!order) return REF_ENOMEM;
  for (int64_t i = 0; i < job->N; ++i) {
    for (int64_t k = 0; k < F; ++k) {
      order[k].count = count[i * F + k];
      order[k].first = first[i * F + k] >= 0 ? first[i * F + k] : INT64_MAX;
      order[k].id = (int32_t)k;
    }
    qsort(order, (size_t)F, sizeof(ranked_t), cmp_ranked);
    int64_t pos = 0;
    for (int32_t j = 0; j < J; ++j) {
      int64_t u = 0;
      while (pos < F && u + sizes[order[pos].id] <= caps[j]) {
        tier[i * F + order[pos].id] = (int8_t)j;
        u += sizes[order[pos].id];
        pos++;
      }
      used[i * J + j] = u;
    }
    for (int64_t q = pos; q < F; ++q) tier[i * F + order[q].id] = -1;
  }
  free(order);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Prefetch order (Design: a worker fills each storage class in the order it */
/* will first need the samples -- the first rule of optimal prefetching of   */
/* I/O Access Patterns, fetch the next sample of R that is not cached).      */
/* Walk R_i; at the first read of a sample placed in tier j, append it to    */
/* tier j's queue.                                                           */
/* ------------------------------------------------------------------------ */
int nopfs_ref_prefetch_order(const nopfs_ref_job* job, const int32_t* R,
                             const int32_t* first, const int8_t* tier, int32_t J,
                             int32_t* order, int64_t* qlen) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if ((!R && M_max > 0) || !first || !tier || !qlen || (!order && M_max > 0)) return REF_EINVAL;
  if (J < 1) return REF_EINVAL;
  if (J > 127) return REF_ERANGE;
  int64_t F = job->F;
  for (int64_t i = 0; i < job->N; ++i) {
    const int32_t* Ri = R ? R + i * M_max : NULL;
    int64_t Mi = job->E * epoch_len(job, i);
    /* pass 1: queue lengths; pass 2: each queue in stream order */
    for (int32_t j = 0; j < J; ++j) qlen[i * J + j] = 0;
    for (int64_t f = 0; f < Mi; ++f) {
      int32_t k = Ri[f];
      int8_t t = tier[i * F + k];
      if (first[i * F + k] == f && t >= 0 && t < J) qlen[i * J + t]++;
    }
    int64_t start[128];
    int64_t acc = 0;
    for (int32_t j = 0; j < J; ++j) {
      start[j] = acc;
      acc += qlen[i * J + j];
    }
    for (int64_t f = 0; f < Mi; ++f) {
      int32_t k = Ri[f];
      int8_t t = tier[i * F + k];
      if (first[i * F + k] == f && t >= 0 && t < J) order[i * M_max + start[t]++] = k;
    }
    for (int64_t q = acc; q < M_max; ++q) order[i * M_max + q] = -1;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Staging schedule (Design: the staging buffer is filled in the order of R  */
/* and a sample is dropped as soon as it has been read; Implementation: the  */
/* buffer is filled circularly). While the worker has read positions < f,    */
/* the buffer holds the samples at f, f+1, ...; the sample at h can be       */
/* fetched once those at f..h fit in d0 bytes. The window's left end only    */
/* moves forward as h grows (sizes are >= 1), so one running sum does.       */
/* ------------------------------------------------------------------------ */
int nopfs_ref_staging_schedule(const nopfs_ref_job* job, const int32_t* R,
                               const int64_t* sizes, int64_t d0, int32_t* fill) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if ((!R && M_max > 0) || !sizes || (!fill && M_max > 0)) return REF_EINVAL;
  if (d0 < 0) return REF_EINVAL;
  for (int64_t i = 0; i < job->N; ++i) {
    const int32_t* Ri = R ? R + i * M_max : NULL;
    int64_t Mi = job->E * epoch_len(job, i);
    int64_t f = 0, sum = 0; /* sum of sizes at positions f..h */
    for (int64_t h = 0; h < Mi; ++h) {
      sum += sizes[Ri[h]];
      while (sum > d0 && f < h) {
        sum -= sizes[Ri[f]];
        f++;
      }
      fill[i * M_max + h] = (int32_t)f; /* f == h: alone, or alone too large */
    }
    for (int64_t h = Mi; h < M_max; ++h) fill[i * M_max + h] = -1;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Performance model (section 4). Worker i consumes its f-th read at         */
/*   t(f) = max(avail(f), t(f-1) + s(R[f-1]) / c),                          */
/* where avail(f) = (read time of R[0..f] summed) / p0 is when the read is  */
/* in the staging buffer (prefetch threads load-balanced), and a read takes */
/* fetch + write: write = max(s / beta, s / (w0 / p0)) (preprocessing and   */
/* buffer writes pipelined), fetch = s over the fastest applicable          */
/* throughput among the PFS (t(gamma) / gamma), another worker's tier j     */
/* (min(b_c, r_j / p_j)) and the worker's own tier j (r_j / p_j). The first */
/* read has no predecessor: t(0) = avail(0). Placement is static: a sample  */
/* is in tier j of worker i exactly when tier[i][k] == j.                   */
/* ------------------------------------------------------------------------ */
static int model_ok(const nopfs_ref_model* m) {
  if (!m || m->J < 1 || m->J > 32) return 0;
  const double v[7] = {m->c, m->beta, m->b_c, m->pfs_t, m->pfs_gamma, m->w0, m->p0};
  for (int q = 0; q < 7; ++q)
    if (!(v[q] > 0) || v[q] * 0 != 0) return 0; /* positive and finite */
  for (int32_t j = 0; j < m->J; ++j)
    if (!(m->r[j] > 0) || !(m->p[j] > 0) || m->r[j] * 0 != 0 || m->p[j] * 0 != 0) return 0;
  return 1;
}

int nopfs_ref_fetch_model_rows(const nopfs_ref_job* job, const int32_t* R,
                               const int8_t* tier, const int64_t* sizes,
                               const nopfs_ref_model* m, int64_t i0, int64_t i1,
                               int16_t* src, double* t) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if (!tier || !sizes || !model_ok(m)) return REF_EINVAL;
  if (i0 < 0 || i1 > job->N || i0 > i1) return REF_EINVAL;
  if (M_max > 0 && i1 > i0 && (!R || !src || !t)) return REF_EINVAL;
  const int64_t F = job->F, N = job->N;
  const int32_t J = m->J;
  /* holders[k][j]: how many workers hold sample k in tier j */
  int32_t* holders = (int32_t*)calloc((size_t)F * (size_t)J, sizeof(int32_t));
  if (!holders) return REF_ENOMEM;
  for (int64_t w = 0; w < N; ++w)
    for (int64_t k = 0; k < F; ++k) {
      int8_t q = tier[w * F + k];
      if (q >= 0 && q < J) holders[k * J + q]++;
    }
  const double pfs = m->pfs_t / m->pfs_gamma;
  for (int64_t i = i0; i < i1; ++i) {
    const int32_t* Ri = R + (i - i0) * M_max;
    int16_t* si = src + (i - i0) * M_max;
    double* ti = t + (i - i0) * M_max;
    int64_t Mi = job->E * epoch_len(job, i);
    double read_sum = 0, t_prev = 0, s_prev = 0;
    for (int64_t f = 0; f < Mi; ++f) {
      int32_t k = Ri[f];
      double s = (double)sizes[k];
      int8_t own = tier[i * F + k];
      /* candidates in order of preference; a later one must be strictly faster */
      double best = -1;
      int16_t code = 0;
      if (own >= 0 && own < J) {
        best = m->r[own] / m->p[own];
        code = (int16_t)(256 + own);
      }
      for (int32_t j = 0; j < J; ++j) {
        int32_t elsewhere = holders[(int64_t)k * J + j] - (own == j ? 1 : 0);
        if (elsewhere > 0) {
          double thr = m->r[j] / m->p[j];
          if (m->b_c < thr) thr = m->b_c;
          if (thr > best) {
            best = thr;
            code = (int16_t)(128 + j);
          }
        }
      }
      if (pfs > best) {
        best = pfs;
        code = 0;
      }
      double fetch = s / best;
      double wr = s / m->beta;
      double wb = s / (m->w0 / m->p0);
      if (wb > wr) wr = wb;
      read_sum += fetch + wr;
      double avail = read_sum / m->p0;
      double tf = avail;
      if (f > 0 && t_prev + s_prev / m->c > tf) tf = t_prev + s_prev / m->c;
      si[f] = code;
      ti[f] = tf;
      t_prev = tf;
      s_prev = s;
    }
    for (int64_t f = Mi; f < M_max; ++f) {
      si[f] = -1;
      ti[f] = -1.0;
    }
  }
  free(holders);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Policy simulation (section 6: the Perfect, Naive, StagingBuffer and       */
/* NoPFS policies on the section 4 model). For read f of a worker, with      */
/* s its size: u(f) = s / c is its compute time, read(f) = fetch(f) +       */
/* write(f) the time to stage it, write(f) = max(s / beta, s / (w0 / p0)),  */
/* fetch(f) = s over the throughput of its source.                          */
/*   Perfect:       never stalls: t(0) = 0, t(f) = t(f-1) + u(f-1).         */
/*   Naive:         one read at a time from the PFS, after the previous     */
/*                  compute: t(0) = read(0), t(f) = t(f-1) + u(f-1) + read(f)*/
/*   StagingBuffer: p0 threads stage the reads in stream order from the PFS */
/*   NoPFS:         the same, each read from the source src gives.          */
/* The two staging policies keep Q(f), the thread-time spent staging reads  */
/* 0..f (so avail(f) = Q(f) / p0 as in section 4), with the buffer of d0    */
/* bytes as the extra condition that read f can start only once the reads   */
/* before fill(f) (the staging schedule) are consumed:                      */
/*   Q(f) = max(Q(f-1), p0 * t(fill(f) - 1)) + read(f)   (t(-1) = 0),       */
/*   t(0) = Q(0) / p0,  t(f) = max(Q(f) / p0, t(f-1) + u(f-1)).             */
/* finish = t(last) + u(last); io[c] sums fetch times by source class c:    */
/* 0 the PFS, 1 + j another worker's tier j, 1 + J + j the own tier j.      */
/* ------------------------------------------------------------------------ */
int nopfs_ref_policy_sim_rows(const nopfs_ref_job* job, const int32_t* R, const int64_t* sizes,
                              const int16_t* src, const int32_t* fill, const nopfs_ref_model* m,
                              int32_t policy, int64_t i0, int64_t i1, double* t, double* finish,
                              double* io) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if (!sizes || !model_ok(m) || policy < 0 || policy > 3) return REF_EINVAL;
  if (i0 < 0 || i1 > job->N || i0 > i1) return REF_EINVAL;
  if (i1 > i0 && (!finish || !io)) return REF_EINVAL;
  if (M_max > 0 && i1 > i0) {
    if (!R || !t) return REF_EINVAL;
    if (policy >= 2 && !fill) return REF_EINVAL;
    if (policy == 3 && !src) return REF_EINVAL;
  }
  const int32_t J = m->J;
  const int64_t K = 1 + 2 * (int64_t)J;
  const double pfs = m->pfs_t / m->pfs_gamma;
  for (int64_t i = i0; i < i1; ++i) {
    const int64_t row = (i - i0) * M_max;
    double* ti = t ? t + row : NULL;
    double* ioi = io + (i - i0) * K;
    for (int64_t c = 0; c < K; ++c) ioi[c] = 0.0;
    int64_t Mi = job->E * epoch_len(job, i);
    double Q = 0, t_prev = 0, u_prev = 0;
    for (int64_t f = 0; f < Mi; ++f) {
      double s = (double)sizes[R[row + f]];
      double u = s / m->c;
      /* the source: the PFS unless NoPFS names a valid tier */
      double thr = pfs;
      int64_t cls = 0;
      if (policy == 3) {
        int32_t code = src[row + f];
        if (code >= 128 && code < 128 + J) {
          int32_t j = code - 128;
          thr = m->r[j] / m->p[j];
          if (m->b_c < thr) thr = m->b_c;
          cls = 1 + j;
        } else if (code >= 256 && code < 256 + J) {
          int32_t j = code - 256;
          thr = m->r[j] / m->p[j];
          cls = 1 + J + j;
        }
      }
      double fetch = s / thr;
      double wr = s / m->beta;
      double wb = s / (m->w0 / m->p0);
      if (wb > wr) wr = wb;
      double rd = fetch + wr;
      double tf;
      if (policy == 0) {
        tf = f == 0 ? 0.0 : t_prev + u_prev;
      } else if (policy == 1) {
        tf = f == 0 ? rd : (t_prev + u_prev) + rd;
      } else {
        /* the latest consumed read the buffer must wait for */
        int64_t g = (int64_t)fill[row + f] - 1;
        if (g > f - 1) g = f - 1;
        double wait = g >= 0 ? m->p0 * ti[g] : 0.0;
        if (wait > Q) Q = wait;
        Q = Q + rd;
        tf = Q / m->p0;
        if (f > 0 && t_prev + u_prev > tf) tf = t_prev + u_prev;
      }
      if (policy != 0) ioi[cls] += fetch;
      ti[f] = tf;
      t_prev = tf;
      u_prev = u;
    }
    for (int64_t f = Mi; f < M_max; ++f) ti[f] = -1.0;
    finish[i - i0] = Mi > 0 ? t_prev + u_prev : 0.0;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Clairvoyant buffer (section 3). Held entries are keyed by the stream     */
/* position of their next use, so at position f the sample read is held     */
/* exactly when key f is. A binary max-heap of keys with lazy deletion (a   */
/* popped key that is no longer held is skipped) gives the furthest entry. */
/* ------------------------------------------------------------------------ */
static void heap_push(int32_t* h, int64_t* n, int32_t key) {
  int64_t i = (*n)++;
  h[i] = key;
  while (i > 0 && h[(i - 1) / 2] < h[i]) {
    int32_t t = h[i];
    h[i] = h[(i - 1) / 2];
    h[(i - 1) / 2] = t;
    i = (i - 1) / 2;
  }
}

static int32_t heap_pop(int32_t* h, int64_t* n) {
  int32_t top = h[0];
  h[0] = h[--(*n)];
  int64_t i = 0;
  for (;;) {
    int64_t l = 2 * i + 1, r = l + 1, m = i;
    if (l < *n && h[l] > h[m]) m = l;
    if (r < *n && h[r] > h[m]) m = r;
    if (m == i) break;
    int32_t t = h[i];
    h[i] = h[m];
    h[m] = t;
    i = m;
  }
  return top;
}

int nopfs_ref_buffer_sim(const nopfs_ref_job* job, const int32_t* R, const int32_t* next,
                         const int64_t* sizes, int64_t d0, int8_t* hit, int64_t* hits) {
  return nopfs_ref_buffer_sim_rows(job, R, 0, job ? job->N : 0, next, sizes, d0, hit, hits);
}

int nopfs_ref_buffer_sim_rows(const nopfs_ref_job* job, const int32_t* R, int64_t i0, int64_t i1,
                              const int32_t* next, const int64_t* sizes, int64_t d0, int8_t* hit,
                              int64_t* hits) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if (i0 < 0 || i1 > job->N || i0 > i1) return REF_EINVAL;
  if (!sizes || !hits || d0 < 0) return REF_EINVAL;
  if (M_max > 0 && (!R || !next || !hit)) return REF_EINVAL;
  uint8_t* held = (uint8_t*)malloc((size_t)(M_max > 0 ? M_max : 1));
  int32_t* heap = (int32_t*)malloc((size_t)(M_max > 0 ? M_max : 1) * sizeof(int32_t));
  if (!held || !heap) { free(held); free(heap); return REF_ENOMEM; }
  for (int64_t i = i0; i < i1; ++i) {
    const int32_t* Ri = R + (i - i0) * M_max;
    const int32_t* Xi = next + (i - i0) * M_max;
    int8_t* Hi = hit + (i - i0) * M_max;
    int64_t Mi = job->E * epoch_len(job, i);
    memset(held, 0, (size_t)(M_max > 0 ? M_max : 1));
    int64_t nh = 0, used = 0, h_count = 0, h_bytes = 0;
    for (int64_t f = 0; f < Mi; ++f) {
      int64_t s = sizes[Ri[f]];
      if (held[f]) { /* the sample is in the buffer: a hit; its entry ends here */
        Hi[f] = 1;
        h_count++;
        h_bytes += s;
        held[f] = 0;
        used -= s;
      } else {
        Hi[f] = 0;
      }
      int32_t nx = Xi[f];
      if (nx >= 0 && s <= d0) { /* admit under the next use, then discard furthest */
        held[nx] = 1;
        heap_push(heap, &nh, nx);
        used += s;
        while (used > d0) {
          int32_t x = heap_pop(heap, &nh);
          if (!held[x]) continue; /* stale key */
          held[x] = 0;
          used -= sizes[Ri[x]];
        }
      }
    }
    for (int64_t f = Mi; f < M_max; ++f) Hi[f] = -1;
    hits[(i - i0) * 2] = h_count;
    hits[(i - i0) * 2 + 1] = h_bytes;
    nh = 0;
  }
  free(held);
  free(heap);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Sampled columns. The position of sample s in epoch e is, by definition   */
/* of the sorted order, the number of samples whose (key, id) is smaller.   */
/* Everything else for s follows from its positions in the E epochs.        */
/* ------------------------------------------------------------------------ */
int nopfs_ref_sample_columns(const nopfs_ref_job* job, const int32_t* samples,
                             int64_t S, int64_t* pos, int32_t* occ_worker,
                             int32_t* occ_f, int32_t* occ_next,
                             uint8_t* col_count, int32_t* col_first) {
  int64_t M_max;
  int rc = nopfs_ref_stream_shape(job, NULL, &M_max, NULL);
  if (rc) return rc;
  if (!samples || S < 0 || !pos || !occ_worker || !occ_f || !occ_next ||
      !col_count || !col_first)
    return REF_EINVAL;
  int64_t F = job->F, N = job->N, E = job->E, P = issued(job);
  for (int64_t s = 0; s < S; ++s)
    if (samples[s] < 0 || samples[s] >= F) return REF_EINVAL;
  uint32_t* keys = (uint32_t*)malloc((size_t)F * sizeof(uint32_t));
  if (!keys) return REF_ENOMEM;
  for (int32_t e = 0; e < E; ++e) {
    nopfs_ref_epoch_keys(job, e, keys);
    for (int64_t s = 0; s < S; ++s) {
      int64_t ks = samples[s];
      uint32_t key_s = keys[ks];
      int64_t smaller = 0;
      for (int64_t k = 0; k < F; ++k)
        smaller += (keys[k] < key_s) | ((keys[k] == key_s) & (k < ks));
      pos[e * S + s] = smaller;
    }
  }
  free(keys);
  for (int64_t i = 0; i < N; ++i)
    for (int64_t s = 0; s < S; ++s) {
      col_count[i * S + s] = 0;
      col_first[i * S + s] = -1;
    }
  for (int32_t e = 0; e < E; ++e)
    for (int64_t s = 0; s < S; ++s) {
      int64_t p = pos[e * S + s];
      if (p >= P) { occ_worker[e * S + s] = -1; occ_f[e * S + s] = -1; continue; }
      int64_t i = p % N, j = p / N;
      int64_t f = (int64_t)e * epoch_len(job, i) + j;
      occ_worker[e * S + s] = (int32_t)i;
      occ_f[e * S + s] = (int32_t)f;
      if (col_count[i * S + s] == 0) col_first[i * S + s] = (int32_t)f;
      col_count[i * S + s] += 1;
    }
  for (int32_t e = 0; e < E; ++e)
    for (int64_t s = 0; s < S; ++s) {
      int32_t nx = -1;
      if (occ_worker[e * S + s] >= 0)
        for (int32_t e2 = e + 1; e2 < E; ++e2)
          if (occ_worker[e2 * S + s] == occ_worker[e * S + s]) {
            nx = occ_f[e2 * S + s];
            break;
          }
      occ_next[e * S + s] = nx;
    }
  return 0;
}
