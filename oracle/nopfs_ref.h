/*
 * nopfs_ref.h -- the CPU oracle for clairvoyant access planning.
 *
 * TEST INFRASTRUCTURE. This library is a plain, slow, single-threaded
 * reference implementation used only by the test suite, the smoke check and
 * the benchmark's CPU-baseline leg. The GPU library never includes, links or
 * calls it, and it includes nothing from the GPU library: the job struct below
 * is declared here on its own, with the same field order and widths as the
 * GPU library's, so that one Python-side description can fill both.
 *
 * All array arguments are HOST pointers. Every function returns 0 on success
 * and a negative code on invalid arguments (-1 invalid, -2 out of range,
 * -3 out of memory).
 */
#ifndef NOPFS_REF_H
#define NOPFS_REF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nopfs_ref_job {
  int64_t  F;          /* samples in the dataset (paper notation F)          */
  int32_t  E;          /* epochs                                             */
  int32_t  N;          /* data-parallel workers                              */
  int32_t  B;          /* per-worker mini-batch size                         */
  int32_t  drop_last;  /* 1: drop the last, partial iteration of each epoch  */
  uint64_t seed;       /* shuffle seed (Philox key)                          */
} nopfs_ref_job;

/* Philox-4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11). */
void nopfs_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                             uint32_t out[4]);

/* Iterations per epoch T, longest stream M_max, per-worker stream lengths. */
int nopfs_ref_stream_shape(const nopfs_ref_job* job, int64_t* T, int64_t* M_max,
                           int64_t* M_per_worker /* [N] or NULL */);

/* Shuffle key of every sample in epoch e: keys[k], k in [0, F). */
int nopfs_ref_epoch_keys(const nopfs_ref_job* job, int32_t e, uint32_t* keys);

/* Epoch permutation: perm[p] = sample at global position p of epoch e. */
int nopfs_ref_epoch_perm(const nopfs_ref_job* job, int32_t e, int32_t* perm);

/* Shard the given epoch permutations perms[E][F] into R[N][M_max]. */
int nopfs_ref_streams_from_perms(const nopfs_ref_job* job, const int32_t* perms,
                                 int32_t* R);

/* Rows [i0, i1) of the streams sharded from perms[E][F]; R points at row
 * i0 and holds i1 - i0 rows of M_max entries. */
int nopfs_ref_streams_rows(const nopfs_ref_job* job, const int32_t* perms, int64_t i0,
                           int64_t i1, int32_t* R);

/* Every worker's access stream R[N][M_max] (rows padded with -1). */
int nopfs_ref_access_streams(const nopfs_ref_job* job, int32_t* R);

/* count[N][F] and first[N][F] from R. */
int nopfs_ref_access_stats(const nopfs_ref_job* job, const int32_t* R,
                           uint8_t* count, int32_t* first);

/* The same for workers [i0, i1) only: R, count and first point at row i0. */
int nopfs_ref_access_stats_rows(const nopfs_ref_job* job, const int32_t* R,
                                int64_t i0, int64_t i1, uint8_t* count,
                                int32_t* first);

/* next[N][M_max] from R. */
int nopfs_ref_reuse_next(const nopfs_ref_job* job, const int32_t* R,
                         int32_t* next);

/* The same for workers [i0, i1) only: R and next point at row i0. */
int nopfs_ref_reuse_next_rows(const nopfs_ref_job* job, const int32_t* R,
                              int64_t i0, int64_t i1, int32_t* next);

/* tier[N][F] and used[N][J] from count, first, sizes[F] and caps[J]. Only
 * job->F, job->E and job->N (the number of rows) are read. */
int nopfs_ref_tier_plan(const nopfs_ref_job* job, const uint8_t* count,
                        const int32_t* first, const int64_t* sizes,
                        const int64_t* caps, int32_t J, int8_t* tier,
                        int64_t* used);

/* Prefetch order per cache tier: for worker i and tier j in [0, J), the
 * samples k with tier[i][k] == j that worker i reads, each once, in order of
 * first read. order[N][M_max]: tier 0's queue, then tier 1's, ..., then -1;
 * qlen[N][J]: the queue lengths. */
int nopfs_ref_prefetch_order(const nopfs_ref_job* job, const int32_t* R,
                             const int32_t* first, const int8_t* tier, int32_t J,
                             int32_t* order, int64_t* qlen);

/* Staging-buffer schedule for a buffer of d0 bytes: fill[i][h] is the
 * smallest f <= h such that the samples at stream positions f..h of worker i
 * fit together (sum of sizes <= d0), or h when the sample at h alone is
 * larger than d0; -1 in padding. */
int nopfs_ref_staging_schedule(const nopfs_ref_job* job, const int32_t* R,
                               const int64_t* sizes, int64_t d0, int32_t* fill);

/* Parameters of the performance model (section 4), in bytes, bytes per
 * second and seconds. Cache tier j (j = 0..J-1) is the model's storage class
 * j + 1; class 0 is the staging buffer. */
typedef struct nopfs_ref_model {
  double c;          /* compute throughput for training                      */
  double beta;       /* preprocessing rate                                   */
  double b_c;        /* inter-worker network bandwidth                       */
  double pfs_t;      /* aggregate random read throughput of the PFS, t(gamma) */
  double pfs_gamma;  /* the number of PFS readers gamma it is measured at     */
  double w0;         /* staging-buffer write throughput with p0 threads      */
  double p0;         /* prefetch threads of the staging buffer               */
  int32_t J;         /* cache tiers, 1..32                                   */
  int32_t pad_;
  double r[32];      /* tier j: aggregate random read throughput, p[j] threads */
  double p[32];      /* tier j: prefetch threads                             */
} nopfs_ref_model;

/* Fetch source and consumption time of every read (section 4) for workers
 * [i0, i1): R points at row i0 of the streams, tier is the placement of all
 * N workers ([N][F]), src and t point at row i0 of their [N][M_max] tables.
 * src: 0 = the PFS, 128 + j = another worker's tier j, 256 + j = the
 * worker's own tier j (the fastest applicable source; on equal throughput
 * own before remote before PFS, lower tier first); t: the time the worker
 * consumes the read, in seconds. Padding: src -1, t -1. */
int nopfs_ref_fetch_model_rows(const nopfs_ref_job* job, const int32_t* R,
                               const int8_t* tier, const int64_t* sizes,
                               const nopfs_ref_model* m, int64_t i0, int64_t i1,
                               int16_t* src, double* t);

/* Policy simulation (section 6) for workers [i0, i1): policy 0 Perfect (no
 * stalls), 1 Naive (one PFS read at a time after each compute), 2
 * StagingBuffer (p0 threads stage reads in stream order from the PFS into a
 * buffer whose schedule is fill, from nopfs_ref_staging_schedule), 3 NoPFS
 * (the same, each read from the source in src, from
 * nopfs_ref_fetch_model_rows; other codes read from the PFS). R, src, fill
 * and t point at row i0 of their [N][M_max] tables (src only for policy 3,
 * fill for 2 and 3). Outputs: t, when each read is consumed (-1 padding);
 * finish[i1 - i0], when the last read's compute ends; io[i1 - i0][1 + 2J],
 * fetch time summed by source class (0 the PFS, 1 + j another worker's tier
 * j, 1 + J + j the own tier j). */
int nopfs_ref_policy_sim_rows(const nopfs_ref_job* job, const int32_t* R, const int64_t* sizes,
                              const int16_t* src, const int32_t* fill, const nopfs_ref_model* m,
                              int32_t policy, int64_t i0, int64_t i1, double* t, double* finish,
                              double* io);

/* Clairvoyant buffer of d0 bytes (section 3: Belady's replacement, the
 * optimal-replacement and do-no-harm rules), per worker, from R, next and
 * the sizes. The buffer holds samples keyed by their next use; an access is
 * a hit when its sample is held. After an access with a next use the sample
 * is (re)admitted under that key, then, while the held bytes exceed d0, the
 * entry whose next use is furthest is discarded (possibly the admitted one:
 * nothing used before it is ever discarded for it). A sample with no next
 * use, or larger than d0, is not admitted.
 *   hit[N][M_max]: 1 hit, 0 miss, -1 padding; hits[N][2]: hit count and
 *   hit bytes per worker. */
int nopfs_ref_buffer_sim(const nopfs_ref_job* job, const int32_t* R, const int32_t* next,
                         const int64_t* sizes, int64_t d0, int8_t* hit, int64_t* hits);
/* The same for workers [i0, i1) only: R, next and hit hold those rows,
 * hits holds their [i1 - i0][2] totals. */
int nopfs_ref_buffer_sim_rows(const nopfs_ref_job* job, const int32_t* R, int64_t i0, int64_t i1,
                              const int32_t* next, const int64_t* sizes, int64_t d0, int8_t* hit,
                              int64_t* hits);

/* Per-sample columns for S chosen samples, computed one sample at a time
 * from the definition of the shuffle (for checks at sizes where the full
 * oracle is too slow):
 *   pos[e][s]       global position of samples[s] in epoch e's order
 *   occ_worker[e][s] worker that reads it in epoch e (-1: dropped tail)
 *   occ_f[e][s]     stream position of that read (-1: dropped)
 *   occ_next[e][s]  next read of the same sample by the same worker (-1: none)
 *   col_count[i][s], col_first[i][s]  count / first column for worker i     */
int nopfs_ref_sample_columns(const nopfs_ref_job* job, const int32_t* samples,
                             int64_t S, int64_t* pos, int32_t* occ_worker,
                             int32_t* occ_f, int32_t* occ_next,
                             uint8_t* col_count, int32_t* col_first);

#ifdef __cplusplus
}
#endif
#endif /* NOPFS_REF_H */
