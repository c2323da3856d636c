/*
 * nopfs.h -- C ABI of the MI355X (gfx950) clairvoyant access planner.
 *
 * Given the shuffle seed of a data-parallel training job, the library expands
 * it into every worker's exact sample-access stream for all epochs, and from
 * those streams derives per-(worker, sample) access frequencies and first
 * reads, next-reuse positions, and a frequency-ordered placement of samples
 * into capacity-limited storage tiers. This is the clairvoyant planning of
 * NoPFS (Dryden et al., SC'21): section 2 (reproducible shuffles), section 3
 * (access patterns, Belady's next use, the access-frequency distribution),
 * section 4 (batches, worker batches and the stream R) and section 5.1 (the
 * placement rule).
 *
 * CONVENTIONS (all entry points)
 *  - Array arguments are DEVICE pointers owned by the caller, except where
 *    marked "host". Outputs are preallocated by the caller; the library writes
 *    every element of every output (no zeroing needed) and keeps no pointer
 *    after the enqueued work completes.
 *  - `hip_stream` is a hipStream_t (NULL = the null stream). GPU calls
 *    enqueue work on it and return; the caller keeps the buffers alive until
 *    the stream has completed. Internal scratch comes from one block of
 *    device memory per (device, stream), reused in stream order by every call
 *    on that stream: a call that needs more than the block allocates the rest
 *    (hipMalloc) and replaces the block by one of its peak size at its end,
 *    so later calls of that size allocate nothing. The block is kept until
 *    nopfs_scratch_release (or the end of the process): at most the largest
 *    call's scratch per stream. Calls on one stream from several host
 *    threads are enqueued one at a time.
 *  - Host waits: a GPU call returns without waiting for the device, except
 *    a call that outgrows its stream's block (the first call of a larger job
 *    on a stream, or the first after nopfs_scratch_release), which
 *    synchronises the stream after enqueueing its work, before it frees and
 *    replaces the block. nopfs_scratch_release and nopfs_profile_query wait
 *    too; nothing else does.
 *  - Return 0 on success, a negative NOPFS_E* code otherwise. Argument errors
 *    are detected on the host before anything is enqueued. No C++ exception
 *    crosses this boundary. nopfs_last_error() gives a thread-local detail.
 *  - An array with no elements (R and next when M_max == 0) may be NULL.
 *  - Layouts are row-major; [N][F] tables are indexed i*F + k with 64-bit
 *    arithmetic (N*F may exceed 2^31).
 *  - Entry points keep no state but the scratch blocks and are reentrant:
 *    several jobs (say a training and a validation job) can be planned
 *    concurrently on different streams.
 *  - Every result is exact integer work and deterministic: the output is a
 *    pure function of the inputs.
 *
 * READINGS of points the paper leaves open (binding for every entry point):
 *  - Shuffle: epoch e orders samples by a 32-bit key, word (k mod 4) of
 *    Philox-4x32-10 (Salmon et al., SC'11) at counter (k div 4, e, 0, 0) with
 *    key (seed low 32 bits, seed high 32 bits); equal keys go by smaller id.
 *  - Ids, epochs and stream positions are 0-based.
 *  - B is the per-worker batch; the global batch is N*B. Worker i reads the
 *    global positions p of each epoch with p mod N == i, in order.
 *  - drop_last=1: T = F div (N*B) iterations, every worker reads L = T*B
 *    samples per epoch, positions p >= T*N*B are not read. drop_last=0:
 *    T = ceil(F / (N*B)), worker i reads L_i = ceil((F - i) / N) samples per
 *    epoch (0 when i >= F); rows shorter than M_max are padded with -1.
 *  - Stream positions f index a worker's own stream R_i: f = e*L_i + j for
 *    its j-th read in epoch e. "Never" is -1.
 */
#ifndef NOPFS_H
#define NOPFS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define NOPFS_OK        0
#define NOPFS_EINVAL  (-1) /* null pointer, F<1, E<1, N<1, B<1, drop_last not
                              0/1, J<1, a negative capacity                  */
#define NOPFS_ERANGE  (-2) /* F >= 2^31, E > 255, M_max >= 2^31, J > 127     */
#define NOPFS_ENOMEM  (-3) /* internal scratch could not be allocated        */
#define NOPFS_EDEVICE (-4) /* HIP runtime or launch error (see last_error)   */

/* A training job as the paper states it (section 4 and the Python Job of
 * section 5.2.1): F samples, E epochs, N data-parallel workers, per-worker
 * mini-batch B, whether the last partial iteration is dropped, and the seed. */
typedef struct nopfs_job {
  int64_t  F;          /* samples, 1 <= F < 2^31                            */
  int32_t  E;          /* epochs, 1 <= E <= 255 (counts are uint8)          */
  int32_t  N;          /* workers, >= 1                                     */
  int32_t  B;          /* per-worker batch, >= 1                            */
  int32_t  drop_last;  /* 0 or 1                                            */
  uint64_t seed;       /* shuffle seed                                      */
} nopfs_job;

/* Host only, no GPU. Iterations per epoch *T, the longest stream *M_max
 * (= E * max_i L_i), and if M_per_worker != NULL (host, [N]) each worker's
 * stream length M_i = E * L_i. Section 4: T is floor (or ceil when the last
 * small iteration is kept) of F over the global batch. Any output pointer may
 * be NULL. Errors: EINVAL, ERANGE. */
int nopfs_stream_shape(const nopfs_job* job, int64_t* T, int64_t* M_max,
                       int64_t* M_per_worker);

/* Access streams (section 2: the seed reproduces every epoch's shuffle;
 * section 4: worker batches partition each global batch and R is the
 * concatenation of a worker's batches).
 *   R: int32 [N][M_max], R[i][f] = sample read by worker i at position f,
 *      -1 in padding (drop_last=0 only).
 * Errors: EINVAL, ERANGE, ENOMEM, EDEVICE. */
int nopfs_access_streams(const nopfs_job* job, int32_t* R, void* hip_stream);

/* The access streams of epochs [e_begin, e_end) only, as a job resumed at
 * epoch e_begin would regenerate them (every epoch's shuffle depends only on
 * the seed and the epoch). R is laid out as the streams of a job with the
 * same F, N, B, drop_last and e_end - e_begin epochs: int32
 * [N][(e_end - e_begin) * max_i L_i], row i = columns [e_begin * L_i,
 * e_end * L_i) of nopfs_access_streams' row i, then -1 padding. That job
 * (E = e_end - e_begin) is the shape to pass to nopfs_access_stats,
 * nopfs_reuse_next and nopfs_tier_plan for the remaining epochs. An empty
 * range writes nothing. Errors: EINVAL (also unless 0 <= e_begin <= e_end
 * <= E), ERANGE, ENOMEM, EDEVICE. */
int nopfs_access_streams_range(const nopfs_job* job, int32_t e_begin, int32_t e_end,
                               int32_t* R, void* hip_stream);

/* Access frequencies and first reads (section 3.1: worker i's access
 * frequency X of sample k over all E epochs; section 5.1 names it r_k).
 *   R:     int32 [N][M_max], as written by nopfs_access_streams for this job
 *          (precondition; other contents give unspecified but in-bounds
 *          results as long as every entry is in [0, F) or padding).
 *   count: uint8 [N][F], number of reads of k in R_i.
 *   first: int32 [N][F], smallest f with R_i[f] == k, or -1.
 * Errors: EINVAL, ERANGE, ENOMEM, EDEVICE. */
int nopfs_access_stats(const nopfs_job* job, const int32_t* R, uint8_t* count,
                       int32_t* first, void* hip_stream);

/* Next reuse (section 3: Belady's replacement evicts the sample whose next
 * use is furthest; the four rules of Cao et al. need it).
 *   R:    int32 [N][M_max], as for nopfs_access_stats.
 *   next: int32 [N][M_max], smallest f' > f with R_i[f'] == R_i[f], or -1
 *         (also -1 in padding). The reuse distance is next - f; every reuse
 *         lies in a later epoch.
 * Errors: EINVAL, ERANGE, ENOMEM, EDEVICE. */
int nopfs_reuse_next(const nopfs_job* job, const int32_t* R, int32_t* next,
                     void* hip_stream);

/* Tier placement (section 5.1: a worker caches the samples with the largest
 * access frequency in its fastest storage class, then the next, until the
 * dataset is cached or its storage is full).
 * Per worker i, samples are ranked by (count desc, first asc with -1 last,
 * id asc); tier 0 takes samples along the ranking while they fit in caps[0],
 * the first sample that does not fit starts tier 1, and so on; what remains
 * after tier J-1 is uncached. Samples a worker never reads are ranked last
 * and are still placed (they can serve other workers). Tiers are independent
 * per worker. The staging buffer (storage class 0 of section 4) is not a
 * placement tier: pass only cache classes, fastest first.
 *   count, first: as written by nopfs_access_stats for this job.
 *   sizes: int64 [F] sample sizes in bytes, each >= 1 (precondition; other
 *          values give unspecified but in-bounds results).
 *   caps:  HOST int64 [J] per-worker tier capacities in bytes, >= 0.
 *   tier:  int8 [N][F], tier index of k on worker i, or -1 (uncached).
 *   used:  int64 [N][J], bytes placed in each tier.
 * Errors: EINVAL, ERANGE (J > 127), ENOMEM, EDEVICE. */
int nopfs_tier_plan(const nopfs_job* job, const uint8_t* count,
                    const int32_t* first, const int64_t* sizes,
                    const int64_t* caps, int32_t J, int8_t* tier,
                    int64_t* used, void* hip_stream);

/* The whole planning path in one call: the shuffle seed expanded into every
 * worker's streams (sections 2 and 4), access frequencies, first reads and
 * next uses (section 3), and the tier placement (section 5.1), i.e. the
 * preparation a worker does once before training starts.
 * Outputs are exactly those of nopfs_access_streams, nopfs_access_stats,
 * nopfs_reuse_next and nopfs_tier_plan called in that order with the same
 * arguments (same layouts, same readings); every pointer is as documented
 * there. R and next may be NULL when M_max == 0. Fewer passes over memory:
 * the counting and next-use passes share their partition of R where they
 * can, and the tier plan reads a compact list of the read cells produced by
 * the counting pass (scratch of about 8 bytes per read, returned to the
 * stream's scratch block when the call returns).
 * Errors: EINVAL, ERANGE, ENOMEM, EDEVICE, all detected before any launch
 * except ENOMEM/EDEVICE from a later stage (outputs are then unspecified). */
int nopfs_plan_job(const nopfs_job* job, const int64_t* sizes, const int64_t* caps,
                   int32_t J, int32_t* R, uint8_t* count, int32_t* first, int32_t* next,
                   int8_t* tier, int64_t* used, void* hip_stream);

/* nopfs_plan_job for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, outputs and errors, but no call to hipMalloc, hipFree
 * or any allocating routine, and no host wait. Its scratch is one fixed
 * array of 64 MiB (67,108,864 bytes) per device, part of the library's code
 * object, held by every device the library runs on until the process ends;
 * its address on a device is looked up once, on the first call there. A job
 * whose scratch exceeds it is rejected with ERANGE before anything is
 * enqueued (the peak is the shuffle's exchange, about 16 bytes per sample
 * and epoch: F = 200,000 samples over 10 epochs fits, F = 1,000,000 over 10
 * epochs needs 164 MB and is rejected). Every call on a
 * device shares that device's array, and each call initialises what it
 * reads there, so consecutive calls need nothing from each other; calls
 * that overlap in time on one device (other streams, other host threads'
 * streams) race on the array and must be ordered by the caller (one stream,
 * or events). Calls from several host threads are enqueued one at a time. */
int nopfs_plan_job_noalloc(const nopfs_job* job, const int64_t* sizes, const int64_t* caps,
                           int32_t J, int32_t* R, uint8_t* count, int32_t* first,
                           int32_t* next, int8_t* tier, int64_t* used, void* hip_stream);

/* Prefetch order of the cache tiers (section 5.1: samples are always fetched
 * in their order of access, following the first of the prefetching rules of
 * section 3; a worker fills each storage class with the samples placed
 * there). For worker i, tier j's queue lists the samples k with
 * tier[i][k] == j that the worker reads, by increasing first read (the
 * smallest f with R_i[f] == k); the queues are concatenated fastest tier
 * first and the row is padded with -1. Samples placed in tier j that the
 * worker never reads are not listed (they can be fetched after the queue, in
 * any order). First reads are taken from R itself, so the dense first-read
 * table is not an argument.
 *   R:     int32 [N][M_max], as for nopfs_access_stats.
 *   tier:  int8 [N][F], a placement (as written by nopfs_tier_plan); entries
 *          outside [0, J) are not queued.
 *   J:     number of cache tiers, 1 <= J <= 127.
 *   order: int32 [N][M_max], output: queue of tier 0, then tier 1, ..., then -1.
 *   qlen:  int64 [N][J], output: queue lengths (tier j's queue starts at
 *          the sum of qlen[i][0..j-1]).
 * Scratch: about 5 bytes per stream position. Errors: EINVAL (also J < 1),
 * ERANGE (J > 127), ENOMEM, EDEVICE. */
int nopfs_prefetch_order(const nopfs_job* job, const int32_t* R, const int8_t* tier, int32_t J,
                         int32_t* order, int64_t* qlen, void* hip_stream);

/* Staging-buffer schedule (section 5.1: samples enter the staging buffer in
 * access order and leave it as soon as they are read; section 5.2: the
 * buffer is filled circularly). While worker i has read the positions
 * before f, its buffer of d0 bytes holds the samples at positions f, f+1, ...
 * of R_i that fit; the sample at position h can be fetched once the worker
 * has read position fill[i][h] - 1:
 *   fill[i][h] = smallest f <= h with sizes[R_i[f]] + ... + sizes[R_i[h]] <= d0,
 *                or h when sizes[R_i[h]] alone exceeds d0;
 * -1 in padding. fill never decreases along a row.
 *   R:     int32 [N][M_max], as for nopfs_access_stats.
 *   sizes: int64 [F] sample sizes in bytes, each >= 1 (precondition; other
 *          values give unspecified but in-bounds results).
 *   d0:    staging buffer capacity in bytes, >= 0.
 *   fill:  int32 [N][M_max], output.
 * Scratch: about 16 bytes per stream position, plus 4 bytes per (span of
 * 16384 positions of a row, window of 32768 samples). Errors: EINVAL (also d0 < 0),
 * ERANGE, ENOMEM, EDEVICE. */
int nopfs_staging_schedule(const nopfs_job* job, const int32_t* R, const int64_t* sizes,
                           int64_t d0, int32_t* fill, void* hip_stream);

/* Parameters of the performance model (section 4), in bytes, bytes per
 * second and seconds (the paper's MB/s are 10^6 bytes per second). Cache
 * tier j (j = 0..J-1, as in nopfs_tier_plan) is the model's storage class
 * j + 1; class 0 is the staging buffer. Host memory. */
typedef struct nopfs_model {
  double c;          /* compute throughput for training                        */
  double beta;       /* preprocessing rate                                     */
  double b_c;        /* inter-worker network bandwidth                         */
  double pfs_t;      /* aggregate random read throughput of the PFS, t(gamma)  */
  double pfs_gamma;  /* the number of concurrent PFS readers gamma            */
  double w0;         /* staging-buffer write throughput with p0 threads        */
  double p0;         /* prefetch threads of the staging buffer                 */
  int32_t J;         /* cache tiers, 1 <= J <= 32                              */
  int32_t reserved;  /* ignored                                                */
  double r[32];      /* tier j: aggregate random read throughput, p[j] threads */
  double p[32];      /* tier j: prefetch threads                               */
} nopfs_model;

/* Fetch sources and consumption times under the performance model
 * (section 4), with the placement static: sample k is in tier j of worker i
 * exactly when tier[i][k] == j. Worker i fetches its read f of sample k
 * (s bytes) from the fastest of the PFS (t(gamma)/gamma), another worker's
 * tier j (min(b_c, r_j/p_j)) and its own tier j (r_j/p_j), preprocesses and
 * writes it to the staging buffer (max(s/beta, s/(w0/p0))), and consumes it
 * at t(f) = max(avail(f), t(f-1) + s(f-1)/c), avail(f) = (sum of the read
 * times of reads 0..f) / p0; t(0) = avail(0).
 *   R:     int32 [N][M_max], as for nopfs_access_stats.
 *   tier:  int8 [N][F], the placement of all workers (entries outside
 *          [0, J) hold nothing).
 *   sizes: int64 [F] sample sizes in bytes, 1 <= size < 2^56 (precondition).
 *   model: HOST, the parameters; all positive and finite.
 *   src:   int16 [N][M_max], output: 0 = the PFS, 128 + j = another worker's
 *          tier j, 256 + j = the worker's own tier j; on equal throughput the
 *          own tier, then a remote one (lower tier first), then the PFS; -1 in
 *          padding. Exact.
 *   t:     double [N][M_max], output: consumption times in seconds, -1 in
 *          padding. Evaluated as prefix sums and a prefix maximum of the
 *          unrolled recurrence, so it differs from the sequential recurrence
 *          only by floating-point summation order (at most a few units of
 *          (f + 2) * 2^-53 * t(f) in practice).
 * Scratch: about 20 bytes per stream position. Errors: EINVAL (also an invalid
 * model), ERANGE (J > 32), ENOMEM, EDEVICE. */
int nopfs_fetch_model(const nopfs_job* job, const int32_t* R, const int8_t* tier,
                      const int64_t* sizes, const nopfs_model* model, int16_t* src,
                      double* t, void* hip_stream);

/* Clairvoyant buffer of d0 bytes per worker (section 3: Belady's
 * replacement, discard the sample whose next use is furthest in the future,
 * and never one used before the sample being brought in). The buffer holds
 * samples keyed by their next use; read f of worker i hits when its sample
 * is held. After a read with a next use the sample is (re)admitted under
 * it, then, while the held bytes exceed d0, the entry used furthest in the
 * future is discarded (possibly the admitted one). A sample with no next
 * use, or larger than d0, is not admitted. With all sizes equal this is
 * Belady's optimal replacement with bypass.
 *   R, next: int32 [N][M_max], as written by nopfs_access_streams and
 *            nopfs_reuse_next for this job (precondition; other contents give
 *            unspecified but in-bounds results).
 *   sizes:   int64 [F] sample sizes in bytes, >= 1.
 *   d0:      buffer capacity in bytes, >= 0.
 *   hit:     int8 [N][M_max], output: 1 hit, 0 miss, -1 padding.
 *   hits:    int64 [N][2], output: hits and hit bytes per worker.
 * The replay is sequential per worker (one wave each). M_max < 2^24.
 * Scratch: one bit per stream position. Errors: EINVAL (also d0 < 0),
 * ERANGE (M_max >= 2^24), ENOMEM, EDEVICE. */
int nopfs_buffer_sim(const nopfs_job* job, const int32_t* R, const int32_t* next,
                     const int64_t* sizes, int64_t d0, int8_t* hit, int64_t* hits,
                     void* hip_stream);

/* Data-loading policies of section 6, simulated on the model of section 4
 * (nopfs_policy_sim). */
#define NOPFS_POLICY_PERFECT 0 /* no stalls: only compute (a lower bound)        */
#define NOPFS_POLICY_NAIVE 1   /* one PFS read at a time, after each compute      */
#define NOPFS_POLICY_STAGING 2 /* a staging buffer filled in stream order from    */
                               /* the PFS, each sample dropped once consumed      */
#define NOPFS_POLICY_NOPFS 3   /* the same buffer, each read from the fastest     */
                               /* source of the placement (nopfs_fetch_model)     */

/* Simulated training time of every worker under one of the policies of
 * section 6, on the performance model of section 4. For read f of a worker,
 * with s its size: u(f) = s / c (compute), read(f) = fetch(f) + write(f),
 * write(f) = max(s / beta, s / (w0 / p0)), fetch(f) = s over its source's
 * throughput (PFS t(gamma) / gamma; another worker's tier j
 * min(b_c, r_j / p_j); own tier j r_j / p_j).
 *   PERFECT: t(0) = 0, t(f) = t(f-1) + u(f-1).
 *   NAIVE:   t(0) = read(0), t(f) = t(f-1) + u(f-1) + read(f), every read
 *            from the PFS.
 *   STAGING, NOPFS: p0 threads stage reads in stream order (from the PFS,
 *            or from the source src names), and read f can start only once
 *            the reads before fill(f) are consumed (fill: the schedule of
 *            nopfs_staging_schedule for the buffer's d0). With Q(f) the
 *            thread-time spent staging reads 0..f:
 *              Q(f) = max(Q(f-1), p0 t(fill(f) - 1)) + read(f), t(-1) = 0,
 *              t(0) = Q(0) / p0, t(f) = max(Q(f) / p0, t(f-1) + u(f-1)).
 *            With fill all 0 (an unlimited buffer), NOPFS is
 *            nopfs_fetch_model's t (avail = the summed read times / p0).
 * The evaluation is sequential per worker, in this order, with IEEE double
 * operations: results do not depend on the launch.
 *   R:      int32 [N][M_max], nopfs_access_streams' output for this job.
 *   sizes:  int64 [F] sample sizes in bytes.
 *   src:    int16 [N][M_max], nopfs_fetch_model's sources (NOPFS only; may
 *           be NULL otherwise). Codes other than 0, 128 + j, 256 + j with
 *           j < J read from the PFS.
 *   fill:   int32 [N][M_max], nopfs_staging_schedule's output (STAGING and
 *           NOPFS; may be NULL otherwise).
 *   t:      double [N][M_max], output: when each read is consumed, seconds;
 *           -1 in padding.
 *   finish: double [N], output: when the worker's last compute ends (0 for a
 *           worker with no reads).
 *   io:     double [N][1 + 2J], output: fetch time summed by source class,
 *           0 the PFS, 1 + j another worker's tier j, 1 + J + j the own tier
 *           j (all 0 for PERFECT).
 * One wave per worker replays its stream. No scratch. Errors: EINVAL (also
 * a policy outside 0..3, or a missing src or fill the policy needs), ERANGE
 * (J > 32), EDEVICE. */
int nopfs_policy_sim(const nopfs_job* job, const int32_t* R, const int64_t* sizes,
                     const int16_t* src, const int32_t* fill, const nopfs_model* model,
                     int32_t policy, double* t, double* finish, double* io, void* hip_stream);

/* Static description of a status code. Never NULL. */
const char* nopfs_strerror(int code);

/* Thread-local detail of the last failing call on this thread ("" if none). */
const char* nopfs_last_error(void);

/* ---- Measurement aids ------------------------------------------------- */

/* Per-kernel timing with HIP events recorded on the caller's stream around
 * every kernel the library launches. enable=1 starts (and clears) the
 * record, enable=0 stops. Timing is off by default. */
int nopfs_profile_enable(int enable);

/* Synchronises on the recorded events and reports, for the idx-th kernel
 * name seen since profiling was enabled, its name (static string), number of
 * launches and total milliseconds. Returns NOPFS_EINVAL when idx is past the
 * end. */
int nopfs_profile_query(int idx, const char** name, int64_t* launches,
                        double* total_ms);

/* A plain device-to-device copy of `bytes` bytes (multiple of 16, 16-byte
 * aligned pointers) with a kernel of known traffic, used to calibrate HBM
 * byte counters. */
int nopfs_calibration_copy(const void* src, void* dst, int64_t bytes,
                           void* hip_stream);

/* Returns the scratch block of (current device, hip_stream) to the device:
 * waits for the work enqueued on the stream (hipStreamSynchronize), then
 * frees the block (hipFree). The next call on that stream allocates a new
 * one. A call being enqueued on the stream from another host thread
 * finishes first. Nothing to release is not an error. Errors: EDEVICE. */
int nopfs_scratch_release(void* hip_stream);

/* ---- Test hooks ------------------------------------------------------- */

/* Overrides internal capacities so tests can drive the slow paths on small
 * inputs (0 restores the default):
 *   which=1  largest bucket the stream sort keeps in LDS (elements)
 *   which=2  candidate records per worker in the tier plan's fast path, and
 *            reads per window in the next-use fast path
 *   which=3  fail the next internal scratch allocation (value 1)
 *   which=4  longest range of buffer starts the staging schedule keeps in
 *            LDS per chunk (wider ranges take the global-memory search)
 *   which=5  doublings (at most 4) of the sample windows of the staging
 *            schedule and the fetch model, so each window tile covers its
 *            window in several LDS passes, as for F above 2^27
 * The overrides are per host thread: they apply only to calls made from the
 * thread that set them. Meant for tests only. */
int nopfs_debug_set(int which, int64_t value);

#ifdef __cplusplus
}
#endif
#endif /* NOPFS_H */
