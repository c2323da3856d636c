// nopfs_access_streams: every worker's access stream for every epoch.
//
// Section 2 of the paper: an epoch is a random shuffle of all sample ids and
// the seed reproduces it. Section 4: each global batch is partitioned among
// the N workers and a worker's stream R is the concatenation of its batches.
//
// Epoch e orders the samples by (key_e(k), k), key_e(k) a Philox-4x32-10
// word. The order is a bucket sort with one level of buckets: bucket
// b = key >> (32 - m) (2^m buckets per epoch, a few thousand keys each), all
// epochs of a batch at once. The ids of an epoch are cut into chunks of C
// consecutive ids; inside a bucket the keys of each chunk form one run, runs
// in chunk order. Every element travels as ONE 32-bit word:
//     word = kb << cbits | (id - chunk * C)
// where kb is the top (32 - cbits) bits of the key below the bucket bits.
// The chunk of a word follows from its position in the bucket (the run
// bounds are known from the counting pass), so the id is exact; kb orders
// the bucket except where two words share kb, which is resolved by the full
// keys (regenerated from the ids) and then the ids.
//   1. stream_count   -- Philox keys in registers; per (epoch, chunk)
//                        histogram of the buckets.
//   2. stream_offsets -- per (epoch, bucket) running sum over chunks: the
//                        run starts, in chunk-major and bucket-major copies.
//   3. stream_scan    -- bucket starts per epoch.
//   4. stream_scatter -- keys regenerated; each chunk counting-sorted by
//                        bucket in LDS (rounds of 24,576 ids, one workgroup
//                        per CU) and written as words, one contiguous run per
//                        bucket and round.
//   5. stream_sort    -- one workgroup per bucket: words decoded (chunk from
//                        the run table), counting sort in LDS by the top 13
//                        bits of kb, the digit groups of two or more (a fifth
//                        of them) insertion-sorted, and the sorted positions p
//                        sharded straight into R: R[p mod N][e*L_i + p div N],
//                        through an LDS transpose so each worker row gets a
//                        run of consecutive positions.
// At most 4,096 buckets are handled per pass ("window" of buckets); larger
// jobs (F above ~31M) make several passes over the keys, each keeping the
// keys of its window. Buckets larger than the LDS capacity (not expected for
// uniform keys, but possible in principle) are sorted in place in global
// memory by a bitonic network inside the same workgroup.
#include <limits.h>

#include "common.hpp"
#include "philox.hpp"

namespace nopfs {
namespace {

constexpr int kThreads = 1024;
constexpr int kRoundBlocks = 6;                            // Philox blocks per thread and round
constexpr int kRound = kThreads * 4 * kRoundBlocks;        // 24,576 ids per scatter round
#ifndef NOPFS_CHUNK_ROUNDS
#define NOPFS_CHUNK_ROUNDS 1
#endif
constexpr int kChunkRounds = NOPFS_CHUNK_ROUNDS;           // smallest chunk, in rounds
constexpr uint32_t kMaxChunks = 2048;                      // chunks per epoch (sort's run table)
constexpr uint32_t kMaxWin = 4096;                         // buckets per pass
constexpr int64_t kMeanBucket = 7700;                      // largest mean bucket size
constexpr int kBlkShift = 3;                               // run-table lookup granularity

#ifndef NOPFS_SORT_CAP
#define NOPFS_SORT_CAP 8192
#endif
constexpr int kSortCap = NOPFS_SORT_CAP;  // largest bucket sorted in LDS
constexpr int kItems = kSortCap / kThreads;
static_assert(kSortCap % kThreads == 0 && kSortCap < 65536, "16-bit digit counts");
static_assert(kItems % 4 == 0, "the sort loads its words in quads");

struct StreamParams {
  int64_t F, N, B, P, L, M_max;
  int32_t drop_last;
  uint32_t seed_lo, seed_hi;
  uint32_t m;        // log2 of the buckets per epoch
  uint32_t wb0;      // first bucket of this pass
  uint32_t nbw;      // buckets of this pass
  uint32_t C;        // ids per chunk (a multiple of kRound)
  uint32_t cbits;    // C <= 2^cbits
  uint32_t nchunks;  // chunks per epoch
  int32_t e0;        // epoch of the batch's first keys
  int32_t e_first;   // epoch written at the start of the rows
  int32_t cap;       // largest bucket sorted in LDS
};

__device__ __forceinline__ uint32_t bucket_of(uint32_t key, uint32_t m) {
  return m ? key >> (32u - m) : 0u;
}

// kb: the top (32 - cbits) bits of the key's offset inside its bucket
// (32 - m bits); monotone in the key inside a bucket.
__device__ __forceinline__ uint32_t stored_bits(uint32_t key, uint32_t m, uint32_t cbits) {
  const uint32_t off = m ? key & (0xFFFFFFFFu >> m) : key;
  return cbits >= m ? off >> (cbits - m) : off << (m - cbits);
}

__device__ __forceinline__ uint32_t philox_key(uint32_t id, uint32_t e, uint32_t slo, uint32_t shi) {
  const Philox4 r = philox_block(id >> 2, e, slo, shi);
  const uint32_t s = id & 3u;
  return s == 0 ? r.x : (s == 1 ? r.y : (s == 2 ? r.z : r.w));
}

// -- 1. histogram of buckets per chunk ----------------------------------------
// cnt layout: [epoch][chunk][bucket of the pass]
__global__ void __launch_bounds__(kThreads)
stream_count(StreamParams p, uint32_t* __restrict__ cnt) {
  extern __shared__ uint32_t hist[];
  const uint32_t nbw = p.nbw;
  for (uint32_t b = threadIdx.x; b < nbw; b += kThreads) hist[b] = 0;
  __syncthreads();
  const uint32_t e = uint32_t(p.e0) + blockIdx.y;
  const int64_t blk0 = int64_t(blockIdx.x) * (p.C / 4);
  const int iters = int(p.C / (4 * kThreads));
  for (int it = 0; it < iters; ++it) {
    const int64_t blk = blk0 + int64_t(it) * kThreads + threadIdx.x;
    const int64_t id0 = blk * 4;
    if (id0 < p.F) {
      const Philox4 r = philox_block(uint32_t(blk), e, p.seed_lo, p.seed_hi);
      const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t b = bucket_of(w[c], p.m) - p.wb0;
        if (id0 + c < p.F && b < nbw) atomicAdd(&hist[b], 1u);
      }
    }
  }
  __syncthreads();
  uint32_t* out = cnt + (int64_t(blockIdx.y) * p.nchunks + blockIdx.x) * nbw;
  for (uint32_t b = threadIdx.x; b < nbw; b += kThreads) out[b] = hist[b];
}

// -- 2. run starts --------------------------------------------------------------
// In place: cnt[e][c][b] becomes the number of bucket-b keys of epoch e in
// chunks before c; offb[e][b][c] receives the same values bucket-major, with
// offb[e][b][nchunks] and tot[e][b] the bucket size.
__global__ void __launch_bounds__(256)
stream_offsets(StreamParams p, uint32_t* __restrict__ cnt, uint32_t* __restrict__ offb,
               uint32_t* __restrict__ tot) {
  __shared__ uint32_t tile[64][65];
  const uint32_t nbw = p.nbw, nch = p.nchunks;
  const int64_t e = blockIdx.y;
  const uint32_t b0 = blockIdx.x * 64;
  const uint32_t tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  uint32_t* ce = cnt + e * int64_t(nch) * nbw;
  uint32_t* oe = offb + e * int64_t(nbw) * (nch + 1);
  uint32_t run = 0;  // column threadIdx.x (< 64): running sum of bucket b0 + threadIdx.x
  for (uint32_t c0 = 0; c0 < nch; c0 += 64) {
    for (uint32_t y = ty; y < 64; y += 4) {
      const uint32_t c = c0 + y, b = b0 + tx;
      tile[y][tx] = (c < nch && b < nbw) ? ce[int64_t(c) * nbw + b] : 0u;
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      for (int y = 0; y < 64; ++y) {
        const uint32_t v = tile[y][threadIdx.x];
        tile[y][threadIdx.x] = run;
        run += v;
      }
    }
    __syncthreads();
    for (uint32_t y = ty; y < 64; y += 4) {
      const uint32_t c = c0 + y, b = b0 + tx;
      if (c < nch && b < nbw) ce[int64_t(c) * nbw + b] = tile[y][tx];
      const uint32_t bb = b0 + y, cc = c0 + tx;
      if (bb < nbw && cc < nch) oe[int64_t(bb) * (nch + 1) + cc] = tile[tx][y];
    }
    __syncthreads();
  }
  if (threadIdx.x < 64 && b0 + threadIdx.x < nbw) {
    const uint32_t b = b0 + threadIdx.x;
    oe[int64_t(b) * (nch + 1) + nch] = run;
    tot[e * nbw + b] = run;
  }
}

// -- 3. bucket starts ----------------------------------------------------------
// wst[e][b]: start of bucket b inside the pass's part of epoch e (its words'
// position), wst[e][nbw] the part's size; wbase[e]: the part's first
// position in the epoch (the keys of earlier passes), wpos[e] advanced past
// the part for the next pass.
__global__ void __launch_bounds__(1024)
stream_scan(uint32_t nbw, const uint32_t* __restrict__ tot, uint32_t* __restrict__ wst,
            uint32_t* __restrict__ wpos, uint32_t* __restrict__ wbase) {
  __shared__ uint32_t tmp[65];
  const uint32_t* t = tot + int64_t(blockIdx.x) * nbw;
  uint32_t* st = wst + int64_t(blockIdx.x) * (nbw + 1);
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nbw; base += blockDim.x) {
    const uint32_t b = base + threadIdx.x;
    const uint32_t v = b < nbw ? t[b] : 0u;
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(v, tmp, &total);
    if (b < nbw) st[b] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) {
    st[nbw] = carry;
    const uint32_t w = wpos[blockIdx.x];
    wbase[blockIdx.x] = w;
    wpos[blockIdx.x] = w + carry;
  }
}

__global__ void stream_zero(uint32_t* __restrict__ a, uint32_t n) {
  for (uint32_t x = threadIdx.x; x < n; x += blockDim.x) a[x] = 0;
}

// -- 4. scatter ------------------------------------------------------------------
// One workgroup per (chunk, epoch). Per round of kRound ids (the larger the
// round, the longer each bucket's run and the fewer partly written cache
// lines: 24,576 ids take 126 KB of LDS, one workgroup per CU, which measured
// 1.54 ms at ImageNet-22k against 1.82 ms for 12,288-id rounds at two per
// CU): the pass's keys
// are counting-sorted by bucket in LDS (16-bit counts, two per word) and
// written as words, consecutive threads on consecutive positions; the bucket
// of staged position q is found from a table of the bucket at every 8th
// position and a short forward walk over the bucket starts.
__global__ void __launch_bounds__(kThreads)
stream_scatter(StreamParams p, const uint32_t* __restrict__ wst, const uint32_t* __restrict__ offc,
               uint32_t* __restrict__ words) {
  __shared__ uint32_t stage[kRound];                      // staged words
  __shared__ uint32_t cntw[kMaxWin / 2 + 1];              // 16-bit counts / starts
  __shared__ int32_t dl[kMaxWin];                         // run position - start, per bucket
  __shared__ uint16_t blk[kRound >> kBlkShift];           // bucket at every 8th position
  __shared__ uint32_t tmp[65];
  const uint32_t nbw = p.nbw;
  uint16_t* c16 = reinterpret_cast<uint16_t*>(cntw);      // bucket b at [b]
  const uint32_t chunk = xcd_logical(blockIdx.x, gridDim.x);
  if (chunk >= p.nchunks) return;
  const uint32_t e = uint32_t(p.e0) + blockIdx.y;
  const uint32_t* st = wst + int64_t(blockIdx.y) * (nbw + 1);
  const uint32_t* oc = offc + (int64_t(blockIdx.y) * p.nchunks + chunk) * nbw;
  uint32_t* out = words + int64_t(blockIdx.y) * p.F;
  // the chunk's run positions per bucket: requested here (unconditionally),
  // stored to LDS once the first round's keys are counted
  constexpr int kDl = kMaxWin / kThreads;
  static_assert(kMaxWin % kThreads == 0, "run positions per thread");
  int32_t dlv[kDl];
#pragma unroll
  for (int m = 0; m < kDl; ++m) {
    const uint32_t b = threadIdx.x + uint32_t(m) * kThreads;
    const uint32_t bc = b < nbw ? b : 0u;
    dlv[m] = int32_t(st[bc] + oc[bc]);
  }
  const int64_t id_chunk = int64_t(chunk) * p.C;
  for (int64_t r0 = id_chunk; r0 < id_chunk + p.C && r0 < p.F; r0 += kRound) {
    for (uint32_t x = threadIdx.x; x < (nbw + 2) / 2; x += kThreads) cntw[x] = 0;
    __syncthreads();
    // per id: its word, and its bucket and slot packed as b << 16 | slot
    // (b < 4096, slot < kRound), or ~0 when the id is not in this pass
    uint32_t wd[kRoundBlocks][4], bs[kRoundBlocks][4];
#pragma unroll
    for (int it = 0; it < kRoundBlocks; ++it) {
      const int64_t blk4 = r0 / 4 + it * kThreads + threadIdx.x;
      const int64_t id0 = blk4 * 4;
      const Philox4 r = philox_block(uint32_t(blk4), e, p.seed_lo, p.seed_hi);
      const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t b = bucket_of(w[c], p.m) - p.wb0;
        wd[it][c] = (stored_bits(w[c], p.m, p.cbits) << p.cbits) | uint32_t(id0 + c - id_chunk);
        bs[it][c] = 0xFFFFFFFFu;
        if (id0 + c < p.F && b < nbw) {
          const uint32_t half = (b & 1u) * 16u;
          bs[it][c] = (b << 16) | ((atomicAdd(&cntw[b >> 1], 1u << half) >> half) & 0xFFFFu);
        }
      }
    }
    if (r0 == id_chunk) {  // uniform
#pragma unroll
      for (int m = 0; m < kDl; ++m) {
        const uint32_t b = threadIdx.x + uint32_t(m) * kThreads;
        if (b < nbw) dl[b] = dlv[m];
      }
    }
    __syncthreads();
    // exclusive scan of the 16-bit counts (nbw <= 4096: at most two words
    // per thread); c16[nbw] receives the round's total
    uint32_t total;
    {
      const uint32_t nw = (nbw + 1) / 2;
      const uint32_t w0 = 2 * threadIdx.x, w1 = w0 + 1;
      const uint32_t v0 = w0 < nw ? cntw[w0] : 0u, v1 = w1 < nw ? cntw[w1] : 0u;
      const uint32_t s = (v0 & 0xFFFFu) + (v0 >> 16) + (v1 & 0xFFFFu) + (v1 >> 16);
      uint32_t ex = block_exclusive_scan<false>(s, tmp, &total);  // closed below
      if (w0 < nw) {
        const uint32_t a = ex, b = a + (v0 & 0xFFFFu);
        cntw[w0] = a | (b << 16);
        ex = b + (v0 >> 16);
      }
      if (w1 < nw) {
        const uint32_t a = ex, b = a + (v1 & 0xFFFFu);
        cntw[w1] = a | (b << 16);
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) c16[nbw] = uint16_t(total);
#pragma unroll
    for (int it = 0; it < kRoundBlocks; ++it)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (bs[it][c] != 0xFFFFFFFFu) stage[c16[bs[it][c] >> 16] + (bs[it][c] & 0xFFFFu)] = wd[it][c];
    __syncthreads();
    // bucket of every 8th staged position
    for (uint32_t b = threadIdx.x; b < nbw; b += kThreads) {
      const uint32_t a = c16[b], z = c16[b + 1];
      for (uint32_t k = (a + (1u << kBlkShift) - 1) >> kBlkShift; (k << kBlkShift) < z; ++k)
        blk[k] = uint16_t(b);
    }
    __syncthreads();
    for (uint32_t q = threadIdx.x; q < total; q += kThreads) {
      uint32_t b = blk[q >> kBlkShift];
      while (c16[b + 1] <= q) ++b;
      out[uint32_t(dl[b]) + q - c16[b]] = stage[q];
    }
    __syncthreads();
    for (uint32_t b = threadIdx.x; b < nbw; b += kThreads) dl[b] += int32_t(c16[b + 1] - c16[b]);
    __syncthreads();  // the counts are read above before the next round clears them
  }
}

// -- 5. per-bucket sort and shard ------------------------------------------------
__device__ __forceinline__ bool key_id_greater(uint32_t ka, uint32_t ia, uint32_t kb, uint32_t ib) {
  return ka > kb || (ka == kb && ia > ib);
}

// In-place bitonic sort of n ids in global memory by one workgroup, by
// (key, id) with the keys regenerated per comparison. Every merge starts
// with a "flip" comparator, so all comparators point the same way and the
// virtual padding (+inf beyond n) never moves.
__device__ void global_bitonic(int32_t* gi, uint32_t n, uint32_t e, uint32_t slo, uint32_t shi) {
  uint32_t P2 = 1;
  while (P2 < n) P2 <<= 1;
  for (uint32_t k = 2; k <= P2; k <<= 1) {
    for (uint32_t s = k >> 1; s >= 1; s >>= 1) {
      for (uint32_t t = threadIdx.x; t < P2 / 2; t += blockDim.x) {
        const uint32_t blk = t / s, off = t % s;
        uint32_t i, j;
        if (s == (k >> 1)) {
          i = blk * k + off;
          j = blk * k + k - 1 - off;
        } else {
          i = blk * 2 * s + off;
          j = i + s;
        }
        if (j < n) {
          const uint32_t ia = uint32_t(gi[i]), ib = uint32_t(gi[j]);
          if (key_id_greater(philox_key(ia, e, slo, shi), ia, philox_key(ib, e, slo, shi), ib)) {
            gi[i] = int32_t(ib);
            gi[j] = int32_t(ia);
          }
        }
      }
      __threadfence_block();
      __syncthreads();
    }
  }
}

__device__ __forceinline__ int64_t row_offset(const StreamParams& p, uint32_t i, int64_t e) {
  const int64_t Li = p.drop_last ? p.L : epoch_len(p.F, p.N, p.B, 0, i);
  return int64_t(i) * p.M_max + (e - p.e_first) * Li;
}

// Largest c with ob[c] <= q (the run holding position q; empty runs share
// their start with the next run, which the largest index skips).
__device__ __forceinline__ uint32_t run_search(const uint32_t* ob, uint32_t nch, uint32_t q) {
  uint32_t lo = 0, hi = nch;  // ob[lo] <= q < ob[hi] (ob[nch] = n > q)
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (ob[mid] <= q) lo = mid;
    else hi = mid;
  }
  return lo;
}

// A bucket larger than the LDS capacity: its words decoded into ids in
// place (run table in LDS), sorted by (key, id) in global memory, sharded.
__device__ void sort_in_global(const StreamParams& p, const uint32_t* ob, uint32_t* gw, uint32_t n,
                               uint32_t e, uint32_t pos0, int64_t pend64, int32_t* __restrict__ R) {
  const uint32_t lmask = (1u << p.cbits) - 1u;
  for (uint32_t q = threadIdx.x; q < n; q += kThreads) {
    const uint32_t w = gw[q];
    const uint32_t c = run_search(ob, p.nchunks, q);
    gw[q] = c * p.C + (w & lmask);
  }
  __threadfence_block();
  __syncthreads();
  int32_t* gi = reinterpret_cast<int32_t*>(gw);
  global_bitonic(gi, n, e, p.seed_lo, p.seed_hi);
  const uint32_t N = uint32_t(p.N);
  for (int64_t q = threadIdx.x; int64_t(pos0) + q < pend64; q += kThreads) {
    const uint32_t pp = pos0 + uint32_t(q);
    const uint32_t i = pp % N, j = pp / N;
    R[row_offset(p, i, e) + j] = gi[q];
  }
}

// LDS: 64 KB of 8-byte entries (kb << 32 | id), later kb and the ids by
// position (kb then gives way to full keys and the shard stage), and 16 KB
// that first hold the run table (bucket-major run starts, the run at every
// 8th position), then the 16-bit digit counts, then the list of tied runs:
// 80 KB, two workgroups per CU.
constexpr int kSortDigitBits = 13;
constexpr int kSortDigits = 1 << kSortDigitBits;
constexpr int kCountWords = kSortDigits / 2;
constexpr uint32_t kSlotBits = 13;  // bits of a counting-sort slot
static_assert(kSortCap <= (1 << kSlotBits), "slots fit kSlotBits");
// kb has 32 - cbits bits and C >= kRound, so cbits >= kSlotBits and
// kb << kSlotBits | slot fits 32 bits
static_assert((1 << kSlotBits) <= kRound, "kb and slot fit one word");
static_assert(kMaxChunks + 1 + (kSortCap >> kBlkShift) / 2 <= kCountWords,
              "the run table fits the digit counts' space");

__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(8)))
stream_sort(StreamParams p, const uint32_t* __restrict__ wst, const uint32_t* __restrict__ wbase,
            const uint32_t* __restrict__ offb, uint32_t* __restrict__ words, int32_t* __restrict__ R) {
  __shared__ uint64_t kv[kSortCap];
  __shared__ uint32_t cw[kCountWords];
  uint32_t* ob = cw;                                                 // [nchunks + 1]
  uint16_t* blk = reinterpret_cast<uint16_t*>(cw + p.nchunks + 1);  // [kSortCap >> kBlkShift]
  const uint16_t* h16 = reinterpret_cast<const uint16_t*>(cw);      // digit d at [d]
  const uint32_t nbw = p.nbw, nch = p.nchunks;
  const uint32_t b = xcd_logical(blockIdx.x, gridDim.x);
  if (b >= nbw) return;
  const uint32_t e = uint32_t(p.e0) + blockIdx.y;
  const uint32_t* st = wst + int64_t(blockIdx.y) * (nbw + 1);
  const uint32_t lo = st[b];
  const uint32_t n = st[b + 1] - lo;
  if (n == 0) return;
  const uint32_t pos0 = wbase[blockIdx.y] + lo;  // epoch position of the bucket's first element
  uint32_t* gw = words + int64_t(blockIdx.y) * p.F + lo;
  const uint32_t N = uint32_t(p.N);
  const int64_t pend64 = int64_t(pos0) + n < p.P ? int64_t(pos0) + n : p.P;
  const uint32_t lmask = (1u << p.cbits) - 1u;
  const uint32_t* obg = offb + (int64_t(blockIdx.y) * nbw + b) * (nch + 1);
  const bool fast = n <= uint32_t(p.cap);
  // Item r of a thread is position item_pos(r): four consecutive positions
  // per quad, quads kQuad positions apart. The words are requested before
  // the run table, so both round trips overlap: each quad as one 16-byte
  // load (4-byte aligned; words past the bucket are not used) where it
  // stays inside the words of the launch, else word by word.
  constexpr uint32_t kQuad = 4 * kThreads;
  auto item_pos = [](int r) { return uint32_t(r >> 2) * kQuad + 4 * threadIdx.x + uint32_t(r & 3); };
  uint32_t kb[kItems], id[kItems];
  if (fast) {
    const int64_t room = int64_t(gridDim.y - blockIdx.y) * p.F - lo;  // words from gw to the end
#pragma unroll
    for (int h = 0; h < kItems / 4; ++h) {
      const uint32_t q0 = item_pos(4 * h);
      if (int64_t(q0) + 4 <= room) {
        uint4 w;
        __builtin_memcpy(&w, gw + q0, 16);
        kb[4 * h] = w.x;
        kb[4 * h + 1] = w.y;
        kb[4 * h + 2] = w.z;
        kb[4 * h + 3] = w.w;
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) kb[4 * h + u] = q0 + u < n ? gw[q0 + u] : 0u;
      }
    }
  }
  for (uint32_t c = threadIdx.x; c <= nch; c += kThreads) ob[c] = obg[c];
  __syncthreads();
  if (!fast) {
    sort_in_global(p, ob, gw, n, e, pos0, pend64, R);
    return;
  }

  // run at every 8th position of the bucket
  for (uint32_t c = threadIdx.x; c < nch; c += kThreads) {
    const uint32_t a = ob[c], z = ob[c + 1];
    for (uint32_t k = (a + (1u << kBlkShift) - 1) >> kBlkShift; (k << kBlkShift) < z; ++k)
      blk[k] = uint16_t(c);
  }
  __syncthreads();
  // a quad's first position finds its run from the table, the next three
  // step on from there
#pragma unroll
  for (int h = 0; h < kItems / 4; ++h) {
    const uint32_t q0 = item_pos(4 * h);
    uint32_t c = q0 < n ? blk[q0 >> kBlkShift] : 0u;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t q = q0 + u;
      if (q < n) {
        while (ob[c + 1] <= q) ++c;
        id[4 * h + u] = c * p.C + (kb[4 * h + u] & lmask);
        kb[4 * h + u] >>= p.cbits;
      }
    }
  }
  __syncthreads();  // the run table is no longer needed: its space holds the digit counts
  const uint32_t kbits = 32u - p.cbits;
  const uint32_t dbits = kbits < uint32_t(kSortDigitBits) ? kbits : uint32_t(kSortDigitBits);
  const uint32_t dshift = kbits - dbits;
  const uint32_t ndig = 1u << dbits;
  for (int x = threadIdx.x; x < kCountWords; x += kThreads) cw[x] = 0;
  __syncthreads();
  uint32_t pos[kItems];
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = item_pos(r);
    if (q < n) {
      const uint32_t d = kb[r] >> dshift;
      const uint32_t half = (d & 1u) * 16u;
      pos[r] = (atomicAdd(&cw[d >> 1], 1u << half) >> half) & 0xFFFFu;
    }
  }
  __syncthreads();
  {
    constexpr int kPerW = kCountWords / kThreads;  // count words per thread
    uint32_t v[kPerW];
    uint32_t sum = 0;
#pragma unroll
    for (int j = 0; j < kPerW; ++j) {
      v[j] = cw[threadIdx.x * kPerW + j];
      sum += (v[j] & 0xFFFFu) + (v[j] >> 16);
    }
    uint32_t total;
    uint32_t ex = block_exclusive_scan<false>(sum, reinterpret_cast<uint32_t*>(kv), &total);  // closed below
#pragma unroll
    for (int j = 0; j < kPerW; ++j) {
      const uint32_t lo16 = ex;
      ex += v[j] & 0xFFFFu;
      cw[threadIdx.x * kPerW + j] = lo16 | (ex << 16);
      ex += v[j] >> 16;
    }
  }
  __syncthreads();
  // Each counting-sort slot holds kb << kSlotBits | slot: one comparison
  // orders two entries by (kb, slot), and an entry of a later digit group
  // compares above every entry of an earlier one.
#ifndef NOPFS_SORT_GROUP_LOADS
#define NOPFS_SORT_GROUP_LOADS 4
#endif
  constexpr uint32_t kGroupLoads = NOPFS_SORT_GROUP_LOADS;
  uint32_t* kbs = reinterpret_cast<uint32_t*>(kv);  // [kSortCap + kGroupLoads] by slot
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = item_pos(r);
    if (q < n) {
      pos[r] += h16[kb[r] >> dshift];
      kbs[pos[r]] = (kb[r] << kSlotBits) | pos[r];
    }
  }
  if (threadIdx.x < kGroupLoads) kbs[n + threadIdx.x] = 0xFFFFFFFFu;  // above every entry
  __syncthreads();
  // Inside its digit group (about two entries), an entry's place in kb
  // order is the group start plus the group entries below it in (kb, slot)
  // order (runs of equal kb are re-sorted by full key and id below). The
  // first kGroupLoads slots from the group start are compared
  // unconditionally: slots past the group belong to later groups or are
  // the guards past the end, and compare above. A larger group walks the
  // rest.
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = item_pos(r);
    if (q < n) {
      const uint32_t d = kb[r] >> dshift;
      const uint32_t a0 = h16[d];
      const uint32_t a1 = d + 1 < ndig ? h16[d + 1] : n;
      const uint32_t me = (kb[r] << kSlotBits) | pos[r];
      uint32_t below = 0;
#pragma unroll
      for (uint32_t j = 0; j < kGroupLoads; ++j) below += kbs[a0 + j] < me;
      for (uint32_t v = a0 + kGroupLoads; v < a1; ++v) below += kbs[v] < me;
      pos[r] = a0 + below;
    }
  }
  __syncthreads();  // the slots and the digit counts are no longer needed
  // kb and ids by (kb, id) position, then runs of equal kb (a few percent of
  // the entries) re-sorted by (full key, id), one thread per run.
  uint32_t* kbp = reinterpret_cast<uint32_t*>(kv);  // [kSortCap] kb, later full keys, later the shard stage
  uint32_t* sorted = kbp + kSortCap;                // [kSortCap] ids in (key, id) order
  uint16_t* runs = reinterpret_cast<uint16_t*>(cw); // [0..1]: run count (32-bit), then run starts
  uint32_t* nruns = cw;
  if (threadIdx.x == 0) *nruns = 0;
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = item_pos(r);
    if (q < n) {
      kbp[pos[r]] = kb[r];
      sorted[pos[r]] = id[r];
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = uint32_t(r * kThreads) + threadIdx.x;
    if (q + 1 < n) {
      const uint32_t k0 = kbp[q];
      if (k0 == kbp[q + 1] && (q == 0 || kbp[q - 1] != k0)) runs[2 + atomicAdd(nruns, 1u)] = uint16_t(q);
    }
  }
  __syncthreads();
  {
    const uint32_t nr = *nruns;  // at most n / 2 runs: the list fits
    for (uint32_t t = threadIdx.x; t < nr; t += kThreads) {
      const uint32_t a0 = runs[2 + t];
      const uint32_t kk = kbp[a0];
      uint32_t a1 = a0 + 2;
      while (a1 < n && kbp[a1] == kk) ++a1;
      for (uint32_t x = a0; x < a1; ++x) kbp[x] = philox_key(sorted[x], e, p.seed_lo, p.seed_hi);
      for (uint32_t x = a0 + 1; x < a1; ++x) {
        const uint32_t fx = kbp[x], ix = sorted[x];
        uint32_t y = x;
        while (y > a0 && key_id_greater(kbp[y - 1], sorted[y - 1], fx, ix)) {
          kbp[y] = kbp[y - 1];
          sorted[y] = sorted[y - 1];
          --y;
        }
        kbp[y] = fx;
        sorted[y] = ix;
      }
    }
  }
  __syncthreads();

  if (pend64 <= int64_t(pos0)) return;
  const uint32_t pend = uint32_t(pend64);
  const uint32_t j0 = pos0 / N, j1 = (pend - 1) / N;
  const uint32_t nj = j1 - j0 + 1;
  const uint32_t Np = (N & 1u) ? N : N + 1u;  // odd row pitch: conflict-free columns
  // (j, i) of position pos0 + threadIdx.x, stepped by kThreads positions per
  // iteration without dividing
  const uint32_t step_i = kThreads % N, step_j = kThreads / N;
  uint32_t ci = (pos0 + threadIdx.x) % N, cj = (pos0 + threadIdx.x) / N;
  if (uint64_t(nj) * Np <= uint64_t(kSortCap)) {
    uint32_t* stage = kbp;
    for (uint32_t q = threadIdx.x; pos0 + q < pend; q += kThreads) {
      stage[(cj - j0) * Np + ci] = sorted[q];
      ci += step_i;
      cj += step_j;
      if (ci >= N) {
        ci -= N;
        ++cj;
      }
    }
    __syncthreads();
    // t -> (row i, column jj) with consecutive t on consecutive columns of a
    // row: one division per thread, then stepped by kThreads per iteration
    const uint32_t total = nj * N;
    const uint32_t si = kThreads / nj, sj = kThreads % nj;
    auto write = [&](auto row) {
      uint32_t i = threadIdx.x / nj, jj = threadIdx.x % nj;
      for (uint32_t t = threadIdx.x; t < total; t += kThreads) {
        const uint32_t pp = (j0 + jj) * N + i;
        if (pp >= pos0 && pp < pend) row(i)[jj] = int32_t(stage[jj * Np + i]);
        i += si;
        jj += sj;
        if (jj >= nj) {
          jj -= nj;
          ++i;
        }
      }
    };
    if (p.drop_last) {  // every row holds L reads per epoch: one offset for all rows
      int32_t* const Re = R + (int64_t(e) - p.e_first) * p.L + j0;
      write([&](uint32_t i) { return Re + int64_t(i) * p.M_max; });
    } else {
      write([&](uint32_t i) { return R + row_offset(p, i, e) + j0; });
    }
  } else {
    for (uint32_t q = threadIdx.x; pos0 + q < pend; q += kThreads) {
      R[row_offset(p, ci, e) + cj] = int32_t(sorted[q]);
      ci += step_i;
      cj += step_j;
      if (ci >= N) {
        ci -= N;
        ++cj;
      }
    }
  }
}

// drop_last=0: rows shorter than M_max end with -1.
__global__ void stream_pad(StreamParams p, int32_t* __restrict__ R) {
  const int64_t E = p.M_max / p.L;
  const int64_t i = blockIdx.x;
  const int64_t Mi = E * epoch_len(p.F, p.N, p.B, 0, i);
  for (int64_t f = Mi + threadIdx.x; f < p.M_max; f += blockDim.x) R[i * p.M_max + f] = -1;
}

}  // namespace

int streams_impl(const nopfs_job* job, int32_t* R, hipStream_t st, int32_t e_begin,
                 int32_t e_end) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (e_begin < 0) e_begin = 0, e_end = int32_t(s.E);  // the whole job
  if (e_end < e_begin || e_end > s.E) return fail(NOPFS_EINVAL, "epochs must satisfy 0 <= e_begin <= e_end <= E");
  // rows of the range: a job of e_end - e_begin epochs (same F, N, B)
  if (e_end - e_begin != s.E) {
    if (e_end == e_begin) return NOPFS_OK;  // no epochs: R has no elements
    nopfs_job sub = *job;
    sub.E = e_end - e_begin;
    if ((rc = make_shape(&sub, &s))) return rc;
  }
  if (s.M_max == 0) return NOPFS_OK;  // no reads: R has no elements and may be NULL
  if (!R) return fail(NOPFS_EINVAL, "R is NULL");

  int64_t cap = kSortCap;
  if (debug_value(1) > 0 && debug_value(1) < cap) cap = debug_value(1);
  // 2^m buckets per epoch, the fewest with a mean of at most kMeanBucket
  uint32_t m = 0;
  while (m < 31 && (s.F >> m) > kMeanBucket) ++m;
  const uint32_t nb = 1u << m;
  const uint32_t nbw = nb < kMaxWin ? nb : kMaxWin;
  // chunks: multiples of a scatter round, at most kMaxChunks per epoch
  int64_t C = int64_t(kRound) * kChunkRounds;
  while (ceil_div(s.F, C) > int64_t(kMaxChunks)) C *= 2;
  uint32_t cbits = 0;
  while ((int64_t(1) << cbits) < C) ++cbits;
  const uint32_t nchunks = uint32_t(ceil_div(s.F, C));

  StreamParams p;
  p.F = s.F; p.N = s.N; p.B = s.B; p.P = s.P; p.L = s.L; p.M_max = s.M_max;
  p.drop_last = s.drop_last;
  p.seed_lo = uint32_t(s.seed);
  p.seed_hi = uint32_t(s.seed >> 32);
  p.m = m;
  p.nbw = nbw;
  p.C = uint32_t(C);
  p.cbits = cbits;
  p.nchunks = nchunks;
  p.cap = int32_t(cap);
  p.e_first = e_begin;

  // epochs per batch: the words of a batch stay under ~16 GB of scratch
  const int64_t budget = int64_t(16) << 30;
  int64_t EB = budget / (4 * s.F);
  if (EB < 1) EB = 1;
  if (EB > s.E) EB = s.E;

  Scratch scr(st);
  uint32_t *words, *cnt, *offb, *tot, *wst, *wpos, *wbase;
  if ((rc = scr.alloc_n(&words, size_t(EB * s.F)))) return rc;
  if ((rc = scr.alloc_n(&cnt, size_t(EB) * nchunks * nbw))) return rc;
  if ((rc = scr.alloc_n(&offb, size_t(EB) * nbw * (nchunks + 1)))) return rc;
  if ((rc = scr.alloc_n(&tot, size_t(EB) * nbw))) return rc;
  if ((rc = scr.alloc_n(&wst, size_t(EB) * (nbw + 1)))) return rc;
  if ((rc = scr.alloc_n(&wpos, size_t(EB)))) return rc;
  if ((rc = scr.alloc_n(&wbase, size_t(EB)))) return rc;


  for (int64_t e0 = 0; e0 < s.E; e0 += EB) {
    const uint32_t eb = uint32_t(e0 + EB <= s.E ? EB : s.E - e0);
    p.e0 = int32_t(e_begin + e0);
    if ((rc = launch("stream_zero", stream_zero, dim3(1), dim3(256), 0, st, wpos, eb))) return rc;
    for (uint32_t wb0 = 0; wb0 < nb; wb0 += nbw) {
      p.wb0 = wb0;
      if ((rc = launch("stream_count", stream_count, dim3(nchunks, eb), dim3(kThreads),
                       size_t(nbw) * 4, st, p, cnt)))
        return rc;
      if ((rc = launch("stream_offsets", stream_offsets, dim3(uint32_t(ceil_div(nbw, 64)), eb),
                       dim3(256), 0, st, p, cnt, offb, tot)))
        return rc;
      if ((rc = launch("stream_scan", stream_scan, dim3(eb), dim3(1024), 0, st, nbw,
                       (const uint32_t*)tot, wst, wpos, wbase)))
        return rc;
      if ((rc = launch("stream_scatter", stream_scatter, dim3(xcd_padded(nchunks), eb),
                       dim3(kThreads), 0, st, p, (const uint32_t*)wst,
                       (const uint32_t*)cnt, words)))
        return rc;
      if ((rc = launch("stream_sort", stream_sort, dim3(xcd_padded(nbw), eb), dim3(kThreads),
                       0, st, p, (const uint32_t*)wst, (const uint32_t*)wbase,
                       (const uint32_t*)offb, words, R)))
        return rc;
    }
  }
  if (!s.drop_last && s.F % s.N != 0) {
    if ((rc = launch("stream_pad", stream_pad, dim3(uint32_t(s.N)), dim3(64), 0, st, p, R))) return rc;
  }
  return NOPFS_OK;
}

}  // namespace nopfs

extern "C" int nopfs_access_streams(const nopfs_job* job, int32_t* R, void* hip_stream) {
  try {
    return nopfs::streams_impl(job, R, static_cast<hipStream_t>(hip_stream), -1, -1);
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}

extern "C" int nopfs_access_streams_range(const nopfs_job* job, int32_t e_begin, int32_t e_end,
                                          int32_t* R, void* hip_stream) {
  try {
    if (e_begin < 0) return nopfs::fail(NOPFS_EINVAL, "epochs must satisfy 0 <= e_begin <= e_end <= E");
    return nopfs::streams_impl(job, R, static_cast<hipStream_t>(hip_stream), e_begin, e_end);
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}
