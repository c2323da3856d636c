// nopfs_access_streams: every worker's access stream for every epoch.
//
// Section 2 of the paper: an epoch is a random shuffle of all sample ids and
// the seed reproduces it. Section 4: each global batch is partitioned among
// the N workers and a worker's stream R is the concatenation of its batches.
//
// Epoch e orders the samples by (key_e(k), k), key_e(k) a Philox-4x32-10
// word. The order is built as a bucket sort over all epochs of a batch at
// once. Fine bucket b = umulhi(key, nb) holds a few thousand keys; coarse
// bucket c = umulhi(key, nb1) (nb = nb1 * nf) groups nf consecutive fine ones.
//   1. stream_count   -- Philox keys in registers; per (epoch, chunk of 64K
//                        ids) histogram of the fine buckets.
//   2. stream_offsets -- per (epoch, fine bucket) running sum over chunks.
//   3. stream_scan    -- fine bucket start positions per epoch.
//   4. stream_scatter -- keys regenerated and (key, id) pairs written into
//                        their coarse bucket (at most 64 per epoch, so each
//                        workgroup's open cache lines fit in L2 and every
//                        line is completed there before it is written back).
//   5. stream_split   -- each coarse bucket read back in 16K-pair pieces and
//                        split into its nf fine buckets (skipped when nf = 1).
//   6. stream_sort    -- one workgroup per fine bucket: counting sort in LDS
//                        by the top 13 bits of the key inside the bucket,
//                        each pair then placed inside its (tiny) digit group
//                        by its rank in (key, id) order, and
//                        the sorted positions p sharded straight into R:
//                        R[p mod N][e*L_i + p div N], through an LDS
//                        transpose so each worker row gets a run.
// Buckets larger than the LDS capacity (not expected for uniform keys, but
// possible in principle) are sorted in place in global memory by a bitonic
// network inside the same workgroup.
#include <limits.h>

#include "common.hpp"
#include "philox.hpp"

namespace nopfs {
namespace {

constexpr int kChunkThreads = 1024;
constexpr int kBlocksPerThread = 16;                                   // Philox blocks
constexpr int64_t kChunkIds = int64_t(kChunkThreads) * kBlocksPerThread * 4;  // 65536
constexpr uint32_t kMaxBuckets = 8192;

// Tuning knobs: bucket capacity = threads x items (identical results).
#ifndef NOPFS_SORT_THREADS
#define NOPFS_SORT_THREADS 1024
#endif
#ifndef NOPFS_SORT_ITEMS
#define NOPFS_SORT_ITEMS 8
#endif
constexpr int kSortThreads = NOPFS_SORT_THREADS;
constexpr int kItems = NOPFS_SORT_ITEMS;
constexpr int kSortCap = kSortThreads * kItems;  // 8192 (key, id) pairs in LDS
constexpr int kDigitBits = 13;
constexpr int kDigits = 1 << kDigitBits;

struct StreamParams {
  int64_t F, N, B, P, L, M_max;
  int32_t drop_last;
  uint32_t seed_lo, seed_hi;
  uint32_t nb;        // fine buckets per epoch
  uint32_t nb1;       // coarse buckets per epoch
  uint32_t nf;        // fine buckets per coarse bucket (nb = nb1 * nf)
  int32_t e0;         // first epoch of the batch (the epoch its keys are drawn for)
  int32_t e_first;    // epoch written at the start of the rows
  int32_t sort_bits;  // significant bits of a key inside its bucket
  int32_t cap;        // largest bucket sorted in LDS
};

// -- 1. histogram of buckets per chunk ----------------------------------------
// cnt layout: [epoch][chunk][bucket]
__global__ void __launch_bounds__(kChunkThreads)
stream_count(StreamParams p, uint32_t nchunks, uint32_t* __restrict__ cnt) {
  extern __shared__ uint32_t hist[];
  const uint32_t nb = p.nb;
  for (uint32_t b = threadIdx.x; b < nb; b += blockDim.x) hist[b] = 0;
  __syncthreads();
  const uint32_t e = uint32_t(p.e0) + blockIdx.y;
  const int64_t blk0 = int64_t(blockIdx.x) * (kChunkIds / 4);
#pragma unroll 4
  for (int it = 0; it < kBlocksPerThread; ++it) {
    const int64_t blk = blk0 + it * kChunkThreads + threadIdx.x;
    const int64_t id0 = blk * 4;
    if (id0 < p.F) {
      const Philox4 r = philox_block(uint32_t(blk), e, p.seed_lo, p.seed_hi);
      const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (id0 + c < p.F) atomicAdd(&hist[__umulhi(w[c], nb)], 1u);
    }
  }
  __syncthreads();
  uint32_t* out = cnt + (int64_t(blockIdx.y) * nchunks + blockIdx.x) * nb;
  for (uint32_t b = threadIdx.x; b < nb; b += blockDim.x) out[b] = hist[b];
}

// -- 2. chunk offsets inside each bucket --------------------------------------
// In place: cnt[e][c][b] becomes the number of bucket-b keys of epoch e in
// chunks before c; tot[e][b] receives the bucket size.
__global__ void __launch_bounds__(256)
stream_offsets(uint32_t nb, uint32_t nchunks, uint32_t* __restrict__ cnt,
               uint32_t* __restrict__ tot) {
  const uint32_t b = blockIdx.x * 256 + threadIdx.x;
  if (b >= nb) return;
  uint32_t* col = cnt + int64_t(blockIdx.y) * nchunks * nb + b;
  uint32_t run = 0;
  uint32_t c = 0;
  for (; c + 8 <= nchunks; c += 8) {
    uint32_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = col[int64_t(c + u) * nb];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      col[int64_t(c + u) * nb] = run;
      run += v[u];
    }
  }
  for (; c < nchunks; ++c) {
    const uint32_t v = col[int64_t(c) * nb];
    col[int64_t(c) * nb] = run;
    run += v;
  }
  tot[int64_t(blockIdx.y) * nb + b] = run;
}

// -- 3. bucket starts --------------------------------------------------------
__global__ void __launch_bounds__(1024)
stream_scan(uint32_t nb, const uint32_t* __restrict__ tot, uint32_t* __restrict__ start,
            uint32_t* __restrict__ cursor) {
  __shared__ uint32_t tmp[65];
  const uint32_t* t = tot + int64_t(blockIdx.x) * nb;
  uint32_t* st = start + int64_t(blockIdx.x) * (nb + 1);
  uint32_t* cu = cursor + int64_t(blockIdx.x) * nb;
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nb; base += blockDim.x) {
    const uint32_t b = base + threadIdx.x;
    const uint32_t v = b < nb ? t[b] : 0u;
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(v, tmp, &total);
    if (b < nb) {
      st[b] = carry + ex;
      cu[b] = carry + ex;
    }
    carry += total;
  }
  if (threadIdx.x == 0) st[nb] = carry;
}

// -- 4. scatter into coarse buckets ------------------------------------------
// Target bucket t = umulhi(key, nt): the fine bucket when nf = 1 (nt = nb),
// else the coarse bucket (nt = nb1); nt <= 64 either way. A chunk's share of
// bucket t starts at the bucket's first fine start plus the chunk's offsets
// in each of its fine buckets. The chunk is processed in rounds of 8K ids:
// each round is counting-sorted by bucket in LDS and every bucket's part of
// the round is written as one contiguous run after the previous rounds'.
constexpr int kRoundIds = 8192;
constexpr int kRoundBlocks = kRoundIds / 4 / kChunkThreads;  // Philox blocks per thread
constexpr int kMaxTargets = 64;

struct ScatterSmem {
  uint32_t key[kRoundIds];
  int32_t id[kRoundIds];
  uint32_t cnt[kMaxTargets];
  uint32_t off[kMaxTargets];   // start of each bucket's run in the round
  uint32_t base[kMaxTargets];  // next free position of each bucket (global)
};

__global__ void __launch_bounds__(kChunkThreads)
stream_scatter(StreamParams p, uint32_t nchunks, const uint32_t* __restrict__ cnt,
               const uint32_t* __restrict__ start, uint32_t* __restrict__ keys,
               int32_t* __restrict__ ids) {
  __shared__ ScatterSmem s;
  const uint32_t nb = p.nb, nf = p.nf;
  const uint32_t nt = nf == 1 ? nb : p.nb1;
  const uint32_t chunk = xcd_logical(blockIdx.x, gridDim.x);
  if (chunk >= nchunks) return;
  const uint32_t* off = cnt + (int64_t(blockIdx.y) * nchunks + chunk) * nb;
  const uint32_t* st = start + int64_t(blockIdx.y) * (nb + 1);
  for (uint32_t b = threadIdx.x; b < nt; b += blockDim.x) {
    uint32_t o = 0;
    for (uint32_t f = b * nf; f < (b + 1) * nf; ++f) o += off[f];
    s.base[b] = st[b * nf] + o;
  }
  const uint32_t e = uint32_t(p.e0) + blockIdx.y;
  uint32_t* ko = keys + int64_t(blockIdx.y) * p.F;
  int32_t* io = ids + int64_t(blockIdx.y) * p.F;
  const int64_t id_chunk = int64_t(chunk) * kChunkIds;
  for (int64_t r0 = id_chunk; r0 < id_chunk + kChunkIds && r0 < p.F; r0 += kRoundIds) {
    if (threadIdx.x < nt) s.cnt[threadIdx.x] = 0;
    __syncthreads();
    uint32_t w[kRoundBlocks][4], slot[kRoundBlocks][4];
#pragma unroll
    for (int it = 0; it < kRoundBlocks; ++it) {
      const int64_t blk = r0 / 4 + it * kChunkThreads + threadIdx.x;
      const int64_t id0 = blk * 4;
      const Philox4 r = philox_block(uint32_t(blk), e, p.seed_lo, p.seed_hi);
      w[it][0] = r.x; w[it][1] = r.y; w[it][2] = r.z; w[it][3] = r.w;
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (id0 + c < p.F) slot[it][c] = atomicAdd(&s.cnt[__umulhi(w[it][c], nt)], 1u);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      const uint32_t v = threadIdx.x < nt ? s.cnt[threadIdx.x] : 0u;
      const uint32_t inc = wave_inclusive_scan(v);
      if (threadIdx.x < nt) s.off[threadIdx.x] = inc - v;
    }
    __syncthreads();
#pragma unroll
    for (int it = 0; it < kRoundBlocks; ++it) {
      const int64_t blk = r0 / 4 + it * kChunkThreads + threadIdx.x;
      const int64_t id0 = blk * 4;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (id0 + c < p.F) {
          const uint32_t q = s.off[__umulhi(w[it][c], nt)] + slot[it][c];
          s.key[q] = w[it][c];
          s.id[q] = int32_t(id0 + c);
        }
      }
    }
    __syncthreads();
    const uint32_t n = uint32_t(p.F - r0 < kRoundIds ? p.F - r0 : kRoundIds);
    for (uint32_t q = threadIdx.x; q < n; q += kChunkThreads) {
      const uint32_t k = s.key[q];
      const uint32_t b = __umulhi(k, nt);
      const uint32_t dst = s.base[b] + (q - s.off[b]);
      ko[dst] = k;
      io[dst] = s.id[q];
    }
    __syncthreads();
    if (threadIdx.x < nt) s.base[threadIdx.x] += s.cnt[threadIdx.x];
  }
}

// -- 5. split coarse buckets into fine buckets ---------------------------------
// A piece of 8K pairs of coarse bucket c per round: counting sort by fine
// bucket in LDS, then one contiguous run per fine bucket at a position taken
// from the bucket's cursor.
constexpr int kSplitThreads = 1024;
constexpr int kSplitItems = 8;
constexpr uint32_t kSplitPiece = kSplitThreads * kSplitItems;
constexpr uint32_t kMaxFine = 256;

struct SplitSmem {
  uint32_t key[kSplitPiece];
  int32_t id[kSplitPiece];
  uint32_t cnt[kMaxFine];
  uint32_t off[kMaxFine];
  uint32_t base[kMaxFine];
  uint32_t tmp[65];
};

__global__ void __launch_bounds__(kSplitThreads)
stream_split(StreamParams p, const uint32_t* __restrict__ start, uint32_t* __restrict__ cursor,
             const uint32_t* __restrict__ keys1, const int32_t* __restrict__ ids1,
             uint32_t* __restrict__ keys, int32_t* __restrict__ ids) {
  __shared__ SplitSmem s;
  const uint32_t nb = p.nb, nf = p.nf;
  const uint32_t c = blockIdx.y;
  const int64_t eoff = int64_t(blockIdx.z) * p.F;
  const uint32_t* st = start + int64_t(blockIdx.z) * (nb + 1);
  uint32_t* cur = cursor + int64_t(blockIdx.z) * nb;
  const uint32_t r0 = st[c * nf], r1 = st[(c + 1) * nf];
  for (uint32_t q0 = r0 + blockIdx.x * kSplitPiece; q0 < r1; q0 += gridDim.x * kSplitPiece) {
    for (uint32_t f = threadIdx.x; f < nf; f += kSplitThreads) s.cnt[f] = 0;
    __syncthreads();
    uint32_t k[kSplitItems], sl[kSplitItems];
    int32_t id[kSplitItems];
#pragma unroll
    for (int r = 0; r < kSplitItems; ++r) {
      const uint32_t q = q0 + r * kSplitThreads + threadIdx.x;
      if (q < r1) {
        k[r] = keys1[eoff + q];
        id[r] = ids1[eoff + q];
        sl[r] = atomicAdd(&s.cnt[__umulhi(k[r], nb) - c * nf], 1u);
      }
    }
    __syncthreads();
    {
      const uint32_t f = threadIdx.x;
      const uint32_t v = f < nf ? s.cnt[f] : 0u;
      uint32_t tot;
      const uint32_t ex = block_exclusive_scan(v, s.tmp, &tot);
      if (f < nf) {
        s.off[f] = ex;
        if (v) s.base[f] = atomicAdd(&cur[c * nf + f], v);
      }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSplitItems; ++r) {
      const uint32_t q = q0 + r * kSplitThreads + threadIdx.x;
      if (q < r1) {
        const uint32_t d = s.off[__umulhi(k[r], nb) - c * nf] + sl[r];
        s.key[d] = k[r];
        s.id[d] = id[r];
      }
    }
    __syncthreads();
    const uint32_t n = r1 - q0 < kSplitPiece ? r1 - q0 : kSplitPiece;
    for (uint32_t q = threadIdx.x; q < n; q += kSplitThreads) {
      const uint32_t kk = s.key[q];
      const uint32_t f = __umulhi(kk, nb) - c * nf;
      const uint32_t dst = s.base[f] + (q - s.off[f]);
      keys[eoff + dst] = kk;
      ids[eoff + dst] = s.id[q];
    }
    __syncthreads();
  }
}

// -- 6. per-bucket sort and shard --------------------------------------------
// 80 KB: two workgroups per CU. Digit counts and group starts are at most
// kSortCap (< 2^16), so they are kept as 16-bit halves of 32-bit words, and
// the scan's scratch lives in the pair array, which is unused until the
// pairs are placed.
struct SortSmem {
  uint2 kv[kSortCap];          // (key, id) pairs; later the sorted ids and the shard stage
  uint32_t hist[kDigits / 2];  // 16-bit digit counts, then group starts, two per word
};
static_assert(kSortCap < 65536, "16-bit digit counts");

__device__ __forceinline__ bool pair_greater(uint32_t ka, int32_t ia, uint32_t kb, int32_t ib) {
  return ka > kb || (ka == kb && ia > ib);
}

// In-place bitonic sort of n (key, id) pairs in global memory by one
// workgroup. Every merge starts with a "flip" comparator, so all comparators
// point the same way and the virtual padding (+inf beyond n) never moves.
__device__ void global_bitonic(uint32_t* gk, int32_t* gi, uint32_t n) {
  uint32_t P2 = 1;
  while (P2 < n) P2 <<= 1;
  for (uint32_t k = 2; k <= P2; k <<= 1) {
    for (uint32_t s = k >> 1; s >= 1; s >>= 1) {
      for (uint32_t t = threadIdx.x; t < P2 / 2; t += blockDim.x) {
        uint32_t i, j;
        if (s == (k >> 1)) {
          const uint32_t blk = t / s, off = t % s;
          i = blk * k + off;
          j = blk * k + k - 1 - off;
        } else {
          const uint32_t blk = t / s, off = t % s;
          i = blk * 2 * s + off;
          j = i + s;
        }
        if (j < n) {
          const uint32_t ka = gk[i], kb = gk[j];
          const int32_t ia = gi[i], ib = gi[j];
          if (pair_greater(ka, ia, kb, ib)) {
            gk[i] = kb; gi[i] = ib;
            gk[j] = ka; gi[j] = ia;
          }
        }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ int64_t row_offset(const StreamParams& p, uint32_t i, int64_t e) {
  const int64_t Li = p.drop_last ? p.L : epoch_len(p.F, p.N, p.B, 0, i);
  return int64_t(i) * p.M_max + (e - p.e_first) * Li;
}

__global__ void __launch_bounds__(kSortThreads)
stream_sort(StreamParams p, const uint32_t* __restrict__ start, uint32_t* __restrict__ keys,
            int32_t* __restrict__ ids, int32_t* __restrict__ R) {
  __shared__ SortSmem s;
  const uint32_t nb = p.nb;
  const uint32_t b = xcd_logical(blockIdx.x, gridDim.x);
  if (b >= nb) return;
  const int64_t e = int64_t(p.e0) + blockIdx.y;
  const uint32_t* st = start + int64_t(blockIdx.y) * (nb + 1);
  const uint32_t lo = st[b];
  const uint32_t n = st[b + 1] - lo;
  if (n == 0) return;
  uint32_t* gk = keys + int64_t(blockIdx.y) * p.F + lo;
  int32_t* gi = ids + int64_t(blockIdx.y) * p.F + lo;
  const uint32_t N = uint32_t(p.N);
  const int64_t pend64 = int64_t(lo) + n < p.P ? int64_t(lo) + n : p.P;

  if (n > uint32_t(p.cap)) {
    global_bitonic(gk, gi, n);
    for (int64_t q = threadIdx.x; int64_t(lo) + q < pend64; q += blockDim.x) {
      const uint32_t pp = lo + uint32_t(q);
      const uint32_t i = pp % N, j = pp / N;
      R[row_offset(p, i, e) + j] = gi[q];
    }
    return;
  }

  const uint32_t key_lo = uint32_t(((uint64_t(b) << 32) + nb - 1) / nb);
  const int db = p.sort_bits < kDigitBits ? p.sort_bits : kDigitBits;
  const int dshift = p.sort_bits - db;
  for (int x = threadIdx.x; x < kDigits / 2; x += kSortThreads) s.hist[x] = 0;
  const uint16_t* h16 = reinterpret_cast<const uint16_t*>(s.hist);  // digit d at [d]
  __syncthreads();
  // counting sort by the top bits of the key inside the bucket
  uint32_t k[kItems], slot[kItems];
  int32_t id[kItems];
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = uint32_t(r * kSortThreads) + threadIdx.x;
    if (q < n) {
      k[r] = gk[q] - key_lo;
      id[r] = gi[q];
    }
  }
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = uint32_t(r * kSortThreads) + threadIdx.x;
    if (q < n) {
      const uint32_t d = k[r] >> dshift;
      const uint32_t half = (d & 1u) * 16u;
      slot[r] = (atomicAdd(&s.hist[d >> 1], 1u << half) >> half) & 0xFFFFu;
    }
  }
  __syncthreads();
  {
    constexpr int kPerW = kDigits / 2 / kSortThreads;  // count words per thread
    uint32_t v[kPerW];
    uint32_t sum = 0;
#pragma unroll
    for (int j = 0; j < kPerW; ++j) {
      v[j] = s.hist[threadIdx.x * kPerW + j];
      sum += (v[j] & 0xFFFFu) + (v[j] >> 16);
    }
    uint32_t total;
    uint32_t ex = block_exclusive_scan(sum, reinterpret_cast<uint32_t*>(s.kv), &total);
#pragma unroll
    for (int j = 0; j < kPerW; ++j) {
      const uint32_t lo16 = ex;
      ex += v[j] & 0xFFFFu;
      s.hist[threadIdx.x * kPerW + j] = lo16 | (ex << 16);
      ex += v[j] >> 16;
    }
  }
  __syncthreads();
  uint32_t dst[kItems];
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = uint32_t(r * kSortThreads) + threadIdx.x;
    if (q < n) {
      dst[r] = h16[k[r] >> dshift] + slot[r];
      s.kv[dst[r]] = make_uint2(k[r], uint32_t(id[r]));
    }
  }
  __syncthreads();
  // Inside its digit group (a few pairs), every pair's final position is
  // the group start plus the number of group pairs ordered before it by
  // (key, id); the loads of one pair's scan do not depend on each other.
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = uint32_t(r * kSortThreads) + threadIdx.x;
    if (q < n) {
      const uint32_t d = k[r] >> dshift;
      const uint32_t a0 = h16[d];
      const uint32_t a1 = d + 1 < uint32_t(kDigits) ? h16[d + 1] : n;
      uint32_t rank = 0;
      for (uint32_t v = a0; v < a1; ++v) {
        const uint2 o = s.kv[v];
        rank += pair_greater(k[r], id[r], o.x, int32_t(o.y));
      }
      dst[r] = a0 + rank;
    }
  }
  __syncthreads();
  int32_t* sorted = reinterpret_cast<int32_t*>(s.kv);  // ids in (key, id) order
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = uint32_t(r * kSortThreads) + threadIdx.x;
    if (q < n) sorted[dst[r]] = id[r];
  }
  __syncthreads();

  if (pend64 <= int64_t(lo)) return;
  const uint32_t pend = uint32_t(pend64);
  const uint32_t j0 = lo / N, j1 = (pend - 1) / N;
  const uint32_t nj = j1 - j0 + 1;
  const uint32_t Np = (N & 1u) ? N : N + 1u;  // odd row pitch: conflict-free columns
  // (j, i) of position lo + threadIdx.x, stepped by kSortThreads positions
  // per iteration without dividing
  const uint32_t step_i = kSortThreads % N, step_j = kSortThreads / N;
  uint32_t ci = (lo + threadIdx.x) % N, cj = (lo + threadIdx.x) / N;
  if (uint64_t(nj) * Np <= uint64_t(kSortCap)) {
    uint32_t* stage = reinterpret_cast<uint32_t*>(s.kv) + kSortCap;
    for (uint32_t q = threadIdx.x; lo + q < pend; q += kSortThreads) {
      stage[(cj - j0) * Np + ci] = uint32_t(sorted[q]);
      ci += step_i;
      cj += step_j;
      if (ci >= N) {
        ci -= N;
        ++cj;
      }
    }
    __syncthreads();
    // t -> (row i, column jj) with consecutive t on consecutive columns of a
    // row; t < 2^13, so the float reciprocal gives t / nj up to one step
    const uint32_t total = nj * N;
    const float inv_nj = 1.0f / float(nj);
    auto write = [&](auto row) {
      for (uint32_t t = threadIdx.x; t < total; t += kSortThreads) {
        uint32_t i = uint32_t(float(t) * inv_nj);
        if (i * nj > t) --i;
        else if ((i + 1) * nj <= t) ++i;
        const uint32_t jj = t - i * nj;
        const uint32_t pp = (j0 + jj) * N + i;
        if (pp >= lo && pp < pend) row(i)[jj] = int32_t(stage[jj * Np + i]);
      }
    };
    if (p.drop_last) {  // every row holds L reads per epoch: one offset for all rows
      int32_t* const Re = R + (e - p.e_first) * p.L + j0;
      write([&](uint32_t i) { return Re + int64_t(i) * p.M_max; });
    } else {
      write([&](uint32_t i) { return R + row_offset(p, i, e) + j0; });
    }
  } else {
    for (uint32_t q = threadIdx.x; lo + q < pend; q += kSortThreads) {
      R[row_offset(p, ci, e) + cj] = sorted[q];
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
  int64_t nb64 = ceil_div(s.F, cap * 3 / 4 > 0 ? cap * 3 / 4 : 1);
  if (nb64 < 1) nb64 = 1;
  if (nb64 > int64_t(kMaxBuckets)) nb64 = kMaxBuckets;
  // coarse buckets: at most 64 per epoch, nf fine buckets each
  const uint32_t nb1 = uint32_t(nb64 < 64 ? nb64 : 64);
  const uint32_t nf = uint32_t(ceil_div(nb64, nb1));
  const uint32_t nb = nb1 * nf;
  const uint64_t width = ((uint64_t(1) << 32) + nb - 1) / nb;
  int bits = 0;
  while ((uint64_t(1) << bits) < width) ++bits;

  StreamParams p;
  p.F = s.F; p.N = s.N; p.B = s.B; p.P = s.P; p.L = s.L; p.M_max = s.M_max;
  p.drop_last = s.drop_last;
  p.seed_lo = uint32_t(s.seed);
  p.seed_hi = uint32_t(s.seed >> 32);
  p.nb = nb;
  p.nb1 = nb1;
  p.nf = nf;
  p.sort_bits = bits;
  p.cap = int32_t(cap);
  p.e_first = e_begin;

  // epochs per batch: the pair arrays of a batch stay under ~16 GB of scratch
  const int64_t budget = int64_t(16) << 30;
  int64_t EB = budget / ((nf > 1 ? 16 : 8) * s.F);
  if (EB < 1) EB = 1;
  if (EB > s.E) EB = s.E;

  const uint32_t nchunks = uint32_t(ceil_div(s.F, kChunkIds));
  Scratch scr(st);
  uint32_t *keys, *keys1 = nullptr, *cnt, *tot, *start, *cursor;
  int32_t *ids, *ids1 = nullptr;
  if ((rc = scr.alloc_n(&keys, size_t(EB * s.F)))) return rc;
  if ((rc = scr.alloc_n(&ids, size_t(EB * s.F)))) return rc;
  if (nf > 1) {
    if ((rc = scr.alloc_n(&keys1, size_t(EB * s.F)))) return rc;
    if ((rc = scr.alloc_n(&ids1, size_t(EB * s.F)))) return rc;
  }
  if ((rc = scr.alloc_n(&cnt, size_t(EB) * nchunks * nb))) return rc;
  if ((rc = scr.alloc_n(&tot, size_t(EB * nb)))) return rc;
  if ((rc = scr.alloc_n(&start, size_t(EB * (nb + 1))))) return rc;
  if ((rc = scr.alloc_n(&cursor, size_t(EB * nb)))) return rc;
  // pieces per coarse bucket for the split: about 1.25x the mean size
  const uint32_t pieces = uint32_t(ceil_div(ceil_div(s.F, nb1) * 5 / 4, kSplitPiece));

  for (int64_t e0 = 0; e0 < s.E; e0 += EB) {
    const uint32_t eb = uint32_t(e0 + EB <= s.E ? EB : s.E - e0);
    p.e0 = int32_t(e_begin + e0);
    if ((rc = launch("stream_count", stream_count, dim3(nchunks, eb), dim3(kChunkThreads),
                     size_t(nb) * 4, st, p, nchunks, cnt)))
      return rc;
    if ((rc = launch("stream_offsets", stream_offsets, dim3(uint32_t(ceil_div(nb, 256)), eb),
                     dim3(256), 0, st, nb, nchunks, cnt, tot)))
      return rc;
    if ((rc = launch("stream_scan", stream_scan, dim3(eb), dim3(1024), 0, st, nb,
                     (const uint32_t*)tot, start, cursor)))
      return rc;
    if ((rc = launch("stream_scatter", stream_scatter, dim3(xcd_padded(nchunks), eb),
                     dim3(kChunkThreads), 0, st, p, nchunks, (const uint32_t*)cnt,
                     (const uint32_t*)start, nf > 1 ? keys1 : keys, nf > 1 ? ids1 : ids)))
      return rc;
    if (nf > 1) {
      if ((rc = launch("stream_split", stream_split, dim3(pieces, nb1, eb), dim3(kSplitThreads),
                       0, st, p, (const uint32_t*)start, cursor,
                       (const uint32_t*)keys1, (const int32_t*)ids1, keys, ids)))
        return rc;
    }
    if ((rc = launch("stream_sort", stream_sort, dim3(xcd_padded(nb), eb), dim3(kSortThreads), 0, st,
                     p, (const uint32_t*)start, keys, ids, R)))
      return rc;
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
