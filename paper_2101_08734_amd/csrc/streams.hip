// nopfs_access_streams: every worker's access stream for every epoch.
//
// Section 2 of the paper: an epoch is a random shuffle of all sample ids and
// the seed reproduces it. Section 4: each global batch is partitioned among
// the N workers and a worker's stream R is the concatenation of its batches.
//
// Epoch e orders the samples by (key_e(k), k), key_e(k) a Philox-4x32-10
// word. The order is built as a two-level radix sort over all epochs of a
// batch at once:
//   1. stream_count   -- Philox keys in registers, histogram of the bucket
//                        umulhi(key, nb) per epoch (LDS-privatised).
//   2. stream_scan    -- bucket start positions per epoch.
//   3. stream_scatter -- keys regenerated, (key, id) pairs written into their
//                        bucket (order inside a bucket is arbitrary).
//   4. stream_sort    -- one workgroup per bucket: LSD radix sort of the
//                        bucket in LDS, ranked with wavefront ballots (8-bit
//                        digits), equal keys put back in id order, and the
//                        sorted positions p sharded straight into R:
//                        R[p mod N][e*L_i + p div N]. The write goes through
//                        an LDS transpose so each worker row gets a run.
// Buckets larger than the LDS capacity (not expected for uniform keys, but
// possible in principle) are sorted in place in global memory by a bitonic
// network inside the same workgroup.
#include <limits.h>

#include "common.hpp"
#include "philox.hpp"

namespace nopfs {
namespace {

constexpr int kChunkThreads = 256;
constexpr int kBlocksPerThread = 16;                                   // Philox blocks
constexpr int64_t kChunkIds = int64_t(kChunkThreads) * kBlocksPerThread * 4;  // 16384
constexpr uint32_t kMaxBuckets = 8192;

constexpr int kSortThreads = 512;
constexpr int kSortWaves = kSortThreads / 64;
constexpr int kItems = 16;
constexpr int kSortCap = kSortThreads * kItems;  // 8192 (key, id) pairs in LDS
constexpr int kDigits = 256;

struct StreamParams {
  int64_t F, N, B, P, L, M_max;
  int32_t drop_last;
  uint32_t seed_lo, seed_hi;
  uint32_t nb;        // buckets per epoch
  int32_t e0;         // first epoch of the batch
  int32_t sort_bits;  // significant bits of a key inside its bucket
  int32_t cap;        // largest bucket sorted in LDS
};

__global__ void fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (; i < n; i += stride) p[i] = v;
}

// -- 1. histogram of buckets ------------------------------------------------
__global__ void __launch_bounds__(kChunkThreads)
stream_count(StreamParams p, uint32_t* __restrict__ tot) {
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
  uint32_t* t = tot + int64_t(blockIdx.y) * nb;
  for (uint32_t b = threadIdx.x; b < nb; b += blockDim.x)
    if (hist[b]) atomicAdd(&t[b], hist[b]);
}

// -- 2. bucket starts --------------------------------------------------------
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

// -- 3. scatter into buckets -------------------------------------------------
__global__ void __launch_bounds__(kChunkThreads)
stream_scatter(StreamParams p, uint32_t nchunks, uint32_t* __restrict__ cursor,
               uint32_t* __restrict__ keys, int32_t* __restrict__ ids) {
  extern __shared__ uint32_t smem[];
  const uint32_t nb = p.nb;
  uint32_t* cnt = smem;
  uint32_t* base = smem + nb;
  const uint32_t chunk = xcd_logical(blockIdx.x, gridDim.x);
  if (chunk >= nchunks) return;
  for (uint32_t b = threadIdx.x; b < nb; b += blockDim.x) cnt[b] = 0;
  __syncthreads();
  const uint32_t e = uint32_t(p.e0) + blockIdx.y;
  const int64_t blk0 = int64_t(chunk) * (kChunkIds / 4);
  uint32_t kr[kBlocksPerThread][4];
#pragma unroll
  for (int it = 0; it < kBlocksPerThread; ++it) {
    const int64_t blk = blk0 + it * kChunkThreads + threadIdx.x;
    const int64_t id0 = blk * 4;
    if (id0 < p.F) {
      const Philox4 r = philox_block(uint32_t(blk), e, p.seed_lo, p.seed_hi);
      kr[it][0] = r.x; kr[it][1] = r.y; kr[it][2] = r.z; kr[it][3] = r.w;
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (id0 + c < p.F) atomicAdd(&cnt[__umulhi(kr[it][c], nb)], 1u);
    }
  }
  __syncthreads();
  uint32_t* cur = cursor + int64_t(blockIdx.y) * nb;
  for (uint32_t b = threadIdx.x; b < nb; b += blockDim.x) {
    const uint32_t c = cnt[b];
    if (c) base[b] = atomicAdd(&cur[b], c);
    cnt[b] = 0;
  }
  __syncthreads();
  uint32_t* ko = keys + int64_t(blockIdx.y) * p.F;
  int32_t* io = ids + int64_t(blockIdx.y) * p.F;
#pragma unroll
  for (int it = 0; it < kBlocksPerThread; ++it) {
    const int64_t blk = blk0 + it * kChunkThreads + threadIdx.x;
    const int64_t id0 = blk * 4;
    if (id0 < p.F) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (id0 + c < p.F) {
          const uint32_t key = kr[it][c];
          const uint32_t b = __umulhi(key, nb);
          const uint32_t dst = base[b] + atomicAdd(&cnt[b], 1u);
          ko[dst] = key;
          io[dst] = int32_t(id0 + c);
        }
      }
    }
  }
}

// -- 4. per-bucket sort and shard --------------------------------------------
struct SortSmem {
  uint32_t keys[kSortCap];
  int32_t ids[kSortCap];
  uint32_t cnt[kDigits * kSortWaves];
  uint32_t tmp[65];
};

// One stable counting-sort pass over an 8-bit digit. Items live in registers
// in wave-striped order: item r of lane l in wave w has local index
// (w*kItems + r)*64 + l, which is also the stability order. Within a wave,
// lanes holding the same digit are found with 8 ballots; per-wave running
// counters in LDS give each item its rank among equal digits of its wave.
__device__ __forceinline__ void rank_pass(uint32_t (&k)[kItems], int32_t (&id)[kItems], int shift,
                                          SortSmem& s) {
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < kDigits * kSortWaves; i += kSortThreads) s.cnt[i] = 0;
  __syncthreads();
  const uint64_t lt = lanemask_lt();
  uint32_t rank[kItems];
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t d = (k[r] >> shift) & 0xFFu;
    uint64_t m = ~0ull;
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool set = (d >> bit) & 1u;
      const uint64_t bb = __ballot(set);
      m &= set ? bb : ~bb;
    }
    uint32_t* c = &s.cnt[d * kSortWaves + wave];
    const uint32_t before = *c;
    rank[r] = before + uint32_t(__popcll(m & lt));
    if ((m >> lane) == 1ull) *c = before + uint32_t(__popcll(m));
  }
  __syncthreads();
  // exclusive scan of the counters in (digit, wave) order
  constexpr int kPer = kDigits * kSortWaves / kSortThreads;
  uint32_t v[kPer];
  uint32_t sum = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    v[j] = s.cnt[threadIdx.x * kPer + j];
    sum += v[j];
  }
  uint32_t total;
  uint32_t ex = block_exclusive_scan(sum, s.tmp, &total);
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    s.cnt[threadIdx.x * kPer + j] = ex;
    ex += v[j];
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t d = (k[r] >> shift) & 0xFFu;
    const uint32_t dst = s.cnt[d * kSortWaves + wave] + rank[r];
    s.keys[dst] = k[r];
    s.ids[dst] = id[r];
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int q = (wave * kItems + r) * 64 + lane;
    k[r] = s.keys[q];
    id[r] = s.ids[q];
  }
  __syncthreads();
}

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
  return int64_t(i) * p.M_max + e * Li;
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
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  uint32_t k[kItems];
  int32_t id[kItems];
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const uint32_t q = uint32_t((wave * kItems + r) * 64 + lane);
    if (q < n) {
      k[r] = gk[q] - key_lo;
      id[r] = gi[q];
    } else {
      k[r] = 0xFFFFFFFFu;  // padding sorts last (it starts last and passes are stable)
      id[r] = INT_MAX;
    }
  }
  for (int shift = 0; shift < p.sort_bits; shift += 8) rank_pass(k, id, shift, s);

  // equal keys: restore ascending id order inside each run of ties
  for (uint32_t q = threadIdx.x; q + 1 < n; q += kSortThreads) {
    if (s.keys[q] == s.keys[q + 1] && (q == 0 || s.keys[q - 1] != s.keys[q])) {
      uint32_t end = q + 2;
      while (end < n && s.keys[end] == s.keys[q]) ++end;
      for (uint32_t a = q + 1; a < end; ++a) {
        const int32_t v = s.ids[a];
        uint32_t c = a;
        while (c > q && s.ids[c - 1] > v) {
          s.ids[c] = s.ids[c - 1];
          --c;
        }
        s.ids[c] = v;
      }
    }
  }
  __syncthreads();

  if (pend64 <= int64_t(lo)) return;
  const uint32_t pend = uint32_t(pend64);
  const uint32_t j0 = lo / N, j1 = (pend - 1) / N;
  const uint32_t nj = j1 - j0 + 1;
  const uint32_t Np = (N & 1u) ? N : N + 1u;  // odd row pitch: conflict-free columns
  if (uint64_t(nj) * Np <= uint64_t(kSortCap)) {
    uint32_t* stage = s.keys;
    for (uint32_t q = threadIdx.x; lo + q < pend; q += kSortThreads) {
      const uint32_t pp = lo + q;
      stage[(pp / N - j0) * Np + pp % N] = uint32_t(s.ids[q]);
    }
    __syncthreads();
    const uint32_t total = nj * N;
    for (uint32_t t = threadIdx.x; t < total; t += kSortThreads) {
      const uint32_t i = t / nj, jj = t - i * nj;
      const uint32_t pp = (j0 + jj) * N + i;
      if (pp >= lo && pp < pend) R[row_offset(p, i, e) + j0 + jj] = int32_t(stage[jj * Np + i]);
    }
  } else {
    for (uint32_t q = threadIdx.x; lo + q < pend; q += kSortThreads) {
      const uint32_t pp = lo + q;
      const uint32_t i = pp % N, j = pp / N;
      R[row_offset(p, i, e) + j] = s.ids[q];
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

int streams_impl(const nopfs_job* job, int32_t* R, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (s.M_max == 0) return NOPFS_OK;  // no reads: R has no elements and may be NULL
  if (!R) return fail(NOPFS_EINVAL, "R is NULL");

  int64_t cap = kSortCap;
  if (debug_value(1) > 0 && debug_value(1) < cap) cap = debug_value(1);
  int64_t nb64 = ceil_div(s.F, cap * 3 / 4 > 0 ? cap * 3 / 4 : 1);
  if (nb64 < 1) nb64 = 1;
  if (nb64 > int64_t(kMaxBuckets)) nb64 = kMaxBuckets;
  const uint32_t nb = uint32_t(nb64);
  const uint64_t width = ((uint64_t(1) << 32) + nb - 1) / nb;
  int bits = 0;
  while ((uint64_t(1) << bits) < width) ++bits;

  StreamParams p;
  p.F = s.F; p.N = s.N; p.B = s.B; p.P = s.P; p.L = s.L; p.M_max = s.M_max;
  p.drop_last = s.drop_last;
  p.seed_lo = uint32_t(s.seed);
  p.seed_hi = uint32_t(s.seed >> 32);
  p.nb = nb;
  p.sort_bits = bits;
  p.cap = int32_t(cap);

  // epochs per batch: keys + ids of a batch stay under ~6 GB of scratch
  const int64_t budget = int64_t(6) << 30;
  int64_t EB = budget / (8 * s.F);
  if (EB < 1) EB = 1;
  if (EB > s.E) EB = s.E;

  Scratch scr(st);
  uint32_t *keys, *tot, *start, *cursor;
  int32_t* ids;
  if ((rc = scr.alloc_n(&keys, size_t(EB * s.F)))) return rc;
  if ((rc = scr.alloc_n(&ids, size_t(EB * s.F)))) return rc;
  if ((rc = scr.alloc_n(&tot, size_t(EB * nb)))) return rc;
  if ((rc = scr.alloc_n(&start, size_t(EB * (nb + 1))))) return rc;
  if ((rc = scr.alloc_n(&cursor, size_t(EB * nb)))) return rc;

  const uint32_t nchunks = uint32_t(ceil_div(s.F, kChunkIds));
  for (int64_t e0 = 0; e0 < s.E; e0 += EB) {
    const uint32_t eb = uint32_t(e0 + EB <= s.E ? EB : s.E - e0);
    p.e0 = int32_t(e0);
    if ((rc = launch("fill_u32", fill_u32, dim3(uint32_t(ceil_div(eb * nb, 256))), dim3(256), 0, st,
                     tot, int64_t(eb) * nb, 0u)))
      return rc;
    if ((rc = launch("stream_count", stream_count, dim3(nchunks, eb), dim3(kChunkThreads),
                     size_t(nb) * 4, st, p, tot)))
      return rc;
    if ((rc = launch("stream_scan", stream_scan, dim3(eb), dim3(1024), 0, st, nb, tot, start, cursor)))
      return rc;
    if ((rc = launch("stream_scatter", stream_scatter, dim3(xcd_padded(nchunks), eb),
                     dim3(kChunkThreads), size_t(nb) * 8, st, p, nchunks, cursor, keys, ids)))
      return rc;
    if ((rc = launch("stream_sort", stream_sort, dim3(xcd_padded(nb), eb), dim3(kSortThreads), 0, st,
                     p, start, keys, ids, R)))
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
    return nopfs::streams_impl(job, R, static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}
