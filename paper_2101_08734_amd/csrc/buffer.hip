// nopfs_buffer_sim: a clairvoyant buffer of d0 bytes per worker (the
// replacement rules of the I/O Access Patterns section: discard the sample
// whose next use is furthest in the future, and never one used before the
// sample being brought in).
//
// The buffer holds samples keyed by the stream position of their next use,
// so the read at position f hits exactly when key f is held. After a read
// with a next use n the sample is (re)admitted under key n, then, while the
// held bytes exceed d0, the furthest key is discarded (possibly n itself).
// The size of the sample held under key x is that of the sample read at x.
// The replay is sequential per worker and the workers are independent.
//
//   bs_sizes -- every position's sample size, sizes[R[f]], in parallel, so
//               the replay reads sizes with plain coalesced loads.
//   bs_sim   -- one wave per worker. Held keys in a three-level bitmap: a
//               bit per position in 64-bit words in global memory, one word
//               per batch of 64 reads, changed and read only by lane 0's
//               atomics so it is always current; a bit per nonzero word, and
//               a bit per nonzero word of that, in LDS. A batch of 64 reads
//               arrives one per lane (sizes, next uses and the batch's word
//               loaded a batch ahead, with changes to that word made meanwhile
//               kept as set and clear masks); only the reads that can change
//               anything are visited, in order: those whose key is held (a
//               hit) and those with a next use that fits (an admission).
//               The top word, the highest word holding a key, lives in
//               registers with the size of each of its keys in the lane of
//               its bit: the furthest key is discarded from there, and only
//               when that word empties is the next one found through the LDS
//               levels and loaded. An admission above the top key that does
//               not fit is a bypass and touches nothing.
#include <algorithm>
#include <new>

#include "common.hpp"

namespace nopfs {
namespace {

constexpr int kBsMaxLog = 24;                          // positions per worker: < 2^24
constexpr int kBsW1 = (1 << kBsMaxLog) / 64 / 32;      // level-1 words: 8192
constexpr int kBsW2 = kBsW1 / 32;                      // level-2 words: 256

struct BsShape {
  int64_t F, N, B, M_max, E;
  int32_t drop_last;
};

__device__ __forceinline__ int64_t bs_row_len(const BsShape& r, int64_t i) {
  return r.E * epoch_len(r.F, r.N, r.B, r.drop_last, i);
}

__device__ __forceinline__ int64_t rl64(int64_t v, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane(uint32_t(uint64_t(v)), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(uint32_t(uint64_t(v) >> 32), lane);
  return int64_t((uint64_t(hi) << 32) | lo);
}

__device__ __forceinline__ uint64_t rfl64(uint64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(v >> 32));
  return (uint64_t(hi) << 32) | lo;
}

__device__ __forceinline__ int hi_bit(uint32_t v) { return 31 - __builtin_clz(v); }
__device__ __forceinline__ int hi_bit64(uint64_t v) { return 63 - __builtin_clzll(v); }

__device__ __forceinline__ uint64_t l0_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// z[i][f] = sizes[R[i][f]] for f < M_i (0 for an id outside [0, F))
__global__ void __launch_bounds__(256)
bs_sizes(BsShape r, const int32_t* __restrict__ R, const int64_t* __restrict__ sizes,
         int64_t* __restrict__ z) {
  for (int64_t i = blockIdx.y; i < r.N; i += gridDim.y) {
    const int64_t Mi = bs_row_len(r, i);
    const int32_t* Rr = R + i * r.M_max;
    int64_t* zr = z + i * r.M_max;
    // four independent reads in flight per thread
    const int64_t S = int64_t(gridDim.x) * blockDim.x;
    for (int64_t f = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; f < Mi; f += 4 * S) {
      int32_t k[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) k[u] = f + u * S < Mi ? Rr[f + u * S] : -1;
      int64_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = (k[u] >= 0 && k[u] < r.F) ? sizes[k[u]] : 0;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (f + u * S < Mi) zr[f + u * S] = v[u];
    }
  }
}

__global__ void __launch_bounds__(64)
bs_sim(BsShape r, const int32_t* __restrict__ next, const int64_t* __restrict__ z, int64_t d0,
       uint64_t* __restrict__ L0, int8_t* __restrict__ hit, int64_t* __restrict__ hits) {
  __shared__ uint32_t l1[kBsW1];
  __shared__ uint32_t l2[kBsW2];
  const int64_t i = blockIdx.x;
  const int lane = threadIdx.x;
  const int64_t Mi = bs_row_len(r, i);
  const int64_t W0 = (r.M_max + 63) >> 6;
  const int64_t W1 = (W0 + 31) >> 5;
  const int64_t W2 = (W1 + 31) >> 5;
  uint64_t* l0 = L0 + i * W0;
  const int32_t* Xr = next + i * r.M_max;
  const int64_t* zr = z + i * r.M_max;
  int8_t* hrow = hit + i * r.M_max;
  for (int64_t w = lane; w < W0; w += 64) l0[w] = 0u;
  for (int64_t w = lane; w < W1; w += 64) l1[w] = 0u;
  for (int64_t w = lane; w < W2; w += 64) l2[w] = 0u;
  __threadfence();  // the cleared words reach L2 before the atomics below
  __syncthreads();

  int64_t used = 0, hc = 0, hb = 0;
  // top word (-1: nothing held), its bits, lane b: size of key 64 tw + b
  int64_t tw = -1;
  uint64_t tv = 0;
  int64_t zs = 0;

  // clears the level bits above a level-0 word that has become zero
  auto word_emptied = [&](int64_t w) {
    if (lane == 0) {
      const int64_t a = w >> 5;
      const uint32_t v1 = atomicAnd(&l1[a], ~(1u << (w & 31))) & ~(1u << (w & 31));
      if (v1 == 0u) atomicAnd(&l2[a >> 5], ~(1u << (a & 31)));
    }
  };
  // finds the highest word holding a key and loads it with its sizes
  auto descend = [&]() {
    int64_t w2 = -1;
    for (int64_t base = ((W2 - 1) >> 6) << 6; base >= 0; base -= 64) {
      const int64_t idx = base + lane;
      const uint32_t v = idx < W2 ? l2[idx] : 0u;
      const uint64_t b = __ballot(v != 0u);
      if (b) {
        w2 = base + (63 - __builtin_clzll(b));
        break;
      }
    }
    tw = -1;
    tv = 0;
    if (w2 < 0) return;
    const int64_t w1 = (w2 << 5) + hi_bit(l2[w2]);
    const uint32_t v1 = l1[w1];
    if (v1 == 0u) return;  // cannot happen: the level bits mirror level 0
    const int64_t w0 = (w1 << 5) + hi_bit(v1);
    uint64_t v0 = 0;
    if (lane == 0) v0 = l0_load(&l0[w0]);
    const int64_t x = (w0 << 6) + lane;
    zs = x < Mi ? zr[x] : 0;
    v0 = rfl64(v0);
    // the sizes are complete here, so later reads of zs wait for nothing
    __builtin_amdgcn_s_waitcnt(0);
    if (v0 == 0u) return;  // cannot happen either
    tw = w0;
    tv = v0;
  };

  // the next batch: sizes, next uses, lane 0's copy of its word, and the
  // changes made to that word since it was loaded
  int64_t sN = lane < Mi ? zr[lane] : 0;
  int32_t nN = lane < Mi ? Xr[lane] : -1;
  uint64_t hN = 0, nset = 0, nclr = 0;  // every word starts empty
  for (int64_t f0 = 0, b = 0; f0 < Mi; f0 += 64, ++b) {
    const int64_t f = f0 + lane;
    const int64_t s = sN;
    int32_t nx = nN;
    if (nx <= f || nx >= Mi) nx = -1;
    uint64_t hw = (rfl64(hN) & ~nclr) | nset;  // held keys among this batch's positions
    const uint64_t cand = __ballot(nx >= 0 && s <= d0);
    nset = nclr = 0;
    hN = 0;
    {  // the next batch's loads, after this batch's values are in use
      const int64_t g = f + 64;
      sN = g < Mi ? zr[g] : 0;
      nN = g < Mi ? Xr[g] : -1;
      if (lane == 0 && b + 1 < W0) hN = l0_load(&l0[b + 1]);
    }
    uint64_t mask = cand | hw;
    uint64_t hm = 0;
    while (mask) {
      const int q = __builtin_ctzll(mask);
      const uint64_t bit = uint64_t(1) << q;
      mask &= ~bit;
      const int64_t sq = rl64(s, q);
      if (hw & bit) {  // key f0 + q held: a hit, and its entry ends here
        hc += 1;
        hb += sq;
        hm |= bit;
        used -= sq;
        hw &= ~bit;
        if (lane == 0) atomicAnd(reinterpret_cast<unsigned long long*>(&l0[b]), ~bit);
        if (b == tw) tv = hw;
        if (hw == 0u) {
          word_emptied(b);
          if (b == tw) descend();
        }
      }
      if (!(cand & bit)) continue;
      const int32_t nq = __builtin_amdgcn_readlane(nx, q);
      const int64_t top = tw >= 0 ? (tw << 6) + hi_bit64(tv) : -1;
      if (nq > top && sq > d0 - used) continue;  // the furthest and it does not fit: bypass
      {  // admit under the next use
        const int64_t w = nq >> 6;
        const uint64_t bn = uint64_t(1) << (nq & 63);
        if (lane == 0) {
          atomicOr(reinterpret_cast<unsigned long long*>(&l0[w]), bn);
          atomicOr(&l1[w >> 5], 1u << (w & 31));
          atomicOr(&l2[w >> 10], 1u << ((w >> 5) & 31));
        }
        if (w == b) {  // a later read of this batch
          hw |= bn;
          mask |= bn;
        } else if (w == b + 1) {
          nset |= bn;
          nclr &= ~bn;
        }
        if (w > tw) {  // every word above the top is empty
          tw = w;
          tv = 0;
        }
        if (w == tw) {
          tv |= bn;
          if (lane == (nq & 63)) zs = sq;
        }
        used += sq;
      }
      // discard the furthest while over capacity
      while (used > d0) {
        if (tw < 0) {  // nothing held (only if sizes break the precondition)
          used = 0;
          break;
        }
        const int xb = hi_bit64(tv);
        const uint64_t bx = uint64_t(1) << xb;
        used -= rl64(zs, xb);
        tv &= ~bx;
        if (lane == 0) atomicAnd(reinterpret_cast<unsigned long long*>(&l0[tw]), ~bx);
        if (tw == b) {
          hw &= ~bx;
        } else if (tw == b + 1) {
          nclr |= bx;
          nset &= ~bx;
        }
        if (tv == 0u) {
          word_emptied(tw);
          descend();
        }
      }
    }
    if (f < Mi) hrow[f] = int8_t((hm >> lane) & 1u);
  }
  for (int64_t f = Mi + lane; f < r.M_max; f += 64) hrow[f] = -1;
  if (lane == 0) {
    hits[i * 2] = hc;
    hits[i * 2 + 1] = hb;
  }
}

int buffer_impl(const nopfs_job* job, const int32_t* R, const int32_t* next, const int64_t* sizes,
                int64_t d0, int8_t* hit, int64_t* hits, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (!sizes || !hits) return fail(NOPFS_EINVAL, "sizes and hits must be non-NULL");
  if (d0 < 0) return fail(NOPFS_EINVAL, "d0 must be >= 0");
  if (s.M_max > 0 && (!R || !next || !hit)) return fail(NOPFS_EINVAL, "R, next and hit must be non-NULL");
  if (s.M_max >= (int64_t(1) << kBsMaxLog)) return fail(NOPFS_ERANGE, "M_max must be < 2^24");
  if (s.N >= (int64_t(1) << 31)) return fail(NOPFS_ERANGE, "N too large for one launch");
  BsShape r{s.F, s.N, s.B, s.M_max, s.E, s.drop_last};
  const int64_t W0 = (s.M_max + 63) >> 6;
  Scratch scr(st);
  uint64_t* L0;
  int64_t* z;
  if ((rc = scr.alloc_n(&L0, size_t(s.N * W0)))) return rc;
  if ((rc = scr.alloc_n(&z, size_t(s.N * s.M_max)))) return rc;
  if (s.M_max > 0) {
    const int64_t bx = std::min<int64_t>((s.M_max + 1023) / 1024, 64);
    const int64_t by = std::min<int64_t>(s.N, 65535);
    if ((rc = launch("bs_sizes", bs_sizes, dim3(uint32_t(bx), uint32_t(by)), dim3(256), 0, st, r,
                     R, sizes, z)))
      return rc;
  }
  return launch("bs_sim", bs_sim, dim3(uint32_t(s.N)), dim3(64), 0, st, r, next, z, d0, L0, hit,
                hits);
}

}  // namespace
}  // namespace nopfs

extern "C" int nopfs_buffer_sim(const nopfs_job* job, const int32_t* R, const int32_t* next,
                                const int64_t* sizes, int64_t d0, int8_t* hit, int64_t* hits,
                                void* hip_stream) {
  try {
    return nopfs::buffer_impl(job, R, next, sizes, d0, hit, hits,
                              static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}
