// nopfs_buffer_sim: a clairvoyant buffer of d0 bytes per worker (the
// replacement rules of the I/O Access Patterns section: discard the sample
// whose next use is furthest in the future, and never one used before the
// sample being brought in).
//
// The buffer holds samples keyed by the stream position of their next use,
// so the read at position f hits exactly when key f is held. After a read
// with a next use n the sample is (re)admitted under key n, then, while the
// held bytes exceed d0, the furthest key is discarded (possibly n itself).
// The size of the sample held under key x is that of the sample read at x,
// sizes[R[x]].
// The replay is sequential per worker and the workers are independent.
//
//   bs_sim   -- one wave per worker. Held keys in a three-level bitmap: a
//               bit per position in 64-bit words in global memory, one word
//               per batch of 64 reads, changed and read only by atomics so it
//               is always current; a bit per word that may hold keys, and a
//               bit per such level-1 word, in LDS. A batch of 64 reads
//               arrives one per lane (ids and next uses loaded two batches
//               ahead, sizes gathered and the batch's word loaded one ahead,
//               with changes to that word made meanwhile kept as set and
//               clear masks); only the reads that can change
//               anything are visited, in order: those whose key is held (a
//               hit) and those with a next use that fits (an admission). The
//               highest held keys (up to 64) live in registers, ascending
//               across the lanes with their sizes: the furthest key is
//               discarded from there, an admitted key above the lowest cached
//               one joins in order, and an admission above the highest that
//               does not fit is a bypass that touches nothing. Only when the
//               cache empties are the highest keys gathered again from the two
//               highest level-1 words, one word per lane (discards do not
//               clear level bits; words found empty clear theirs then).

#include <algorithm>
#include <climits>
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

// whole-wave lane shifts: lane i takes lane i + 1 (shl1) or lane i - 1
// (shr1); the lane with no source keeps `edge`
__device__ __forceinline__ int32_t shl1(int32_t v, int32_t edge) {
  return __builtin_amdgcn_update_dpp(edge, v, 0x130, 0xf, 0xf, false);
}
__device__ __forceinline__ int32_t shr1(int32_t v, int32_t edge) {
  return __builtin_amdgcn_update_dpp(edge, v, 0x138, 0xf, 0xf, false);
}
__device__ __forceinline__ int64_t shl1_64(int64_t v) {
  const uint32_t lo = uint32_t(shl1(int32_t(uint32_t(uint64_t(v))), 0));
  const uint32_t hi = uint32_t(shl1(int32_t(uint32_t(uint64_t(v) >> 32)), 0));
  return int64_t((uint64_t(hi) << 32) | lo);
}
__device__ __forceinline__ int64_t shr1_64(int64_t v) {
  const uint32_t lo = uint32_t(shr1(int32_t(uint32_t(uint64_t(v))), 0));
  const uint32_t hi = uint32_t(shr1(int32_t(uint32_t(uint64_t(v) >> 32)), 0));
  return int64_t((uint64_t(hi) << 32) | lo);
}
__device__ __forceinline__ int hi_bit64(uint64_t v) { return 63 - __builtin_clzll(v); }

__device__ __forceinline__ uint64_t l0_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void __launch_bounds__(64)
bs_sim(BsShape r, const int32_t* __restrict__ R, const int32_t* __restrict__ next,
       const int64_t* __restrict__ sizes, int64_t d0,
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
  const int32_t* Rr = R + i * r.M_max;
  // a sample's size (0 for an id outside [0, F))
  auto size_at_id = [&](int32_t k) -> int64_t {
    return (k >= 0 && k < r.F) ? sizes[k] : int64_t(0);
  };
  int8_t* hrow = hit + i * r.M_max;
  for (int64_t w = lane; w < W0; w += 64) l0[w] = 0u;
  for (int64_t w = lane; w < W1; w += 64) l1[w] = 0u;
  for (int64_t w = lane; w < W2; w += 64) l2[w] = 0u;
  __threadfence();  // the cleared words reach L2 before the atomics below
  __syncthreads();

  __shared__ int32_t kslot[64];
  int64_t used = 0, hc = 0, hb = 0;
  // the highest held keys, ascending in lanes 0..n-1, with their sizes;
  // every held key >= ck[0] is cached, and n == 0 only when nothing is held
  int32_t ck = INT32_MAX;
  int64_t cz = 0;
  int n = 0;
  int64_t nheld = 0;

  // clears the level bits above a level-0 word that has become zero
  auto word_emptied = [&](int64_t w) {
    if (lane == 0) {
      const int64_t a = w >> 5;
      const uint32_t v1 = atomicAnd(&l1[a], ~(1u << (w & 31))) & ~(1u << (w & 31));
      if (v1 == 0u) atomicAnd(&l2[a >> 5], ~(1u << (a & 31)));
    }
  };
  // the cache's lowest key leaves (it stays held in the bitmap)
  auto drop_min = [&]() {
    ck = shl1(ck, INT32_MAX);
    cz = shl1_64(cz);
    --n;
  };
  // a key above ck[0] (or into an empty cache) joins in order; a full cache
  // first lets its lowest key go
  auto cache_insert = [&](int32_t key, int64_t sz) {
    if (n == 64) drop_min();
    const int p = __builtin_popcountll(__ballot(lane < n && ck < key));
    const int32_t uk = shr1(ck, INT32_MAX);
    const int64_t uz = shr1_64(cz);
    if (lane > p && lane <= n) {
      ck = uk;
      cz = uz;
    }
    if (lane == p) {
      ck = key;
      cz = sz;
    }
    ++n;
  };
  // fills the empty cache with the highest held keys: the words of the two
  // highest level-1 words that have set bits, one word per lane, highest
  // first; level bits of words found empty (keys discarded from the cache
  // leave them set) are cleared on the way
  auto refill = [&]() {
    __builtin_amdgcn_s_waitcnt(0);  // lane 0's atomics are in L2 before other lanes load
    n = 0;
    while (n == 0 && nheld > 0) {
      int64_t w2 = -1;
      for (int64_t base = ((W2 - 1) >> 6) << 6; base >= 0; base -= 64) {
        const int64_t idx = base + lane;
        const uint32_t v = idx < W2 ? l2[idx] : 0u;
        const uint64_t bl = __ballot(v != 0u);
        if (bl) {
          w2 = base + (63 - __builtin_clzll(bl));
          break;
        }
      }
      if (w2 < 0) break;  // nothing marked (only if sizes or next uses break the precondition)
      const uint32_t v2 = l2[w2];
      const int64_t a1 = (w2 << 5) + hi_bit(v2);
      const uint32_t v1a = l1[a1];
      if (v1a == 0u) {  // a level-2 bit over an empty level-1 word
        if (lane == 0) atomicAnd(&l2[w2], ~(1u << (a1 & 31)));
        __builtin_amdgcn_s_waitcnt(0);
        continue;
      }
      // the next level-1 word with a level-2 bit, below a1
      int64_t a2 = -1;
      const uint32_t below = v2 & ((1u << (a1 & 31)) - 1u);
      if (below) {
        a2 = (w2 << 5) + hi_bit(below);
      } else {
        for (int64_t base = ((w2 - 1) >> 6) << 6; w2 > 0 && base >= 0; base -= 64) {
          const int64_t idx = base + lane;
          const uint32_t v = idx < w2 ? l2[idx] : 0u;
          const uint64_t bl = __ballot(v != 0u);
          if (bl) {
            const int64_t w2b = base + (63 - __builtin_clzll(bl));
            a2 = (w2b << 5) + hi_bit(l2[w2b]);
            break;
          }
        }
      }
      const uint32_t v1b = a2 >= 0 ? l1[a2] : 0u;
      const int jj = lane & 31;
      const uint32_t v1 = lane < 32 ? v1a : v1b;
      const int64_t a = lane < 32 ? a1 : a2;
      const bool has = a >= 0 && ((v1 >> (31 - jj)) & 1u);
      const int64_t w = a * 32 + (31 - jj);
      uint64_t v = has ? l0_load(&l0[w]) : uint64_t(0);
      if (has && v == 0u) {  // marked but empty: clear the marks
        const uint32_t m1 = 1u << (w & 31);
        const uint32_t left = atomicAnd(&l1[w >> 5], ~m1) & ~m1;
        if (left == 0u) atomicAnd(&l2[w >> 10], ~(1u << ((w >> 5) & 31)));
      }
      const uint32_t pop = uint32_t(__builtin_popcountll(v));
      const uint32_t incl = wave_inclusive_scan(pop);
      const uint32_t ex = incl - pop;
      const uint32_t sum = __builtin_amdgcn_readlane(incl, 63);
      const int total = sum < 64u ? int(sum) : 64;
      __builtin_amdgcn_s_waitcnt(0);
      if (total == 0) continue;  // only empty words: their marks are gone now
      const int k = ex >= 64u ? 0 : (int(pop) < 64 - int(ex) ? int(pop) : 64 - int(ex));
      for (int it = 0; it < 64; ++it) {
        if (!__ballot(it < k)) break;
        if (it < k) {
          const int bp = hi_bit64(v);
          v &= ~(uint64_t(1) << bp);
          kslot[total - 1 - (int(ex) + it)] = int32_t((w << 6) + bp);
        }
      }
      __builtin_amdgcn_wave_barrier();
      const int32_t key = lane < total ? kslot[lane] : INT32_MAX;
      ck = key;
      const int32_t kid = (lane < total && key >= 0 && key < Mi) ? Rr[key] : -1;
      cz = size_at_id(kid);
      n = total;
      // wait for the sizes here, once: an empty asm that takes and redefines
      // them, so no later use of the cache waits on memory (such a wait would
      // also wait for lane 0's latest atomics)
      asm volatile("" : "+v"(cz), "+v"(ck));
    }
  };
  // the batch: its index, held keys among its positions, and the changes
  // made to the next batch's word since lane 0 loaded it
  int64_t b = 0;
  uint64_t hw = 0, nset = 0, nclr = 0;
  // discards the highest key
  auto evict = [&]() -> bool {
    const int32_t x = __builtin_amdgcn_readlane(ck, n - 1);
    const int64_t sx = rl64(cz, n - 1);
    --n;
    if (x < 0 || x >= Mi) return false;  // cannot happen: cached keys are held positions
    const int64_t w = x >> 6;
    const uint64_t bx = uint64_t(1) << (x & 63);
    if (lane == 0) atomicAnd(reinterpret_cast<unsigned long long*>(&l0[w]), ~bx);
    // this batch's word or the next one's (branch-free: keeps them in registers)
    const uint64_t mb = w == b ? bx : uint64_t(0);
    const uint64_t mn = w == b + 1 ? bx : uint64_t(0);
    hw &= ~mb;
    nclr |= mn;
    nset &= ~mn;
    used -= sx;
    --nheld;
    if (n == 0 && nheld > 0) refill();
    return true;
  };

  // the next batch: sizes, next uses, lane 0's copy of its word, and the
  // changes made to that word since it was loaded
  // pipeline: ids and next uses two batches ahead, sizes one
  int32_t kN2 = 64 + lane < Mi ? Rr[64 + lane] : -1;
  int32_t nN2 = 64 + lane < Mi ? Xr[64 + lane] : -1;
  int64_t sN = size_at_id(lane < Mi ? Rr[lane] : -1);
  int32_t nN = lane < Mi ? Xr[lane] : -1;
  uint64_t hN = 0;  // every word starts empty
  for (int64_t f0 = 0; f0 < Mi; f0 += 64, ++b) {
    const int64_t f = f0 + lane;
    const int64_t s = sN;
    int32_t nx = nN;
    if (nx <= f || nx >= Mi) nx = -1;
    hw = (rfl64(hN) & ~nclr) | nset;
    const uint64_t cand = __ballot(nx >= 0 && s <= d0);
    nset = nclr = 0;
    hN = 0;
    {  // the next batches' loads, after this batch's values are in use
      sN = size_at_id(kN2);
      nN = nN2;
      const int64_t g = f + 128;
      kN2 = g < Mi ? Rr[g] : -1;
      nN2 = g < Mi ? Xr[g] : -1;
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
        --nheld;
        hw &= ~bit;
        if (lane == 0) atomicAnd(reinterpret_cast<unsigned long long*>(&l0[b]), ~bit);
        if (hw == 0u) word_emptied(b);
        if (n > 0 && __builtin_amdgcn_readlane(ck, 0) == int32_t(f0 + q)) {
          drop_min();
          if (n == 0 && nheld > 0) refill();
        }
      }
      if (!(cand & bit)) continue;
      const int32_t nq = __builtin_amdgcn_readlane(nx, q);
      const int64_t top = n > 0 ? int64_t(__builtin_amdgcn_readlane(ck, n - 1)) : -1;
      if (nq > top && sq > d0 - used) continue;  // the furthest and it does not fit: bypass
      {  // admit under the next use
        const int64_t w = nq >> 6;
        const uint64_t bn = uint64_t(1) << (nq & 63);
        if (lane == 0) {
          atomicOr(reinterpret_cast<unsigned long long*>(&l0[w]), bn);
          atomicOr(&l1[w >> 5], 1u << (w & 31));
          atomicOr(&l2[w >> 10], 1u << ((w >> 5) & 31));
        }
        // a later read of this batch, or of the next one
        const uint64_t mb = w == b ? bn : uint64_t(0);
        const uint64_t mn = w == b + 1 ? bn : uint64_t(0);
        hw |= mb;
        mask |= mb;
        nset |= mn;
        nclr &= ~mn;
        if (n == 0 || nq > __builtin_amdgcn_readlane(ck, 0)) cache_insert(nq, sq);
        ++nheld;
        used += sq;
      }
      // discard the furthest while over capacity
      while (used > d0) {
        if (n == 0 || !evict()) {  // nothing held (broken precondition)
          used = 0;
          break;
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
  if ((rc = scr.alloc_n(&L0, size_t(s.N * W0)))) return rc;
  return launch("bs_sim", bs_sim, dim3(uint32_t(s.N)), dim3(64), 0, st, r, R, next, sizes, d0, L0, hit,
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
