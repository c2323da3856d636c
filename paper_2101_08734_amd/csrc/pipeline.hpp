// Internal interface of the fused planning call (nopfs_plan_job): the
// counting pass hands the tier plan a compact list of the cells each worker
// reads, so the plan's passes read that list instead of the dense [N][F]
// count and first-read tables.
#pragma once

#include "common.hpp"

namespace nopfs {

// Rank-ordered bins of the tier plan for read cells (count class c >= 1,
// first read f): one 8-byte record per class, the bin scale and, packed, the
// class's first bin (high 16 bits) and its last bin offset (low 16). Classes
// above E (outside the precondition) hold class E's record.
struct ClassTable {
  float2 e[256];  // x = scale, y = bits of (base << 16 | top)
};

// Bin of a read cell with first read f from its class's record (scale, bits).
__device__ __forceinline__ uint32_t bin_of(float scale, uint32_t bt, int32_t f) {
  // a negative f (not a first read) lands in the class's first bin
  const uint32_t xi0 = uint32_t(fmaxf(float(f) * scale, 0.f));
  const uint32_t top = bt & 0xFFFFu;
  return (bt >> 16) + (xi0 < top ? xi0 : top);
}

__device__ __forceinline__ uint32_t bin_read(const ClassTable& t, uint32_t c, int32_t f) {
  const float2 r = t.e[c];
  return bin_of(r.x, __float_as_uint(r.y), f);
}

// Read-cell list entry: bin << kListOffBits | offset of the sample in its
// window (bins of classes >= 1 are fewer than 2^13, windows at most 2^19).
constexpr int kListOffBits = 19;
constexpr uint32_t kListOffMask = (1u << kListOffBits) - 1;

// Read cells per (worker i, sample window kb) tile, windows of 2^ws samples.
// Tile (i, kb) owns entries ent[i * M_max + base[i * nbk + kb] + t] for
// t < num[i * nbk + kb] (a worker reads at most M_max cells, and base is the
// number of its reads in earlier windows, so tiles never overlap). One entry
// per read cell, in no particular order inside the tile.
struct CompactCells {
  uint32_t* ent = nullptr;
  int32_t* base = nullptr;
  uint32_t* num = nullptr;
  int32_t ws = 0;
  uint32_t nbk = 0;
};

// Counting pass, first reads and next uses of R (the stages of
// nopfs_access_stats and nopfs_reuse_next); the counting pass also fills *cc,
// binning the read cells with `classes`. Scratch that must outlive the call
// (the list) is taken from `keep`. Requires M_max > 0.
int access_fused(const Shape& s, const int32_t* R, const ClassTable* classes, uint8_t* count,
                 int32_t* first, int32_t* next, CompactCells* cc, Scratch& keep, hipStream_t st);

// Tier plan (the stage of nopfs_tier_plan) from the compact list, in two
// steps: prepare() checks the arguments, allocates from `keep` and fills the
// class table the counting pass bins with; run() does the rest. count and
// first are the dense tables of the same call (first read for candidate
// cells, both for a worker whose candidate list overflows).
struct CompactPlan;
int compact_plan_prepare(const Shape& s, const int64_t* caps, int32_t J, Scratch& keep,
                         hipStream_t st, CompactPlan** out, const ClassTable** classes);
int compact_plan_run(CompactPlan* cp, const CompactCells& cc, const uint8_t* count,
                     const int32_t* first, const int64_t* sizes, int8_t* tier, int64_t* used,
                     hipStream_t st);
void compact_plan_free(CompactPlan* cp);

// Argument checks of the tier plan (J and the capacities).
int plan_check(const int64_t* caps, int32_t J);

// Stage bodies shared by the separate entry points and the fused call.
// Streams of epochs [e_begin, e_end) (e_begin < 0: all epochs), written as
// the rows of a job of e_end - e_begin epochs.
int streams_impl(const nopfs_job* job, int32_t* R, hipStream_t st, int32_t e_begin,
                 int32_t e_end);
int stats_impl(const nopfs_job* job, const int32_t* R, uint8_t* count, int32_t* first,
               hipStream_t st);
int plan_impl(const nopfs_job* job, const uint8_t* count, const int32_t* first,
              const int64_t* sizes, const int64_t* caps, int32_t J, int8_t* tier, int64_t* used,
              hipStream_t st);

}  // namespace nopfs
