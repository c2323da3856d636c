// Internal interface of the fused planning call (nopfs_plan_job): the
// counting pass hands the tier plan a compact list of the cells each worker
// reads, so the plan's passes read that list instead of the dense [N][F]
// count and first-read tables.
#pragma once

#include "common.hpp"

namespace nopfs {

// Read cells per (worker i, sample window kb) tile, windows of 2^ws samples.
// Tile (i, kb) owns entries ent[i * M_max + base[i * nbk + kb] + t] for
// t < num[i * nbk + kb] (a worker reads at most M_max cells, and base is the
// number of its reads in earlier windows, so tiles never overlap). Entry =
// {first read f, count << 24 | offset of the sample in its window}, in no
// particular order inside the tile.
struct CompactCells {
  uint2* ent = nullptr;
  int32_t* base = nullptr;
  uint32_t* num = nullptr;
  int32_t ws = 0;
  uint32_t nbk = 0;
};

// Counting pass, first reads and next uses of R (the stages of
// nopfs_access_stats and nopfs_reuse_next) that also fills *cc. The next-use
// kernels go on `side_st` after side.begin(); every buffer comes from `keep`,
// which the caller frees only after `side` has joined. Requires M_max > 0.
int access_fused(const Shape& s, const int32_t* R, uint8_t* count, int32_t* first,
                 int32_t* next, CompactCells* cc, Scratch& keep, SideWork& side,
                 hipStream_t side_st, hipStream_t st);

// Tier plan (the stage of nopfs_tier_plan) from the compact list; count and
// first are the dense tables of the same pass (read only if a worker's
// candidate list overflows).
int plan_compact(const Shape& s, const CompactCells& cc, const uint8_t* count,
                 const int32_t* first, const int64_t* sizes, const int64_t* caps, int32_t J,
                 int8_t* tier, int64_t* used, hipStream_t st);

// Argument checks of the tier plan (J and the capacities).
int plan_check(const int64_t* caps, int32_t J);

// Stage bodies shared by the separate entry points and the fused call.
int streams_impl(const nopfs_job* job, int32_t* R, hipStream_t st);
int stats_impl(const nopfs_job* job, const int32_t* R, uint8_t* count, int32_t* first,
               hipStream_t st);
int plan_impl(const nopfs_job* job, const uint8_t* count, const int32_t* first,
              const int64_t* sizes, const int64_t* caps, int32_t J, int8_t* tier, int64_t* used,
              hipStream_t st);

}  // namespace nopfs
