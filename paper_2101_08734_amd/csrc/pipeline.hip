// nopfs_plan_job: the four stages in one call. The outputs equal those of
// nopfs_access_streams, nopfs_access_stats, nopfs_reuse_next and
// nopfs_tier_plan called in order; inside, the counting pass and the
// next-use pass share one partition of the streams when their sample
// windows agree, and the counting pass lists each worker's read cells (bin
// and offset, 4 bytes) so the tier plan reads that list instead of the dense
// count and first tables.
#include <new>

#include "pipeline.hpp"

namespace nopfs {
namespace {

int plan_job_impl(const nopfs_job* job, const int64_t* sizes, const int64_t* caps, int32_t J,
                  int32_t* R, uint8_t* count, int32_t* first, int32_t* next, int8_t* tier,
                  int64_t* used, hipStream_t st) {
  Shape s;
  int rc = make_shape(job, &s);
  if (rc) return rc;
  if (!sizes || !caps || !count || !first || !tier || !used)
    return fail(NOPFS_EINVAL, "sizes, caps, count, first, tier and used must be non-NULL");
  if (s.M_max > 0 && (!R || !next)) return fail(NOPFS_EINVAL, "R and next must be non-NULL");
  if ((rc = plan_check(caps, J))) return rc;
  if ((rc = streams_impl(job, R, st, -1, -1))) return rc;
  if (s.M_max == 0) {  // nothing is read: every cell is class 0
    if ((rc = stats_impl(job, R, count, first, st))) return rc;
    return plan_impl(job, count, first, sizes, caps, J, tier, used, st);
  }
  Scratch keep(st);
  CompactPlan* cp = nullptr;
  struct FreePlan {
    CompactPlan*& cp;
    ~FreePlan() {
      if (cp) compact_plan_free(cp);
    }
  } free_plan{cp};
  const ClassTable* classes = nullptr;
  if ((rc = compact_plan_prepare(s, caps, J, keep, st, &cp, &classes))) return rc;
  CompactCells cc;
  if ((rc = access_fused(s, R, classes, count, first, next, &cc, keep, st))) return rc;
  return compact_plan_run(cp, cc, count, first, sizes, tier, used, st);
}

}  // namespace
}  // namespace nopfs

extern "C" int nopfs_plan_job(const nopfs_job* job, const int64_t* sizes, const int64_t* caps,
                              int32_t J, int32_t* R, uint8_t* count, int32_t* first, int32_t* next,
                              int8_t* tier, int64_t* used, void* hip_stream) {
  try {
    return nopfs::plan_job_impl(job, sizes, caps, J, R, count, first, next, tier, used,
                                static_cast<hipStream_t>(hip_stream));
  } catch (const std::bad_alloc&) {
    return nopfs::fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return nopfs::fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}
