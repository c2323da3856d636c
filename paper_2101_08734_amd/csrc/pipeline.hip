// nopfs_plan_job: the four stages in one call. The outputs equal those of
// nopfs_access_streams, nopfs_access_stats, nopfs_reuse_next and
// nopfs_tier_plan called in order; inside, the counting pass and the
// next-use pass share one partition of the streams when their sample
// windows agree, and the counting pass lists each worker's read cells (bin
// and offset, 4 bytes) so the tier plan reads that list instead of the dense
// count and first tables.
#include <map>
#include <mutex>
#include <new>
#include <string>

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

// Scratch of nopfs_plan_job_noalloc: one array per device, in the library's
// code object, held by every device the library runs on until the process
// ends. Host code must not pass `scratch` itself to a kernel (on the host it
// names a stand-in, not device memory): its device address is looked up once
// per device with hipGetSymbolAddress and used everywhere instead.
constexpr size_t kNoAllocScratch = size_t(64) << 20;
__device__ __align__(256) char scratch[kNoAllocScratch];

int noalloc_block(char** block) {
  static std::mutex mu;
  static std::map<int, char*> addr;  // device -> address of `scratch` on it
  int dev = 0;
  NOPFS_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> g(mu);
  auto it = addr.find(dev);
  if (it == addr.end()) {
    void* q = nullptr;
    const hipError_t e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !q) {
      (void)hipGetLastError();
      return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol,
                      "hipGetSymbolAddress of the allocation-free scratch");
    }
    it = addr.emplace(dev, static_cast<char*>(q)).first;
  }
  *block = it->second;
  return NOPFS_OK;
}

}  // namespace
}  // namespace nopfs

extern "C" int nopfs_plan_job_noalloc(const nopfs_job* job, const int64_t* sizes,
                                      const int64_t* caps, int32_t J, int32_t* R, uint8_t* count,
                                      int32_t* first, int32_t* next, int8_t* tier, int64_t* used,
                                      void* hip_stream) {
  using namespace nopfs;
  try {
    const hipStream_t st = static_cast<hipStream_t>(hip_stream);
    auto call = [&]() {
      return plan_job_impl(job, sizes, caps, J, R, count, first, next, tier, used, st);
    };
    // the scratch the job needs, found without launching anything; argument
    // errors come back from this pass
    size_t need = 0;
    int rc = run_sizing(call, &need);
    if (rc) return rc;
    if (need > kNoAllocScratch)
      return fail(NOPFS_ERANGE, "the job needs " + std::to_string(need) +
                                    " bytes of scratch; the allocation-free entry point holds " +
                                    std::to_string(kNoAllocScratch) + " per device");
    char* block = nullptr;
    if ((rc = noalloc_block(&block))) return rc;
    return run_in_fixed_block(block, kNoAllocScratch, call);
  } catch (const std::bad_alloc&) {
    return fail(NOPFS_ENOMEM, "host allocation failed");
  } catch (...) {
    return fail(NOPFS_EDEVICE, "unexpected host exception");
  }
}

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
