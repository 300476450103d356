// Dynamic LDS above 64 KB: a kernel's limit has to be raised once on each
// device before such a launch (gfx950 has 160 KB of LDS per CU).  The record
// of the (kernel, device) pairs already raised is the library's only shared
// host state; a mutex guards it, so concurrent first calls from several
// threads are safe and every later call is a lookup.
#include <hip/hip_runtime_api.h>

#include <mutex>
#include <set>
#include <utility>

namespace oc {

hipError_t raise_lds_limit(const void *kernel, size_t bytes) {
    if (bytes <= 65536) return hipSuccess;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    static std::mutex mu;
    static std::set<std::pair<const void *, int>> done;
    std::lock_guard<std::mutex> lock(mu);
    const auto key = std::make_pair(kernel, dev);
    if (done.count(key)) return hipSuccess;
    e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e == hipSuccess) done.insert(key);
    return e;
}

}  // namespace oc
