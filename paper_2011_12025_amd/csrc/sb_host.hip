// Launch-setup state of the library, kept per device and shared by every
// host thread: the number of compute units (grid sizing) and the dynamic-LDS
// limit raised on each kernel.  Both tables are guarded, so calls may come
// from several host threads at once.
#include <atomic>
#include <map>
#include <mutex>
#include <utility>

#include "sb_kernels.h"

namespace sb {

namespace {

constexpr int MAXDEV = 64;
std::atomic<int> g_cus[MAXDEV];
std::mutex g_attr_mu;
std::map<std::pair<const void*, int>, int> g_attr;  // (kernel, device) -> dynamic LDS bytes allowed

}  // namespace

int device_cus() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAXDEV) return 256;
    int n = g_cus[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    g_cus[dev].store(n, std::memory_order_relaxed);
    return n;
}

hipError_t ensure_dyn_lds(const void* kernel, int bytes) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lk(g_attr_mu);
    int& cur = g_attr[std::make_pair(kernel, dev)];
    if (bytes > cur) {
        e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
        if (e != hipSuccess) return e;
        cur = bytes;
    }
    return hipSuccess;
}

}  // namespace sb
