// The fixed scratch buffer of gspmm_noalloc: a file-scope device array, of
// which every GPU that runs the library holds its own copy from the moment
// the library's code is loaded on it until the process ends.  Host code
// never passes the array's name to a kernel (on the host that name stands
// for a host-side shadow, not a device address): the device address of the
// copy on a GPU is looked up once, with that GPU current, and kept.
#include "host.h"

namespace gnnk {

static __device__ __align__(256) unsigned char scratch[STATIC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_mu;
void* g_addr[MAX_DEVICES] = {};

}  // namespace

gnnk_status static_scratch(hipStream_t stream, Scratch& sc) {
    int dev = -1;
    hipError_t e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return hip_fail(e, "gspmm_noalloc: device of the stream");
    if (dev < 0 || dev >= MAX_DEVICES) return fail(GNNK_EUNSUPPORTED, "gspmm_noalloc: device %d", dev);
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_addr[dev]) {
        int cur = -1;
        e = hipGetDevice(&cur);
        if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
        void* p = nullptr;
        if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur >= 0 && cur != dev) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess) e = e2;
        }
        if (e != hipSuccess) return hip_fail(e, "gspmm_noalloc: address of the fixed scratch buffer");
        g_addr[dev] = p;
    }
    sc.base = reinterpret_cast<char*>(g_addr[dev]);
    sc.bytes = STATIC_SCRATCH_BYTES;
    sc.used = 0;
    return GNNK_OK;
}

}  // namespace gnnk
