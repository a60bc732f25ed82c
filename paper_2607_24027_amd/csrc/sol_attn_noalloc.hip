// Built-in device scratch for the forward entry point that allocates nothing
// (sol_attn_forward_noalloc).  The array lives in the library's code object, so every GPU the
// library runs on holds its own copy, at its own address, until the process ends.  Host code
// never passes the array's name to a kernel (on the host it names a host-side stand-in): the
// device address is looked up once per device with hipGetSymbolAddress and used instead.
#include <map>
#include <mutex>

#include "sol_attn_internal.h"

namespace sol {
namespace {

constexpr size_t kNoallocScratchBytes = size_t(64) << 20;   // 64 MiB per device

static __device__ __align__(256) char scratch[kNoallocScratchBytes];

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_addr;   // device -> device address of `scratch`

}  // namespace

size_t noalloc_scratch_bytes() { return kNoallocScratchBytes; }

hipError_t noalloc_scratch(void** addr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    auto it = g_scratch_addr.find(dev);
    if (it == g_scratch_addr.end()) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // with `dev` current
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        it = g_scratch_addr.emplace(dev, p).first;
    }
    *addr = it->second;
    return hipSuccess;
}

}  // namespace sol
