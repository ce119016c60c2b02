// Exact LRU stack distance without any allocation (pc_stack_distance_noalloc):
// the dominance count of pc_stack_distance, with its workspace taken from a
// fixed device array instead of the caller.
//
// The array is a file-scope __device__ variable, so every GPU the library
// runs on holds its own copy for the life of the process.  In host code its
// name is only a stand-in for the symbol, never a device address: the first
// call on a device (with that device current) asks the runtime for the
// device address once, and every later use -- the workspace handed to the
// kernels, the header the fill kernel clears -- goes through that address.
// pc_stack_distance clears everything it reads before reading it (with a
// kernel, not a memset, so the call stays valid under graph capture), so the
// contents left by the previous call do not matter; calls that overlap on one
// device share the array and race.
#include <mutex>

#include "pc_internal.h"

namespace pc {

constexpr size_t NOALLOC_BYTES = (size_t)128 << 20;   // 128 MiB per device
constexpr int NOALLOC_MAX_DEVICES = 64;

static __device__ __align__(256) unsigned char scratch[NOALLOC_BYTES];

static void *g_scratch[NOALLOC_MAX_DEVICES];
static std::once_flag g_scratch_once[NOALLOC_MAX_DEVICES];

// device address of this device's scratch array (nullptr if the runtime
// cannot give it); resolved once per device, with that device current
static void *scratch_address(int dev) {
    std::call_once(g_scratch_once[dev], [dev] {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess) g_scratch[dev] = p;
    });
    return g_scratch[dev];
}

}  // namespace pc

extern "C" {

uint64_t pc_stack_distance_noalloc_max_n(void) {
    // largest n whose pc_stack_distance workspace fits the array (the
    // workspace grows monotonically with n)
    uint64_t lo = 0, hi = pc::NOALLOC_BYTES;
    while (lo < hi) {
        const uint64_t mid = (lo + hi + 1) / 2;
        if (pc_stack_distance_ws(mid) <= pc::NOALLOC_BYTES) lo = mid; else hi = mid - 1;
    }
    return lo;
}

pc_status pc_stack_distance_noalloc(const uint32_t *prev, const uint32_t *next, uint64_t n, uint32_t *dist,
                                    void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n > 0 && (!prev || !next || !dist)) return PC_ERR_INVALID;
    if (pc_stack_distance_ws(n) > pc::NOALLOC_BYTES) return PC_ERR_TOO_LARGE;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= pc::NOALLOC_MAX_DEVICES) return PC_ERR_DEVICE;
    void *ws = pc::scratch_address(dev);
    if (!ws) return PC_ERR_DEVICE;
    return pc_stack_distance(prev, next, n, dist, ws, pc::NOALLOC_BYTES, stream);
}

}  // extern "C"
