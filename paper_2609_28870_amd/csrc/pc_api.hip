// libpc: status strings, workspace status, fill kernel and the optional
// per-kernel event timing shared by every entry point.
#include <vector>

#include "pc_internal.h"

namespace pc {

// one case per kernel id (a missing one is a -Wswitch warning)
static const char *kernel_name(KernelId k) {
    switch (k) {
    case K_FILL32: return "fill_u32";
    case K_HASH: return "hash_blocks";
    case K_SORT_HIST: return "sort_digit_hist";
    case K_SORT_SCAN: return "sort_digit_scan";
    case K_SORT_PASS: return "sort_onesweep_pass";
    case K_LINK: return "link_partition";
    case K_PERM: return "perm_partition";
    case K_PERM_LOCAL: return "perm_local";
    case K_SD_COLD: return "sd_cold_count";
    case K_SD_SCAN: return "sd_scan";
    case K_SD_TILES: return "sd_tile_map";
    case K_SD_COUNT: return "sd_count";
    case K_SD_SEG: return "sd_seg_scan";
    case K_SD_PASS: return "sd_dominance_pass";
    case K_SD_LOCAL: return "sd_local_finish";
    case K_MRC_HIST: return "mrc_hist";
    case K_MRC_COST: return "mrc_cost";
    case K_REQ_ORDER: return "request_order";
    case K_REQ_DIST: return "request_distance";
    case K_SESS_REQ: return "session_requests";
    case K_SESS_DIST: return "session_distance";
    case K_SESS_PROFILE: return "session_profile";
    case K_PROF_PACK: return "reuse_profile_pack";
    case K_PROF_WALK: return "reuse_profile_walk";
    case K_CHAIN_ANCHOR: return "chain_anchor";
    case K_CHAIN_STAIR: return "chain_stair";
    case K_CHAIN_SCAN: return "chain_scan";
    case K_CHAIN_COMPACT: return "chain_compact";
    case K_CHAIN_MERGE: return "chain_merge";
    case K_RUNS_COUNT: return "runs_count";
    case K_RUNS_SCAN: return "runs_scan";
    case K_RUNS_COMPACT: return "runs_compact";
    case K_RUNS_MERGE: return "runs_merge";
    case K_RUNS_FILL: return "runs_fill";
    case K_BELADY: return "belady";
    case K_MRC_MAP: return "mrc_map";
    case K_COUNT: break;
    }
    return "";
}

struct ProfEvent {
    int kid;
    hipEvent_t a, b;
};

static bool g_prof = false;
static std::vector<ProfEvent> g_events;
static std::vector<hipEvent_t> g_pool;
static hipEvent_t g_pending = nullptr;
static uint64_t g_launches[K_COUNT];
static double g_ms[K_COUNT];

static hipEvent_t get_event() {
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

void prof_begin(int kid, hipStream_t s) {
    (void)kid;
    if (!g_prof) return;
    g_pending = get_event();
    if (g_pending && hipEventRecord(g_pending, s) != hipSuccess) g_pending = nullptr;
}

void prof_end(int kid, hipStream_t s) {
    if (!g_prof || !g_pending) return;
    hipEvent_t b = get_event();
    if (!b) return;
    if (hipEventRecord(b, s) != hipSuccess) return;
    g_events.push_back({kid, g_pending, b});
    g_pending = nullptr;
}

int device_cus() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        return 256;
    return cus;
}

unsigned capped(uint64_t items, int per_cu) {
    const uint64_t cap = (uint64_t)device_cus() * per_cu;
    const uint64_t g = items < cap ? items : cap;
    return (unsigned)(g ? g : 1);
}

__global__ void fill_u32_kernel(uint32_t *__restrict__ p, uint32_t value, size_t count) {
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    size_t stride = (size_t)gridDim.x * blockDim.x;
    for (; i < count; i += stride) p[i] = value;
}

__global__ void fill_u32_gated_kernel(uint32_t *__restrict__ p, uint32_t value, size_t count,
                                      const int32_t *__restrict__ gate) {
    if (*gate == 0) return;
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    size_t stride = (size_t)gridDim.x * blockDim.x;
    for (; i < count; i += stride) p[i] = value;
}

static unsigned fill_blocks(size_t count) {
    size_t blocks = (count + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    return (unsigned)blocks;
}

pc_status fill_u32(uint32_t *p, uint32_t value, size_t count, hipStream_t s) {
    if (count == 0) return PC_OK;
    PC_LAUNCH(K_FILL32, fill_u32_kernel, dim3(fill_blocks(count)), dim3(256), 0, s, p, value, count);
    return PC_OK;
}

pc_status fill_u32_gated(uint32_t *p, uint32_t value, size_t count, hipStream_t s, const int32_t *gate) {
    if (!gate) return fill_u32(p, value, count, s);
    if (count == 0) return PC_OK;
    PC_LAUNCH(K_FILL32, fill_u32_gated_kernel, dim3(fill_blocks(count)), dim3(256), 0, s, p, value, count, gate);
    return PC_OK;
}

}  // namespace pc

extern "C" {

const char *pc_status_string(pc_status s) {
    switch (s) {
        case PC_OK: return "ok";
        case PC_ERR_INVALID: return "invalid argument";
        case PC_ERR_TOO_LARGE: return "too large: positions must fit uint32 below 0xFFFFFFFF";
        case PC_ERR_WORKSPACE: return "workspace missing or too small";
        case PC_ERR_DEVICE: return "HIP device call or kernel launch failed";
        case PC_ERR_UNSUPPORTED: return "unsupported device";
    }
    return "unknown status";
}

int pc_version(void) { return 100; }

pc_status pc_workspace_status(const void *ws, size_t ws_bytes, void *stream, int32_t *code_out) {
    if (!ws || !code_out) return PC_ERR_INVALID;
    if (ws_bytes < pc::WS_HEADER) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    int32_t v = 0;
    if (hipMemcpyAsync(&v, ws, sizeof(v), hipMemcpyDeviceToHost, s) != hipSuccess) return PC_ERR_DEVICE;
    if (hipStreamSynchronize(s) != hipSuccess) return PC_ERR_DEVICE;
    *code_out = v;
    return PC_OK;
}

void pc_prof_enable(int on) { pc::g_prof = on != 0; }

int pc_prof_kernel_count(void) { return pc::K_COUNT; }

const char *pc_prof_kernel_name(int i) {
    return (i >= 0 && i < pc::K_COUNT) ? pc::kernel_name((pc::KernelId)i) : "";
}

pc_status pc_prof_read(uint64_t *launches, double *total_ms, int n) {
    for (auto &e : pc::g_events) {
        float ms = 0.f;
        if (hipEventSynchronize(e.b) != hipSuccess) return PC_ERR_DEVICE;
        if (hipEventElapsedTime(&ms, e.a, e.b) != hipSuccess) return PC_ERR_DEVICE;
        pc::g_launches[e.kid] += 1;
        pc::g_ms[e.kid] += ms;
        pc::g_pool.push_back(e.a);
        pc::g_pool.push_back(e.b);
    }
    pc::g_events.clear();
    for (int i = 0; i < n && i < pc::K_COUNT; ++i) {
        if (launches) launches[i] = pc::g_launches[i];
        if (total_ms) total_ms[i] = pc::g_ms[i];
        pc::g_launches[i] = 0;
        pc::g_ms[i] = 0.0;
    }
    return PC_OK;
}

}  // extern "C"
