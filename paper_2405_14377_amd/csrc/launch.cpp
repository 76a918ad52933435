// Launch check mode: the compute calls run their whole host path, but each
// kernel launch is validated against the gfx950 launch limits and recorded
// instead of being issued (comera_debug_launch_check in comera.h).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

namespace comera {
namespace {

struct LaunchRec {
    std::string name;
    uint32_t grid[3], block[3];
    uint64_t lds;
    bool ok;
};

std::atomic<bool> g_check{false};
std::mutex g_mu;
std::vector<LaunchRec> g_log;
thread_local int g_pending = 0;     // first failed check since the last launch_status()

constexpr size_t kMaxRecords = 1 << 20;
constexpr uint64_t kMaxLds = 160 * 1024;   // LDS of one gfx950 CU

}  // namespace

bool launch_check_mode() { return g_check.load(std::memory_order_relaxed); }

void launch_check(const char *name, dim3 grid, dim3 block, size_t lds) {
    const uint64_t threads = uint64_t(block.x) * block.y * block.z;
    const bool ok = grid.x >= 1 && grid.x <= 0x7fffffffu && grid.y >= 1 && grid.y <= 65535 && grid.z >= 1 &&
                    grid.z <= 65535 && threads >= 1 && threads <= 1024 && lds <= kMaxLds;
    if (!ok && !g_pending) g_pending = int(hipErrorInvalidConfiguration);
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_log.size() < kMaxRecords)
        g_log.push_back({name, {grid.x, grid.y, grid.z}, {block.x, block.y, block.z}, uint64_t(lds), ok});
}

int launch_status() {
    if (!launch_check_mode()) return int(hipGetLastError());
    const int e = g_pending;
    g_pending = 0;
    return e;
}

}  // namespace comera

using namespace comera;

extern "C" {

comera_status comera_debug_launch_check(int32_t enable) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_log.clear();
    g_pending = 0;
    g_check.store(enable != 0);
    return COMERA_OK;
}

int32_t comera_debug_launch_count(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    return int32_t(g_log.size());
}

comera_status comera_debug_launch_info(int32_t i, char *name, size_t len, uint32_t *grid3, uint32_t *block3,
                                       uint64_t *lds, int32_t *ok) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (i < 0 || size_t(i) >= g_log.size()) return COMERA_ERR_INVALID_ARG;
    const LaunchRec &r = g_log[size_t(i)];
    if (name && len > 0) {
        std::strncpy(name, r.name.c_str(), len - 1);
        name[len - 1] = 0;
    }
    if (grid3) std::memcpy(grid3, r.grid, sizeof(r.grid));
    if (block3) std::memcpy(block3, r.block, sizeof(r.block));
    if (lds) *lds = r.lds;
    if (ok) *ok = r.ok ? 1 : 0;
    return COMERA_OK;
}

}  // extern "C"
