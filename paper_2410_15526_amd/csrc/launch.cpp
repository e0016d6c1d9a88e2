// launch.cpp -- grid sizing shared by every launcher.
#include "launch.hpp"

#include <hip/hip_runtime.h>

#include <mutex>
#include <unordered_map>

namespace sdp4 {

namespace {
std::mutex g_mu;
std::unordered_map<const void *, int> g_occ; // kernel -> resident blocks per CU
int g_cus[64];
int g_khz[64];
} // namespace

int wall_clock_khz(hipError_t &err)
{
    int dev = 0;
    err = hipGetDevice(&dev);
    if (err != hipSuccess)
        return 0;
    std::lock_guard<std::mutex> lk(g_mu);
    if (dev < 64 && g_khz[dev] != 0)
        return g_khz[dev];
    int v = 0;
    err = hipDeviceGetAttribute(&v, hipDeviceAttributeWallClockRate, dev);
    if (err != hipSuccess)
        return 0;
    if (dev < 64)
        g_khz[dev] = v;
    return v;
}

namespace {
// LDS of `kernel` itself, and of one compute unit (cached).
std::unordered_map<const void *, int> g_static_lds;
int g_lds_per_cu[64], g_lds_per_block[64];

size_t reserve_lds(const void *kernel, int per_cu, hipError_t &err)
{
    int dev = 0;
    err = hipGetDevice(&dev);
    if (err != hipSuccess)
        return 0;
    std::lock_guard<std::mutex> lk(g_mu);
    if (dev < 64 && g_lds_per_cu[dev] == 0) {
        int v = 0, b = 0;
        err = hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev);
        if (err == hipSuccess)
            err = hipDeviceGetAttribute(&b, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
        if (err != hipSuccess)
            return 0;
        g_lds_per_cu[dev] = v;
        g_lds_per_block[dev] = b;
    }
    const int lds = dev < 64 ? g_lds_per_cu[dev] : 160 * 1024;
    const int lds_block = dev < 64 ? g_lds_per_block[dev] : 64 * 1024;
    auto it = g_static_lds.find(kernel);
    if (it == g_static_lds.end()) {
        hipFuncAttributes a;
        err = hipFuncGetAttributes(&a, kernel);
        if (err != hipSuccess)
            return 0;
        it = g_static_lds.emplace(kernel, (int)a.sharedSizeBytes).first;
    }
    // per_cu blocks fit, one more does not: each takes lds / per_cu less a
    // margin of one allocation granule or so
    int64_t each = lds / per_cu - 1024;
    if (each > lds_block) // a block cannot hold more: residency is then bounded by the block limit
        each = lds_block;
    const int64_t dyn = each - it->second;
    return dyn > 0 ? (size_t)dyn : 0;
}
} // namespace

LaunchShape shape_for(const void *kernel, int64_t nwork_blocks, int per_cu_cap, int block_threads, hipError_t &err)
{
    err = hipSuccess;
    if (per_cu_cap < 0) { // one block per work block, dispatched in address order
        const int grid = (int)(nwork_blocks < 1 ? 1 : nwork_blocks < kMaxGrid ? nwork_blocks : kMaxGrid);
        if (per_cu_cap == kFullGrid)
            return {grid, 0};
        const size_t dyn = reserve_lds(kernel, -per_cu_cap, err);
        return {grid, dyn};
    }
    return {grid_for(kernel, nwork_blocks, per_cu_cap, block_threads, err), 0};
}

int grid_for(const void *kernel, int64_t nwork_blocks, int per_cu_cap, int block_threads, hipError_t &err)
{
    int dev = 0;
    err = hipGetDevice(&dev);
    if (err != hipSuccess)
        return 0;
    int per_cu, cus;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        if (dev < 64 && g_cus[dev] == 0) {
            int v = 0;
            err = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev);
            if (err != hipSuccess)
                return 0;
            g_cus[dev] = v;
        }
        cus = dev < 64 ? g_cus[dev] : 256;
        auto it = g_occ.find(kernel);
        if (it == g_occ.end()) {
            int nb = 0;
            err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, block_threads, 0);
            if (err != hipSuccess)
                return 0;
            it = g_occ.emplace(kernel, nb > 0 ? nb : 1).first;
        }
        per_cu = it->second;
    }
    // A launch whose work blocks all fit the device at full occupancy runs
    // them all at once: it has no steady state for the per-CU cap to pace,
    // and one round of tiles beats two.
    if (nwork_blocks <= (int64_t)cus * per_cu)
        return (int)(nwork_blocks > 0 ? nwork_blocks : 1);
    if (per_cu_cap > 0 && per_cu > per_cu_cap)
        per_cu = per_cu_cap;
    int64_t g = (int64_t)cus * per_cu;
    if (nwork_blocks < g)
        g = nwork_blocks;
    return (int)(g > 0 ? g : 1);
}

} // namespace sdp4
