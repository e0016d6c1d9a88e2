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
