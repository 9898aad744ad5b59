// Device helpers shared by the fp32 and bf16 worker-product kernels.
#pragma once

#include "internal.h"

namespace coded {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ inline double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Maps this wavefront to (worker, index of the wave within the worker,
// parity?), given wsys / wpar waves per systematic / parity worker.  Returns
// false when the wavefront has no work.
__device__ inline bool wave_task(const WorkerArgs& a, int64_t wsys, int64_t wpar, int& worker, int64_t& idx,
                                 bool& parity) {
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWaves +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nsys_waves = wsys * a.n_sys;
    if (wave < nsys_waves) {
        worker = a.sys_ids[wave / wsys];
        idx = wave % wsys;
        parity = false;
        return true;
    }
    const int64_t w2 = wave - nsys_waves;
    if (w2 >= wpar * a.n_par) return false;
    worker = a.par_ids[w2 / wpar];
    idx = w2 % wpar;
    parity = true;
    return true;
}

__device__ inline void store_y(const WorkerArgs& a, int worker, int64_t t, int64_t col, double v) {
    const int64_t off = (static_cast<int64_t>(worker) * a.qb + t) * a.s + col;
    if (a.y_f64)
        static_cast<double*>(a.Y)[off] = v;
    else
        static_cast<float*>(a.Y)[off] = static_cast<float>(v);
}

}  // namespace
}  // namespace coded
