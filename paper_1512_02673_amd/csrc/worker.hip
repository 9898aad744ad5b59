// Worker products Y_i = A'_i X for the simulated workers (Sec. III-A: each
// worker multiplies its stored coded block by the multicast input).
//
// All n blocks are served by one launch.  A systematic block is a window of A
// itself (rows i*qb .. i*qb+qb-1; rows at or beyond q are the zero padding and
// are never read).  A parity block is `planes` planes (hi, lo) in the parity
// buffer; its product is sum_h plane_h X.
//
// The work unit of a wavefront is R consecutive "plane rows": rows of a
// systematic block, or (row, plane) pairs of a parity block taken row-major,
// so every wavefront streams the same number of bytes whatever block it
// serves.  Lanes split the row's columns in 16-byte vectors (64 lanes x 16 B
// per load instruction, fully coalesced); each lane multiplies in fp64 (the
// product of two fp32 values is exact in fp64) and the 64 partial sums of a
// row are combined with cross-lane shuffles.  The kernel is bound by HBM: a
// row is read exactly once, X (at most a few hundred KB) stays in L2.
#include "internal.h"

namespace coded {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

typedef float f32x4 __attribute__((ext_vector_type(4)));

// 16-byte streaming load: the data is used once, so it is marked non-temporal
// to keep it from displacing X in the caches.
__device__ inline float4 load_stream(const float* p) {
    const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ inline double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

struct RowRef {
    const float* ptr;   // start of the plane row (null: zero padding / out of range)
    int64_t t;          // block row
};

// Plane row `pr` of worker `w`.
__device__ inline RowRef plane_row(const WorkerArgs& a, int w, int64_t pr, bool parity) {
    RowRef rr{nullptr, 0};
    if (!parity) {
        rr.t = pr;
        const int64_t row = static_cast<int64_t>(w) * a.qb + pr;
        if (pr < a.qb && row < a.q) rr.ptr = static_cast<const float*>(a.A) + row * a.lda;
    } else {
        const int64_t t = pr / a.planes;
        const int h = static_cast<int>(pr % a.planes);
        rr.t = t;
        if (t < a.qb) {
            const int64_t plane = static_cast<int64_t>(a.n - a.k) * a.qb * a.r;
            rr.ptr = static_cast<const float*>(a.parity) + h * plane +
                     (static_cast<int64_t>(w - a.k) * a.qb + t) * a.r;
        }
    }
    return rr;
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

// s == 1, 16-byte vectors.  R plane rows per wave, U vectors per lane in flight per row.
template <int R, int U>
__global__ __launch_bounds__(kThreads) void gemv_f32_kernel(WorkerArgs a) {
    int worker;
    int64_t idx;
    bool parity;
    if (!wave_task(a, ceil_div(a.qb, R), ceil_div(a.qb * a.planes, R), worker, idx, parity)) return;
    const int64_t pr0 = idx * R;
    const int lane = threadIdx.x & 63;

    const float* rp[R];
    int64_t rt[R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
        RowRef ref = plane_row(a, worker, pr0 + i, parity);
        rp[i] = ref.ptr;
        rt[i] = ref.t;
    }
    const float* x = static_cast<const float*>(a.X);

    double acc[R];
#pragma unroll
    for (int i = 0; i < R; ++i) acc[i] = 0.0;

    constexpr int kStep = 64 * 4 * U;                 // columns per iteration
    const int64_t full = (a.r / kStep) * kStep;
    for (int64_t c0 = 0; c0 < full; c0 += kStep) {
        float4 xv[U];
        float4 av[R][U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            xv[u] = *reinterpret_cast<const float4*>(x + c0 + u * 256 + lane * 4);
#pragma unroll
        for (int i = 0; i < R; ++i) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (rp[i])
                    av[i][u] = load_stream(rp[i] + c0 + u * 256 + lane * 4);
                else
                    av[i][u] = make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const double x0 = xv[u].x, x1 = xv[u].y, x2 = xv[u].z, x3 = xv[u].w;
#pragma unroll
            for (int i = 0; i < R; ++i) {
                acc[i] = fma(static_cast<double>(av[i][u].x), x0, acc[i]);
                acc[i] = fma(static_cast<double>(av[i][u].y), x1, acc[i]);
                acc[i] = fma(static_cast<double>(av[i][u].z), x2, acc[i]);
                acc[i] = fma(static_cast<double>(av[i][u].w), x3, acc[i]);
            }
        }
    }
    // Tail: remaining columns, one vector per lane per step.
    for (int64_t c = full + lane * 4; c < a.r; c += 256) {
        const float4 xv = *reinterpret_cast<const float4*>(x + c);
        const double x0 = xv.x, x1 = xv.y, x2 = xv.z, x3 = xv.w;
#pragma unroll
        for (int i = 0; i < R; ++i) {
            if (rp[i]) {
                const float4 v = *reinterpret_cast<const float4*>(rp[i] + c);
                acc[i] = fma(static_cast<double>(v.x), x0, acc[i]);
                acc[i] = fma(static_cast<double>(v.y), x1, acc[i]);
                acc[i] = fma(static_cast<double>(v.z), x2, acc[i]);
                acc[i] = fma(static_cast<double>(v.w), x3, acc[i]);
            }
        }
    }
#pragma unroll
    for (int i = 0; i < R; ++i) acc[i] = wave_sum(acc[i]);

    if (lane == 0) {
        if (!parity || a.planes == 1) {
#pragma unroll
            for (int i = 0; i < R; ++i)
                if (rt[i] < a.qb) store_y(a, worker, rt[i], 0, acc[i]);
        } else {
            // planes == 2 and R even: plane rows (2t, 2t+1) are (hi, lo) of row t.
#pragma unroll
            for (int i = 0; i < R; i += 2)
                if (rt[i] < a.qb) store_y(a, worker, rt[i], 0, acc[i] + acc[i + 1]);
        }
    }
}

// General shapes (any r, s, strides): one block row per wave (all planes of a
// parity row), scalar loads, columns of X in groups of SC.  Used for s > 1
// and for unaligned inputs.
template <int SC>
__global__ __launch_bounds__(kThreads) void gemm_small_f32_kernel(WorkerArgs a) {
    int worker;
    int64_t t;
    bool parity;
    if (!wave_task(a, a.qb, a.qb, worker, t, parity)) return;
    const int lane = threadIdx.x & 63;
    const int nplanes = parity ? a.planes : 1;
    const float* x = static_cast<const float*>(a.X);
    for (int64_t c0 = 0; c0 < a.s; c0 += SC) {
        double acc[SC];
#pragma unroll
        for (int j = 0; j < SC; ++j) acc[j] = 0.0;
        for (int h = 0; h < nplanes; ++h) {
            const float* rowp = plane_row(a, worker, parity ? t * a.planes + h : t, parity).ptr;
            if (!rowp) continue;
            for (int64_t c = lane; c < a.r; c += 64) {
                const double av = rowp[c];
                const float* xr = x + c * a.ldx + c0;
#pragma unroll
                for (int j = 0; j < SC; ++j)
                    if (c0 + j < a.s) acc[j] = fma(av, static_cast<double>(xr[j]), acc[j]);
            }
        }
#pragma unroll
        for (int j = 0; j < SC; ++j) acc[j] = wave_sum(acc[j]);
        if (lane == 0) {
#pragma unroll
            for (int j = 0; j < SC; ++j)
                if (c0 + j < a.s) store_y(a, worker, t, c0 + j, acc[j]);
        }
    }
}

// bf16 blocks and X, fp32 accumulation (products of two bf16 values are exact
// in fp32), same work split as gemm_small_f32_kernel.
template <int SC>
__global__ __launch_bounds__(kThreads) void gemm_small_bf16_kernel(WorkerArgs a) {
    int worker;
    int64_t t;
    bool parity;
    if (!wave_task(a, a.qb, a.qb, worker, t, parity)) return;
    const int lane = threadIdx.x & 63;
    const int nplanes = parity ? a.planes : 1;
    const uint16_t* x = static_cast<const uint16_t*>(a.X);
    const int64_t plane = static_cast<int64_t>(a.n - a.k) * a.qb * a.r;
    for (int64_t c0 = 0; c0 < a.s; c0 += SC) {
        float acc[SC];
#pragma unroll
        for (int j = 0; j < SC; ++j) acc[j] = 0.0f;
        for (int h = 0; h < nplanes; ++h) {
            const uint16_t* rowp = nullptr;
            if (!parity) {
                const int64_t row = static_cast<int64_t>(worker) * a.qb + t;
                if (row < a.q) rowp = static_cast<const uint16_t*>(a.A) + row * a.lda;
            } else {
                rowp = static_cast<const uint16_t*>(a.parity) + h * plane +
                       (static_cast<int64_t>(worker - a.k) * a.qb + t) * a.r;
            }
            if (!rowp) continue;
            for (int64_t c = lane; c < a.r; c += 64) {
                const float av = __uint_as_float(static_cast<uint32_t>(rowp[c]) << 16);
                const uint16_t* xr = x + c * a.ldx + c0;
#pragma unroll
                for (int j = 0; j < SC; ++j)
                    if (c0 + j < a.s) acc[j] = fmaf(av, __uint_as_float(static_cast<uint32_t>(xr[j]) << 16), acc[j]);
            }
        }
#pragma unroll
        for (int j = 0; j < SC; ++j) {
            float v = acc[j];
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
            acc[j] = v;
        }
        if (lane == 0) {
#pragma unroll
            for (int j = 0; j < SC; ++j)
                if (c0 + j < a.s) store_y(a, worker, t, c0 + j, acc[j]);
        }
    }
}

bool aligned(const void* p, int bytes) { return (reinterpret_cast<uintptr_t>(p) % bytes) == 0; }

template <typename K>
hipError_t launch_waves(K kernel, const WorkerArgs& a, int64_t wsys, int64_t wpar, hipStream_t st) {
    const int64_t waves = wsys * a.n_sys + wpar * a.n_par;
    if (waves == 0) return hipSuccess;
    const int64_t blocks = ceil_div(waves, kWaves);
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_worker_f32(const WorkerArgs& a, hipStream_t st) {
    if (a.qb == 0) return hipSuccess;
    const bool vec = a.s == 1 && a.ldx == 1 && (a.r % 4 == 0) && (a.lda % 4 == 0) && aligned(a.A, 16) &&
                     aligned(a.X, 16) && (a.parity == nullptr || aligned(a.parity, 16));
    if (vec) {
        constexpr int R = 4, U = 4;   // R even keeps a parity row's hi and lo in one wave
        return launch_waves(gemv_f32_kernel<R, U>, a, ceil_div(a.qb, R), ceil_div(a.qb * a.planes, R), st);
    }
    return launch_waves(gemm_small_f32_kernel<4>, a, a.qb, a.qb, st);
}

hipError_t launch_worker_bf16(const WorkerArgs& a, hipStream_t st) {
    if (a.qb == 0) return hipSuccess;
    return launch_waves(gemm_small_bf16_kernel<4>, a, a.qb, a.qb, st);
}

}  // namespace coded
