// Worker products Y_i = A'_i X for the simulated workers (Sec. III-A: each
// worker multiplies its stored coded block by the multicast input).
//
// All n blocks are served by one launch.  A systematic block is a window of A
// itself (rows i*qb .. i*qb+qb-1; rows at or beyond q are the zero padding and
// are never read).  A parity block is `planes` planes (hi, lo) in the parity
// buffer; its product is sum_h plane_h X.
//
// The single-vector case (s == 1) is the HBM-bound GEMV: every byte of A and
// of the parity planes is read exactly once, in 16-byte non-temporal loads
// that a whole workgroup issues over one contiguous stretch of a row at a time
// (streaming each row through a single wavefront instead measurably loses
// bandwidth).  Products of two fp32 values are exact in fp64 and are summed
// in fp64.  s > 1 runs on the fp64 matrix cores (worker_f32_mfma.hip);
// unaligned shapes take a general vector kernel.
#include "internal.h"
#include "worker_common.h"

namespace coded {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// 16-byte streaming load: the data is used once, so it is marked non-temporal
// to keep it from displacing X in the caches.
__device__ inline float4 load_stream(const float* p) {
    // a global-memory pointer, so the load is a global (not flat) load
    typedef const __attribute__((address_space(1))) f32x4* gptr;
    const f32x4 v = __builtin_nontemporal_load((gptr)(p));
    return make_float4(v.x, v.y, v.z, v.w);
}
__device__ inline float4 load_global4(const float* p) {
    typedef const __attribute__((address_space(1))) f32x4* gptr;
    const f32x4 v = *(gptr)(p);
    return make_float4(v.x, v.y, v.z, v.w);
}

// Four bfloat16 values (8 bytes, streamed) as raw bits, and their exact
// widening to fp32 (kept apart so a select can take the raw load).
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
__device__ inline u32x2 load_stream_bf16x4(const uint16_t* p) {
    // a global-memory pointer, so the load is a global (not flat) load
    typedef const __attribute__((address_space(1))) u32x2* gptr;
    return __builtin_nontemporal_load((gptr)(p));
}
__device__ inline float4 widen_bf16x4(u32x2 v) {
    return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
                       __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u));
}

__device__ inline float bf16_bits_to_f32(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// First element of the lo plane when it is stored as bfloat16: directly after
// the fp32 hi plane, in the same (worker, block row, column) order.
__device__ inline const uint16_t* lo16_base(const WorkerArgs& a) {
    return reinterpret_cast<const uint16_t*>(static_cast<const float*>(a.parity) +
                                             static_cast<int64_t>(a.n - a.k) * a.qb * a.r);
}

struct RowRef {
    const float* ptr;     // start of the plane row (null: zero padding / out of range)
    const uint16_t* p16;  // instead of ptr for a bfloat16 lo plane
    int64_t t;            // block row
};

// Plane row `pr` of worker `w`.
__device__ inline RowRef plane_row(const WorkerArgs& a, int w, int64_t pr, bool parity) {
    RowRef rr{nullptr, nullptr, 0};
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
            const int64_t off = (static_cast<int64_t>(w - a.k) * a.qb + t) * a.r;
            if (h == 1 && a.lo_bf16)
                rr.p16 = lo16_base(a) + off;
            else
                rr.ptr = static_cast<const float*>(a.parity) + h * plane + off;
        }
    }
    return rr;
}

// s == 1, 16-byte vectors.  A workgroup of NT threads owns a tile of T
// consecutive rows of one worker's block and sweeps it one row at a time:
// thread tid covers column slots c = tid*4 + j*NT*4 (j < XR) of every row, so
// each load instruction of the workgroup reads NT*16 contiguous bytes, and
// its slice of x stays in registers for all T rows.  Rows wider than
// NT*4*XR are swept in column chunks (x reloaded per chunk).  A parity row's
// planes (hi, lo) are summed into the same fp64 accumulator.  Partial sums
// are combined across lanes (shuffles) and waves (LDS) in a fixed order.
// LO16: the lo plane is bfloat16 (8-byte loads of four values, widened
// exactly to fp32, so the products stay exact in fp64).
template <int T, int XR, int NT, bool LO16>
__global__ __launch_bounds__(NT) void gemv_wg_kernel(WorkerArgs a) {
    constexpr int NW = NT / 64;
    constexpr int kChunk = NT * 4 * XR;
    __shared__ double red[NW][T];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    // The arguments the first loads depend on, fetched in one batch and held
    // in scalar registers (left alone, the compiler fetches them one
    // dependent round trip after another, inside the branches that use them).
    const float* Ap = static_cast<const float*>(a.A);
    const float* Pp = static_cast<const float*>(a.parity);
    const float* x = static_cast<const float*>(a.X);
    int64_t q = a.q, r = a.r, lda = a.lda, qb = a.qb;
    int32_t n = a.n, k = a.k, planes = a.planes, n_sys = a.n_sys, n_par = a.n_par;
    asm volatile("" : "+s"(Ap), "+s"(Pp), "+s"(x), "+s"(q), "+s"(r), "+s"(lda), "+s"(qb), "+s"(n), "+s"(k),
                 "+s"(planes), "+s"(n_sys), "+s"(n_par));
    // The grid has fewer than 2^31 workgroups (checked at launch), so the
    // tile arithmetic fits 32 bits.
    const uint32_t groups = static_cast<uint32_t>(ceil_div(qb, T));
    const uint32_t npar = groups * static_cast<uint32_t>(n_par);
    const uint32_t g = blockIdx.x;
    int worker;
    int64_t grp;
    bool parity;
    // Parity workgroups stream `planes` times the bytes: dispatch them first so
    // the launch does not end on a tail of long workgroups.  With every worker
    // active (the usual case) the worker follows from the index; otherwise
    // from the lists of active workers.
    if (g < npar) {
        const uint32_t wi = g / groups;
        worker = n_par == n - k ? k + static_cast<int>(wi) : a.par_ids[wi];
        grp = g - wi * groups;
        parity = true;
    } else {
        if (g - npar >= groups * static_cast<uint32_t>(n_sys)) return;
        const uint32_t wi = (g - npar) / groups;
        worker = n_sys == k ? static_cast<int>(wi) : a.sys_ids[wi];
        grp = (g - npar) - wi * groups;
        parity = false;
    }
    const int64_t t0 = grp * T;
    const int nplanes = parity ? planes : 1;
    const int64_t plane = static_cast<int64_t>(n - k) * qb * r;

    // Row pointers of the tile (null: padding row or beyond the block).
    const float* rows[T][2];
    const uint16_t* lo16[T];
#pragma unroll
    for (int i = 0; i < T; ++i) {
        const int64_t t = t0 + i;
        rows[i][0] = rows[i][1] = nullptr;
        lo16[i] = nullptr;
        if (t >= qb) continue;
        if (!parity) {
            const int64_t rr = static_cast<int64_t>(worker) * qb + t;
            if (rr < q) rows[i][0] = Ap + rr * lda;
        } else {
            const int64_t off = (static_cast<int64_t>(worker - k) * qb + t) * r;
            const float* base = Pp + off;
            rows[i][0] = base;
            if (nplanes == 2) {
                if constexpr (LO16)
                    lo16[i] = reinterpret_cast<const uint16_t*>(Pp + plane) + off;
                else
                    rows[i][1] = base + plane;
            }
        }
    }

    double acc[T];
#pragma unroll
    for (int i = 0; i < T; ++i) acc[i] = 0.0;

    for (int64_t cb = 0; cb < r; cb += kChunk) {
        float4 xv[XR];
#pragma unroll
        for (int j = 0; j < XR; ++j) {
            const int64_t c = cb + tid * 4 + j * NT * 4;
            xv[j] = c < r ? load_global4(x + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < T; ++i) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const float* row = rows[i][h];
                const bool bf = LO16 && h == 1;
                if (bf ? !lo16[i] : !row) continue;
                float4 av[XR];
#pragma unroll
                for (int j = 0; j < XR; ++j) {
                    const int64_t c = cb + tid * 4 + j * NT * 4;
                    // selects, not branches, so the loads stay in flight together
                    if constexpr (LO16) {
                        if (h == 1) continue;
                    }
                    av[j] = c < r ? load_stream(row + c) : make_float4(0.f, 0.f, 0.f, 0.f);
                }
                if constexpr (LO16) {
                    if (h == 1) {
                        u32x2 raw[XR];
#pragma unroll
                        for (int j = 0; j < XR; ++j) {
                            const int64_t c = cb + tid * 4 + j * NT * 4;
                            raw[j] = c < r ? load_stream_bf16x4(lo16[i] + c) : u32x2{0u, 0u};
                        }
#pragma unroll
                        for (int j = 0; j < XR; ++j) av[j] = widen_bf16x4(raw[j]);
                    }
                }
#pragma unroll
                for (int j = 0; j < XR; ++j) {
                    acc[i] = fma(static_cast<double>(av[j].x), static_cast<double>(xv[j].x), acc[i]);
                    acc[i] = fma(static_cast<double>(av[j].y), static_cast<double>(xv[j].y), acc[i]);
                    acc[i] = fma(static_cast<double>(av[j].z), static_cast<double>(xv[j].z), acc[i]);
                    acc[i] = fma(static_cast<double>(av[j].w), static_cast<double>(xv[j].w), acc[i]);
                }
            }
        }
    }
#pragma unroll
    for (int i = 0; i < T; ++i) {
        const double v = wave_sum(acc[i]);
        if (lane == 0) red[wv][i] = v;
    }
    __syncthreads();
    if (tid < T) {
        double v = 0.0;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += red[w][tid];
        const int64_t t = t0 + tid;
        if (t < a.qb) store_y(a, worker, t, 0, v);
    }
}

// General shapes (any r, s, strides): one block row per wave (all planes of a
// parity row), scalar loads, columns of X in groups of SC.  Used for inputs
// the vector GEMV and the matrix-core kernel cannot take (r or lda not a
// multiple of 4, or unaligned pointers).
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
            const RowRef rr = plane_row(a, worker, parity ? t * a.planes + h : t, parity);
            if (!rr.ptr && !rr.p16) continue;
            for (int64_t c = lane; c < a.r; c += 64) {
                const double av = rr.p16 ? bf16_bits_to_f32(rr.p16[c]) : rr.ptr[c];
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

template <int T, int XR>
hipError_t launch_gemv_wg(const WorkerArgs& a, hipStream_t st) {
    const int64_t blocks = ceil_div(a.qb, T) * (a.n_sys + a.n_par);
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    // Rows of 8 column slots per thread: at most three workgroups per compute
    // unit (each requests 40 KB of the 160 KB of LDS, which it does not use),
    // which streams these long rows best (measured: two, three and four).
    const size_t cap = XR >= 8 ? 40 * 1024 : 0;
    if (a.lo_bf16 && a.planes == 2)
        hipLaunchKernelGGL((gemv_wg_kernel<T, XR, 256, true>), dim3(static_cast<unsigned>(blocks)), dim3(256), cap,
                           st, a);
    else
        hipLaunchKernelGGL((gemv_wg_kernel<T, XR, 256, false>), dim3(static_cast<unsigned>(blocks)), dim3(256), cap,
                           st, a);
    return hipGetLastError();
}

template <int XR>
hipError_t launch_gemv_t(const WorkerArgs& a, hipStream_t st) {
    // Four rows per workgroup (x is read once per four rows) unless that
    // leaves fewer than four workgroups per compute unit (256 CUs); then fewer.
    const int64_t workers = a.n_sys + a.n_par;
    if (ceil_div(a.qb, 4) * workers >= 1024) return launch_gemv_wg<4, XR>(a, st);
    if (ceil_div(a.qb, 2) * workers >= 1024) return launch_gemv_wg<2, XR>(a, st);
    return launch_gemv_wg<1, XR>(a, st);
}

hipError_t launch_worker_f32(const WorkerArgs& a, hipStream_t st) {
    if (a.qb == 0) return hipSuccess;
    const bool vec = a.s == 1 && a.ldx == 1 && (a.r % 4 == 0) && (a.lda % 4 == 0) && aligned(a.A, 16) &&
                     aligned(a.X, 16) && (a.parity == nullptr || aligned(a.parity, 16));
    if (vec) {
        // Column slots per thread: the whole row in registers up to 8192 columns.
        if (a.r > 4096) return launch_gemv_t<8>(a, st);
        if (a.r > 2048) return launch_gemv_t<4>(a, st);
        if (a.r > 1024) return launch_gemv_t<2>(a, st);
        return launch_gemv_t<1>(a, st);
    }
    if (gemm_f32_mfma_supported(a)) return launch_gemm_f32_mfma(a, st);
    return launch_waves(gemm_small_f32_kernel<4>, a, a.qb, a.qb, st);
}

}  // namespace coded
