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
// in fp64.  s > 1 and unaligned shapes take a general kernel.
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

// s == 1, 16-byte vectors.  A workgroup of NT threads owns a tile of T
// consecutive rows of one worker's block and sweeps it one row at a time:
// thread tid covers column slots c = tid*4 + j*NT*4 (j < XR) of every row, so
// each load instruction of the workgroup reads NT*16 contiguous bytes, and
// its slice of x stays in registers for all T rows.  Rows wider than
// NT*4*XR are swept in column chunks (x reloaded per chunk).  A parity row's
// planes (hi, lo) are summed into the same fp64 accumulator.  Partial sums
// are combined across lanes (shuffles) and waves (LDS) in a fixed order.
template <int T, int XR, int NT>
__global__ __launch_bounds__(NT) void gemv_wg_kernel(WorkerArgs a) {
    constexpr int NW = NT / 64;
    constexpr int kChunk = NT * 4 * XR;
    __shared__ double red[NW][T];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t groups = ceil_div(a.qb, T);
    const int64_t npar = groups * a.n_par;
    const int64_t g = blockIdx.x;
    int worker;
    int64_t grp;
    bool parity;
    // Parity workgroups stream `planes` times the bytes: dispatch them first so
    // the launch does not end on a tail of long workgroups.
    if (g < npar) {
        worker = a.par_ids[g / groups];
        grp = g % groups;
        parity = true;
    } else {
        if (g - npar >= groups * a.n_sys) return;
        worker = a.sys_ids[(g - npar) / groups];
        grp = (g - npar) % groups;
        parity = false;
    }
    const int64_t t0 = grp * T;
    const int nplanes = parity ? a.planes : 1;
    const int64_t plane = static_cast<int64_t>(a.n - a.k) * a.qb * a.r;
    const float* x = static_cast<const float*>(a.X);

    // Row pointers of the tile (null: padding row or beyond the block).
    const float* rows[T][2];
#pragma unroll
    for (int i = 0; i < T; ++i) {
        const int64_t t = t0 + i;
        rows[i][0] = rows[i][1] = nullptr;
        if (t >= a.qb) continue;
        if (!parity) {
            const int64_t rr = static_cast<int64_t>(worker) * a.qb + t;
            if (rr < a.q) rows[i][0] = static_cast<const float*>(a.A) + rr * a.lda;
        } else {
            const float* base = static_cast<const float*>(a.parity) + (static_cast<int64_t>(worker - a.k) * a.qb + t) * a.r;
            rows[i][0] = base;
            if (nplanes == 2) rows[i][1] = base + plane;
        }
    }

    double acc[T];
#pragma unroll
    for (int i = 0; i < T; ++i) acc[i] = 0.0;

    for (int64_t cb = 0; cb < a.r; cb += kChunk) {
        float4 xv[XR];
#pragma unroll
        for (int j = 0; j < XR; ++j) {
            const int64_t c = cb + tid * 4 + j * NT * 4;
            xv[j] = c < a.r ? *reinterpret_cast<const float4*>(x + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < T; ++i) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const float* row = rows[i][h];
                if (!row) continue;
                float4 av[XR];
#pragma unroll
                for (int j = 0; j < XR; ++j) {
                    const int64_t c = cb + tid * 4 + j * NT * 4;
                    av[j] = c < a.r ? load_stream(row + c) : make_float4(0.f, 0.f, 0.f, 0.f);
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


// ---------------------------------------------------------------- bf16, matrix cores
// Worker products of bf16 blocks with a bf16 X of up to 64 columns per pass,
// fp32 accumulation on v_mfma_f32_16x16x32_bf16.  Lane layouts (checked on
// the device): A operand lane l element e = A[l%16][8*(l/16)+e], B operand
// lane l element e = B[8*(l/16)+e][l%16], result lane l item v =
// C[4*(l/16)+v][l%16].  Both operands are read along K in 16-byte pieces, so
// X is first transposed (X^T, s x r) into the workspace.  A workgroup of four
// wavefronts owns 4*SLABS*16 rows of one worker's block.  X^T is staged in
// LDS in K chunks of kBK, double-buffered: the next chunk is read into
// registers while the current one feeds the matrix cores, so each chunk costs
// one barrier.  A fragments are plain 16-byte loads: each instruction reads
// 64 bytes of 16 rows, and the other half of every 128-byte line is read by
// the next instruction, which a non-temporal hint would evict first.  A
// parity row's hi and lo planes accumulate into the same tile; parity
// workgroups (twice the bytes) are scheduled first.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kBK = 64;      // K chunk of X^T staged in LDS
constexpr int kXPad = 8;     // bf16 padding per LDS row (spreads the 16-byte reads over banks)

template <int NTILE, int SLABS>
__global__ __launch_bounds__(kThreads) void gemm_bf16_mfma_kernel(WorkerArgs a, int64_t tiles, int64_t c0) {
    constexpr int ROWS = kWaves * SLABS * 16;
    constexpr int KS = kBK / 32;
    constexpr int XV = (16 * NTILE * (kBK / 8) + kThreads - 1) / kThreads;   // X^T vectors per thread per chunk
    __shared__ __align__(16) uint16_t sXT[2][16 * NTILE][kBK + kXPad];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int li = lane & 15, lk = lane >> 4;
    const int64_t g = blockIdx.x;
    const int64_t npar = tiles * a.n_par;
    int worker;
    int64_t tile;
    bool parity;
    if (g < npar) {
        worker = a.par_ids[g / tiles];
        tile = g % tiles;
        parity = true;
    } else {
        worker = a.sys_ids[(g - npar) / tiles];
        tile = (g - npar) % tiles;
        parity = false;
    }
    const int nplanes = parity ? a.planes : 1;
    const int64_t plane = static_cast<int64_t>(a.n - a.k) * a.qb * a.r;
    const uint16_t* XT = static_cast<const uint16_t*>(a.xt);
    const int64_t ncols = min<int64_t>(16 * NTILE, a.s - c0);
    const uint16_t* rp[SLABS][2];
    int64_t trow[SLABS];
#pragma unroll
    for (int sl = 0; sl < SLABS; ++sl) {
        trow[sl] = tile * ROWS + (wv * SLABS + sl) * 16;
        const int64_t t = trow[sl] + li;
        rp[sl][0] = rp[sl][1] = nullptr;
        if (t < a.qb) {
            if (!parity) {
                const int64_t rr = static_cast<int64_t>(worker) * a.qb + t;
                if (rr < a.q) rp[sl][0] = static_cast<const uint16_t*>(a.A) + rr * a.lda;
            } else {
                const uint16_t* base =
                    static_cast<const uint16_t*>(a.parity) + (static_cast<int64_t>(worker - a.k) * a.qb + t) * a.r;
                rp[sl][0] = base;
                if (nplanes == 2) rp[sl][1] = base + plane;
            }
        }
    }
    f32x4_t acc[SLABS][NTILE];
#pragma unroll
    for (int sl = 0; sl < SLABS; ++sl)
#pragma unroll
        for (int j = 0; j < NTILE; ++j) acc[sl][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const bf16x8 zero8 = __builtin_bit_cast(bf16x8, u32x4_t{0u, 0u, 0u, 0u});

    u32x4_t xr[XV];
    auto xload = [&](int64_t kc) {
#pragma unroll
        for (int i = 0; i < XV; ++i) {
            const int e = tid + kThreads * i;
            const int col = e / (kBK / 8), v = e % (kBK / 8);
            const int64_t k = kc + 8 * v;
            xr[i] = (col < ncols && k < a.r) ? *reinterpret_cast<const u32x4_t*>(XT + (c0 + col) * a.r + k)
                                             : u32x4_t{0u, 0u, 0u, 0u};
        }
    };
    auto xstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < XV; ++i) {
            const int e = tid + kThreads * i;
            const int col = e / (kBK / 8), v = e % (kBK / 8);
            if (col < 16 * NTILE) *reinterpret_cast<u32x4_t*>(&sXT[buf][col][8 * v]) = xr[i];
        }
    };
    xload(0);
    xstore(0);
    __syncthreads();
    int buf = 0;
    for (int64_t kc = 0; kc < a.r; kc += kBK) {
        bf16x8 af[KS][SLABS][2];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int64_t k = kc + 32 * ks + 8 * lk;
#pragma unroll
            for (int sl = 0; sl < SLABS; ++sl)
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    af[ks][sl][h] = (rp[sl][h] && h < nplanes && k < a.r)
                                        ? __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4_t*>(rp[sl][h] + k))
                                        : zero8;
        }
        const bool more = kc + kBK < a.r;
        if (more) xload(kc + kBK);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            bf16x8 bfr[NTILE];
#pragma unroll
            for (int j = 0; j < NTILE; ++j)
                bfr[j] = *reinterpret_cast<const bf16x8*>(&sXT[buf][16 * j + li][32 * ks + 8 * lk]);
#pragma unroll
            for (int sl = 0; sl < SLABS; ++sl)
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    if (h < nplanes)
#pragma unroll
                        for (int j = 0; j < NTILE; ++j)
                            acc[sl][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[ks][sl][h], bfr[j], acc[sl][j], 0, 0, 0);
        }
        if (more) xstore(buf ^ 1);
        __syncthreads();
        buf ^= 1;
    }
    float* Y = static_cast<float*>(a.Y);
#pragma unroll
    for (int sl = 0; sl < SLABS; ++sl)
#pragma unroll
        for (int j = 0; j < NTILE; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t t = trow[sl] + 4 * lk + v;
                const int64_t col = 16 * j + li;
                if (t < a.qb && col < ncols) Y[(static_cast<int64_t>(worker) * a.qb + t) * a.s + c0 + col] = acc[sl][j][v];
            }
}

// X (r x s, row stride ldx) -> X^T (s x r) in 64 x 64 tiles through LDS.
__global__ __launch_bounds__(256) void transpose_x_bf16_kernel(const uint16_t* __restrict__ X, int64_t r, int64_t s,
                                                               int64_t ldx, uint16_t* __restrict__ XT, int64_t tiles_s) {
    __shared__ uint16_t tile[64][65];
    const int64_t tr = blockIdx.x / tiles_s, ts = blockIdx.x % tiles_s;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int64_t k = tr * 64 + i, c = ts * 64 + tx;
        tile[i][tx] = (k < r && c < s) ? X[k * ldx + c] : static_cast<uint16_t>(0);
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int64_t c = ts * 64 + i, k = tr * 64 + tx;
        if (c < s && k < r) XT[c * r + k] = tile[tx][i];
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
    hipLaunchKernelGGL((gemv_wg_kernel<T, XR, 256>), dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, a);
    return hipGetLastError();
}

template <int XR>
hipError_t launch_gemv_t(const WorkerArgs& a, hipStream_t st) {
    // Four rows per workgroup unless that leaves too few workgroups to fill
    // the chip (256 CUs); then fewer.
    const int64_t workers = a.n_sys + a.n_par;
    if (ceil_div(a.qb, 4) * workers >= 4096) return launch_gemv_wg<4, XR>(a, st);
    if (ceil_div(a.qb, 2) * workers >= 4096) return launch_gemv_wg<2, XR>(a, st);
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
    return launch_waves(gemm_small_f32_kernel<4>, a, a.qb, a.qb, st);
}

int64_t worker_workspace_bytes_bf16(int64_t r, int64_t s) { return (r * s * 2 + 255) / 256 * 256; }

hipError_t launch_worker_bf16(const WorkerArgs& a, hipStream_t st) {
    if (a.qb == 0 || a.s == 0) return hipSuccess;
    const bool mfma = a.xt != nullptr && a.r > 0 && a.r % 8 == 0 && a.lda % 8 == 0 && aligned(a.A, 16) &&
                      (a.parity == nullptr || aligned(a.parity, 16)) && aligned(a.xt, 16);
    if (!mfma) return launch_waves(gemm_small_bf16_kernel<4>, a, a.qb, a.qb, st);
    const int64_t tr = ceil_div(a.r, 64), ts = ceil_div(a.s, 64);
    hipLaunchKernelGGL(transpose_x_bf16_kernel, dim3(static_cast<unsigned>(tr * ts)), dim3(256), 0, st,
                       static_cast<const uint16_t*>(a.X), a.r, a.s, a.ldx, static_cast<uint16_t*>(a.xt), ts);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    constexpr int SLABS = 2, ROWS = kWaves * SLABS * 16;
    const int64_t tiles = ceil_div(a.qb, ROWS);
    const int64_t blocks = tiles * (a.n_sys + a.n_par);
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    for (int64_t c0 = 0; c0 < a.s; c0 += 64) {
        const int64_t cols = std::min<int64_t>(64, a.s - c0);
        if (cols > 32)
            hipLaunchKernelGGL((gemm_bf16_mfma_kernel<4, SLABS>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0,
                               st, a, tiles, c0);
        else if (cols > 16)
            hipLaunchKernelGGL((gemm_bf16_mfma_kernel<2, SLABS>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0,
                               st, a, tiles, c0);
        else
            hipLaunchKernelGGL((gemm_bf16_mfma_kernel<1, SLABS>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0,
                               st, a, tiles, c0);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace coded
