// bf16 worker products Y_i = A'_i X (Sec. III-A: each worker multiplies its
// stored coded block by the multicast input), fp32 accumulation.  The
// matrix-core kernel serves aligned shapes given a workspace; a vector kernel
// serves the rest.
#include "internal.h"
#include <type_traits>

#include "worker_common.h"

namespace coded {
namespace {

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
    const int64_t plane = static_cast<int64_t>(a.n - a.k) * a.qb * a.r;
    const uint16_t* XT = static_cast<const uint16_t*>(a.xt);
    const int64_t ncols = min<int64_t>(16 * NTILE, a.s - c0);
    // Every load in the K loop is unconditional, which lets the loads of a
    // chunk and the next chunk's X^T all be in flight together (a load under
    // a condition makes the compiler wait for everything in flight first).
    // A padding row (past the block, or a systematic row past A) reads a
    // clamped valid row instead: row i of the product depends on row i of
    // the block only, and such rows are stored as zeros or not at all.
    const uint16_t* rp[SLABS][2];
    int64_t trow[SLABS];
#pragma unroll
    for (int sl = 0; sl < SLABS; ++sl) {
        trow[sl] = tile * ROWS + (wv * SLABS + sl) * 16;
        const int64_t t = min<int64_t>(trow[sl] + li, a.qb - 1);
        if (!parity) {
            const int64_t rr = min<int64_t>(static_cast<int64_t>(worker) * a.qb + t, a.q - 1);
            rp[sl][0] = rp[sl][1] = static_cast<const uint16_t*>(a.A) + rr * a.lda;
        } else {
            rp[sl][0] = static_cast<const uint16_t*>(a.parity) + (static_cast<int64_t>(worker - a.k) * a.qb + t) * a.r;
            rp[sl][1] = rp[sl][0] + plane;
        }
    }
    f32x4_t acc[SLABS][NTILE];
#pragma unroll
    for (int sl = 0; sl < SLABS; ++sl)
#pragma unroll
        for (int j = 0; j < NTILE; ++j) acc[sl][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    u32x4_t xr[XV];
    // X^T from clamped addresses; out-of-range values are zeroed when they
    // are stored to LDS, so tail columns of A meet zeros.
    auto xload = [&](int64_t kc) {
#pragma unroll
        for (int i = 0; i < XV; ++i) {
            const int e = tid + kThreads * i;
            const int col = e / (kBK / 8), v = e % (kBK / 8);
            const int64_t k = kc + 8 * v;
            xr[i] = *reinterpret_cast<const u32x4_t*>(XT + (c0 + min<int64_t>(col, ncols - 1)) * a.r +
                                                      min<int64_t>(k, a.r - 8));
        }
    };
    auto xstore = [&](int buf, int64_t kc) {
#pragma unroll
        for (int i = 0; i < XV; ++i) {
            const int e = tid + kThreads * i;
            const int col = e / (kBK / 8), v = e % (kBK / 8);
            const bool ok = col < ncols && kc + 8 * v < a.r;
            if (col < 16 * NTILE)
                *reinterpret_cast<u32x4_t*>(&sXT[buf][col][8 * v]) = ok ? xr[i] : u32x4_t{0u, 0u, 0u, 0u};
        }
    };
    // NPL planes per row (compile time, so the loop has no per-plane branch).
    // The A fragments of chunk c + 1 are loaded while chunk c feeds the
    // matrix cores (two register sets, used alternately).
    auto sweep = [&](auto npl) {
        constexpr int NPL = decltype(npl)::value;
        bf16x8 fa[KS][SLABS][NPL], fb[KS][SLABS][NPL];
        auto aload = [&](int64_t kc, bf16x8 (&af)[KS][SLABS][NPL]) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int64_t k = min<int64_t>(kc + 32 * ks + 8 * lk, a.r - 8);
#pragma unroll
                for (int sl = 0; sl < SLABS; ++sl)
#pragma unroll
                    for (int h = 0; h < NPL; ++h)
                        af[ks][sl][h] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4_t*>(rp[sl][h] + k));
            }
        };
        auto step = [&](int64_t kc, int buf, bf16x8 (&cur)[KS][SLABS][NPL], bf16x8 (&nxt)[KS][SLABS][NPL]) {
            const bool more = kc + kBK < a.r;
            if (more) {
                xload(kc + kBK);
                aload(kc + kBK, nxt);
            }
            // keep the scheduler from sinking these loads into the MFMA
            // sequence (it would serialise them one at a time)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                bf16x8 bfr[NTILE];
#pragma unroll
                for (int j = 0; j < NTILE; ++j)
                    bfr[j] = *reinterpret_cast<const bf16x8*>(&sXT[buf][16 * j + li][32 * ks + 8 * lk]);
#pragma unroll
                for (int sl = 0; sl < SLABS; ++sl)
#pragma unroll
                    for (int h = 0; h < NPL; ++h)
#pragma unroll
                        for (int j = 0; j < NTILE; ++j)
                            acc[sl][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur[ks][sl][h], bfr[j], acc[sl][j], 0, 0, 0);
            }
            if (more) xstore(buf ^ 1, kc + kBK);
            __syncthreads();
        };
        xload(0);
        aload(0, fa);
        xstore(0, 0);
        __syncthreads();
        for (int64_t kc = 0; kc < a.r; kc += 2 * kBK) {
            step(kc, 0, fa, fb);
            if (kc + kBK < a.r) step(kc + kBK, 1, fb, fa);
        }
    };
    if (parity && a.planes == 2)
        sweep(std::integral_constant<int, 2>{});
    else
        sweep(std::integral_constant<int, 1>{});

    float* Y = static_cast<float*>(a.Y);
#pragma unroll
    for (int sl = 0; sl < SLABS; ++sl)
#pragma unroll
        for (int j = 0; j < NTILE; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t t = trow[sl] + 4 * lk + v;
                const int64_t col = 16 * j + li;
                // systematic rows past A are the zero padding of the last block
                const bool inside = parity || static_cast<int64_t>(worker) * a.qb + t < a.q;
                if (t < a.qb && col < ncols)
                    Y[(static_cast<int64_t>(worker) * a.qb + t) * a.s + c0 + col] = inside ? acc[sl][j][v] : 0.0f;
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

int64_t worker_workspace_bytes_bf16(int64_t r, int64_t s) { return (r * s * 2 + 255) / 256 * 256; }

hipError_t launch_transpose_x_bf16(const WorkerArgs& a, hipStream_t st) {
    if (a.r == 0 || a.s == 0) return hipSuccess;
    const int64_t tr = ceil_div(a.r, 64), ts = ceil_div(a.s, 64);
    hipLaunchKernelGGL(transpose_x_bf16_kernel, dim3(static_cast<unsigned>(tr * ts)), dim3(256), 0, st,
                       static_cast<const uint16_t*>(a.X), a.r, a.s, a.ldx, static_cast<uint16_t*>(a.xt), ts);
    return hipGetLastError();
}

hipError_t launch_worker_bf16(const WorkerArgs& a, hipStream_t st) {
    if (a.qb == 0 || a.s == 0) return hipSuccess;
    const bool mfma = a.xt != nullptr && a.r > 0 && a.r % 8 == 0 && a.lda % 8 == 0 && aligned(a.A, 16) &&
                      (a.parity == nullptr || aligned(a.parity, 16)) && aligned(a.xt, 16);
    if (!mfma) return launch_waves(gemm_small_bf16_kernel<4>, a, a.qb, a.qb, st);
    hipError_t e = a.xt_ready ? hipSuccess : launch_transpose_x_bf16(a, st);
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
