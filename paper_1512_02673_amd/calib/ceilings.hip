// Device ceilings of the part the library runs on, measured by plain probe
// kernels: HBM read and write bandwidth for streaming and for the row-window
// read patterns the worker kernels use, and the sustained rates of the matrix
// instructions the kernels issue.  The design figures are quoted against
// these numbers next to the published peaks.  Every entry point times its
// kernel with HIP events on the null stream and returns milliseconds per
// launch (a mean over `reps` launches after two untimed ones).
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef double d4 __attribute__((ext_vector_type(4)));
typedef float fl4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

// Grid-stride streaming read, eight 16-byte non-temporal loads in flight per thread.
__global__ __launch_bounds__(256) void read_stream(const f4* __restrict__ p, int64_t n4, float* out) {
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
    int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    for (; i + 7 * stride < n4; i += 8 * stride) {
        f4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc += v[u];
    }
    for (; i < n4; i += stride) acc += __builtin_nontemporal_load(p + i);
    if (acc.x + acc.y + acc.z + acc.w == 1.2345678e30f) out[0] = acc.x;   // keeps the loads
}

// Grid-stride streaming write of 16-byte pieces (NT: non-temporal stores).
template <bool NT>
__global__ __launch_bounds__(256) void write_stream(f4* __restrict__ p, int64_t n4) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
    const f4 v = {1.f, 2.f, 3.f, 4.f};
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n4; i += stride) {
        if constexpr (NT)
            __builtin_nontemporal_store(v, p + i);
        else
            p[i] = v;
    }
}

// Row-window reads: a workgroup of 256 threads streams R rows of r floats in
// chunks of KC columns, PF chunks in flight (16-byte non-temporal loads, KC/4
// consecutive threads per row), optionally staging each chunk through LDS
// with a barrier as the matrix-core kernels do.  Prefetches past the last
// chunk read the matrix's first 16 bytes.
template <int R, int KC, int PF, bool LDS>
__global__ __launch_bounds__(256) void read_rows(const float* __restrict__ A, int64_t rows, int r, float* out) {
    constexpr int NL = R * KC / 4 / 256;
    __shared__ f4 sm[LDS ? 2 * R * (KC / 4 + 1) : 1];
    const int tid = threadIdx.x;
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * R;
    const float* rp[NL];
    int col[NL], ofs[NL];
#pragma unroll
    for (int p = 0; p < NL; ++p) {
        const int f = tid + 256 * p;
        const int rho = f / (KC / 4);
        col[p] = (f % (KC / 4)) * 4;
        ofs[p] = rho * (KC / 4 + 1) + f % (KC / 4);
        const int64_t row = r0 + rho < rows ? r0 + rho : rows - 1;
        rp[p] = A + row * r;
    }
    const int nch = r / KC;
    f4 ring[PF][NL];
    f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < PF; ++j)
#pragma unroll
        for (int p = 0; p < NL; ++p)
            ring[j][p] = __builtin_nontemporal_load(reinterpret_cast<const f4*>(j < nch ? rp[p] + j * KC + col[p] : A));
    for (int cb = 0; cb < nch; cb += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int c = cb + j;
            if (c >= nch) break;
            if constexpr (LDS) {
#pragma unroll
                for (int p = 0; p < NL; ++p) sm[(c & 1) * R * (KC / 4 + 1) + ofs[p]] = ring[j][p];
                __syncthreads();
                acc += sm[(c & 1) * R * (KC / 4 + 1) + (tid * 7) % (R * (KC / 4))];
            } else {
#pragma unroll
                for (int p = 0; p < NL; ++p) acc += ring[j][p];
            }
            const bool more = c + PF < nch;
#pragma unroll
            for (int p = 0; p < NL; ++p)
                ring[j][p] = __builtin_nontemporal_load(reinterpret_cast<const f4*>(more ? rp[p] + (c + PF) * KC + col[p] : A));
        }
    }
#pragma unroll
    for (int j = 0; j < PF; ++j)
#pragma unroll
        for (int p = 0; p < NL; ++p) acc += ring[j][p];
    if (acc.x + acc.y + acc.z + acc.w == 1.2345678e30f) out[0] = acc.x;
}

// The memory pattern of the bf16 single pass (encode + products) with nothing
// else: a 512-thread workgroup per compute unit walks an equal run of units
// (16-row tile, column range of RUN = max(RUNR, RUNW) bytes) of a (k = 24,
// n - k = 8) code, reading the tile's 16 rows of all 24 blocks and writing 16
// rows of each of the 16 parity rows (8 per plane), with the next unit's
// loads in flight (two register sets).  A wave's load instruction covers
// 1024 / RUNR rows x RUNR contiguous bytes, a store 1024 / RUNW rows x RUNW
// bytes (RUN / RUNR such runs of a row are read by successive instructions).
// Rows past q read the last row; rows past a block's end are not written.
struct TileArgs {
    const uint16_t* A;   // q x r bf16
    uint16_t* P;         // 2 planes x 8 x qb x r bf16
    int64_t q, r, qb, ranges, units, per;
};

template <int RUNR, int RUNW>
__global__ __launch_bounds__(512, 1) void tile_pattern(TileArgs a) {
    constexpr int RUN = RUNR > RUNW ? RUNR : RUNW;
    constexpr int T = 512, PRr = RUNR / 16, PRw = RUNW / 16;   // lanes per row run
    constexpr int LD = 24 * 16 * (RUN / 16) / T, ST = 16 * 16 * (RUN / 16) / T;
    const int tid = threadIdx.x;
    const int64_t u0 = static_cast<int64_t>(blockIdx.x) * a.per;
    const int64_t u1 = u0 + a.per < a.units ? u0 + a.per : a.units;
    if (u0 >= u1) return;
    f4 R[2][LD];
    auto load = [&](int set, int64_t u) __attribute__((always_inline)) {
        const int64_t t0 = (u / a.ranges) * 16, c0 = (u % a.ranges) * (RUN / 2);
#pragma unroll
        for (int i = 0; i < LD; ++i) {
            // piece e: run qq of the row outermost, then block row, then lane in the run
            const int e = tid + T * i;
            const int pc = e % PRr, jrow = (e / PRr) % 384, qq = e / (PRr * 384);
            const int j = jrow / 16, row = jrow % 16;
            const int64_t t = t0 + row < a.qb ? t0 + row : a.qb - 1;
            const int64_t g = j * a.qb + t < a.q ? j * a.qb + t : a.q - 1;
            R[set][i] = *reinterpret_cast<const f4*>(a.A + g * a.r + c0 + (qq * PRr + pc) * 8);
        }
    };
    auto store = [&](int set, int64_t u) __attribute__((always_inline)) {
        const int64_t t0 = (u / a.ranges) * 16, c0 = (u % a.ranges) * (RUN / 2);
#pragma unroll
        for (int i = 0; i < ST; ++i) {
            const int e = tid + T * i;
            const int pc = e % PRw, prow = (e / PRw) % 256, qq = e / (PRw * 256);
            const int pl = prow / 16, row = prow % 16;
            if (t0 + row < a.qb) {
                const int64_t off = ((pl / 8) * 8 * a.qb + (pl % 8) * a.qb + t0 + row) * a.r + c0 + (qq * PRw + pc) * 8;
                __builtin_nontemporal_store(R[set][i % LD] + R[set][(i + 1) % LD], reinterpret_cast<f4*>(a.P + off));
            }
        }
    };
    load(0, u0);
    for (int64_t u = u0; u < u1; u += 2) {
        if (u + 1 < u1) load(1, u + 1);
        store(0, u);
        if (u + 2 < u1) load(0, u + 2);
        if (u + 1 < u1) store(1, u + 1);
    }
}

// Matrix-instruction rates: CH independent accumulator chains per wave,
// `iters` rounds; the result is written so nothing is optimised away.
template <int CH>
__global__ __launch_bounds__(256) void rate_f64_16x16x4(int iters, double* out) {
    const double a = 1.0 + threadIdx.x * 1e-9, b = 1.0 - threadIdx.x * 1e-9;
    d4 acc[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[c] = d4{0.0, 0.0, 0.0, 0.0};
    for (int it = 0; it < iters; ++it)
#pragma unroll
        for (int c = 0; c < CH; ++c) acc[c] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc[c], 0, 0, 0);
    double s = 0.0;
#pragma unroll
    for (int c = 0; c < CH; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
    out[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = s;
}

template <int CH>
__global__ __launch_bounds__(256) void rate_f64_4x4x4(int iters, double* out) {
    const double a = 1.0 + threadIdx.x * 1e-9, b = 1.0 - threadIdx.x * 1e-9;
    double acc[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[c] = 0.0;
    for (int it = 0; it < iters; ++it)
#pragma unroll
        for (int c = 0; c < CH; ++c) acc[c] = __builtin_amdgcn_mfma_f64_4x4x4f64(a, b, acc[c], 0, 0, 0);
    double s = 0.0;
#pragma unroll
    for (int c = 0; c < CH; ++c) s += acc[c];
    out[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = s;
}

template <int CH>
__global__ __launch_bounds__(256) void rate_bf16_16x16x32(int iters, double* out) {
    bf8 a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = static_cast<__bf16>(1.0f + (threadIdx.x + e) * 1e-3f);
        b[e] = static_cast<__bf16>(1.0f - e * 1e-3f);
    }
    fl4 acc[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[c] = fl4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it)
#pragma unroll
        for (int c = 0; c < CH; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[c], 0, 0, 0);
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < CH; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
    out[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = s;
}

// Vector fp64 FMA rate: CH independent chains per lane.
template <int CH>
__global__ __launch_bounds__(256) void rate_fma64(int iters, double* out) {
    double acc[CH];
    const double m = 1.0 + threadIdx.x * 1e-12, ad = 1e-9;
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[c] = c;
    for (int it = 0; it < iters; ++it)
#pragma unroll
        for (int c = 0; c < CH; ++c) acc[c] = fma(acc[c], m, ad);
    double s = 0.0;
#pragma unroll
    for (int c = 0; c < CH; ++c) s += acc[c];
    out[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = s;
}

template <typename F>
int time_ms(F launch, int reps, float* ms_out) {
    hipEvent_t e0, e1;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return 1;
    for (int i = 0; i < 2; ++i) launch();
    if (hipGetLastError() != hipSuccess || hipDeviceSynchronize() != hipSuccess) return 1;
    hipEventRecord(e0, nullptr);
    for (int i = 0; i < reps; ++i) launch();
    hipEventRecord(e1, nullptr);
    if (hipEventSynchronize(e1) != hipSuccess) return 1;
    float ms = 0.f;
    hipEventElapsedTime(&ms, e0, e1);
    *ms_out = ms / reps;
    hipEventDestroy(e0);
    hipEventDestroy(e1);
    return hipGetLastError() == hipSuccess ? 0 : 1;
}

}  // namespace

extern "C" {

// Streaming read of `bytes` (a multiple of 16) from device buffer `buf` with `blocks` workgroups.
int calib_read(const void* buf, int64_t bytes, int blocks, int reps, float* scratch, float* ms) {
    return time_ms([&] { hipLaunchKernelGGL(read_stream, dim3(blocks), dim3(256), 0, nullptr,
                                            static_cast<const f4*>(buf), bytes / 16, scratch); }, reps, ms);
}

// Streaming write of `bytes` (a multiple of 16); nontemporal selects the store hint.
int calib_write(void* buf, int64_t bytes, int blocks, int nontemporal, int reps, float* ms) {
    if (nontemporal)
        return time_ms([&] { hipLaunchKernelGGL(write_stream<true>, dim3(blocks), dim3(256), 0, nullptr,
                                                static_cast<f4*>(buf), bytes / 16); }, reps, ms);
    return time_ms([&] { hipLaunchKernelGGL(write_stream<false>, dim3(blocks), dim3(256), 0, nullptr,
                                            static_cast<f4*>(buf), bytes / 16); }, reps, ms);
}

// Row-window reads of a rows x r fp32 matrix (r a multiple of 4096).  pattern:
// 0: 1 row x 16 KB chunks; 1: 4 rows x 4 KB, 2 in flight; 2: 8 rows x 1 KB, 8 in
// flight, LDS; 3: 16 rows x 512 B, 4 in flight, LDS.
int calib_read_rows(const float* A, int64_t rows, int r, int pattern, int reps, float* scratch, float* ms) {
    if (r <= 0 || r % 4096 != 0 || rows <= 0) return 2;
    switch (pattern) {
        case 0:
            return time_ms([&] { hipLaunchKernelGGL((read_rows<1, 4096, 1, false>), dim3(rows), dim3(256), 0, nullptr,
                                                    A, rows, r, scratch); }, reps, ms);
        case 1:
            return time_ms([&] { hipLaunchKernelGGL((read_rows<4, 1024, 2, false>), dim3((rows + 3) / 4), dim3(256), 0,
                                                    nullptr, A, rows, r, scratch); }, reps, ms);
        case 2:
            return time_ms([&] { hipLaunchKernelGGL((read_rows<8, 256, 8, true>), dim3((rows + 7) / 8), dim3(256), 0,
                                                    nullptr, A, rows, r, scratch); }, reps, ms);
        case 3:
            return time_ms([&] { hipLaunchKernelGGL((read_rows<16, 128, 4, true>), dim3((rows + 15) / 16), dim3(256),
                                                    0, nullptr, A, rows, r, scratch); }, reps, ms);
    }
    return 2;
}

// The single pass's memory pattern (tile_pattern above) over a q x r bf16
// matrix A (r a multiple of 256) and parity planes P of 2 x 8 x ceil(q/24) x r
// bf16, both device buffers, with read and write runs of run_read and
// run_write bytes per row (128, 256 or 512 each; the pairs 128/128, 256/256,
// 512/512, 512/128 and 512/256); one workgroup per compute unit (`cus`).  Bytes moved
// per launch: 2 q r read + 4 x 8 x ceil(q/24) x r written.
int calib_tile_pattern(const void* A, void* P, int64_t q, int64_t r, int run_read, int run_write, int cus, int reps,
                       float* ms) {
    if (q <= 0 || r <= 0 || r % 256 != 0 || cus <= 0) return 2;
    TileArgs a{static_cast<const uint16_t*>(A), static_cast<uint16_t*>(P), q, r, (q + 23) / 24, 0, 0, 0};
    const int run = run_read > run_write ? run_read : run_write;
    a.ranges = r * 2 / run;
    a.units = (a.qb + 15) / 16 * a.ranges;
    a.per = (a.units + cus - 1) / cus;
    a.per = a.per > a.ranges ? a.per : a.ranges;
    const unsigned blocks = static_cast<unsigned>((a.units + a.per - 1) / a.per);
    auto go = [&](auto kernel) { return time_ms([&] { hipLaunchKernelGGL(kernel, dim3(blocks), dim3(512), 0, nullptr, a); }, reps, ms); };
    if (run_read == 128 && run_write == 128) return go(tile_pattern<128, 128>);
    if (run_read == 256 && run_write == 256) return go(tile_pattern<256, 256>);
    if (run_read == 512 && run_write == 512) return go(tile_pattern<512, 512>);
    if (run_read == 512 && run_write == 128) return go(tile_pattern<512, 128>);
    if (run_read == 512 && run_write == 256) return go(tile_pattern<512, 256>);
    return 2;
}

// Matrix-instruction and vector rates.  kind: 0 v_mfma_f64_16x16x4f64, 1
// v_mfma_f64_4x4x4f64, 2 v_mfma_f32_16x16x32_bf16, 3 v_fma_f64.  `blocks`
// workgroups of 4 waves, `iters` rounds of 8 independent chains; out must hold
// blocks * 256 doubles.  flops_out: flops executed per launch.
int calib_rate(int kind, int blocks, int iters, int reps, double* out, double* flops_out, float* ms) {
    const double waves = blocks * 4.0, chains = 8.0;
    switch (kind) {
        case 0:
            *flops_out = waves * iters * chains * 2.0 * 16 * 16 * 4;
            return time_ms([&] { hipLaunchKernelGGL(rate_f64_16x16x4<8>, dim3(blocks), dim3(256), 0, nullptr, iters,
                                                    out); }, reps, ms);
        case 1:
            *flops_out = waves * iters * chains * 2.0 * 4 * 4 * 4 * 4;
            return time_ms([&] { hipLaunchKernelGGL(rate_f64_4x4x4<8>, dim3(blocks), dim3(256), 0, nullptr, iters,
                                                    out); }, reps, ms);
        case 2:
            *flops_out = waves * iters * chains * 2.0 * 16 * 16 * 32;
            return time_ms([&] { hipLaunchKernelGGL(rate_bf16_16x16x32<8>, dim3(blocks), dim3(256), 0, nullptr, iters,
                                                    out); }, reps, ms);
        case 3:
            *flops_out = waves * 64.0 * iters * chains * 2.0;
            return time_ms([&] { hipLaunchKernelGGL(rate_fma64<8>, dim3(blocks), dim3(256), 0, nullptr, iters, out); },
                           reps, ms);
    }
    return 2;
}

}  // extern "C"
