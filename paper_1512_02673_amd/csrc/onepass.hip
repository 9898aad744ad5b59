// One launch for the whole coded product of a small fp32 problem with one
// column (Sec. III-A: encode, the n worker products, dec(indices, results)).
//
// Every step works along block rows: parity row t is sum_j P[p][j] A_j[t],
// worker i's result at t is its row t times x, and the decoded outputs at t
// need only the survivors' results at t.  So one workgroup per block row t
// reads row t of the k data blocks once, forms the parity rows (writing both
// planes, or reads the stored planes), computes all n products into Y, and
// decodes the k outputs of that row: systematic survivors are copied, the
// missing blocks are sum_c D[b][c] Y_{S[c]}[t] with the decoding matrix D
// eliminated by wave 0 while the other waves stream.  For a problem of a
// few MB this replaces three launch latencies with one.
//
// The parity arithmetic is the encode kernel's, element for element (fp64
// fma chain over j in order, hi = round(sum), lo = round(sum - hi)), so the
// stored planes equal coded_encode's bit for bit.  Products are exact in
// fp64 and summed in fp64.
#include "internal.h"
#include "decode_common.h"
#include "worker_common.h"

namespace coded {
namespace {

typedef float f32x4o __attribute__((ext_vector_type(4)));

__device__ inline f32x4o load4(const float* p) { return *reinterpret_cast<const f32x4o*>(p); }

__device__ inline double dot4(f32x4o a, f32x4o x, double acc) {
    acc = fma(static_cast<double>(a.x), static_cast<double>(x.x), acc);
    acc = fma(static_cast<double>(a.y), static_cast<double>(x.y), acc);
    acc = fma(static_cast<double>(a.z), static_cast<double>(x.z), acc);
    acc = fma(static_cast<double>(a.w), static_cast<double>(x.w), acc);
    return acc;
}

template <int NT>
__global__ __launch_bounds__(NT) void onepass_f32_kernel(OnePassArgs a) {
    constexpr int NW = NT / 64;
    constexpr int MN = kOnePassMaxN;
    __shared__ SetMeta sm;
    __shared__ double sD[64 * kFastLd];
    __shared__ double sP[MN * MN];
    __shared__ double red[NW][MN];
    __shared__ double sy[MN];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int n = a.n, k = a.k, npar = n - k;
    const int64_t t = blockIdx.x;

    DecodeArgs da{};
    da.G = a.G;
    da.info = a.info;
    da.q = a.q;
    da.qb = a.qb;
    da.s = 1;
    da.ldo = a.ldo;
    da.n = n;
    da.k = k;
    da.batch = 1;
    setup_set<NT>(da, a.set, 0, false, sm);     // the host has checked the set
    for (int e = tid; e < npar * k; e += NT) sP[e] = a.G[static_cast<int64_t>(k) * k + e];
    __syncthreads();
    const int m = sm.m;
    if (m > 0 && wv == 0) eliminate_wave(da, sm, m, k - m, lane, sD);   // read after the barrier below

    // Row t of the data blocks (zero past q), the parity rows, and the n products.
    double y[MN];
#pragma unroll
    for (int i = 0; i < MN; ++i) y[i] = 0.0;
    int kin = 0;                                  // data blocks whose row t lies inside A
    while (kin < k && static_cast<int64_t>(kin) * a.qb + t < a.q) ++kin;
    const int64_t plane = static_cast<int64_t>(npar) * a.qb * a.r;
    for (int64_t c = static_cast<int64_t>(tid) * 4; c < a.r; c += NT * 4) {
        const f32x4o xv = load4(a.x + c);
        f32x4o av[MN];
#pragma unroll
        for (int j = 0; j < MN; ++j) {
            av[j] = f32x4o{0.f, 0.f, 0.f, 0.f};
            if (j < kin) av[j] = load4(a.A + (static_cast<int64_t>(j) * a.qb + t) * a.lda + c);
        }
#pragma unroll
        for (int j = 0; j < MN; ++j)
            if (j < kin) y[j] = dot4(av[j], xv, y[j]);
        for (int p = 0; p < npar; ++p) {
            float* prow = a.parity + (static_cast<int64_t>(p) * a.qb + t) * a.r + c;
            f32x4o hi, lo = f32x4o{0.f, 0.f, 0.f, 0.f};
            if (a.encode) {
                double s4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
                for (int j = 0; j < MN; ++j) {
                    if (j < kin) {
                        const double g = sP[p * k + j];
                        s4[0] = fma(g, static_cast<double>(av[j].x), s4[0]);
                        s4[1] = fma(g, static_cast<double>(av[j].y), s4[1]);
                        s4[2] = fma(g, static_cast<double>(av[j].z), s4[2]);
                        s4[3] = fma(g, static_cast<double>(av[j].w), s4[3]);
                    }
                }
                hi = f32x4o{static_cast<float>(s4[0]), static_cast<float>(s4[1]), static_cast<float>(s4[2]),
                            static_cast<float>(s4[3])};
                *reinterpret_cast<f32x4o*>(prow) = hi;
                if (a.planes == 2) {
                    lo = f32x4o{static_cast<float>(s4[0] - static_cast<double>(hi.x)),
                                static_cast<float>(s4[1] - static_cast<double>(hi.y)),
                                static_cast<float>(s4[2] - static_cast<double>(hi.z)),
                                static_cast<float>(s4[3] - static_cast<double>(hi.w))};
                    *reinterpret_cast<f32x4o*>(prow + plane) = lo;
                }
            } else {
                hi = load4(prow);
                if (a.planes == 2) lo = load4(prow + plane);
            }
            // the worker multiplies its stored planes: hi, then lo
            double yp = dot4(hi, xv, 0.0);
            if (a.planes == 2) yp = dot4(lo, xv, yp);
#pragma unroll
            for (int i = 0; i < MN; ++i)
                if (i == k + p) y[i] += yp;
        }
    }
#pragma unroll
    for (int i = 0; i < MN; ++i) {
        if (i < n) {
            const double v = wave_sum(y[i]);
            if (lane == 0) red[wv][i] = v;
        }
    }
    __syncthreads();
    if (tid < n) {
        double v = 0.0;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += red[w][tid];
        sy[tid] = v;
        a.Y[static_cast<int64_t>(tid) * a.qb + t] = v;
    }
    __syncthreads();

    // Decode block row t (out is not written for a singular survivor system).
    const int status = sm.status;
    if (t == 0 && tid == 0) a.info[0] = status;
    if (status != 0 || tid >= k) return;
    const int j = tid;
    if (t >= sm.lim[j]) return;                  // padding row
    double v;
    if (sm.present[j]) {
        v = sy[j];
    } else {
        int b = 0;                               // rank of j among the missing blocks
        for (int i = 0; i < j; ++i) b += sm.present[i] ? 0 : 1;
        v = 0.0;
        for (int c = 0; c < k; ++c) v = fma(sD[c * kFastLd + b], sy[sm.S[c]], v);
    }
    a.out[(static_cast<int64_t>(j) * a.qb + t) * a.ldo] = static_cast<float>(v);
}

bool aligned16p(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

bool onepass_supported(int n, int k, int64_t q, int64_t r, int64_t lda, const void* A, const void* parity,
                       const void* x) {
    // Small problems only (up to 16 MB of A): there three launch latencies
    // dominate; larger ones stream better through the dedicated kernels.
    return n <= kOnePassMaxN && n > k && q > 0 && r >= 4 && r % 4 == 0 && lda % 4 == 0 && q * r <= (int64_t{1} << 22) &&
           aligned16p(A) && aligned16p(parity) && aligned16p(x);
}

hipError_t launch_onepass_f32(const OnePassArgs& a, hipStream_t st) {
    if (a.qb == 0) return hipSuccess;
    if (a.qb > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(a.qb));
    if (a.r <= 256)
        hipLaunchKernelGGL(onepass_f32_kernel<64>, grid, dim3(64), 0, st, a);
    else if (a.r <= 512)
        hipLaunchKernelGGL(onepass_f32_kernel<128>, grid, dim3(128), 0, st, a);
    else
        hipLaunchKernelGGL(onepass_f32_kernel<256>, grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace coded
