// Parity encoding: A'_{k+p} = sum_j P[p][j] A_j for the n-k parity blocks
// (Sec. III-A: the (n,k) code applied to every element of the k row-blocks;
// the k systematic blocks are A itself and are never copied).
//
// The contraction has k (<= a few dozen) terms per output element and the
// whole pass streams A once and writes the parity planes once, so it is bound
// by HBM bandwidth, not arithmetic (about 2 flops per byte, far below the
// matrix cores' ridge): each thread owns a short vector of columns of one
// block row t, walks the k blocks j with kBatch loads in flight, and keeps up
// to kGroup parity accumulators in registers; the sum runs over j in order.  Parity rows beyond kGroup are
// handled by further groups (grid.y), each re-reading A.
//
// Storage: with planes == 2 the exact sum (fp64 for fp32 inputs, fp32 for
// bf16 inputs) is stored as hi = round(sum) and lo = round(sum - hi).
#include "internal.h"

namespace coded {
namespace {

constexpr int kGroup = 8;       // parity rows per pass
constexpr int kThreads = 256;
constexpr int kBatch = 8;       // blocks whose loads are in flight together

__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t b = __float_as_uint(f);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return static_cast<uint16_t>(b >> 16);
}
__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

// One thread: VEC consecutive columns of block row t, parity rows
// [p0, p0 + np) with np <= kGroup.
template <int VEC>
__global__ __launch_bounds__(kThreads) void encode_f32_kernel(EncodeArgs a, int64_t col_chunks) {
    __shared__ double sP[kGroup * kMaxN];
    const int64_t t = blockIdx.x;
    const int64_t chunk = blockIdx.y % col_chunks;
    const int p0 = static_cast<int>(blockIdx.y / col_chunks) * kGroup;
    const int npar = a.n - a.k;
    const int np = min(kGroup, npar - p0);
    const int k = a.k;
    for (int e = threadIdx.x; e < np * k; e += kThreads) {
        const int p = e / k, j = e % k;
        sP[p * k + j] = a.G[(a.k + p0 + p) * k + j];
    }
    __syncthreads();
    const int64_t c = (chunk * kThreads + threadIdx.x) * VEC;
    if (c >= a.r) return;
    const float* A = static_cast<const float*>(a.A);

    double acc[kGroup][VEC];
#pragma unroll
    for (int p = 0; p < kGroup; ++p)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[p][v] = 0.0;

    // Blocks whose row t lies inside A (rows of later blocks are the zero
    // padding and contribute nothing); their loads go out kBatch at a time.
    const int kv = static_cast<int>(min<int64_t>(k, (a.q - t + a.qb - 1) / a.qb));
    for (int j0 = 0; j0 < kv; j0 += kBatch) {
        float v4[kBatch][VEC];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int j = min(j0 + u, kv - 1);   // past the last block: re-read it, not used
            const float* src = A + (static_cast<int64_t>(j) * a.qb + t) * a.lda + c;
            if constexpr (VEC == 4) {
                const float4 f = *reinterpret_cast<const float4*>(src);
                v4[u][0] = f.x; v4[u][1] = f.y; v4[u][2] = f.z; v4[u][3] = f.w;
            } else {
#pragma unroll
                for (int v = 0; v < VEC; ++v) v4[u][v] = src[v];
            }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (j0 + u >= kv) break;
#pragma unroll
            for (int p = 0; p < kGroup; ++p) {
                if (p < np) {
                    const double g = sP[p * k + j0 + u];
#pragma unroll
                    for (int v = 0; v < VEC; ++v) acc[p][v] = fma(g, static_cast<double>(v4[u][v]), acc[p][v]);
                }
            }
        }
    }

    float* par = static_cast<float*>(a.parity);
    const int64_t plane = static_cast<int64_t>(npar) * a.qb * a.r;
    // lo plane as bfloat16: after the fp32 hi plane, same element order
    uint16_t* par16 = reinterpret_cast<uint16_t*>(par + plane);
#pragma unroll
    for (int p = 0; p < kGroup; ++p) {
        if (p >= np) break;
        float hi[VEC], lo[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            hi[v] = static_cast<float>(acc[p][v]);
            lo[v] = static_cast<float>(acc[p][v] - static_cast<double>(hi[v]));   // exact remainder, rounded to fp32
        }
        const int64_t off = (static_cast<int64_t>(p0 + p) * a.qb + t) * a.r + c;
        float* dst = par + off;
        if constexpr (VEC == 4) {
            *reinterpret_cast<float4*>(dst) = make_float4(hi[0], hi[1], hi[2], hi[3]);
            if (a.planes == 2) {
                if (a.lo_bf16) {
                    uint2 l;
                    l.x = f32_to_bf16_rne(lo[0]) | (static_cast<uint32_t>(f32_to_bf16_rne(lo[1])) << 16);
                    l.y = f32_to_bf16_rne(lo[2]) | (static_cast<uint32_t>(f32_to_bf16_rne(lo[3])) << 16);
                    *reinterpret_cast<uint2*>(par16 + off) = l;
                } else {
                    *reinterpret_cast<float4*>(dst + plane) = make_float4(lo[0], lo[1], lo[2], lo[3]);
                }
            }
        } else {
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                dst[v] = hi[v];
                if (a.planes == 2) {
                    if (a.lo_bf16)
                        par16[off + v] = f32_to_bf16_rne(lo[v]);
                    else
                        dst[plane + v] = lo[v];
                }
            }
        }
    }
}

// bf16: products of two bf16 values are exact in fp32; the k-term sum is
// accumulated in fp32 and split into bf16 hi + lo.
template <int VEC>
__global__ __launch_bounds__(kThreads) void encode_bf16_kernel(EncodeArgs a, int64_t col_chunks) {
    __shared__ float sP[kGroup * kMaxN];
    const int64_t t = blockIdx.x;
    const int64_t chunk = blockIdx.y % col_chunks;
    const int p0 = static_cast<int>(blockIdx.y / col_chunks) * kGroup;
    const int npar = a.n - a.k;
    const int np = min(kGroup, npar - p0);
    const int k = a.k;
    for (int e = threadIdx.x; e < np * k; e += kThreads) {
        const int p = e / k, j = e % k;
        sP[p * k + j] = static_cast<float>(a.G[(a.k + p0 + p) * k + j]);
    }
    __syncthreads();
    const int64_t c = (chunk * kThreads + threadIdx.x) * VEC;
    if (c >= a.r) return;
    const uint16_t* A = static_cast<const uint16_t*>(a.A);

    float acc[kGroup][VEC];
#pragma unroll
    for (int p = 0; p < kGroup; ++p)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[p][v] = 0.0f;

    const int kv = static_cast<int>(min<int64_t>(k, (a.q - t + a.qb - 1) / a.qb));   // blocks with row t inside A
    for (int j0 = 0; j0 < kv; j0 += kBatch) {
        float v8[kBatch][VEC];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int j = min(j0 + u, kv - 1);   // past the last block: re-read it, not used
            const uint16_t* src = A + (static_cast<int64_t>(j) * a.qb + t) * a.lda + c;
            if constexpr (VEC == 8) {
                const uint4 q4 = *reinterpret_cast<const uint4*>(src);
                const uint32_t w[4] = {q4.x, q4.y, q4.z, q4.w};
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    v8[u][2 * h] = __uint_as_float(w[h] << 16);
                    v8[u][2 * h + 1] = __uint_as_float(w[h] & 0xFFFF0000u);
                }
            } else {
#pragma unroll
                for (int v = 0; v < VEC; ++v) v8[u][v] = bf16_to_f32(src[v]);
            }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (j0 + u >= kv) break;
#pragma unroll
            for (int p = 0; p < kGroup; ++p) {
                if (p < np) {
                    const float g = sP[p * k + j0 + u];
#pragma unroll
                    for (int v = 0; v < VEC; ++v) acc[p][v] = fmaf(g, v8[u][v], acc[p][v]);
                }
            }
        }
    }

    uint16_t* par = static_cast<uint16_t*>(a.parity);
    const int64_t plane = static_cast<int64_t>(npar) * a.qb * a.r;
#pragma unroll
    for (int p = 0; p < kGroup; ++p) {
        if (p >= np) break;
        uint16_t hi[VEC], lo[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            hi[v] = f32_to_bf16_rne(acc[p][v]);
            lo[v] = f32_to_bf16_rne(acc[p][v] - bf16_to_f32(hi[v]));
        }
        uint16_t* dst = par + (static_cast<int64_t>(p0 + p) * a.qb + t) * a.r + c;
        if constexpr (VEC == 8) {
            uint4 h4, l4;
            h4.x = hi[0] | (uint32_t(hi[1]) << 16); h4.y = hi[2] | (uint32_t(hi[3]) << 16);
            h4.z = hi[4] | (uint32_t(hi[5]) << 16); h4.w = hi[6] | (uint32_t(hi[7]) << 16);
            l4.x = lo[0] | (uint32_t(lo[1]) << 16); l4.y = lo[2] | (uint32_t(lo[3]) << 16);
            l4.z = lo[4] | (uint32_t(lo[5]) << 16); l4.w = lo[6] | (uint32_t(lo[7]) << 16);
            *reinterpret_cast<uint4*>(dst) = h4;
            if (a.planes == 2) *reinterpret_cast<uint4*>(dst + plane) = l4;
        } else {
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                dst[v] = hi[v];
                if (a.planes == 2) dst[plane + v] = lo[v];
            }
        }
    }
}

bool aligned(const void* p, int bytes) { return (reinterpret_cast<uintptr_t>(p) % bytes) == 0; }

}  // namespace

hipError_t launch_encode_f32(const EncodeArgs& a, hipStream_t st) {
    const int npar = a.n - a.k;
    if (npar == 0 || a.qb == 0 || a.r == 0) return hipSuccess;
    const int groups = static_cast<int>(ceil_div(npar, kGroup));
    const bool vec = (a.r % 4 == 0) && (a.lda % 4 == 0) && aligned(a.A, 16) && aligned(a.parity, 16);
    const int V = vec ? 4 : 1;
    const int64_t chunks = ceil_div(a.r, static_cast<int64_t>(kThreads) * V);
    if (chunks * groups > 65535) return hipErrorInvalidConfiguration;
    dim3 grid(static_cast<unsigned>(a.qb), static_cast<unsigned>(chunks * groups));
    if (vec)
        hipLaunchKernelGGL(encode_f32_kernel<4>, grid, dim3(kThreads), 0, st, a, chunks);
    else
        hipLaunchKernelGGL(encode_f32_kernel<1>, grid, dim3(kThreads), 0, st, a, chunks);
    return hipGetLastError();
}

hipError_t launch_encode_bf16(const EncodeArgs& a, hipStream_t st) {
    const int npar = a.n - a.k;
    if (npar == 0 || a.qb == 0 || a.r == 0) return hipSuccess;
    const int groups = static_cast<int>(ceil_div(npar, kGroup));
    const bool vec = (a.r % 8 == 0) && (a.lda % 8 == 0) && aligned(a.A, 16) && aligned(a.parity, 16);
    const int V = vec ? 8 : 1;
    const int64_t chunks = ceil_div(a.r, static_cast<int64_t>(kThreads) * V);
    if (chunks * groups > 65535) return hipErrorInvalidConfiguration;
    dim3 grid(static_cast<unsigned>(a.qb), static_cast<unsigned>(chunks * groups));
    if (vec)
        hipLaunchKernelGGL(encode_bf16_kernel<8>, grid, dim3(kThreads), 0, st, a, chunks);
    else
        hipLaunchKernelGGL(encode_bf16_kernel<1>, grid, dim3(kThreads), 0, st, a, chunks);
    return hipGetLastError();
}

}  // namespace coded
