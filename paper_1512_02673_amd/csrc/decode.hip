// Decoding from any k worker results: dec(indices, results) of Sec. III-A.
//
// For a systematic generator G = [I_k; P] and a survivor set S, let M be the
// systematic blocks that did not arrive and S_par the parity survivors
// (|M| = |S_par| = m).  Every parity survivor a satisfies
//     Y_a = sum_{j in S_sys} G[a][j] Y_j + sum_{b in M} G[a][b] (A_b X),
// so the missing block products solve the m x m system
//     G[S_par, M] Z = Y_{S_par} - G[S_par, S_sys] Y_{S_sys}.
// This is exactly the LU of the k x k survivor sub-matrix G_S with the
// systematic rows (unit rows) taken as the first k-m pivots; the remaining
// m x m block is eliminated with partial pivoting (largest |entry|, lowest row
// on ties).  The kernel forms the m x k decoding matrix
//     D = G[S_par, M]^{-1} [ -G[S_par, S_sys] | I_m ]
// (columns indexed by the sorted survivor positions) in LDS, in fp64, and
// then applies it: out block M[b] = sum_c D[b][c] Y_{S[c]}, while systematic
// survivors are copied.  Survivors are canonicalised by sorting, so the
// result does not depend on the order in which they were given.
//
// Grid: (survivor set, chunk of block-row elements), flattened.  Every
// workgroup of a set rebuilds the same D (it is small next to the apply), so
// no global scratch or second launch is needed; the arithmetic is identical
// in every workgroup, so results are deterministic.
//
// Apply: a thread takes E consecutive elements of a block row (E = 4 when a
// row's columns come in aligned groups of four, so every output goes out as
// one 16-byte store; E = 1 otherwise, lanes on consecutive elements) and
// computes the missing outputs PASS at a time in registers; each pair of D
// entries read from LDS feeds 2*E fused multiply-adds.
#include "internal.h"

namespace coded {
namespace {

constexpr int kThreads = 256;

__device__ inline int set_entry(const DecodeSet& s, int c) {
    // Pick byte c of the packed set with constant-index reads of the argument.
    uint32_t word = 0;
#pragma unroll
    for (int i = 0; i < kMaxN / 4; ++i) word = (c / 4 == i) ? s.packed[i] : word;
    return static_cast<int>((word >> (8 * (c % 4))) & 0xFFu);
}

template <int E, typename YT>
struct Vec;
template <>
struct Vec<1, double> {
    __device__ static void load(const double* p, double* y) { y[0] = p[0]; }
};
template <>
struct Vec<4, double> {
    __device__ static void load(const double* p, double* y) {
        const double2 lo = reinterpret_cast<const double2*>(p)[0], hi = reinterpret_cast<const double2*>(p)[1];
        y[0] = lo.x; y[1] = lo.y; y[2] = hi.x; y[3] = hi.y;
    }
};
template <>
struct Vec<1, float> {
    __device__ static void load(const float* p, double* y) { y[0] = p[0]; }
};
template <>
struct Vec<4, float> {
    __device__ static void load(const float* p, double* y) {
        const float4 v = *reinterpret_cast<const float4*>(p);
        y[0] = v.x; y[1] = v.y; y[2] = v.z; y[3] = v.w;
    }
};

// out = v, or alpha * v + beta * c when an epilogue operand is given (c has
// out's layout; the element is read before it is written, so c may be out).
template <int E>
__device__ inline void store_out(const DecodeArgs& a, float* p, int64_t off, const double* v) {
    double w[E];
#pragma unroll
    for (int i = 0; i < E; ++i) w[i] = v[i];
    if (a.c) {
        float cv[E];
        if constexpr (E == 4) {
            const float4 f = *reinterpret_cast<const float4*>(a.c + off);
            cv[0] = f.x; cv[1] = f.y; cv[2] = f.z; cv[3] = f.w;
        } else {
            cv[0] = a.c[off];
        }
#pragma unroll
        for (int i = 0; i < E; ++i) w[i] = fma(a.alpha, w[i], a.beta * static_cast<double>(cv[i]));
    }
    if constexpr (E == 4)
        *reinterpret_cast<float4*>(p + off) = make_float4(static_cast<float>(w[0]), static_cast<float>(w[1]),
                                                          static_cast<float>(w[2]), static_cast<float>(w[3]));
    else
        p[off] = static_cast<float>(w[0]);
}

// PASS: missing outputs computed per sweep over the survivors (register
// bucket); E: elements per thread; ST (>= every m of the launch, even) is the
// row stride of the LDS matrices, sized on the host.
template <int PASS, int E, typename YT>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeArgs a, DecodeSet single, int64_t chunks,
                                                          int elems_per_block, int ST) {
    __shared__ int32_t sRaw[kMaxN];
    __shared__ int32_t sS[kMaxN];        // sorted survivors
    __shared__ int32_t sPresent[kMaxN];
    __shared__ int32_t sMiss[kMaxN];     // missing systematic blocks, ascending
    __shared__ int64_t sYoff[kMaxN];     // element offset of survivor c's result in Y
    __shared__ int64_t sOoff[kMaxN];     // element offset of block j's first row in out
    __shared__ int32_t sLim[kMaxN];      // rows of block j that lie inside A (the rest is padding)
    __shared__ int32_t sStatus, sM;
    extern __shared__ __align__(16) double dyn[];
    double* sD = dyn;                    // D column-major: sD[c * ST + b], c < k
    double* sMat = dyn + a.k * ST;       // m x m, row stride ST
    double* sL = sMat + ST * ST;         // multipliers of one elimination step

    const int tid = threadIdx.x;
    const int n = a.n, k = a.k;
    const int64_t b = blockIdx.x / chunks;
    const int64_t chunk = blockIdx.x % chunks;
    const bool writer = (chunk == 0 && tid == 0);

    if (tid == 0) sStatus = 0;
    for (int i = tid; i < n; i += kThreads) sPresent[i] = 0;
    for (int c = tid; c < k; c += kThreads) sRaw[c] = a.sets ? a.sets[b * k + c] : set_entry(single, c);
    __syncthreads();

    // Validate (range, repeats), sort by rank, mark present workers.
    for (int c = tid; c < k; c += kThreads) {
        const int v = sRaw[c];
        if (v < 0 || v >= n) {
            sStatus = -1;
            continue;
        }
        int rank = 0, same = 0;
        for (int j = 0; j < k; ++j) {
            rank += sRaw[j] < v;
            same += sRaw[j] == v;
        }
        if (same != 1) {
            sStatus = -1;
            continue;
        }
        sS[rank] = v;
        sPresent[v] = 1;
    }
    __syncthreads();
    if (sStatus != 0) {
        if (writer) a.info[b] = sStatus;
        return;
    }
    if (tid == 0) {
        int m = 0;
        for (int j = 0; j < k; ++j)
            if (!sPresent[j]) sMiss[m++] = j;
        sM = m;
    }
    for (int c = tid; c < k; c += kThreads) sYoff[c] = static_cast<int64_t>(sS[c]) * a.qb * a.s;
    for (int j = tid; j < k; j += kThreads) {
        sOoff[j] = static_cast<int64_t>(j) * a.qb * a.ldo;
        const int64_t lim = a.q - static_cast<int64_t>(j) * a.qb;
        sLim[j] = static_cast<int32_t>(lim < 0 ? 0 : (lim > a.qb ? a.qb : lim));
    }
    __syncthreads();
    const int m = sM;
    const int first_par = k - m;          // sorted: systematic survivors first, then parity

    if (m > 0) {
        // sMat[r][cb] = G[S_par[r]][M[cb]];  column c of D starts as column c
        // of the right-hand side [-G[S_par, S_sys] | I]; rows >= m stay 0.
        for (int e = tid; e < m * m; e += kThreads) {
            const int ra = e / m, cb = e % m;
            sMat[ra * ST + cb] = a.G[static_cast<int64_t>(sS[first_par + ra]) * k + sMiss[cb]];
        }
        for (int e = tid; e < ST * k; e += kThreads) {
            const int c = e / ST, ra = e % ST;
            double v = 0.0;
            if (ra < m) {
                const int sc = sS[c];
                v = sc < k ? -a.G[static_cast<int64_t>(sS[first_par + ra]) * k + sc]
                           : ((c - first_par == ra) ? 1.0 : 0.0);
            }
            sD[c * ST + ra] = v;
        }
        __syncthreads();

        // Gaussian elimination with partial pivoting on sMat, applied to the
        // right-hand sides as it goes.
        for (int j = 0; j < m; ++j) {
            if (tid == 0) {
                int p = j;
                double best = fabs(sMat[j * ST + j]);
                for (int i = j + 1; i < m; ++i) {
                    const double v = fabs(sMat[i * ST + j]);
                    if (v > best) {
                        best = v;
                        p = i;
                    }
                }
                if (best == 0.0) sStatus = first_par + j + 1;
                sRaw[0] = p;                       // reuse: pivot row of this step
            }
            __syncthreads();
            if (sStatus != 0) break;
            const int p = sRaw[0];
            if (p != j) {
                for (int c = tid; c < m; c += kThreads) {
                    const double t0 = sMat[j * ST + c];
                    sMat[j * ST + c] = sMat[p * ST + c];
                    sMat[p * ST + c] = t0;
                }
                for (int c = tid; c < k; c += kThreads) {
                    const double t0 = sD[c * ST + j];
                    sD[c * ST + j] = sD[c * ST + p];
                    sD[c * ST + p] = t0;
                }
            }
            __syncthreads();
            for (int i = j + 1 + tid; i < m; i += kThreads) sL[i] = sMat[i * ST + j] / sMat[j * ST + j];
            __syncthreads();
            const int rows = m - j - 1;
            if (rows > 0) {
                for (int e = tid; e < rows * rows; e += kThreads) {
                    const int i = j + 1 + e / rows, c = j + 1 + e % rows;
                    sMat[i * ST + c] -= sL[i] * sMat[j * ST + c];
                }
                for (int e = tid; e < rows * k; e += kThreads) {
                    const int i = j + 1 + e / k, c = e % k;
                    sD[c * ST + i] -= sL[i] * sD[c * ST + j];
                }
            }
            __syncthreads();
        }
        if (sStatus != 0) {
            if (writer) a.info[b] = sStatus;
            return;
        }
        // Back substitution with U, one right-hand side column per thread.
        for (int c = tid; c < k; c += kThreads) {
            for (int i = m - 1; i >= 0; --i) {
                double v = sD[c * ST + i];
                for (int jj = i + 1; jj < m; ++jj) v -= sMat[i * ST + jj] * sD[c * ST + jj];
                sD[c * ST + i] = v / sMat[i * ST + i];
            }
        }
        __syncthreads();
    }
    if (writer) a.info[b] = 0;

    // Apply.
    const YT* Y = static_cast<const YT*>(a.Y);
    float* out = a.out + b * a.out_stride;
    const int total = static_cast<int>(a.qb * a.s);
    const int s = static_cast<int>(a.s);
    const int e0 = static_cast<int>(chunk) * elems_per_block;
    const int e1 = min(total, e0 + elems_per_block);
    const int passes = m > 0 ? (m + PASS - 1) / PASS : 1;
    for (int e = e0 + E * tid; e < e1; e += E * kThreads) {
        const int t = e / s, col = e - t * s;      // E = 4: the four elements share row t
        for (int pass = 0; pass < passes; ++pass) {
            const int p0 = pass * PASS;
            double acc[PASS][E];
#pragma unroll
            for (int bb = 0; bb < PASS; ++bb)
#pragma unroll
                for (int v = 0; v < E; ++v) acc[bb][v] = 0.0;
            for (int c = 0; c < k; ++c) {
                double y[E];
                Vec<E, YT>::load(Y + sYoff[c] + e, y);
                const int w = sS[c];
                if (pass == 0 && w < k && t < sLim[w]) store_out<E>(a, out, sOoff[w] + static_cast<int64_t>(t) * a.ldo + col, y);
                const double* dp = sD + c * ST + p0;
#pragma unroll
                for (int bb = 0; bb < PASS; bb += 2) {
                    if (p0 + bb < m) {
                        const double2 d = *reinterpret_cast<const double2*>(dp + bb);
#pragma unroll
                        for (int v = 0; v < E; ++v) {
                            acc[bb][v] = fma(d.x, y[v], acc[bb][v]);
                            acc[bb + 1][v] = fma(d.y, y[v], acc[bb + 1][v]);
                        }
                    }
                }
            }
#pragma unroll
            for (int bb = 0; bb < PASS; ++bb) {
                if (p0 + bb < m) {
                    const int w = sMiss[p0 + bb];
                    if (t < sLim[w]) store_out<E>(a, out, sOoff[w] + static_cast<int64_t>(t) * a.ldo + col, acc[bb]);
                }
            }
        }
    }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) % 16) == 0; }

template <int PASS, int E>
hipError_t launch_pe(const DecodeArgs& a, const DecodeSet& single, int st_rows, hipStream_t st) {
    const int64_t total = a.qb * a.s;
    // One workgroup per set once the batch fills the chip; a few sets are split
    // over several workgroups.
    const int64_t max_chunks = std::max<int64_t>(1, ceil_div(total, static_cast<int64_t>(kThreads) * E));
    const int64_t want = std::max<int64_t>(1, ceil_div(2048, a.batch));
    const int64_t chunks = std::min(max_chunks, want);
    const int64_t per = ceil_div(ceil_div(std::max<int64_t>(total, 1), chunks), E) * E;
    const int64_t blocks = chunks * a.batch;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const size_t shmem = decode_lds_bytes(a.k, st_rows);
    if (a.y_f64)
        hipLaunchKernelGGL((decode_kernel<PASS, E, double>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads),
                           shmem, st, a, single, chunks, static_cast<int>(per), st_rows);
    else
        hipLaunchKernelGGL((decode_kernel<PASS, E, float>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads),
                           shmem, st, a, single, chunks, static_cast<int>(per), st_rows);
    return hipGetLastError();
}

template <int PASS>
hipError_t launch_p(const DecodeArgs& a, const DecodeSet& single, int st_rows, hipStream_t st) {
    const bool vec4 = a.s % 4 == 0 && a.ldo % 4 == 0 && aligned16(a.out) && aligned16(a.Y) &&
                      (a.batch == 1 || a.out_stride % 4 == 0) && (a.c == nullptr || aligned16(a.c));
    return vec4 ? launch_pe<PASS, 4>(a, single, st_rows, st) : launch_pe<PASS, 1>(a, single, st_rows, st);
}

}  // namespace

size_t decode_lds_bytes(int k, int mmax) {
    const int st = (std::max(mmax, 1) + 1) / 2 * 2;
    return static_cast<size_t>(k * st + st * st + st) * sizeof(double);
}

hipError_t launch_decode(const DecodeArgs& a, const DecodeSet* single, int mmax, hipStream_t st) {
    if (a.batch == 0) return hipSuccess;
    if (a.qb * a.s > 0x7FFFFFFF) return hipErrorInvalidValue;
    DecodeSet s{};
    if (single) s = *single;
    const int rows = (std::max(mmax, 1) + 1) / 2 * 2;   // even: D pairs are read 16 bytes at a time
    if (mmax <= 2) return launch_p<2>(a, s, rows, st);
    if (mmax <= 4) return launch_p<4>(a, s, rows, st);
    return launch_p<8>(a, s, rows, st);
}

}  // namespace coded
