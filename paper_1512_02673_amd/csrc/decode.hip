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
// Grid: (chunks of block-row elements, survivor sets).  Every workgroup of a
// set rebuilds the same D (it is tiny next to the apply) so no global
// scratch or second launch is needed; the arithmetic is identical in every
// workgroup, so results are deterministic.
#include "internal.h"

namespace coded {
namespace {

constexpr int kThreads = 256;

// MAXM: register bound on m (a template bucket); ST (>= every m of the
// launch) is the row stride of the LDS matrices, sized on the host.
template <int MAXM, typename YT>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeArgs a, DecodeSet single, int64_t chunks,
                                                          int64_t elems_per_block, int ST) {
    __shared__ int32_t sRaw[kMaxN];
    __shared__ int32_t sS[kMaxN];       // sorted survivors
    __shared__ int32_t sPresent[kMaxN];
    __shared__ int32_t sMiss[MAXM];     // missing systematic blocks, ascending
    __shared__ int32_t sStatus, sM;
    __shared__ double sL[MAXM];
    extern __shared__ double dyn[];
    double* sD = dyn;                   // D column-major: sD[c * ST + b], c < k
    double* sMat = dyn + a.k * ST;      // m x m, row stride ST

    const int tid = threadIdx.x;
    const int n = a.n, k = a.k;
    const int64_t b = blockIdx.x / chunks;
    const int64_t chunk = blockIdx.x % chunks;
    const bool writer = (chunk == 0 && tid == 0);

    if (tid == 0) sStatus = 0;
    for (int i = tid; i < n; i += kThreads) sPresent[i] = 0;
    for (int c = tid; c < k; c += kThreads) sRaw[c] = a.sets ? a.sets[b * k + c] : single.idx[c];
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
    __syncthreads();
    const int m = sM;
    const int first_par = k - m;          // sorted: systematic survivors first, then parity

    if (m > 0) {
        // sMat[a][bb] = G[S_par[a]][M[bb]];  D[c][a] = right-hand side column c.
        for (int e = tid; e < m * m; e += kThreads) {
            const int ra = e / m, cb = e % m;
            sMat[ra * ST + cb] = a.G[static_cast<int64_t>(sS[first_par + ra]) * k + sMiss[cb]];
        }
        for (int e = tid; e < m * k; e += kThreads) {
            const int c = e / m, ra = e % m;
            const int sc = sS[c];
            double v;
            if (sc < k)
                v = -a.G[static_cast<int64_t>(sS[first_par + ra]) * k + sc];
            else
                v = (c - first_par == ra) ? 1.0 : 0.0;
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
                for (int e = tid; e < rows * (m - j - 1); e += kThreads) {
                    const int i = j + 1 + e / (m - j - 1), c = j + 1 + e % (m - j - 1);
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

    // Apply: element e of a block is (row t, column col) with t = e / s.
    const YT* Y = static_cast<const YT*>(a.Y);
    float* out = a.out + b * a.out_stride;
    const int64_t total = a.qb * a.s;
    const int64_t e0 = chunk * elems_per_block;
    const int64_t e1 = min(total, e0 + elems_per_block);
    for (int64_t e = e0 + tid; e < e1; e += kThreads) {
        const int64_t t = e / a.s, col = e - t * a.s;
        double acc[MAXM];
#pragma unroll
        for (int bb = 0; bb < MAXM; ++bb) acc[bb] = 0.0;
        for (int c = 0; c < k; ++c) {
            const int w = sS[c];
            const double y = static_cast<double>(Y[(static_cast<int64_t>(w) * a.qb + t) * a.s + col]);
            if (w < k) {
                const int64_t row = static_cast<int64_t>(w) * a.qb + t;
                if (row < a.q) out[row * a.ldo + col] = static_cast<float>(y);
            }
#pragma unroll
            for (int bb = 0; bb < MAXM; ++bb)
                if (bb < m) acc[bb] = fma(sD[c * ST + bb], y, acc[bb]);
        }
#pragma unroll
        for (int bb = 0; bb < MAXM; ++bb) {
            if (bb < m) {
                const int64_t row = static_cast<int64_t>(sMiss[bb]) * a.qb + t;
                if (row < a.q) out[row * a.ldo + col] = static_cast<float>(acc[bb]);
            }
        }
    }
}

template <int MAXM>
hipError_t launch_m(const DecodeArgs& a, const DecodeSet& single, int st_rows, hipStream_t st) {
    const int64_t total = a.qb * a.s;
    const int64_t max_chunks = std::max<int64_t>(1, ceil_div(total, kThreads));
    const int64_t want = std::max<int64_t>(1, ceil_div(2048, a.batch));
    const int64_t chunks = std::min(max_chunks, want);
    const int64_t per = ceil_div(std::max<int64_t>(total, 1), chunks);
    const int64_t blocks = chunks * a.batch;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const size_t shmem = decode_lds_bytes(a.k, st_rows);
    if (a.y_f64)
        hipLaunchKernelGGL((decode_kernel<MAXM, double>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), shmem,
                           st, a, single, chunks, per, st_rows);
    else
        hipLaunchKernelGGL((decode_kernel<MAXM, float>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), shmem,
                           st, a, single, chunks, per, st_rows);
    return hipGetLastError();
}

}  // namespace

size_t decode_lds_bytes(int k, int mmax) {
    return static_cast<size_t>(k * mmax + mmax * mmax) * sizeof(double);
}

hipError_t launch_decode(const DecodeArgs& a, const DecodeSet* single, int mmax, hipStream_t st) {
    if (a.batch == 0) return hipSuccess;
    DecodeSet s{};
    if (single) s = *single;
    const int rows = std::max(mmax, 1);
    if (mmax <= 4) return launch_m<4>(a, s, rows, st);
    if (mmax <= 8) return launch_m<8>(a, s, rows, st);
    if (mmax <= 16) return launch_m<16>(a, s, rows, st);
    if (mmax <= 32) return launch_m<32>(a, s, rows, st);
    return launch_m<64>(a, s, rows, st);
}

}  // namespace coded
