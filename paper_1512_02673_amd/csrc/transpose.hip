// Column split of A for the transposed code of coded gradient descent
// (Sec. III-E: worker i stores the i-th row-split of A and, for the second
// product, the i-th column-split, i.e. a row-split of A^T).  A^T is formed
// once, in 64 x 64 tiles staged through LDS so that both the reads of A and
// the writes of A^T are coalesced rows.
#include "internal.h"

namespace coded {
namespace {

constexpr int kTile = 64;

__global__ __launch_bounds__(256) void transpose_f32_kernel(const float* __restrict__ A, int64_t q, int64_t r,
                                                            int64_t lda, float* __restrict__ AT, int64_t ldat,
                                                            int64_t tiles_r) {
    __shared__ float tile[kTile][kTile + 1];     // +1 column: no bank conflicts on the transposed read
    const int64_t tq = blockIdx.x / tiles_r, tr = blockIdx.x % tiles_r;
    const int64_t row0 = tq * kTile, col0 = tr * kTile;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;   // 64 x 4 threads
    for (int i = ty; i < kTile; i += 4) {
        const int64_t row = row0 + i, col = col0 + tx;
        tile[i][tx] = (row < q && col < r) ? A[row * lda + col] : 0.0f;
    }
    __syncthreads();
    for (int i = ty; i < kTile; i += 4) {
        const int64_t orow = col0 + i, ocol = row0 + tx;    // AT[orow][ocol] = A[ocol][orow]
        if (orow < r && ocol < q) AT[orow * ldat + ocol] = tile[tx][i];
    }
}

}  // namespace

hipError_t launch_transpose_f32(const float* A, int64_t q, int64_t r, int64_t lda, float* AT, int64_t ldat,
                                hipStream_t st) {
    if (q == 0 || r == 0) return hipSuccess;
    const int64_t tq = ceil_div(q, kTile), tr = ceil_div(r, kTile);
    if (tq * tr > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(transpose_f32_kernel, dim3(static_cast<unsigned>(tq * tr)), dim3(256), 0, st, A, q, r, lda, AT,
                       ldat, tr);
    return hipGetLastError();
}

}  // namespace coded
