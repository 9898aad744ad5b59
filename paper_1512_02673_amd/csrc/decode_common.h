// Decoding pieces shared by the decode kernels and the one-pass product:
// reading a survivor set, its bookkeeping, and the register elimination
// that forms the decoding matrix D (Sec. III-A, dec(indices, results)).
#pragma once
#include "internal.h"

namespace coded {
namespace {

__device__ inline int set_entry(const DecodeSet& s, int c) {
    // Pick byte c of the packed set with constant-index reads of the argument.
    uint32_t word = 0;
#pragma unroll
    for (int i = 0; i < kMaxN / 4; ++i) word = (c / 4 == i) ? s.packed[i] : word;
    return static_cast<int>((word >> (8 * (c % 4))) & 0xFFu);
}

// Per-set bookkeeping in LDS.
struct SetMeta {
    int32_t raw[kMaxN];
    int32_t S[kMaxN];          // sorted survivors
    int32_t present[kMaxN];
    int32_t miss[kMaxN];       // missing systematic blocks, ascending
    int64_t yoff[kMaxN];       // element offset of survivor c's result in Y
    int64_t ooff[kMaxN];       // element offset of block j's first row in out
    int32_t lim[kMaxN];        // rows of block j that lie inside A (the rest is padding)
    int32_t status, m;
};

// Reads set b, validates it (range, repeats), sorts it and fills the
// bookkeeping.  Returns false (after writing info = -1) for an invalid set.
// Every thread of the workgroup (NT threads) must call it.
template <int NT>
__device__ __forceinline__ bool setup_set(const DecodeArgs& a, const DecodeSet& single, int64_t b, bool writer, SetMeta& sm) {
    const int tid = threadIdx.x;
    const int n = a.n, k = a.k;
    if (tid == 0) sm.status = 0;
    for (int i = tid; i < n; i += NT) sm.present[i] = 0;
    for (int c = tid; c < k; c += NT) sm.raw[c] = a.sets ? a.sets[b * k + c] : set_entry(single, c);
    __syncthreads();
    for (int c = tid; c < k; c += NT) {
        const int v = sm.raw[c];
        if (v < 0 || v >= n) {
            sm.status = -1;
            continue;
        }
        int rank = 0, same = 0;
        for (int j = 0; j < k; ++j) {
            rank += sm.raw[j] < v;
            same += sm.raw[j] == v;
        }
        if (same != 1) {
            sm.status = -1;
            continue;
        }
        sm.S[rank] = v;
        sm.present[v] = 1;
    }
    __syncthreads();
    if (sm.status != 0) {
        if (writer) a.info[b] = sm.status;
        return false;
    }
    if (tid == 0) {
        int m = 0;
        for (int j = 0; j < k; ++j)
            if (!sm.present[j]) sm.miss[m++] = j;
        sm.m = m;
    }
    for (int c = tid; c < k; c += NT) sm.yoff[c] = static_cast<int64_t>(sm.S[c]) * a.qb * a.s;
    for (int j = tid; j < k; j += NT) {
        sm.ooff[j] = static_cast<int64_t>(j) * a.qb * a.ldo;
        const int64_t lim = a.q - static_cast<int64_t>(j) * a.qb;
        sm.lim[j] = static_cast<int32_t>(lim < 0 ? 0 : (lim > a.qb ? a.qb : lim));
    }
    __syncthreads();
    return true;
}

// Codes with at most kFastM missing blocks per set and m + k <= 64 eliminate
// the m x (m + k) system [G[S_par, M] | -G[S_par, S_sys] | I] in the
// registers of one wave (Gauss-Jordan, partial pivoting: the same pivots as
// an LU with the systematic rows first, one column per lane, no workgroup
// barriers).
constexpr int kFastM = 16;
constexpr int kFastLd = kFastM + 1;      // odd LDS column stride of D: spreads the banks

__device__ inline double lane_value(double v, int lane) {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(u), lane);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(u >> 32), lane);
    return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}

// Wave-level elimination for sets with m <= MM <= kFastM.  Lane l holds
// column l of the augmented matrix: lanes < m the columns of G[S_par, M],
// lanes m..m+k-1 the right-hand sides (sorted survivor order).  On success
// D[b][c] = sD[c * kFastLd + b] for b < kFastM (rows >= m zero); on a zero
// pivot sm.status = first_par + j + 1.  The operations on rows < m do not
// depend on MM, so every MM >= m gives the same D.
// Meta: any bookkeeping with S (sorted survivors), miss and status as in SetMeta.
template <int MM, typename Meta>
__device__ __forceinline__ void eliminate_wave(const DecodeArgs& a, Meta& sm, int m, int first_par, int lane, double* sD) {
    static_assert(MM <= kFastM, "MM");
    const int k = a.k;
    const int c = lane - m;
    double col[MM];
#pragma unroll
    for (int r = 0; r < MM; ++r) {
        double v = 0.0;
        if (r < m) {
            const int64_t prow = static_cast<int64_t>(sm.S[first_par + r]) * k;
            if (lane < m) {
                v = a.G[prow + sm.miss[lane]];
            } else if (c < k) {
                const int sc = sm.S[c];
                v = sc < k ? -a.G[prow + sc] : ((c - first_par == r) ? 1.0 : 0.0);
            }
        }
        col[r] = v;
    }
    int status = 0;
#pragma unroll
    for (int j = 0; j < MM; ++j) {
        // uniform guards instead of an early exit keep the loop fully unrolled
        // (every register index a constant)
        if (j < m && status == 0) {
            // pivot: largest |entry| of column j in rows j..m-1, lowest row on ties
            int p = j;
            double best = fabs(col[j]);
#pragma unroll
            for (int i = j + 1; i < MM; ++i) {
                const double v = fabs(col[i]);
                if (i < m && v > best) {
                    best = v;
                    p = i;
                }
            }
            p = __builtin_amdgcn_readlane(p, j);
            best = lane_value(best, j);
            if (best == 0.0) {
                status = first_par + j + 1;
            } else {
#pragma unroll
                for (int i = j + 1; i < MM; ++i) {
                    if (i == p) {
                        const double t = col[i];
                        col[i] = col[j];
                        col[j] = t;
                    }
                }
                // Row i -= l_i * row j with l_i = a_ij / pivot, as in the LU
                // (so an exactly dependent row cancels to an exact zero), then
                // row j /= pivot.  l_i is the reciprocal product corrected once
                // by its exact residual (Markstein's division step).
                const double piv = lane_value(col[j], j);
                const double inv = 1.0 / piv;
#pragma unroll
                for (int i = 0; i < MM; ++i) {
                    if (i != j && i < m) {
                        const double aij = lane_value(col[i], j);
                        const double l0 = aij * inv;
                        const double li = fma(fma(-l0, piv, aij), inv, l0);
                        col[i] = fma(-li, col[j], col[i]);
                    }
                }
                col[j] = col[j] / piv;
            }
        }
    }
    if (status == 0 && c >= 0 && c < k) {
#pragma unroll
        for (int r = 0; r < kFastM; ++r) sD[c * kFastLd + r] = r < MM ? col[r] : 0.0;
    }
    if (lane == 0) sm.status = status;
}

// The smallest register size that holds a set with m missing blocks.
template <typename Meta>
__device__ __forceinline__ void eliminate_set(const DecodeArgs& a, Meta& sm, int m, int first_par, int lane,
                                              double* sD) {
    if (m <= 4)
        eliminate_wave<4>(a, sm, m, first_par, lane, sD);
    else if (m <= 8)
        eliminate_wave<8>(a, sm, m, first_par, lane, sD);
    else if (m <= 12)
        eliminate_wave<12>(a, sm, m, first_par, lane, sD);
    else
        eliminate_wave<kFastM>(a, sm, m, first_par, lane, sD);
}

}  // namespace
}  // namespace coded
