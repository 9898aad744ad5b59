// Coded shuffling on the device (Sec. IV, Algorithm 1 and the decoding rule).
//
// encode: message row m is the sum of the data rows of its terms,
//         enc_rows[enc_off[m] .. enc_off[m+1]), in that order;
// decode: term d (row enc_rows[d], needed by one worker) is its message
//         term_msg[d] minus the other terms' rows of that message, in order;
//         one wave per message writes all of its terms.
// The data are coded over their own representation (fp32 sums and
// differences, no fused operations), so a decoded row is bit-identical to a
// sequential evaluation of the same sums.
//
// Both are row gathers bound by HBM: one wave per message row, 16-byte loads
// when the rows allow them; the encode issues a row's term loads four at a
// time.  Every table entry is checked against its range: an entry outside it
// turns its output rows into NaN instead of reading out of bounds (a term
// that no valid message range covers is left unwritten).
#include "internal.h"

namespace coded {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
typedef float f32x4s __attribute__((ext_vector_type(4)));

template <int V>
struct Row;
template <>
struct Row<4> {
    typedef f32x4s T;
    __device__ static T load(const float* p) { return *reinterpret_cast<const f32x4s*>(p); }
    __device__ static void store(float* p, T v) { __builtin_nontemporal_store(v, reinterpret_cast<f32x4s*>(p)); }
    __device__ static T nan() {
        const float x = __builtin_nanf("");
        return T{x, x, x, x};
    }
};
template <>
struct Row<1> {
    typedef float T;
    __device__ static T load(const float* p) { return *p; }
    __device__ static void store(float* p, T v) { __builtin_nontemporal_store(v, p); }
    __device__ static T nan() { return __builtin_nanf(""); }
};

// Validated term range of message m (false: a bad table entry).
__device__ inline bool term_range(const int64_t* off, int64_t m, int64_t terms, int64_t& b, int64_t& e) {
    b = off[m];
    e = off[m + 1];
    return 0 <= b && b <= e && e <= terms;
}

template <int V>
__global__ __launch_bounds__(kThreads) void shuffle_encode_kernel(const float* __restrict__ A, int64_t q, int64_t r,
                                                                  int64_t lda, const int64_t* __restrict__ off,
                                                                  const int32_t* __restrict__ rows, int64_t msgs,
                                                                  int64_t terms, float* __restrict__ M, int64_t ldm) {
    using R = Row<V>;
    const int lane = threadIdx.x & 63;
    const int64_t m = static_cast<int64_t>(blockIdx.x) * kWaves + (threadIdx.x >> 6);
    if (m >= msgs) return;
    int64_t b, e;
    bool ok = term_range(off, m, terms, b, e) && e > b;
    float* dst = M + m * ldm;
    if (ok && e - b <= 64) {
        // lane j holds term j's row; one vote checks them all
        const int cnt = static_cast<int>(e - b);
        int32_t rj = 0;
        bool bad = false;
        if (lane < cnt) {
            rj = rows[b + lane];
            bad = rj < 0 || rj >= q;
        }
        ok = __ballot(bad) == 0;
        for (int64_t c = static_cast<int64_t>(lane) * V; c < r; c += 64 * V) {
            if (!ok) {
                R::store(dst + c, R::nan());
                continue;
            }
            auto row = [&](int j) __attribute__((always_inline)) {
                return R::load(A + static_cast<int64_t>(__builtin_amdgcn_readlane(rj, j)) * lda + c);
            };
            typename R::T acc = row(0);
            int j = 1;
            for (; j + 4 <= cnt; j += 4) {
                const typename R::T x0 = row(j), x1 = row(j + 1), x2 = row(j + 2), x3 = row(j + 3);
                acc = acc + x0;
                acc = acc + x1;
                acc = acc + x2;
                acc = acc + x3;
            }
            for (; j < cnt; ++j) acc = acc + row(j);
            R::store(dst + c, acc);
        }
        return;
    }
    // more than 64 terms (no plan has them: n <= 64), or a bad range
    for (int64_t t = b; ok && t < e; ++t) ok = rows[t] >= 0 && rows[t] < q;
    for (int64_t c = static_cast<int64_t>(lane) * V; c < r; c += 64 * V) {
        if (!ok) {
            R::store(dst + c, R::nan());
            continue;
        }
        typename R::T acc = R::load(A + static_cast<int64_t>(rows[b]) * lda + c);
        int64_t t = b + 1;
        for (; t + 4 <= e; t += 4) {
            const typename R::T x0 = R::load(A + static_cast<int64_t>(rows[t]) * lda + c);
            const typename R::T x1 = R::load(A + static_cast<int64_t>(rows[t + 1]) * lda + c);
            const typename R::T x2 = R::load(A + static_cast<int64_t>(rows[t + 2]) * lda + c);
            const typename R::T x3 = R::load(A + static_cast<int64_t>(rows[t + 3]) * lda + c);
            acc = acc + x0;
            acc = acc + x1;
            acc = acc + x2;
            acc = acc + x3;
        }
        for (; t < e; ++t) acc = acc + R::load(A + static_cast<int64_t>(rows[t]) * lda + c);
        R::store(dst + c, acc);
    }
}

// One wave per message m: its row and its terms' rows are read once (up to
// kTermRegs of them held in registers) and every term d of the message is
// written as the message minus the other terms' rows, in order.
constexpr int kTermRegs = 8;

template <int V>
__global__ __launch_bounds__(kThreads) void shuffle_decode_kernel(const float* __restrict__ A, int64_t q, int64_t r,
                                                                  int64_t lda, const float* __restrict__ M,
                                                                  int64_t ldm, const int64_t* __restrict__ off,
                                                                  const int32_t* __restrict__ rows,
                                                                  const int32_t* __restrict__ msg, int64_t msgs,
                                                                  int64_t terms, float* __restrict__ out,
                                                                  int64_t ldo) {
    using R = Row<V>;
    const int lane = threadIdx.x & 63;
    const int64_t m = static_cast<int64_t>(blockIdx.x) * kWaves + (threadIdx.x >> 6);
    if (m >= msgs) return;
    int64_t b, e;
    if (!term_range(off, m, terms, b, e)) return;          // no term of this message can be placed
    const int64_t cnt = e - b;
    if (cnt <= kTermRegs) {
        // lane j holds term j's row; one vote checks them all
        int32_t rj = 0;
        bool bad = false;
        if (lane < cnt) {
            rj = rows[b + lane];
            bad = rj < 0 || rj >= q || msg[b + lane] != m;
        }
        const bool okv = __ballot(bad) == 0;
        for (int64_t c = static_cast<int64_t>(lane) * V; c < r; c += 64 * V) {
            if (!okv) {
                for (int64_t d = b; d < e; ++d) R::store(out + d * ldo + c, R::nan());
                continue;
            }
            const typename R::T mv = R::load(M + m * ldm + c);
            typename R::T x[kTermRegs];
#pragma unroll
            for (int j = 0; j < kTermRegs; ++j)
                if (j < cnt) x[j] = R::load(A + static_cast<int64_t>(__builtin_amdgcn_readlane(rj, j)) * lda + c);
#pragma unroll
            for (int i = 0; i < kTermRegs; ++i) {
                if (i < cnt) {
                    typename R::T acc = mv;
#pragma unroll
                    for (int j = 0; j < kTermRegs; ++j)
                        if (j < cnt && j != i) acc = acc - x[j];
                    R::store(out + (b + i) * ldo + c, acc);
                }
            }
        }
        return;
    }
    bool ok = true;
    for (int64_t t = b; ok && t < e; ++t) ok = rows[t] >= 0 && rows[t] < q && msg[t] == m;
    for (int64_t c = static_cast<int64_t>(lane) * V; c < r; c += 64 * V) {
        if (!ok) {
            for (int64_t d = b; d < e; ++d) R::store(out + d * ldo + c, R::nan());
            continue;
        }
        const typename R::T mv = R::load(M + m * ldm + c);
        if (cnt <= kTermRegs) {
            typename R::T x[kTermRegs];
#pragma unroll
            for (int j = 0; j < kTermRegs; ++j)
                if (j < cnt) x[j] = R::load(A + static_cast<int64_t>(rows[b + j]) * lda + c);
#pragma unroll
            for (int i = 0; i < kTermRegs; ++i) {
                if (i < cnt) {
                    typename R::T acc = mv;
#pragma unroll
                    for (int j = 0; j < kTermRegs; ++j)
                        if (j < cnt && j != i) acc = acc - x[j];
                    R::store(out + (b + i) * ldo + c, acc);
                }
            }
        } else {
            for (int64_t d = b; d < e; ++d) {
                typename R::T acc = mv;
                for (int64_t t = b; t < e; ++t)
                    if (t != d) acc = acc - R::load(A + static_cast<int64_t>(rows[t]) * lda + c);
                R::store(out + d * ldo + c, acc);
            }
        }
    }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) % 16) == 0; }

}  // namespace

hipError_t launch_shuffle_encode(const float* A, int64_t q, int64_t r, int64_t lda, const int64_t* off,
                                 const int32_t* rows, int64_t msgs, int64_t terms, float* M, int64_t ldm,
                                 hipStream_t st) {
    if (msgs == 0 || r == 0) return hipSuccess;
    const int64_t blocks = ceil_div(msgs, kWaves);
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const bool vec = r % 4 == 0 && lda % 4 == 0 && ldm % 4 == 0 && aligned16(A) && aligned16(M);
    if (vec)
        hipLaunchKernelGGL(shuffle_encode_kernel<4>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, st, A, q,
                           r, lda, off, rows, msgs, terms, M, ldm);
    else
        hipLaunchKernelGGL(shuffle_encode_kernel<1>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, st, A, q,
                           r, lda, off, rows, msgs, terms, M, ldm);
    return hipGetLastError();
}

hipError_t launch_shuffle_decode(const float* A, int64_t q, int64_t r, int64_t lda, const float* M, int64_t ldm,
                                 const int64_t* off, const int32_t* rows, const int32_t* msg, int64_t msgs,
                                 int64_t terms, float* out, int64_t ldo, hipStream_t st) {
    if (terms == 0 || msgs == 0 || r == 0) return hipSuccess;
    const int64_t blocks = ceil_div(msgs, kWaves);
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const bool vec = r % 4 == 0 && lda % 4 == 0 && ldm % 4 == 0 && ldo % 4 == 0 && aligned16(A) && aligned16(M) &&
                     aligned16(out);
    if (vec)
        hipLaunchKernelGGL(shuffle_decode_kernel<4>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, st, A, q,
                           r, lda, M, ldm, off, rows, msg, msgs, terms, out, ldo);
    else
        hipLaunchKernelGGL(shuffle_decode_kernel<1>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, st, A, q,
                           r, lda, M, ldm, off, rows, msg, msgs, terms, out, ldo);
    return hipGetLastError();
}

}  // namespace coded
