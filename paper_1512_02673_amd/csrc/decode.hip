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
#include "decode_common.h"

namespace coded {
namespace {

constexpr int kThreads = 256;

typedef float f32x4v __attribute__((ext_vector_type(4)));

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
template <int E, typename T>
__device__ inline void store_out(const DecodeArgs& a, float* p, int64_t off, const T* v) {
    float w[E];
    if (a.c) {
        float cv[E];
        if constexpr (E == 4) {
            const float4 f = *reinterpret_cast<const float4*>(a.c + off);
            cv[0] = f.x; cv[1] = f.y; cv[2] = f.z; cv[3] = f.w;
        } else {
            cv[0] = a.c[off];
        }
#pragma unroll
        for (int i = 0; i < E; ++i)
            w[i] = static_cast<float>(fma(a.alpha, static_cast<double>(v[i]), a.beta * static_cast<double>(cv[i])));
    } else {
#pragma unroll
        for (int i = 0; i < E; ++i) w[i] = static_cast<float>(v[i]);
    }
    // decoded outputs are written once and not read again here: non-temporal
    if constexpr (E == 4) {
        const f32x4v q = {w[0], w[1], w[2], w[3]};
        __builtin_nontemporal_store(q, reinterpret_cast<f32x4v*>(p + off));
    } else {
        __builtin_nontemporal_store(w[0], p + off);
    }
}

// E consecutive elements of Y as fp32 (a copied systematic block is the
// worker's result rounded to the output type).
template <int E, typename YT>
__device__ inline void load_f32(const YT* p, float* v) {
    if constexpr (E == 4 && sizeof(YT) == 4) {
        const float4 f = *reinterpret_cast<const float4*>(p);
        v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
    } else if constexpr (E == 4) {
        const double2 lo = reinterpret_cast<const double2*>(p)[0], hi = reinterpret_cast<const double2*>(p)[1];
        v[0] = static_cast<float>(lo.x); v[1] = static_cast<float>(lo.y);
        v[2] = static_cast<float>(hi.x); v[3] = static_cast<float>(hi.y);
    } else {
        v[0] = static_cast<float>(p[0]);
    }
}

// PASS: missing outputs computed per sweep over the survivors (register
// bucket); E: elements per thread; ST (>= every m of the launch, even) is the
// row stride of the LDS matrices, sized on the host.
template <int PASS, int E, typename YT>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeArgs a, DecodeSet single, int64_t chunks,
                                                          int elems_per_block, int ST) {
    __shared__ SetMeta sm;
    extern __shared__ __align__(16) double dyn[];
    double* sD = dyn;                    // D column-major: sD[c * ST + b], c < k
    double* sMat = dyn + a.k * ST;       // m x m, row stride ST
    double* sL = sMat + ST * ST;         // multipliers of one elimination step

    const int tid = threadIdx.x;
    const int k = a.k;
    const int64_t b = blockIdx.x / chunks;
    const int64_t chunk = blockIdx.x % chunks;
    const bool writer = (chunk == 0 && tid == 0);
    if (!setup_set<kThreads>(a, single, b, writer, sm)) return;
    const int32_t* sS = sm.S;
    const int32_t* sMiss = sm.miss;
    const int64_t* sYoff = sm.yoff;
    const int64_t* sOoff = sm.ooff;
    const int32_t* sLim = sm.lim;
    const int m = sm.m;
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
                if (best == 0.0) sm.status = first_par + j + 1;
                sm.raw[0] = p;                     // reuse: pivot row of this step
            }
            __syncthreads();
            if (sm.status != 0) break;
            const int p = sm.raw[0];
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
                // consecutive threads walk down a column of D (contiguous in LDS)
                for (int e = tid; e < rows * k; e += kThreads) {
                    const int c = e / rows, i = j + 1 + e % rows;
                    sD[c * ST + i] -= sL[i] * sD[c * ST + j];
                }
            }
            __syncthreads();
        }
        if (sm.status != 0) {
            if (writer) a.info[b] = sm.status;
            return;
        }
        // Back substitution with U, one step per pivot from the bottom: scale
        // row i of D, then eliminate it from the rows above (consecutive
        // threads walk down a column, contiguous in LDS).
        for (int i = m - 1; i >= 0; --i) {
            for (int c = tid; c < k; c += kThreads) sD[c * ST + i] /= sMat[i * ST + i];
            __syncthreads();
            if (i > 0) {
                for (int e = tid; e < i * k; e += kThreads) {
                    const int c = e / i, ii = e % i;
                    sD[c * ST + ii] -= sMat[ii * ST + i] * sD[c * ST + i];
                }
                __syncthreads();
            }
        }
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

// ---------------------------------------------------------------- fast path
// Codes with at most kFastM missing blocks per set and m + k <= 64: one wave
// eliminates the m x (m + k) system [G[S_par, M] | -G[S_par, S_sys] | I] in
// registers (Gauss-Jordan, partial pivoting: the same pivots as the LU above,
// one column per lane, no workgroup barriers), and the combination of the
// survivors is one 16-row matrix-core tile:
//     out[M] (16 x 16 elements) += D (16 x 4 survivors) * Y (4 x 16 elements)
// on v_mfma_f64_16x16x4f64, with D held in registers for the whole set.
typedef double f64x4v __attribute__((ext_vector_type(4)));

// Consecutive elements per lane in the combination's loads (E == 4 path);
// 4 needs 192 registers at k = 48 (2 waves per SIMD) and measured slower.
constexpr int kDecodePE = 2;

// PE consecutive elements of Y (16-byte aligned for fp64 pairs, PE * 4-byte
// aligned for fp32) with vector loads.
template <int PE, typename YT>
__device__ inline void load_pe(const YT* p, YT (&v)[PE]) {
    if constexpr (sizeof(YT) == 8) {
#pragma unroll
        for (int i = 0; i < PE; i += 2) {
            const double2 d = reinterpret_cast<const double2*>(p)[i / 2];
            v[i] = d.x;
            v[i + 1] = d.y;
        }
    } else if constexpr (PE == 4) {
        const float4 f = *reinterpret_cast<const float4*>(p);
        v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
    } else {
        const float2 f = *reinterpret_cast<const float2*>(p);
        v[0] = f.x; v[1] = f.y;
    }
}

// SIMD of the calling wave within its compute unit (hardware register
// HW_ID, bits 5:4).  The four waves of a 256-thread workgroup run on four
// different SIMDs.
__device__ inline int simd_id() {
    return static_cast<int>(__builtin_amdgcn_s_getreg(4 | (4 << 6) | ((2 - 1) << 11)) & 3);
}

// One workgroup per (set, chunk).
// E == 4: the wave on SIMD 0 of its compute unit (wave 0 if none is) forms
// D and then copies the systematic survivors; the other three waves combine
// the missing blocks on the fp64 matrix cores.  Vector instructions do not
// overlap with fp64 matrix instructions on the same SIMD, so every compute
// unit keeps the copies and the elimination on one SIMD and the matrix work
// on the other three.  Which wave takes which role changes only the timing.
// E == 1: wave 0 eliminates while the others start copying; then all four
// combine.
// KS: matrix-core K steps (4 survivors each) the kernel is built for, k <= 4 KS;
// FULL: k == 4 KS (no padding steps).
// Raw buffer over `bytes` bytes (gfx9 dword-3 value: no stride, no format).
__device__ inline __amdgpu_buffer_rsrc_t y_buffer(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0), static_cast<int>(bytes),
                                             0x00020000);
}

// YBUF (E == 4, Y's byte offsets below 2^31): the combining waves read Y as a
// raw buffer, each lane's offset per survivor fixed for the set and the
// group's offset in a scalar register, so the loads need no vector address
// arithmetic.
// Six waves per SIMD (80 registers, six workgroups per compute unit) for the
// variants with whole survivor groups and buffer-addressed Y up to 12 groups,
// which then spill one word in the elimination; the others keep the default
// register budget.
template <int KS, bool FULL, bool YBUF>
constexpr int decode_min_waves() {
    return FULL && YBUF && KS <= 12 ? 6 : 1;
}

template <int KS, int E, typename YT, bool FULL, bool YBUF>
__global__ __launch_bounds__(kThreads, (decode_min_waves<KS, FULL, YBUF>())) void decode_mfma_kernel(
    DecodeArgs args, DecodeSet single, int64_t chunks, int elems_per_block) {
    __shared__ SetMeta sm;
    __shared__ double sD[64 * kFastLd];
    __shared__ double sOut[E == 4 ? kThreads / 64 - 1 : 1][E == 4 ? 256 * kDecodePE : 1];   // per combining wave output tile
    __shared__ int32_t sSimd[kThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    DecodeArgs a = args;
    if constexpr (E == 1) {
        // Short chunks, latency bound: the sizes the set-up and the first
        // loads depend on are fetched in one batch and held in scalar
        // registers (left alone, the compiler fetches them one dependent
        // round trip after another).
        asm volatile("" : "+s"(a.q), "+s"(a.qb), "+s"(a.s), "+s"(a.ldo), "+s"(a.n), "+s"(a.k), "+s"(chunks),
                     "+s"(elems_per_block));
    }
    const int k = a.k;
    // fewer than 2^31 workgroups (checked at launch): 32-bit division
    const uint32_t bid = blockIdx.x, nch = static_cast<uint32_t>(chunks);
    const int64_t b = bid / nch;
    const int64_t chunk = bid - static_cast<uint32_t>(b) * nch;
    const bool writer = (chunk == 0 && tid == 0);
    if (lane == 0) sSimd[wv] = simd_id();             // read after setup_set's barriers
    if (!setup_set<kThreads>(a, single, b, writer, sm)) return;
    const int m = sm.m;
    const int first_par = k - m;
    const YT* Y = static_cast<const YT*>(a.Y);
    float* out = a.out + b * a.out_stride;
    const int s = static_cast<int>(a.s);
    const int total = static_cast<int>(a.qb * a.s);
    const int e0 = static_cast<int>(chunk) * elems_per_block;
    const int e1 = min(total, e0 + elems_per_block);
    constexpr int kWaves = kThreads / 64;

    // E == 1 (chunks of single elements, often short): the systematic
    // survivors are copied as (element, survivor) items spread over the
    // waves that do not eliminate, and the first CI items of each thread are
    // loaded before the barrier that publishes the elimination's status (and
    // stored only after it: a singular set writes nothing).
    constexpr int CI = 4;
    const int len = e1 - e0, items = len * first_par;
    const int cw = m > 0 ? 1 : 0, nthr = kThreads - 64 * cw, ctid = tid - 64 * cw;
    YT cy[CI];
    int64_t co[CI];                      // output offset of item i, -1 for none
    if constexpr (E == 1) {
#pragma unroll
        for (int i = 0; i < CI; ++i) {
            const int it = ctid + i * nthr;
            co[i] = -1;
            cy[i] = YT(0);
            if (ctid >= 0 && it < items) {
                const int c = it / len, e = e0 + (it - c * len);
                const int t = e / s, col = e - t * s;
                const int w = sm.S[c];
                if (t < sm.lim[w]) {
                    cy[i] = Y[sm.yoff[c] + e];
                    co[i] = sm.ooff[w] + static_cast<int64_t>(t) * a.ldo + col;
                }
            }
        }
    }

    // E == 1: each wave's first tile of Y (Y_{S[4 st + lk]} at element li of
    // the tile, as the tile loop below reads it) is requested before the
    // barrier that publishes D, so its latency overlaps the elimination.
    const int ntiles1 = (e1 - e0 + 15) / 16;
    YT yfirst[E == 1 ? KS : 1];
    if constexpr (E == 1) {
        if (m > 0 && wv < ntiles1) {
            const int li = lane & 15, lk = lane >> 4;
            const int el = min(e0 + wv * 16 + li, e1 - 1);
#pragma unroll
            for (int st = 0; st < KS; ++st) {
                const int c = 4 * st + lk;
                yfirst[st] = Y[(c < k ? static_cast<int32_t>(sm.yoff[c]) : 0) + el];
            }
        }
    }

    // the eliminating wave (E == 4: also the copying wave)
    int ew = 0;
    if constexpr (E == 4) {
#pragma unroll
        for (int w = kWaves - 1; w >= 0; --w) ew = sSimd[w] == 0 ? w : ew;
    }
    if (m > 0 && wv == ew) eliminate_set(a, sm, m, first_par, lane, sD);
    __syncthreads();
    if (sm.status != 0) {
        if (writer) a.info[b] = sm.status;
        return;
    }
    if (writer) a.info[b] = 0;

    if constexpr (E == 1) {
#pragma unroll
        for (int i = 0; i < CI; ++i) {
            if (co[i] >= 0) {
                const float fv = static_cast<float>(cy[i]);   // the worker's result in the output type
                store_out<1>(a, out, co[i], &fv);
            }
        }
        for (int it = ctid + CI * nthr; ctid >= 0 && it < items; it += nthr) {
            const int c = it / len, e = e0 + (it - c * len);
            const int t = e / s, col = e - t * s;
            const int w = sm.S[c];
            if (t < sm.lim[w]) {
                const float fv = static_cast<float>(Y[sm.yoff[c] + e]);
                store_out<1>(a, out, sm.ooff[w] + static_cast<int64_t>(t) * a.ldo + col, &fv);
            }
        }
    }

    // E == 4: the copying wave takes the systematic survivors block by block,
    // U four-element items per lane in flight (a batch past the block's end
    // re-reads its last item and stores nothing).  With dense output rows
    // (ldo == s) element e of a block is at offset e from its first row.
    if constexpr (E == 4) {
        if (wv == ew) {
            constexpr int U = 4;
            const bool dense = a.ldo == a.s;
            for (int c = 0; c < first_par; ++c) {
                const int w = sm.S[c];
                const YT* yr = Y + sm.yoff[c];
                float* ob = out + sm.ooff[w];
                const int elim = min(e1, sm.lim[w] * s);    // the block's elements inside A
                for (int e = e0 + 4 * lane; e < elim; e += 256 * U) {
                    float v[U][4];
#pragma unroll
                    for (int u = 0; u < U; ++u) load_f32<4, YT>(yr + min(e + 256 * u, elim - 4), v[u]);
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        const int ee = e + 256 * u;
                        if (ee < elim) {
                            const int64_t off = dense ? ee : static_cast<int64_t>(ee / s) * a.ldo + ee % s;
                            store_out<4>(a, ob, off, v[u]);
                        }
                    }
                }
            }
            return;
        }
    }
    if (m == 0) return;

    // Missing blocks: 16-element tiles, one wave per tile.  Lane (li, lk)
    // holds D[li][4 st + lk] (A operand) and loads Y_{S[4 st + lk]}[e] (B);
    // accumulator item v is out block M[4 v + lk], element li of the tile.
    const int li = lane & 15, lk = lane >> 4;
    double af[KS];
    int32_t yo[KS];
    uint32_t valid = 0;                   // bit st: survivor 4 st + lk exists
#pragma unroll
    for (int st = 0; st < KS; ++st) {
        const int c = 4 * st + lk;
        af[st] = c < k ? sD[c * kFastLd + li] : 0.0;
        yo[st] = c < k ? static_cast<int32_t>(sm.yoff[c]) : 0;
        valid |= (c < k ? 1u : 0u) << st;
    }
    if constexpr (E == 4) {
        // Tiles in groups of PE: lane (li, lk) loads elements PE li .. PE li +
        // PE - 1 of a 16 PE-element group at once, and PE matrix-core
        // products take the elements in each phase.  The results go through
        // this wave's LDS tile (16 blocks x 16 PE elements, fp64) back into
        // element order, and each lane writes 4 consecutive elements of one
        // block per 16-byte store.  (E == 4: s % 4 == 0 and Y, out 16-byte
        // aligned, so the chunk bounds and the total are multiples of 4.)
        constexpr int PE = kDecodePE;
        constexpr int W = 16 * PE;
        const int ngroups = (e1 - e0 + W - 1) / W;
        const int crank = __builtin_amdgcn_readfirstlane(wv < ew ? wv : wv - 1);   // rank among the combining waves
        double* buf = sOut[crank];
        // each store instruction covers 16 / PE blocks, 4 PE lanes (W
        // elements, whole 128-byte lines for PE = 2) per block; this lane's
        // block, its first row in out and its element limit are fixed for the set
        constexpr int QPB = 4 * PE;
        const int g4 = lane % QPB;
        float* obase[PE];
        int elim[PE];
#pragma unroll
        for (int h = 0; h < PE; ++h) {
            const int bb = lane / QPB + (16 / PE) * h;
            const int w = sm.miss[bb < m ? bb : 0];
            obase[h] = out + sm.ooff[w];
            elim[h] = bb < m ? min(e1, sm.lim[w] * s) : 0;   // 0: no block for this lane
        }
        const bool dense = a.ldo == a.s;
        // YBUF: byte offset of this lane's elements of survivor 4 st + lk (a
        // group's elements past the block's end read the next result or zeros
        // past the buffer; those columns are not stored)
        uint32_t yb[YBUF ? KS : 1];
        const __amdgpu_buffer_rsrc_t yrs =
            y_buffer(Y, static_cast<uint32_t>(YBUF ? static_cast<int64_t>(a.n) * total * sizeof(YT) : 0));
        if constexpr (YBUF) {
#pragma unroll
            for (int st = 0; st < KS; ++st) yb[st] = static_cast<uint32_t>((yo[st] + PE * li) * sizeof(YT));
        }
        for (int gp = crank; gp < ngroups; gp += kWaves - 1) {
            const int base = e0 + gp * W;
            YT yv[KS][PE];
            if constexpr (YBUF) {
                static_assert(PE == 2, "one 2-element load per survivor");
                const uint32_t so = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(base) * sizeof(YT));
#pragma unroll
                for (int st = 0; st < KS; ++st) {
                    if constexpr (sizeof(YT) == 8) {
                        const double2 d = __builtin_bit_cast(double2, __builtin_amdgcn_raw_buffer_load_b128(yrs, yb[st], so, 0));
                        yv[st][0] = d.x;
                        yv[st][1] = d.y;
                    } else {
                        const float2 f = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(yrs, yb[st], so, 0));
                        yv[st][0] = f.x;
                        yv[st][1] = f.y;
                    }
                }
            } else {
                // a group past the chunk's end reads the block's last PE elements
                // instead (in bounds; those columns are not stored)
                const int el = min(base + PE * li, total - PE);
#pragma unroll
                for (int st = 0; st < KS; ++st) load_pe<PE>(Y + yo[st] + el, yv[st]);
            }
            f64x4v acc[PE];
#pragma unroll
            for (int q = 0; q < PE; ++q) acc[q] = f64x4v{0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int st = 0; st < KS; ++st) {
                // padding steps (k not a multiple of 4) contribute exact zeros
                const bool ok = FULL || ((valid >> st) & 1u);
#pragma unroll
                for (int q = 0; q < PE; ++q)
                    acc[q] = __builtin_amdgcn_mfma_f64_16x16x4f64(af[st], ok ? static_cast<double>(yv[st][q]) : 0.0,
                                                                  acc[q], 0, 0, 0);
            }
            // item v of lane (li, lk): block 4 v + lk, element PE li + q of acc[q],
            // kept in the tile at [block][q][li] (one 8-byte write per item, no
            // register moves)
#pragma unroll
            for (int v = 0; v < 4; ++v)
#pragma unroll
                for (int q = 0; q < PE; ++q) buf[(4 * v + lk) * W + 16 * q + li] = acc[q][v];
#pragma unroll
            for (int h = 0; h < PE; ++h) {
                const int bb = lane / QPB + (16 / PE) * h, eg = base + 4 * g4;
                if (eg < elim[h]) {
                    // elements 4 g4 .. 4 g4 + 3: (li, q) = (2 g4, 0), (2 g4, 1), (2 g4 + 1, 0), (2 g4 + 1, 1)
                    static_assert(PE == 2, "tile order");
                    const double2 r0 = *reinterpret_cast<const double2*>(&buf[bb * W + 2 * g4]);
                    const double2 r1 = *reinterpret_cast<const double2*>(&buf[bb * W + 16 + 2 * g4]);
                    const double v4[4] = {r0.x, r1.x, r0.y, r1.y};
                    // s % 4 == 0: the four share one row; dense rows (ldo == s) need no division
                    const int64_t off = dense ? eg : static_cast<int64_t>(eg / s) * a.ldo + eg % s;
                    store_out<4>(a, obase[h], off, v4);
                }
            }
        }
    } else {
        for (int tile = wv; tile < ntiles1; tile += kWaves) {
            const int e = e0 + tile * 16 + li;
            // Straight-line loads, all issued before the first is used (the
            // first tile's before the barrier).  A lane past the chunk's end
            // reads its last element instead: column li of the product
            // depends on column li of Y only, and is not stored.
            const int el = min(e, e1 - 1);
            YT yv[KS];
#pragma unroll
            for (int st = 0; st < KS; ++st) yv[st] = tile == wv ? yfirst[st] : Y[yo[st] + el];
            f64x4v acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int st = 0; st < KS; ++st) {
                const double bv = (FULL || ((valid >> st) & 1u)) ? static_cast<double>(yv[st]) : 0.0;
                acc = __builtin_amdgcn_mfma_f64_16x16x4f64(af[st], bv, acc, 0, 0, 0);
            }
            if (e < e1) {
                const int t = e / s, col = e - t * s;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int bb = 4 * v + lk;
                    if (bb < m) {
                        const int w = sm.miss[bb];
                        const double val = acc[v];
                        if (t < sm.lim[w]) store_out<1>(a, out, sm.ooff[w] + static_cast<int64_t>(t) * a.ldo + col, &val);
                    }
                }
            }
        }
    }
}

// The fast path takes codes (not sets) by their largest possible m, so a set
// decodes with the same arithmetic alone or in a batch.
bool fast_path_ok(const DecodeArgs& a) {
    const int mmax = std::min(a.k, a.n - a.k);
    return mmax <= kFastM && a.k + mmax <= 64 && static_cast<int64_t>(a.n) * a.qb * a.s <= 0x7FFFFFFF;
}

template <int E>
hipError_t launch_fast(const DecodeArgs& a, const DecodeSet& single, hipStream_t st) {
    // About 1024 workgroups when the batch is small: a set is cut into chunks
    // of at least 64 elements (each workgroup repeats the small elimination),
    // which keeps the per-wave tile chains of a single decode short while the
    // repeated eliminations, one per workgroup on its first SIMD, stay few
    // (one (32,24) set of 64 columns: 45.6 us with 2048 workgroups, 34.0 with
    // 1024, 34.4 with 512, 40.9 with 256).
    const int64_t total = a.qb * a.s;
    const int64_t want = std::max<int64_t>(1, ceil_div(1024, a.batch));
    const int64_t per = std::max<int64_t>(64, ceil_div(ceil_div(std::max<int64_t>(total, 1), want), 16) * 16);
    const int64_t chunks = std::max<int64_t>(1, ceil_div(total, per));
    const int64_t blocks = chunks * a.batch;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const int ksteps = (a.k + 3) / 4;
    const dim3 grid(static_cast<unsigned>(blocks));
    const int per32 = static_cast<int>(per);
    // Y read as a raw buffer (E == 4) when its byte offsets fit in 31 bits
    const bool ybuf = E == 4 && static_cast<int64_t>(a.n) * total * (a.y_f64 ? 8 : 4) < (int64_t(1) << 31);
#define CODED_FAST_Y(KS, FULL, YB)                                                                             \
    do {                                                                                                       \
        if (a.y_f64)                                                                                           \
            hipLaunchKernelGGL((decode_mfma_kernel<KS, E, double, FULL, YB>), grid, dim3(kThreads), 0, st, a,  \
                               single, chunks, per32);                                                         \
        else                                                                                                   \
            hipLaunchKernelGGL((decode_mfma_kernel<KS, E, float, FULL, YB>), grid, dim3(kThreads), 0, st, a,   \
                               single, chunks, per32);                                                         \
    } while (0)
#define CODED_FAST_F(KS, FULL)                       \
    do {                                             \
        if (ybuf)                                    \
            CODED_FAST_Y(KS, FULL, E == 4);          \
        else                                         \
            CODED_FAST_Y(KS, FULL, false);           \
    } while (0)
#define CODED_FAST(KS)                          \
    do {                                        \
        if (a.k == 4 * (KS))                    \
            CODED_FAST_F(KS, true);             \
        else                                    \
            CODED_FAST_F(KS, false);            \
    } while (0)
    if (ksteps <= 4) CODED_FAST(4);
    else if (ksteps <= 8) CODED_FAST(8);
    else if (ksteps <= 12) CODED_FAST(12);
    else CODED_FAST(16);
#undef CODED_FAST
#undef CODED_FAST_F
#undef CODED_FAST_Y
    return hipGetLastError();
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
    if (fast_path_ok(a)) {
        const bool vec4 = a.s % 4 == 0 && a.ldo % 4 == 0 && aligned16(a.out) && aligned16(a.Y) &&
                          (a.batch == 1 || a.out_stride % 4 == 0) && (a.c == nullptr || aligned16(a.c));
        return vec4 ? launch_fast<4>(a, s, st) : launch_fast<1>(a, s, st);
    }
    const int rows = (std::max(mmax, 1) + 1) / 2 * 2;   // even: D pairs are read 16 bytes at a time
    if (mmax <= 2) return launch_p<2>(a, s, rows, st);
    if (mmax <= 4) return launch_p<4>(a, s, rows, st);
    return launch_p<8>(a, s, rows, st);
}

}  // namespace coded
