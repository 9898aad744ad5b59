// Encode and worker products in one pass over A (Sec. III-A: the parity
// blocks A'_{k+p} = sum_j P[p][j] A_j, then every worker's product A'_i X),
// for bf16 inputs with hi + lo parity planes and fp32 accumulation.
//
// Run separately, the encode reads A and writes the parity planes, and the
// worker products read A and the planes again.  Here each 16-row tile of
// every block is read from HBM once, into LDS, and serves three uses there:
//   the encode, on the matrix cores: for one column of the tile the parity
//     values of all n-k rows are P (n-k x k, bf16 values, exact) times the
//     k block values of that column, one 16x16x32 product per column with P
//     as the first operand (rows p, K = j) and the column's values as the
//     second (K = j, N = the 16 rows of the tile);
//   the parity planes: hi = bf16(sum), lo = bf16(sum - hi), staged in LDS
//     and written to HBM with row-contiguous 16-byte stores;
//   the worker products of the systematic blocks and of both parity planes
//     (PRODUCTS), 16x16x32 products against X^T staged in LDS.
// HBM traffic falls from 2(q r + 2(n-k) qb r) + 2 q r bytes (encode, then
// products) to 2 q r + 4 (n-k) qb r bytes.  The separate encode of the same
// shapes runs this kernel without PRODUCTS, so both write the same planes.
//
// Work split: one workgroup per compute unit, over the units (16-row tile,
// 64-deep K stage) in order; each workgroup takes an equal run of units, so
// a tile is shared by at most two workgroups (the run is at least one tile).
// Partial tiles are added into Y with float atomics on a zero-filled Y; with
// at most two addends onto zero the result does not depend on their order.
//
// LDS tiles hold rows of 128 bytes (eight 16-byte pieces); piece c of row i
// is stored at position c ^ (i & 7) ^ ((i >> 3) & 1), so a 16-byte access of
// the same piece in 8 or 16 consecutive rows, and a row write, touch distinct
// banks.
#include "internal.h"

namespace coded {
namespace {

typedef __bf16 bf16x8f __attribute__((ext_vector_type(8)));
typedef float f32x4f __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4f __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2f __attribute__((ext_vector_type(2)));
typedef float f32x2f __attribute__((ext_vector_type(2)));
typedef unsigned int u32x2f __attribute__((ext_vector_type(2)));

constexpr int kStage = 64;   // K elements per stage (one 128-byte row piece set)

__device__ inline int swz(int row, int piece) { return row * 8 + (piece ^ (row & 7) ^ ((row >> 3) & 1)); }

template <int WAVES, int K, int NPAR, bool PRODUCTS>
__global__ __launch_bounds__(WAVES * 64, 1) void fused_bf16_kernel(FusedArgs a) {
    constexpr int T = WAVES * 64;
    constexpr int AP = K * 16 * 8 / T;        // A pieces per thread per stage
    constexpr int XPn = 64 * 8 / T;           // X^T pieces per thread per stage
    constexpr int PP = 2 * NPAR * 16 * 8 / T; // parity pieces per thread per stage
    constexpr int SL = 8 / WAVES;             // encode column groups (of 8) per wave
    constexpr int KW = K / WAVES, PW = NPAR / WAVES;
    static_assert(K * 16 * 8 % T == 0 && 2 * NPAR * 16 * 8 % T == 0 && 8 % WAVES == 0, "shape");
    static_assert(K <= 32 && NPAR <= 16 && K % WAVES == 0 && NPAR % WAVES == 0 && NPAR % 4 == 0, "shape");

    __shared__ u32x4f sA[2][K * 16 * 8];
    __shared__ u32x4f sP[2 * NPAR * 16 * 8];
    __shared__ u32x4f sX[PRODUCTS ? 2 : 1][PRODUCTS ? 64 * 8 : 1];

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, lk = lane >> 4;
    const int64_t plane = static_cast<int64_t>(NPAR) * a.qb * a.r;

    // P as the encode's first operand: lane (li, lk) holds P[li][8 lk + e]
    u32x4f pf;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        uint32_t lo = 0, hi = 0;
        const int j0 = 8 * lk + 2 * d;
        if (li < NPAR && j0 < K) lo = __float_as_uint(a.P[li * K + j0]) >> 16;
        if (li < NPAR && j0 + 1 < K) hi = __float_as_uint(a.P[li * K + j0 + 1]) >> 16;
        pf[d] = lo | (hi << 16);
    }
    const bf16x8f pfrag = __builtin_bit_cast(bf16x8f, pf);

    f32x4f acc[PRODUCTS ? KW + PW : 1][4];
    auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int b = 0; b < (PRODUCTS ? KW + PW : 1); ++b)
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[b][c] = f32x4f{0.f, 0.f, 0.f, 0.f};
    };
    zero_acc();

    const int64_t u0 = static_cast<int64_t>(blockIdx.x) * a.per;
    const int64_t u1 = min<int64_t>(a.units, u0 + a.per);

    // Two sets of staging registers: the loads of unit u + 2 are issued into
    // the set that unit u has just been written to LDS from, so two stages of
    // loads are in flight while one is computed.
    u32x4f ar[2][AP], xr[2][PRODUCTS ? XPn : 1];
    int64_t aoff[AP];
    int64_t cur_tile = -1;
    auto set_tile = [&](int64_t tile) __attribute__((always_inline)) {
        const int64_t t0 = tile * 16;
#pragma unroll
        for (int i = 0; i < AP; ++i) {
            const int e = tid + T * i;
            const int j = e >> 7, row = (e >> 3) & 15, p8 = e & 7;
            const int64_t rg = static_cast<int64_t>(j) * a.qb + min<int64_t>(t0 + row, a.qb - 1);
            aoff[i] = min<int64_t>(rg, a.q - 1) * a.lda + 8 * p8;
        }
        cur_tile = tile;
    };
    // (tile, stage) of a unit, advanced one unit at a time (no division in the loop)
    const int nst = static_cast<int>(a.stages);
    struct Cursor {
        int tile, s;
    };
    auto advance = [&](Cursor& c) __attribute__((always_inline)) {
        if (++c.s == nst) {
            c.s = 0;
            ++c.tile;
        }
    };
    auto load = [&](int set, const Cursor& cu) __attribute__((always_inline)) {
        const int64_t tile = cu.tile;
        if (tile != cur_tile) set_tile(tile);
        const int64_t kc = cu.s * kStage;
#pragma unroll
        for (int i = 0; i < AP; ++i) ar[set][i] = *reinterpret_cast<const u32x4f*>(a.A + aoff[i] + kc);
        if constexpr (PRODUCTS) {
#pragma unroll
            for (int i = 0; i < XPn; ++i) {
                const int e = tid + T * i;
                xr[set][i] =
                    *reinterpret_cast<const u32x4f*>(a.xt + static_cast<int64_t>(e >> 3) * a.r + 8 * (e & 7) + kc);
            }
        }
    };

    Cursor cc{static_cast<int>(u0 / a.stages), static_cast<int>(u0 % a.stages)};   // the unit being computed
    Cursor cl = cc;                              // the unit being loaded
    auto body = [&](int set, int64_t u) __attribute__((always_inline)) {
        const int b = set;
        const int64_t tile = cc.tile;
        const int64_t s = cc.s;
        const int64_t t0 = tile * 16;
        const bool masked = tile >= a.clean_tiles;
        // stage u into LDS (padding rows as zeros), then start the loads of u + 2
#pragma unroll
        for (int i = 0; i < AP; ++i) {
            const int e = tid + T * i;
            u32x4f v = ar[set][i];
            if (masked) {
                const int64_t t = t0 + ((e >> 3) & 15);
                if (t >= a.qb || static_cast<int64_t>(e >> 7) * a.qb + t >= a.q) v = u32x4f{0u, 0u, 0u, 0u};
            }
            sA[b][(e >> 7) * 128 + swz((e >> 3) & 15, e & 7)] = v;
        }
        if constexpr (PRODUCTS) {
#pragma unroll
            for (int i = 0; i < XPn; ++i) {
                const int e = tid + T * i;
                sX[b][swz(e >> 3, e & 7)] = xr[set][i];
            }
        }
        if (u + 2 < u1) advance(cl);             // else the last unit is loaded again
        load(set, cl);
        __syncthreads();

        // encode: column groups g of this wave; lane (li, lk) reads blocks 8 lk .. 8 lk + 7
#pragma unroll
        for (int sl = 0; sl < SL; ++sl) {
            const int g = w * SL + sl;
            u32x4f R[8];
#pragma unroll
            for (int bb = 0; bb < 8; ++bb) {
                const int j = 8 * lk + bb;
                R[bb] = j < K ? sA[b][j * 128 + swz(li, g)] : u32x4f{0u, 0u, 0u, 0u};
            }
            // two halves of four columns: column e of the group is blocks
            // 8 lk .. 8 lk + 7 of row li, packed in pairs
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                f32x4f C[4];
#pragma unroll
                for (int ee = 0; ee < 4; ++ee) {
                    const int e = 4 * hf + ee;
                    u32x4f tv;
                    const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
                    for (int d = 0; d < 4; ++d)
                        tv[d] = __builtin_amdgcn_perm(R[2 * d + 1][e >> 1], R[2 * d][e >> 1], sel);
                    C[ee] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pfrag, __builtin_bit_cast(bf16x8f, tv),
                                                                   f32x4f{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                }
                // lane (li, lk) holds parity rows p = 4 lk + v of tile row li, columns 8 g + 4 hf + ee
                if (lk < NPAR / 4) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        u32x2f hv, lv;
#pragma unroll
                        for (int d = 0; d < 2; ++d) {
                            // round to nearest even, two values per conversion
                            const float x0 = C[2 * d][v], x1 = C[2 * d + 1][v];
                            const uint32_t h =
                                __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2f{x0, x1}, bf16x2f));
                            const f32x2f rr{x0 - __uint_as_float(h << 16), x1 - __uint_as_float(h & 0xFFFF0000u)};
                            hv[d] = h;
                            lv[d] = __builtin_bit_cast(uint32_t, __builtin_convertvector(rr, bf16x2f));
                        }
                        const int p = 4 * lk + v;
                        u32x2f* hp = reinterpret_cast<u32x2f*>(&sP[(p * 16) * 8 + swz(li, g)]);
                        u32x2f* lp = reinterpret_cast<u32x2f*>(&sP[((NPAR + p) * 16) * 8 + swz(li, g)]);
                        hp[hf] = hv;
                        lp[hf] = lv;
                    }
                }
            }
        }
        __syncthreads();

        // parity planes to HBM: 8 threads per 128-byte row piece set
        const int64_t kc = s * kStage;
#pragma unroll
        for (int i = 0; i < PP; ++i) {
            const int e = tid + T * i;
            const int pl = e >> 7, row = (e >> 3) & 15, p8 = e & 7;
            const int pln = pl / NPAR, p = pl % NPAR;
            if (!masked || t0 + row < a.qb)
                __builtin_nontemporal_store(sP[pl * 128 + swz(row, p8)],
                                            reinterpret_cast<u32x4f*>(a.parity + pln * plane +
                                                                      (p * a.qb + t0 + row) * a.r + kc + 8 * p8));
        }

        if constexpr (PRODUCTS) {
            bf16x8f bx[2][4];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    bx[ks][c] = __builtin_bit_cast(bf16x8f, sX[b][swz(16 * c + li, 4 * ks + lk)]);
#pragma unroll
            for (int jj = 0; jj < KW; ++jj) {
                const int j = w * KW + jj;
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const bf16x8f af = __builtin_bit_cast(bf16x8f, sA[b][j * 128 + swz(li, 4 * ks + lk)]);
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        acc[jj][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bx[ks][c], acc[jj][c], 0, 0, 0);
                }
            }
#pragma unroll
            for (int pp = 0; pp < PW; ++pp) {
                const int p = w * PW + pp;
#pragma unroll
                for (int pln = 0; pln < 2; ++pln)
#pragma unroll
                    for (int ks = 0; ks < 2; ++ks) {
                        const bf16x8f af =
                            __builtin_bit_cast(bf16x8f, sP[((pln * NPAR + p) * 16) * 8 + swz(li, 4 * ks + lk)]);
#pragma unroll
                        for (int c = 0; c < 4; ++c)
                            acc[KW + pp][c] =
                                __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bx[ks][c], acc[KW + pp][c], 0, 0, 0);
                    }
            }
            if (s == a.stages - 1 || u == u1 - 1) {
                // this workgroup's share of the tile (result lane l item v = C[4 lk + v][li])
#pragma unroll
                for (int bb = 0; bb < KW + PW; ++bb) {
                    const int64_t blk = bb < KW ? w * KW + bb : K + w * PW + (bb - KW);
#pragma unroll
                    for (int c = 0; c < 4; ++c)
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            const int64_t t = t0 + 4 * lk + v;
                            if (!masked || t < a.qb)
                                unsafeAtomicAdd(a.Y + (blk * a.qb + t) * 64 + 16 * c + li, acc[bb][c][v]);
                        }
                }
                zero_acc();
            }
        }
        advance(cc);
    };

    load(0, cl);
    if (u0 + 1 < u1) advance(cl);
    load(1, cl);
    for (int64_t u = u0; u < u1; u += 2) {
        body(0, u);
        if (u + 1 < u1) body(1, u + 1);
    }
}

__global__ void zero_f32_kernel(float* p, int64_t n) {
    const int64_t i = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 4;
    if (i + 4 <= n)
        *reinterpret_cast<f32x4f*>(p + i) = f32x4f{0.f, 0.f, 0.f, 0.f};
    else
        for (int64_t j = i; j < n; ++j) p[j] = 0.0f;
}

// Eight wavefronts per workgroup (two per SIMD): each owns three systematic
// blocks and one parity row of the products and one 8-column group of the
// encode.
constexpr int kWaves = 8;

}  // namespace

bool fused_bf16_supported(int n, int k, int planes, int64_t r, int64_t lda) {
    return planes == 2 && k == 24 && n - k == 8 && r > 0 && r % kStage == 0 && lda % 8 == 0;
}

hipError_t launch_fused_bf16(FusedArgs a, bool products, int compute_units, hipStream_t st) {
    if (a.qb == 0 || a.r == 0) return hipSuccess;
    hipError_t e;
    if (products) {
        const int64_t ny = static_cast<int64_t>(a.n) * a.qb * 64;
        hipLaunchKernelGGL(zero_f32_kernel, dim3(static_cast<unsigned>(ceil_div(ny, 4 * 256))), dim3(256), 0, st, a.Y,
                           ny);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const int64_t tiles = ceil_div(a.qb, 16);
    a.stages = a.r / kStage;
    a.units = tiles * a.stages;
    const int64_t groups = std::max<int64_t>(1, std::min<int64_t>(compute_units, tiles));
    a.per = std::max(ceil_div(a.units, groups), a.stages);   // a tile is shared by at most two workgroups
    const int64_t blocks = ceil_div(a.units, a.per);
    // tiles whose 16 rows lie inside every block (no clamped or zeroed row)
    const int64_t lim = std::min(a.qb, a.q - static_cast<int64_t>(a.k - 1) * a.qb);
    a.clean_tiles = lim > 0 ? lim / 16 : 0;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    if (products)
        hipLaunchKernelGGL((fused_bf16_kernel<kWaves, 24, 8, true>), dim3(static_cast<unsigned>(blocks)),
                           dim3(kWaves * 64), 0, st, a);
    else
        hipLaunchKernelGGL((fused_bf16_kernel<kWaves, 24, 8, false>), dim3(static_cast<unsigned>(blocks)),
                           dim3(kWaves * 64), 0, st, a);
    return hipGetLastError();
}

}  // namespace coded
