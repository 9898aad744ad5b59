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
// 64-deep K stage) in order; each workgroup takes an equal, even run of
// units, so a tile is shared by at most two workgroups (the run is at least
// one tile).  A is loaded four stages at a time: one wave instruction covers
// 2 rows x 512 contiguous bytes (four stages' columns) instead of 8 rows x
// 128 B, which HBM serves much faster; the last group of a tile whose stage
// count is not a multiple of four has empty stages, loaded but not computed.
// X^T, small and read from the cache, is loaded two stages at a time.
// Partial tiles are added into Y with float atomics on a zero-filled Y; with
// at most two addends onto zero the result does not depend on their order.
//
// Addressing: every load and store goes through a raw buffer resource whose
// base is the current 16-row tile of one block (of A, or of one parity row
// and plane) and whose size covers only that tile's rows inside the block.
// A lane's byte offset inside such a tile is fixed for the whole kernel and
// the stage's column offset is a scalar, so the K loop does no address
// arithmetic; rows past a block's end read as zeros (the zero padding of the
// last block) and their stores are dropped by the range check.
//
// LDS tiles hold rows of 128 bytes (eight 16-byte pieces); piece c of row i
// is stored at position c ^ (i & 7) ^ ((i >> 3) & 1), so a 16-byte access of
// the same piece in 8 or 16 consecutive rows, and a row write, touch distinct
// banks.
#include "internal.h"
#include "fused.h"

namespace coded {
namespace {

typedef __bf16 bf16x8f __attribute__((ext_vector_type(8)));
typedef float f32x4f __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4f __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2f __attribute__((ext_vector_type(2)));
typedef float f32x2f __attribute__((ext_vector_type(2)));
typedef unsigned int u32x2f __attribute__((ext_vector_type(2)));

constexpr int kStage = 64;   // K elements per stage (one 128-byte row piece set)
constexpr int kAuxNonTemporal = 2;   // cache-policy bits of a buffer access: nt

// Raw buffer resource over `bytes` bytes from `base` (no stride, no format);
// loads at offsets >= bytes return zeros and stores there are dropped.
__device__ inline __amdgpu_buffer_rsrc_t raw_buffer(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0), static_cast<int>(bytes),
                                             0x00020000);
}

__device__ inline int swz(int row, int piece) { return row * 8 + (piece ^ (row & 7) ^ ((row >> 3) & 1)); }

template <int WAVES, int K, int NPAR, bool PRODUCTS>
__global__ __launch_bounds__(WAVES * 64, 1) void fused_bf16_kernel(FusedArgs a) {
    constexpr int AB = K / WAVES;             // blocks of A each wave loads and stages
    constexpr int AQ = 8 * AB;                // A pieces per thread per four stages (8 row pairs per block)
    constexpr int XQ = 16 / WAVES;            // row quads of X^T per wave per pair of stages
    constexpr int PB = 2 * NPAR / WAVES;      // parity rows (of either plane) each wave stores
    constexpr int SL = 8 / WAVES;             // encode column groups (of 8) per wave
    constexpr int KW = K / WAVES, PW = NPAR / WAVES;
    static_assert(2 * NPAR % WAVES == 0 && 16 % WAVES == 0 && 8 % WAVES == 0, "shape");
    static_assert(K <= 32 && NPAR <= 16 && K % WAVES == 0 && NPAR % WAVES == 0 && NPAR % 4 == 0, "shape");

    __shared__ u32x4f sA[2][K * 16 * 8];
    __shared__ u32x4f sP[2 * NPAR * 16 * 8];
    __shared__ u32x4f sX[PRODUCTS ? 2 : 1][PRODUCTS ? 64 * 8 : 1];

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, lk = lane >> 4;
    const int64_t plane = static_cast<int64_t>(NPAR) * a.qb * a.r;
    // A wave moves whole 16-row tiles: blocks AB w .. AB w + AB - 1 of A,
    // X^T rows 4 XQ w .. 4 XQ w + 4 XQ - 1 and parity rows PB w .. PB w + PB - 1
    // (hi plane rows, then lo plane rows).  A loads: lane (rh, p32) takes the
    // 16-byte piece p32 of the 512 bytes (four stages) of row rh of a row
    // pair; the piece belongs to stage qs = p32 / 8 of the four.  X^T loads:
    // lane (rq, p16) takes piece p16 of the 256 bytes (two stages) of row rq
    // of a row quad, stage hs = p16 / 8 of the two.  Stores: lane (rr, p8)
    // writes piece p8 of rows rr and rr + 8.  Piece p8 = lane % 8 of its stage
    // in all three; the row pair's, quad's or second row's offset is a scalar.
    const int rh = lane >> 5, p32 = lane & 31, qs = p32 >> 3;
    const int rq = lane >> 4, p16 = lane & 15, hs = p16 >> 3, p8 = lane & 7, rr = lane >> 3;
    const uint32_t voA = static_cast<uint32_t>((rh * a.lda + 8 * p32) * 2);
    const uint32_t voX = static_cast<uint32_t>((rq * a.r + 8 * p16) * 2);
    const uint32_t voP = static_cast<uint32_t>((rr * a.r + 8 * p8) * 2);
    const uint32_t pairA = static_cast<uint32_t>(2 * a.lda * 2), quadX = static_cast<uint32_t>(4 * a.r * 2);
    const uint32_t halfP = static_cast<uint32_t>(8 * a.r * 2);

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

    // Staging registers: A for four stages, X^T for two, each loaded two
    // stages before it is staged.
    u32x4f ar[AQ], xr[PRODUCTS ? XQ : 1];
    // the loading tile's blocks of A: base and bytes inside the block
    const uint16_t* abase[AB];
    uint32_t abytes[AB];
    int64_t cur_tile = -1;
    auto set_tile = [&](int64_t tile) __attribute__((always_inline)) {
        const int64_t t0 = tile * 16;
#pragma unroll
        for (int i = 0; i < AB; ++i) {
            const int64_t j = AB * w + i;
            int64_t rows = min<int64_t>(a.qb, a.q - j * a.qb) - t0;
            rows = rows > 16 ? 16 : rows;
            abase[i] = a.A + (j * a.qb + t0) * a.lda;
            // the tile's rows inside A, up to the last row's r-th column
            abytes[i] = static_cast<uint32_t>(rows > 0 ? ((rows - 1) * a.lda + a.r) * 2 : 0);
        }
        cur_tile = tile;
    };
    const __amdgpu_buffer_rsrc_t rsX = raw_buffer(a.xt, static_cast<uint32_t>(PRODUCTS ? 64 * a.r * 2 : 0));
    // (tile, stage) of a unit, advanced four units at a time (no division in the loop)
    const int nst = static_cast<int>(a.stages);
    struct Cursor {
        int tile, s;
    };
    auto advance4 = [&](Cursor& c) __attribute__((always_inline)) {
        c.s += 4;
        if (c.s >= nst) {
            c.s = 0;
            ++c.tile;
        }
    };
    // A for stages cu.s .. cu.s + 3
    auto load_a = [&](const Cursor& cu) __attribute__((always_inline)) {
        const int64_t tile = cu.tile;
        if (tile != cur_tile) set_tile(tile);
        const uint32_t sk = static_cast<uint32_t>(cu.s) * kStage * 2;
#pragma unroll
        for (int i = 0; i < AQ; ++i)
            ar[i] = __builtin_bit_cast(u32x4f, __builtin_amdgcn_raw_buffer_load_b128(
                                                   raw_buffer(abase[i >> 3], abytes[i >> 3]), voA,
                                                   sk + (i & 7) * pairA, 0));
    };
    // X^T for stages s, s + 1
    auto load_x = [&](int s) __attribute__((always_inline)) {
        if constexpr (PRODUCTS) {
            const uint32_t sk = static_cast<uint32_t>(s) * kStage * 2;
#pragma unroll
            for (int i = 0; i < XQ; ++i)
                xr[i] = __builtin_bit_cast(u32x4f, __builtin_amdgcn_raw_buffer_load_b128(
                                                       rsX, voX, sk + (XQ * w + i) * quadX, 0));
        }
    };

    const int64_t slots = (a.stages + 3) / 4 * 4;      // stage slots per tile, a multiple of four
    Cursor cc{static_cast<int>(u0 / slots), static_cast<int>(u0 % slots)};   // the four stages being computed
    Cursor cl = cc;                              // the four stages being loaded
    // body b computes stage b of the four (tile cc.tile, stages cc.s .. cc.s + 3)
    auto body = [&](int b, int64_t u) __attribute__((always_inline)) {
        const int64_t tile = cc.tile;
        const int64_t s = cc.s + b;
        const int64_t t0 = tile * 16;
        const bool masked = tile >= a.clean_tiles;
        const int lb = b & 1;                    // LDS buffer of this stage
        // the previous stage's products have finished with the LDS tiles
        __syncthreads();
        if (b == 0 || b == 2) {
            // stage stages b, b + 1 into LDS from the lanes that hold them
            // (padding rows were read as zeros), then start the next loads:
            // X^T for stages b + 2, b + 3 and, after the second half, A for
            // the next four stages
            if ((qs >> 1) == (b >> 1)) {
#pragma unroll
                for (int i = 0; i < AQ; ++i)
                    sA[qs & 1][(AB * w + (i >> 3)) * 128 + swz(2 * (i & 7) + rh, p8)] = ar[i];
            }
            if constexpr (PRODUCTS) {
#pragma unroll
                for (int i = 0; i < XQ; ++i) sX[hs][swz(4 * (XQ * w + i) + rq, p8)] = xr[i];
            }
            if (b == 2) {
                if (u + 2 < u1) advance4(cl);    // else the last four stages are loaded again
                load_a(cl);
                load_x(cl.s);
            } else {
                load_x(cl.s + 2);
            }
            __syncthreads();
        }
        const bool live = s < a.stages;          // false for the empty stages of the last group

        if (live) {
            // encode: column groups g of this wave; lane (li, lk) reads blocks 8 lk .. 8 lk + 7
#pragma unroll
            for (int sl = 0; sl < SL; ++sl) {
                const int g = w * SL + sl;
                // two halves of four columns: column e of the group is blocks
                // 8 lk .. 8 lk + 7 of row li, packed in pairs; each half reads
                // the 8 bytes of its four columns from the 8 blocks
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) {
                    u32x2f R[8];
#pragma unroll
                    for (int bb = 0; bb < 8; ++bb) {
                        const int j = 8 * lk + bb;
                        R[bb] = j < K ? reinterpret_cast<const u32x2f*>(&sA[lb][j * 128 + swz(li, g)])[hf]
                                      : u32x2f{0u, 0u};
                    }
                    f32x4f C[4];
#pragma unroll
                    for (int ee = 0; ee < 4; ++ee) {
                        const int e = 4 * hf + ee;
                        u32x4f tv;
                        const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
                        for (int d = 0; d < 4; ++d)
                            tv[d] = __builtin_amdgcn_perm(R[2 * d + 1][(e >> 1) & 1], R[2 * d][(e >> 1) & 1], sel);
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
        }
        __syncthreads();

        // parity planes to HBM: 8 threads per 128-byte row piece set; rows
        // past the block's end fall outside the tile's buffer and are dropped
        const uint32_t sk = static_cast<uint32_t>(s) * kStage * 2;
        const int64_t prows = a.qb - t0;
        const uint32_t pbytes = live ? static_cast<uint32_t>((prows > 16 ? 16 : prows) * a.r * 2) : 0u;
#pragma unroll
        for (int i = 0; i < PB; ++i) {
            const int pl = PB * w + i;
            const int pln = pl / NPAR, p = pl % NPAR;
            const __amdgpu_buffer_rsrc_t rp = raw_buffer(a.parity + pln * plane + (p * a.qb + t0) * a.r, pbytes);
#pragma unroll
            for (int h = 0; h < 2; ++h)
                __builtin_amdgcn_raw_buffer_store_b128(sP[pl * 128 + swz(8 * h + rr, p8)], rp, voP, sk + h * halfP,
                                                       kAuxNonTemporal);
        }

        if constexpr (PRODUCTS) {
            if (live) {
                bf16x8f bx[2][4];
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        bx[ks][c] = __builtin_bit_cast(bf16x8f, sX[lb][swz(16 * c + li, 4 * ks + lk)]);
#pragma unroll
                for (int jj = 0; jj < KW; ++jj) {
                    const int j = w * KW + jj;
#pragma unroll
                    for (int ks = 0; ks < 2; ++ks) {
                        const bf16x8f af = __builtin_bit_cast(bf16x8f, sA[lb][j * 128 + swz(li, 4 * ks + lk)]);
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
        }
    };

    // The first loads are followed by as many stores as two stages write,
    // here into an empty buffer (the range check drops them): the queue of
    // memory operations entering the loop then has the shape it has after
    // every pass, and the wait before each staging covers only its loads.
    load_a(cl);
    load_x(cl.s);
    {
        const __amdgpu_buffer_rsrc_t none = raw_buffer(a.parity, 0);
        // distinct offsets, so that none of them is merged away as a repeated store
#pragma unroll
        for (int i = 0; i < 4 * PB; ++i)
            __builtin_amdgcn_raw_buffer_store_b128(u32x4f{0u, 0u, 0u, 0u}, none, 16u * i, 0u, 0);
    }
    for (int64_t u = u0; u < u1; u += 4) {
        body(0, u);
        body(1, u + 1);
        body(2, u + 2);
        body(3, u + 3);
        advance4(cc);
    }
}

__global__ void zero_f32_kernel(float* p, int64_t n) {
    const int64_t i = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 4;
    if (i + 4 <= n)
        *reinterpret_cast<f32x4f*>(p + i) = f32x4f{0.f, 0.f, 0.f, 0.f};
    else
        for (int64_t j = i; j < n; ++j) p[j] = 0.0f;
}

// What the single pass with products needs before it starts, in one launch:
// X (r x s bf16, row stride ldx) transposed into XT (s x r) by the first
// `ttiles` workgroups, 64 x 64 tiles through LDS, and Y (ny floats) zeroed by
// the others, 16384 floats each with 16-byte stores.  With vec (s = 64, r a
// multiple of 64, X 16-byte aligned, ldx a multiple of 8) the tiles move in
// 16-byte pieces; otherwise element by element.
__global__ __launch_bounds__(256) void fused_prep_kernel(const uint16_t* __restrict__ X, int64_t r, int64_t s,
                                                         int64_t ldx, uint16_t* __restrict__ XT, int64_t tiles_s,
                                                         int64_t ttiles, float* __restrict__ Y, int64_t ny, int vec) {
    __shared__ uint16_t tile[64][72];            // rows of 144 bytes: 16-byte aligned pieces
    const int64_t bid = blockIdx.x;
    if (bid < ttiles) {
        const int64_t tr = bid / tiles_s, ts = bid % tiles_s;
        if (vec) {
            // 64 rows x 8 pieces of X in, 64 rows x 8 pieces of X^T out: two of each per thread
            for (int p = threadIdx.x; p < 512; p += 256) {
                const int i = p >> 3, j = p & 7;
                *reinterpret_cast<uint4*>(&tile[i][8 * j]) =
                    *reinterpret_cast<const uint4*>(X + (tr * 64 + i) * ldx + 8 * j);
            }
            __syncthreads();
            for (int p = threadIdx.x; p < 512; p += 256) {
                const int c = p >> 3, j = p & 7;
                uint32_t w[4];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    w[u] = static_cast<uint32_t>(tile[8 * j + 2 * u][c]) |
                           (static_cast<uint32_t>(tile[8 * j + 2 * u + 1][c]) << 16);
                *reinterpret_cast<uint4*>(XT + c * r + tr * 64 + 8 * j) = uint4{w[0], w[1], w[2], w[3]};
            }
            return;
        }
        const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
        for (int i = ty; i < 64; i += 4) {
            const int64_t k = tr * 64 + i, c = ts * 64 + tx;
            tile[i][tx] = (k < r && c < s) ? X[k * ldx + c] : static_cast<uint16_t>(0);
        }
        __syncthreads();
        for (int i = ty; i < 64; i += 4) {
            const int64_t c = ts * 64 + i, k = tr * 64 + tx;
            if (c < s && k < r) XT[c * r + k] = tile[tx][i];
        }
        return;
    }
    const int64_t base = (bid - ttiles) * 16384 + threadIdx.x * 4;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
        const int64_t i = base + u * 1024;
        if (i + 4 <= ny)
            *reinterpret_cast<f32x4f*>(Y + i) = f32x4f{0.f, 0.f, 0.f, 0.f};
        else
            for (int64_t j = i; j < ny; ++j) Y[j] = 0.0f;
    }
}

// Eight wavefronts per workgroup (two per SIMD): each owns three systematic
// blocks and one parity row of the products and one 8-column group of the
// encode.
constexpr int kWaves = 8;

hipError_t launch_single_pass(FusedArgs a, bool products, int compute_units, hipStream_t st) {
    const int64_t tiles = ceil_div(a.qb, 16);
    a.stages = a.r / kStage;
    const int64_t slots = (a.stages + 3) / 4 * 4;           // stage slots per tile, a multiple of four
    a.units = tiles * slots;
    const int64_t groups = std::max<int64_t>(1, std::min<int64_t>(compute_units, tiles));
    a.per = std::max(ceil_div(a.units, groups), slots);     // a tile is shared by at most two workgroups
    a.per = (a.per + 3) / 4 * 4;                             // whole groups of four stages
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

}  // namespace

bool fused_bf16_supported(int n, int k, int planes, int64_t r, int64_t lda) {
    // a 64-row buffer of X^T and a 16-row tile of A must stay below 2^31 bytes
    return planes == 2 && k == 24 && n - k == 8 && r > 0 && r % kStage == 0 && lda % 8 == 0 && r < (1 << 23) &&
           lda < (1 << 25);
}

hipError_t launch_fused_bf16(FusedArgs a, bool products, int compute_units, hipStream_t st) {
    if (a.qb == 0 || a.r == 0) return hipSuccess;
    if (products) {
        const int64_t ny = static_cast<int64_t>(a.n) * a.qb * 64;
        hipLaunchKernelGGL(zero_f32_kernel, dim3(static_cast<unsigned>(ceil_div(ny, 4 * 256))), dim3(256), 0, st, a.Y,
                           ny);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return launch_single_pass(a, products, compute_units, st);
}

hipError_t launch_fused_bf16_from_x(FusedArgs a, const uint16_t* X, int64_t s, int64_t ldx, int compute_units,
                                    hipStream_t st) {
    if (a.qb == 0 || a.r == 0) return hipSuccess;
    const int64_t tiles_s = ceil_div(s, 64), ttiles = ceil_div(a.r, 64) * tiles_s;
    const int64_t ny = static_cast<int64_t>(a.n) * a.qb * 64;
    const int64_t blocks = ttiles + ceil_div(ny, 16384);
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    const int vec = s == 64 && a.r % 64 == 0 && ldx % 8 == 0 && (reinterpret_cast<uintptr_t>(X) & 15u) == 0 &&
                    (reinterpret_cast<uintptr_t>(a.xt) & 15u) == 0;
    hipLaunchKernelGGL(fused_prep_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, X, a.r, s, ldx,
                       const_cast<uint16_t*>(a.xt), tiles_s, ttiles, a.Y, ny, vec);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_single_pass(a, true, compute_units, st);
}

}  // namespace coded
