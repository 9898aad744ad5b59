// Multi-column fp32 worker products Y_i = A'_i X on the fp64 matrix cores
// (Sec. III-A: each worker multiplies its stored coded block by the multicast
// input; here X has s > 1 columns).
//
// Products of two fp32 values are exact in fp64, so the blocks and X are
// widened to fp64 and the sums run on v_mfma_f64_*: every element of A and of
// the parity planes is read from HBM once for all the columns of a launch.
//
// Tiles.  A workgroup of 256 threads owns 16 * RT row slots of one worker and
// up to 16 * NCT (or 4 * NCT) columns of X.  For a systematic worker, or a
// parity worker with one plane, slot rho is block row t0 + rho.  For a parity
// worker with two planes, slot rho is row t0 + rho % (8 RT) of plane
// rho / (8 RT): the hi and lo rows of a block row sit in one tile and their
// results are added at the end, so every workgroup streams the same bytes
// (two-plane rows as longer K loops would leave the parity workgroups running
// alone at the end of the launch).
//
// K loop.  K is walked in chunks of KC.  A chunk's slot rows are loaded with
// 16-byte loads (KC/4 consecutive threads cover one row's KC contiguous
// elements) into a ring of PF register sets, so PF chunks are in flight; the
// chunk is then stored to a double-buffered LDS tile with 16-byte row padding
// (conflict-free 16-byte reads down a column of rows), X's KC x SP slice is
// stored transposed and widened to fp64, one barrier, and the load of chunk
// c + PF is issued before the chunk is multiplied.  Every chunk, the last one
// with a K tail included, runs the same straight-line loads (positions past
// r read a clamped address and are zeroed at the LDS store, and prefetches
// past the last chunk read one fixed line), so each step waits for exactly
// one chunk.  Rows past the block read a clamped row; padding rows (past q)
// are written as zero in the epilogue.
//
// With buffer addressing (BUF, used when every offset fits in 31 bits) each
// load is one per-thread offset, fixed for the whole K loop, from one base per
// operand, plus the chunk's byte offset in a scalar register: no vector
// instruction is spent on addresses, and the prefetches past the last chunk
// get an offset beyond the buffer's size, which the hardware answers with
// zeros and no memory access.  Vector instructions do not overlap with the
// fp64 matrix instructions on a SIMD, so every one removed from the K loop
// shortens it.
//
// The four waves take quarters of each chunk's K range and keep partial sums
// of the whole tile; the partials are added through LDS in a fixed order.
//
// Matrix-core shapes.  v_mfma_f64_16x16x4f64 (16 rows x 16 columns x 4 k)
// for s > 8; for s <= 8 v_mfma_f64_4x4x4f64, four 4 x 4 x 4 products per
// instruction, used as 16 rows x 4 columns sharing one B operand, so no
// matrix-core work is spent on absent columns.  Lane layouts (checked on the
// device): A lane l = A[l % 16][l / 16] for both; B lane l = B[l / 16][l % 16]
// (16x16x4) or B[l / 16][l % 4] (4x4x4, replicated over the four products);
// results: item v of lane l = C[4v + l/16][l % 16] (16x16x4), or lane l =
// C[4((l % 16) / 4) + l / 16][l % 4] (4x4x4).  The k index a lane supplies
// is free as long as A and B agree, so lane group g = l/16 takes the four
// consecutive k of one 16-byte LDS read, one per instruction.
#include "internal.h"
#include "worker_common.h"

namespace coded {
namespace {

typedef float f32x4m __attribute__((ext_vector_type(4)));
typedef double f64x4m __attribute__((ext_vector_type(4)));

constexpr int kMmThreads = 256;

template <int RT, int NCT, bool NARROW, int KC>
struct MmCfg {
    static constexpr int kRows = 16 * RT;                     // row slots per workgroup
    static constexpr int kTileCols = NARROW ? 4 : 16;         // columns per matrix-core tile
    static constexpr int kSP = kTileCols * NCT;               // columns per launch
    static constexpr int kStride = KC + 4;                    // floats per A row in LDS (16-byte pad)
    static constexpr int kXStride = KC + 2;                   // doubles per X^T row in LDS (16-byte pad)
    static constexpr int kABytes = 2 * kRows * kStride * 4;   // double-buffered A tile
    static constexpr int kXBytes = 2 * kSP * kXStride * 8;    // double-buffered X^T slice (fp64)
    static constexpr int kRedCols = kSP < 16 ? kSP : 16;      // columns per reduction pass
    static constexpr int kRedBytes = 4 * kRows * kRedCols * 8;
    static constexpr int kLds = (kABytes + kXBytes) > kRedBytes ? (kABytes + kXBytes) : kRedBytes;
    static constexpr int kALoads = kRows * KC / 4 / kMmThreads;  // 16-byte A loads per thread and chunk
    static constexpr int kXLoads = kSP * KC / kMmThreads;        // X elements per thread and chunk
    static constexpr int kKW = KC / 4;                           // k per wave and chunk
    static_assert(kRows * KC / 4 % kMmThreads == 0, "A tile must split evenly over the threads");
    static_assert(kSP * KC % kMmThreads == 0, "X slice must split evenly over the threads");
    static_assert(kKW % 16 == 0, "each wave takes whole groups of 16 k");
    static_assert(kLds <= 64 * 1024, "LDS budget");
};

__device__ inline f32x4m load_stream4(const float* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4m*>(p));
}

// Raw buffer resource over `bytes` bytes from `base` (no stride, no format:
// the gfx9 dword-3 value); loads at offsets >= bytes return zeros.
__device__ inline __amdgpu_buffer_rsrc_t raw_buffer(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0), static_cast<int>(bytes),
                                             0x00020000);
}
constexpr int kAuxNonTemporal = 2;   // cache-policy bits of the load: nt

template <int RT, int NCT, bool NARROW, int KC, int PF, bool BUF>
__global__ __launch_bounds__(kMmThreads) void gemm_f32_mfma_kernel(WorkerArgs a, int64_t stiles, int64_t ptiles,
                                                                   int64_t c0) {
    using C = MmCfg<RT, NCT, NARROW, KC>;
    __shared__ __attribute__((aligned(16))) char smem[C::kLds];
    float* As = reinterpret_cast<float*>(smem);                // [2][kRows][kStride]
    double* Xs = reinterpret_cast<double*>(smem + C::kABytes);  // [2][kSP][kXStride]
    double* Red = reinterpret_cast<double*>(smem);              // [4][kRows][kRedCols], after the K loop

    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);

    // Tile -> (worker, first block row); parity tiles first.
    const int64_t g = blockIdx.x;
    int worker;
    int64_t tile;
    bool parity;
    if (g < ptiles * a.n_par) {
        worker = a.par_ids[g / ptiles];
        tile = g % ptiles;
        parity = true;
    } else {
        const int64_t g2 = g - ptiles * a.n_par;
        if (g2 >= stiles * a.n_sys) return;
        worker = a.sys_ids[g2 / stiles];
        tile = g2 % stiles;
        parity = false;
    }
    const int hrows = (parity && a.planes == 2) ? C::kRows / 2 : C::kRows;   // block rows of the tile
    const int64_t t0 = tile * hrows;
    const int64_t plane_elems = static_cast<int64_t>(a.n - a.k) * a.qb * a.r;
    const int r = static_cast<int>(a.r);
    const int nch = (r + KC - 1) / KC;

    // Row start of each slot this thread loads (a real row in every case).
    auto slot_row = [&](int rho) -> const float* {
        int64_t t = t0 + rho % hrows;
        t = t < a.qb ? t : a.qb - 1;
        if (parity)
            return static_cast<const float*>(a.parity) + (rho / hrows) * plane_elems +
                   (static_cast<int64_t>(worker - a.k) * a.qb + t) * a.r;
        int64_t row = static_cast<int64_t>(worker) * a.qb + t;
        row = row < a.q ? row : a.q - 1;
        return static_cast<const float*>(a.A) + row * a.lda;
    };
    const float* gp[C::kALoads];
    int ofs_a[C::kALoads], acol[C::kALoads];
#pragma unroll
    for (int p = 0; p < C::kALoads; ++p) {
        const int f = tid + kMmThreads * p;
        const int rho = f / (KC / 4);
        acol[p] = (f % (KC / 4)) * 4;
        ofs_a[p] = rho * C::kStride + acol[p];
        gp[p] = slot_row(rho);
    }
    const float* dummy = slot_row(0);   // one line every past-the-end prefetch reads
    const float* X = static_cast<const float*>(a.X);
    const float* gx[C::kXLoads];
    int ofs_x[C::kXLoads], xk[C::kXLoads];
    uint32_t xoff[C::kXLoads];
#pragma unroll
    for (int i = 0; i < C::kXLoads; ++i) {
        const int e = tid + kMmThreads * i;
        const int kk = e / C::kSP, cc = e % C::kSP;
        xk[i] = kk;
        ofs_x[i] = cc * C::kXStride + kk;
        const int64_t col = c0 + cc < a.s ? c0 + cc : a.s - 1;   // absent columns read a real one, never stored
        gx[i] = X + col;
        xoff[i] = static_cast<uint32_t>((static_cast<int64_t>(kk) * a.ldx + col) * 4);
    }

    // Buffer addressing: the operands' buffers and this thread's byte offsets
    // (a systematic block's rows past q read as zeros; padding rows are
    // stored as zeros in the epilogue).
    const float* abase;
    int64_t rows_in, rstride;
    uint32_t abytes;
    if (parity) {
        abase = static_cast<const float*>(a.parity) + static_cast<int64_t>(worker - a.k) * a.qb * a.r;
        rows_in = a.qb;
        rstride = a.r;
        abytes = static_cast<uint32_t>(((a.planes == 2 ? plane_elems : 0) + a.qb * a.r) * 4);
    } else {
        abase = static_cast<const float*>(a.A) + static_cast<int64_t>(worker) * a.qb * a.lda;
        rows_in = a.q - static_cast<int64_t>(worker) * a.qb;
        rows_in = rows_in < a.qb ? rows_in : a.qb;
        rstride = a.lda;
        // the block's rows inside A, up to the last row's r-th column
        abytes = static_cast<uint32_t>(rows_in > 0 ? ((rows_in - 1) * a.lda + a.r) * 4 : 0);
    }
    uint32_t aoff[C::kALoads];
#pragma unroll
    for (int p = 0; p < C::kALoads; ++p) {
        const int rho = (tid + kMmThreads * p) / (KC / 4);
        int64_t t = t0 + rho % hrows;
        t = t < rows_in ? t : rows_in - 1;
        t = t > 0 ? t : 0;
        aoff[p] = static_cast<uint32_t>(((parity ? (rho / hrows) * plane_elems : 0) + t * rstride + acol[p]) * 4);
    }
    const uint32_t xbytes = static_cast<uint32_t>(a.r * a.ldx * 4);
    const __amdgpu_buffer_rsrc_t rsA = raw_buffer(abase, abytes);
    const __amdgpu_buffer_rsrc_t rsX = raw_buffer(X, xbytes);

    auto load_chunk = [&](int c, f32x4m* R, float* XR) {
        const bool live = c < nch;
        if constexpr (BUF) {
            // scalar chunk offsets; past the last chunk, offsets beyond the buffers
            const uint32_t sa = live ? static_cast<uint32_t>(c) * KC * 4 : abytes;
            const uint32_t sx = live ? static_cast<uint32_t>(c) * KC * static_cast<uint32_t>(a.ldx) * 4 : xbytes;
#pragma unroll
            for (int p = 0; p < C::kALoads; ++p)
                R[p] = __builtin_bit_cast(f32x4m, __builtin_amdgcn_raw_buffer_load_b128(rsA, aoff[p], sa, kAuxNonTemporal));
#pragma unroll
            for (int i = 0; i < C::kXLoads; ++i)
                XR[i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsX, xoff[i], sx, 0));
            return;
        }
#pragma unroll
        for (int p = 0; p < C::kALoads; ++p) {
            int kk = c * KC + acol[p];
            kk = kk < r ? kk : r - 4;
            R[p] = load_stream4(live ? gp[p] + kk : dummy);
        }
#pragma unroll
        for (int i = 0; i < C::kXLoads; ++i) {
            int kk = c * KC + xk[i];
            kk = kk < r ? kk : r - 1;
            XR[i] = gx[i][live ? static_cast<int64_t>(kk) * a.ldx : 0];
        }
    };
    // kvalid: K positions of the chunk below r; the rest are stored as zeros.
    auto store_chunk = [&](int buf, int kvalid, const f32x4m* R, const float* XR) {
        float* Ab = As + buf * C::kRows * C::kStride;
        double* Xb = Xs + buf * C::kSP * C::kXStride;
        if (BUF && kvalid >= KC) {     // a whole chunk: nothing to zero
#pragma unroll
            for (int p = 0; p < C::kALoads; ++p) *reinterpret_cast<f32x4m*>(Ab + ofs_a[p]) = R[p];
#pragma unroll
            for (int i = 0; i < C::kXLoads; ++i) Xb[ofs_x[i]] = static_cast<double>(XR[i]);
            return;
        }
#pragma unroll
        for (int p = 0; p < C::kALoads; ++p)
            *reinterpret_cast<f32x4m*>(Ab + ofs_a[p]) = acol[p] < kvalid ? R[p] : f32x4m{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < C::kXLoads; ++i) Xb[ofs_x[i]] = xk[i] < kvalid ? static_cast<double>(XR[i]) : 0.0;
    };

    const int r16 = lane & 15, g4 = lane >> 4;
    const int xc = NARROW ? (lane & 3) : (lane & 15);
    double accn[RT][NCT];
    f64x4m accw[RT][NCT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
            accn[rt][ct] = 0.0;
            accw[rt][ct] = f64x4m{0.0, 0.0, 0.0, 0.0};
        }
    auto multiply = [&](int buf) {
        const float* Ab = As + buf * C::kRows * C::kStride;
        const double* Xb = Xs + buf * C::kSP * C::kXStride;
#pragma unroll
        for (int jj = 0; jj < C::kKW / 16; ++jj) {
            const int koff = wv * C::kKW + jj * 16 + 4 * g4;
            f32x4m af[RT];
            f64x4m xf[NCT];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                af[rt] = *reinterpret_cast<const f32x4m*>(Ab + (rt * 16 + r16) * C::kStride + koff);
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                const double* xp = Xb + (ct * C::kTileCols + xc) * C::kXStride + koff;
                const double2 lo = *reinterpret_cast<const double2*>(xp);
                const double2 hi = *reinterpret_cast<const double2*>(xp + 2);
                xf[ct] = f64x4m{lo.x, lo.y, hi.x, hi.y};
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                double ad[RT];
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) ad[rt] = static_cast<double>(af[rt][e]);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) {
                        if constexpr (NARROW)
                            accn[rt][ct] = __builtin_amdgcn_mfma_f64_4x4x4f64(ad[rt], xf[ct][e], accn[rt][ct], 0, 0, 0);
                        else
                            accw[rt][ct] = __builtin_amdgcn_mfma_f64_16x16x4f64(ad[rt], xf[ct][e], accw[rt][ct], 0, 0, 0);
                    }
            }
        }
    };

    f32x4m aring[PF][C::kALoads];
    float xring[PF][C::kXLoads];
    if (nch > 0) {
#pragma unroll
        for (int j = 0; j < PF; ++j) load_chunk(j, aring[j], xring[j]);
    }
    for (int cb = 0; cb < nch; cb += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int c = cb + j;
            if (c >= nch) break;
            const int buf = c & 1;
            store_chunk(buf, r - c * KC, aring[j], xring[j]);
            __syncthreads();
            load_chunk(c + PF, aring[j], xring[j]);
            multiply(buf);
        }
    }

    // Add the four waves' partial sums (wave 0, 1, 2, 3 in that order) and,
    // for a two-plane parity tile, the lo rows to the hi rows, kRedCols
    // columns per pass; padding rows of a systematic block are stored as 0.
    constexpr int kPasses = C::kSP / C::kRedCols;
    const int w = C::kRows * C::kRedCols;
#pragma unroll
    for (int pass = 0; pass < kPasses; ++pass) {
        __syncthreads();   // every wave is done with the tiles (or with the last pass)
        double* Rw = Red + wv * w;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            if constexpr (NARROW) {
                const int row = rt * 16 + 4 * (r16 >> 2) + g4;
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) Rw[row * C::kRedCols + ct * 4 + (lane & 3)] = accn[rt][ct];
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v) Rw[(rt * 16 + 4 * v + g4) * C::kRedCols + r16] = accw[rt][pass][v];
            }
        }
        __syncthreads();
        for (int idx = tid; idx < hrows * C::kRedCols; idx += kMmThreads) {
            const int row = idx / C::kRedCols, col = idx % C::kRedCols;
            const int64_t t = t0 + row, cc = c0 + pass * C::kRedCols + col;
            if (t >= a.qb || cc >= a.s) continue;
            const int o = row * C::kRedCols + col;
            double v = ((Red[o] + Red[w + o]) + Red[2 * w + o]) + Red[3 * w + o];
            if (hrows != C::kRows) {
                const int o2 = o + hrows * C::kRedCols;
                v += ((Red[o2] + Red[w + o2]) + Red[2 * w + o2]) + Red[3 * w + o2];
            }
            if (!parity && static_cast<int64_t>(worker) * a.qb + t >= a.q) v = 0.0;
            store_y(a, worker, t, cc, v);
        }
    }
}

// Buffer addressing needs every byte offset (and the past-the-end offsets,
// which equal a buffer's size) below 2^31.
bool buffer_offsets_fit(const WorkerArgs& a) {
    const int64_t lim = (int64_t(1) << 31) - 1;
    const int64_t sys = a.qb * a.lda * 4;
    const int64_t par = ((a.planes == 2 ? static_cast<int64_t>(a.n - a.k) * a.qb * a.r : 0) + a.qb * a.r) * 4;
    const int64_t x = a.r * a.ldx * 4 + a.s * 4;
    return sys < lim && par < lim && x < lim;
}

template <int RT, int NCT, bool NARROW, int KC, int PF>
hipError_t launch_mm(const WorkerArgs& a, int64_t c0, hipStream_t st) {
    using C = MmCfg<RT, NCT, NARROW, KC>;
    const int64_t stiles = ceil_div(a.qb, C::kRows);
    const int64_t ptiles = a.planes == 2 ? ceil_div(a.qb, C::kRows / 2) : stiles;
    const int64_t blocks = stiles * a.n_sys + ptiles * a.n_par;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    if (buffer_offsets_fit(a))
        hipLaunchKernelGGL((gemm_f32_mfma_kernel<RT, NCT, NARROW, KC, PF, true>), dim3(static_cast<unsigned>(blocks)),
                           dim3(kMmThreads), 0, st, a, stiles, ptiles, c0);
    else
        hipLaunchKernelGGL((gemm_f32_mfma_kernel<RT, NCT, NARROW, KC, PF, false>),
                           dim3(static_cast<unsigned>(blocks)), dim3(kMmThreads), 0, st, a, stiles, ptiles, c0);
    return hipGetLastError();
}

}  // namespace

bool gemm_f32_mfma_supported(const WorkerArgs& a) {
    // K positions are 32-bit inside the kernel; rows need 16-byte alignment;
    // planes are fp32 (a bfloat16 lo plane takes the general kernel).
    return a.s > 1 && !a.lo_bf16 && a.r > 0 && a.r % 4 == 0 && a.r <= (1ll << 30) && a.lda % 4 == 0 &&
           (reinterpret_cast<uintptr_t>(a.A) & 15u) == 0 && (reinterpret_cast<uintptr_t>(a.parity) & 15u) == 0;
}

// Up to 8 columns: 4-column tiles, one launch.  More: 16-column tiles in
// launches of at most 32 columns (two 32-column launches measured faster
// than one 64-column launch at s = 64: the wider tile halves occupancy).
hipError_t launch_gemm_f32_mfma(const WorkerArgs& a, hipStream_t st) {
    if (a.s <= 4) return launch_mm<1, 1, true, 128, 4>(a, 0, st);
    if (a.s <= 8) return launch_mm<1, 2, true, 128, 2>(a, 0, st);
    for (int64_t c0 = 0; c0 < a.s; c0 += 32) {
        const hipError_t e = a.s - c0 <= 16 ? launch_mm<2, 1, false, 64, 2>(a, c0, st)
                                            : launch_mm<2, 2, false, 64, 2>(a, c0, st);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace coded
