// One launch for the whole coded product of a small fp32 problem with one
// column (Sec. III-A: encode, the n worker products, dec(indices, results)).
//
// Every step works along block rows: parity row t is sum_j P[p][j] A_j[t],
// worker i's result at t is its row t times x, and the decoded outputs at t
// need only the survivors' results at t.  So one workgroup per block row t
// reads row t of the k data blocks once, forms the parity rows (writing both
// planes, or reads the stored planes), computes all n products into Y, and
// decodes the k outputs of that row: systematic survivors are copied, the
// missing blocks are sum_c D[b][c] Y_{S[c]}[t] with the decoding matrix D
// eliminated by wave 0 while the other waves stream.  For a problem of a
// few MB this replaces three launch latencies with one.
//
// The parity arithmetic is the encode kernel's, element for element (fp64
// fma chain over j in order, hi = round(sum), lo = round(sum - hi)), so the
// stored planes equal coded_encode's bit for bit.  Products are exact in
// fp64 and summed in fp64.
#include "internal.h"
#include "onepass.h"
#include "decode_common.h"
#include "worker_common.h"

namespace coded {
namespace {

typedef float f32x4o __attribute__((ext_vector_type(4)));

__device__ inline f32x4o load4(const float* p) { return *reinterpret_cast<const f32x4o*>(p); }

// Pointers into device (global) memory, so that loads through them stay
// global loads once the compiler can no longer trace them to an argument.
typedef __attribute__((address_space(1))) const float gfloat;
typedef __attribute__((address_space(1))) const f32x4o gf32x4o;
__device__ inline f32x4o load4(const gfloat* p) { return *reinterpret_cast<const gf32x4o*>(p); }

// Sum of v over the wavefront, in every lane: cross-lane moves within each
// 16-lane row (DPP: quad swaps, then half-row and row mirrors), then the
// four row sums read from lanes 0, 16, 32 and 48.  No LDS round trips.
template <int CTRL>
__device__ inline double dpp_f64(double v) {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
    const uint32_t lo = static_cast<uint32_t>(
        __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(u)), CTRL, 0xF, 0xF, false));
    const uint32_t hi = static_cast<uint32_t>(
        __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(u >> 32)), CTRL, 0xF, 0xF, false));
    return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}

__device__ inline double wave_total(double v) {
    v += dpp_f64<0xB1>(v);    // quad_perm [1,0,3,2]
    v += dpp_f64<0x4E>(v);    // quad_perm [2,3,0,1]
    v += dpp_f64<0x141>(v);   // row_half_mirror
    v += dpp_f64<0x140>(v);   // row_mirror: every lane holds its row's sum
    return ((lane_value(v, 0) + lane_value(v, 16)) + lane_value(v, 32)) + lane_value(v, 48);
}

// The set's bookkeeping, by one wave (the host has validated the set; k <= n
// <= 16, so lane j stands for block j).  The survivors form a bit mask; from
// it every entry is written by one lane without reading another's: the
// survivors in ascending order, presence, the missing systematic blocks in
// ascending order, and the rows of each block that lie inside A.  No
// workgroup barrier: the wave orders its own LDS writes before its
// elimination reads them, and the other waves read them after the barrier
// that precedes the decode.  Returns the number of missing blocks.
__device__ inline int setup_set_wave(const OnePassArgs& a, int lane, SetMeta& sm) {
    const int n = a.n, k = a.k;
    uint32_t mask = 0;
    for (int c = 0; c < k; ++c) mask |= 1u << set_entry(a.set, c);
    const uint32_t below = static_cast<uint32_t>((uint64_t{1} << lane) - 1u);   // blocks below this lane's
    const bool in = lane < 32 && ((mask >> lane) & 1u) != 0;
    if (lane < n) {
        sm.present[lane] = in ? 1 : 0;
        if (in) sm.S[__builtin_popcount(mask & below)] = lane;
    }
    if (lane < k) {
        if (!in) sm.miss[__builtin_popcount(~mask & below)] = lane;
        const int64_t lim = a.q - static_cast<int64_t>(lane) * a.qb;
        sm.lim[lane] = static_cast<int32_t>(lim < 0 ? 0 : (lim > a.qb ? a.qb : lim));
    }
    const int m = k - __builtin_popcount(mask & ((1u << k) - 1u));
    if (lane == 0) {
        sm.status = 0;
        sm.m = m;
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
    return m;
}

__device__ inline double lane_xor(double v, int lane, int mask) {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
    const int addr = (lane ^ mask) * 4;
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(addr, static_cast<int>(static_cast<uint32_t>(u))));
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(addr, static_cast<int>(static_cast<uint32_t>(u >> 32))));
    return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}

// Sums of four values v0..v3 over the wavefront at once: the first two
// exchanges (lanes 1 and 2 apart) halve the values a lane carries, so that
// lane l keeps value ((l & 1) << 1) | ((l >> 1) & 1) summed over its quad;
// rotations by 4 and 8 within each 16-lane row and exchanges 16 and 32 lanes
// apart then add the quads of the wavefront.  Lane l < 4 returns the total
// of that value.
__device__ inline double quad_class_total(double v0, double v1, double v2, double v3, int lane) {
    const bool b0 = (lane & 1) != 0, b1 = (lane & 2) != 0;
    // lanes 1 apart: keep values 2 b0 and 2 b0 + 1, send the other pair
    const double k0 = b0 ? v2 : v0, k1 = b0 ? v3 : v1;
    const double s0 = b0 ? v0 : v2, s1 = b0 ? v1 : v3;
    const double z0 = k0 + dpp_f64<0xB1>(s0), z1 = k1 + dpp_f64<0xB1>(s1);
    // lanes 2 apart: keep value 2 b0 + b1
    double w = (b1 ? z1 : z0) + dpp_f64<0x4E>(b1 ? z0 : z1);
    w += dpp_f64<0x124>(w);   // row_ror:4
    w += dpp_f64<0x128>(w);   // row_ror:8: every lane holds its row's sum of its value
    w += lane_xor(w, lane, 16);
    w += lane_xor(w, lane, 32);
    return w;
}

// The same for eight values v[0..7]: exchanges 1 and 2 lanes apart and a
// rotation by 4 halve them three times, so lane l keeps value
// ((l & 1) << 2) | (l & 2) | ((l >> 2) & 1) summed over its half-row; a
// rotation by 8 and permutes 16 and 32 lanes apart then add the rest.  Lane
// l < 8 returns the total of that value.
__device__ inline double octet_class_total(const double (&v)[8], int lane) {
    const bool b0 = (lane & 1) != 0, b1 = (lane & 2) != 0, b2 = (lane & 4) != 0;
    double z[4], w[2];
#pragma unroll
    for (int j = 0; j < 4; ++j) z[j] = (b0 ? v[j + 4] : v[j]) + dpp_f64<0xB1>(b0 ? v[j] : v[j + 4]);
#pragma unroll
    for (int j = 0; j < 2; ++j) w[j] = (b1 ? z[j + 2] : z[j]) + dpp_f64<0x4E>(b1 ? z[j] : z[j + 2]);
    double x = (b2 ? w[1] : w[0]) + dpp_f64<0x124>(b2 ? w[0] : w[1]);   // row_ror:4
    x += dpp_f64<0x128>(x);                                             // row_ror:8
    x += lane_xor(x, lane, 16);
    x += lane_xor(x, lane, 32);
    return x;
}

__device__ inline double dot4(f32x4o a, f32x4o x, double acc) {
    acc = fma(static_cast<double>(a.x), static_cast<double>(x.x), acc);
    acc = fma(static_cast<double>(a.y), static_cast<double>(x.y), acc);
    acc = fma(static_cast<double>(a.z), static_cast<double>(x.z), acc);
    acc = fma(static_cast<double>(a.w), static_cast<double>(x.w), acc);
    return acc;
}

// KM >= k: data rows held per thread (registers are sized by it).
template <int NT, int KM>
__global__ __launch_bounds__(NT) void onepass_f32_kernel(OnePassArgs a) {
    constexpr int NW = NT / 64;
    constexpr int MN = kOnePassMaxN;
    __shared__ SetMeta sm;
    __shared__ double sD[64 * kFastLd];
    __shared__ double red[NW][MN];
    __shared__ double sy[MN];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t t = blockIdx.x;
    // The arguments the first loads depend on, fetched in one batch before
    // anything else and then held in scalar registers (left alone, the
    // compiler fetches each inside the branch that first uses it, one
    // dependent round trip after another before the first load goes out).
    const gfloat* Ap = (const gfloat*)a.A;
    const gfloat* xp = (const gfloat*)a.x;
    int64_t q = a.q, qb = a.qb, r = a.r, lda = a.lda;
    int32_t n = a.n, k = a.k, missing = a.missing;
    asm volatile("" : "+s"(Ap), "+s"(xp), "+s"(q), "+s"(qb), "+s"(r), "+s"(lda), "+s"(n), "+s"(k), "+s"(missing));
    const int npar = n - k;
    int kin = 0;                                  // data blocks whose row t lies inside A
#pragma unroll
    for (int j = 0; j < KM; ++j) kin += (j < k && static_cast<int64_t>(j) * qb + t < q) ? 1 : 0;
    // With blocks to solve for, wave 0 forms D while the other waves stream
    // the columns (the two chains run side by side); otherwise all stream.
    const int cw = (missing > 0 && NW > 1) ? 1 : 0;

    // This thread's first columns are requested before anything else, so the
    // memory latency overlaps the set bookkeeping and the elimination.
    auto load_chunk = [&](int64_t c, f32x4o (&av)[KM], f32x4o& xv) __attribute__((always_inline)) {
        xv = load4(xp + c);
#pragma unroll
        for (int j = 0; j < KM; ++j) {
            av[j] = f32x4o{0.f, 0.f, 0.f, 0.f};
            if (j < kin) av[j] = load4(Ap + (static_cast<int64_t>(j) * qb + t) * lda + c);
        }
    };
    f32x4o avA[KM], avB[KM], xA, xB;
    const int64_t kStep = static_cast<int64_t>(NT - 64 * cw) * 4;
    int64_t c = wv < cw ? r : static_cast<int64_t>(tid - 64 * cw) * 4;
    if (c < r) load_chunk(c, avA, xA);

    // Wave 0 sets up the set and forms D (read by all after the barrier
    // below); the streaming waves go straight on to their columns.
    if (wv == 0) {
        const int m = setup_set_wave(a, lane, sm);
        if (m > 0) {
            DecodeArgs da{};
            da.G = a.G;
            da.info = a.info;
            da.q = q;
            da.qb = qb;
            da.s = 1;
            da.ldo = a.ldo;
            da.n = n;
            da.k = k;
            da.batch = 1;
            eliminate_set(da, sm, m, k - m, lane, sD);
        }
    }

    // Row t of the data blocks (zero past q), the parity rows, and the n products.
    double y[MN];
#pragma unroll
    for (int i = 0; i < MN; ++i) y[i] = 0.0;
    const int64_t plane = static_cast<int64_t>(npar) * qb * r;
    auto process = [&](int64_t c, const f32x4o (&av)[KM], f32x4o xv) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < KM; ++j)
            if (j < kin) y[j] = dot4(av[j], xv, y[j]);
        for (int p = 0; p < npar; ++p) {
            float* prow = a.parity + (static_cast<int64_t>(p) * qb + t) * r + c;
            const double* g = a.G + static_cast<int64_t>(k + p) * k;    // parity row p of G (uniform)
            f32x4o hi, lo = f32x4o{0.f, 0.f, 0.f, 0.f};
            if (a.encode) {
                double s4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
                for (int j = 0; j < KM; ++j) {
                    if (j < kin) {
                        const double gj = g[j];
                        s4[0] = fma(gj, static_cast<double>(av[j].x), s4[0]);
                        s4[1] = fma(gj, static_cast<double>(av[j].y), s4[1]);
                        s4[2] = fma(gj, static_cast<double>(av[j].z), s4[2]);
                        s4[3] = fma(gj, static_cast<double>(av[j].w), s4[3]);
                    }
                }
                hi = f32x4o{static_cast<float>(s4[0]), static_cast<float>(s4[1]), static_cast<float>(s4[2]),
                            static_cast<float>(s4[3])};
                *reinterpret_cast<f32x4o*>(prow) = hi;
                if (a.planes == 2) {
                    lo = f32x4o{static_cast<float>(s4[0] - static_cast<double>(hi.x)),
                                static_cast<float>(s4[1] - static_cast<double>(hi.y)),
                                static_cast<float>(s4[2] - static_cast<double>(hi.z)),
                                static_cast<float>(s4[3] - static_cast<double>(hi.w))};
                    *reinterpret_cast<f32x4o*>(prow + plane) = lo;
                }
            } else {
                hi = load4(prow);
                if (a.planes == 2) lo = load4(prow + plane);
            }
            // the worker multiplies its stored planes: hi, then lo
            double yp = dot4(hi, xv, 0.0);
            if (a.planes == 2) yp = dot4(lo, xv, yp);
#pragma unroll
            for (int i = 0; i < MN; ++i)
                if (i == k + p) y[i] += yp;
        }
    };
    // one chunk of loads in flight ahead of the chunk being combined
    while (c < r) {
        if (c + kStep < r) load_chunk(c + kStep, avB, xB);
        process(c, avA, xA);
        c += kStep;
        if (c >= r) break;
        if (c + kStep < r) load_chunk(c + kStep, avA, xA);
        process(c, avB, xB);
        c += kStep;
    }
    if (n <= 4) {
        // lane l < 4 holds the total of value ((l & 1) << 1) | ((l >> 1) & 1)
        const double v = quad_class_total(y[0], y[1], y[2], y[3], lane);
        const int i = ((lane & 1) << 1) | ((lane >> 1) & 1);
        if (lane < 4 && i < n) red[wv][i] = v;
    } else if (n <= 8) {
        // lane l < 8 holds the total of value ((l & 1) << 2) | (l & 2) | ((l >> 2) & 1)
        const double y8[8] = {y[0], y[1], y[2], y[3], y[4], y[5], y[6], y[7]};
        const double v = octet_class_total(y8, lane);
        const int i = ((lane & 1) << 2) | (lane & 2) | ((lane >> 2) & 1);
        if (lane < 8 && i < n) red[wv][i] = v;
    } else {
#pragma unroll
        for (int i = 0; i < MN; ++i) {
            if (i < n) {
                const double v = wave_total(y[i]);
                if (lane == 0) red[wv][i] = v;
            }
        }
    }
    __syncthreads();
    if (tid < n) {
        double v = 0.0;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += red[w][tid];
        sy[tid] = v;
        a.Y[static_cast<int64_t>(tid) * a.qb + t] = v;
    }
    __syncthreads();

    // Decode block row t (out is not written for a singular survivor system).
    const int status = sm.status;
    if (t == 0 && tid == 0) a.info[0] = status;
    if (status != 0 || tid >= k) return;
    const int j = tid;
    if (t >= sm.lim[j]) return;                  // padding row
    double v;
    if (sm.present[j]) {
        v = sy[j];
    } else {
        int b = 0;                               // rank of j among the missing blocks
        for (int i = 0; i < j; ++i) b += sm.present[i] ? 0 : 1;
        v = 0.0;
        for (int c2 = 0; c2 < k; ++c2) v = fma(sD[c2 * kFastLd + b], sy[sm.S[c2]], v);
    }
    a.out[(static_cast<int64_t>(j) * a.qb + t) * a.ldo] = static_cast<float>(v);
}

template <int NT>
void launch_nt(const OnePassArgs& a, dim3 grid, hipStream_t st) {
    if (a.k <= 4)
        hipLaunchKernelGGL((onepass_f32_kernel<NT, 4>), grid, dim3(NT), 0, st, a);
    else if (a.k <= 8)
        hipLaunchKernelGGL((onepass_f32_kernel<NT, 8>), grid, dim3(NT), 0, st, a);
    else
        hipLaunchKernelGGL((onepass_f32_kernel<NT, 16>), grid, dim3(NT), 0, st, a);
}

bool aligned16p(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

bool onepass_supported(int n, int k, int64_t q, int64_t r, int64_t lda, const void* A, const void* parity,
                       const void* x) {
    // Small problems only (up to 16 MB of A): there three launch latencies
    // dominate; larger ones stream better through the dedicated kernels.
    return n <= kOnePassMaxN && n > k && q > 0 && r >= 4 && r % 4 == 0 && lda % 4 == 0 && q * r <= (int64_t{1} << 22) &&
           aligned16p(A) && aligned16p(parity) && aligned16p(x);
}

hipError_t launch_onepass_f32(const OnePassArgs& a, hipStream_t st) {
    if (a.qb == 0) return hipSuccess;
    if (a.qb > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    // Wave 0 forms D while the others stream: one streaming wave per 256
    // columns up to two, then three.
    const dim3 grid(static_cast<unsigned>(a.qb));
    if (a.r <= 256)
        launch_nt<128>(a, grid, st);
    else if (a.r <= 512)
        launch_nt<192>(a, grid, st);
    else
        launch_nt<256>(a, grid, st);
    return hipGetLastError();
}

}  // namespace coded
