// C ABI of the coded matrix-multiplication library: argument checking, code
// objects, survivor draws and kernel launches.  Every entry point validates
// on the host before enqueueing anything and never throws.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <exception>
#include <new>
#include <set>
#include <string>
#include <thread>
#include <vector>

#include "internal.h"
#include "fused.h"
#include "onepass.h"

namespace coded {

static thread_local std::string g_last_error;

coded_status fail(coded_status st, const std::string& msg) {
    g_last_error = msg;
    return st;
}

coded_status hip_fail(hipError_t e, const char* what) {
    return fail(CODED_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

namespace {

constexpr size_t kMaxDecodeLds = 56 * 1024;   // dynamic part; static LDS adds under 5 KB

#define CODED_GUARD_BEGIN try {
#define CODED_GUARD_END                                                   \
    }                                                                     \
    catch (const std::bad_alloc&) {                                       \
        return fail(CODED_ERR_ARG, "host allocation failed");             \
    }                                                                     \
    catch (...) {                                                         \
        return fail(CODED_ERR_ARG, "unexpected host exception");          \
    }

coded_status check_code(const coded_code* c) {
    if (!c) return fail(CODED_ERR_ARG, "code is NULL");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != c->device)
        return fail(CODED_ERR_ARG, "code was created on device " + std::to_string(c->device) +
                                       " but device " + std::to_string(dev) + " is current");
    return CODED_OK;
}

int64_t block_rows(int64_t q, int k) { return (q + k - 1) / k; }

int64_t align256(int64_t b) { return (b + 255) / 256 * 256; }

// The code's device buffer: G (n*k doubles), then P ((n-k)*k floats), each 256-byte aligned.
int64_t code_device_bytes(int n, int k) {
    return align256(static_cast<int64_t>(n) * k * 8) + (n > k ? align256(static_cast<int64_t>(n - k) * k * 4) : 0);
}

// coded_matmul's workspace: its worker results Y (fp64 for fp32 inputs, fp32
// for bf16), 256-byte aligned, then the worker workspace.
int64_t matmul_y_bytes(const coded_code* c, coded_dtype dt, int64_t q, int64_t s) {
    const int64_t b = static_cast<int64_t>(c->n) * block_rows(q, c->k) * s * (dt == CODED_F32 ? 8 : 4);
    return (b + 255) / 256 * 256;
}

size_t dtype_size(coded_dtype d) {
    switch (d) {
        case CODED_F32: return 4;
        case CODED_BF16: return 2;
        case CODED_F64: return 8;
    }
    return 0;
}

coded_status check_dt(coded_dtype dt, coded_dtype y_dt) {
    if (dt != CODED_F32 && dt != CODED_BF16) return fail(CODED_ERR_ARG, "dt must be CODED_F32 or CODED_BF16");
    if (dt == CODED_F32 && y_dt != CODED_F64 && y_dt != CODED_F32)
        return fail(CODED_ERR_ARG, "with dt = CODED_F32, y_dt must be CODED_F64 or CODED_F32");
    if (dt == CODED_BF16 && y_dt != CODED_F32) return fail(CODED_ERR_ARG, "with dt = CODED_BF16, y_dt must be CODED_F32");
    return CODED_OK;
}

coded_status check_ar(int64_t q, int64_t r, int64_t lda) {
    if (q < 0 || r < 0) return fail(CODED_ERR_SHAPE, "q and r must be >= 0");
    if (lda < std::max<int64_t>(r, 1)) return fail(CODED_ERR_SHAPE, "lda must be >= max(r, 1)");
    return CODED_OK;
}

bool is_bf16_value(double v) {
    const float f = static_cast<float>(v);
    if (static_cast<double>(f) != v) return false;
    uint32_t b;
    std::memcpy(&b, &f, 4);
    return (b & 0xFFFFu) == 0;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// bf16 shapes served by the single-pass encode (and encode + products) kernel.
bool single_pass_bf16(const coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                      const void* parity) {
    return dt == CODED_BF16 && q > 0 && c->dPf && fused_bf16_supported(c->n, c->k, c->planes, r, lda) &&
           aligned16(A) && aligned16(parity);
}

FusedArgs fused_args(const coded_code* c, const void* A, int64_t q, int64_t r, int64_t lda, void* parity,
                     const void* xt, void* Y) {
    FusedArgs f{};
    f.A = static_cast<const uint16_t*>(A);
    f.parity = static_cast<uint16_t*>(parity);
    f.xt = static_cast<const uint16_t*>(xt);
    f.Y = static_cast<float*>(Y);
    f.P = c->dPf;
    f.q = q;
    f.r = r;
    f.lda = lda;
    f.qb = block_rows(q, c->k);
    f.n = c->n;
    f.k = c->k;
    return f;
}

coded_status do_encode(const coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                       void* parity, hipStream_t st) {
    const int64_t qb = block_rows(q, c->k);
    if (c->n == c->k || qb == 0 || r == 0) return CODED_OK;
    if (!A && q > 0) return fail(CODED_ERR_ARG, "A is NULL");
    if (!parity) return fail(CODED_ERR_ARG, "parity is NULL");
    if (dt == CODED_BF16) {
        for (size_t i = static_cast<size_t>(c->k) * c->k; i < c->G.size(); ++i)
            if (!is_bf16_value(c->G[i]))
                return fail(CODED_ERR_ARG, "bf16 encode needs every parity coefficient to be a bfloat16 value");
    }
    hipError_t e;
    if (single_pass_bf16(c, dt, A, q, r, lda, parity)) {
        e = launch_fused_bf16(fused_args(c, A, q, r, lda, parity, nullptr, nullptr), false, c->compute_units, st);
    } else {
        EncodeArgs a{A, parity, c->dG, q, r, lda, qb, c->n, c->k, c->planes, c->lo_bf16 && dt == CODED_F32};
        e = dt == CODED_F32 ? launch_encode_f32(a, st) : launch_encode_bf16(a, st);
    }
    if (e != hipSuccess) return hip_fail(e, "encode launch");
    return CODED_OK;
}

coded_status do_workers(const coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                        const void* parity, const void* X, int64_t s, int64_t ldx, const uint8_t* mask, void* Y,
                        coded_dtype y_dt, void* workspace, hipStream_t st, bool xt_ready = false) {
    if (s < 0) return fail(CODED_ERR_SHAPE, "s must be >= 0");
    if (ldx < std::max<int64_t>(s, 1)) return fail(CODED_ERR_SHAPE, "ldx must be >= max(s, 1)");
    if (s == 1 && ldx != 1 && dt == CODED_F32) {
        // a single column is read as a contiguous vector
        return fail(CODED_ERR_UNSUPPORTED, "s == 1 needs ldx == 1");
    }
    const int64_t qb = block_rows(q, c->k);
    if (qb == 0 || s == 0) return CODED_OK;
    if (!Y) return fail(CODED_ERR_ARG, "Y is NULL");
    if (r > 0) {
        if (!A && q > 0) return fail(CODED_ERR_ARG, "A is NULL");
        if (!X) return fail(CODED_ERR_ARG, "X is NULL");
        if (!parity && c->n > c->k) return fail(CODED_ERR_ARG, "parity is NULL");
    }
    WorkerArgs a{};
    a.A = A;
    a.parity = parity;
    a.X = X;
    a.Y = Y;
    a.q = q;
    a.r = r;
    a.lda = lda;
    a.qb = qb;
    a.s = s;
    a.ldx = ldx;
    a.n = c->n;
    a.k = c->k;
    a.planes = c->planes;
    a.lo_bf16 = c->lo_bf16 && dt == CODED_F32;
    a.y_f64 = y_dt == CODED_F64;
    a.xt = dt == CODED_BF16 ? workspace : nullptr;
    a.xt_ready = xt_ready ? 1 : 0;
    for (int i = 0; i < c->n; ++i) {
        if (mask && !mask[i]) continue;
        if (i < c->k)
            a.sys_ids[a.n_sys++] = static_cast<uint8_t>(i);
        else
            a.par_ids[a.n_par++] = static_cast<uint8_t>(i);
    }
    hipError_t e = dt == CODED_F32 ? launch_worker_f32(a, st) : launch_worker_bf16(a, st);
    if (e != hipSuccess) return hip_fail(e, "worker launch");
    return CODED_OK;
}

// Parity blocks, then every worker's product.  bf16 inputs of a shape the
// single-pass kernel serves, with 64 columns, read A once for both; any
// other input runs the encode and the products one after the other.
coded_status do_encode_workers(const coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                               void* parity, const void* X, int64_t s, int64_t ldx, void* Y, coded_dtype y_dt,
                               void* workspace, hipStream_t st) {
    const bool one_pass = single_pass_bf16(c, dt, A, q, r, lda, parity) && s == 64 && ldx >= 64 && X && Y &&
                          workspace && aligned16(workspace) && y_dt == CODED_F32;
    if (!one_pass) {
        if (coded_status e = do_encode(c, dt, A, q, r, lda, parity, st)) return e;
        return do_workers(c, dt, A, q, r, lda, parity, X, s, ldx, nullptr, Y, y_dt, workspace, st);
    }
    for (size_t i = static_cast<size_t>(c->k) * c->k; i < c->G.size(); ++i)
        if (!is_bf16_value(c->G[i]))
            return fail(CODED_ERR_ARG, "bf16 encode needs every parity coefficient to be a bfloat16 value");
    const hipError_t e = launch_fused_bf16_from_x(fused_args(c, A, q, r, lda, parity, workspace, Y),
                                                  static_cast<const uint16_t*>(X), s, ldx, c->compute_units, st);
    if (e != hipSuccess) return hip_fail(e, "encode and worker launch");
    return CODED_OK;
}

// First k of `count` survivors: range and repeat checks; returns the sorted set.
coded_status take_survivors(const coded_code* c, const int32_t* survivors, int32_t count, DecodeSet& set, int& m) {
    if (!survivors) return fail(CODED_ERR_ARG, "survivors is NULL");
    if (count < c->k)
        return fail(CODED_ERR_TOO_FEW, "need k = " + std::to_string(c->k) + " survivors, got " + std::to_string(count));
    std::vector<int32_t> v(survivors, survivors + c->k);
    for (int32_t w : v)
        if (w < 0 || w >= c->n) return fail(CODED_ERR_ARG, "survivor index " + std::to_string(w) + " outside [0, n)");
    std::sort(v.begin(), v.end());
    if (std::adjacent_find(v.begin(), v.end()) != v.end()) return fail(CODED_ERR_ARG, "repeated survivor index");
    std::memset(&set, 0, sizeof(set));
    m = 0;
    for (int i = 0; i < c->k; ++i) {
        set.packed[i / 4] |= static_cast<uint32_t>(v[i]) << (8 * (i % 4));
        m += v[i] >= c->k;
    }
    return CODED_OK;
}

coded_status do_decode_single(const coded_code* c, const DecodeSet& set, int m, const void* Y, coded_dtype y_dt,
                              int64_t q, int64_t s, float* out, int64_t ldo, int32_t* info, hipStream_t st,
                              const float* cvec = nullptr, double alpha = 1.0, double beta = 0.0) {
    if (y_dt != CODED_F64 && y_dt != CODED_F32) return fail(CODED_ERR_ARG, "y_dt must be CODED_F64 or CODED_F32");
    if (q < 0 || s < 0) return fail(CODED_ERR_SHAPE, "q and s must be >= 0");
    if (ldo < std::max<int64_t>(s, 1)) return fail(CODED_ERR_SHAPE, "ldo must be >= max(s, 1)");
    if (!info) return fail(CODED_ERR_ARG, "info is NULL");
    const int64_t qb = block_rows(q, c->k);
    if (qb * s > 0 && (!Y || !out)) return fail(CODED_ERR_ARG, "Y or out is NULL");
    if (decode_lds_bytes(c->k, std::max(m, 1)) > kMaxDecodeLds)
        return fail(CODED_ERR_UNSUPPORTED, "survivor system too large for one workgroup's LDS");
    DecodeArgs a{c->dG, Y, out, info, nullptr, q, qb, s, ldo, 0, c->n, c->k, 1, y_dt == CODED_F64};
    a.c = cvec;
    a.alpha = alpha;
    a.beta = beta;
    hipError_t e = launch_decode(a, &set, m, st);
    if (e != hipSuccess) return hip_fail(e, "decode launch");
    return CODED_OK;
}

// Number of k-subsets of the n workers holding at least min_parity of the n-k
// parity workers, saturating at 2^64 - 1 (binomials from Pascal's triangle in
// saturating arithmetic; n <= CODED_MAX_N).
uint64_t qualifying_sets(int n, int k, int min_parity) {
    constexpr uint64_t kSat = ~0ull;
    std::vector<std::vector<uint64_t>> C(n + 1, std::vector<uint64_t>(n + 1, 0));
    for (int a = 0; a <= n; ++a) {
        C[a][0] = 1;
        for (int b = 1; b <= a; ++b) {
            const uint64_t x = C[a - 1][b - 1], y = C[a - 1][b];
            C[a][b] = x > kSat - y ? kSat : x + y;
        }
    }
    uint64_t total = 0;
    for (int m = min_parity; m <= std::min(k, n - k); ++m) {
        const uint64_t x = C[k][m], y = C[n - k][m];
        const uint64_t prod = (x != 0 && y > kSat / x) ? kSat : x * y;
        total = prod > kSat - total ? kSat : total + prod;
    }
    return total;
}

}  // namespace
}  // namespace coded

using namespace coded;

extern "C" {

coded_status coded_code_bytes(int32_t n, int32_t k, int64_t* bytes) {
    CODED_GUARD_BEGIN
    if (!bytes) return fail(CODED_ERR_ARG, "bytes is NULL");
    if (k < 1 || n < k || n > CODED_MAX_N) return fail(CODED_ERR_ARG, "need 1 <= k <= n <= CODED_MAX_N");
    *bytes = code_device_bytes(n, k);
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_code_create(int32_t n, int32_t k, const double* G, int32_t planes, void* device_buf,
                               int64_t device_buf_bytes, coded_code** out) {
    CODED_GUARD_BEGIN
    if (!out) return fail(CODED_ERR_ARG, "out is NULL");
    *out = nullptr;
    if (!G) return fail(CODED_ERR_ARG, "G is NULL");
    if (k < 1 || n < k || n > CODED_MAX_N) return fail(CODED_ERR_ARG, "need 1 <= k <= n <= CODED_MAX_N");
    if (planes != 1 && planes != 2 && planes != CODED_PLANES_LO_BF16)
        return fail(CODED_ERR_ARG, "planes must be 1, 2 or CODED_PLANES_LO_BF16");
    for (int64_t i = 0; i < static_cast<int64_t>(n) * k; ++i)
        if (!std::isfinite(G[i])) return fail(CODED_ERR_ARG, "G has a non-finite entry");
    for (int i = 0; i < k; ++i)
        for (int j = 0; j < k; ++j)
            if (G[i * k + j] != (i == j ? 1.0 : 0.0))
                return fail(CODED_ERR_UNSUPPORTED, "only systematic codes (rows 0..k-1 of G equal to I_k) are supported");
    const int64_t need = code_device_bytes(n, k);
    if (!device_buf) return fail(CODED_ERR_ARG, "device_buf is NULL");
    if (device_buf_bytes < need)
        return fail(CODED_ERR_ARG, "device_buf holds " + std::to_string(device_buf_bytes) + " bytes; the code needs " +
                                       std::to_string(need));
    if (!aligned16(device_buf)) return fail(CODED_ERR_ARG, "device_buf must be 16-byte aligned");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    hipPointerAttribute_t attr{};
    e = hipPointerGetAttributes(&attr, device_buf);
    if (e != hipSuccess || attr.type != hipMemoryTypeDevice || attr.device != dev) {
        (void)hipGetLastError();
        return fail(CODED_ERR_ARG, "device_buf must be device memory of the current device");
    }
    auto* c = new coded_code();
    c->n = n;
    c->k = k;
    c->planes = planes == CODED_PLANES_LO_BF16 ? 2 : planes;
    c->lo_bf16 = planes == CODED_PLANES_LO_BF16;
    c->device = dev;
    c->G.assign(G, G + static_cast<size_t>(n) * k);
    c->dG = static_cast<double*>(device_buf);
    e = hipMemcpy(c->dG, c->G.data(), c->G.size() * sizeof(double), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&c->compute_units, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess && n > k) {
        std::vector<float> pf(static_cast<size_t>(n - k) * k);
        for (size_t i = 0; i < pf.size(); ++i) pf[i] = static_cast<float>(c->G[static_cast<size_t>(k) * k + i]);
        c->dPf = reinterpret_cast<float*>(static_cast<char*>(device_buf) + align256(static_cast<int64_t>(n) * k * 8));
        e = hipMemcpy(c->dPf, pf.data(), pf.size() * sizeof(float), hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) {
        delete c;
        return hip_fail(e, "coded_code_create");
    }
    *out = c;
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_code_destroy(coded_code* c) {
    CODED_GUARD_BEGIN
    if (!c) return CODED_OK;
    // teardown: a failure to release one handle must not stop the others
    for (hipEvent_t ev : c->worker_events) (void)hipEventDestroy(ev);
    if (c->start_event) (void)hipEventDestroy(c->start_event);
    for (hipStream_t w : c->worker_streams) (void)hipStreamDestroy(w);
    delete c;
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_code_info(const coded_code* c, int32_t* n, int32_t* k, int32_t* planes) {
    if (!c) return fail(CODED_ERR_ARG, "code is NULL");
    if (n) *n = c->n;
    if (k) *k = c->k;
    if (planes) *planes = c->lo_bf16 ? CODED_PLANES_LO_BF16 : c->planes;
    return CODED_OK;
}

coded_status coded_sizes(const coded_code* c, coded_dtype dt, coded_dtype y_dt, int64_t q, int64_t r, int64_t s,
                         int64_t* parity_bytes, int64_t* y_bytes, int64_t* workspace_bytes,
                         int64_t* worker_workspace_bytes) {
    CODED_GUARD_BEGIN
    if (!c) return fail(CODED_ERR_ARG, "code is NULL");
    if (coded_status st = check_dt(dt, y_dt)) return st;
    if (q < 0 || r < 0 || s < 0) return fail(CODED_ERR_SHAPE, "q, r, s must be >= 0");
    const int64_t qb = block_rows(q, c->k);
    if (parity_bytes)
        *parity_bytes = (c->lo_bf16 && dt == CODED_F32 ? 6 : static_cast<int64_t>(c->planes) * dtype_size(dt)) *
                        (c->n - c->k) * qb * r;
    if (y_bytes) *y_bytes = static_cast<int64_t>(c->n) * qb * s * static_cast<int64_t>(dtype_size(y_dt));
    const int64_t wws = dt == CODED_BF16 ? worker_workspace_bytes_bf16(r, s) : 0;
    if (workspace_bytes) *workspace_bytes = matmul_y_bytes(c, dt, q, s) + wws;
    if (worker_workspace_bytes) *worker_workspace_bytes = wws;
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_encode(const coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                          void* parity, void* stream) {
    CODED_GUARD_BEGIN
    if (coded_status st = check_code(c)) return st;
    if (dt != CODED_F32 && dt != CODED_BF16) return fail(CODED_ERR_ARG, "dt must be CODED_F32 or CODED_BF16");
    if (coded_status st = check_ar(q, r, lda)) return st;
    return do_encode(c, dt, A, q, r, lda, parity, static_cast<hipStream_t>(stream));
    CODED_GUARD_END
}

coded_status coded_worker_mm(const coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                             const void* parity, const void* X, int64_t s, int64_t ldx, const uint8_t* worker_mask,
                             void* Y, coded_dtype y_dt, void* workspace, void* stream) {
    CODED_GUARD_BEGIN
    if (coded_status st = check_code(c)) return st;
    if (coded_status st = check_dt(dt, y_dt)) return st;
    if (coded_status st = check_ar(q, r, lda)) return st;
    return do_workers(c, dt, A, q, r, lda, parity, X, s, ldx, worker_mask, Y, y_dt, workspace,
                      static_cast<hipStream_t>(stream));
    CODED_GUARD_END
}

coded_status coded_encode_worker_mm(const coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r,
                                    int64_t lda, void* parity, const void* X, int64_t s, int64_t ldx, void* Y,
                                    coded_dtype y_dt, void* workspace, void* stream) {
    CODED_GUARD_BEGIN
    if (coded_status st = check_code(c)) return st;
    if (coded_status st = check_dt(dt, y_dt)) return st;
    if (coded_status st = check_ar(q, r, lda)) return st;
    if (s < 0) return fail(CODED_ERR_SHAPE, "s must be >= 0");
    if (ldx < std::max<int64_t>(s, 1)) return fail(CODED_ERR_SHAPE, "ldx must be >= max(s, 1)");
    if (block_rows(q, c->k) * s > 0 && r > 0 && (!X || !Y)) return fail(CODED_ERR_ARG, "X or Y is NULL");
    if (dt == CODED_BF16 && !workspace && block_rows(q, c->k) * s > 0 && r > 0)
        return fail(CODED_ERR_ARG, "bf16 needs the worker workspace");
    return do_encode_workers(c, dt, A, q, r, lda, parity, X, s, ldx, Y, y_dt, workspace,
                             static_cast<hipStream_t>(stream));
    CODED_GUARD_END
}

coded_status coded_decode(const coded_code* c, const int32_t* survivors, int32_t count, const void* Y,
                          coded_dtype y_dt, int64_t q, int64_t s, float* out, int64_t ldo, int32_t* info,
                          void* stream) {
    CODED_GUARD_BEGIN
    if (coded_status st = check_code(c)) return st;
    DecodeSet set;
    int m = 0;
    if (coded_status st = take_survivors(c, survivors, count, set, m)) return st;
    return do_decode_single(c, set, m, Y, y_dt, q, s, out, ldo, info, static_cast<hipStream_t>(stream));
    CODED_GUARD_END
}

coded_status coded_decode_batched(const coded_code* c, const int32_t* sets, int32_t batch, const void* Y,
                                  coded_dtype y_dt, int64_t q, int64_t s, float* out, int64_t ldo,
                                  int64_t out_stride, int32_t* info, void* stream) {
    CODED_GUARD_BEGIN
    if (coded_status st = check_code(c)) return st;
    if (y_dt != CODED_F64 && y_dt != CODED_F32) return fail(CODED_ERR_ARG, "y_dt must be CODED_F64 or CODED_F32");
    if (batch < 0) return fail(CODED_ERR_ARG, "batch must be >= 0");
    if (batch == 0) return CODED_OK;
    if (q < 0 || s < 0) return fail(CODED_ERR_SHAPE, "q and s must be >= 0");
    if (ldo < std::max<int64_t>(s, 1)) return fail(CODED_ERR_SHAPE, "ldo must be >= max(s, 1)");
    if (batch > 1 && out_stride < q * ldo) return fail(CODED_ERR_SHAPE, "out_stride must be >= q * ldo");
    if (!sets || !info) return fail(CODED_ERR_ARG, "sets or info is NULL");
    const int64_t qb = block_rows(q, c->k);
    if (qb * s > 0 && (!Y || !out)) return fail(CODED_ERR_ARG, "Y or out is NULL");
    const int mmax = std::min(c->k, c->n - c->k);
    if (decode_lds_bytes(c->k, std::max(mmax, 1)) > kMaxDecodeLds)
        return fail(CODED_ERR_UNSUPPORTED, "survivor system too large for one workgroup's LDS");
    DecodeArgs a{c->dG, Y, out, info, sets, q, qb, s, ldo, out_stride, c->n, c->k, batch, y_dt == CODED_F64};
    hipError_t e = launch_decode(a, nullptr, mmax, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "decode launch");
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_draw_survivors(int32_t n, int32_t k, uint64_t seed, uint64_t draw, double shift, double rate,
                                  int32_t* survivors_out, double* t_overall_out) {
    CODED_GUARD_BEGIN
    if (k < 1 || n < k || n > CODED_MAX_N) return fail(CODED_ERR_ARG, "need 1 <= k <= n <= CODED_MAX_N");
    if (!survivors_out) return fail(CODED_ERR_ARG, "survivors_out is NULL");
    if (!(rate > 0.0) || !std::isfinite(shift)) return fail(CODED_ERR_ARG, "need rate > 0 and a finite shift");
    if (draw >= (1ull << 40)) return fail(CODED_ERR_ARG, "draw must be < 2^40");
    const double t = coded_rng::draw_survivors(n, k, seed, draw, shift, rate, survivors_out);
    if (t_overall_out) *t_overall_out = t;
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_draw_survivor_sets(int32_t n, int32_t k, uint64_t seed, uint64_t first_draw, int32_t batch,
                                      int32_t min_parity, int32_t* sets_out, uint64_t* next_draw_out) {
    CODED_GUARD_BEGIN
    if (k < 1 || n < k || n > CODED_MAX_N) return fail(CODED_ERR_ARG, "need 1 <= k <= n <= CODED_MAX_N");
    if (batch < 0) return fail(CODED_ERR_ARG, "batch must be >= 0");
    if (batch > 0 && !sets_out) return fail(CODED_ERR_ARG, "sets_out is NULL");
    if (min_parity < 0 || min_parity > std::min(k, n - k))
        return fail(CODED_ERR_ARG, "min_parity must lie in [0, min(k, n-k)]");
    // Distinct sets with m >= min_parity parity members: sum_m C(k, m) C(n-k, m)
    // (m parity workers in, m systematic ones out).  More are never found.
    if (static_cast<uint64_t>(batch) > qualifying_sets(n, k, min_parity))
        return fail(CODED_ERR_ARG, "batch exceeds the number of distinct survivor sets with at least min_parity "
                                   "parity workers");
    std::set<std::vector<int32_t>> seen;
    std::vector<int32_t> cur(k);
    uint64_t d = first_draw;
    int32_t got = 0;
    while (got < batch) {
        if (d >= (1ull << 40)) return fail(CODED_ERR_ARG, "ran out of draws");
        coded_rng::draw_survivors(n, k, seed, d, 1.0, 1.0, cur.data());
        ++d;
        int m = 0;
        for (int32_t w : cur) m += w >= k;
        if (m < min_parity) continue;
        if (!seen.insert(cur).second) continue;
        std::copy(cur.begin(), cur.end(), sets_out + static_cast<int64_t>(got) * k);
        ++got;
    }
    if (next_draw_out) *next_draw_out = d;
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_matmul(const coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                          void* parity, int32_t parity_ready, const void* X, int64_t s, int64_t ldx, uint64_t seed,
                          uint64_t draw, double shift, double rate, int32_t* survivors_out, double* t_overall_out,
                          float* out, int64_t ldo, void* workspace, int32_t* info, void* stream) {
    CODED_GUARD_BEGIN
    if (coded_status st = check_code(c)) return st;
    const coded_dtype y_dt = dt == CODED_F32 ? CODED_F64 : CODED_F32;
    if (coded_status st = check_dt(dt, y_dt)) return st;
    if (coded_status st = check_ar(q, r, lda)) return st;
    if (s < 0) return fail(CODED_ERR_SHAPE, "s must be >= 0");
    if (ldo < std::max<int64_t>(s, 1)) return fail(CODED_ERR_SHAPE, "ldo must be >= max(s, 1)");
    if (!info) return fail(CODED_ERR_ARG, "info is NULL");
    if (!(rate > 0.0) || !std::isfinite(shift)) return fail(CODED_ERR_ARG, "need rate > 0 and a finite shift");
    if (draw >= (1ull << 40)) return fail(CODED_ERR_ARG, "draw must be < 2^40");
    const int64_t qb = block_rows(q, c->k);
    if (qb * s > 0 && (!workspace || !out)) return fail(CODED_ERR_ARG, "workspace or out is NULL");
    hipStream_t st = static_cast<hipStream_t>(stream);

    // Survivors first: a host-only step, so a bad argument enqueues nothing.
    int32_t surv[CODED_MAX_N];
    const double t = coded_rng::draw_survivors(c->n, c->k, seed, draw, shift, rate, surv);
    DecodeSet set;
    int m = 0;
    if (coded_status s2 = take_survivors(c, surv, c->k, set, m)) return s2;
    if (decode_lds_bytes(c->k, std::max(m, 1)) > kMaxDecodeLds)
        return fail(CODED_ERR_UNSUPPORTED, "survivor system too large for one workgroup's LDS");
    if (s == 1 && ldx != 1 && dt == CODED_F32) return fail(CODED_ERR_UNSUPPORTED, "s == 1 needs ldx == 1");
    if (ldx < std::max<int64_t>(s, 1)) return fail(CODED_ERR_SHAPE, "ldx must be >= max(s, 1)");

    void* wws = static_cast<char*>(workspace) + matmul_y_bytes(c, dt, q, s);
    if (dt == CODED_F32 && s == 1 && ldx == 1 && c->n > c->k && A && X && parity && !c->lo_bf16 &&
        onepass_supported(c->n, c->k, q, r, lda, A, parity, X)) {
        // small problem: encode (unless ready), products and decode in one launch
        OnePassArgs oa{};
        oa.A = static_cast<const float*>(A);
        oa.parity = static_cast<float*>(parity);
        oa.x = static_cast<const float*>(X);
        oa.Y = static_cast<double*>(workspace);
        oa.out = out;
        oa.info = info;
        oa.G = c->dG;
        oa.set = set;
        oa.q = q;
        oa.r = r;
        oa.lda = lda;
        oa.qb = qb;
        oa.ldo = ldo;
        oa.n = c->n;
        oa.k = c->k;
        oa.planes = c->planes;
        oa.encode = parity_ready ? 0 : 1;
        oa.missing = m;
        const hipError_t e = launch_onepass_f32(oa, st);
        if (e != hipSuccess) return hip_fail(e, "one-pass product launch");
        if (survivors_out) std::copy(surv, surv + c->k, survivors_out);
        if (t_overall_out) *t_overall_out = t;
        return CODED_OK;
    }
    if (!parity_ready) {
        if (coded_status s2 = do_encode_workers(c, dt, A, q, r, lda, parity, X, s, ldx, workspace, y_dt, wws, st))
            return s2;
    } else if (coded_status s2 = do_workers(c, dt, A, q, r, lda, parity, X, s, ldx, nullptr, workspace, y_dt, wws, st)) {
        return s2;
    }
    if (coded_status s2 = do_decode_single(c, set, m, workspace, y_dt, q, s, out, ldo, info, st)) return s2;
    if (survivors_out) std::copy(surv, surv + c->k, survivors_out);
    if (t_overall_out) *t_overall_out = t;
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_matmul_noalloc(const coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r,
                                  int64_t lda, void* parity, int32_t parity_ready, const void* X, int64_t s,
                                  int64_t ldx, uint64_t seed, uint64_t draw, double shift, double rate,
                                  int32_t* survivors_out, double* t_overall_out, float* out, int64_t ldo,
                                  int32_t* info, void* stream) {
    CODED_GUARD_BEGIN
    if (coded_status st = check_code(c)) return st;
    const coded_dtype y_dt = dt == CODED_F32 ? CODED_F64 : CODED_F32;
    if (coded_status st = check_dt(dt, y_dt)) return st;
    if (q < 0 || r < 0 || s < 0) return fail(CODED_ERR_SHAPE, "q, r, s must be >= 0");
    const int64_t need = matmul_y_bytes(c, dt, q, s) + (dt == CODED_BF16 ? worker_workspace_bytes_bf16(r, s) : 0);
    if (need > static_cast<int64_t>(CODED_NOALLOC_SCRATCH_BYTES))
        return fail(CODED_ERR_UNSUPPORTED, "the product needs " + std::to_string(need) +
                                               " bytes of workspace; the static scratch holds " +
                                               std::to_string(static_cast<int64_t>(CODED_NOALLOC_SCRATCH_BYTES)));
    void* ws = nullptr;
    if (coded_status st = static_scratch(&ws)) return st;
    return coded_matmul(c, dt, A, q, r, lda, parity, parity_ready, X, s, ldx, seed, draw, shift, rate, survivors_out,
                        t_overall_out, out, ldo, ws, info, stream);
    CODED_GUARD_END
}

namespace {

constexpr int kStragglerStreams = 4;          // the device's default number of hardware queues
constexpr double kStragglerMaxStartUs = 60e6;  // latest start the host waits for

coded_status ensure_straggler_state(coded_code* c) {
    if (!c->worker_streams.empty()) return CODED_OK;
    std::vector<hipStream_t> streams;
    std::vector<hipEvent_t> events;
    hipEvent_t start = nullptr;
    hipError_t e = hipEventCreateWithFlags(&start, hipEventDisableTiming);
    for (int i = 0; e == hipSuccess && i < kStragglerStreams; ++i) {
        hipStream_t w = nullptr;
        e = hipStreamCreateWithFlags(&w, hipStreamNonBlocking);
        if (e == hipSuccess) streams.push_back(w);
    }
    for (int i = 0; e == hipSuccess && i < c->n; ++i) {
        hipEvent_t ev = nullptr;
        e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e == hipSuccess) events.push_back(ev);
    }
    if (e != hipSuccess) {
        // undo what was created; the first error is the one reported
        for (hipEvent_t ev : events) (void)hipEventDestroy(ev);
        for (hipStream_t w : streams) (void)hipStreamDestroy(w);
        if (start) (void)hipEventDestroy(start);
        return hip_fail(e, "straggler streams and events");
    }
    c->worker_streams = std::move(streams);
    c->worker_events = std::move(events);
    c->start_event = start;
    return CODED_OK;
}

}  // namespace

coded_status coded_straggler_matmul(coded_code* c, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                                    const void* parity, const void* X, int64_t s, int64_t ldx, uint64_t seed,
                                    uint64_t draw, double shift, double rate, double time_unit_us,
                                    int32_t launch_all, void* Y, coded_dtype y_dt, void* workspace, float* out,
                                    int64_t ldo, int32_t* info, int32_t* survivors_out, double* timeline_out,
                                    double* latency_us_out, void* stream) {
    CODED_GUARD_BEGIN
    using clock = std::chrono::steady_clock;
    const auto t0 = clock::now();
    auto now_us = [&]() { return std::chrono::duration<double, std::micro>(clock::now() - t0).count(); };
    if (coded_status st = check_code(c)) return st;
    if (coded_status st = check_dt(dt, y_dt)) return st;
    if (coded_status st = check_ar(q, r, lda)) return st;
    if (s < 0) return fail(CODED_ERR_SHAPE, "s must be >= 0");
    if (ldx < std::max<int64_t>(s, 1)) return fail(CODED_ERR_SHAPE, "ldx must be >= max(s, 1)");
    if (s == 1 && ldx != 1 && dt == CODED_F32) return fail(CODED_ERR_UNSUPPORTED, "s == 1 needs ldx == 1");
    if (ldo < std::max<int64_t>(s, 1)) return fail(CODED_ERR_SHAPE, "ldo must be >= max(s, 1)");
    if (!info) return fail(CODED_ERR_ARG, "info is NULL");
    if (!(rate > 0.0) || !std::isfinite(shift)) return fail(CODED_ERR_ARG, "need rate > 0 and a finite shift");
    if (!(time_unit_us >= 0.0) || !std::isfinite(time_unit_us)) return fail(CODED_ERR_ARG, "need time_unit_us >= 0");
    if (draw >= (1ull << 40)) return fail(CODED_ERR_ARG, "draw must be < 2^40");
    const int64_t qb = block_rows(q, c->k);
    if (qb * s > 0 && (!Y || !out)) return fail(CODED_ERR_ARG, "Y or out is NULL");
    if (qb * s > 0 && r > 0 && (!X || (q > 0 && !A) || (!parity && c->n > c->k)))
        return fail(CODED_ERR_ARG, "A, parity or X is NULL");
    if (dt == CODED_BF16 && qb * s > 0 && r > 0 && !workspace)
        return fail(CODED_ERR_ARG, "bf16 needs the worker workspace");
    if (decode_lds_bytes(c->k, std::max(std::min(c->k, c->n - c->k), 1)) > kMaxDecodeLds)
        return fail(CODED_ERR_UNSUPPORTED, "survivor system too large for one workgroup's LDS");

    // Start times from the runtime model (Sec. III-C), in the order they fall.
    const int n = c->n, k = c->k;
    std::vector<double> sched(n);
    coded_rng::worker_times(n, k, seed, draw, shift, rate, sched.data());
    for (double& t : sched) t *= time_unit_us;
    std::vector<int> order(n);
    for (int i = 0; i < n; ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return sched[a] < sched[b]; });
    if (sched[order[k - 1]] > kStragglerMaxStartUs)
        return fail(CODED_ERR_ARG, "the k-th start time exceeds 60 s; use a smaller time unit");
    if (coded_status st = ensure_straggler_state(c)) return st;

    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e = hipSuccess;
    if (dt == CODED_BF16 && qb * s > 0 && r > 0) {
        // X is transposed once, before any worker starts (the workers share it)
        WorkerArgs xa{};
        xa.X = X;
        xa.r = r;
        xa.s = s;
        xa.ldx = ldx;
        xa.xt = workspace;
        e = launch_transpose_x_bf16(xa, st);
        if (e != hipSuccess) return hip_fail(e, "transpose launch");
    }
    // Products start after everything already enqueued on the caller's stream.
    e = hipEventRecord(c->start_event, st);
    for (int i = 0; e == hipSuccess && i < kStragglerStreams; ++i) e = hipStreamWaitEvent(c->worker_streams[i], c->start_event, 0);
    if (e != hipSuccess) return hip_fail(e, "ordering the worker streams");

    std::vector<double> launched_at(n, -1.0), seen_at(n, -1.0);
    std::vector<int> pending, arrivals;
    std::vector<uint8_t> mask(n, 0);
    int next = 0, launches = 0;
    auto launch = [&](int i) -> coded_status {
        std::fill(mask.begin(), mask.end(), 0);
        mask[i] = 1;
        hipStream_t ws = c->worker_streams[launches % kStragglerStreams];
        launched_at[i] = now_us();
        if (coded_status s2 = do_workers(c, dt, A, q, r, lda, parity, X, s, ldx, mask.data(), Y, y_dt, workspace, ws,
                                         dt == CODED_BF16))
            return s2;
        hipError_t e2 = hipEventRecord(c->worker_events[i], ws);
        if (e2 != hipSuccess) return hip_fail(e2, "worker event");
        ++launches;
        pending.push_back(i);
        return CODED_OK;
    };
    // The master's loop: start the workers whose time has come, collect
    // completions, stop at the k-th.
    while (static_cast<int>(arrivals.size()) < k) {
        const double t = now_us();
        while (next < n && sched[order[next]] <= t)
            if (coded_status s2 = launch(order[next++])) return s2;
        for (size_t j = 0; j < pending.size();) {
            const int i = pending[j];
            const hipError_t qe = hipEventQuery(c->worker_events[i]);
            if (qe == hipSuccess) {
                seen_at[i] = now_us();
                arrivals.push_back(i);
                pending.erase(pending.begin() + j);
            } else if (qe == hipErrorNotReady) {
                ++j;
            } else {
                return hip_fail(qe, "worker event query");
            }
        }
        if (static_cast<int>(arrivals.size()) >= k) break;
        if (t > kStragglerMaxStartUs + 60e6) return fail(CODED_ERR_HIP, "workers did not complete within 60 s");
        // sleep through long gaps before the next start, poll otherwise
        const double gap = next < n ? sched[order[next]] - now_us() : 0.0;
        if (pending.empty() && gap > 300.0)
            std::this_thread::sleep_for(std::chrono::microseconds(static_cast<int64_t>(std::min(gap - 200.0, 1000.0))));
        else
            std::this_thread::yield();
    }
    arrivals.resize(k);

    // Decode from the first k arrivals, in arrival order.
    DecodeSet set;
    int m = 0;
    if (coded_status s2 = take_survivors(c, arrivals.data(), k, set, m)) return s2;
    for (int i : arrivals) {
        e = hipStreamWaitEvent(st, c->worker_events[i], 0);
        if (e != hipSuccess) return hip_fail(e, "ordering the decode");
    }
    if (coded_status s2 = do_decode_single(c, set, m, Y, y_dt, q, s, out, ldo, info, st)) return s2;
    e = hipEventRecord(c->start_event, st);     // reused: marks the decode's end
    if (e != hipSuccess) return hip_fail(e, "decode event");
    // The rest of the workers: started now (launch_all) or never (survivors only).
    if (launch_all)
        while (next < n)
            if (coded_status s2 = launch(order[next++])) return s2;
    e = hipEventSynchronize(c->start_event);
    if (e != hipSuccess) return hip_fail(e, "decode wait");
    const double latency = now_us();
    // Later work on the caller's stream waits for every product started here.
    for (int i : pending) {
        e = hipStreamWaitEvent(st, c->worker_events[i], 0);
        if (e != hipSuccess) return hip_fail(e, "ordering the stragglers");
    }
    if (survivors_out) std::copy(arrivals.begin(), arrivals.end(), survivors_out);
    if (latency_us_out) *latency_us_out = latency;
    if (timeline_out)
        for (int i = 0; i < n; ++i) {
            timeline_out[3 * i] = sched[i];
            timeline_out[3 * i + 1] = launched_at[i];
            timeline_out[3 * i + 2] = seen_at[i];
        }
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_transpose(const float* A, int64_t q, int64_t r, int64_t lda, float* AT, int64_t ldat,
                             void* stream) {
    CODED_GUARD_BEGIN
    if (q < 0 || r < 0) return fail(CODED_ERR_SHAPE, "q and r must be >= 0");
    if (lda < std::max<int64_t>(r, 1) || ldat < std::max<int64_t>(q, 1)) return fail(CODED_ERR_SHAPE, "bad lda / ldat");
    if (q > 0 && r > 0 && (!A || !AT)) return fail(CODED_ERR_ARG, "A or AT is NULL");
    hipError_t e = launch_transpose_f32(A, q, r, lda, AT, ldat, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "transpose launch");
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_gd_sizes(const coded_code* cA, const coded_code* cT, int64_t q, int64_t r,
                            int64_t* workspace_bytes) {
    if (!cA || !cT) return fail(CODED_ERR_ARG, "code is NULL");
    if (q < 0 || r < 0) return fail(CODED_ERR_SHAPE, "q and r must be >= 0");
    const int64_t y1 = static_cast<int64_t>(cA->n) * block_rows(q, cA->k) * 8;
    const int64_t y2 = static_cast<int64_t>(cT->n) * block_rows(r, cT->k) * 8;
    if (workspace_bytes) *workspace_bytes = align256(y1) + align256(y2) + align256(q * 4);
    return CODED_OK;
}

coded_status coded_gd_step(const coded_code* cA, const coded_code* cT, const float* A, int64_t lda,
                           const float* parityA, const float* AT, int64_t ldat, const float* parityAT, int64_t q,
                           int64_t r, const float* y, float* x, double eta, uint64_t seed, uint64_t iteration,
                           double shift, double rate, void* workspace, int32_t* info, int32_t* survivors_out,
                           void* stream) {
    CODED_GUARD_BEGIN
    if (coded_status st = check_code(cA)) return st;
    if (coded_status st = check_code(cT)) return st;
    if (coded_status st = check_ar(q, r, lda)) return st;
    if (coded_status st = check_ar(r, q, ldat)) return st;
    if (q == 0 || r == 0) return fail(CODED_ERR_SHAPE, "q and r must be > 0");
    if (!y || !x || !workspace || !info) return fail(CODED_ERR_ARG, "y, x, workspace or info is NULL");
    if (!(rate > 0.0) || !std::isfinite(shift) || !std::isfinite(eta)) return fail(CODED_ERR_ARG, "need rate > 0, finite shift and eta");
    if (iteration >= (1ull << 38)) return fail(CODED_ERR_ARG, "iteration must be < 2^38");
    hipStream_t st = static_cast<hipStream_t>(stream);
    // Survivors of both products first (host only; nothing is enqueued on failure).
    int32_t s1[CODED_MAX_N], s2[CODED_MAX_N];
    coded_rng::draw_survivors(cA->n, cA->k, seed, 2 * iteration, shift, rate, s1);
    coded_rng::draw_survivors(cT->n, cT->k, seed, 2 * iteration + 1, shift, rate, s2);
    DecodeSet set1, set2;
    int m1 = 0, m2 = 0;
    if (coded_status e = take_survivors(cA, s1, cA->k, set1, m1)) return e;
    if (coded_status e = take_survivors(cT, s2, cT->k, set2, m2)) return e;
    if (decode_lds_bytes(cA->k, std::max(m1, 1)) > kMaxDecodeLds || decode_lds_bytes(cT->k, std::max(m2, 1)) > kMaxDecodeLds)
        return fail(CODED_ERR_UNSUPPORTED, "survivor system too large for one workgroup's LDS");
    char* ws = static_cast<char*>(workspace);
    double* Y1 = reinterpret_cast<double*>(ws);
    double* Y2 = reinterpret_cast<double*>(ws + align256(static_cast<int64_t>(cA->n) * block_rows(q, cA->k) * 8));
    float* z = reinterpret_cast<float*>(reinterpret_cast<char*>(Y2) +
                                        align256(static_cast<int64_t>(cT->n) * block_rows(r, cT->k) * 8));
    // z = A x - y  (coded product with code A, residual fused into the decode)
    if (coded_status e = do_workers(cA, CODED_F32, A, q, r, lda, parityA, x, 1, 1, nullptr, Y1, CODED_F64, nullptr, st)) return e;
    if (coded_status e = do_decode_single(cA, set1, m1, Y1, CODED_F64, q, 1, z, 1, info, st, y, 1.0, -1.0)) return e;
    // x = x - eta A^T z  (coded product with the code of A^T, update fused into the decode)
    if (coded_status e = do_workers(cT, CODED_F32, AT, r, q, ldat, parityAT, z, 1, 1, nullptr, Y2, CODED_F64, nullptr, st)) return e;
    if (coded_status e = do_decode_single(cT, set2, m2, Y2, CODED_F64, r, 1, x, 1, info + 1, st, x, -eta, 1.0)) return e;
    if (survivors_out) {
        std::copy(s1, s1 + cA->k, survivors_out);
        std::copy(s2, s2 + cT->k, survivors_out + cA->k);
    }
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_simulate_runtimes(int32_t n, int32_t k, uint64_t seed, uint64_t first_draw, int64_t count,
                                     double shift, double rate, double* t_uncoded, double* t_repetition, double* t_mds,
                                     void* stream) {
    CODED_GUARD_BEGIN
    if (k < 1 || n < k || n > CODED_MAX_N) return fail(CODED_ERR_ARG, "need 1 <= k <= n <= CODED_MAX_N");
    if (count < 0) return fail(CODED_ERR_ARG, "count must be >= 0");
    if (!(rate > 0.0) || !std::isfinite(shift)) return fail(CODED_ERR_ARG, "need rate > 0 and a finite shift");
    if (first_draw + static_cast<uint64_t>(count) > (1ull << 40)) return fail(CODED_ERR_ARG, "draws must stay below 2^40");
    if (t_repetition && n % k != 0) return fail(CODED_ERR_ARG, "repetition needs k to divide n");
    hipError_t e = launch_runtime_sim(n, k, seed, first_draw, count, shift, rate, t_uncoded, t_repetition, t_mds,
                                      static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "runtime simulation launch");
    return CODED_OK;
    CODED_GUARD_END
}

coded_status coded_optimal_k(int32_t n, double rate, double* k_star, double* t_star, int32_t* k_best) {
    CODED_GUARD_BEGIN
    if (n < 1) return fail(CODED_ERR_ARG, "n must be >= 1");
    if (!(rate > 0.0) || !std::isfinite(rate)) return fail(CODED_ERR_ARG, "rate must be > 0");
    const double w = coded_rng::lambert_w_lower(-std::exp(-rate - 1.0));
    if (k_star) *k_star = (1.0 + 1.0 / w) * n;
    if (t_star) *t_star = -w / (rate * n);
    if (k_best) {
        // exact expected MDS runtime (1/k)(1 + (H_n - H_{n-k})/rate), smallest over integer k
        std::vector<double> H(n + 1, 0.0);
        for (int i = 1; i <= n; ++i) H[i] = H[i - 1] + 1.0 / i;
        int best = 1;
        double bv = 1e300;
        for (int kk = 1; kk <= n; ++kk) {
            const double v = (1.0 + (H[n] - H[n - kk]) / rate) / kk;
            if (v < bv) { bv = v; best = kk; }
        }
        *k_best = best;
    }
    return CODED_OK;
    CODED_GUARD_END
}

const char* coded_status_string(coded_status status) {
    switch (status) {
        case CODED_OK: return "CODED_OK";
        case CODED_ERR_ARG: return "CODED_ERR_ARG";
        case CODED_ERR_SHAPE: return "CODED_ERR_SHAPE";
        case CODED_ERR_TOO_FEW: return "CODED_ERR_TOO_FEW";
        case CODED_ERR_SINGULAR: return "CODED_ERR_SINGULAR";
        case CODED_ERR_HIP: return "CODED_ERR_HIP";
        case CODED_ERR_UNSUPPORTED: return "CODED_ERR_UNSUPPORTED";
    }
    return "unknown coded_status";
}

const char* coded_last_error(void) { return g_last_error.c_str(); }

const char* coded_version(void) { return "coded-mi355x 0.1.0 (gfx950)"; }

}  // extern "C"
