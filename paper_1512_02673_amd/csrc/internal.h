// Internal declarations shared by the host glue and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/coded.h"

struct coded_code {
    int32_t n = 0, k = 0, planes = 2;
    bool lo_bf16 = false;      // CODED_PLANES_LO_BF16: planes == 2, the lo plane stored as bfloat16 for fp32 inputs
    std::vector<double> G;     // host copy, n*k row-major
    double* dG = nullptr;      // device copy, n*k row-major (in the caller's buffer)
    float* dPf = nullptr;      // device copy of the parity rows P ((n-k) x k) in fp32 (same buffer)
    int device = 0;
    int compute_units = 0;     // of the device, for kernels that place one workgroup per unit
    // Created on first use by coded_straggler_matmul, released with the code:
    // default-priority streams the worker products run on, one completion
    // event per worker, and an event that orders them after the caller.
    std::vector<hipStream_t> worker_streams;
    std::vector<hipEvent_t> worker_events;
    hipEvent_t start_event = nullptr;
};

namespace coded {

constexpr int kMaxN = CODED_MAX_N;

// Status plumbing: every API function funnels its failures through fail().
coded_status fail(coded_status st, const std::string& msg);
coded_status hip_fail(hipError_t e, const char* what);

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------- encode
struct EncodeArgs {
    const void* A;        // q x r, row stride lda (f32 or bf16 bits)
    void* parity;         // planes x (n-k) x qb x r
    const double* G;      // device n x k
    int64_t q, r, lda, qb;
    int32_t n, k, planes;
    int32_t lo_bf16;      // fp32 with planes == 2: lo plane stored as bfloat16
};
hipError_t launch_encode_f32(const EncodeArgs& a, hipStream_t st);
hipError_t launch_encode_bf16(const EncodeArgs& a, hipStream_t st);

// ---------------------------------------------------------------- workers
struct WorkerArgs {
    const void* A;        // q x r, row stride lda
    const void* parity;   // planes x (n-k) x qb x r
    const void* X;        // r x s, row stride ldx
    void* Y;              // n x qb x s
    int64_t q, r, lda, qb, s, ldx;
    int32_t n, k, planes;
    int32_t y_f64;        // 1: Y is fp64, 0: Y is fp32
    int32_t n_sys, n_par; // active systematic / parity workers
    void* xt;             // bf16 only: scratch for X transposed (s x r), or null
    int32_t xt_ready;     // bf16 only: xt already holds X transposed (skip the transpose)
    int32_t lo_bf16;      // fp32 with planes == 2: the lo plane is bfloat16 (after the fp32 hi plane)
    uint8_t sys_ids[kMaxN];
    uint8_t par_ids[kMaxN];
};
hipError_t launch_worker_f32(const WorkerArgs& a, hipStream_t st);
// fp32 with s > 1 on the fp64 matrix cores (worker_f32_mfma.hip); supported
// when r and lda are multiples of 4, 0 < r <= 2^30 and A, parity are 16-byte
// aligned.
bool gemm_f32_mfma_supported(const WorkerArgs& a);
hipError_t launch_gemm_f32_mfma(const WorkerArgs& a, hipStream_t st);
hipError_t launch_worker_bf16(const WorkerArgs& a, hipStream_t st);
// bf16: X (r x s, row stride ldx) transposed into a.xt.
hipError_t launch_transpose_x_bf16(const WorkerArgs& a, hipStream_t st);
// Bytes of the bf16 worker workspace (X transposed), 256-byte aligned.
int64_t worker_workspace_bytes_bf16(int64_t r, int64_t s);

// ---------------------------------------------------------------- fused encode + workers (bf16)
struct FusedArgs {
    const uint16_t* A;    // q x r bf16, row stride lda
    uint16_t* parity;     // 2 planes x (n-k) x qb x r, written
    const uint16_t* xt;   // X^T, s x r (s = 64)
    float* Y;             // n x qb x 64, written (zero-filled, then accumulated)
    const float* P;       // device (n-k) x k parity coefficients (bf16 values)
    int64_t q, r, lda, qb;
    int32_t n, k;
    int64_t stages = 0, units = 0, per = 0, clean_tiles = 0;   // set by the launcher
};
bool fused_bf16_supported(int n, int k, int planes, int64_t r, int64_t lda);
hipError_t launch_fused_bf16(FusedArgs a, bool products, int compute_units, hipStream_t st);

// ---------------------------------------------------------------- decode
// One survivor set passed by value (worker indices < 128 fit in a byte;
// packed four to a word so the kernel can pick them out of its arguments).
struct DecodeSet {
    uint32_t packed[kMaxN / 4];
};
struct DecodeArgs {
    const double* G;      // device n x k
    const void* Y;        // n x qb x s
    float* out;           // batch x (q x s, row stride ldo), set stride out_stride
    int32_t* info;        // batch
    const int32_t* sets;  // device batch x k, or null when `single` is used
    int64_t q, qb, s, ldo, out_stride;
    int32_t n, k, batch, y_f64;
    // Epilogue: out = alpha * decoded + beta * c (c: same layout as out, or
    // null for out = decoded).  c may alias out.
    const float* c = nullptr;
    double alpha = 1.0, beta = 0.0;
};
// LDS bytes of the decode kernel's matrices for k survivors and at most mmax
// missing blocks; launch_decode sizes its dynamic LDS with it.
size_t decode_lds_bytes(int k, int mmax);
hipError_t launch_decode(const DecodeArgs& a, const DecodeSet* single, int mmax, hipStream_t st);

// ---------------------------------------------------------------- transpose
hipError_t launch_transpose_f32(const float* A, int64_t q, int64_t r, int64_t lda, float* AT, int64_t ldat,
                                hipStream_t st);

// ---------------------------------------------------------------- coded shuffling
hipError_t launch_shuffle_encode(const float* A, int64_t q, int64_t r, int64_t lda, const int64_t* off,
                                 const int32_t* rows, int64_t msgs, int64_t terms, float* M, int64_t ldm,
                                 hipStream_t st);
hipError_t launch_shuffle_decode(const float* A, int64_t q, int64_t r, int64_t lda, const float* M, int64_t ldm,
                                 const int64_t* off, const int32_t* rows, const int32_t* msg, int64_t msgs,
                                 int64_t terms, float* out, int64_t ldo, hipStream_t st);

// ---------------------------------------------------------------- static scratch
// Device address of the library's static scratch array on the current device
// (CODED_NOALLOC_SCRATCH_BYTES bytes, looked up once per device).
coded_status static_scratch(void** out);

// ---------------------------------------------------------------- runtime model
hipError_t launch_runtime_sim(int n, int k, uint64_t seed, uint64_t first, int64_t count, double shift, double rate,
                              double* t_uncoded, double* t_repetition, double* t_mds, hipStream_t st);

}  // namespace coded

// Host runtime model (survivors.cpp); plain C++, no device code.
namespace coded_rng {
uint64_t splitmix64_output(uint64_t seed, uint64_t index);
uint64_t runtime_word(uint64_t seed, uint64_t stream, uint64_t draw, uint64_t worker);
// Survivors of one draw: k worker indices ascending; returns T_(k).
double draw_survivors(int n, int k, uint64_t seed, uint64_t draw, double shift, double rate, int32_t* out);
// Task times of the n workers of one draw: t[i] = (shift - ln U_i / rate) / k.
void worker_times(int n, int k, uint64_t seed, uint64_t draw, double shift, double rate, double* t);
// W_{-1}(x) for -1/e <= x < 0 (lower real branch of Lambert W).
double lambert_w_lower(double x);
}  // namespace coded_rng
