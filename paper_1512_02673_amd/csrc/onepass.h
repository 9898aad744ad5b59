// The whole coded product of a small fp32 problem with one column (encode
// unless the planes are stored, all n worker products, the decode) in one
// launch: block row t of every output depends on block row t of the k data
// blocks only.
#pragma once
#include "internal.h"

namespace coded {

constexpr int kOnePassMaxN = 16;
struct OnePassArgs {
    const float* A;       // q x r, row stride lda
    float* parity;        // planes x (n-k) x qb x r: written when encode, read otherwise
    const float* x;       // r
    double* Y;            // n x qb: every worker's product
    float* out;           // q values, stride ldo
    int32_t* info;        // 1
    const double* G;      // device n x k
    DecodeSet set;        // the k survivors, checked on the host
    int64_t q, r, lda, qb, ldo;
    int32_t n, k, planes, encode;
    int32_t missing;      // survivors at or past k (the blocks to solve for), from the same set
};
bool onepass_supported(int n, int k, int64_t q, int64_t r, int64_t lda, const void* A, const void* parity,
                       const void* x);
hipError_t launch_onepass_f32(const OnePassArgs& a, hipStream_t st);

}  // namespace coded
