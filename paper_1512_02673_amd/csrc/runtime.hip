// Monte-Carlo of the runtime model (Sec. III-B to III-D): for each draw the
// n worker samples T0_i = shift - ln(U_i) / rate come from the counter-based
// SplitMix64 word of (draw, worker), as in the survivor draw, and the job's
// overall runtime is formed for three schemes from the same samples:
//   uncoded      n subtasks of T0/n, the slowest one (eq. uncoded);
//   repetition   k subtasks of T0/k, each on n/k consecutive workers, the
//                slowest task's fastest replica (eq. rep_coded);
//   MDS (n,k)    subtasks of T0/k, the k-th finisher (eq. mds_coded).
// T0 falls as the word grows, so every order statistic is taken on the
// integer words and only the selected word goes through the logarithm.
// One thread per draw; words live in registers for n <= 32 (loops unrolled
// over the register count, so no word is indexed at run time) and are
// recomputed for larger n.
#include "internal.h"

namespace coded {
namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kRuntimeStream = 4;

// SplitMix64 output of counter c is mix(seed + (c + 1) * gamma).  With the
// counter 4 << 56 | draw << 16 | worker (worker < 2^16, so the OR is a sum)
// the state is base(draw) + worker * gamma, modulo 2^64.
__device__ inline uint64_t mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ inline uint64_t base_of(uint64_t seed, uint64_t draw) {
    return seed + (((kRuntimeStream << 56) | (draw << 16)) + 1) * kGamma;
}

__device__ inline uint64_t word_of(uint64_t base, int worker) {
    return mix(base + static_cast<uint64_t>(worker) * kGamma);
}

__device__ inline double mother(uint64_t w, double shift, double rate) {
    const double u = (static_cast<double>(w >> 11) + 0.5) * 0x1.0p-53;
    return shift - log(u) / rate;
}

// "a finishes no later than b": larger word, then lower index.
__device__ inline bool before(uint64_t ua, int a, uint64_t ub, int b) { return ua > ub || (ua == ub && a < b); }

template <int NMAX>
__global__ __launch_bounds__(256) void runtime_sim_kernel(int n, int k, uint64_t seed, uint64_t first_draw, int64_t count,
                                                          double shift, double rate, double* t_unc, double* t_rep,
                                                          double* t_mds) {
    const int64_t d = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (d >= count) return;
    const uint64_t base = base_of(seed, first_draw + static_cast<uint64_t>(d));
    if constexpr (NMAX > 0) {
        // Words in registers: every loop runs over the compile-time NMAX with
        // uniform guards (i < n), so each register index is a constant.
        uint64_t u[NMAX];
#pragma unroll
        for (int i = 0; i < NMAX; ++i) u[i] = i < n ? word_of(base, i) : 0;
        if (t_unc) {
            // the slowest worker: the smallest word (ties: the higher index finishes later)
            int slow = 0;
            uint64_t us = u[0];
#pragma unroll
            for (int i = 1; i < NMAX; ++i)
                if (i < n && before(us, slow, u[i], i)) {
                    us = u[i];
                    slow = i;
                }
            t_unc[d] = mother(us, shift, rate) / n;
        }
        if (t_mds) {
            // the k-th finisher: the worker with exactly k-1 workers before it
            uint64_t uk = 0;
#pragma unroll
            for (int i = 0; i < NMAX; ++i) {
                if (i < n) {
                    int rank = 0;
#pragma unroll
                    for (int j = 0; j < NMAX; ++j)
                        if (j < n && j != i) rank += before(u[j], j, u[i], i) ? 1 : 0;
                    uk = rank == k - 1 ? u[i] : uk;
                }
            }
            t_mds[d] = mother(uk, shift, rate) / k;
        }
        if (t_rep) {
            // per task (n/k consecutive workers) the fastest replica, then the slowest task
            const int g = n / k;
            uint64_t worst = ~0ull, best = 0;
            int pos = 0;
#pragma unroll
            for (int i = 0; i < NMAX; ++i) {
                if (i < n) {
                    best = u[i] > best ? u[i] : best;
                    if (++pos == g) {
                        worst = best < worst ? best : worst;
                        best = 0;
                        pos = 0;
                    }
                }
            }
            t_rep[d] = mother(worst, shift, rate) / k;
        }
    } else {
        // n > 32: words recomputed where needed
        auto W = [&](int i) { return word_of(base, i); };
        if (t_unc) {
            int slow = 0;
            uint64_t us = W(0);
            for (int i = 1; i < n; ++i) {
                const uint64_t ui = W(i);
                if (before(us, slow, ui, i)) {
                    us = ui;
                    slow = i;
                }
            }
            t_unc[d] = mother(us, shift, rate) / n;
        }
        if (t_mds) {
            uint64_t uk = 0;
            for (int i = 0; i < n; ++i) {
                const uint64_t ui = W(i);
                int rank = 0;
                for (int j = 0; j < n; ++j) rank += j != i && before(W(j), j, ui, i);
                if (rank == k - 1) uk = ui;
            }
            t_mds[d] = mother(uk, shift, rate) / k;
        }
        if (t_rep) {
            const int g = n / k;
            uint64_t worst = ~0ull;
            for (int task = 0; task < k; ++task) {
                uint64_t best = 0;
                for (int j = 0; j < g; ++j) {
                    const uint64_t uj = W(task * g + j);
                    best = uj > best ? uj : best;
                }
                worst = best < worst ? best : worst;
            }
            t_rep[d] = mother(worst, shift, rate) / k;
        }
    }
}

template <int NMAX>
hipError_t launch_sim(int n, int k, uint64_t seed, uint64_t first, int64_t count, double shift, double rate,
                      double* tu, double* tr, double* tm, hipStream_t st) {
    const int64_t blocks = ceil_div(count, 256);
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(runtime_sim_kernel<NMAX>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, n, k, seed,
                       first, count, shift, rate, tu, tr, tm);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_runtime_sim(int n, int k, uint64_t seed, uint64_t first, int64_t count, double shift, double rate,
                              double* tu, double* tr, double* tm, hipStream_t st) {
    if (count == 0) return hipSuccess;
    if (n <= 8) return launch_sim<8>(n, k, seed, first, count, shift, rate, tu, tr, tm, st);
    if (n <= 12) return launch_sim<12>(n, k, seed, first, count, shift, rate, tu, tr, tm, st);
    if (n <= 16) return launch_sim<16>(n, k, seed, first, count, shift, rate, tu, tr, tm, st);
    if (n <= 24) return launch_sim<24>(n, k, seed, first, count, shift, rate, tu, tr, tm, st);
    if (n <= 32) return launch_sim<32>(n, k, seed, first, count, shift, rate, tu, tr, tm, st);
    return launch_sim<0>(n, k, seed, first, count, shift, rate, tu, tr, tm, st);
}

}  // namespace coded
