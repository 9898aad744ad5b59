// Host side of the straggler model: which k of the n simulated workers finish
// first in a given draw (Sec. III-B, eq. mds_coded; Sec. III-C).
//
// Worker i's mother-runtime sample is T0 = shift + E/rate with E = -ln U, U
// uniform on (0,1); its coded task is 1/k of the job, so it takes T0/k.  U is
// taken from a 64-bit word of the counter-based SplitMix64 generator (Steele,
// Lea, Flood, OOPSLA 2014): word = output number c of SplitMix64 seeded with
// `seed`, c = stream<<56 | draw<<16 | worker, and U = ((word>>11)+0.5)*2^-53.
// T0 falls as the word grows, so the k fastest workers are the k largest
// words: the set is chosen with integer comparisons only.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>

namespace coded_rng {

static constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
static constexpr uint64_t kRuntimeStream = 4;

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

uint64_t splitmix64_output(uint64_t seed, uint64_t index) {
    // After index+1 steps the generator's state is seed + (index+1)*gamma.
    return mix64(seed + (index + 1) * kGamma);
}

uint64_t runtime_word(uint64_t seed, uint64_t stream, uint64_t draw, uint64_t worker) {
    return splitmix64_output(seed, (stream << 56) | (draw << 16) | worker);
}

double draw_survivors(int n, int k, uint64_t seed, uint64_t draw, double shift, double rate, int32_t* out) {
    uint64_t words[256];
    int order[256];
    for (int i = 0; i < n; ++i) {
        words[i] = runtime_word(seed, kRuntimeStream, draw, static_cast<uint64_t>(i));
        order[i] = i;
    }
    // Fastest first: larger word, then lower index.
    std::sort(order, order + n, [&](int a, int b) {
        return words[a] != words[b] ? words[a] > words[b] : a < b;
    });
    for (int c = 0; c < k; ++c) out[c] = order[c];
    std::sort(out, out + k);
    const uint64_t wk = words[order[k - 1]];
    const double u = (static_cast<double>(wk >> 11) + 0.5) * 0x1.0p-53;
    return (shift + (-std::log(u)) / rate) / static_cast<double>(k);
}

void worker_times(int n, int k, uint64_t seed, uint64_t draw, double shift, double rate, double* t) {
    for (int i = 0; i < n; ++i) {
        const uint64_t w = runtime_word(seed, kRuntimeStream, draw, static_cast<uint64_t>(i));
        const double u = (static_cast<double>(w >> 11) + 0.5) * 0x1.0p-53;
        t[i] = (shift + (-std::log(u)) / rate) / static_cast<double>(k);
    }
}

double lambert_w_lower(double x) {
    // Halley's iteration on f(w) = w e^w - x, started from the branch-point
    // series near -1/e or from the asymptotic logarithmic form near 0.
    const double e = 2.718281828459045235;
    if (x <= -1.0 / e) return -1.0;
    double w;
    if (x < -0.25) {
        const double p = -std::sqrt(2.0 * (1.0 + e * x));
        w = -1.0 + p - p * p / 3.0;
    } else {
        const double lx = std::log(-x);
        w = lx - std::log(-lx);
    }
    for (int it = 0; it < 100; ++it) {
        const double ew = std::exp(w), f = w * ew - x, wp1 = w + 1.0;
        if (wp1 == 0.0) break;
        const double step = f / (ew * wp1 - (w + 2.0) * f / (2.0 * wp1));
        w -= step;
        if (std::fabs(step) <= 1e-15 * std::fabs(w)) break;
    }
    return w;
}

}  // namespace coded_rng
