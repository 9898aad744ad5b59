// Coded shuffling (Sec. IV): the master's state and transmission plan.
//
// Rows are partitioned among n workers before every iteration; worker i's
// cache C_i holds its S_i plus (s - q/n) more rows.  A row's cache signature
// is the set of workers caching it (bit i: worker i).  For the next
// partition, a row that worker i needs and lacks, with signature J, belongs
// to the multicast message of the group I = J + {i} (Algorithm 1: it lies in
// S_i cap C~_{I - i}); each member's rows of a group are listed in increasing
// row order and the group's message rows sum the members' j-th rows, zero
// padded to the longest list.  Every term of a message is one row that one
// worker lacks, so the decode of that term is its message minus the others.
//
// Random draws use the counter-based SplitMix64 (Steele, Lea, Flood, OOPSLA
// 2014): the partition of iteration t ranks rows by the stream-8 word of
// (t, row) and deals them out q/n at a time; the cache rule of iteration t
// keeps, for worker i, the rows of (old C_i minus new S_i) with the smallest
// stream-9 words of (t, row, i).  The first caches are that rule applied to
// the whole data set.
#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

#include "internal.h"

struct coded_shuffle {
    int32_t n = 0;
    int64_t q = 0, cache_rows = 0, t = 0;
    uint64_t seed = 0;
    std::vector<int32_t> assign;   // S^t: worker of each row
    std::vector<uint64_t> sig;     // C^t: cache signature of each row
    bool planned = false;          // a plan for iteration t+1 is pending
    std::vector<int32_t> next_assign;
    std::vector<int64_t> enc_off;
    std::vector<int32_t> enc_rows, term_worker, term_msg;
};

namespace coded {
namespace {

constexpr uint64_t kPartitionStream = 8;
constexpr uint64_t kCacheStream = 9;

std::vector<int32_t> partition(int n, int64_t q, uint64_t seed, int64_t t) {
    std::vector<std::pair<uint64_t, int64_t>> keyed(q);
    for (int64_t r = 0; r < q; ++r)
        keyed[r] = {coded_rng::splitmix64_output(seed, (kPartitionStream << 56) | (static_cast<uint64_t>(t) << 40) |
                                                           static_cast<uint64_t>(r)),
                    r};
    std::sort(keyed.begin(), keyed.end());
    std::vector<int32_t> assign(q);
    const int64_t per = q / n;
    for (int64_t p = 0; p < q; ++p) assign[keyed[p].second] = static_cast<int32_t>(p / per);
    return assign;
}

// The cache rule of iteration t: worker i keeps its S_i and (s - q/n) rows of
// (old cache minus S_i), those with the smallest stream-9 words.
std::vector<uint64_t> apply_cache_rule(const coded_shuffle& st, int64_t t, const std::vector<int32_t>& assign,
                                       const std::vector<uint64_t>& old_sig) {
    const int64_t q = st.q, extra = st.cache_rows - st.q / st.n;
    std::vector<uint64_t> sig(q, 0);
    for (int64_t r = 0; r < q; ++r) sig[r] |= uint64_t{1} << assign[r];
    std::vector<std::pair<uint64_t, int64_t>> pool;
    for (int i = 0; i < st.n; ++i) {
        pool.clear();
        for (int64_t r = 0; r < q; ++r)
            if (((old_sig[r] >> i) & 1u) && assign[r] != i)
                pool.push_back({coded_rng::splitmix64_output(
                                    st.seed, (kCacheStream << 56) | (static_cast<uint64_t>(t) << 40) |
                                                 (static_cast<uint64_t>(r) << 6) | static_cast<uint64_t>(i)),
                                r});
        const int64_t take = std::min<int64_t>(extra, static_cast<int64_t>(pool.size()));
        std::nth_element(pool.begin(), pool.begin() + take, pool.end());
        for (int64_t j = 0; j < take; ++j) sig[pool[j].second] |= uint64_t{1} << i;
    }
    return sig;
}

}  // namespace
}  // namespace coded

using namespace coded;

coded_status coded_shuffle_create(int32_t n, int64_t q, int64_t cache_rows, uint64_t seed, coded_shuffle** out) {
    try {
        if (!out) return fail(CODED_ERR_ARG, "out is NULL");
        *out = nullptr;
        if (n < 1 || n > 64) return fail(CODED_ERR_ARG, "need 1 <= n <= 64 workers");
        if (q < n || q % n) return fail(CODED_ERR_SHAPE, "q must be a positive multiple of n");
        if (q >= (int64_t{1} << 31)) return fail(CODED_ERR_SHAPE, "q must be below 2^31");
        if (cache_rows < q / n || cache_rows > q) return fail(CODED_ERR_ARG, "need q/n <= cache_rows <= q");
        auto* st = new coded_shuffle;
        st->n = n;
        st->q = q;
        st->cache_rows = cache_rows;
        st->seed = seed;
        st->t = 0;
        st->assign = partition(n, q, seed, 0);
        const uint64_t all = n == 64 ? ~uint64_t{0} : (uint64_t{1} << n) - 1;
        st->sig = apply_cache_rule(*st, 0, st->assign, std::vector<uint64_t>(q, all));
        *out = st;
        return CODED_OK;
    } catch (const std::bad_alloc&) {
        return fail(CODED_ERR_ARG, "host allocation failed");
    } catch (...) {
        return fail(CODED_ERR_ARG, "unexpected host exception");
    }
}

coded_status coded_shuffle_destroy(coded_shuffle* st) {
    delete st;
    return CODED_OK;
}

coded_status coded_shuffle_state(const coded_shuffle* st, int64_t* t, int32_t* assign, uint64_t* cache_sig) {
    if (!st) return fail(CODED_ERR_ARG, "shuffle state is NULL");
    if (t) *t = st->t;
    if (assign) std::copy(st->assign.begin(), st->assign.end(), assign);
    if (cache_sig) std::copy(st->sig.begin(), st->sig.end(), cache_sig);
    return CODED_OK;
}

coded_status coded_shuffle_plan(coded_shuffle* st, int64_t* coded_rows, int64_t* terms) {
    try {
        if (!st) return fail(CODED_ERR_ARG, "shuffle state is NULL");
        if (st->t + 1 >= (int64_t{1} << 16)) return fail(CODED_ERR_ARG, "at most 65535 iterations");
        st->planned = false;
        st->next_assign = partition(st->n, st->q, st->seed, st->t + 1);
        struct Entry {
            uint64_t key;
            int32_t worker;
            int64_t row;
        };
        std::vector<Entry> need;
        for (int64_t r = 0; r < st->q; ++r) {
            const int i = st->next_assign[r];
            if (!((st->sig[r] >> i) & 1u)) need.push_back({st->sig[r] | (uint64_t{1} << i), i, r});
        }
        std::sort(need.begin(), need.end(), [](const Entry& a, const Entry& b) {
            if (a.key != b.key) return a.key < b.key;
            if (a.worker != b.worker) return a.worker < b.worker;
            return a.row < b.row;
        });
        st->enc_off.assign(1, 0);
        st->enc_rows.clear();
        st->term_worker.clear();
        st->term_msg.clear();
        int64_t m = 0;
        for (size_t g0 = 0; g0 < need.size();) {
            size_t g1 = g0;
            while (g1 < need.size() && need[g1].key == need[g0].key) ++g1;
            // members' runs inside the group [g0, g1)
            std::vector<std::pair<size_t, size_t>> runs;
            size_t longest = 0;
            for (size_t a = g0; a < g1;) {
                size_t b = a;
                while (b < g1 && need[b].worker == need[a].worker) ++b;
                runs.push_back({a, b});
                longest = std::max(longest, b - a);
                a = b;
            }
            for (size_t j = 0; j < longest; ++j) {
                for (const auto& run : runs) {
                    if (run.first + j < run.second) {
                        const Entry& e = need[run.first + j];
                        st->enc_rows.push_back(static_cast<int32_t>(e.row));
                        st->term_worker.push_back(e.worker);
                        st->term_msg.push_back(static_cast<int32_t>(m));
                    }
                }
                st->enc_off.push_back(static_cast<int64_t>(st->enc_rows.size()));
                ++m;
            }
            g0 = g1;
        }
        st->planned = true;
        if (coded_rows) *coded_rows = m;
        if (terms) *terms = static_cast<int64_t>(st->enc_rows.size());
        return CODED_OK;
    } catch (const std::bad_alloc&) {
        return fail(CODED_ERR_ARG, "host allocation failed");
    } catch (...) {
        return fail(CODED_ERR_ARG, "unexpected host exception");
    }
}

coded_status coded_shuffle_tables(const coded_shuffle* st, int64_t* enc_off, int32_t* enc_rows, int32_t* term_worker,
                                  int32_t* term_msg, int32_t* next_assign) {
    if (!st) return fail(CODED_ERR_ARG, "shuffle state is NULL");
    if (!st->planned) return fail(CODED_ERR_ARG, "no pending plan: call coded_shuffle_plan first");
    if (enc_off) std::copy(st->enc_off.begin(), st->enc_off.end(), enc_off);
    if (enc_rows) std::copy(st->enc_rows.begin(), st->enc_rows.end(), enc_rows);
    if (term_worker) std::copy(st->term_worker.begin(), st->term_worker.end(), term_worker);
    if (term_msg) std::copy(st->term_msg.begin(), st->term_msg.end(), term_msg);
    if (next_assign) std::copy(st->next_assign.begin(), st->next_assign.end(), next_assign);
    return CODED_OK;
}

coded_status coded_shuffle_commit(coded_shuffle* st) {
    try {
        if (!st) return fail(CODED_ERR_ARG, "shuffle state is NULL");
        if (!st->planned) return fail(CODED_ERR_ARG, "no pending plan: call coded_shuffle_plan first");
        st->sig = apply_cache_rule(*st, st->t + 1, st->next_assign, st->sig);
        st->assign.swap(st->next_assign);
        st->t += 1;
        st->planned = false;
        return CODED_OK;
    } catch (const std::bad_alloc&) {
        return fail(CODED_ERR_ARG, "host allocation failed");
    } catch (...) {
        return fail(CODED_ERR_ARG, "unexpected host exception");
    }
}

coded_status coded_shuffle_encode(const float* A, int64_t q, int64_t r, int64_t lda, const int64_t* enc_off,
                                  const int32_t* enc_rows, int64_t coded_rows, int64_t terms, float* M, int64_t ldm,
                                  void* stream) {
    if (q < 0 || r < 0 || coded_rows < 0 || terms < 0) return fail(CODED_ERR_SHAPE, "sizes must be >= 0");
    if (lda < std::max<int64_t>(r, 1) || ldm < std::max<int64_t>(r, 1)) return fail(CODED_ERR_SHAPE, "bad lda / ldm");
    if (coded_rows > 0 && r > 0 && (!A || !enc_off || !enc_rows || !M)) return fail(CODED_ERR_ARG, "NULL pointer");
    hipError_t e = launch_shuffle_encode(A, q, r, lda, enc_off, enc_rows, coded_rows, terms, M, ldm,
                                         static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "shuffle encode launch");
    return CODED_OK;
}

coded_status coded_shuffle_decode(const float* A, int64_t q, int64_t r, int64_t lda, const float* M, int64_t ldm,
                                  const int64_t* enc_off, const int32_t* enc_rows, const int32_t* term_msg,
                                  int64_t coded_rows, int64_t terms, float* out, int64_t ldo, void* stream) {
    if (q < 0 || r < 0 || coded_rows < 0 || terms < 0) return fail(CODED_ERR_SHAPE, "sizes must be >= 0");
    if (lda < std::max<int64_t>(r, 1) || ldm < std::max<int64_t>(r, 1) || ldo < std::max<int64_t>(r, 1))
        return fail(CODED_ERR_SHAPE, "bad lda / ldm / ldo");
    if (terms > 0 && r > 0 && (!A || !M || !enc_off || !enc_rows || !term_msg || !out))
        return fail(CODED_ERR_ARG, "NULL pointer");
    hipError_t e = launch_shuffle_decode(A, q, r, lda, M, ldm, enc_off, enc_rows, term_msg, coded_rows, terms, out, ldo,
                                         static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "shuffle decode launch");
    return CODED_OK;
}

