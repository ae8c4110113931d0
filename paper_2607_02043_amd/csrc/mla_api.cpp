// C ABI of libmlastep: argument checks, work planning and launches.
// The entry points and their contracts are declared in include/mla_step.h.
#include "mla_step.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <atomic>
#include <mutex>
#include <vector>

#include "mla_kernels.h"
#include "api_util.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(MLA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Compute units of the current device (cached per device ordinal).
int cu_count(int *status) {
    static std::mutex mu;
    static int cache[64] = {0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        *status = hip_fail(e, "hipGetDevice");
        return 0;
    }
    if (dev < 0 || dev >= 64) dev = 0;
    std::lock_guard<std::mutex> lk(mu);
    if (cache[dev] == 0) {
        int n = 0;
        e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess || n <= 0) {
            *status = hip_fail(e, "hipDeviceGetAttribute(multiProcessorCount)");
            return 0;
        }
        cache[dev] = n;
    }
    return cache[dev];
}

// Debug settings (mla_debug_set): check mode, first value from the
// environment variable MLASTEP_CHECK (read once), and the spin limit of the
// kernels' bounded waits.
std::atomic<int> &debug_value(int knob) {
    static std::atomic<int> v[MLA_DEBUG_COUNT] = {};
    static std::once_flag once;
    std::call_once(once, [] {
        const char *e = std::getenv("MLASTEP_CHECK");
        v[MLA_DEBUG_CHECK].store(e && std::atoi(e) != 0 ? 1 : 0);
        v[MLA_DEBUG_SPIN_LIMIT].store(mla::kSpinLimit);
        v[MLA_DEBUG_CHUNK_KEYS].store(0);
        v[MLA_DEBUG_WARM_PLAN].store(1);
        v[MLA_DEBUG_DEC_FIRST].store(-1);
    });
    return v[knob];
}

bool check_mode() { return debug_value(MLA_DEBUG_CHECK).load(std::memory_order_relaxed) != 0; }

int ilog2_exact(int v) {
    int l = 0;
    while ((1 << l) < v) ++l;
    return (1 << l) == v ? l : -1;
}

long long ceil_div_ll(long long a, long long b) { return (a + b - 1) / b; }

struct Shape {
    int R = 0;
    int T = 0;
    int log2_page = 0;
};

// Host checks shared by both entry points.
int check_batch(const mla_batch *b, Shape *sh) {
    g_err[0] = '\0';
    if (!b) return fail(MLA_ERR_INVALID_ARG, "batch is NULL");
    if (b->num_reqs < 0) return fail(MLA_ERR_INVALID_ARG, "num_reqs = %d < 0", b->num_reqs);
    sh->R = b->num_reqs;
    if (b->num_reqs == 0) return MLA_OK;
    const int lg = ilog2_exact(b->page_size);
    if (b->page_size < 1 || b->page_size > 1024 || lg < 0)
        return fail(MLA_ERR_UNSUPPORTED, "page_size = %d is not a power of two in [1, 1024]", b->page_size);
    sh->log2_page = lg;
    if (b->num_pages < 1) return fail(MLA_ERR_INVALID_ARG, "num_pages = %d < 1", b->num_pages);
    if (b->max_pages_per_req < 1)
        return fail(MLA_ERR_INVALID_ARG, "max_pages_per_req = %d < 1", b->max_pages_per_req);
    if (!b->q_lens || !b->prefix_lens) return fail(MLA_ERR_INVALID_ARG, "host q_lens / prefix_lens is NULL");
    if (!b->cu_q_dev || !b->prefix_lens_dev || !b->block_table_dev)
        return fail(MLA_ERR_INVALID_ARG, "a device batch array is NULL");
    const long long cap = (long long)b->max_pages_per_req * b->page_size;
    long long T = 0;
    for (int r = 0; r < b->num_reqs; ++r) {
        const long long c = b->q_lens[r], p = b->prefix_lens[r];
        if (c < 1) return fail(MLA_ERR_INVALID_ARG, "q_lens[%d] = %lld < 1", r, c);
        if (p < 0) return fail(MLA_ERR_INVALID_ARG, "prefix_lens[%d] = %lld < 0", r, p);
        if (p + c > cap)
            return fail(MLA_ERR_INVALID_ARG, "request %d: prefix %lld + q_len %lld exceeds the block table (%lld keys)",
                        r, p, c, cap);
        if (p + c > (1LL << 30)) return fail(MLA_ERR_INVALID_ARG, "request %d: more than 2^30 keys", r);
        T += c;
        if (T > (1LL << 30) / mla::kHeads) return fail(MLA_ERR_INVALID_ARG, "too many rows in the step");
    }
    sh->T = (int)T;
    return MLA_OK;
}

struct Plan {
    int ks_chunk = 0, n_chunk_items = 0;
    int n_dec_units = 0, dec_unit_tiles = 0, dec_total_tiles = 0, grid = 0, merge_hsplit = 1;
    int dec_first_wgs = 0;  // workgroups that take decode items before chunk items
    bool chunk_split = false, dec_split = false, chunk_rev = false;
    size_t off_chunk_o = 0, off_chunk_ml = 0, off_dec_o = 0, off_dec_ml = 0, bytes = 0;
    // what a warm start compares: the work of the batch the plan was made for
    double chunk_pairs = 0.0;  // query-key pairs of the chunk requests
    long long chunk_keys_max = 0;  // keys of the longest chunk request
    int n_chunk_reqs = 0, n_dec_reqs = 0;
    bool warm = false;  // key split and unit size taken from an earlier plan
    double est_us = 0.0;  // the cost model's finishing time of a full plan (0 when warm-started)
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Per-CU costs (us) used only to size the work items: calibrated so that
// the planner's choice of key split and decode unit size is close to the
// fastest measured one over a set of MI355X steps (small and large decode
// batches, chunks of 124 to 4096 tokens over prefixes up to 8192).
constexpr double kChunkTileUs = 2.0;    // one chunk tile: 8 tokens x 32 keys
constexpr double kChunkItemUs = 18.0;   // chunk item: lookup, queries, ring fill; epilogue stores
constexpr double kEmptyItemUs = 1.5;    // a chunk item past its block's causal limit
constexpr double kDecTileUs = 3.5;      // one decode tile of a unit (the two units of an item run side by side)
constexpr double kDecUnitUs = 8.0;      // decode item start-up
constexpr double kDecTileLoUs = 2.65;   // a decode tile when few workgroups stream (per-CU rate bound)
constexpr double kTwoQueueGain = 0.03;  // decode-first workgroups only for at least this much less time
constexpr double kTwoQueueMinUs = 5.0;  // and at least this many microseconds less
constexpr double kMergeGBs = 3000.0;    // partial rows written and merged, whole chip
constexpr double kMergeLaunchUs = 7.0;  // the merge launch itself, when any row is split
constexpr int kCounterBytes = 256;     // work-queue counters at the start of the workspace

struct DecReq {
    long long first_tile, tiles, p;
};

// Does a decode unit of S tiles respect the kernel's limits (segments and
// page-window entries per unit)?
bool dec_share_fits(const std::vector<DecReq> &reqs, long long total, long long S, int page_size,
                    long long min_tiles) {
    // a unit of S tiles touches at most S / min_tiles + 2 requests (min_tiles:
    // the shortest request's tiles) and, per request, at most its keys /
    // page_size + 2 pages
    const long long segs = std::min(S, S / std::max(1LL, min_tiles) + 2);
    if (segs <= mla::kMaxDecSegments && S * mla::kKeysPerTile / page_size + 2 * segs <= mla::kPageWindow) return true;
    const int lg = __builtin_ctz((unsigned)page_size);  // page_size is a power of two
    size_t k = 0;
    for (long long R0 = 0; R0 < total; R0 += S) {
        const long long R1 = std::min(R0 + S, total);
        while (k < reqs.size() && reqs[k].first_tile + reqs[k].tiles <= R0) ++k;
        long long segs = 0, pages = 0;
        for (size_t j = k; j < reqs.size() && reqs[j].first_tile < R1; ++j) {
            const long long t0 = std::max(R0 - reqs[j].first_tile, 0LL);
            const long long t1 = std::min(R1 - reqs[j].first_tile, reqs[j].tiles);
            const long long k0 = t0 * mla::kKeysPerTile;
            const long long klast = std::min(t1 * mla::kKeysPerTile, reqs[j].p + 1) - 1;
            pages += (klast >> lg) - (k0 >> lg) + 1;
            ++segs;
        }
        if (segs > mla::kMaxDecSegments || pages > mla::kPageWindow) return false;
    }
    return true;
}

// Loads of the G workgroups after the chunk items, each item taken in queue
// order by the first free workgroup; `init` (G loads) is where the
// workgroups start, all at 0 when it is null.
std::vector<double> simulate_chunks(const std::vector<double> &items, int G, const std::vector<double> *init = nullptr) {
    // each item goes to the workgroup that finishes first (the root of a
    // min-heap, sifted down); from idle workgroups the first G items start
    // directly
    const size_t g = (size_t)G, n0 = init != nullptr ? 0 : std::min(g, items.size());
    std::vector<double> heap = init != nullptr ? *init : std::vector<double>(g, 0.0);
    for (size_t i = 0; i < n0; ++i) heap[i] = items[i];
    std::make_heap(heap.begin(), heap.end(), [](double x, double y) { return x > y; });
    for (size_t i = n0; i < items.size(); ++i) {
        const double v = heap[0] + items[i];
        size_t k = 0;
        for (;;) {
            size_t c = 2 * k + 1;
            if (c >= g) break;
            if (c + 1 < g && heap[c + 1] < heap[c]) ++c;
            if (heap[c] >= v) break;
            heap[k] = heap[c];
            k = c;
        }
        heap[k] = v;
    }
    return heap;
}

// Workgroup loads as runs of equal values, ascending, with the sum and the
// count of the loads up to and including each run.
struct LoadRun {
    double load;
    long long count;
    double sum_to;
    long long count_to;
};
std::vector<LoadRun> load_runs(std::vector<double> loads) {
    std::sort(loads.begin(), loads.end());
    std::vector<LoadRun> runs;
    for (double L : loads) {
        if (!runs.empty() && runs.back().load == L)
            ++runs.back().count;
        else
            runs.push_back(LoadRun{L, 1, 0.0, 0});
    }
    double sum = 0.0;
    long long cnt = 0;
    for (LoadRun &r : runs) {
        sum += r.load * (double)r.count;
        cnt += r.count;
        r.sum_to = sum;
        r.count_to = cnt;
    }
    return runs;
}

// The first run k at which pred(k) holds, pred being false up to some run and
// true from there on (the last run if it never holds): a binary search.
template <typename Pred>
size_t first_run(const std::vector<LoadRun> &runs, Pred pred) {
    size_t lo = 0, hi = runs.size() - 1;
    while (lo < hi) {
        const size_t mid = (lo + hi) / 2;
        if (pred(mid))
            hi = mid;
        else
            lo = mid + 1;
    }
    return lo;
}

// Water level of n units of cost u poured onto the workgroup loads: the t
// with sum over loads L < t of (t - L) = n u.  No schedule of the units
// finishes before it.
double water_level(const std::vector<LoadRun> &runs, long long n, double u) {
    if (runs.empty()) return 0.0;
    // the level over the loads up to run k, which only falls below the next
    // load once k reaches the answer
    auto level = [&](size_t k) { return (runs[k].sum_to + (double)n * u) / (double)runs[k].count_to; };
    return level(first_run(runs, [&](size_t k) { return k + 1 == runs.size() || level(k) <= runs[k + 1].load; }));
}

// A lower bound on the finishing time below.  A workgroup with load L has
// started at most (t - L) / u + 1 units by t >= L, so the last of the n units
// cannot start before the t at which that bound, summed over the loads, first
// reaches n (searched for over the segments between the sorted loads).
double fill_bound(const std::vector<LoadRun> &runs, long long n, double u) {
    if (n <= 0 || runs.empty()) return runs.empty() ? 0.0 : runs.back().load;
    auto start = [&](size_t k) {
        return std::max(runs[k].load, (runs[k].sum_to + (double)(n - runs[k].count_to) * u) / (double)runs[k].count_to);
    };
    const size_t k = first_run(runs, [&](size_t k) { return k + 1 == runs.size() || start(k) <= runs[k + 1].load; });
    return std::max(runs.back().load, start(k) + u);
}

// Finishing time when n equal units of cost u follow, each taken by the first
// free workgroup, on top of the workgroup loads.  The last unit starts at the
// smallest t with sum over loads L < t of ceil((t - L) / u) >= n, which lies
// in [level - u, level].  That sum is a step function of t: a run of loads L
// has started ceil((lo - L) / u) units by lo and one more just after each
// L + j u inside the interval (at most two such steps, the interval being
// one unit long), so t is the step at which the count reaches n.
double fill_units(const std::vector<LoadRun> &runs, long long n, double u) {
    const double mx = runs.empty() ? 0.0 : runs.back().load;
    if (n <= 0 || runs.empty()) return mx;
    const double level = water_level(runs, n, u);
    const double lo = std::max(0.0, level - u), hi = level, inv_u = 1.0 / u;
    struct Step {
        double t;
        long long count;
        int bucket;
    };
    // the steps are counted in equal buckets of [lo, hi) (bucket order is t
    // order); only the bucket where the count reaches n is sorted
    constexpr int kBuckets = 64;
    const double scale = hi > lo ? kBuckets / (hi - lo) : 0.0;
    long long hist[kBuckets] = {};
    thread_local std::vector<Step> steps;
    steps.clear();
    long long base = 0;  // units started by lo
    for (const LoadRun &r : runs) {
        if (r.load >= hi) break;
        long long j = 0;  // ceil((lo - L) / u), less a rounding margin
        if (r.load < lo) {
            const double x = (lo - r.load) * inv_u - 1e-9;
            j = (long long)x;
            j += (double)j < x;
        }
        base += r.count * j;
        for (double t = r.load + (double)j * u; t < hi; t += u) {
            const int k = std::min(kBuckets - 1, std::max(0, (int)((t - lo) * scale)));
            hist[k] += r.count;
            steps.push_back(Step{t, r.count, k});
        }
    }
    if (base >= n) return std::max(mx, lo + u);
    // the smallest step t with base + (units of the steps <= t) >= n
    long long need = n - base;
    int kb = 0;
    while (kb < kBuckets && need > hist[kb]) need -= hist[kb++];
    if (kb < kBuckets) {
        size_t m = 0;
        for (const Step &st : steps)
            if (st.bucket == kb) steps[m++] = st;
        std::sort(steps.begin(), steps.begin() + (std::ptrdiff_t)m, [](const Step &x, const Step &y) { return x.t < y.t; });
        for (size_t i = 0; i < m; ++i)
            if ((need -= steps[i].count) <= 0) return std::max(mx, steps[i].t + u);
    }
    return std::max(mx, hi + u);
}

// Work layout of one call.
//  * chunk requests -> items of (8 tokens) x (a range of keys): every block
//    of 8 query tokens (longest rows first) takes nks = ceil((p + c) /
//    ks_chunk) queue slots and cuts its causal keys klim into
//    ceil(klim / ks_chunk) equal ranges (multiples of 64 keys; the other
//    slots are empty items); ks_chunk is picked
//    from a closed-form estimate of the finishing time (work spread over the
//    CUs plus half the largest item) plus the merge of the partials a split
//    leaves.  Chunk requests are numbered from the last to the first when the
//    last one has the larger items, so that large items start first.
//  * decode requests -> one list of 32-key tiles cut into units of
//    dec_unit_tiles; the units fill the tail after the chunk items.
// The device recomputes the same mapping from the device copies of the
// lengths.  Cost: a closed form per request and candidate key split, then a
// queue simulation of the best one (and of the runner-up while its work
// bound can still win), with the decode fill of each unit size evaluated
// exactly until a lower bound rules the rest out.
int make_plan_uncached(const mla_batch *b, const Shape &sh, int ncu, mla::ChunkRoute route, Plan *pl,
                       const Plan *warm = nullptr) {
    const long long P = b->page_size;
    long long cap = ((long long)(mla::kPageWindow - 1) * P) / 64 * 64;  // keys per chunk item
    if (cap < 64) cap = 64;
    const int BM = mla::kChunkBlockTokens, KT = mla::kKeysPerTile;

    std::vector<DecReq> dec;
    std::vector<std::pair<long long, long long>> chunks;  // (p, c) of each chunk request, request order
    dec.reserve(sh.R);
    long long dec_total = 0;
    for (int r = 0; r < sh.R; ++r) {
        const long long c = b->q_lens[r], p = b->prefix_lens[r];
        if (c == 1) {
            const long long nt = ceil_div_ll(p + 1, KT);
            dec.push_back(DecReq{dec_total, nt, p});
            dec_total += nt;
        } else if (!route.multi_head(p, c)) {
            chunks.emplace_back(p, c);
        }
    }
    if (dec_total > (1LL << 30)) return fail(MLA_ERR_INVALID_ARG, "too many decode keys in the step");
    long long min_tiles = 1LL << 40;
    for (const DecReq &d : dec) min_tiles = std::min(min_tiles, d.tiles);
    const int G = std::max(1, ncu);
    const double row_bytes = (double)mla::kPartialFloats * 4.0;
    double chunk_pairs = 0.0;
    long long chunk_keys_max = 0;
    for (const auto &pc : chunks) {
        chunk_pairs += (double)pc.second * ((double)pc.first + 0.5 * (double)(pc.second + 1));
        chunk_keys_max = std::max(chunk_keys_max, pc.first + pc.second);
    }
    // large items first: number the chunk requests from the last one when
    // its items are the larger ones
    const bool rev = chunks.size() > 1 && chunks.back().first + chunks.back().second >
                                              chunks.front().first + chunks.front().second;

    // Warm start: a batch with as many chunk requests as an earlier plan's,
    // and within 1/16 of its decode requests, decode tiles, chunk pairs and
    // longest chunk (a serving step whose decode lengths grew by a token, or
    // that gained or lost a few requests), keeps that plan's key split and
    // unit size when the unit still fits the kernel's limits; only the
    // derived counts below are recomputed.
    if (warm != nullptr) {
        const auto near = [](double x, double y) { return std::fabs(x - y) <= y / 16.0; };
        const long long U = warm->dec_unit_tiles;
        const bool ok = (int)chunks.size() == warm->n_chunk_reqs && near((double)dec.size(), warm->n_dec_reqs) &&
                        near((double)dec_total, (double)warm->dec_total_tiles) && near(chunk_pairs, warm->chunk_pairs) &&
                        near((double)chunk_keys_max, (double)warm->chunk_keys_max) &&
                        warm->ks_chunk >= 64 && warm->ks_chunk <= cap &&
                        (dec_total == 0 || (U >= 1 && U <= dec_total && dec_share_fits(dec, dec_total, U, (int)P, min_tiles)));
        if (!ok) warm = nullptr;
    }

    // Chunk work for a key split ks: total cost, largest item, items, and
    // the partial rows a split adds (each part written, then read back by the
    // merge, whose merged row replaces the direct store).  Per
    // request in closed form: the blocks' causal limits p + 8 (rb + 1) form
    // an arithmetic sequence (the last block ends at p + c).
    struct ChunkEst {
        double total = 0.0, max_item = 0.0, merge_us = 0.0;
        long long items = 0;
        bool split = false;
    };
    auto chunk_est = [&](long long ks) {
        ChunkEst e;
        double split_rows = 0.0;
        for (const auto &pc : chunks) {
            const long long p = pc.first, c = pc.second;
            const long long nrb = ceil_div_ll(c, BM), nks = ceil_div_ll(p + c, ks);
            // sum over blocks of their tiles: limits p + 8, p + 16, .., p + c
            const double keys = (double)nrb * (double)p + 4.0 * (double)(nrb - 1) * (double)nrb + (double)c;
            const double tiles = keys / KT + 0.5 * (double)nrb * (double)nks;  // + rounding of each range
            e.total += tiles * kChunkTileUs + (double)(nrb * nks) * kChunkItemUs;
            const long long kp = ceil_div_ll(ceil_div_ll(p + c, nks), 64) * 64;
            e.max_item = std::max(e.max_item, kChunkItemUs + kChunkTileUs * (double)ceil_div_ll(kp, KT));
            if (nks > 1) {
                // rows of the blocks whose keys span more than one range
                const double first_split = std::max(0.0, (double)(ks - p) / BM);  // blocks within ks keys
                split_rows += (double)(2 * nks) * std::max(0.0, (double)c - first_split * BM);
            }
            e.items += nrb * nks;
        }
        e.merge_us = split_rows * row_bytes / (kMergeGBs * 1e3);
        e.split = split_rows > 0.0;
        return e;
    };
    // Chunk items of key split ks in device queue order (requests forward or
    // from the last, blocks longest first, nks ranges per block; an empty
    // range still takes a queue slot), as costs.
    auto chunk_items = [&](long long ks, bool rev, std::vector<double> &items) {
        // 32-bit arithmetic: keys per request stay below 2^30
        const uint32_t k32 = (uint32_t)ks;
        size_t n = 0;
        for (const auto &pc : chunks)
            n += (size_t)(((uint32_t)pc.second + BM - 1) / BM) * (((uint32_t)(pc.first + pc.second) + k32 - 1) / k32);
        items.resize(n);
        double *out = items.data();
        for (size_t i = 0; i < chunks.size(); ++i) {
            const auto &pc = chunks[rev ? chunks.size() - 1 - i : i];
            const uint32_t p = (uint32_t)pc.first, c = (uint32_t)pc.second;
            const uint32_t nrb = (c + BM - 1) / BM, nks = (p + c + k32 - 1) / k32;
            // klim falls by at most BM keys a block, so nr = ceil(klim / ks)
            // and q = ceil(klim / (64 nr)) (kp = 64 q) are stepped down
            // rather than divided out again
            uint32_t nr = 0, q = 0;
            for (uint32_t rb = nrb; rb-- > 0;) {
                const uint32_t klim = p + std::min(c, (rb + 1) * (uint32_t)BM);
                if (nr == 0 || (nr - 1) * k32 >= klim) {
                    nr = (klim + k32 - 1) / k32;
                    q = (klim + 64 * nr - 1) / (64 * nr);
                }
                while ((q - 1) * 64 * nr >= klim) --q;
                const uint32_t kp = 64 * q;
                // ranges of kp keys, the last one shorter, then empty slots
                uint32_t full = nr;  // floor(klim / kp): nr, or nr - 1 when ks is a multiple of 64
                while (full * kp > klim) --full;
                const uint32_t rest = klim - full * kp;
                out = std::fill_n(out, full, kChunkItemUs + kChunkTileUs * (double)((kp + KT - 1) / KT));
                if (rest > 0) *out++ = kChunkItemUs + kChunkTileUs * (double)((rest + KT - 1) / KT);
                out = std::fill_n(out, nks - full - (rest > 0), kEmptyItemUs);
            }
        }
    };
    // A decode unit size made smaller until it respects the kernel's
    // per-unit segment and page-window limits (0 if even one tile does not).
    auto fit_unit = [&](long long U) {
        U = std::max(1LL, std::min(U, dec_total));
        bool fits;
        while (!(fits = dec_share_fits(dec, dec_total, U, (int)P, min_tiles)) && U > 1) U = std::max(1LL, U * 3 / 4);
        return fits ? U : 0LL;
    };
    // Decode units: the candidate sizes (tiles) that respect those limits.
    std::vector<long long> units;
    if (dec_total > 0 && warm == nullptr) {
        const long long forced_unit = debug_value(MLA_DEBUG_DEC_UNIT).load(std::memory_order_relaxed);
        std::vector<long long> cands{8, 16, 32, 64, ceil_div_ll(dec_total, 3LL * G), ceil_div_ll(dec_total, 2LL * G),
                                     ceil_div_ll(dec_total, G)};
        if (forced_unit > 0) cands.assign(1, forced_unit);
        for (long long U : cands) {
            U = fit_unit(U);
            if (U > 0 && std::find(units.begin(), units.end(), U) == units.end()) units.push_back(U);
        }
        if (units.empty())
            return fail(MLA_ERR_UNSUPPORTED, "decode work does not fit the per-unit segment / page limits");
    }
    // Per unit size U: the work items (pairs of units), a unit's cost and the
    // merge of the request rows it splits.
    struct DecFill {
        long long n;
        double u, merge_us;
        bool split;
    };
    auto dec_fill = [&](long long U) {
        long long split_parts = 0;
        const uint32_t u32 = (uint32_t)U;  // tile indices stay below 2^30
        const uint64_t inv = (1ull << 32) / u32;
        auto unit_of = [&](uint32_t x) {  // x / U: x floor(2^32 / U) / 2^32 is short by at most one
            uint32_t q = (uint32_t)(((uint64_t)x * inv) >> 32);
            q += (q + 1) * u32 <= x;
            return q;
        };
        // the requests' tiles are contiguous: each one starts in the unit of
        // its predecessor's last tile or in the next one
        uint32_t first = 0;  // unit of the request's first tile
        for (const DecReq &d : dec) {
            const uint32_t l = (uint32_t)(d.first_tile + d.tiles - 1), last = unit_of(l);
            if (last > first) split_parts += 2 * (last - first + 1);  // each part written and read back
            first = last + ((last + 1) * u32 == l + 1);
        }
        return DecFill{ceil_div_ll(ceil_div_ll(dec_total, U), 2), kDecUnitUs + kDecTileUs * (double)U,
                       (double)split_parts * row_bytes / (kMergeGBs * 1e3), split_parts > 0};
    };

    // Key split: the closed-form estimate keeps the best candidate (and the
    // runner-up when within 10%), whose queue is then simulated (with the
    // decode units after it).
    long long ks_best = cap, U_best = units.empty() ? 1 : units.back(), dec_first = 0;
    const long long ks_forced = debug_value(MLA_DEBUG_CHUNK_KEYS).load(std::memory_order_relaxed);
    if (warm != nullptr) {
        ks_best = warm->ks_chunk;
        U_best = std::max(1, warm->dec_unit_tiles);
    } else {
        struct Cand {
            long long ks;
            double est, merge_us;
            bool split;
            ChunkEst e;
        };
        std::vector<Cand> cands;
        // the decode work fills the CUs after the chunk items: about
        // kDecTileUs / 2 per tile (the two units of an item run side by side)
        const double dec_work = 0.5 * kDecTileUs * (double)dec_total;
        if (!chunks.empty() && ks_forced > 0) {
            const ChunkEst e = chunk_est(std::min(ks_forced, cap));
            cands.push_back(Cand{std::min(ks_forced, cap), 0.0, e.merge_us, e.split, e});
        } else if (!chunks.empty()) {
            for (long long ks = 64;; ks *= 2) {
                const long long k = std::min(ks, cap);
                const ChunkEst e = chunk_est(k);
                if (e.items <= 8LL * G || k >= cap) {
                    const double tail = e.items <= G ? 0.0 : 0.5 * e.total / (double)e.items;
                    // (the merge launch is left out here: decode rows may
                    // need it anyway, which only the simulation below knows)
                    cands.push_back(Cand{k, std::max(e.max_item, (e.total + dec_work) / G + tail) + e.merge_us,
                                         e.merge_us, e.split, e});
                }
                if (k >= cap) break;
            }
            std::sort(cands.begin(), cands.end(), [](const Cand &x, const Cand &y) { return x.est < y.est; });
        } else {
            cands.push_back(Cand{cap, 0.0, 0.0, false, ChunkEst{}});
        }
        std::vector<DecFill> fills;
        double dec_min = dec_total > 0 ? 1e300 : 0.0;
        for (long long U : units) {
            fills.push_back(dec_fill(U));
            dec_min = std::min(dec_min, (double)fills.back().n * fills.back().u);
        }
        // merges of a candidate split and a unit size: their traffic and,
        // when any row is split, the merge launch
        auto merges = [](const Cand &cd, const DecFill &df) {
            return cd.merge_us + df.merge_us + ((cd.split || df.split) ? kMergeLaunchUs : 0.0);
        };
        double best = 1e300;
        size_t best_key = 0;
        std::vector<double> items;
        long long items_ks = -1;  // the key split `items` holds
        auto items_for = [&](long long ks) {
            if (ks != items_ks) chunk_items(ks, rev, items);
            items_ks = ks;
        };
        std::vector<std::pair<double, size_t>> order;
        // the best candidate is simulated, and the runner-up too when the
        // estimates are close
        const size_t n_sim = cands.size() > 1 && cands[1].est <= 1.1 * cands[0].est ? 2 : 1;
        for (size_t ci = 0; ci < n_sim; ++ci) {
            const Cand &cd = cands[ci];
            std::vector<LoadRun> loads{LoadRun{0.0, (long long)G, 0.0, (long long)G}};
            if (!chunks.empty()) {
                items_for(cd.ks);
                if (ci > 0) {
                    // the runner-up finishes no earlier than its largest item
                    // or its average load per workgroup (the least decode
                    // work and merge of any unit size added; a shade less,
                    // for rounding): not simulated if that cannot win
                    double sum = 0.0, largest = 0.0;
                    for (double c : items) {
                        sum += c;
                        largest = std::max(largest, c);
                    }
                    double merge_min = dec_total > 0 ? 1e300 : cd.merge_us + (cd.split ? kMergeLaunchUs : 0.0);
                    for (const DecFill &df : fills) merge_min = std::min(merge_min, merges(cd, df));
                    const double lower = std::max(largest, (sum + dec_min) / (double)G) + merge_min;
                    if (lower * (1.0 - 1e-9) >= best) continue;
                }
                loads = load_runs(simulate_chunks(items, G));
            }
            if (dec_total == 0) {
                const double t = loads.back().load + cd.merge_us + (cd.split ? kMergeLaunchUs : 0.0);
                if (t < best) {
                    best = t;
                    ks_best = cd.ks;
                }
                continue;
            }
            // sizes are tried by a lower bound on their finish, up to the
            // first that cannot beat the best one; among equal finishes the
            // earlier candidate and size win
            order.clear();
            for (size_t ui = 0; ui < units.size(); ++ui) {
                const DecFill &df = fills[ui];
                order.emplace_back(fill_bound(loads, df.n, df.u) + merges(cd, df), ui);
            }
            std::sort(order.begin(), order.end());
            for (const auto &o : order) {
                if (o.first > best) break;
                const DecFill &df = fills[o.second];
                const double t = fill_units(loads, df.n, df.u) + merges(cd, df);
                const size_t key = ci * units.size() + o.second;
                if (t < best || (t == best && key < best_key)) {
                    best = t;
                    best_key = key;
                    ks_best = cd.ks;
                    U_best = units[o.second];
                }
            }
        }
        // Decode-first workgroups: D of them stream the decode work, one item
        // each (units of ceil(T / 2D) tiles), while the others run the chunk
        // items; each moves to the chunk items when its decode item is done.
        // Fewer workgroups streaming at once get more of the memory
        // bandwidth each, down to a per-CU floor of kDecTileLoUs a tile, so
        // the decode work takes fewer workgroup-microseconds than at the
        // tail of the chunk-first schedule.  Closed form for every key split
        // and D, then a queue simulation of the best pair (and of the
        // runner-up when within 5%), taken when it beats the chunk-first
        // plan by kTwoQueueGain and kTwoQueueMinUs (or D is forced).
        const long long forced_first = debug_value(MLA_DEBUG_DEC_FIRST).load(std::memory_order_relaxed);
        if (!chunks.empty() && dec_total > 0 && forced_first != 0) {
            const long long forced_unit = debug_value(MLA_DEBUG_DEC_UNIT).load(std::memory_order_relaxed);
            std::vector<long long> firsts;
            if (forced_first > 0)
                firsts.push_back(std::min<long long>(forced_first, G));
            else
                for (int eighths = 2; eighths <= 7; ++eighths) firsts.push_back(std::max(1LL, (long long)G * eighths / 8));
            struct Two {
                long long D, U, n, Dp;
                double c, est;
                size_t ci;
                DecFill df;
            };
            Two top[2] = {};
            top[0].est = top[1].est = 1e300;
            for (long long D : firsts) {
                const long long U2 = fit_unit(forced_unit > 0 ? forced_unit : ceil_div_ll(dec_total, 2 * D));
                if (U2 == 0) continue;
                const DecFill df = dec_fill(U2);
                const long long Dp = std::min(D, df.n);  // workgroups that stream at once
                const double tile = std::max(kDecTileLoUs, kDecTileUs * (double)Dp / (double)G);
                const double c = kDecUnitUs + tile * (double)U2;
                const double t_first = c * (double)ceil_div_ll(df.n, Dp), dec_wg = c * (double)df.n;
                Two mine{D, U2, df.n, Dp, c, 1e300, 0, df};  // this D's best key split
                for (size_t ci = 0; ci < cands.size(); ++ci) {
                    const ChunkEst &e = cands[ci].e;
                    // without the tail, about the least any schedule takes:
                    // a pair that cannot beat the chunk-first plan is dropped
                    const double floor = std::max({e.max_item, t_first, (e.total + dec_wg) / G}) + merges(cands[ci], df);
                    if (forced_first <= 0 && floor >= best) continue;
                    const double tail = e.items <= G ? 0.0 : 0.5 * e.total / (double)e.items;
                    const double est = std::max(floor, (e.total + dec_wg) / G + tail + merges(cands[ci], df));
                    if (est < mine.est) {
                        mine.est = est;
                        mine.ci = ci;
                    }
                }
                if (mine.est < top[0].est) {
                    top[1] = top[0];
                    top[0] = mine;
                } else if (mine.est < top[1].est) {
                    top[1] = mine;
                }
            }
            double best_two = 1e300;
            const Two *pick = nullptr;
            for (const Two &tw : top) {
                if (tw.est >= 1e300 || (&tw != top && tw.est > 1.05 * top[0].est)) continue;
                // decode-first workgroup loads: the items dealt round the Dp
                // streaming ones
                std::vector<double> init((size_t)G, 0.0);
                for (long long j = 0; j < tw.Dp; ++j)
                    init[(size_t)j] = tw.c * (double)(tw.n / tw.Dp + (j < tw.n % tw.Dp ? 1 : 0));
                items_for(cands[tw.ci].ks);
                const std::vector<double> fin = simulate_chunks(items, G, &init);
                const double t = *std::max_element(fin.begin(), fin.end()) + merges(cands[tw.ci], tw.df);
                if (t < best_two) {
                    best_two = t;
                    pick = &tw;
                }
            }
            if (pick != nullptr && (forced_first > 0 || (best_two < best * (1.0 - kTwoQueueGain) &&
                                                         best_two < best - kTwoQueueMinUs))) {
                best = best_two;
                ks_best = cands[pick->ci].ks;
                U_best = pick->U;
                dec_first = pick->D;
            }
        }
        pl->est_us = best;
    }
    const long long U = dec_total > 0 ? U_best : 0;
    const long long n_units = dec_total > 0 ? ceil_div_ll(dec_total, U) : 0;
    long long nci = 0;
    for (const auto &pc : chunks) {
        const long long p = pc.first, c = pc.second;
        nci += ceil_div_ll(c, BM) * ceil_div_ll(p + c, ks_best);
        if (ceil_div_ll(p + c, ks_best) > 1) pl->chunk_split = true;
    }
    if (nci > (1LL << 27)) return fail(MLA_ERR_INVALID_ARG, "step needs too many work items");
    pl->chunk_rev = rev;
    pl->chunk_pairs = chunk_pairs;
    pl->chunk_keys_max = chunk_keys_max;
    pl->n_chunk_reqs = (int)chunks.size();
    pl->n_dec_reqs = (int)dec.size();
    pl->warm = warm != nullptr;
    pl->ks_chunk = (int)ks_best;
    pl->n_chunk_items = (int)nci;
    pl->n_dec_units = (int)ceil_div_ll(n_units, 2);  // a work item is a pair of units, one per wave group
    pl->dec_unit_tiles = (int)U;
    pl->dec_total_tiles = (int)dec_total;
    pl->grid = (int)std::min<long long>(G, nci + pl->n_dec_units);
    {
        const long long forced_first = debug_value(MLA_DEBUG_DEC_FIRST).load(std::memory_order_relaxed);
        const long long first = forced_first >= 0 ? forced_first : warm != nullptr ? warm->dec_first_wgs : dec_first;
        pl->dec_first_wgs = nci > 0 && dec_total > 0 ? (int)std::min<long long>(first, pl->grid) : 0;
    }
    long long max_parts = 1;
    for (const DecReq &d : dec) {
        const long long parts = (d.first_tile + d.tiles - 1) / U - d.first_tile / U + 1;
        if (parts > 1) pl->dec_split = true;
        max_parts = std::max(max_parts, parts);
    }
    // a row merged from many parts is spread over several workgroups
    pl->merge_hsplit = max_parts > 16 ? 8 : max_parts > 4 ? 4 : 1;
    size_t off = kCounterBytes;
    if (pl->chunk_split) {
        pl->off_chunk_o = off;
        off = align256(off + (size_t)nci * BM * mla::kPartialFloats * sizeof(float));
        pl->off_chunk_ml = off;
        off = align256(off + (size_t)nci * BM * mla::kPartialStats * sizeof(float));
    }
    if (pl->dec_split) {
        pl->off_dec_o = off;
        off = align256(off + (size_t)2 * n_units * mla::kPartialFloats * sizeof(float));
        pl->off_dec_ml = off;
        off = align256(off + (size_t)2 * n_units * mla::kPartialStats * sizeof(float));
    }
    pl->bytes = off;
    static const bool log_plan = std::getenv("MLA_PLAN_LOG") != nullptr;
    if (log_plan)
        std::fprintf(stderr,
                     "[mla plan] R=%d CUs=%d chunk items=%d (ks=%d keys, split=%d, rev=%d) decode units=%d x %d "
                     "tiles (total %lld, split=%d, merge x%d) grid=%d decode-first=%d workspace=%zu B%s\n",
                     sh.R, ncu, pl->n_chunk_items, pl->ks_chunk, (int)pl->chunk_split, (int)pl->chunk_rev,
                     pl->n_dec_units, pl->dec_unit_tiles, dec_total, (int)pl->dec_split, pl->merge_hsplit, pl->grid,
                     pl->dec_first_wgs, pl->bytes, pl->warm ? " (warm)" : "");
    return MLA_OK;
}

// The plan depends only on the host lengths, the page size and the CU count;
// the last one is kept per thread so a steady stream of identical steps
// plans once.  The last full plan is kept too, as the warm start of batches
// with nearly the same work (MLA_DEBUG_WARM_PLAN = 0 turns that off).
int make_plan(const mla_batch *b, const Shape &sh, Plan *pl, mla::ChunkRoute route = mla::kAbsorbAll) {
    *pl = Plan{};
    if (sh.R == 0) return MLA_OK;
    int st = MLA_OK;
    const int ncu = cu_count(&st);
    if (st != MLA_OK) return st;
    constexpr size_t kHdr = 9;
    const int32_t hdr[kHdr] = {b->page_size, ncu, sh.R, b->max_pages_per_req, route.min_rows, route.pair_keys,
                               debug_value(MLA_DEBUG_CHUNK_KEYS).load(std::memory_order_relaxed),
                               debug_value(MLA_DEBUG_DEC_UNIT).load(std::memory_order_relaxed),
                               debug_value(MLA_DEBUG_DEC_FIRST).load(std::memory_order_relaxed)};
    const size_t qbytes = (size_t)sh.R * sizeof(int32_t);
    // key: header, query lengths, prefix lengths
    thread_local std::vector<int32_t> key;
    thread_local int32_t anchor_hdr[kHdr] = {};
    thread_local bool have_anchor = false;
    thread_local Plan cached, anchor;
    if (key.size() == kHdr + 2 * (size_t)sh.R && std::memcmp(key.data(), hdr, sizeof hdr) == 0 &&
        std::memcmp(key.data() + kHdr, b->q_lens, qbytes) == 0 &&
        std::memcmp(key.data() + kHdr + sh.R, b->prefix_lens, qbytes) == 0) {
        *pl = cached;
        return MLA_OK;
    }
    // the anchor's header must match except for the request count
    const bool warm = debug_value(MLA_DEBUG_WARM_PLAN).load(std::memory_order_relaxed) != 0 && have_anchor &&
                      std::memcmp(anchor_hdr, hdr, 2 * sizeof(int32_t)) == 0 &&
                      std::memcmp(anchor_hdr + 3, hdr + 3, (kHdr - 3) * sizeof(int32_t)) == 0;
    st = make_plan_uncached(b, sh, ncu, route, pl, warm ? &anchor : nullptr);
    if (st != MLA_OK) return st;
    key.resize(kHdr + 2 * (size_t)sh.R);
    std::memcpy(key.data(), hdr, sizeof hdr);
    std::memcpy(key.data() + kHdr, b->q_lens, qbytes);
    std::memcpy(key.data() + kHdr + sh.R, b->prefix_lens, qbytes);
    cached = *pl;
    if (!pl->warm) {
        anchor = *pl;
        std::memcpy(anchor_hdr, hdr, sizeof hdr);
        have_anchor = true;
    }
    return MLA_OK;
}

// Check mode, before a launch: the device copies of the lengths equal the
// host ones, every block-table entry a request uses lies in the pool, and no
// slot a request writes is written or read by another request (or twice by
// one).  Synchronises the stream first (the device arrays may be produced on
// it).
int check_device_batch(const mla_batch *b, const Shape &sh, hipStream_t s) {
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "check mode: hipStreamSynchronize");
    const size_t R = sh.R, mp = b->max_pages_per_req;
    std::vector<int32_t> cu(R + 1), pre(R), bt(R * mp);
    if ((e = hipMemcpy(cu.data(), b->cu_q_dev, (R + 1) * 4, hipMemcpyDeviceToHost)) != hipSuccess ||
        (e = hipMemcpy(pre.data(), b->prefix_lens_dev, R * 4, hipMemcpyDeviceToHost)) != hipSuccess ||
        (e = hipMemcpy(bt.data(), b->block_table_dev, R * mp * 4, hipMemcpyDeviceToHost)) != hipSuccess)
        return hip_fail(e, "check mode: reading the device batch arrays");
    long long acc = 0;
    for (size_t r = 0; r <= R; ++r) {
        if (cu[r] != acc)
            return fail(MLA_ERR_INVALID_ARG, "check mode: cu_q_dev[%zu] = %d, the host q_lens give %lld", r, cu[r], acc);
        if (r < R) {
            if (pre[r] != b->prefix_lens[r])
                return fail(MLA_ERR_INVALID_ARG, "check mode: prefix_lens_dev[%zu] = %d, host prefix_lens %d", r, pre[r],
                            b->prefix_lens[r]);
            acc += b->q_lens[r];
        }
    }
    const long long P = b->page_size;
    for (size_t r = 0; r < R; ++r) {
        const long long n = ceil_div_ll((long long)b->prefix_lens[r] + b->q_lens[r], P);
        for (long long j = 0; j < n; ++j) {
            const int32_t id = bt[r * mp + j];
            if (id < 0 || id >= b->num_pages)
                return fail(MLA_ERR_INVALID_ARG,
                            "check mode: request %zu, logical page %lld: block-table entry %d outside [0, %d)", r, j, id,
                            b->num_pages);
        }
    }
    const long long slots = (long long)b->num_pages * P;
    if (slots <= (1LL << 28)) {
        std::vector<int32_t> writer(slots, -1);
        for (size_t r = 0; r < R; ++r)
            for (long long t = b->prefix_lens[r]; t < (long long)b->prefix_lens[r] + b->q_lens[r]; ++t) {
                const long long sl = (long long)bt[r * mp + t / P] * P + t % P;
                if (writer[sl] >= 0)
                    return fail(MLA_ERR_INVALID_ARG, "check mode: slot %lld is written by requests %d and %zu", sl,
                                writer[sl], r);
                writer[sl] = (int32_t)r;
            }
        for (size_t r = 0; r < R; ++r)
            for (long long t = 0; t < b->prefix_lens[r]; ++t) {
                const long long sl = (long long)bt[r * mp + t / P] * P + t % P;
                if (writer[sl] >= 0)
                    return fail(MLA_ERR_INVALID_ARG,
                                "check mode: request %zu reads key %lld from slot %lld, which request %d writes", r, t,
                                sl, writer[sl]);
            }
    }
    return MLA_OK;
}

// Check mode, after a launch: wait for the stream and turn the kernels' error
// flags into a status.
int check_after_launch(hipStream_t s, const char *what) {
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, what);
    int flags = 0;
    if ((e = mla::read_flags(&flags, true)) != hipSuccess) return hip_fail(e, "check mode: reading the device flags");
    if (flags & mla::kFlagWaitExpired)
        return fail(MLA_ERR_HIP, "check mode: %s: a bounded wait inside a kernel expired; results are undefined", what);
    if (flags & mla::kFlagBadPage)
        return fail(MLA_ERR_INVALID_ARG, "check mode: %s: a kernel met a block-table entry outside the pool", what);
    return MLA_OK;
}

}  // namespace

namespace mla {

int set_error(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int attn_workspace(const mla_batch *batch, size_t *bytes, ChunkRoute route) {
    *bytes = 0;
    Shape sh;
    int st = check_batch(batch, &sh);
    if (st != MLA_OK || sh.R == 0) return st;
    Plan pl;
    st = make_plan(batch, sh, &pl, route);
    if (st == MLA_OK) *bytes = pl.bytes;
    return st;
}

int batch_rows(const mla_batch *batch, int *num_rows) {
    Shape sh;
    const int st = check_batch(batch, &sh);
    *num_rows = st == MLA_OK ? sh.T : 0;
    return st;
}

}  // namespace mla

extern "C" {

int mla_abi_version(void) { return MLA_ABI_VERSION; }

const char *mla_last_error(void) { return g_err; }

size_t mixed_step_workspace_bytes(const mla_batch *batch) {
    Shape sh;
    if (check_batch(batch, &sh) != MLA_OK) return 0;
    Plan pl;
    if (make_plan(batch, sh, &pl) != MLA_OK) return 0;
    return pl.bytes;
}

int append_latent_kv(const mla_batch *batch, const uint16_t *new_latents, uint16_t *kv_cache, void *stream) {
    Shape sh;
    int st = check_batch(batch, &sh);
    if (st != MLA_OK || sh.R == 0) return st;
    if (!new_latents || !kv_cache) return fail(MLA_ERR_INVALID_ARG, "new_latents / kv_cache is NULL");
    if ((reinterpret_cast<uintptr_t>(new_latents) | reinterpret_cast<uintptr_t>(kv_cache)) & 15)
        return fail(MLA_ERR_INVALID_ARG, "new_latents / kv_cache must be 16-byte aligned");
    mla::AppendArgs a;
    a.src = new_latents;
    a.kv = kv_cache;
    a.cu_q = batch->cu_q_dev;
    a.prefix = batch->prefix_lens_dev;
    a.bt = batch->block_table_dev;
    a.num_reqs = sh.R;
    a.num_rows = sh.T;
    a.page_size = batch->page_size;
    a.log2_page = sh.log2_page;
    a.max_pages = batch->max_pages_per_req;
    a.num_pages = batch->num_pages;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    const bool chk = check_mode();
    if (chk && (st = check_device_batch(batch, sh, s)) != MLA_OK) return st;
    hipError_t e = mla::launch_append(a, s);
    if (e != hipSuccess) return hip_fail(e, "append kernel launch");
    return chk ? check_after_launch(s, "append_latent_kv") : MLA_OK;
}

int mla_device_flags(int32_t clear, int32_t *flags, void *stream) {
    g_err[0] = '\0';
    if (!flags) return fail(MLA_ERR_INVALID_ARG, "flags is NULL");
    *flags = 0;
    hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    int f = 0;
    if ((e = mla::read_flags(&f, clear != 0)) != hipSuccess) return hip_fail(e, "reading the device flags");
    *flags = f;
    return MLA_OK;
}

int mla_debug_set(int32_t knob, int32_t value) {
    g_err[0] = '\0';
    if (knob < 0 || knob >= MLA_DEBUG_COUNT) return fail(MLA_ERR_INVALID_ARG, "unknown debug knob %d", knob);
    if (knob == MLA_DEBUG_CHECK && value != 0 && value != 1)
        return fail(MLA_ERR_INVALID_ARG, "check mode must be 0 or 1, not %d", value);
    if (knob == MLA_DEBUG_SPIN_LIMIT && value < -1) return fail(MLA_ERR_INVALID_ARG, "spin limit %d < -1", value);
    if (knob == MLA_DEBUG_CHUNK_KEYS && (value < -1 || value % 64 != 0) && value != -1)
        return fail(MLA_ERR_INVALID_ARG, "chunk key split %d is not a non-negative multiple of 64", value);
    if (knob == MLA_DEBUG_WARM_PLAN && value != 0 && value != 1 && value != -1)
        return fail(MLA_ERR_INVALID_ARG, "warm planning must be 0 or 1, not %d", value);
    if (knob == MLA_DEBUG_DEC_UNIT && value < -1) return fail(MLA_ERR_INVALID_ARG, "decode unit size %d < -1", value);
    if (knob == MLA_DEBUG_DEC_FIRST && value < -1)
        return fail(MLA_ERR_INVALID_ARG, "decode-first workgroups %d < -1", value);
    const int dflt = knob == MLA_DEBUG_SPIN_LIMIT ? mla::kSpinLimit
                     : knob == MLA_DEBUG_WARM_PLAN ? 1
                     : knob == MLA_DEBUG_DEC_FIRST ? -1
                                                   : 0;
    debug_value(knob).store(value != -1 ? value : dflt);
    return MLA_OK;
}

}  // extern "C"

namespace {

// Shared by mixed_step_attn (new_latents == NULL) and mixed_step (fused append).
int attend(const mla_batch *batch, const uint16_t *q, const uint16_t *new_latents, uint16_t *kv_cache,
           float softmax_scale, void *out, int32_t out_dtype, float *lse, void *workspace, size_t workspace_bytes,
           void *stream, mla::ChunkRoute route = mla::kAbsorbAll) {
    Shape sh;
    int st = check_batch(batch, &sh);
    if (st != MLA_OK || sh.R == 0) return st;
    if (!q || !kv_cache || !out) return fail(MLA_ERR_INVALID_ARG, "q / kv_cache / out is NULL");
    if (reinterpret_cast<uintptr_t>(new_latents) & 15)
        return fail(MLA_ERR_INVALID_ARG, "new_latents must be 16-byte aligned");
    if (out_dtype != MLA_OUT_F32 && out_dtype != MLA_OUT_BF16)
        return fail(MLA_ERR_INVALID_ARG, "out_dtype = %d is neither MLA_OUT_F32 nor MLA_OUT_BF16", out_dtype);
    if (!std::isfinite(softmax_scale) || softmax_scale <= 0.f)
        return fail(MLA_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
    if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(kv_cache) | reinterpret_cast<uintptr_t>(out) |
         reinterpret_cast<uintptr_t>(workspace)) & 15)
        return fail(MLA_ERR_INVALID_ARG, "q / kv_cache / out / workspace must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(lse) & 3) return fail(MLA_ERR_INVALID_ARG, "lse must be 4-byte aligned");
    Plan pl;
    st = make_plan(batch, sh, &pl, route);
    if (st != MLA_OK) return st;
    if (pl.bytes > 0 && (!workspace || workspace_bytes < pl.bytes))
        return fail(MLA_ERR_WORKSPACE, "workspace of %zu bytes at %p; this batch needs %zu", workspace_bytes,
                    workspace, pl.bytes);
    mla::AttnArgs a;
    a.q = q;
    a.kv = kv_cache;
    a.new_kv = new_latents;
    a.kv_out = new_latents ? kv_cache : nullptr;
    a.cu_q = batch->cu_q_dev;
    a.prefix = batch->prefix_lens_dev;
    a.bt = batch->block_table_dev;
    a.out = out;
    a.lse = lse;
    char *ws = static_cast<char *>(workspace);
    a.ws_chunk_o = pl.chunk_split ? reinterpret_cast<float *>(ws + pl.off_chunk_o) : nullptr;
    a.ws_chunk_ml = pl.chunk_split ? reinterpret_cast<float *>(ws + pl.off_chunk_ml) : nullptr;
    a.ws_dec_o = pl.dec_split ? reinterpret_cast<float *>(ws + pl.off_dec_o) : nullptr;
    a.ws_dec_ml = pl.dec_split ? reinterpret_cast<float *>(ws + pl.off_dec_ml) : nullptr;
    a.work = reinterpret_cast<int32_t *>(ws);
    a.num_reqs = sh.R;
    a.num_rows = sh.T;
    a.page_size = batch->page_size;
    a.log2_page = sh.log2_page;
    a.max_pages = batch->max_pages_per_req;
    a.num_pages = batch->num_pages;
    a.scale_log2 = (float)((double)softmax_scale * 1.4426950408889634);
    a.ks_chunk = pl.ks_chunk;
    a.chunk_rev = pl.chunk_rev ? 1 : 0;
    a.n_chunk_items = pl.n_chunk_items;
    a.n_dec_units = pl.n_dec_units;
    a.dec_unit_tiles = pl.dec_unit_tiles;
    a.grid = pl.grid;
    a.dec_first_wgs = pl.dec_first_wgs;
    a.merge_hsplit = pl.merge_hsplit;
    a.dec_total_tiles = pl.dec_total_tiles;
    a.out_bf16 = out_dtype == MLA_OUT_BF16 ? 1 : 0;
    a.spin_limit = debug_value(MLA_DEBUG_SPIN_LIMIT).load(std::memory_order_relaxed);
    a.route = route;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    const bool chk = check_mode();
    if (chk && (st = check_device_batch(batch, sh, s)) != MLA_OK) return st;
    hipError_t e = mla::launch_attention(a, s);
    if (e != hipSuccess) return hip_fail(e, "attention kernel launch");
    if (pl.chunk_split || pl.dec_split) {
        e = mla::launch_combine(a, s);
        if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
    }
    return chk ? check_after_launch(s, new_latents ? "mixed_step" : "mixed_step_attn") : MLA_OK;
}

}  // namespace

namespace mla {

int attend_rows(const mla_batch *batch, const uint16_t *q, const uint16_t *new_latents, uint16_t *kv_cache,
                float softmax_scale, void *out, int32_t out_dtype, void *workspace, size_t workspace_bytes, void *stream,
                ChunkRoute route) {
    return attend(batch, q, new_latents, kv_cache, softmax_scale, out, out_dtype, nullptr, workspace, workspace_bytes,
                  stream, route);
}

}  // namespace mla

extern "C" {

int mixed_step_attn(const mla_batch *batch, const uint16_t *q, const uint16_t *kv_cache, float softmax_scale,
                    void *out, int32_t out_dtype, float *lse, void *workspace, size_t workspace_bytes,
                    void *stream) {
    return attend(batch, q, nullptr, const_cast<uint16_t *>(kv_cache), softmax_scale, out, out_dtype, lse, workspace,
                  workspace_bytes, stream);
}

static_assert(MLA_NOALLOC_SCRATCH_BYTES == mla::kNoAllocScratchBytes, "scratch size of the header and the library");

int mixed_step_noalloc(const mla_batch *batch, const uint16_t *q, const uint16_t *new_latents, uint16_t *kv_cache,
                       float softmax_scale, void *out, int32_t out_dtype, float *lse, void *stream) {
    g_err[0] = '\0';
    if (batch && batch->num_reqs > 0 && !new_latents) return fail(MLA_ERR_INVALID_ARG, "new_latents is NULL");
    void *ws = nullptr;
    const hipError_t e = mla::noalloc_scratch(&ws);
    if (e != hipSuccess) return hip_fail(e, "no-allocation scratch set-up");
    const int st = attend(batch, q, new_latents, kv_cache, softmax_scale, out, out_dtype, lse, ws,
                          mla::kNoAllocScratchBytes, stream);
    if (st == MLA_ERR_WORKSPACE)
        return fail(MLA_ERR_WORKSPACE, "mixed_step_noalloc: this batch needs %zu bytes of scratch, more than the %zu "
                    "bytes the no-allocation entry point holds; use mixed_step with a workspace",
                    mixed_step_workspace_bytes(batch), mla::kNoAllocScratchBytes);
    return st;
}

int mixed_step(const mla_batch *batch, const uint16_t *q, const uint16_t *new_latents, uint16_t *kv_cache,
               float softmax_scale, void *out, int32_t out_dtype, float *lse, void *workspace,
               size_t workspace_bytes, void *stream) {
    if (batch && batch->num_reqs > 0 && !new_latents) {
        g_err[0] = '\0';
        return fail(MLA_ERR_INVALID_ARG, "new_latents is NULL");
    }
    return attend(batch, q, new_latents, kv_cache, softmax_scale, out, out_dtype, lse, workspace, workspace_bytes,
                  stream);
}

}  // extern "C"
