// Host-only harness around the library's work planner (the translation unit
// is included as is; the launch functions are stubbed because nothing is
// launched here, and the device queries answer for a 256-CU device).  Input on
// stdin, one batch per line:
//   ncu page_size R q_0 p_0 q_1 p_1 ...
// (PLAN_ROUTE, PLAN_CHUNK_KEYS, PLAN_DEC_UNIT, PLAN_DEC_FIRST and PLAN_SERVING in the
// environment: see main)
// Output, one line per batch:
//   ok ks n_chunk_items n_dec_items unit_tiles dec_total grid merge_hsplit chunk_split dec_split bytes
//      off_chunk_o off_chunk_ml off_dec_o off_dec_ml plan_us warm est_us dec_first_wgs
// or "err <status> <message>".
// A line "ws <bytes> page_size R q_0 p_0 ..." instead calls the real
// mixed_step_attn entry point with fake device pointers and a workspace of
// <bytes> bytes and prints "rc <status> <needed bytes> <message>"; "na 0 ..."
// calls mixed_step_noalloc the same way (its scratch stubbed by a fake address).
// A line "cm <seed> <cases>" checks the planner's cost model on random
// workgroup loads against brute force and prints "cm ok <cases>" or the first
// case that fails.
#include <hip/hip_runtime.h>

static hipError_t harness_get_device(int *d) {
    *d = 0;
    return hipSuccess;
}
static hipError_t harness_get_attribute(int *v, hipDeviceAttribute_t, int) {
    *v = 256;
    return hipSuccess;
}
#define hipGetDevice harness_get_device
#define hipDeviceGetAttribute harness_get_attribute
#include "../../paper_2607_02043_amd/csrc/mla_api.cpp"
#undef hipGetDevice
#undef hipDeviceGetAttribute

#include <chrono>
#include <iostream>
#include <queue>
#include <random>
#include <sstream>
#include <string>

namespace mla {
hipError_t launch_append(const AppendArgs &, hipStream_t) { return hipSuccess; }
hipError_t launch_attention(const AttnArgs &, hipStream_t) { return hipSuccess; }
hipError_t launch_combine(const AttnArgs &, hipStream_t) { return hipSuccess; }
hipError_t read_flags(int *flags, bool) {
    *flags = 0;
    return hipSuccess;
}
hipError_t noalloc_scratch(void **ptr) {
    alignas(256) static char fake[256];
    *ptr = fake;
    return hipSuccess;
}
}  // namespace mla

// Each item or unit to the workgroup that is free first, one at a time; the
// finishing time of the last one (or the largest load).
static std::vector<double> brute_schedule(std::vector<double> loads, const std::vector<double> &items) {
    for (double c : items) *std::min_element(loads.begin(), loads.end()) += c;
    return loads;
}

static std::string cost_model_check(unsigned seed, int cases) {
    std::mt19937 g(seed);
    for (int k = 0; k < cases; ++k) {
        const int G = 1 + (int)(g() % 300);
        std::vector<double> items(g() % 1500);
        for (double &c : items) c = g() % 4 == 0 ? 1.5 : 14.0 + 2.2 * (double)(1 + g() % 40);
        // the chunk queue: same loads as one at a time to the least loaded
        std::vector<double> sim = simulate_chunks(items, G), ref = brute_schedule(std::vector<double>(G, 0.0), items);
        std::sort(sim.begin(), sim.end());
        std::sort(ref.begin(), ref.end());
        if (sim != ref) return "simulate_chunks differs, case " + std::to_string(k);
        // decode units after it: exact fill, its bounds
        const long long n = 1 + (long long)(g() % 3000);
        const double u = 5.5 + 3.5 * (double)(1 + g() % 64);
        const std::vector<LoadRun> runs = load_runs(sim);
        std::vector<double> ld = brute_schedule(sim, std::vector<double>((size_t)n, u));
        const double want = *std::max_element(ld.begin(), ld.end());
        const double got = fill_units(runs, n, u), lower = fill_bound(runs, n, u);
        const double level = std::max(runs.back().load, water_level(runs, n, u));
        if (std::abs(got - want) > 1e-9 * want)
            return "fill_units " + std::to_string(got) + " vs " + std::to_string(want) + ", case " + std::to_string(k);
        if (lower > got * (1 + 1e-12) || level > got * (1 + 1e-12))
            return "a lower bound exceeds the fill, case " + std::to_string(k);
    }
    return "ok " + std::to_string(cases);
}

int main() {
    // PLAN_ROUTE="min_rows pair_keys": leave the chunk requests that this
    // route sends to the multi-head path out of the plan
    mla::ChunkRoute route = mla::kAbsorbAll;
    if (const char *e = std::getenv("PLAN_ROUTE")) {
        std::istringstream r(e);
        r >> route.min_rows >> route.pair_keys;
    }
    // PLAN_SERVING=1: plan through the library's cached, warm-started
    // planner (the device's CU count, 256 here), as consecutive calls do
    const bool serving = std::getenv("PLAN_SERVING") != nullptr;
    // PLAN_CHUNK_KEYS=k: the forced chunk key split of the debug knob
    if (const char *e = std::getenv("PLAN_CHUNK_KEYS")) mla_debug_set(MLA_DEBUG_CHUNK_KEYS, std::atoi(e));
    // PLAN_DEC_UNIT=u: the forced decode unit size of the debug knob
    if (const char *e = std::getenv("PLAN_DEC_UNIT")) mla_debug_set(MLA_DEBUG_DEC_UNIT, std::atoi(e));
    // PLAN_DEC_FIRST=d: the forced decode-first workgroups of the debug knob
    if (const char *e = std::getenv("PLAN_DEC_FIRST")) mla_debug_set(MLA_DEBUG_DEC_FIRST, std::atoi(e));
    std::string line;
    while (std::getline(std::cin, line)) {
        if (line.rfind("cm ", 0) == 0) {
            std::istringstream in(line.substr(3));
            unsigned seed = 0;
            int cases = 0;
            in >> seed >> cases;
            std::cout << "cm " << cost_model_check(seed, cases) << "\n";
            continue;
        }
        const bool noalloc = line.rfind("na ", 0) == 0;
        if (line.rfind("ws ", 0) == 0 || noalloc) {
            std::istringstream in(line.substr(3));
            long long bytes = 0;
            int P = 0, R = 0;
            in >> bytes >> P >> R;
            std::vector<int32_t> q(R), p(R);
            long long maxk = 1;
            for (int i = 0; i < R; ++i) {
                in >> q[i] >> p[i];
                maxk = std::max<long long>(maxk, (long long)q[i] + p[i]);
            }
            static const int32_t fake = 0;
            mla_batch b{};
            b.num_reqs = R;
            b.page_size = P;
            b.num_pages = 1 << 20;
            b.max_pages_per_req = (int)((maxk + P - 1) / P);
            b.q_lens = q.data();
            b.prefix_lens = p.data();
            b.cu_q_dev = &fake;
            b.prefix_lens_dev = &fake;
            b.block_table_dev = &fake;
            alignas(16) static char fake_dev[16];
            const size_t need = mixed_step_workspace_bytes(&b);
            const uint16_t *fq = reinterpret_cast<const uint16_t *>(fake_dev);
            const int rc = noalloc ? mixed_step_noalloc(&b, fq, fq, reinterpret_cast<uint16_t *>(fake_dev), 0.07f,
                                                        fake_dev, MLA_OUT_F32, nullptr, nullptr)
                                   : mixed_step_attn(&b, fq, fq, 0.07f, fake_dev, MLA_OUT_F32, nullptr,
                                                     bytes > 0 ? fake_dev : nullptr, (size_t)bytes, nullptr);
            std::cout << "rc " << rc << " " << need << " " << mla_last_error() << "\n";
            continue;
        }
        std::istringstream in(line);
        int ncu = 0, P = 0, R = 0;
        if (!(in >> ncu >> P >> R)) continue;
        std::vector<int32_t> q(R), p(R);
        long long maxk = 1;
        for (int i = 0; i < R; ++i) {
            in >> q[i] >> p[i];
            maxk = std::max<long long>(maxk, (long long)q[i] + p[i]);
        }
        static const int32_t fake = 0;  // device pointers are never dereferenced by the planner
        mla_batch b{};
        b.num_reqs = R;
        b.page_size = P;
        b.num_pages = 1 << 30;
        b.max_pages_per_req = (int)((maxk + P - 1) / P);
        b.q_lens = q.data();
        b.prefix_lens = p.data();
        b.cu_q_dev = &fake;
        b.prefix_lens_dev = &fake;
        b.block_table_dev = &fake;
        Shape sh;
        int st = check_batch(&b, &sh);
        Plan pl{};
        double us = 0.0;
        if (st == MLA_OK && sh.R > 0) {
            const auto t0 = std::chrono::steady_clock::now();
            st = serving ? make_plan(&b, sh, &pl, route) : make_plan_uncached(&b, sh, ncu, route, &pl);
            us = std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
        }
        if (st != MLA_OK) {
            std::cout << "err " << st << " " << g_err << "\n";
            continue;
        }
        std::cout << "ok " << pl.ks_chunk << " " << pl.n_chunk_items << " " << pl.n_dec_units << " "
                  << pl.dec_unit_tiles << " " << pl.dec_total_tiles << " " << pl.grid << " " << pl.merge_hsplit << " "
                  << (int)pl.chunk_split << " " << (int)pl.dec_split << " " << pl.bytes << " " << pl.off_chunk_o << " "
                  << pl.off_chunk_ml << " " << pl.off_dec_o << " " << pl.off_dec_ml << " " << us << " "
                  << (int)pl.warm << " " << pl.est_us << " " << pl.dec_first_wgs << "\n";
    }
    return 0;
}
