// Host-only check of the planner (csrc/plan.cpp), built by the CPU tests with
// AddressSanitizer and UndefinedBehaviorSanitizer (g++, no device code).
//
// Sweeps seeded pseudo-random problem shapes through plan_fwd, plan_fwd_all,
// plan_decode and plan_gemm with the built-in gfx950 description (register
// footprints estimated, no device), and checks that every plan satisfies the
// legality rules the kernels rely on -- tile symbols from the compiled
// domains, LDS within capacity, the grid the launch will use, key splits that
// leave no split empty -- that the prefill pick is the minimum of the
// enumerated candidates, and that the plan formatters truncate safely.
// Prints "plan_check ok: N plans" and exits 0, or names the first violation
// and exits 1.  With --planted it corrupts one plan's grid and exits 0 only if
// the checks report it.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "common.h"

using namespace attn;

namespace {

int failures = 0;

#define CHECK(cond, ...)                                              \
    do {                                                              \
        if (!(cond)) {                                                \
            std::fprintf(stderr, "violation: %s -- ", #cond);         \
            std::fprintf(stderr, __VA_ARGS__);                        \
            std::fprintf(stderr, "\n");                               \
            if (++failures > 20) return false;                        \
        }                                                             \
    } while (0)

// splitmix64: a seeded stream of shapes
uint64_t state = 0x5eed1234abcdULL;
uint64_t next() {
    uint64_t z = (state += 0x9e3779b97f4a7c15ULL);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}
// log-uniform integer in [1, hi]
int log_uniform(int hi) {
    const double u = (next() >> 11) * (1.0 / 9007199254740992.0);
    const int v = (int)std::floor(std::exp(u * std::log((double)hi + 1.0)));
    return v < 1 ? 1 : (v > hi ? hi : v);
}

bool in(int v, const int* set, int n) {
    for (int i = 0; i < n; ++i)
        if (set[i] == v) return true;
    return false;
}

bool check_fwd(const attn_device_desc& desc, const FwdPlan& p, int B, int H, int Sq, int Skv,
               int d, int causal) {
    CHECK(p.d == d, "d %d", p.d);
    CHECK(in(p.block_n, kFwdBlockN, 3) && in(p.waves, kFwdWaves, 2) && in(p.pipe, kFwdPipe, 4),
          "tile (%d, %d, %d)", p.block_n, p.waves, p.pipe);
    CHECK(p.block_m == 32 * p.waves, "block_m %d", p.block_m);
    CHECK(p.pipe != 2 || p.waves == 8, "ping-pong needs 8 waves");
    CHECK(p.pipe != 3 || p.block_n <= 64, "pipe 3 needs BN <= 64");
    CHECK(p.lds_bytes > 0 && p.lds_bytes <= desc.lds_bytes_per_cu, "lds %d", p.lds_bytes);
    CHECK(p.wg_per_cu >= 1, "wg_per_cu %d", p.wg_per_cu);
    CHECK(p.n_qtiles == (Sq + p.block_m - 1) / p.block_m, "n_qtiles %d", p.n_qtiles);
    CHECK(p.kv_splits >= 1, "splits %d", p.kv_splits);
    const long long grid = (long long)B * H *
                           (causal ? (p.n_qtiles + 1) / 2 : (long long)p.n_qtiles * p.kv_splits);
    CHECK(p.grid == grid && p.grid > 0 && p.grid <= 0x7fffffffLL, "grid %lld (want %lld)",
          p.grid, grid);
    if (p.kv_splits > 1) {
        CHECK(!causal && p.pipe != 2, "splits with causal or ping-pong");
        CHECK(p.kv_chunk % p.block_n == 0, "chunk %d not whole tiles", p.kv_chunk);
        CHECK((long long)(p.kv_splits - 1) * p.kv_chunk < Skv, "empty last split");
        CHECK((long long)p.kv_splits * p.kv_chunk >= Skv, "keys not covered");
    } else {
        CHECK(p.kv_chunk == Skv, "unsplit chunk %d != Skv %d", p.kv_chunk, Skv);
    }
    CHECK(std::isfinite(p.modeled_us) && p.modeled_us > 0.0, "modeled %g", p.modeled_us);
    CHECK(p.bound && *p.bound, "no bound");
    return true;
}

bool check_decode(const DecodePlan& p, int B, int Hq, int Hkv, int Skv, int d) {
    CHECK(p.d == d, "d %d", p.d);
    CHECK(p.n_splits >= 1 && p.n_splits <= Skv, "splits %d", p.n_splits);
    CHECK(p.chunk == (Skv + p.n_splits - 1) / p.n_splits ||
              (Skv + p.chunk - 1) / p.chunk == p.n_splits,
          "chunk %d for %d splits of %d keys", p.chunk, p.n_splits, Skv);
    CHECK((long long)(p.n_splits - 1) * p.chunk < Skv, "empty last split");
    CHECK(p.grid > 0 && p.grid <= 0x7fffffffLL, "grid %lld", p.grid);
    const int group = Hq / Hkv;
    if (p.mfma) {
        CHECK(group >= kGqaMinGroup, "matrix-core decode for group %d", group);
        CHECK(p.q_blocks == (group + 15) / 16, "q_blocks %d", p.q_blocks);
        CHECK(p.grid == (long long)B * Hkv * p.q_blocks * p.n_splits, "mfma grid %lld", p.grid);
    } else {
        CHECK(group % p.heads_per_wg == 0, "heads per workgroup %d for group %d",
              p.heads_per_wg, group);
        CHECK(p.grid == (long long)B * Hq / p.heads_per_wg * p.n_splits, "grid %lld", p.grid);
    }
    CHECK(std::isfinite(p.modeled_us) && p.modeled_us > 0.0, "modeled %g", p.modeled_us);
    return true;
}

bool check_gemm(const attn_device_desc& desc, const GemmPlan& p, int M, int N, int K) {
    CHECK(p.block_m % (32 * p.waves_m) == 0 && p.block_n % (32 * p.waves_n) == 0,
          "tile %dx%d over %dx%d waves", p.block_m, p.block_n, p.waves_m, p.waves_n);
    CHECK(p.block_k == 32 || p.block_k == 64, "BK %d", p.block_k);
    // the 256 x 256 tile on 2 x 2 waves (hand-scheduled) runs pipes 1..3, the others 0..2
    const bool scheduled = p.block_m == 256 && p.block_n == 256 && p.waves_m == 2 && p.waves_n == 2;
    CHECK(scheduled ? p.pipe >= 1 && p.pipe <= 3 : p.pipe >= 0 && p.pipe <= 2, "pipe %d", p.pipe);
    CHECK(p.lds_bytes > 0 && p.lds_bytes <= desc.lds_bytes_per_cu, "lds %d", p.lds_bytes);
    CHECK(p.tiles_m == (M + p.block_m - 1) / p.block_m &&
              p.tiles_n == (N + p.block_n - 1) / p.block_n,
          "tiles %dx%d", p.tiles_m, p.tiles_n);
    CHECK(p.k_splits >= 1 && (p.k_splits == 1 || scheduled), "k_splits %d", p.k_splits);
    CHECK(p.grid == (long long)p.tiles_m * p.tiles_n * p.k_splits, "grid %lld", p.grid);
    if (p.k_splits > 1) {
        CHECK(p.k_chunk % p.block_k == 0, "k_chunk %d not whole k-tiles", p.k_chunk);
        CHECK((long long)(p.k_splits - 1) * p.k_chunk < K, "empty last K split");
        CHECK((long long)p.k_splits * p.k_chunk >= K, "K not covered");
        CHECK(gemm_workspace_bytes(p, M, N) <= kGemmMaxWorkspaceBytes, "workspace %lld",
              gemm_workspace_bytes(p, M, N));
    } else {
        CHECK(p.k_chunk == K, "unsplit k_chunk %d != K %d", p.k_chunk, K);
    }
    CHECK(std::isfinite(p.modeled_us) && p.modeled_us > 0.0, "modeled %g", p.modeled_us);
    CHECK(!scheduled || K % p.block_k == 0, "hand-scheduled tile with K %d not whole k-tiles", K);
    return true;
}

// A formatter writes at most buflen bytes, NUL-terminated, and returns the
// full length whatever buflen is.
template <typename P, typename F>
bool check_format(const P& p, F fmt) {
    char full[1024];
    const int n = fmt(p, full, (int)sizeof full);
    CHECK(n > 0 && n < (int)sizeof full && (int)std::strlen(full) == n, "length %d", n);
    for (int len : {0, 1, 7, n, n + 1}) {
        std::vector<char> buf((size_t)len + 8, '#');
        const int m = fmt(p, len ? buf.data() : nullptr, len);
        CHECK(m == n, "buflen %d returned %d, not %d", len, m, n);
        if (len > 0) {
            CHECK(std::strlen(buf.data()) == (size_t)std::min(n, len - 1), "buflen %d", len);
            CHECK(std::strncmp(buf.data(), full, (size_t)std::min(n, len - 1)) == 0,
                  "buflen %d prefix", len);
        }
        for (int i = len; i < len + 8; ++i) CHECK(buf[(size_t)i] == '#', "wrote past %d", len);
    }
    return true;
}

}  // namespace

int main(int argc, char** argv) {
    attn_device_desc desc;
    default_desc(&desc);
    if (argc > 1 && std::strcmp(argv[1], "--planted") == 0) {
        // the checks must see a plan whose grid disagrees with its tiles
        FwdPlan p;
        if (!plan_fwd(desc, 2, 3, 1000, 1000, 128, 0, &p)) return 1;
        p.grid += 1;
        check_fwd(desc, p, 2, 3, 1000, 1000, 128, 0);
        std::printf(failures ? "planted violation caught\n" : "planted violation missed\n");
        return failures ? 0 : 1;
    }
    int plans = 0;
    std::vector<FwdPlan> all(512);
    for (int it = 0; it < 2000 && failures == 0; ++it) {
        const int d = (next() & 1) ? 128 : 64;
        const int causal = (int)(next() & 1);
        const int B = log_uniform(8), H = log_uniform(64);
        const int Skv = log_uniform(1 << 17);
        const int Sq = causal ? 1 + (int)(next() % (uint64_t)Skv) : log_uniform(1 << 14);
        FwdPlan p;
        if (!plan_fwd(desc, B, H, Sq, Skv, d, causal, &p)) {
            std::fprintf(stderr, "no prefill plan for B=%d H=%d Sq=%d Skv=%d d=%d causal=%d\n",
                         B, H, Sq, Skv, d, causal);
            return 1;
        }
        if (!check_fwd(desc, p, B, H, Sq, Skv, d, causal)) break;
        const int n = plan_fwd_all(desc, B, H, Sq, Skv, d, causal, all.data(), (int)all.size());
        CHECK(n >= 1 && n <= (int)all.size(), "candidates %d", n);
        for (int i = 0; i < n && i < (int)all.size(); ++i) {
            check_fwd(desc, all[(size_t)i], B, H, Sq, Skv, d, causal);
            CHECK(p.modeled_us <= all[(size_t)i].modeled_us, "pick %.3f above candidate %.3f",
                  p.modeled_us, all[(size_t)i].modeled_us);
        }
        check_format(p, format_fwd_plan);
        ++plans;

        const int Hkv = log_uniform(16), group = log_uniform(32);
        const int dSkv = log_uniform(1 << 20);
        const int n_req = (next() & 3) == 0 ? log_uniform(600) : 0;
        DecodePlan q;
        if (!plan_decode(desc, B, Hkv * group, Hkv, dSkv, d, n_req, &q)) {
            std::fprintf(stderr, "no decode plan for B=%d Hq=%d Hkv=%d Skv=%d d=%d n=%d\n", B,
                         Hkv * group, Hkv, dSkv, d, n_req);
            return 1;
        }
        check_decode(q, B, Hkv * group, Hkv, dSkv, d);
        check_format(q, format_decode_plan);
        ++plans;

        const int M = log_uniform(16384), N = 8 * log_uniform(2048), K = 8 * log_uniform(2048);
        GemmPlan g;
        if (!plan_gemm(desc, M, N, K, (int)(next() & 1), &g)) {
            std::fprintf(stderr, "no GEMM plan for %dx%dx%d\n", M, N, K);
            return 1;
        }
        check_gemm(desc, g, M, N, K);
        check_format(g, format_gemm_plan);
        ++plans;
    }
    if (failures) return 1;
    std::printf("plan_check ok: %d plans\n", plans);
    return 0;
}
