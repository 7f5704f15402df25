// Host-side code of the library driven through its C entry points under
// AddressSanitizer and UndefinedBehaviorSanitizer (built and run by
// tests/test_host_sanitizers.py): the seeded weight generator, the elastic
// allocator (Algorithm 1, Eq. (2), monitor, refinement) on random tables and
// on invalid input, and the rollout scheduler (group pipeline, Algorithm 2)
// through random event sequences.  Exits non-zero on any failed check; the
// sanitizers abort on the first finding.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "ebrl.h"
#include "ebrl_alloc.h"
#include "ebrl_sched.h"
#include "../paper_2609_27547_amd/csrc/weights.h"

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd() {
    g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(g_state >> 33);
}
static double urand() { return (rnd() + 0.5) / 2147483648.0; }

#define CHECK(c)                                                        \
    do {                                                                \
        if (!(c)) {                                                     \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            exit(1);                                                    \
        }                                                               \
    } while (0)

static void weights() {
    for (int64_t count : {0, 1, 2, 3, 17, 1000, 100001}) {
        std::vector<uint16_t> b(count + 1, 0xABCD);
        std::vector<float> f(count + 1, -7.f);
        ebrl::generate_weight(7, 1003, count, 0.02, true, b.data());
        ebrl::generate_weight(7, 1003, count, 0.02, false, f.data());
        CHECK(b[count] == 0xABCD && f[count] == -7.f);   // nothing written past the end
        for (int64_t i = 0; i < count; ++i) CHECK(f[i] > -1.f && f[i] < 1.f);
    }
}

static void allocator() {
    for (int trial = 0; trial < 300; ++trial) {
        const int nc = 1 + rnd() % 3, ns = 1 + rnd() % 3, ng = 1 + rnd() % 5, nb = 1 + rnd() % 4,
                  nt = 1 + rnd() % 5, nbt = 1 + rnd() % 3;
        std::vector<int32_t> cenv(nc), ssim(ns), sgen(ng), bgen(nb), strain(nt), btrain(nbt);
        for (int i = 0; i < nc; ++i) cenv[i] = i + 1;
        for (int i = 0; i < ns; ++i) ssim[i] = i * 10;
        for (int i = 0; i < ng; ++i) sgen[i] = 10 + 20 * i;
        for (int i = 0; i < nb; ++i) bgen[i] = 8 << i;
        for (int i = 0; i < nt; ++i) strain[i] = 10 + 20 * i;
        for (int i = 0; i < nbt; ++i) btrain[i] = 16 << i;
        std::vector<double> sim(nc * ns), gen(ng * nb), gmem(nb), train(nt * nbt), tmem(nbt);
        for (auto& v : sim) v = 100 * urand();
        for (auto& v : gen) v = 100 * urand();
        for (auto& v : train) v = 100 * urand();
        for (auto& v : gmem) v = 1e9 * urand();
        for (auto& v : tmem) v = 1e9 * urand();
        ebrl_alloc_profiles P = {nc, cenv.data(), ns, ssim.data(), sim.data(), ng, sgen.data(), nb, bgen.data(),
                                 gen.data(), gmem.data(), nt, strain.data(), nbt, btrain.data(), train.data(),
                                 tmem.data()};
        ebrl_alloc_limits L = {(int32_t)(1 + rnd() % 64), 2e9 * urand(), 10, 10, 0.05};
        ebrl_alloc_result r;
        const int rc = ebrl_alloc_solve(&P, &L, &r);
        CHECK(rc == EBRL_OK || rc == EBRL_E_OOM || rc == EBRL_E_INVALID);
        if (rc == EBRL_OK) {
            ebrl_alloc_result o = r;
            CHECK(ebrl_alloc_objective(&P, &o) == EBRL_OK);
            std::vector<double> g2(gen.size()), t2(train.size());
            CHECK(ebrl_alloc_refine(&P, &r, 50 * urand(), 50 * urand(), g2.data(), t2.data()) == EBRL_OK);
        }
    }
    ebrl_alloc_result r;
    CHECK(ebrl_alloc_solve(nullptr, nullptr, &r) == EBRL_E_INVALID);
    ebrl_alloc_monitor* m = nullptr;
    CHECK(ebrl_alloc_monitor_create(20, 0.15, 20, &m) == EBRL_OK);
    int triggers = 0;
    for (int i = 0; i < 500; ++i) {
        int32_t t = 0;
        CHECK(ebrl_alloc_monitor_observe(m, 10 * urand(), i < 250 ? 1.0 : 10 * urand(), &t) == EBRL_OK);
        triggers += t;
    }
    CHECK(triggers > 0);
    ebrl_alloc_monitor_destroy(m);
}

static void scheduler() {
    for (int trial = 0; trial < 50; ++trial) {
        const int n_envs = 1 + rnd() % 40, n_groups = 1 + rnd() % n_envs, chunk = 1 + rnd() % 6;
        ebrl_sched* s = nullptr;
        CHECK(ebrl_sched_create(n_envs, n_groups, chunk, &s) == EBRL_OK);
        std::vector<int32_t> ids(n_envs);
        std::vector<int> running;
        const int cores = 1 + rnd() % 8;
        const int stride = rnd() % 2 ? cores : 0;
        for (int step = 0; step < 4000; ++step) {
            const int op = rnd() % 3;
            if (op == 0) {
                int32_t env = -1;
                CHECK(ebrl_sched_dispatch(s, rnd() % cores, stride, &env) == EBRL_OK);
                if (env >= 0) running.push_back(env);
            } else if (op == 1 && !running.empty()) {
                const size_t k = rnd() % running.size();
                int32_t done = 0;
                CHECK(ebrl_sched_complete(s, running[k], 0.04 * urand(), &done) == EBRL_OK);
                running.erase(running.begin() + k);
            } else {
                int32_t g = -1, n = 0;
                CHECK(ebrl_sched_next_group(s, &g, ids.data(), n_envs, &n) == EBRL_OK);
                if (g >= 0) CHECK(ebrl_sched_deliver(s, g) == EBRL_OK);
            }
        }
        int32_t sd, ru, hc;
        double ld;
        for (int e = 0; e < n_envs; ++e) CHECK(ebrl_sched_env_state(s, e, &sd, &ru, &hc, &ld) == EBRL_OK);
        CHECK(ebrl_sched_env_state(s, n_envs, &sd, &ru, &hc, &ld) == EBRL_E_INVALID);
        int32_t dummy = 0;
        CHECK(ebrl_sched_complete(s, -1, 0.0, &dummy) != EBRL_OK);
        ebrl_sched_destroy(s);
    }
}

int main() {
    weights();
    allocator();
    scheduler();
    printf("host code clean under the sanitizers\n");
    return 0;
}
