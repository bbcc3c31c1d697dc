// Host-side exercise of the library's C ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer (built by tests/test_host_sanitizers.py): the planner
// (App. A.7 FLOPs, FIR, Algorithm 1, the Sec. 2.5 placements, maps), the page allocator
// and the runtime's argument checks.  Nothing here touches a GPU: every runtime call is
// one that must be rejected before any device work, so the program is safe to run on a
// machine with a GPU as well.  Exit status 0 = every check held; sanitizer reports abort.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <set>
#include <vector>

#include "kvpipe.h"

static int g_fail = 0;
#define CHECK(c)                                                             \
    do {                                                                     \
        if (!(c)) {                                                          \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            ++g_fail;                                                        \
        }                                                                    \
    } while (0)

static void planner(std::mt19937_64& rng) {
    for (int it = 0; it < 3000; ++it) {
        const int L = 1 + (int)(rng() % 80);
        const int P = 1 + (int)(rng() % std::min(L, 16));
        // A random partition of L layers into P non-empty, ordered stages.
        std::vector<int> cuts;
        std::set<int> pick;
        while ((int)pick.size() < P - 1) pick.insert(1 + (int)(rng() % (L - 1 > 0 ? L - 1 : 1)));
        std::vector<int32_t> stage(L);
        int s = 0;
        for (int l = 0; l < L; ++l) {
            if (pick.count(l)) ++s;
            stage[l] = s;
        }
        std::vector<double> f0(L), f1(L);
        for (int l = 0; l < L; ++l) {
            f0[l] = (double)(1000 + rng() % 100000);
            f1[l] = f0[l] - (double)(1 + rng() % 900);
        }
        std::vector<uint8_t> adm(L);
        for (int l = 0; l < L; ++l) adm[l] = (uint8_t)(rng() % 4 != 0);
        kvp_plan_in in{};
        in.L = L;
        in.P = P;
        in.stage_of_layer = stage.data();
        in.f_full = f0.data();
        in.f_share = f1.data();
        in.f_lmhead = (double)(rng() % 50000);
        in.eps = 1e-4 + (double)(rng() % 1000) * 1e-4;
        in.m = (int)(rng() % (L + 2)) - 1;
        in.admissible = (rng() % 2) ? adm.data() : nullptr;
        in.alpha = (rng() % 3 == 0) ? (double)(rng() % 100) / 100.0 : -1.0;
        std::vector<uint8_t> z(L, 7);
        std::vector<double> sf(P, -1.0);
        kvp_plan_out out{z.data(), sf.data(), 0.0, 0, 0};
        const int rc = kvp_plan_fir(&in, &out);
        CHECK(rc == KVP_OK || P > L);
        if (rc == KVP_OK) {
            CHECK(z[0] == 0);
            CHECK(out.n_converted >= 0 && out.n_converted < L);
            std::vector<int32_t> tau(L);
            CHECK(kvp_map_from_mask(L, z.data(), tau.data()) == KVP_OK);
            std::vector<int32_t> canon(L);
            CHECK(kvp_canonicalize_map(L, tau.data(), canon.data()) == KVP_OK);
            std::vector<double> sf2(P);
            CHECK(kvp_stage_flops(L, P, stage.data(), f0.data(), f1.data(), z.data(), in.f_lmhead, sf2.data()) ==
                  KVP_OK);
            for (int i = 0; i < P; ++i) CHECK(sf2[i] == sf[i]);
            double fir = 0.0;
            CHECK(kvp_fir(P, sf2.data(), &fir) == KVP_OK && fir == out.fir);
        }
        for (int strat = 0; strat < 2; ++strat) {
            std::vector<uint8_t> zp(L, 9);
            int32_t n_placed = -1, stop = -1;
            const int k = (int)(rng() % (L + 3));
            CHECK(kvp_place(strat, L, P, stage.data(), k, in.admissible, in.alpha, zp.data(), &n_placed, &stop) ==
                  KVP_OK);
            CHECK(n_placed >= 0 && n_placed <= k && zp[0] == 0);
        }
        // Maps with random (often invalid) entries.
        std::vector<int32_t> tau(L), outm(L);
        for (int l = 0; l < L; ++l) tau[l] = (int)(rng() % (L + 2)) - 1;
        const int rc2 = kvp_canonicalize_map(L, tau.data(), outm.data());
        CHECK(rc2 == KVP_OK || rc2 == KVP_E_BAD_MAP);
        std::vector<uint8_t> zz(L);
        for (int l = 0; l < L; ++l) zz[l] = (uint8_t)(rng() % 2);
        const int rc3 = kvp_map_from_mask(L, zz.data(), outm.data());
        CHECK(rc3 == (zz[0] ? KVP_E_BAD_MAP : KVP_OK));
    }
    // Rejections.
    kvp_plan_in bad{};
    std::vector<uint8_t> z(4);
    std::vector<double> sf(4);
    kvp_plan_out out{z.data(), sf.data(), 0.0, 0, 0};
    CHECK(kvp_plan_fir(&bad, &out) == KVP_E_INVALID_ARG);
    CHECK(kvp_plan_fir(nullptr, &out) == KVP_E_INVALID_ARG);
    CHECK(kvp_fir(0, sf.data(), nullptr) == KVP_E_INVALID_ARG);
    CHECK(kvp_map_from_mask(0, z.data(), nullptr) == KVP_E_INVALID_ARG);
    for (int it = 0; it < 2000; ++it) {
        kvp_shape sh{};
        sh.b = (int64_t)(rng() % 8) - 1;
        sh.s = (int64_t)(rng() % 20000) - 1;
        sh.h = 64 * (int64_t)(rng() % 200);
        sh.a = (int64_t)(rng() % 70);
        sh.g = (int64_t)(rng() % 10);
        sh.ffn = (int64_t)(rng() % 30000) - 1;
        sh.causal = (int32_t)(rng() % 2);
        double a = 0, b = 0;
        const int rc = kvp_layer_flops(&sh, (int)(rng() % 3), &a, &b);
        CHECK(rc == KVP_OK || rc == KVP_E_INVALID_ARG);
        if (rc == KVP_OK) CHECK(a > b && b > 0);
    }
}

static void pager(std::mt19937_64& rng) {
    for (int trial = 0; trial < 20; ++trial) {
        const int n_pages = 1 + (int)(rng() % 500), seqs = 1 + (int)(rng() % 40), row = 1 + (int)(rng() % 40);
        kvp_pager* p = nullptr;
        CHECK(kvp_pager_create(n_pages, seqs, row, &p) == KVP_OK && p);
        std::vector<int32_t> ids(seqs);
        for (int i = 0; i < seqs; ++i) ids[i] = i;
        std::vector<int32_t> rows((size_t)seqs * row);
        for (int op = 0; op < 2000; ++op) {
            const int s = (int)(rng() % (seqs + 2)) - 1;
            if (rng() % 3) {
                const int rc = kvp_pager_reserve(p, s, (int)(rng() % (64 * row + 130)) - 1);
                CHECK(rc == KVP_OK || rc == KVP_E_CAPACITY || rc == KVP_E_INVALID_ARG);
            } else {
                const int rc = kvp_pager_release(p, s);
                CHECK(rc == KVP_OK || rc == KVP_E_INVALID_ARG);
            }
            int free_pages = -1;
            CHECK(kvp_pager_free_pages(p, &free_pages) == KVP_OK && free_pages >= 0 && free_pages <= n_pages);
            if (op % 97 == 0) {
                CHECK(kvp_pager_rows(p, ids.data(), seqs, rows.data()) == KVP_OK);
                std::set<int32_t> seen;
                int used = 0;
                for (int32_t v : rows)
                    if (v >= 0) {
                        CHECK(v < n_pages && !seen.count(v));
                        seen.insert(v);
                        ++used;
                    }
                CHECK(used + free_pages == n_pages);
            }
        }
        kvp_pager_destroy(p);
    }
    kvp_pager* p = nullptr;
    CHECK(kvp_pager_create(0, 1, 1, &p) == KVP_E_INVALID_ARG);
    kvp_pager_destroy(nullptr);
}

static void runtime_checks(std::mt19937_64& rng) {
    // Random descriptors: accepted ones must give consistent workspace sizes; rejected ones
    // leave *out NULL.
    for (int it = 0; it < 3000; ++it) {
        kvp_model_desc d{};
        d.L = (int)(rng() % 6);
        d.a = (int)(rng() % 9);
        d.g = 1 + (int)(rng() % 4);
        d.d_h = (rng() % 2) ? 128 : 16 << (rng() % 4);
        d.h = d.a * d.d_h + ((rng() % 8 == 0) ? 1 : 0);
        d.dtype = (int)(rng() % 3);
        d.rope_base = (rng() % 10 == 0) ? -1.0 : 10000.0;
        d.max_batch = (int)(rng() % 70);
        d.max_seq = (int)(rng() % 600);
        d.kv_capacity = 64 * (int)(rng() % 12) + ((rng() % 6 == 0) ? 3 : 0);
        std::vector<int32_t> tau(d.L > 0 ? d.L : 1);
        for (int l = 0; l < (int)tau.size(); ++l) tau[l] = (rng() % 3) ? 0 : l;
        kvp_ctx* c = (kvp_ctx*)0x1;
        const int rc = kvp_create(&d, tau.data(), &c);
        if (rc != KVP_OK) {
            CHECK(c == nullptr);
            CHECK(kvp_last_error()[0] != 0);
            continue;
        }
        size_t a = 0, b = 0, t = 0;
        const int B = 1 + (int)(rng() % d.max_batch), S = 1 + (int)(rng() % d.max_seq);
        CHECK(kvp_workspace_size(c, KVP_PHASE_PREFILL, B, S, &a) == KVP_OK && a > 0);
        CHECK(kvp_workspace_size(c, KVP_PHASE_DECODE, B, S, &b) == KVP_OK && b > 0);
        const int rcb = kvp_workspace_size(c, KVP_PHASE_BACKWARD, B, S, &t);
        CHECK(rcb == KVP_OK || rcb == KVP_E_SHAPE);
        CHECK(kvp_workspace_size(c, KVP_PHASE_PREFILL, d.max_batch + 1, S, &a) == KVP_E_CAPACITY);
        CHECK(kvp_train_saved_size(c, B, S, &t) == KVP_OK);
        std::vector<int32_t> got(d.L);
        CHECK(kvp_get_map(c, got.data()) == KVP_OK);
        // Weights never set: every call stops at the state check, before any device work.
        void* fake = (void*)(uintptr_t)0x10000;
        CHECK(kvp_prefill(c, fake, (char*)fake + 4096, B, S, fake, a, nullptr) == KVP_E_STATE);
        CHECK(kvp_decode_step(c, fake, (const int32_t*)fake, 0, (char*)fake + 4096, B, fake, b, nullptr) ==
              KVP_E_STATE);
        CHECK(kvp_prefill(c, fake, fake, B, S, fake, a, nullptr) == KVP_E_INVALID_ARG);
        CHECK(kvp_set_layer(c, d.L, fake, nullptr, nullptr, fake) == KVP_E_INVALID_ARG);
        CHECK(kvp_set_layer(c, 0, (char*)fake + 2, fake, fake, fake) == KVP_E_INVALID_ARG);
        CHECK(kvp_set_kv_slot(c, 0, nullptr, fake) == KVP_E_INVALID_ARG);
        CHECK(kvp_set_layer_grads(c, -1, fake, fake, fake, fake) == KVP_E_INVALID_ARG);
        double ms[KVP_NUM_KERNEL_KINDS];
        int64_t n[KVP_NUM_KERNEL_KINDS];
        CHECK(kvp_profile_read(c, ms, n) == KVP_OK);
        CHECK(kvp_destroy(c) == KVP_OK);
    }
    CHECK(kvp_create(nullptr, nullptr, nullptr) == KVP_E_INVALID_ARG);
    CHECK(kvp_destroy(nullptr) == KVP_OK);
    for (int s = 1; s >= -8; --s) CHECK(std::strlen(kvp_status_string(s)) > 0);
}

int main() {
    std::mt19937_64 rng(20261202);
    planner(rng);
    pager(rng);
    runtime_checks(rng);
    if (g_fail) {
        std::fprintf(stderr, "%d checks failed\n", g_fail);
        return 1;
    }
    std::printf("host checks passed\n");
    return 0;
}
