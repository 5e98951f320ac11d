// Host exerciser of the library's tree, plan and table code, built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_host_sanitizers.py: random forks, appends,
// releases and raw allocations over small pools (evictions, copy-on-write, OOM), block
// tables, decode plans for every supported head layout, rank and RoPE setting, coverage and
// capacity queries, table validation and the argument checks shared by the attention entry
// points (those live in the GPU sources, which this build leaves out).
// Exit status 0 and no sanitizer report is the pass condition.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <vector>

#include "../include/forkkv.h"

namespace fkv {
fkv_status validate_attn_common(const fkv_attn_args *a, const char *who);  // the entry points' shared checks
}

#define CHECK(c)                                                          \
    do {                                                                  \
        if (!(c)) {                                                       \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            return 1;                                                     \
        }                                                                 \
    } while (0)

static int run_tree(unsigned seed, int ps, int nb, int nr) {
    std::mt19937 rng(seed);
    fkv_tree_config cfg{ps, nb, nr};
    fkv_tree *t = nullptr;
    CHECK(fkv_tree_create(&cfg, &t) == FKV_OK);
    std::vector<std::vector<int32_t>> toks;
    std::set<int> live;
    std::vector<int32_t> raw[2];
    int next = 0;
    for (int op = 0; op < 600; ++op) {
        const int kind = rng() % 8;
        fkv_fill_plan fp;
        if (kind < 3) {  // fork: continue a prefix of a live sequence, cut anywhere
            std::vector<int32_t> c;
            if (!live.empty() && rng() % 4) {
                auto it = live.begin();
                std::advance(it, rng() % live.size());
                const auto &src = toks[*it];
                c.assign(src.begin(), src.begin() + rng() % (src.size() + 1));
            }
            const int extra = 1 + rng() % 20;
            for (int i = 0; i < extra; ++i) c.push_back(rng() % 3);
            const int id = next;
            const fkv_status st = fkv_fork(t, id, rng() % 4, c.data(), (int64_t)c.size(), &fp);
            CHECK(st == FKV_OK || st == FKV_ERR_OOM);
            if (st == FKV_OK) {
                live.insert(id);
                if ((int)toks.size() <= id) toks.resize(id + 1);
                toks[id] = c;
                ++next;
            }
        } else if (kind < 5 && !live.empty()) {  // append
            auto it = live.begin();
            std::advance(it, rng() % live.size());
            std::vector<int32_t> c(rng() % (2 * ps + 2));
            for (auto &x : c) x = rng() % 3;
            const fkv_status st = fkv_cow_append(t, *it, c.data(), (int64_t)c.size(), &fp);
            CHECK(st == FKV_OK || st == FKV_ERR_OOM);
            if (st == FKV_OK) toks[*it].insert(toks[*it].end(), c.begin(), c.end());
        } else if (kind == 5 && !live.empty()) {  // release
            auto it = live.begin();
            std::advance(it, rng() % live.size());
            CHECK(fkv_release(t, *it) == FKV_OK);
            live.erase(it);
        } else if (kind == 6) {  // raw pages
            const int pool = rng() % 2, n = rng() % 4;
            std::vector<int32_t> ids(n + 1);
            const fkv_status st = fkv_alloc_pages(t, pool, n, ids.data());
            CHECK(st == FKV_OK || st == FKV_ERR_OOM);
            if (st == FKV_OK) raw[pool].insert(raw[pool].end(), ids.begin(), ids.begin() + n);
        } else if (!raw[op % 2].empty()) {
            const int pool = op % 2;
            CHECK(fkv_free_pages(t, pool, (int32_t)raw[pool].size(), raw[pool].data()) == FKV_OK);
            raw[pool].clear();
        }
        // tables of every live sequence, then a plan and a table check over them
        if (!live.empty() && op % 10 == 0) {
            std::vector<int32_t> ids(live.begin(), live.end());
            const int n = (int)ids.size();
            int mp = 1;
            for (int id : ids) mp = std::max<int>(mp, (int)((toks[id].size() + ps - 1) / ps));
            mp += 3;
            std::vector<int32_t> bb((size_t)n * mp), rb((size_t)n * mp), sl(n), ad(n);
            CHECK(fkv_get_block_tables(t, ids.data(), n, mp, bb.data(), rb.data(), sl.data()) == FKV_OK);
            for (int i = 0; i < n; ++i) ad[i] = (i % 3 == 2) ? -1 : i;
            CHECK(fkv_validate_tables(bb.data(), rb.data(), sl.data(), ad.data(), n, mp, ps, nb, nr) == FKV_OK);
            bb[0] = nb;  // one bad id
            CHECK(fkv_validate_tables(bb.data(), rb.data(), sl.data(), ad.data(), n, mp, ps, nb, nr) == FKV_ERR_INVALID);
            bb[0] = 0;
            for (int g : {4, 8})
                for (int r : {0, 8, 16, 32, 64})
                    for (int rope : {0, 1}) {
                        fkv_decode_plan_params prm{n, 8 * g, 8, ps, mp, 0, 0, 0, r, rope, 0};
                        fkv_plan *plan = nullptr;
                        CHECK(fkv_decode_plan_create(&prm, bb.data(), rb.data(), sl.data(), ad.data(), &plan) == FKV_OK);
                        fkv_plan_info info;
                        CHECK(fkv_decode_plan_info(plan, 128, r, &info) == FKV_OK);
                        std::vector<int32_t> words(info.plan_words);
                        CHECK(fkv_decode_plan_serialize(plan, words.data(), info.plan_words) == FKV_OK);
                        CHECK(fkv_decode_plan_serialize(plan, words.data(), info.plan_words - 1) == FKV_ERR_INVALID);
                        CHECK(fkv_decode_plan_covers(plan, sl.data(), n) == FKV_OK);
                        int64_t cap = 0;
                        CHECK(fkv_decode_plan_capacity(plan, n - 1, &cap) == FKV_OK && cap >= sl[n - 1]);
                        std::vector<int32_t> fp_(info.n_segments), np_(info.n_segments), na(info.n_segments),
                            ag((size_t)info.n_segments * n);
                        CHECK(fkv_decode_plan_segments(plan, fp_.data(), np_.data(), na.data(), ag.data(),
                                                       (int64_t)ag.size()) == FKV_OK);
                        fkv_decode_plan_destroy(plan);
                    }
        }
        fkv_pool_stats s;
        CHECK(fkv_get_pool_stats(t, &s) == FKV_OK);
        CHECK(s.base_pages_free + s.base_pages_referenced + s.base_pages_cached + s.base_pages_raw == nb);
        CHECK(s.res_pages_free + s.res_pages_referenced + s.res_pages_cached + s.res_pages_raw == nr);
    }
    fkv_tree_destroy(t);
    return 0;
}

int main() {
    // argument checks: every failure path returns an error without touching device memory
    CHECK(fkv_tree_create(nullptr, nullptr) == FKV_ERR_INVALID);
    fkv_attn_args a{};
    CHECK(fkv::validate_attn_common(&a, "decode") == FKV_ERR_INVALID);
    CHECK(fkv::validate_attn_common(nullptr, "decode") == FKV_ERR_INVALID);
    int dummy = 0;
    a.q = a.base_kv = a.out = &dummy;
    a.base_bt = a.seq_lens = &dummy;
    a.n_agents = a.hq = a.hkv = a.max_pages = 1;
    a.d = 64;
    a.page_size = 16;
    a.scale = 0.1f;
    CHECK(fkv::validate_attn_common(&a, "decode") == FKV_ERR_UNSUPPORTED);
    a.d = 128;
    CHECK(fkv::validate_attn_common(&a, "decode") == FKV_OK);
    std::vector<float> c(64 * 64), s(64 * 64);
    CHECK(fkv_rope_table(128, 64, 500000.0, c.data(), s.data()) == FKV_OK);
    CHECK(fkv_rope_table(128, 60, 500000.0, c.data(), s.data()) == FKV_ERR_INVALID);
    for (unsigned seed = 0; seed < 6; ++seed)
        for (int ps : {1, 4, 16})
            if (run_tree(seed * 31 + ps, ps, ps == 16 ? 24 : 90, ps == 16 ? 40 : 140)) return 1;
    std::puts("sanitized host run: ok");
    return 0;
}
