// Decode plan: shared-base segments, work items and the workgroup order.
//
// A segment is a maximal run of logical pages over which a fixed set of agents
// maps every page to the same physical base page (what the base tree's prefix
// sharing produces, Section 5.2).  Each segment is cut into work items of up to
// four agent groups (a group is floor(16 / g) agents: 16 query rows per KV head)
// and a page range.  The split kernel runs one workgroup per (work item, KV head);
// the base tiles of a page range are therefore read once per item and applied to
// all of its agents' query heads.
//
// Workgroup order: on MI355X consecutive workgroup ids are dealt round-robin to
// the 8 XCDs, each with its own L2.  All workgroups that read the same base pages
// (the agent groups of one segment split) or the same rCache rows (the KV heads of
// one item) are placed on one XCD so those re-reads hit that XCD's L2.
#include <algorithm>
#include <cmath>
#include <functional>
#include <queue>
#include <string>
#include <unordered_map>

#include "internal.hpp"

namespace {
constexpr int kNumXcd = 8;
// Estimated time of one item page (in units of a single agent's page) and of an item's
// prologue, used to size and order the work items.
double item_page_cost(int32_t agents) { return 1.0 + 0.095 * (double)agents; }
constexpr double kItemOverhead = 24.0;
}

extern "C" {

fkv_status fkv_decode_plan_create(const fkv_decode_plan_params *prm, const int32_t *base_bt,
                                  const int32_t *res_bt, const int32_t *seq_lens, const int32_t *adapter_idx,
                                  fkv_plan **out) {
    fkv::clear_error();
    if (!prm || !base_bt || !seq_lens || !out) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_create: null argument");
    (void)res_bt;  // page ids, lengths and adapters are read by the kernels at launch
    (void)adapter_idx;
    const int32_t A = prm->n_agents, ps = prm->page_size, mp = prm->max_pages;
    if (A < 1 || prm->hkv < 1 || prm->hq < 1 || ps < 1 || mp < 1 || prm->pages_per_split < 0)
        return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_create: bad sizes");
    if (prm->hq % prm->hkv) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_create: hq % hkv != 0");
    const int32_t g = prm->hq / prm->hkv;
    if (g > fkv::kMaxRows) return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_decode_plan_create: more than 16 query heads per KV head");
    if (prm->r < 0 || prm->max_item_agents < 0) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_create: bad r / max_item_agents");
    const bool rope = prm->rope != 0 && prm->r > 0;
    // agents per group: the slots one wave serves (RoPE) or that fill a 16-row tile
    const int32_t ag = rope ? fkv::decode_rope_wave_agents(g, prm->r) : fkv::kMaxRows / g;
    const int32_t hpb = fkv::decode_heads_per_block(prm->hkv, rope);
    const int32_t cap = fkv::decode_item_agent_cap(g, prm->hkv, prm->r, rope);
    if (cap < 1) return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_decode_plan_create: rank too large for the decode kernels");
    const int32_t item_agents = prm->max_item_agents > 0 ? std::min(prm->max_item_agents, cap) : cap;
    std::vector<int32_t> npages(A);
    int32_t P = 0;
    for (int32_t a = 0; a < A; ++a) {
        if (seq_lens[a] < 1) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_create: seq_len < 1");
        npages[a] = (seq_lens[a] + ps - 1) / ps;
        if (npages[a] > mp) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_create: seq_len exceeds max_pages * page_size");
        P = std::max(P, npages[a]);
    }

    // 1. segments
    struct Seg { int32_t first, n; std::vector<int32_t> agents; };
    std::vector<Seg> segs;
    std::vector<int32_t> open(A, -1);
    std::unordered_map<int32_t, int32_t> group_of_page;
    std::vector<std::vector<int32_t>> groups;
    for (int32_t i = 0; i < P; ++i) {
        group_of_page.clear();
        groups.clear();
        for (int32_t a = 0; a < A; ++a) {
            if (i >= npages[a]) continue;
            const int32_t pg = base_bt[(int64_t)a * mp + i];
            auto it = group_of_page.find(pg);
            if (it == group_of_page.end()) {
                group_of_page.emplace(pg, (int32_t)groups.size());
                groups.push_back({a});
            } else {
                groups[it->second].push_back(a);
            }
        }
        for (auto &gr : groups) {
            const int32_t s = open[gr[0]];
            if (s >= 0 && segs[s].first + segs[s].n == i && segs[s].agents == gr) {
                segs[s].n += 1;
            } else {
                segs.push_back({i, 1, gr});
                for (int32_t a : gr) open[a] = (int32_t)segs.size() - 1;
            }
        }
    }

    // 2. agent chunks per segment: up to item_agents agents, in whole groups of ag where
    //    possible.  With RoPE, chunks of 3 groups are split 2 + 1 (12 agents over a 32K
    //    prefix: 114-117 us against 119-123 us as one item); without RoPE they stay one item,
    //    run as four groups with one idle, so each base page is streamed once instead of
    //    twice (56.1 -> 51.5 us)
    auto chunk_sizes = [&](size_t na) {
        std::vector<size_t> out;
        const size_t full = (size_t)item_agents;
        while (na > 0) {
            size_t c = std::min(na, full);
            const size_t groups = (c + ag - 1) / ag;
            if (groups == 3 && rope) c = std::min(c, (size_t)(2 * ag));
            out.push_back(c);
            na -= c;
        }
        return out;
    };
    // 3. pages per item.
    //    RoPE off: the split kernel keeps two workgroups per compute unit resident.  A page
    //    of an item with more agents costs more (its agents' rCache rows and more
    //    matrix-core work per base byte; about 2.5x a single agent's page at 16 agents, as
    //    measured), and every item pays a fixed prologue worth about 24 pages (see below
    //    for how the split sizes are chosen).  Splits of a segment are equal.
    //    RoPE on: items of 32 pages (see below).
    const int64_t cus = prm->num_cus > 0 ? prm->num_cus : 256;
    const int32_t nhb_units = prm->hkv / hpb;
    std::vector<int32_t> seg_pps(segs.size());
    {
        struct SegCost { int32_t n, cap; double cpp; };  // pages, page limit, cost per page
        std::vector<SegCost> sc(segs.size());
        for (size_t i = 0; i < segs.size(); ++i) {
            const std::vector<size_t> ch = chunk_sizes(segs[i].agents.size());
            double cpp = 0;
            int32_t cap = fkv::kMaxPagesSingle;
            for (size_t c : ch) {  // every chunk is an item of its own: the largest sets the time
                cpp = std::max(cpp, item_page_cost((int32_t)c));
                if ((c + ag - 1) / ag > 2) cap = fkv::kMaxPagesMulti;
            }
            if (rope) cap = fkv::kMaxPagesSingle;
            sc[i] = {segs[i].n, cap, cpp};
        }
        const int64_t slots = std::max<int64_t>(1, 2 * cus / nhb_units);  // items per round
        // Items of three or four agent groups stream every base page through LDS to four
        // waves and are bound by the compute unit's vector-memory issue rate, so two of them
        // on one compute unit slow each other down: they get at most one workgroup per
        // compute unit (pages split evenly over that budget, within their page limit), and
        // at least 12 pages each: below that an item spends most of its time starting up
        // (one KV head, 16 agents sharing 32K tokens: 8-page items 34.1 us per split and
        // merge, 12 pages 28.7, 16 pages 29.7; 2K shared tokens at eight KV heads: 4-page
        // items 45.0 us, 12 pages 36.8).  The other items take a uniform page count, chosen by a simulated greedy longest-first
        // fill of the resident slots (what the dispatcher does with the block order below).
        auto is_multi = [&](size_t i) { return sc[i].cap == fkv::kMaxPagesMulti && !rope; };
        int64_t multi_pages = 0;
        for (size_t i = 0; i < sc.size(); ++i)
            if (is_multi(i)) {
                multi_pages += (int64_t)sc[i].n * (int64_t)chunk_sizes(segs[i].agents.size()).size();
            }
        const int64_t multi_budget = std::max<int64_t>(1, cus / nhb_units);
        constexpr int64_t kMinMultiPages = 12;
        const int32_t multi_pps = multi_pages > 0
            ? (int32_t)std::min<int64_t>(fkv::kMaxPagesMulti, std::max<int64_t>(kMinMultiPages, (multi_pages + multi_budget - 1) / multi_budget))
            : fkv::kMaxPagesMulti;
        std::vector<int32_t> cand_pps(sc.size());
        auto sim = [&](auto &&pages_of) {
            std::vector<double> costs;
            for (size_t i = 0; i < sc.size(); ++i) {
                const int32_t pps_i = pages_of(i);
                const int64_t k = (sc[i].n + pps_i - 1) / pps_i;
                const int32_t pages = (int32_t)((sc[i].n + k - 1) / k);
                for (size_t c : chunk_sizes(segs[i].agents.size()))
                    for (int64_t j = 0; j < k; ++j) costs.push_back(kItemOverhead + pages * item_page_cost((int32_t)c));
            }
            std::sort(costs.begin(), costs.end(), std::greater<double>());
            std::priority_queue<double, std::vector<double>, std::greater<double>> free_at;
            for (int64_t s = 0; s < slots; ++s) free_at.push(0.0);
            double end = 0;
            for (double c : costs) {
                const double t0 = free_at.top();
                free_at.pop();
                free_at.push(t0 + c);
                end = std::max(end, t0 + c);
            }
            return end;
        };
        // The largest page count whose estimate is within 5% of the best (fewer items, fewer
        // partial rows to merge) among those that give every resident slot a workgroup; the
        // simulation sees slots as independent, but a compute unit whose second slot idles
        // streams less than one that runs two workgroups (measured: 448 workgroups of up to
        // 128 pages at the 16-agent, 32K-prefix workload take 3 % longer than 512 of up to
        // 112).  Without such a count, the largest within 1% of the best.
        const int32_t cands[] = {32, 40, 48, 56, 64, 80, 96, 112, 128};
        double est[9], best = 1e300;
        int64_t units[9];
        for (int c = 0; c < 9; ++c) {
            const int32_t u = cands[c];
            auto pages_of = [&](size_t i) { return is_multi(i) ? multi_pps : std::min(u, sc[i].cap); };
            est[c] = sim(pages_of);
            best = std::min(best, est[c]);
            units[c] = 0;
            for (size_t i = 0; i < sc.size(); ++i)
                units[c] += (int64_t)((sc[i].n + pages_of(i) - 1) / pages_of(i)) * (int64_t)chunk_sizes(segs[i].agents.size()).size();
        }
        int32_t best_u = -1;
        for (int c = 8; c >= 0 && best_u < 0; --c)
            if (est[c] <= best * 1.05 && units[c] * nhb_units >= 2 * cus) best_u = cands[c];
        if (best_u < 0 && units[0] * nhb_units * 2 < cus) {
            // a small workload (items of 32 pages would occupy fewer than half the compute
            // units): shorter items shorten the longest chain of pages (4 agents over a
            // 512-token root at two KV heads: 16 workgroups of up to 32 pages -> 32 of up to 4,
            // 12.3 -> 7.9 us; where the 32-page items already occupy most compute units, as
            // for one KV head of 16 agents over 32K, items of 16 pages were slower, 21.3 ->
            // 24.3 us)
            double small_est[3];
            const int32_t small_u[3] = {16, 8, 4};
            for (int c = 0; c < 3; ++c) {
                const int32_t u = small_u[c];
                small_est[c] = sim([&](size_t i) { return is_multi(i) ? multi_pps : std::min(u, sc[i].cap); });
                best = std::min(best, small_est[c]);
            }
            for (int c = 8; c >= 0 && best_u < 0; --c)
                if (est[c] <= best * 1.01) best_u = cands[c];
            for (int c = 0; c < 3 && best_u < 0; ++c)
                if (small_est[c] <= best * 1.01) best_u = small_u[c];
        }
        for (int c = 8; c >= 0 && best_u < 0; --c)
            if (est[c] <= best * 1.01) best_u = cands[c];
        if (best_u < 0) best_u = 64;
        for (size_t i = 0; i < sc.size(); ++i) cand_pps[i] = is_multi(i) ? multi_pps : std::min(best_u, sc[i].cap);
        // RoPE on: the per-page rebuild and rotation of every agent's keys bound the kernel,
        // not the balance of items.  Items of 32 pages (fewer when a segment is shorter) when
        // that gives the two resident workgroups per compute unit few rounds (16 agents over
        // a 32K prefix: 1152 workgroups; 16 to 64 pages within 12 %, 32 best); on larger
        // workloads items of 64 or 128 pages, the largest that still leave at least 2.5
        // workgroups per resident slot: fewer B_K^T builds and partial rows per page (64
        // agents over a 128K tree: 2978 -> 2743 us per step at 128 pages; 70B heads, 24
        // agents: 727 -> 637 us).
        int32_t rope_pages = 32;
        if (rope) {
            auto rope_blocks = [&](int32_t pages) {
                int64_t b = 0;
                for (size_t i = 0; i < segs.size(); ++i)
                    b += (int64_t)((segs[i].n + pages - 1) / pages) * (int64_t)chunk_sizes(segs[i].agents.size()).size();
                return b * nhb_units;
            };
            for (int32_t pages : {64, 128})
                if (rope_blocks(pages) * 2 >= 5 * slots * nhb_units) rope_pages = pages;
            // small workloads: items of 16 or 8 pages when 32 would leave fewer than 1.5
            // workgroups per resident slot (16 agents over a 2K shared prefix: 640 -> 1280
            // workgroups, split and merge 69.1 -> 54.9 us with the spread below)
            if (rope_blocks(32) * 2 < 3 * slots * nhb_units)
                rope_pages = rope_blocks(16) * 2 >= 3 * slots * nhb_units ? 16 : 8;
            // and 4 when even 8-page items occupy fewer than half the compute units (4 agents
            // over a 512-token root: 9.5 -> 7.9 us; one KV head of 16 agents over 32K, 536
            // workgroups of 8 pages: 36.5 us, with 4 pages 46.5)
            if (rope_pages == 8 && rope_blocks(8) * 2 < cus) rope_pages = 4;
        }
        // RoPE on: items of more than one wave group carry most of the work (every page is
        // rebuilt for each of their agents); their pages are spread so that they give every
        // compute unit a workgroup (8 pages an item or more, capped at the size chosen above).
        // One KV head, 16 agents sharing 32K tokens: 64 shared items of 32 pages -> 256 of 8,
        // 84 -> 39 us (36 with the private items at 8 pages too, from the rule above).
        auto is_rope_multi = [&](size_t i) {
            for (size_t c : chunk_sizes(segs[i].agents.size()))
                if ((int64_t)c > ag) return true;
            return false;
        };
        int32_t rope_multi_pages = rope_pages;
        if (rope) {
            int64_t multi = 0;
            for (size_t i = 0; i < segs.size(); ++i)
                if (is_rope_multi(i)) multi += (int64_t)segs[i].n * (int64_t)chunk_sizes(segs[i].agents.size()).size();
            const int64_t budget = std::max<int64_t>(1, cus / nhb_units);
            rope_multi_pages = (int32_t)std::min<int64_t>(rope_pages, std::max<int64_t>(8, (multi + budget - 1) / budget));
        }
        for (size_t i = 0; i < segs.size(); ++i) {
            int32_t pps;
            if (prm->pages_per_split > 0) {
                if (prm->pages_per_split > fkv::kMaxPagesSingle)
                    return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_create: pages_per_split above 128");
                pps = std::min(prm->pages_per_split, sc[i].cap);
            } else {
                const int32_t target = rope ? (is_rope_multi(i) ? rope_multi_pages : rope_pages) : cand_pps[i];
                const int64_t k = (segs[i].n + target - 1) / target;
                pps = (int32_t)((segs[i].n + k - 1) / k);
            }
            seg_pps[i] = pps;
        }
    }

    // 4. work items, clustered by (segment, split).  An item of ng agent groups runs its
    //    groups on 4 / ngp wave copies (ngp = ng rounded up to 1, 2 or 4); the copies of a
    //    group merge their partial rows inside the workgroup, so every slot owns one partial
    //    (the `copies` field of an item: partials per slot, 1): rows = agents * g.
    struct Item {
        int32_t p0, p1, cap, copies;
        double cost;
        std::vector<int32_t> agents;
        bool solo;  // no other item reads its base pages (one item per split of its segment)
    };
    std::vector<Item> items;
    std::vector<std::pair<int32_t, int32_t>> clusters;  // [first item, item count)
    std::vector<double> cluster_cost;
    int64_t total_rows = 0;
    int32_t pps_max = 0;
    for (size_t si = 0; si < segs.size(); ++si) {
        const auto &s = segs[si];
        const int32_t pps = seg_pps[si];
        pps_max = std::max(pps_max, pps);
        const std::vector<size_t> chunks = chunk_sizes(s.agents.size());
        for (int32_t p0 = s.first; p0 < s.first + s.n; p0 += pps) {
            const int32_t p1 = std::min(p0 + pps, s.first + s.n);
            const int32_t first = (int32_t)items.size();
            double cost = 0;
            size_t k = 0;
            for (size_t c : chunks) {
                Item it{p0, p1, p1, 1, 0.0, {}, chunks.size() == 1};
                for (size_t j = k; j < k + c; ++j) it.agents.push_back(s.agents[j]);
                k += c;
                total_rows += (int64_t)it.copies * (int64_t)c * g;
                it.cost = kItemOverhead + (double)(p1 - p0) * item_page_cost((int32_t)c);
                cost += it.cost;
                items.push_back(std::move(it));
            }
            clusters.push_back({first, (int32_t)items.size() - first});
            cluster_cost.push_back(cost);
        }
    }
    // 4b. growth room for decode steps: each agent's last item may read up to `reserve` more
    //     pages (as far as its block-table row reaches) when the agent's length grows, so the
    //     plan stays valid while agents append tokens.  A last item that is the agent's alone
    //     and has room under its page limit is extended; otherwise the agent gets a tail item
    //     of its own that starts empty.
    const int32_t reserve = prm->reserve_pages == 0 ? fkv::kDefaultReservePages : std::max<int32_t>(0, prm->reserve_pages);
    std::vector<int32_t> last_item(A, -1);
    for (size_t i = 0; i < items.size(); ++i)
        for (int32_t a : items[i].agents)
            if (items[i].p1 == npages[a]) last_item[a] = (int32_t)i;
    std::vector<int32_t> cap_pages(npages);
    for (int32_t a = 0; a < A; ++a) {
        const int32_t room = std::min(reserve, mp - npages[a]);
        if (room <= 0) continue;
        Item &last = items[last_item[a]];
        const int32_t limit = fkv::kMaxPagesSingle;
        if (last.agents.size() == 1 && last.p1 - last.p0 + room <= limit) {
            last.cap = last.p1 + room;
        } else {
            const int32_t first = (int32_t)items.size();
            Item it{npages[a], npages[a], npages[a] + room, 1, kItemOverhead, {a}, true};
            total_rows += (int64_t)it.copies * g;
            items.push_back(std::move(it));
            clusters.push_back({first, 1});
            cluster_cost.push_back(kItemOverhead);
        }
        cap_pages[a] = npages[a] + room;
    }
    for (const auto &it : items) pps_max = std::max(pps_max, it.cap - it.p0);
    if (total_rows * prm->hkv > INT32_MAX) return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_decode_plan_create: too many rows");
    const int32_t n_items = (int32_t)items.size();
    const int32_t hkv = prm->hkv;

    // 5. workgroup order: clusters dealt to XCDs by least accumulated cost (all heads of a
    //    cluster on one XCD), then each XCD's units longest-first so the dispatcher's greedy
    //    fill is a longest-processing-time schedule
    std::vector<std::vector<int32_t>> per_xcd(kNumXcd);
    std::vector<double> load(kNumXcd, 0.0);
    std::vector<int32_t> order(clusters.size());
    for (size_t c = 0; c < clusters.size(); ++c) order[c] = (int32_t)c;
    std::stable_sort(order.begin(), order.end(), [&](int32_t x, int32_t y) { return cluster_cost[x] > cluster_cost[y]; });
    const int32_t nhb = hkv / hpb;  // head blocks per item
    for (int32_t c : order) {
        const int32_t x = (int32_t)(std::min_element(load.begin(), load.end()) - load.begin());
        load[x] += cluster_cost[c] * hkv;
        auto &lst = per_xcd[x];
        for (int32_t hb = 0; hb < nhb; ++hb)
            for (int32_t k = 0; k < clusters[c].second; ++k) lst.push_back((clusters[c].first + k) * nhb + hb);
    }
    for (auto &lst : per_xcd)
        std::stable_sort(lst.begin(), lst.end(),
                         [&](int32_t x, int32_t y) { return items[x / nhb].cost > items[y / nhb].cost; });
    size_t depth = 0;
    for (auto &l : per_xcd) depth = std::max(depth, l.size());
    const int32_t n_blocks = (int32_t)(depth * kNumXcd);

    // 6. partials, contiguous per agent (CSR): agent a owns [ptr[a], ptr[a+1]); slot j of an
    //    item writes partial first[j]
    std::vector<int32_t> ptr(A + 1, 0);
    for (const auto &it : items)
        for (int32_t a : it.agents) ptr[a + 1] += it.copies;
    for (int32_t a = 0; a < A; ++a) ptr[a + 1] += ptr[a];
    std::vector<int32_t> next(ptr.begin(), ptr.end() - 1);
    std::vector<std::vector<int32_t>> first(n_items);
    for (int32_t w = 0; w < n_items; ++w)
        for (int32_t a : items[w].agents) {
            first[w].push_back(next[a]);
            next[a] += items[w].copies;
        }

    // 7. serialise
    auto *pl = new fkv_plan();
    pl->hkv = hkv;
    pl->g = g;
    pl->n_agents = A;
    pl->page_size = ps;
    pl->max_pages = mp;
    pl->cap_pages = cap_pages;
    pl->max_pages_used = *std::max_element(cap_pages.begin(), cap_pages.end());
    const int64_t off_items = fkv::kHeaderWords;
    const int64_t off_blocks = off_items + (int64_t)n_items * fkv::kItemWords;
    const int64_t off_ptr = off_blocks + n_blocks;
    const int64_t off_zero = (off_ptr + A + 1 + 3) / 4 * 4;
    const int64_t off_desc = off_zero + fkv::kZeroWords;
    const int64_t total = off_desc + (int64_t)n_blocks * fkv::kDescWords;
    if (total > INT32_MAX) {
        delete pl;
        return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_decode_plan_create: plan too large");
    }
    auto &w = pl->words;
    w.assign(total, 0);
    w[fkv::H_MAGIC] = fkv::kPlanMagic;
    w[fkv::H_N_ITEMS] = n_items;
    w[fkv::H_N_BLOCKS] = n_blocks;
    w[fkv::H_N_AGENTS] = A;
    w[fkv::H_HKV] = hkv;
    w[fkv::H_GROUP] = g;
    w[fkv::H_AGENTS_PER_ITEM] = ag;
    w[fkv::H_OFF_ITEMS] = (int32_t)off_items;
    w[fkv::H_OFF_BLOCKS] = (int32_t)off_blocks;
    w[fkv::H_OFF_AGENT_PTR] = (int32_t)off_ptr;
    w[fkv::H_OFF_AGENT_SLOT] = (int32_t)off_zero;
    w[fkv::H_TOTAL_WORDS] = (int32_t)total;
    w[fkv::H_PAGES_PER_SPLIT] = pps_max;
    w[fkv::H_PAGE_SIZE] = ps;
    w[fkv::H_N_SEGMENTS] = (int32_t)segs.size();
    w[fkv::H_TOTAL_ROWS] = (int32_t)total_rows;
    w[fkv::H_MAX_ITEM_AGENTS] = item_agents;
    w[fkv::H_HEADS_PER_BLOCK] = hpb;
    w[fkv::H_RANK] = prm->r;
    w[fkv::H_ROPE] = rope ? 1 : 0;
    w[fkv::H_OFF_ZERO] = (int32_t)off_zero;
    w[fkv::H_OFF_DESC] = (int32_t)off_desc;
    for (int32_t i = 0; i < n_items; ++i) {
        int32_t *r = &w[off_items + (int64_t)i * fkv::kItemWords];
        const int32_t nag = (int32_t)items[i].agents.size();
        r[fkv::kItemP0] = items[i].p0;
        r[fkv::kItemCap] = items[i].cap;
        r[fkv::kItemLeader] = items[i].agents[0];
        r[fkv::kItemNag] = nag;
        r[fkv::kItemCopies] = items[i].copies;
        r[fkv::kItemEnd] = items[i].p1;
        for (int32_t j = 0; j < fkv::kMaxItemAgents; ++j) {
            r[fkv::kItemAgents + j] = j < nag ? items[i].agents[j] : -1;
            r[fkv::kItemFirst + j] = j < nag ? first[i][j] : -1;
        }
    }
    for (int32_t b = 0; b < n_blocks; ++b) {
        const auto &lst = per_xcd[b % kNumXcd];
        const size_t k = (size_t)(b / kNumXcd);
        w[off_blocks + b] = k < lst.size() ? lst[k] : -1;
    }
    for (int32_t a = 0; a <= A; ++a) w[off_ptr + a] = ptr[a];
    {
        // block descriptors: the item a block serves, at an address that depends on the block
        // index only (the kernel's first load)
        for (int32_t b = 0; b < n_blocks; ++b) {
            int32_t *d = &w[off_desc + (int64_t)b * fkv::kDescWords];
            const int32_t blk = w[off_blocks + b];
            if (blk < 0) continue;  // idle: nag = 0
            const int32_t i = blk / nhb;
            const Item &it = items[i];
            const int32_t nag = (int32_t)it.agents.size();
            d[fkv::kDescPg0] = it.p0;
            d[fkv::kDescCap] = it.cap;
            d[fkv::kDescNag] = nag;
            d[fkv::kDescHead] = (blk % nhb) * hpb;
            d[fkv::kDescLeader] = it.agents[0];
            d[fkv::kDescItem] = i;
            d[fkv::kDescCopies] = it.copies;
            d[fkv::kDescStream] = it.solo ? 1 : 0;
            for (int32_t j = 0; j < nag; ++j) {
                d[fkv::kDescAgent + j] = it.agents[j];
                d[fkv::kDescPart + j] = first[i][j];
            }
        }
    }
    for (auto &s : segs) {
        pl->seg_first_page.push_back(s.first);
        pl->seg_n_pages.push_back(s.n);
        pl->seg_agent_off.push_back((int32_t)pl->seg_agents.size());
        pl->seg_agents.insert(pl->seg_agents.end(), s.agents.begin(), s.agents.end());
    }
    *out = pl;
    return FKV_OK;
}

void fkv_decode_plan_destroy(fkv_plan *plan) { delete plan; }

fkv_status fkv_decode_plan_covers(const fkv_plan *plan, const int32_t *seq_lens, int32_t n_agents) {
    fkv::clear_error();
    if (!plan || !seq_lens) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_covers: null argument");
    if (n_agents != plan->n_agents) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_covers: agent count differs from the plan's");
    for (int32_t a = 0; a < n_agents; ++a) {
        const int64_t cap = (int64_t)plan->cap_pages[a] * plan->page_size;
        if (seq_lens[a] < 1 || seq_lens[a] > cap)
            return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_covers: agent " + std::to_string(a) + " has length " +
                                                  std::to_string(seq_lens[a]) + ", the plan covers 1.." +
                                                  std::to_string(cap) + ": build a new plan");
    }
    return FKV_OK;
}

fkv_status fkv_decode_plan_capacity(const fkv_plan *plan, int32_t agent, int64_t *max_len) {
    fkv::clear_error();
    if (!plan || !max_len || agent < 0 || agent >= plan->n_agents)
        return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_capacity: bad argument");
    *max_len = (int64_t)plan->cap_pages[agent] * plan->page_size;
    return FKV_OK;
}

}  // extern "C"

namespace fkv {
int64_t decode_partials_bytes(const fkv_plan *plan, int32_t d, int32_t r) {
    const int64_t stride = (int64_t)(d + r + 2 + 3) / 4 * 4;
    const int64_t bytes = (int64_t)plan->words[H_TOTAL_ROWS] * plan->hkv * stride * 4;
    return (bytes + 255) / 256 * 256;
}
}  // namespace fkv

extern "C" {

fkv_status fkv_decode_plan_info(const fkv_plan *plan, int32_t d, int32_t r, fkv_plan_info *out) {
    fkv::clear_error();
    if (!plan || !out || d < 1 || r < 0) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_info: bad argument");
    const auto &w = plan->words;
    out->plan_words = (int64_t)w.size();
    out->n_items = w[fkv::H_N_ITEMS];
    out->n_blocks = w[fkv::H_N_BLOCKS];
    out->n_segments = w[fkv::H_N_SEGMENTS];
    out->pages_per_split = w[fkv::H_PAGES_PER_SPLIT];
    out->workspace_bytes = fkv::decode_partials_bytes(plan, d, r);
    return FKV_OK;
}

int32_t fkv_decode_plan_default_agents(int32_t hq, int32_t hkv, int32_t r, int32_t rope) {
    if (hq < 1 || hkv < 1 || hq % hkv) return 0;
    const int32_t g = hq / hkv;
    if (g > fkv::kMaxRows) return 0;
    // Without RoPE the residual key term is one small product per page and agent, so a
    // workgroup serves up to four groups from each staged base page (as many agents as
    // fit one LDS stage).  With RoPE the per-page rebuild (Stage 1 plus the rotation)
    // dominates: each wave serves the agents whose rebuilt keys fit its registers, and an
    // item holds as many such wave groups as 64 KB of B_K^T fragments in LDS allow.
    if (r < 0) return 0;
    return fkv::decode_item_agent_cap(g, hkv, r, rope != 0 && r > 0);
}

fkv_status fkv_decode_plan_serialize(const fkv_plan *plan, int32_t *out, int64_t capacity_words) {
    fkv::clear_error();
    if (!plan || !out) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_serialize: null argument");
    if (capacity_words < (int64_t)plan->words.size())
        return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_serialize: buffer too small");
    std::copy(plan->words.begin(), plan->words.end(), out);
    return FKV_OK;
}

fkv_status fkv_decode_plan_segments(const fkv_plan *plan, int32_t *first_page, int32_t *n_pages,
                                    int32_t *n_agents, int32_t *agents, int64_t cap) {
    fkv::clear_error();
    if (!plan || !first_page || !n_pages || !n_agents || !agents)
        return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_segments: null argument");
    if (cap < (int64_t)plan->seg_agents.size()) return fkv::fail(FKV_ERR_INVALID, "fkv_decode_plan_segments: buffer too small");
    const size_t ns = plan->seg_first_page.size();
    for (size_t s = 0; s < ns; ++s) {
        first_page[s] = plan->seg_first_page[s];
        n_pages[s] = plan->seg_n_pages[s];
        const int32_t e = s + 1 < ns ? plan->seg_agent_off[s + 1] : (int32_t)plan->seg_agents.size();
        n_agents[s] = e - plan->seg_agent_off[s];
    }
    std::copy(plan->seg_agents.begin(), plan->seg_agents.end(), agents);
    return FKV_OK;
}

}  // extern "C"
