// DualRadixTree: page pools and fork / copy-on-write bookkeeping for the two
// caches of ForkKV (Section 5.2).
//
// Each cache has its own radix tree whose edges are single pages: a node owns one
// physical page and the (at most page_size) token ids stored in it.  The base
// tree has one root (key = token ids); the residual tree has one root per agent
// id (key = agent id + token ids, so residual pages never alias across agents).
// A sequence is a path of nodes, one per logical page.  Nodes that no sequence
// references stay cached and are evicted least-recently-used first, each tree
// on its own (the decoupled eviction policy of Section 5.2).
#include <algorithm>
#include <cstring>
#include <queue>
#include <set>
#include <unordered_map>
#include <unordered_set>

#include "internal.hpp"

namespace {

struct Node {
    int32_t page = -1;
    std::vector<int32_t> tokens;
    Node *parent = nullptr;
    std::vector<Node *> children;
    int32_t ref = 0;
    uint64_t last_use = 0;
};

class PageTrie {
public:
    PageTrie(int32_t ps, int32_t capacity) : ps_(ps), capacity_(capacity) {
        for (int32_t i = 0; i < capacity; ++i) free_.insert(i);
    }
    ~PageTrie() {
        for (Node *n : nodes_) delete n;
        for (auto &kv : roots_) delete kv.second;
    }
    PageTrie(const PageTrie &) = delete;
    PageTrie &operator=(const PageTrie &) = delete;

    Node *root(int64_t ns) const {
        auto it = roots_.find(ns);
        return it == roots_.end() ? nullptr : it->second;
    }
    Node *root_create(int64_t ns) {
        Node *&r = roots_[ns];
        if (!r) r = new Node();
        return r;
    }

    // Longest-prefix walk.  `shared` receives the nodes whose tokens cover the next
    // chunk of the query exactly (a final chunk shorter than a page may share a page
    // that holds more tokens: the sequence reads only its own prefix of it).  If the
    // walk stops at a page that matches only k > 0 of the next chunk's tokens, that
    // page is returned as the copy-on-write source for k tokens.
    struct Walk {
        std::vector<Node *> shared;
        int64_t shared_tokens = 0;
        Node *cow_src = nullptr;
        int32_t cow_k = 0;
    };
    Walk walk(Node *root, const int32_t *t, int64_t n) const {
        Walk w;
        if (!root) return w;
        Node *cur = root;
        int64_t pos = 0;
        while (pos < n) {
            const int32_t m = (int32_t)std::min<int64_t>(ps_, n - pos);
            Node *best = nullptr;
            int32_t best_k = 0;
            for (Node *c : cur->children) {
                const int32_t lim = std::min<int32_t>(m, (int32_t)c->tokens.size());
                int32_t k = 0;
                while (k < lim && c->tokens[k] == t[pos + k]) ++k;
                if (k > best_k) { best = c; best_k = k; }
                if (best_k == m) break;
            }
            if (!best) break;
            if (best_k == m) {
                w.shared.push_back(best);
                w.shared_tokens += m;
                pos += m;
                cur = best;
                if (m < ps_) break;
                continue;
            }
            w.cow_src = best;
            w.cow_k = best_k;
            break;
        }
        return w;
    }

    int32_t n_free() const { return (int32_t)free_.size(); }
    int32_t n_unref() const { return n_unref_; }
    int32_t n_nodes() const { return (int32_t)nodes_.size(); }
    int32_t n_raw() const { return (int32_t)raw_.size(); }
    int64_t evictions() const { return evictions_; }
    int32_t capacity() const { return capacity_; }

    void acquire(Node *x) {
        if (x->ref == 0) --n_unref_;
        ++x->ref;
        x->last_use = ++clock_;
    }
    void release(Node *x) {
        --x->ref;
        if (x->ref == 0) ++n_unref_;
        x->last_use = ++clock_;
    }

    // Make sure `need` pages are free, evicting unreferenced leaves LRU-first.
    // Callers check feasibility first (need <= n_free() + evictable).
    bool ensure_free(int32_t need) {
        if (n_free() >= need) return true;
        using Item = std::pair<uint64_t, Node *>;
        auto cmp = [](const Item &a, const Item &b) {
            return a.first != b.first ? a.first > b.first : a.second->page > b.second->page;
        };
        std::priority_queue<Item, std::vector<Item>, decltype(cmp)> heap(cmp);
        for (Node *x : nodes_)
            if (x->ref == 0 && x->children.empty()) heap.push({x->last_use, x});
        while (n_free() < need && !heap.empty()) {
            Node *x = heap.top().second;
            heap.pop();
            Node *p = x->parent;
            auto &sib = p->children;
            sib.erase(std::find(sib.begin(), sib.end(), x));
            free_.insert(x->page);
            nodes_.erase(x);
            --n_unref_;
            ++evictions_;
            delete x;
            if (p->page >= 0 && p->ref == 0 && p->children.empty()) heap.push({p->last_use, p});
        }
        return n_free() >= need;
    }

    int32_t take_page() {
        auto it = free_.begin();
        const int32_t id = *it;
        free_.erase(it);
        return id;
    }

    // New node holding `tokens`, child of `parent`, referenced once.
    Node *add_node(Node *parent, const int32_t *tokens, int32_t m) {
        Node *x = new Node();
        x->page = take_page();
        x->tokens.assign(tokens, tokens + m);
        x->parent = parent;
        x->ref = 1;
        x->last_use = ++clock_;
        parent->children.push_back(x);
        nodes_.insert(x);
        return x;
    }

    bool alloc_raw(int32_t n, int32_t *out) {
        if (n > n_free() + n_unref_) return false;
        ensure_free(n);
        for (int32_t i = 0; i < n; ++i) {
            out[i] = take_page();
            raw_.insert(out[i]);
        }
        return true;
    }
    bool free_raw(int32_t n, const int32_t *ids) {
        for (int32_t i = 0; i < n; ++i)
            if (!raw_.count(ids[i])) return false;
        std::unordered_set<int32_t> seen;
        for (int32_t i = 0; i < n; ++i)
            if (!seen.insert(ids[i]).second) return false;
        for (int32_t i = 0; i < n; ++i) {
            raw_.erase(ids[i]);
            free_.insert(ids[i]);
        }
        return true;
    }
    int32_t page_size() const { return ps_; }

private:
    int32_t ps_, capacity_;
    std::set<int32_t> free_;
    std::unordered_set<Node *> nodes_;
    std::unordered_map<int64_t, Node *> roots_;
    std::unordered_set<int32_t> raw_;
    int32_t n_unref_ = 0;
    uint64_t clock_ = 0;
    int64_t evictions_ = 0;
};

struct Seq {
    int32_t agent = 0;
    int64_t len = 0;
    std::vector<Node *> path[2];  // base, residual
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

struct fkv_tree {
    int32_t ps;
    PageTrie trie[2];
    std::unordered_map<int32_t, Seq> seqs;
    fkv_tree(int32_t page_size, int32_t nb, int32_t nr) : ps(page_size), trie{{page_size, nb}, {page_size, nr}} {}
};

namespace {

// Pages a fork needs from one trie, and the nodes it will reference.
struct ForkPart {
    PageTrie::Walk w;
    int32_t new_pages = 0;
    int32_t protect = 0;  // unreferenced nodes the walk will pin (not evictable during this call)
};

ForkPart plan_fork(const PageTrie &t, Node *root, const int32_t *tok, int64_t n) {
    ForkPart f;
    f.w = t.walk(root, tok, n);
    f.new_pages = (int32_t)(ceil_div(n, t.page_size()) - (int64_t)f.w.shared.size());
    for (Node *x : f.w.shared) f.protect += x->ref == 0;
    if (f.w.cow_src && f.w.cow_src->ref == 0) f.protect += 1;
    return f;
}

void run_fork(PageTrie &t, Node *root, const int32_t *tok, int64_t n, const ForkPart &f, int32_t pool,
              std::vector<Node *> &path, int64_t &valid, fkv_fill_plan *out) {
    const int32_t ps = t.page_size();
    for (Node *x : f.w.shared) t.acquire(x);
    if (f.w.cow_src) t.acquire(f.w.cow_src);  // pinned while pages are allocated
    t.ensure_free(f.new_pages);
    path = f.w.shared;
    Node *cur = path.empty() ? root : path.back();
    int64_t pos = f.w.shared_tokens;
    valid = pos;
    if (f.w.cow_src) {
        const int32_t m = (int32_t)std::min<int64_t>(ps, n - pos);
        Node *x = t.add_node(cur, tok + pos, m);
        fkv_page_copy &c = out->copies[out->n_copies++];
        c.pool = pool;
        c.src = f.w.cow_src->page;
        c.dst = x->page;
        c.n_valid = f.w.cow_k;
        valid += f.w.cow_k;
        t.release(f.w.cow_src);
        path.push_back(x);
        cur = x;
        pos += m;
    }
    while (pos < n) {
        const int32_t m = (int32_t)std::min<int64_t>(ps, n - pos);
        Node *x = t.add_node(cur, tok + pos, m);
        path.push_back(x);
        cur = x;
        pos += m;
    }
}

// Pages an append of n tokens needs from one trie.
int32_t append_pages(const std::vector<Node *> &path, int64_t len, int64_t n, int32_t ps, bool *in_place) {
    const int32_t k = (int32_t)(len % ps);
    int64_t rest = n;
    int32_t need = 0;
    *in_place = false;
    if (k != 0 && n > 0) {
        Node *last = path.back();
        *in_place = last->ref == 1 && (int32_t)last->tokens.size() == k;
        need += *in_place ? 0 : 1;
        rest -= std::min<int64_t>(ps - k, n);
    }
    return need + (int32_t)ceil_div(rest, ps);
}

void run_append(PageTrie &t, std::vector<Node *> &path, int64_t len, const int32_t *tok, int64_t n,
                bool in_place, int32_t pool, fkv_fill_plan *out) {
    const int32_t ps = t.page_size();
    const int32_t k = (int32_t)(len % ps);
    int64_t pos = 0;
    if (k != 0 && n > 0) {
        const int32_t m = (int32_t)std::min<int64_t>(ps - k, n);
        Node *last = path.back();
        if (in_place) {
            last->tokens.insert(last->tokens.end(), tok, tok + m);
            t.acquire(last);
            t.release(last);
        } else {
            std::vector<int32_t> merged(last->tokens.begin(), last->tokens.begin() + k);
            merged.insert(merged.end(), tok, tok + m);
            Node *x = t.add_node(last->parent, merged.data(), (int32_t)merged.size());
            fkv_page_copy &c = out->copies[out->n_copies++];
            c.pool = pool;
            c.src = last->page;
            c.dst = x->page;
            c.n_valid = k;
            t.release(last);
            path.back() = x;
        }
        pos = m;
    }
    while (pos < n) {
        const int32_t m = (int32_t)std::min<int64_t>(ps, n - pos);
        Node *x = t.add_node(path.back(), tok + pos, m);
        path.push_back(x);
        pos += m;
    }
}

}  // namespace

extern "C" {

fkv_status fkv_tree_create(const fkv_tree_config *cfg, fkv_tree **out) {
    fkv::clear_error();
    if (!cfg || !out) return fkv::fail(FKV_ERR_INVALID, "fkv_tree_create: null argument");
    if (cfg->page_size < 1 || cfg->page_size > 1024)
        return fkv::fail(FKV_ERR_INVALID, "fkv_tree_create: page_size must be in 1..1024");
    if (cfg->num_base_pages < 0 || cfg->num_res_pages < 0)
        return fkv::fail(FKV_ERR_INVALID, "fkv_tree_create: negative pool size");
    *out = new fkv_tree(cfg->page_size, cfg->num_base_pages, cfg->num_res_pages);
    return FKV_OK;
}

void fkv_tree_destroy(fkv_tree *tree) { delete tree; }

fkv_status fkv_alloc_pages(fkv_tree *tree, int32_t pool, int32_t n, int32_t *out_ids) {
    fkv::clear_error();
    if (!tree || (n > 0 && !out_ids) || n < 0 || (pool != FKV_POOL_BASE && pool != FKV_POOL_RES))
        return fkv::fail(FKV_ERR_INVALID, "fkv_alloc_pages: bad argument");
    if (!tree->trie[pool].alloc_raw(n, out_ids))
        return fkv::fail(FKV_ERR_OOM, "fkv_alloc_pages: pool exhausted");
    return FKV_OK;
}

fkv_status fkv_free_pages(fkv_tree *tree, int32_t pool, int32_t n, const int32_t *ids) {
    fkv::clear_error();
    if (!tree || (n > 0 && !ids) || n < 0 || (pool != FKV_POOL_BASE && pool != FKV_POOL_RES))
        return fkv::fail(FKV_ERR_INVALID, "fkv_free_pages: bad argument");
    if (!tree->trie[pool].free_raw(n, ids))
        return fkv::fail(FKV_ERR_INVALID, "fkv_free_pages: id not allocated by fkv_alloc_pages (or repeated)");
    return FKV_OK;
}

fkv_status fkv_fork(fkv_tree *tree, int32_t seq_id, int32_t agent_id, const int32_t *tokens, int64_t n,
                    fkv_fill_plan *out) {
    fkv::clear_error();
    if (!tree || !tokens || !out || n < 1) return fkv::fail(FKV_ERR_INVALID, "fkv_fork: bad argument");
    if (tree->seqs.count(seq_id)) return fkv::fail(FKV_ERR_EXISTS, "fkv_fork: sequence id already in use");
    PageTrie &bt = tree->trie[FKV_POOL_BASE];
    PageTrie &rt = tree->trie[FKV_POOL_RES];
    Node *broot = bt.root_create(0);
    ForkPart fb = plan_fork(bt, broot, tokens, n);
    ForkPart fr = plan_fork(rt, rt.root(agent_id), tokens, n);
    if (fb.new_pages > bt.n_free() + bt.n_unref() - fb.protect)
        return fkv::fail(FKV_ERR_OOM, "fkv_fork: base pool exhausted");
    if (fr.new_pages > rt.n_free() + rt.n_unref() - fr.protect)
        return fkv::fail(FKV_ERR_OOM, "fkv_fork: residual pool exhausted");
    std::memset(out, 0, sizeof(*out));
    Seq s;
    s.agent = agent_id;
    s.len = n;
    run_fork(bt, broot, tokens, n, fb, FKV_POOL_BASE, s.path[0], out->base_valid, out);
    run_fork(rt, rt.root_create(agent_id), tokens, n, fr, FKV_POOL_RES, s.path[1], out->res_valid, out);
    out->seq_len = n;
    tree->seqs.emplace(seq_id, std::move(s));
    return FKV_OK;
}

fkv_status fkv_cow_append(fkv_tree *tree, int32_t seq_id, const int32_t *tokens, int64_t n, fkv_fill_plan *out) {
    fkv::clear_error();
    if (!tree || (n > 0 && !tokens) || !out || n < 0) return fkv::fail(FKV_ERR_INVALID, "fkv_cow_append: bad argument");
    auto it = tree->seqs.find(seq_id);
    if (it == tree->seqs.end()) return fkv::fail(FKV_ERR_NOT_FOUND, "fkv_cow_append: unknown sequence");
    Seq &s = it->second;
    bool in_place[2];
    int32_t need[2];
    for (int i = 0; i < 2; ++i) {
        need[i] = append_pages(s.path[i], s.len, n, tree->ps, &in_place[i]);
        if (need[i] > tree->trie[i].n_free() + tree->trie[i].n_unref())
            return fkv::fail(FKV_ERR_OOM, i == 0 ? "fkv_cow_append: base pool exhausted"
                                                 : "fkv_cow_append: residual pool exhausted");
    }
    std::memset(out, 0, sizeof(*out));
    for (int i = 0; i < 2; ++i) {
        tree->trie[i].ensure_free(need[i]);
        run_append(tree->trie[i], s.path[i], s.len, tokens, n, in_place[i], i, out);
    }
    out->base_valid = out->res_valid = s.len;
    s.len += n;
    out->seq_len = s.len;
    return FKV_OK;
}

fkv_status fkv_release(fkv_tree *tree, int32_t seq_id) {
    fkv::clear_error();
    if (!tree) return fkv::fail(FKV_ERR_INVALID, "fkv_release: null tree");
    auto it = tree->seqs.find(seq_id);
    if (it == tree->seqs.end()) return fkv::fail(FKV_ERR_NOT_FOUND, "fkv_release: unknown sequence");
    for (int i = 0; i < 2; ++i)
        for (auto p = it->second.path[i].rbegin(); p != it->second.path[i].rend(); ++p) tree->trie[i].release(*p);
    tree->seqs.erase(it);
    return FKV_OK;
}

fkv_status fkv_seq_info(const fkv_tree *tree, int32_t seq_id, int64_t *seq_len, int32_t *n_pages) {
    fkv::clear_error();
    if (!tree) return fkv::fail(FKV_ERR_INVALID, "fkv_seq_info: null tree");
    auto it = tree->seqs.find(seq_id);
    if (it == tree->seqs.end()) return fkv::fail(FKV_ERR_NOT_FOUND, "fkv_seq_info: unknown sequence");
    if (seq_len) *seq_len = it->second.len;
    if (n_pages) *n_pages = (int32_t)it->second.path[0].size();
    return FKV_OK;
}

fkv_status fkv_get_block_tables(const fkv_tree *tree, const int32_t *seq_ids, int32_t n, int32_t max_pages,
                                int32_t *base_bt, int32_t *res_bt, int32_t *seq_lens) {
    fkv::clear_error();
    if (!tree || n < 0 || max_pages < 1 || (n > 0 && (!seq_ids || !base_bt || !res_bt || !seq_lens)))
        return fkv::fail(FKV_ERR_INVALID, "fkv_get_block_tables: bad argument");
    for (int32_t i = 0; i < n; ++i) {
        auto it = tree->seqs.find(seq_ids[i]);
        if (it == tree->seqs.end()) return fkv::fail(FKV_ERR_NOT_FOUND, "fkv_get_block_tables: unknown sequence");
        if ((int64_t)it->second.path[0].size() > max_pages)
            return fkv::fail(FKV_ERR_INVALID, "fkv_get_block_tables: sequence longer than max_pages pages");
        if (it->second.len > INT32_MAX) return fkv::fail(FKV_ERR_INVALID, "fkv_get_block_tables: sequence too long");
    }
    for (int32_t i = 0; i < n; ++i) {
        const Seq &s = tree->seqs.find(seq_ids[i])->second;
        int32_t *b = base_bt + (int64_t)i * max_pages;
        int32_t *r = res_bt + (int64_t)i * max_pages;
        for (int32_t p = 0; p < max_pages; ++p) {
            b[p] = p < (int32_t)s.path[0].size() ? s.path[0][p]->page : 0;
            r[p] = p < (int32_t)s.path[1].size() ? s.path[1][p]->page : 0;
        }
        seq_lens[i] = (int32_t)s.len;
    }
    return FKV_OK;
}

fkv_status fkv_get_pool_stats(const fkv_tree *tree, fkv_pool_stats *out) {
    fkv::clear_error();
    if (!tree || !out) return fkv::fail(FKV_ERR_INVALID, "fkv_get_pool_stats: null argument");
    const PageTrie &b = tree->trie[0], &r = tree->trie[1];
    out->base_pages_free = b.n_free();
    out->base_pages_cached = b.n_unref();
    out->base_pages_raw = b.n_raw();
    out->base_pages_referenced = b.n_nodes() - b.n_unref();
    out->res_pages_free = r.n_free();
    out->res_pages_cached = r.n_unref();
    out->res_pages_raw = r.n_raw();
    out->res_pages_referenced = r.n_nodes() - r.n_unref();
    out->n_sequences = (int32_t)tree->seqs.size();
    out->base_evictions = b.evictions();
    out->res_evictions = r.evictions();
    return FKV_OK;
}

}  // extern "C"
