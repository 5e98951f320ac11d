/*
 * forkkv.h -- C ABI of the MI355X (gfx950) ResidualAttention library.
 *
 * ForkKV (arXiv 2604.06370) splits the KV cache of many LoRA agents into a
 * shared base cache (bCache = xW, RoPE'd keys, Section 5.1) and a small
 * per-agent residual cache (rCache = xA_i, r values per token for K and for V,
 * Section 2.2, Eq. 2).  This library provides
 *   - the host-side DualRadixTree that hands out pages of both caches with fork
 *     and copy-on-write semantics (Section 5.2), and
 *   - ResidualAttention kernels for decode and chunked prefill (Section 5.3,
 *     Algorithm 1) that rebuild each agent's keys as
 *         K = K_base + RoPE(C_K . B_K)
 *     on chip and fold the value residual in rank space,
 *         O = (sum_p P_p V_base,p + (sum_p P_p C_V,p) . B_V) / l        (Eq. 4),
 *     never writing a reconstructed K or V to memory.
 *
 * Conventions
 *   - Every call returns fkv_status: 0 on success, a negative FKV_ERR_* code on
 *     failure; fkv_last_error() then returns a message (thread-local, valid
 *     until the next failing call on that thread).
 *   - Host-side tree calls are single-threaded per tree (the scheduler owns the
 *     tree).  A failing tree call leaves the tree unchanged.
 *   - Device memory is owned by the caller: pools, queries, outputs, block
 *     tables, plans and workspaces are caller allocations.  The library
 *     allocates no device memory and never synchronises; kernels are enqueued on
 *     the caller's stream (a hipStream_t passed as void*; NULL = null stream).
 *   - Pointers documented as "device" must point to device memory of the
 *     current HIP device; "host" pointers to ordinary host memory.
 *   - bf16 means IEEE bfloat16 stored as 16-bit words.
 *
 * Data layout in HBM (d = head dim, ps = page size, r = rank, Hkv = KV heads):
 *   base pool  [num_base_pages][2][Hkv][ps*d] bf16: slot 0 holds K, slot 1 holds V;
 *              one (page, K|V, head) block of ps*d values is contiguous.  For the
 *              supported ps = 16, d = 128 a block is stored in the order the
 *              kernels' matrix-core fragments read it (one 16-byte load per lane):
 *                K (token t, dim i): (i/32)*512 + (t + 16*((i%16)/4))*8 + 4*((i%32)/16) + i%4
 *                V (token t, dim i): (i/32)*512 + (i%16 + 16*(t/4))*8 + 4*((i/16)%2) + t%4
 *              fkv_scatter_tokens writes this order; other shapes use K [ps][d], V [d][ps].
 *   res pool   [num_res_pages][fkv_res_page_elems(ps, r)] bf16.  For ps = 16 a page
 *              holds ceil(r/16) tiles of 512 values in fragment order: for L = 16*g + c
 *              (0 <= L < 64) tile k holds C_K[token c][16k + 4g + i] at L*8 + i and
 *              C_V[token 4g + i][16k + c] at L*8 + 4 + i (i < 4), so each lane of a
 *              wave reads both of its rCache fragments of a tile with one 16-byte load
 *              (for r = 8 half of a tile is padding).  Other page sizes: C_K as [ps][r], then C_V as
 *              [r][ps].
 *   adapters   [n_adapters][2][r][Hkv*d] bf16: B_K then B_V, each the r x n
 *              up-projection of Eq. 1 in row-major order (n = Hkv*d); KV head h
 *              uses columns h*d .. h*d+d-1.  Any LoRA scaling is folded in by the
 *              caller (Eq. 1 has none).
 *   queries    [n_q][Hq][d] bf16, already RoPE'd.  Output has the same layout.
 *   GQA        query head j reads KV head j / (Hq/Hkv).
 */
#ifndef FORKKV_H
#define FORKKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t fkv_status;

enum {
    FKV_OK = 0,
    FKV_ERR_INVALID = -1,     /* bad argument or inconsistent sizes */
    FKV_ERR_OOM = -2,         /* a page pool cannot satisfy the request (nothing changed) */
    FKV_ERR_NOT_FOUND = -3,   /* unknown sequence id */
    FKV_ERR_EXISTS = -4,      /* sequence id already in use */
    FKV_ERR_UNSUPPORTED = -5, /* a shape the kernels do not implement */
    FKV_ERR_HIP = -6          /* a HIP runtime call failed (message has the HIP error) */
};

enum { FKV_POOL_BASE = 0, FKV_POOL_RES = 1 };

/* Message of the last failing call on this thread ("" if none). */
const char *fkv_last_error(void);
/* Library version string. */
const char *fkv_version(void);

/* ------------------------------------------------------------------------ */
/* DualRadixTree (host).  Section 5.2: a base radix tree keyed by token ids    */
/* indexes bCache pages; a residual radix tree keyed by (agent id, token ids) */
/* indexes rCache pages.  Both are radix trees with one page per edge.        */
/* ------------------------------------------------------------------------ */

/* Determinism contract (both trees; block tables are therefore reproducible bit for bit):
 *   - Matching: a fork walks the tree one page-sized chunk of its tokens at a time; at each
 *     step it takes, among the current page's children in creation order, the child whose
 *     stored tokens match the longest prefix of the chunk (the first such child on ties; a
 *     child matching the whole chunk ends the search).  A whole-chunk match is inherited (a
 *     final chunk shorter than a page may inherit a page that holds more tokens, read-only);
 *     a match of k > 0 tokens short of the chunk makes that page the copy-on-write source of
 *     k tokens for the next new page; the walk stops at the first page it does not inherit.
 *   - Allocation: a pool hands out its lowest free page id.
 *   - Recency: each tree has a clock; a page is stamped with the next tick when it is
 *     created and whenever a sequence starts or stops referencing it.  A fork references its
 *     inherited pages in path order, then pins the copy-on-write source, evicts if needed,
 *     creates its new pages in order and unpins the source (base tree first, then the
 *     residual tree).  An append that writes into its exclusively owned last page stamps it
 *     twice; one that copies it creates the copy, then drops the old page.  A release drops
 *     the pages from last to first.
 *   - Eviction: when a pool has fewer free pages than a call needs, cached pages (referenced
 *     by no sequence) without children are evicted oldest stamp first (lower page id on
 *     ties), a parent becoming a candidate when its last child is evicted. */
typedef struct fkv_tree fkv_tree;

typedef struct {
    int32_t page_size;       /* tokens per page, both pools (1..1024) */
    int32_t num_base_pages;  /* capacity of the base pool */
    int32_t num_res_pages;   /* capacity of the residual pool */
} fkv_tree_config;

/* One device-side page copy the caller must perform (Section 5.2 copy-on-write):
 * copy the first n_valid token slots of page src into page dst of pool `pool`.
 * fkv_page_copy_launch performs a batch of them. */
typedef struct {
    int32_t pool, src, dst, n_valid;
} fkv_page_copy;

/* What the caller must do after fkv_fork / fkv_cow_append for one sequence:
 * first perform `copies`, then write bCache for logical positions
 * [base_valid, seq_len) and rCache for [res_valid, seq_len) into the slots
 * given by the sequence's block tables (page = table[pos / ps], slot = pos % ps).
 * Perform the copies before the next call on the tree. */
typedef struct {
    int64_t seq_len;
    int64_t base_valid;
    int64_t res_valid;
    int32_t n_copies;
    fkv_page_copy copies[2];
} fkv_fill_plan;

typedef struct {
    int32_t base_pages_free, base_pages_referenced, base_pages_cached, base_pages_raw;
    int32_t res_pages_free, res_pages_referenced, res_pages_cached, res_pages_raw;
    int32_t n_sequences;
    int64_t base_evictions, res_evictions;
} fkv_pool_stats;

/* Create / destroy a tree.  The tree owns host memory only. */
fkv_status fkv_tree_create(const fkv_tree_config *cfg, fkv_tree **out);
void fkv_tree_destroy(fkv_tree *tree);

/* Allocate n pages of pool FKV_POOL_BASE or FKV_POOL_RES outside the trees
 * (lowest free ids first, evicting unreferenced cached pages of that pool's
 * tree when needed).  out_ids: host, n entries.  FKV_ERR_OOM if impossible. */
fkv_status fkv_alloc_pages(fkv_tree *tree, int32_t pool, int32_t n, int32_t *out_ids);
/* Return pages obtained from fkv_alloc_pages. */
fkv_status fkv_free_pages(fkv_tree *tree, int32_t pool, int32_t n, const int32_t *ids);

/* Fork (Section 5.2, "Fork Semantics with CoW"): create sequence seq_id for
 * agent agent_id whose context is tokens[0..n) (host).  Step 1: longest-prefix
 * match in the base tree; matched pages are inherited read-only and unmatched
 * tokens get new base pages that extend the tree.  Step 2: the same in the
 * residual tree under key (agent_id, tokens), so a new agent id gets exclusive
 * rCache pages for its whole context.  A match that ends inside a page whose
 * remaining slots the new sequence needs yields a copy of that page.
 * Errors: FKV_ERR_EXISTS (seq_id in use), FKV_ERR_OOM, FKV_ERR_INVALID. */
fkv_status fkv_fork(fkv_tree *tree, int32_t seq_id, int32_t agent_id, const int32_t *tokens, int64_t n,
                    fkv_fill_plan *out);

/* Append n tokens (host) to sequence seq_id (decode steps or a prefill chunk).
 * A partially filled last page is written in place when the sequence is its only
 * user and nothing beyond it is stored, and copied first otherwise
 * (copy-on-write); further tokens go to new pages, which are inserted into the
 * trees so later forks can share them. */
fkv_status fkv_cow_append(fkv_tree *tree, int32_t seq_id, const int32_t *tokens, int64_t n,
                          fkv_fill_plan *out);

/* Drop a sequence.  Its pages stay cached in the trees until evicted (each tree
 * has its own LRU order, Section 5.2 "Decoupled Eviction Policy"). */
fkv_status fkv_release(fkv_tree *tree, int32_t seq_id);

/* Length and page count of a sequence (host outputs). */
fkv_status fkv_seq_info(const fkv_tree *tree, int32_t seq_id, int64_t *seq_len, int32_t *n_pages);

/* Block tables for n sequences (all host buffers): base_bt and res_bt are
 * [n][max_pages] int32 physical page ids, padded with 0 past each sequence's
 * pages; seq_lens [n] int32.  FKV_ERR_INVALID if a sequence needs more than
 * max_pages pages. */
fkv_status fkv_get_block_tables(const fkv_tree *tree, const int32_t *seq_ids, int32_t n, int32_t max_pages,
                                int32_t *base_bt, int32_t *res_bt, int32_t *seq_lens);

fkv_status fkv_get_pool_stats(const fkv_tree *tree, fkv_pool_stats *out);

/* Debug check (host copies) of the tables an attention call will read, for callers that build
 * or edit tables themselves (the kernels trust every page id they are given): for each agent a,
 * seq_lens[a] is in 1 .. max_pages * page_size, the first ceil(seq_lens[a] / page_size) entries
 * of base_bt row a are in [0, num_base_pages), and, when adapter_idx[a] >= 0, those of res_bt
 * row a are in [0, num_res_pages) (res_bt and adapter_idx may be NULL for r = 0).  Tables are
 * [n_agents][max_pages].  FKV_ERR_INVALID names the first bad agent, page and id.  The Python
 * binding runs it before every launch when the environment variable FKV_DEBUG is set. */
fkv_status fkv_validate_tables(const int32_t *base_bt, const int32_t *res_bt, const int32_t *seq_lens,
                               const int32_t *adapter_idx, int32_t n_agents, int32_t max_pages, int32_t page_size,
                               int32_t num_base_pages, int32_t num_res_pages);

/* ------------------------------------------------------------------------ */
/* Decode plan (host).  Agents whose base block tables name the same physical */
/* pages over a range of logical pages form a segment; each segment is split */
/* into work items of at most 16 query rows (agents x query heads per KV head)*/
/* and a bounded page range, so a base tile is streamed once per item and     */
/* applied to all of its agents' query heads.                                 */
/* ------------------------------------------------------------------------ */

typedef struct fkv_plan fkv_plan;

typedef struct {
    int32_t n_agents;
    int32_t hq, hkv;
    int32_t page_size;
    int32_t max_pages;        /* row stride of base_bt */
    int32_t pages_per_split;  /* pages per work item (<= 128 without RoPE, items of several agent
                                 groups <= 64; <= 64 with RoPE); 0 = choose automatically */
    int32_t num_cus;          /* compute units to fill; 0 = 256 */
    int32_t max_item_agents;  /* agents sharing one work item; 0 = as many as the kernel takes
                                 (fkv_decode_plan_default_agents); larger values are clamped */
    int32_t r;                /* residual rank the plan will be run with (0, 8, 16, 32, 64) */
    int32_t rope;             /* nonzero: the plan will be run with RoPE tables */
    int32_t reserve_pages;    /* growth room of each agent, in pages past its current last page (as far
                                 as max_pages allows): the plan stays valid while the agent's length
                                 grows into it.  0 = 16 pages; negative = none */
} fkv_decode_plan_params;

typedef struct {
    int64_t plan_words;       /* int32 words of the serialised plan */
    int64_t workspace_bytes;  /* workspace fkv_residual_attention_decode needs for (d, r) given at query */
    int32_t n_items;          /* work items */
    int32_t n_blocks;         /* workgroups of the split kernel */
    int32_t n_segments;       /* shared / private page ranges found */
    int32_t pages_per_split;
} fkv_plan_info;

/* Most agents one decode work item can hold for (hq, hkv, r, rope).  A group is the
 * floor(16/g) agents whose query heads of one KV head fill a 16-row matrix tile.  Without
 * RoPE: four groups below rank 32, two at rank 32, one (of at most two agents) at rank 64.
 * With RoPE: up to four wave groups of the agents one wave rebuilds (a whole group below
 * rank 32, two agents at rank 32, one at rank 64), at most 16 / ceil(r/16) agents (their
 * B_K^T fragments fill 64 KB of LDS).  Returns 0 for an unsupported head layout. */
int32_t fkv_decode_plan_default_agents(int32_t hq, int32_t hkv, int32_t r, int32_t rope);

/* Build a plan from host copies of the decode call's base block table base_bt
 * [n_agents][max_pages] and seq_lens [n_agents] (res_bt and adapter_idx are not read and may
 * be NULL).  The plan records which agents share which base pages (the segments) and how the
 * work is cut into items and workgroups; it holds no page id, length or adapter: the kernels
 * read those from the launch's block tables, seq_lens and adapter_idx.  So one plan serves
 * consecutive decode steps while
 *   - every agent's length stays within its capacity (fkv_decode_plan_covers checks this;
 *     each agent's last item reads up to reserve_pages further pages as the agent grows), and
 *   - the sharing structure is unchanged: no agent forked, released or replaced, and no
 *     page of the agents' existing block-table entries replaced (a copy-on-write copy reported
 *     by fkv_fork / fkv_cow_append for one of them; new entries past an agent's last page are
 *     fine).
 * Otherwise build a new plan.  Errors: FKV_ERR_INVALID for null or inconsistent arguments,
 * FKV_ERR_UNSUPPORTED for head layouts or ranks the kernels do not take. */
fkv_status fkv_decode_plan_create(const fkv_decode_plan_params *params, const int32_t *base_bt,
                                  const int32_t *res_bt, const int32_t *seq_lens, const int32_t *adapter_idx,
                                  fkv_plan **out);
void fkv_decode_plan_destroy(fkv_plan *plan);
/* FKV_OK if host seq_lens [n_agents] (n_agents as at creation) are all >= 1 and within the
 * plan's capacity; FKV_ERR_INVALID naming the first agent that outgrew it otherwise (build a
 * new plan).  O(n_agents), allocates nothing. */
fkv_status fkv_decode_plan_covers(const fkv_plan *plan, const int32_t *seq_lens, int32_t n_agents);
/* Largest length agent a may reach under this plan (host output). */
fkv_status fkv_decode_plan_capacity(const fkv_plan *plan, int32_t agent, int64_t *max_len);
/* Sizes of the plan; workspace_bytes is computed for head dim d and rank r. */
fkv_status fkv_decode_plan_info(const fkv_plan *plan, int32_t d, int32_t r, fkv_plan_info *out);
/* Write the serialised plan (plan_words int32) to a host buffer; the caller copies
 * it to device memory and passes that copy as fkv_attn_args.plan. */
fkv_status fkv_decode_plan_serialize(const fkv_plan *plan, int32_t *out, int64_t capacity_words);
/* Segment list (host outputs, n_segments entries each): first agent, agent count,
 * first page, page count.  Agents of a segment are listed in seg_agents. */
fkv_status fkv_decode_plan_segments(const fkv_plan *plan, int32_t *seg_first_page, int32_t *seg_n_pages,
                                    int32_t *seg_n_agents, int32_t *seg_agents, int64_t seg_agents_capacity);

/* ------------------------------------------------------------------------ */
/* ResidualAttention (device).                                                */
/* ------------------------------------------------------------------------ */

typedef struct {
    const void *q;              /* device bf16 [n_q][hq][d]; decode: n_q = n_agents, row a = agent a */
    const void *base_kv;        /* device bf16 base pool (layout above) */
    const void *res_kv;         /* device bf16 residual pool (layout above); unused when r == 0 */
    const void *lora_b;         /* device bf16 adapters [n_adapters][2][r][hkv*d] */
    const int32_t *adapter_idx; /* device [n_agents]; -1 = agent has no residual (base-only path) */
    const int32_t *base_bt;     /* device [n_agents][max_pages] */
    const int32_t *res_bt;      /* device [n_agents][max_pages] */
    const int32_t *seq_lens;    /* device [n_agents], >= 1; keys 0..seq_len-1 */
    const float *rope_cos;      /* device fp32 table from fkv_rope_table (rope_max_pos*d/2 values);
                                   NULL = no RoPE on C_K.B_K */
    const float *rope_sin;      /* device fp32 table from fkv_rope_table */
    const int32_t *plan;        /* device copy of a serialised decode plan (decode only) */
    const int32_t *q_indptr;    /* device [n_agents+1] query rows per agent (prefill only) */
    void *workspace;            /* device scratch of workspace_bytes (decode): the partial rows */
    size_t workspace_bytes;
    void *out;                  /* device bf16 [n_q][hq][d] */
    int32_t n_agents, hq, hkv, d, r, page_size, max_pages;
    int32_t rope_max_pos;       /* rows of the RoPE tables; every key position must be below it */
    int32_t n_q;                /* prefill: total query rows (= q_indptr[n_agents]) */
    int32_t max_q_per_agent;    /* prefill: largest q_indptr[a+1] - q_indptr[a] (sizes the grid); 0 = n_q,
                                   always enough.  If understated, the rows of an agent past it are
                                   not computed and are written as NaN. */
    float scale;                /* softmax scale; typically 1/sqrt(d) */
    void *const *timing_events; /* optional, host array of hipEvent_t (created with timing enabled), set by
                                   the launches to the kernels' own execution timestamps: decode [0] start
                                   and [1] end of the split kernel, [2] end of the merge kernel; prefill [0]
                                   start and [1] end of its kernel.  NULL = no events. */
} fkv_attn_args;

/* Decode: one query row per agent attends to all seq_len keys of its agent
 * (the current token's K/V/C is already in the cache).  Section 5.3,
 * Algorithm 1, split over the plan's work items with a log-sum-exp combine.
 * `plan` is the host plan whose serialised copy args->plan points to: the grid and workspace
 * sizes come from it on the host, so the launch needs no read of device memory.  The block
 * tables, seq_lens and adapter_idx in args are read by the kernels; they must keep the sharing
 * structure the plan was built from and the lengths within its capacity (see
 * fkv_decode_plan_create; a length past the capacity leaves those keys out of the result).
 * Supported: d = 128, page_size = 16, r in {0, 8, 16, 32, 64}, hq/hkv in {4, 8}.  The plan must
 * have been built for the same r and RoPE setting (FKV_ERR_INVALID otherwise), so that its work
 * items hold no more agents than fkv_decode_plan_default_agents allows.
 * Two kernels are enqueued (split, merge).  Calls that share a workspace must not overlap.
 * Errors: FKV_ERR_INVALID / FKV_ERR_UNSUPPORTED before any launch, FKV_ERR_HIP when a
 * launch fails. */
fkv_status fkv_residual_attention_decode(const fkv_attn_args *args, const fkv_plan *plan, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, serving loops
 * or harnesses that forbid allocation): the same decode as fkv_residual_attention_decode, with
 * the partial rows kept in a static device array of FKV_NOALLOC_WORKSPACE_BYTES that the library
 * holds on each GPU it runs on (from its first use there until the process ends) instead of
 * args->workspace, which is ignored.  The call allocates and frees nothing; the caller still
 * owns every input and output.  Every call on one GPU shares that GPU's array and nothing in
 * it needs to start at zero (each call writes every partial row it reads); calls that overlap
 * on one GPU (on different streams) race.  Errors as fkv_residual_attention_decode, plus
 * FKV_ERR_INVALID when the plan's partial rows (fkv_plan_info.workspace_bytes) exceed the array. */
#define FKV_NOALLOC_WORKSPACE_BYTES (64u << 20)
fkv_status fkv_residual_attention_decode_noalloc(const fkv_attn_args *args, const fkv_plan *plan, void *stream);

/* Chunked prefill: agent a's query rows q_indptr[a] .. q_indptr[a+1]-1 are the
 * last n_a = q_indptr[a+1]-q_indptr[a] tokens of its sequence (already in the
 * cache); row i sits at position seq_len[a] - n_a + i and attends causally to
 * keys 0 .. that position.  Same shapes as decode; needs no plan or workspace. */
fkv_status fkv_residual_attention_prefill(const fkv_attn_args *args, void *stream);

/* Fill the RoPE tables on the host (fp64 angles rounded to fp32): for position p
 * and pair i < d/2 the entry is cos(p * base^(-2i/d)) (sin likewise), stored at
 * (p/16)*1024 + (i/16)*256 + (p%16 + 16*((i%16)/4))*4 + i%4, the order in which the
 * kernels' fragments read them.  Needs d = 128 and max_pos a multiple of 16;
 * each table holds max_pos*d/2 floats. */
fkv_status fkv_rope_table(int32_t d, int32_t max_pos, double base, float *cos_out, float *sin_out);

/* ------------------------------------------------------------------------ */
/* Cache writes (device): copy-on-write page copies and token scatter.        */
/* ------------------------------------------------------------------------ */

/* Values (bf16) in one residual page for page size ps and rank r (the row stride of the
 * residual pool): ceil(r/16)*512 for ps = 16, 2*ps*r otherwise; 0 for invalid arguments. */
int64_t fkv_res_page_elems(int32_t page_size, int32_t r);

/* Perform page copies (device array of n fkv_page_copy) in both pools.  base_kv
 * and res_kv are the pools; hkv, d, r, page_size describe them. */
fkv_status fkv_page_copy_launch(const fkv_page_copy *copies_dev, int32_t n, void *base_kv, void *res_kv,
                                int32_t hkv, int32_t d, int32_t r, int32_t page_size, void *stream);

/* Write logical rows into the pools through one sequence's block table.
 * Positions pos0 .. pos0+n-1 of the sequence receive
 *   base: k_src/v_src [n][hkv][d] bf16 (device; NULL skips the base pool)
 *   res:  ck_src/cv_src [n][r] bf16 (device; NULL skips the residual pool)
 * bt_base / bt_res: device block-table rows of that sequence. */
fkv_status fkv_scatter_tokens(const int32_t *bt_base, const int32_t *bt_res, int64_t pos0, int64_t n,
                              const void *k_src, const void *v_src, const void *ck_src, const void *cv_src,
                              void *base_kv, void *res_kv, int32_t hkv, int32_t d, int32_t r,
                              int32_t page_size, void *stream);

/* Producer: write n new tokens (positions pos0 .. pos0+n-1 of one sequence) into both pools,
 * the cache-write step that precedes ResidualAttention (Section 5.2 stores the base and
 * residual caches apart; Section 5.3 keeps the residual as the rank-r shrink of the hidden
 * state, K = K_base + RoPE(C_K B_K) being rebuilt later):
 *   base:  K = RoPE_pos(k_raw) (rotate-half pairs (i, i + d/2) with the fp32 tables of
 *          fkv_rope_table; rope_cos = NULL stores k_raw as is) and V, k_raw/v [n][hkv][d] bf16;
 *   res:   C_K = x . A_K^T and C_V = x . A_V^T, x [n][hidden] bf16, lora_a [2][r][hidden] bf16
 *          (A_K then A_V of the sequence's adapter, rows of the shrink), fp32 accumulation,
 *          rounded to bf16; lora_a = NULL (or r = 0) leaves the residual pool untouched.
 * bt_base / bt_res: device block-table rows of the sequence (pages already allocated, e.g. by
 * fkv_cow_append).  Requires d = 128, page_size = 16, r in {0, 8, 16, 32, 64}, hidden a
 * multiple of 1024, pos0 + n <= rope_max_pos with RoPE.  Device pointers; enqueued on
 * `stream`; FKV_ERR_INVALID before any launch on bad arguments. */
fkv_status fkv_produce_tokens(const int32_t *bt_base, const int32_t *bt_res, int64_t pos0, int64_t n, const void *x,
                              int32_t hidden, const void *k_raw, const void *v, const void *lora_a,
                              const float *rope_cos, const float *rope_sin, int64_t rope_max_pos, void *base_kv,
                              void *res_kv, int32_t hkv, int32_t d, int32_t r, int32_t page_size, void *stream);

/* One sequence of a batched producer call (a host array of these; its pointers are device
 * memory). */
typedef struct {
    const int32_t *bt_base;  /* the sequence's base block-table row */
    const int32_t *bt_res;   /* its residual block-table row (may be NULL when lora_a is NULL) */
    const void *lora_a;      /* its adapter's [2][r][hidden] bf16 shrink rows; NULL: base pool only */
    int64_t pos0;            /* position of its first new token */
    int64_t n;               /* its new tokens (0: nothing to do) */
    int64_t row0;            /* row of its first new token in x, k_raw and v */
} fkv_produce_seq;

/* The producer over several sequences in one launch (same writes as fkv_produce_tokens for
 * each sequence; up to 32 sequences per launch, more are enqueued in groups of 32).  x
 * [rows][hidden], k_raw / v [rows][hkv][d] hold every sequence's new tokens, sequence i at
 * rows row0 .. row0 + n - 1.  The sequences must write disjoint page slots (fkv_cow_append
 * gives each appending sequence private pages); overlapping slots race.  Every sequence is
 * checked before anything is launched: FKV_ERR_INVALID names the first bad one. */
fkv_status fkv_produce_tokens_batch(const fkv_produce_seq *seqs, int32_t nseq, const void *x, int32_t hidden,
                                    const void *k_raw, const void *v, const float *rope_cos, const float *rope_sin,
                                    int64_t rope_max_pos, void *base_kv, void *res_kv, int32_t hkv, int32_t d,
                                    int32_t r, int32_t page_size, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* FORKKV_H */
