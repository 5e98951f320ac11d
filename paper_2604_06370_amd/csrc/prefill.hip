// ResidualAttention chunked prefill for gfx950 (Section 6 prefill kernel,
// Algorithm 1 with a block of query rows).
//
// One workgroup of eight waves = (agent a, KV head h, block of 256 query rows); its rows
// are (query token, query head of h), all of the same agent, so every 64-key tile of the
// agent's keys is staged once in LDS and applied to all 256 rows:
//   RoPE on, per tile: U^T = B_K^T C_K^T (MFMA), K_lora = RoPE_p(U) (rotate-half, fp32),
//                      K = K_base + K_lora -> bf16, in place in LDS
//   every wave, for its 32 rows:  S^T = K Q^T              (16x16x32 MFMA)
//                                 RoPE off: S^T += C_K (B_K q)^T
//                                 causal mask + online softmax
//                                 O^T   += V^T P^T          (16x16x32 MFMA)
//                                 acc_r^T += C_V^T P^T
// and at the end O = (O + acc_r . B_V[h]) / l (Eq. 4) is written in bf16.
//
// The contraction index of the 16x16x32 products is permuted so that the
// accumulator tiles of the 16x16x16 rebuild feed them without shuffles: in
// k-step kk, slot j of lane group grp is head-dim index 32kk + 16(j/4) + 4grp +
// j%4 for the key products, and key 16(j/4) + 4grp + j%4 of a 32-key half for the
// value products.  Queries and values are loaded in the same order.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <string>

#include "internal.hpp"
#include "lds_dma.hpp"
#include "mfma.hpp"

using namespace fkvk;

namespace {

constexpr int D = 128;
constexpr int PS = 16;
constexpr int ROWS_PER_WAVE = 32;          // two 16-row tiles
constexpr int TILE_KEYS = 64;              // four pages
constexpr int kXcds = 8;
constexpr float kNegInf = -INFINITY;

struct PrefillArgs {
    const uint16_t *q, *base_kv, *res_kv, *lora_b;
    const int32_t *adapter_idx, *base_bt, *res_bt, *seq_lens, *q_indptr;
    const float *rope_cos, *rope_sin;
    uint16_t *out;
    int32_t n_agents, hq, hkv, max_pages, blocks_per_agent_head;
    float scale_log2;
    int32_t rope_rows;  // positions the RoPE tables hold
};


// Rows of an agent's chunk that its query blocks do not reach (a max_q_per_agent below the
// agent's row count) are written as NaN by the agent's last block, so the shortfall shows in
// the output instead of leaving stale memory there.
__device__ __forceinline__ void poison_unreached_rows(const PrefillArgs &p, int q0, int nq, int h, int g, int reach) {
    const uint32_t nan2 = 0x7fc07fc0u;  // two bf16 quiet NaNs
    for (int64_t i = threadIdx.x; i < (int64_t)(nq - reach) * g * 32; i += blockDim.x) {
        const int64_t row = i / 32, c = i % 32;
        const int tok = reach + (int)(row / g), j = (int)(row % g);
        uint16_t *orow = p.out + ((int64_t)(q0 + tok) * p.hq + h * g + j) * 128;
        *reinterpret_cast<u32x2 *>(orow + 4 * c) = u32x2{nan2, nan2};
    }
}

// ---------------------------------------------------------------------------
// Streaming kernel.  A workgroup of eight waves holds 256 query rows, and 64-key tiles
// stream through a ring of LDS buffers by direct memory-to-LDS copies: wave w < 4 copies
// the K block (and, with an adapter, the rCache page) of page w of a tile, wave 4 + w its
// V block.  One barrier per tile hands a buffer over: every wave has waited (by count)
// for its copies of the tile, and every wave has finished reading the buffer that the
// copies issued after the barrier overwrite.
//  - RoPE off: the key residual folds into the queries (S^T += C_K (B_K q)^T), so the
//    stored blocks are used as they are; three buffers, copies two tiles ahead.
//  - RoPE on: a tile also carries the cos/sin rows of its pages' first positions (each
//    wave copies the 8 + 8 values per lane group that its rebuild uses); the rotation
//    angle of token t of a page starting at p0 comes from those rows and the rows of
//    positions 0..15 (kept in LDS for the launch) by angle addition.  Three buffers up to
//    rank 32, two at rank 64 (copies one tile ahead).  After a tile has landed each wave rebuilds half of one page's keys
//    in place (U^T = B_K^T C_K^T on the matrix cores, rotated, added to K_base) and a
//    second barrier publishes the rebuilt tile.
//
// Buffer layout (bytes): K blocks [page][4 KB], V blocks [page][4 KB], rCache pages as
// [rank tile][page][1 KB] (four pages of one rank tile are 1 KB apart).  All are stored
// verbatim: the K block's 16 bytes at k-step kk, lane l are the A fragment of the score
// product, the V block's 16 bytes at chunk q2, lane l hold dims 32q2 + col (.xy) and
// 32q2 + 16 + col (.zw) of tokens 4grp .. 4grp + 3, and the rCache fragment holds C_K
// (.xy) and C_V (.zw) of the lane.
constexpr float kLazyRescale = 8.f;

constexpr int kStreamWaves = 8;
constexpr int kStreamRows = kStreamWaves * ROWS_PER_WAVE;

template <int R, bool ROPE>
struct StreamShape {
    static constexpr int NBUF = (ROPE && R > 32) ? 2 : 3;  // ring buffers (copies NBUF - 1 tiles ahead)
    // Tile reads the compiler schedules (rank 64: 15.6 instead of 16.6 ms at 70B heads,
    // 8 x 1024 rows) or explicit ones that wait for themselves (below: no gain, 22.6 vs
    // 23.0 ms at 16 x 2048 rows, 8B heads)
    static constexpr bool CV = R >= 64;
    static constexpr int RT = R == 0 ? 0 : (R + 15) / 16;
    static constexpr int SBK_BYTES = ROPE ? RT * 8 * 64 * 8 : 0;  // B_K^T fragments (RoPE on)
    static constexpr int K_OFF = 0;
    static constexpr int V_OFF = 4 * 4096;
    static constexpr int C_OFF = 8 * 4096;
    // RoPE on: table rows [page][half][cos m, cos m + 1, sin m, sin m + 1][1 KB], m = 2 half
    static constexpr int T_OFF = C_OFF + 4 * RT * 1024;
    // RoPE on: [page pw][half][cos, sin][frequency tile j][lane group] 16 B
    static constexpr int BUF_BYTES = T_OFF + (ROPE ? 4 * 2 * 256 : 0);
    static constexpr int SBV_BYTES = R > 0 ? R * D * 4 : 16;
    static constexpr int SACC_BYTES = R > 0 ? kStreamRows * R * 4 : 16;
    static constexpr int EPI_BYTES = SBV_BYTES + SACC_BYTES;
    static constexpr int RING_BYTES = NBUF * BUF_BYTES;
    static constexpr int MAIN_BYTES = RING_BYTES > EPI_BYTES ? RING_BYTES : EPI_BYTES;
    // RoPE on: cos then sin of positions 0..15 in the table's own order ([tile m][lane] 16 B)
    static constexpr int COLT_BYTES = ROPE ? 2 * 4096 : 0;
    static constexpr int LDS_BYTES = MAIN_BYTES + SBK_BYTES + COLT_BYTES;
    static_assert(LDS_BYTES <= 160 * 1024, "LDS of one workgroup");
};

template <int R, int G, bool ROPE>
__global__ __launch_bounds__(64 * kStreamWaves, 1) void prefill_stream_kernel(PrefillArgs p) {
    using S = StreamShape<R, ROPE>;
    constexpr int RT = S::RT;
    constexpr int RTX = RT > 0 ? RT : 1;
    constexpr int TPW = kStreamRows / G;
    __shared__ __attribute__((aligned(16))) u32x4 lds[S::LDS_BYTES / 16];
    float *sBV = reinterpret_cast<float *>(lds);
    float *sAcc = reinterpret_cast<float *>(reinterpret_cast<unsigned char *>(lds) + S::SBV_BYTES);
    const u32x2 *sBK = reinterpret_cast<const u32x2 *>(reinterpret_cast<unsigned char *>(lds) + S::MAIN_BYTES);

    const int hkv = p.hkv;
    const int bpa = p.blocks_per_agent_head;
    const int xcd = blockIdx.x % kXcds, local = blockIdx.x / kXcds;
    const int pair = (local / bpa) * kXcds + xcd;
    const int qb = local - (local / bpa) * bpa;
    if (pair >= p.n_agents * hkv) return;
    const int a = pair / hkv;
    const int h = pair - a * hkv;
    const int q0 = p.q_indptr[a], nq = p.q_indptr[a + 1] - q0;
    const int tok_begin = qb * TPW;
    if (qb == bpa - 1 && nq > bpa * TPW) poison_unreached_rows(p, q0, nq, h, G, bpa * TPW);
    if (tok_begin >= nq) return;
    const int L = p.seq_lens[a];
    const int P0 = L - nq;  // position of the chunk's first query
    const int ad = R > 0 ? p.adapter_idx[a] : -1;

    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int64_t n = (int64_t)hkv * D;

    const int n_pages = (L + PS - 1) / PS;
    const int last_pos = P0 + (tok_begin + TPW < nq ? tok_begin + TPW : nq) - 1;
    const int n_tiles = last_pos / TILE_KEYS + 1;
    const int32_t *btb = p.base_bt + (int64_t)a * p.max_pages;
    const int32_t *btr = R > 0 ? p.res_bt + (int64_t)a * p.max_pages : nullptr;
    const bool use_res = R > 0 && ad >= 0;

    // This wave copies page pw of every tile: its K block and rCache page (waves 0..3) or
    // its V block (waves 4..7).
    const int pw = wave & 3;
    const int half = wave >> 2;
    const bool kwave = wave < 4;
    const bool res_copy = use_res && kwave;
    // Page ids of this wave's pages (page 4 t + pw of tile t), 64 tiles per register:
    // lane i holds the id for tile 64 c + i of chunk c (pages past the sequence repeat its
    // last page, so every copy reads a real page; their keys are masked).
    auto load_ids = [&](int c, int &idb, int &idr) __attribute__((always_inline)) {
        const int pg = min((64 * c + lane) * 4 + pw, n_pages - 1);
        idb = btb[pg];
        idr = res_copy ? btr[pg] : 0;
    };
    int idb_cur, idr_cur, idb_nxt, idr_nxt;
    load_ids(0, idb_cur, idr_cur);
    load_ids(1, idb_nxt, idr_nxt);

    auto buf = [&](int tile) __attribute__((always_inline)) -> LdsU32x4 * {
        return (LdsU32x4 *)(lds + (tile % S::NBUF) * (S::BUF_BYTES / 16));
    };
    // RoPE tables (rope_rows positions of D / 2 floats each)
    const int rope_bytes = ROPE ? p.rope_rows * (D / 2) * 4 : 0;
    const i32x4 rope_rc = block_rsrc(reinterpret_cast<uint64_t>(p.rope_cos), rope_bytes);
    const i32x4 rope_rs = block_rsrc(reinterpret_cast<uint64_t>(p.rope_sin), rope_bytes);
    // this wave's copies of tile `tile` (page 4 tile + pw)
    auto copy_tile = [&](int tile, int idb, int idr) __attribute__((always_inline)) {
        LdsU32x4 *b = buf(tile);
        const uint64_t kaddr = reinterpret_cast<uint64_t>(p.base_kv + ((int64_t)idb * 2 * hkv + h) * (PS * D));
        const i32x4 rs = block_rsrc(kwave ? kaddr : kaddr + (uint64_t)hkv * 4096, 4096);
        LdsU32x4 *dst = b + ((kwave ? S::K_OFF : S::V_OFF) + pw * 4096) / 16;
#pragma unroll
        for (int i = 0; i < 4; ++i) lds_dma16(rs, lane * 16 + i * 1024, dst + i * 64);
        if constexpr (R > 0) {
            if (res_copy) {
                const i32x4 rc = block_rsrc(reinterpret_cast<uint64_t>(p.res_kv + (int64_t)idr * (RT * 512)), RT * 1024);
#pragma unroll
                for (int t = 0; t < RT; ++t) lds_dma16(rc, lane * 16 + t * 1024, b + (S::C_OFF + (t * 4 + pw) * 1024) / 16);
            }
        }
        if constexpr (ROPE && R > 0) {
            if (use_res) {
                // cos and sin at the first position of page pw for the frequencies this wave's
                // rebuild uses: lane 4j + g (< 8) copies the 16 bytes that lane group g holds in
                // frequency tile 2 half + j of the page's first table row
                const int pg = min(tile * 4 + pw, n_pages - 1);
                const int voff = ((pg * (PS * D / 2) + (2 * half + (lane >> 2)) * 256) + 64 * (lane & 3)) * 4;
                LdsU32x4 *td = b + (S::T_OFF + (pw * 2 + half) * 256) / 16;
                if (lane < 8) {
                    lds_dma16(rope_rc, voff, td);
                    lds_dma16(rope_rs, voff, td + 8);
                }
            }
        }
    };

    // queries of this lane's rows in the two 16-row tiles of the wave, in the contraction
    // order of the stored K fragments
    int row_tok[2], row_pos[2];
    bool row_ok[2];
    u32x4 qf[2][4];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        const int r = wave * ROWS_PER_WAVE + nt * 16 + col;
        const int tk = tok_begin + r / G;
        const int jj = r % G;
        row_ok[nt] = tk < nq;
        row_tok[nt] = tk;
        row_pos[nt] = P0 + tk;
        const uint16_t *qr = p.q + ((int64_t)(q0 + (row_ok[nt] ? tk : 0)) * p.hq + h * G + jj) * D;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            u32x4 v = {0, 0, 0, 0};
            if (row_ok[nt]) {
                const u32x2 lo = ldg64(qr + 32 * kk + 4 * grp);
                const u32x2 hi = ldg64(qr + 32 * kk + 16 + 4 * grp);
                v = u32x4{lo.x, lo.y, hi.x, hi.y};
            }
            qf[nt][kk] = v;
        }
    }
    // W^T = (B_K q)^T per row tile and rank tile: the residual key term of row j is
    // (B_K q_j) . c_p, one extra contraction over the rank
    u32x2 wq[2][RTX];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int t = 0; t < RTX; ++t) wq[nt][t] = u32x2{0, 0};
    if constexpr (R > 0 && !ROPE) {
        if (use_res) {
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    f32x4 acc = {0, 0, 0, 0};
                    const int rho = 16 * t + col;
                    const uint16_t *bk = p.lora_b + (int64_t)ad * 2 * R * n + (int64_t)(rho < R ? rho : 0) * n + (int64_t)h * D;
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) {
                        u32x4 av = {0, 0, 0, 0};
                        if (rho < R) {
                            const u32x2 lo = ldg64(bk + 32 * kk + 4 * grp);
                            const u32x2 hi = ldg64(bk + 32 * kk + 16 + 4 * grp);
                            av = u32x4{lo.x, lo.y, hi.x, hi.y};
                        }
                        acc = mfma32(av, qf[nt][kk], acc);
                    }
                    wq[nt][t] = pack4(acc);
                }
        }
    }
    // RoPE on: B_K^T fragments of the agent's adapter (lane holds B_K[16t + 4grp + i][h*D +
    // 16mt + col]) in LDS for the whole launch; this wave rebuilds u tiles 2 half, 2 half + 1
    // and their rotation partners + 4 of page pw, with the table rows of frequency tiles
    // 2 half + j, loaded one tile ahead
    if constexpr (ROPE && R > 0) {
        if (use_res) {
            u32x2 *bkt = const_cast<u32x2 *>(sBK);
            const uint16_t *bk = p.lora_b + (int64_t)ad * 2 * R * n + (int64_t)h * D;
            for (int idx = threadIdx.x; idx < RT * 8 * 64; idx += 64 * kStreamWaves) {
                const int ln = idx & 63, rest = idx >> 6;
                const int mt = rest & 7, t = rest >> 3;
                const int c = ln & 15, gg = ln >> 4;
                uint32_t w[2];
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int r0 = 16 * t + 4 * gg + 2 * j;
                    const uint16_t lo = r0 < R ? bk[(int64_t)r0 * n + 16 * mt + c] : (uint16_t)0;
                    const uint16_t hi = r0 + 1 < R ? bk[(int64_t)(r0 + 1) * n + 16 * mt + c] : (uint16_t)0;
                    w[j] = (uint32_t)lo | ((uint32_t)hi << 16);
                }
                bkt[idx] = u32x2{w[0], w[1]};
            }
            __syncthreads();  // B_K^T fragments written (no copy into LDS is in flight yet)
            // cos and sin of positions 0..15 (the first 4 KB of each table): wave w copies
            // kilobyte w % 4 of cos (w < 4) or sin; they land before the first tile's barrier
            LdsU32x4 *colt = (LdsU32x4 *)(lds + (S::MAIN_BYTES + S::SBK_BYTES) / 16);
            lds_dma16(wave < 4 ? rope_rc : rope_rs, lane * 16 + (wave & 3) * 1024, colt + wave * 64);
        }
    }
    // the page ids must be in registers before the first copies read them
    wait_vmcnt<0>();
    copy_tile(0, __builtin_amdgcn_readlane(idb_cur, 0), __builtin_amdgcn_readlane(idr_cur, 0));
    if (S::NBUF == 3 && n_tiles > 1) copy_tile(1, __builtin_amdgcn_readlane(idb_cur, 1), __builtin_amdgcn_readlane(idr_cur, 1));

    f32x4 oacc[8][2];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) oacc[mt][0] = oacc[mt][1] = f32x4{0, 0, 0, 0};
    f32x4 racc[RTX][2];
#pragma unroll
    for (int t = 0; t < RTX; ++t) racc[t][0] = racc[t][1] = f32x4{0, 0, 0, 0};
    f32x4 lacc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};  // row sums l
    float m_run[2] = {kNegInf, kNegInf};
    const float cl = p.scale_log2;
    const u32x4 kOnes = u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};  // bf16 1.0

    for (int tile = 0; tile < n_tiles; ++tile) {
        // this wave's copies of the tile have landed (only those of the next tile, issued
        // after them, may still be in flight); after the barrier every wave's have, and
        // every wave is done with the tile before, whose buffer the next copies overwrite
        // (last tile, or two buffers: nothing else is in flight)
        if (S::NBUF == 3 && tile + 1 < n_tiles) {
            // per tile a wave copies 4 blocks, plus its rCache page (K waves, with an adapter)
            // and, RoPE on with an adapter, two table rows
            constexpr int kTab = (ROPE && R > 0) ? 2 : 0;
            if (res_copy) wait_vmcnt<4 + RT + kTab>();
            else if (use_res) wait_vmcnt<4 + kTab>();
            else wait_vmcnt<4>();
        } else {
            wait_vmcnt<0>();
        }
        if constexpr (S::CV) lds_fence_barrier();
        else __builtin_amdgcn_s_barrier();
        const int tn = tile + S::NBUF - 1;
        if (tn < n_tiles) {
            if ((tn & 63) == 0) {
                idb_cur = idb_nxt;
                idr_cur = idr_nxt;
                load_ids((tn >> 6) + 1, idb_nxt, idr_nxt);
            }
            copy_tile(tn, __builtin_amdgcn_readlane(idb_cur, tn & 63), __builtin_amdgcn_readlane(idr_cur, tn & 63));
        }
        const uint32_t base = lds_addr(buf(tile)) + lane * 16;
        // keys of the tile at or past the sequence end (the tile that holds it, or pages
        // past it) may hold any bits in V and C_V: zero them
        const bool ragged = (tile + 1) * TILE_KEYS > L;
        if constexpr (ROPE && R > 0) {
            if (use_res) {
                // Stage 1 for a quarter of page pw: U^T tiles, deferred RoPE, K = K_base +
                // K_lora in place (keys past the sequence end are masked out of the scores)
                u32x2 ck[RTX];
                f32x4 u[4];  // u tiles 2 half, 2 half + 1, 2 half + 4, 2 half + 5
#pragma unroll
                for (int j = 0; j < 4; ++j) u[j] = f32x4{0, 0, 0, 0};
                u32x4 rot0[4];  // cos m, cos m + 1, sin m, sin m + 1 at p0 (this lane group)
                u32x4 rotc[2], rots[2];  // cos, sin of tiles m, m + 1 at position col
                const uint32_t colt = lds_addr((LdsU32x4 *)lds) + S::MAIN_BYTES + S::SBK_BYTES + 2 * half * 1024 + lane * 16;
                const uint32_t ka = base + S::K_OFF + pw * 4096 + half * 1024;
                const uint32_t kb = ka + 2 * 1024;
                u32x4 kf[2];
                if constexpr (RT == 1) {
                    // every LDS read of the rebuild under one wait (rCache fragment, B_K^T tiles,
                    // cos/sin pieces, K fragments): 16 agents x 2048-token chunks, 28.0 -> 26.9 ms
                    u32x4 c;
                    u32x2 bkf[4];
                    asm volatile(
                        "ds_read_b128 %0, %15\n\t"
                        "ds_read_b64 %1, %16\n\t"
                        "ds_read_b64 %2, %16 offset:512\n\t"
                        "ds_read_b64 %3, %16 offset:2048\n\t"
                        "ds_read_b64 %4, %16 offset:2560\n\t"
                        "ds_read_b128 %5, %17\n\t"
                        "ds_read_b128 %6, %17 offset:64\n\t"
                        "ds_read_b128 %7, %17 offset:128\n\t"
                        "ds_read_b128 %8, %17 offset:192\n\t"
                        "ds_read_b128 %9, %18\n\t"
                        "ds_read_b128 %10, %18 offset:1024\n\t"
                        "ds_read_b128 %11, %18 offset:4096\n\t"
                        "ds_read_b128 %12, %18 offset:5120\n\t"
                        "ds_read_b128 %13, %19\n\t"
                        "ds_read_b128 %14, %19 offset:2048\n\t"
                        "s_waitcnt lgkmcnt(0)"
                        : "=&v"(c), "=&v"(bkf[0]), "=&v"(bkf[1]), "=&v"(bkf[2]), "=&v"(bkf[3]), "=&v"(rot0[0]), "=&v"(rot0[1]),
                          "=&v"(rot0[2]), "=&v"(rot0[3]), "=&v"(rotc[0]), "=&v"(rotc[1]), "=&v"(rots[0]), "=&v"(rots[1]),
                          "=&v"(kf[0]), "=&v"(kf[1])
                        : "v"(base + S::C_OFF + pw * 1024),
                          "v"(lds_addr((LdsU32x4 *)lds) + S::MAIN_BYTES + ((2 * half) * 64 + lane) * 8),
                          "v"(lds_addr(buf(tile)) + S::T_OFF + (pw * 2 + half) * 256 + grp * 16), "v"(colt), "v"(ka)
                        : "memory");
                    ck[0] = (4 * grp < R) ? u32x2{c.x, c.y} : u32x2{0, 0};
#pragma unroll
                    for (int j = 0; j < 4; ++j) u[j] = mfma16(bkf[j], ck[0], u[j]);
                } else {
                    // two groups under one wait each: the rCache fragments and B_K^T tiles of every
                    // rank tile (rank tile t is 4 KB further in both), then cos/sin and K
                    u32x4 c[RT];
                    u32x2 bkf[RT][4];
                    const uint32_t ca = base + S::C_OFF + pw * 1024;
                    const uint32_t ba = lds_addr((LdsU32x4 *)lds) + S::MAIN_BYTES + ((2 * half) * 64 + lane) * 8;
                    static_assert(RT == 2 || RT == 4, "rank tiles");
                    if constexpr (RT == 2) {
                        asm volatile(
                            "ds_read_b128 %0, %10\n\t"
                            "ds_read_b128 %1, %10 offset:4096\n\t"
                            "ds_read_b64 %2, %11\n\t"
                            "ds_read_b64 %3, %11 offset:512\n\t"
                            "ds_read_b64 %4, %11 offset:2048\n\t"
                            "ds_read_b64 %5, %11 offset:2560\n\t"
                            "ds_read_b64 %6, %11 offset:4096\n\t"
                            "ds_read_b64 %7, %11 offset:4608\n\t"
                            "ds_read_b64 %8, %11 offset:6144\n\t"
                            "ds_read_b64 %9, %11 offset:6656\n\t"
                            "s_waitcnt lgkmcnt(0)"
                            : "=&v"(c[0]), "=&v"(c[1]), "=&v"(bkf[0][0]), "=&v"(bkf[0][1]), "=&v"(bkf[0][2]),
                              "=&v"(bkf[0][3]), "=&v"(bkf[1][0]), "=&v"(bkf[1][1]), "=&v"(bkf[1][2]), "=&v"(bkf[1][3])
                            : "v"(ca), "v"(ba)
                            : "memory");
                    } else {
                        asm volatile(
                            "ds_read_b128 %0, %20\n\t"
                            "ds_read_b128 %1, %20 offset:4096\n\t"
                            "ds_read_b128 %2, %20 offset:8192\n\t"
                            "ds_read_b128 %3, %20 offset:12288\n\t"
                            "ds_read_b64 %4, %21\n\t"
                            "ds_read_b64 %5, %21 offset:512\n\t"
                            "ds_read_b64 %6, %21 offset:2048\n\t"
                            "ds_read_b64 %7, %21 offset:2560\n\t"
                            "ds_read_b64 %8, %21 offset:4096\n\t"
                            "ds_read_b64 %9, %21 offset:4608\n\t"
                            "ds_read_b64 %10, %21 offset:6144\n\t"
                            "ds_read_b64 %11, %21 offset:6656\n\t"
                            "ds_read_b64 %12, %21 offset:8192\n\t"
                            "ds_read_b64 %13, %21 offset:8704\n\t"
                            "ds_read_b64 %14, %21 offset:10240\n\t"
                            "ds_read_b64 %15, %21 offset:10752\n\t"
                            "ds_read_b64 %16, %21 offset:12288\n\t"
                            "ds_read_b64 %17, %21 offset:12800\n\t"
                            "ds_read_b64 %18, %21 offset:14336\n\t"
                            "ds_read_b64 %19, %21 offset:14848\n\t"
                            "s_waitcnt lgkmcnt(0)"
                            : "=&v"(c[0]), "=&v"(c[1]), "=&v"(c[2]), "=&v"(c[3]), "=&v"(bkf[0][0]), "=&v"(bkf[0][1]),
                              "=&v"(bkf[0][2]), "=&v"(bkf[0][3]), "=&v"(bkf[1][0]), "=&v"(bkf[1][1]),
                              "=&v"(bkf[1][2]), "=&v"(bkf[1][3]), "=&v"(bkf[2][0]), "=&v"(bkf[2][1]),
                              "=&v"(bkf[2][2]), "=&v"(bkf[2][3]), "=&v"(bkf[3][0]), "=&v"(bkf[3][1]),
                              "=&v"(bkf[3][2]), "=&v"(bkf[3][3])
                            : "v"(ca), "v"(ba)
                            : "memory");
                    }
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        ck[t] = (16 * t + 4 * grp < R) ? u32x2{c[t].x, c[t].y} : u32x2{0, 0};
#pragma unroll
                        for (int j = 0; j < 4; ++j) u[j] = mfma16(bkf[t][j], ck[t], u[j]);
                    }
                    asm volatile(
                        "ds_read_b128 %0, %10\n\t"
                        "ds_read_b128 %1, %10 offset:64\n\t"
                        "ds_read_b128 %2, %10 offset:128\n\t"
                        "ds_read_b128 %3, %10 offset:192\n\t"
                        "ds_read_b128 %4, %11\n\t"
                        "ds_read_b128 %5, %11 offset:1024\n\t"
                        "ds_read_b128 %6, %11 offset:4096\n\t"
                        "ds_read_b128 %7, %11 offset:5120\n\t"
                        "ds_read_b128 %8, %12\n\t"
                        "ds_read_b128 %9, %12 offset:2048\n\t"
                        "s_waitcnt lgkmcnt(0)"
                        : "=&v"(rot0[0]), "=&v"(rot0[1]), "=&v"(rot0[2]), "=&v"(rot0[3]), "=&v"(rotc[0]), "=&v"(rotc[1]),
                          "=&v"(rots[0]), "=&v"(rots[1]), "=&v"(kf[0]), "=&v"(kf[1])
                        : "v"(lds_addr(buf(tile)) + S::T_OFF + (pw * 2 + half) * 256 + grp * 16), "v"(colt), "v"(ka)
                        : "memory");
                }
                // rotate-half pairs (tile m with m + 4) at the key's position p0 + col: the
                // angle of page start p0 plus the angle of offset col (angle addition)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const f32x4 c0 = __builtin_bit_cast(f32x4, rot0[j]), s0 = __builtin_bit_cast(f32x4, rot0[2 + j]);
                    const f32x4 ct = __builtin_bit_cast(f32x4, rotc[j]), st = __builtin_bit_cast(f32x4, rots[j]);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float c = c0[i] * ct[i] - s0[i] * st[i];
                        const float s = s0[i] * ct[i] + c0[i] * st[i];
                        const float x = u[j][i], y = u[j + 2][i];
                        u[j][i] = x * c - y * s;
                        u[j + 2][i] = y * c + x * s;
                    }
                }
                // K fragments half (u tiles 2 half, 2 half + 1) and half + 2 (tiles + 4), read above
                u32x4 out[2];
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const u32x4 k = kf[j];
                    const f32x4 lo = f32x4{bf16_lo(k.x), bf16_hi(k.x), bf16_lo(k.y), bf16_hi(k.y)} + u[2 * j];
                    const f32x4 hi = f32x4{bf16_lo(k.z), bf16_hi(k.z), bf16_lo(k.w), bf16_hi(k.w)} + u[2 * j + 1];
                    const u32x2 plo = pack4(lo), phi = pack4(hi);
                    out[j] = u32x4{plo.x, plo.y, phi.x, phi.y};
                }
                lds_write2(ka, out[0], kb, out[1]);
                // the rebuilt tile is complete
                if constexpr (S::CV) lds_fence_barrier();
                else __builtin_amdgcn_s_barrier();
            }
        }

        // ---- scores for the 64 keys of the tile, 2 row tiles ----
        // (below rank 64 two pages' K fragments are read per wait, so each wait on the LDS
        // is followed by 16 products instead of 8)
        f32x4 sacc[4][2];
        constexpr int KPW = R < 64 ? 2 : 1;  // pages read per LDS wait
#pragma unroll
        for (int kt = 0; kt < 4; kt += KPW) {
            u32x4 kf[KPW][4];
            if constexpr (KPW == 2) lds_get8<S::CV>(base + S::K_OFF + kt * 4096, base + S::K_OFF + (kt + 1) * 4096, kf[0], kf[1]);
            else lds_get4<S::CV>(base + S::K_OFF + kt * 4096, kf[0]);
#pragma unroll
            for (int j = 0; j < KPW; ++j) {
                sacc[kt + j][0] = sacc[kt + j][1] = f32x4{0, 0, 0, 0};
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    sacc[kt + j][0] = mfma32(kf[j][kk], qf[0][kk], sacc[kt + j][0]);
                    sacc[kt + j][1] = mfma32(kf[j][kk], qf[1][kk], sacc[kt + j][1]);
                }
            }
        }
        if constexpr (R > 0 && !ROPE) {
            if (use_res) {
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    // rCache fragments of the tile's four pages (C_K in .xy)
                    u32x4 cf[4];
                    lds_get4<S::CV>(base + S::C_OFF + t * 4096, cf);
                    // C_K of rank rows 16t + 4grp .. +3 (rank 8: half a tile is padding)
                    const bool kvalid = 16 * t + 4 * grp < R;
#pragma unroll
                    for (int kt = 0; kt < 4; ++kt) {
                        const u32x4 ak = u32x4{kvalid ? cf[kt].x : 0u, kvalid ? cf[kt].y : 0u, 0u, 0u};
                        // zero-padded 16x16x32 form: the chain stays on one instruction form
                        sacc[kt][0] = mfma32(ak, u32x4{wq[0][t].x, wq[0][t].y, 0u, 0u}, sacc[kt][0]);
                        sacc[kt][1] = mfma32(ak, u32x4{wq[1][t].x, wq[1][t].y, 0u, 0u}, sacc[kt][1]);
                    }
                }
            }
        }

        // ---- causal mask + online softmax (rows live in lanes) ----
        // A tile below every row's diagonal needs no mask.  The running maximum moves only
        // when some row's scores exceed it by more than 2^kLazyRescale (then acc, acc_r and
        // the row sums are rescaled); otherwise this tile's weights stay below 2^8.
        const bool full = (tile + 1) * TILE_KEYS - 1 <= P0 + tok_begin;
        u32x2 pf[4][2];
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
            float sv[4][4];
            if (full) {
#pragma unroll
                for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) sv[kt][i] = sacc[kt][nt][i];
            } else {
#pragma unroll
                for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = tile * TILE_KEYS + kt * PS + 4 * grp + i;
                        sv[kt][i] = (row_ok[nt] && key <= row_pos[nt]) ? sacc[kt][nt][i] : kNegInf;
                    }
            }
            float mx = kNegInf;
#pragma unroll
            for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i) mx = fmaxf(mx, sv[kt][i]);
            mx = max_over_groups(mx) * cl;  // the scale is positive
            if (__builtin_amdgcn_ballot_w64(mx > m_run[nt] + kLazyRescale) != 0) {
                const float m_new = fmaxf(m_run[nt], mx);
                const float alpha = fast_exp2(m_run[nt] - (m_new == kNegInf ? 0.f : m_new));
#pragma unroll
                for (int mt = 0; mt < 8; ++mt) oacc[mt][nt] *= alpha;
#pragma unroll
                for (int t = 0; t < RT; ++t) racc[t][nt] *= alpha;
                lacc[nt] *= alpha;
                m_run[nt] = m_new;
            }
            const float m_use = m_run[nt] == kNegInf ? 0.f : m_run[nt];
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                f32x4 pv;
#pragma unroll
                for (int i = 0; i < 4; ++i) pv[i] = fast_exp2(__builtin_fmaf(sv[kt][i], cl, -m_use));
                pf[kt][nt] = pack4(pv);
            }
        }

        // ---- O^T += V^T P^T and acc_r^T += C_V^T P^T over two 32-key halves ----
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const u32x4 pb0 = u32x4{pf[2 * half][0].x, pf[2 * half][0].y, pf[2 * half + 1][0].x, pf[2 * half + 1][0].y};
            const u32x4 pb1 = u32x4{pf[2 * half][1].x, pf[2 * half][1].y, pf[2 * half + 1][1].x, pf[2 * half + 1][1].y};
            u32x4 v0[4], v1[4];
            lds_get8<S::CV>(base + S::V_OFF + (2 * half) * 4096, base + S::V_OFF + (2 * half + 1) * 4096, v0, v1);
            if (ragged) {
                const int vis0 = L - (tile * 4 + 2 * half) * PS, vis1 = vis0 - PS;
#pragma unroll
                for (int q2 = 0; q2 < 4; ++q2) {
                    const u32x2 a0 = mask4(u32x2{v0[q2].x, v0[q2].y}, vis0, grp), b0 = mask4(u32x2{v0[q2].z, v0[q2].w}, vis0, grp);
                    const u32x2 a1 = mask4(u32x2{v1[q2].x, v1[q2].y}, vis1, grp), b1 = mask4(u32x2{v1[q2].z, v1[q2].w}, vis1, grp);
                    v0[q2] = u32x4{a0.x, a0.y, b0.x, b0.y};
                    v1[q2] = u32x4{a1.x, a1.y, b1.x, b1.y};
                }
            }
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2) {
                const u32x4 va = u32x4{v0[q2].x, v0[q2].y, v1[q2].x, v1[q2].y};  // dim 32q2 + col
                const u32x4 vb = u32x4{v0[q2].z, v0[q2].w, v1[q2].z, v1[q2].w};  // dim 32q2 + 16 + col
                oacc[2 * q2][0] = mfma32(va, pb0, oacc[2 * q2][0]);
                oacc[2 * q2][1] = mfma32(va, pb1, oacc[2 * q2][1]);
                oacc[2 * q2 + 1][0] = mfma32(vb, pb0, oacc[2 * q2 + 1][0]);
                oacc[2 * q2 + 1][1] = mfma32(vb, pb1, oacc[2 * q2 + 1][1]);
            }
            // row sums of the bf16 weights (every accumulator row holds the sum)
            lacc[0] = mfma32(kOnes, pb0, lacc[0]);
            lacc[1] = mfma32(kOnes, pb1, lacc[1]);
            if constexpr (R > 0) {
                if (use_res) {
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        // C_V of rank 16t + col, tokens 4grp .. +3 of the two pages (.zw)
                        u32x4 cf[2];
                        lds_get2<S::CV>(base + S::C_OFF + (t * 4 + 2 * half) * 1024, cf);
                        u32x2 c0 = u32x2{cf[0].z, cf[0].w};
                        u32x2 c1 = u32x2{cf[1].z, cf[1].w};
                        if (ragged) {
                            const int vis0 = L - (tile * 4 + 2 * half) * PS;
                            c0 = mask4(c0, vis0, grp);
                            c1 = mask4(c1, vis0 - PS, grp);
                        }
                        const bool vvalid = 16 * t + col < R;
                        const u32x4 ca = vvalid ? u32x4{c0.x, c0.y, c1.x, c1.y} : u32x4{0, 0, 0, 0};
                        racc[t][0] = mfma32(ca, pb0, racc[t][0]);
                        racc[t][1] = mfma32(ca, pb1, racc[t][1]);
                    }
                }
            }
        }
    }
    wait_vmcnt<0>();
    __syncthreads();  // the buffers are reused below

    // ---- epilogue: O = (acc + acc_r . B_V[h]) / l ----
    const float l_run[2] = {lacc[0][0], lacc[1][0]};
    if constexpr (R > 0) {
        if (use_res) {
            const uint16_t *bv = p.lora_b + ((int64_t)ad * 2 + 1) * R * n + (int64_t)h * D;
            for (int e = threadIdx.x; e < R * D; e += 64 * kStreamWaves) sBV[e] = bf16_to_f32(bv[(int64_t)(e / D) * n + (e % D)]);
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int t = 0; t < RT; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int rho = 16 * t + 4 * grp + i;
                        if (rho < R) sAcc[(wave * ROWS_PER_WAVE + nt * 16 + col) * R + rho] = racc[t][nt][i];
                    }
            __syncthreads();
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) {
                const float *ar = sAcc + (wave * ROWS_PER_WAVE + nt * 16 + col) * R;
#pragma unroll 4
                for (int rho = 0; rho < R; ++rho) {
                    const float c = ar[rho];
#pragma unroll
                    for (int mt = 0; mt < 8; ++mt)
#pragma unroll
                        for (int i = 0; i < 4; ++i) oacc[mt][nt][i] += c * sBV[rho * D + 16 * mt + 4 * grp + i];
                }
            }
        }
    }
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        if (!row_ok[nt]) continue;
        const int r = wave * ROWS_PER_WAVE + nt * 16 + col;
        const float inv = l_run[nt] > 0.f ? 1.f / l_run[nt] : 0.f;
        uint16_t *orow = p.out + ((int64_t)(q0 + row_tok[nt]) * p.hq + h * G + r % G) * D;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
            f32x4 o = oacc[mt][nt] * inv;
            *reinterpret_cast<u32x2 *>(orow + 16 * mt + 4 * grp) = pack4(o);
        }
    }
}

template <int R, int G, bool ROPE>
hipError_t launch_prefill(const PrefillArgs &pa, hipStream_t st, void *const *ev) {
    hipError_t e;
    const int pairs = (pa.n_agents * pa.hkv + kXcds - 1) / kXcds * kXcds;
    const int grid = pairs * pa.blocks_per_agent_head;
    // timing events carry the kernel's own start and end timestamps (set by the launch)
    hipEvent_t e0 = ev ? static_cast<hipEvent_t>(ev[0]) : nullptr;
    hipEvent_t e1 = ev ? static_cast<hipEvent_t>(ev[1]) : nullptr;
    hipExtLaunchKernelGGL((prefill_stream_kernel<R, G, ROPE>), dim3(grid), dim3(64 * kStreamWaves), 0, st, e0, e1, 0, pa);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return hipSuccess;
}

template <int G>
hipError_t dispatch_prefill(int r, bool rope, const PrefillArgs &pa, hipStream_t st, void *const *ev) {
    switch (r) {
    case 0: return launch_prefill<0, G, false>(pa, st, ev);
    case 8: return rope ? launch_prefill<8, G, true>(pa, st, ev) : launch_prefill<8, G, false>(pa, st, ev);
    case 16: return rope ? launch_prefill<16, G, true>(pa, st, ev) : launch_prefill<16, G, false>(pa, st, ev);
    case 32: return rope ? launch_prefill<32, G, true>(pa, st, ev) : launch_prefill<32, G, false>(pa, st, ev);
    case 64: return rope ? launch_prefill<64, G, true>(pa, st, ev) : launch_prefill<64, G, false>(pa, st, ev);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

namespace fkv {
fkv_status validate_attn_common(const fkv_attn_args *a, const char *who);
}

extern "C" fkv_status fkv_residual_attention_prefill(const fkv_attn_args *a, void *stream) {
    fkv::clear_error();
    fkv_status st = fkv::validate_attn_common(a, "fkv_residual_attention_prefill");
    if (st != FKV_OK) return st;
    if (!a->q_indptr || a->n_q < 1)
        return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_prefill: q_indptr and n_q >= 1 are required");
    const int g = a->hq / a->hkv;
    if (g != 4 && g != 8)
        return fkv::fail(FKV_ERR_UNSUPPORTED, "fkv_residual_attention_prefill: query heads per KV head must be 4 or 8");
    if (a->rope_cos && (int64_t)a->rope_max_pos < (int64_t)a->max_pages * a->page_size)
        return fkv::fail(FKV_ERR_INVALID,
                         "fkv_residual_attention_prefill: RoPE table must cover max_pages * page_size positions");
    PrefillArgs pa;
    pa.q = static_cast<const uint16_t *>(a->q);
    pa.base_kv = static_cast<const uint16_t *>(a->base_kv);
    pa.res_kv = static_cast<const uint16_t *>(a->res_kv);
    pa.lora_b = static_cast<const uint16_t *>(a->lora_b);
    pa.adapter_idx = a->adapter_idx;
    pa.base_bt = a->base_bt;
    pa.res_bt = a->res_bt;
    pa.seq_lens = a->seq_lens;
    pa.q_indptr = a->q_indptr;
    pa.rope_cos = a->rope_cos;
    pa.rope_sin = a->rope_sin;
    pa.out = static_cast<uint16_t *>(a->out);
    pa.n_agents = a->n_agents;
    pa.hq = a->hq;
    pa.hkv = a->hkv;
    pa.max_pages = a->max_pages;
    pa.rope_rows = a->rope_cos ? a->rope_max_pos : 0;
    // query blocks per (agent, KV head); blocks past an agent's own chunk exit at once
    const bool rope = a->rope_cos != nullptr && a->r > 0;
    const int tok_per_wg = kStreamRows / g;
    const int maxq = a->max_q_per_agent > 0 ? a->max_q_per_agent : a->n_q;
    if (maxq > a->n_q) return fkv::fail(FKV_ERR_INVALID, "fkv_residual_attention_prefill: max_q_per_agent > n_q");
    pa.blocks_per_agent_head = (maxq + tok_per_wg - 1) / tok_per_wg;
    pa.scale_log2 = a->scale * 1.4426950408889634f;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    hipError_t e = g == 4 ? dispatch_prefill<4>(a->r, rope, pa, hs, a->timing_events)
                          : dispatch_prefill<8>(a->r, rope, pa, hs, a->timing_events);
    if (e != hipSuccess)
        return fkv::fail(FKV_ERR_HIP, std::string("fkv_residual_attention_prefill: launch failed: ") + hipGetErrorString(e));
    return FKV_OK;
}
