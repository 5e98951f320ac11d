// Internal declarations shared by the host-side sources of libforkkv.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/forkkv.h"

namespace fkv {

// Record a failure message for fkv_last_error() and return the status.
fkv_status fail(fkv_status code, const std::string &msg);
void clear_error();

// Decode plan, host side.  Serialised layout (all int32):
//   header[kHeaderWords]
//   items   [n_items][kItemWords]  {page_begin, page_cap, leader, n_ag, copies (1), page_end_at_plan,
//                                   agent[16], partial[16]}  (partial[j]: partial of slot j).  The item covers pages page_begin .. min(page_cap,
//                                   ceil(longest length / ps)) - 1 of its agents, the length read
//                                   from the device array at launch, so an item whose agent grows
//                                   reads the new pages (up to page_cap) without a new plan.
//   blocks  [n_blocks]             item * (hkv / H) + head block, or -1 for an idle block
//                                  (H = heads per block, header word H_HEADS_PER_BLOCK)
//   agent_ptr [n_agents+1]         agent a owns partials agent_ptr[a] .. agent_ptr[a+1]-1; query
//                                  head jj of KV head h of partial p is workspace record
//                                  (p * g + jj) * hkv + h
//   (header word H_OFF_AGENT_SLOT is unused and equals H_OFF_ZERO)
//   zero      [kZeroWords]         zeros, 16-byte aligned (read in place of the rCache of an
//                                  agent without adapter or of an empty agent slot)
//   descriptors [n_blocks][kDescWords]  see below
// An item holds up to four agent groups; a group is the floor(16/g) agents whose
// query heads of one KV head fill the 16 rows of one matrix-core tile.  An item of
// ng groups runs on 4 / ngp wave copies (ngp = 1, 2, 4 for ng = 1, 2, 3..4); the copies
// of a group merge their partials in LDS, so the item owns n_ag partials (g rows each) and
// its `copies` field (partials per slot) is 1.
// The plan holds no page id, sequence length or adapter: the kernels read them from the
// block tables, seq_lens and adapter_idx of the launch.
constexpr int kHeaderWords = 24;
constexpr int kMaxRows = 16;        // query rows of one agent group (one wave's row tile)
constexpr int kMaxGroups = 4;       // agent groups per item (one wave each)
constexpr int kMaxItemAgents = 16;  // agents per item
enum ItemField { kItemP0 = 0, kItemCap, kItemLeader, kItemNag, kItemCopies, kItemEnd, kItemAgents };
constexpr int kItemFirst = kItemAgents + kMaxItemAgents;
constexpr int kItemWords = kItemFirst + kMaxItemAgents;
constexpr int kMaxPagesPerItem = 64;  // upper bound of pages_per_split (block tables are staged in LDS)
// RoPE-off plans: item page limits of the split kernel, whose page ids travel in lane
// registers (two per table row: lanes 0..63 and 64..127)
constexpr int kMaxPagesMulti = 64;    // items of three or four agent groups
constexpr int kMaxPagesSingle = 128;  // items of one or two agent groups
constexpr int kDefaultReservePages = 16;  // growth room of an agent's last item (decode steps)

// Block descriptors: block b of the decode kernel (either form) reads the kDescWords words at
// off_desc + b * kDescWords:
//   kDescPg0, kDescCap    item page range start and capacity end (pages read: up to
//                         min(cap, ceil(longest length / ps)))
//   kDescNag              agents in the item (0: idle block)    kDescHead  KV head
//   kDescLeader           agent whose base block-table row names the item's pages
//   kDescItem, kDescCopies
//   kDescStream           1: no other item reads this item's base pages (the kernel loads
//                         them as data read once); 0: other items of the segment do
//   kDescAgent + slot, kDescPart + slot   agent and first partial of each item slot
enum DescField { kDescPg0 = 0, kDescCap, kDescNag, kDescHead, kDescLeader, kDescItem, kDescCopies, kDescStream };
constexpr int kDescAgent = 8;
constexpr int kDescPart = kDescAgent + kMaxItemAgents;
constexpr int kDescWords = kDescPart + kMaxItemAgents;

// Decode: one workgroup per (work item, KV head).  Without RoPE an item holds up to four
// agent groups below rank 32 and up to two at rank 32 (and at rank 64 with eight query heads
// per KV head), their base pages shared through LDS; otherwise one group, of at most two
// agents at rank 64 (the wave keeps every slot's rCache fragments of a stage in registers).
// With RoPE see decode_rope_wave_agents below.  Agent slots one wave serves without RoPE:
constexpr int decode_wave_slots(int g, int r) {
    return r >= 64 ? (kMaxRows / g < 2 ? kMaxRows / g : 2) : kMaxRows / g;
}
constexpr int decode_heads_per_block(int, bool) { return 1; }
// With RoPE a wave serves NSW agents (all the agents of a 16-row group below rank 32, two at
// rank 32, one at rank 64: the wave keeps their rCache fragments of two pages in registers),
// and an item holds up to four such wave groups, as many slots as 64 KB of B_K^T fragments
// (kept in LDS for the launch) allow.
constexpr int decode_rope_wave_agents(int g, int r) {
    const int ag = kMaxRows / g;
    return r >= 64 ? 1 : (r >= 32 ? (ag < 2 ? ag : 2) : ag);
}
constexpr int decode_rope_item_agents(int g, int r) {
    const int rt = r <= 16 ? 1 : (r + 15) / 16;
    const int ms = 4 * decode_rope_wave_agents(g, r);
    return ms < 16 / rt ? ms : 16 / rt;
}
// Agent groups one RoPE-off work item may hold: four below rank 32; two at rank 32 and at
// rank 64 when one wave serves a whole group (a stage's rCache fragments of a group then fit the
// registers of four groups at rank 16); one otherwise.
constexpr int decode_item_groups(int g, int r) {
    return r < 32 ? kMaxGroups : (decode_wave_slots(g, r) >= kMaxRows / g ? 2 : 1);
}
constexpr int decode_item_agent_cap(int g, int hkv, int r, bool rope) {
    (void)hkv;
    const int ag = kMaxRows / g;
    if (rope && r > 0) return decode_rope_item_agents(g, r);
    const int ng = decode_item_groups(g, r);
    if (ng == 1) return decode_wave_slots(g, r);
    return ng * ag < kMaxItemAgents ? ng * ag : kMaxItemAgents;
}

enum PlanHeader {
    H_MAGIC = 0, H_N_ITEMS, H_N_BLOCKS, H_N_AGENTS, H_HKV, H_GROUP, H_AGENTS_PER_ITEM,
    H_OFF_ITEMS, H_OFF_BLOCKS, H_OFF_AGENT_PTR, H_OFF_AGENT_SLOT, H_TOTAL_WORDS, H_PAGES_PER_SPLIT,
    H_PAGE_SIZE, H_N_SEGMENTS, H_TOTAL_ROWS, H_MAX_ITEM_AGENTS, H_HEADS_PER_BLOCK, H_RANK, H_ROPE, H_OFF_ZERO,
    H_OFF_DESC, H_FIELDS
};
constexpr int kZeroWords = 1024;  // zeroed area of a plan: stand-in rCache page for agents without one
static_assert(H_FIELDS <= kHeaderWords, "plan header fields overflow the header");
constexpr int32_t kPlanMagic = 0x464b5631;  // "FKV1"

}  // namespace fkv

struct fkv_plan;
namespace fkv {
// Decode workspace: the partial rows, rounded up to 256 bytes.
int64_t decode_partials_bytes(const fkv_plan *plan, int32_t d, int32_t r);
}  // namespace fkv

struct fkv_plan {
    std::vector<int32_t> words;
    std::vector<int32_t> seg_first_page, seg_n_pages, seg_agent_off, seg_agents;
    std::vector<int32_t> cap_pages;  // per agent: pages its items can read (length capacity / ps)
    int32_t hkv = 0, g = 0, n_agents = 0, page_size = 0, max_pages = 0;
    int32_t max_pages_used = 0;  // largest page capacity of any agent
};
