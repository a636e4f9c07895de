// Layout of the int32 launch plan shared by the host planner and the device
// kernels.  A plan is a header followed by fixed-size records.
#pragma once

#include <cstdint>

namespace pa {

constexpr int32_t kPlanMagic = 0x31304150;  // "PA01"

// Header words.
//
// Work is described once, as templates for kv-head 0, and a dispatch list
// assigns each workgroup of the attention launch a kv-head and a template:
// dispatch word (g << kDispatchHeadShift) | i, where i indexes the shared-
// prefix, tile and row templates in that order: i < N_SHARED_TMPL names
// shared-prefix template i, the next N_TILE_TMPL indices the tile templates,
// the rest the first of four row templates (one per wavefront); the kinds
// may interleave in the dispatch list.  Kv-head g's items
// write the partial rows of head 0's template plus g * HEAD_PARTIAL; merge
// group b of the merge launch is group template b % N_GROUP_TMPL of kv-head
// b / N_GROUP_TMPL.
enum : int32_t {
  H_MAGIC = 0,
  H_KIND,
  H_N_SHARED,      // shared-prefix (cascade) workgroups, all kv-heads
  H_N_TILE,        // tile workgroups (128-row items), all kv-heads
  H_N_ROW,         // row items (one wavefront each), all kv-heads, padded to whole workgroups
  H_N_GROUPS,      // merge groups, all kv-heads
  H_GRID,          // workgroups of the attention launch = N_SHARED + N_TILE + N_ROW / 4
  H_HQ,
  H_HKV,
  H_D,
  H_N_SEQS,
  H_TOTAL_Q,
  H_SHARED_OFF,    // word offset of the shared-prefix templates
  H_TILE_OFF,      // word offset of the tile templates
  H_ROW_OFF,       // word offset of the row templates (whole quads, padded)
  H_GROUP_OFF,     // word offset of the merge-group templates
  H_MEMBER_OFF,    // word offset of the cascade member tables (kv-head 0)
  H_PARTIAL_ROWS,  // rows of partial results in the workspace, all kv-heads
  H_DISPATCH_OFF,  // word offset of the dispatch list (GRID words): kHeaderWords
  H_HEAD_PARTIAL,  // partial rows of one kv-head
  H_N_SHARED_TMPL, // templates of each kind
  H_N_TILE_TMPL,
  H_N_ROW_TMPL,
  H_N_GROUP_TMPL,
  H_TAIL_OFF,      // word offset of the tail table: kXcdQueues list offsets, then lengths
                   // (each list in dispatch order)
  H_N_TAIL,        // tile items in all tail lists
  H_N_WILD,        // wildcard workgroups (dispatch words kWildcard), one per tail item
  H_CTR_OFF,       // word offset of the counters (kCounterWords apart; zero in a fresh plan)
  H_PAD28, H_PAD29, H_PAD30, H_PAD31,
  kHeaderWords = 32
};
constexpr int32_t kDispatchHeadShift = 24;  // template index < 2^24 (all kinds), kv-head < 2^7
constexpr int32_t kDispatchIndexMask = (1 << kDispatchHeadShift) - 1;
// Dispatch word of a wildcard workgroup: it takes tile items one at a time
// from the tail list of its own XCD queue (workgroup b runs on XCD
// b % kXcdQueues), then from the other queues' lists in turn, each list
// claimed through its own device-scope counter, until none is left: XCDs
// that run ahead finish the work of the ones that fall behind, and an XCD
// reads other kv-heads' keys only for the items it takes over at the end.
// Counter q (claims of list q) is at word H_CTR_OFF + q * kCounterWords, the
// count of finished wildcard workgroups after them; the last wildcard
// workgroup resets them all to zero.
constexpr int32_t kWildcard = kDispatchIndexMask;
constexpr int32_t kXcdQueues = 8;
constexpr int32_t kCounterWords = 32;  // one 128-byte line per counter
constexpr int32_t kCounterBlockWords = (kXcdQueues + 1) * kCounterWords;

// Work item (tile or row item; templates hold kvh = 0): rows [row0, row0 +
// nrows) of sequence seq's packed (query, head-in-group) rows for kv-head
// kvh, keys [kv0, kv1).
// Row rho is query rho / G, q-head kvh * G + rho % G.  part = -1: write the
// final output; otherwise the item writes normalised partial outputs and
// log-sum-exps at workspace rows part + (rho - row0).  seq = -1: empty slot.
// flags: kItemStream = no other item reads the item's keys (a few-row
// sequence's private key range), so its copies need not stay in L2.
enum : int32_t {
  I_SEQ = 0, I_KVH, I_ROW0, I_NROWS, I_KV0, I_KV1, I_PART, I_FLAGS,
  kItemWords = 8
};

constexpr int32_t kItemStream = 1;

// Shared-prefix item: gathered rows [row0, row0 + nrows) of a cascade group's
// members (member m owns gathered rows m * rpm .. m * rpm + rpm - 1, its own
// rows in order) for kv-head kvh, over the group's shared keys [kv0, kv1),
// which every member's block table maps to the same blocks (read from
// sequence block_seq's row).  The member table at word offset members holds
// (sequence, partial base) pairs for kv-head 0; member m's row rho goes to
// partial row base + rho (+ the kv-head's partial offset).
enum : int32_t {
  S_MEMBERS = 0, S_KVH, S_ROW0, S_NROWS, S_KV0, S_KV1, S_RPM, S_BLOCK_SEQ,
  kSharedWords = 8
};

// Merge group: rows [row0, row0 + nrows) of (seq, kvh) were computed by
// nsplit parts; part s of row rho is at partial row part + s * stride + (rho - row0).
enum : int32_t {
  G_SEQ = 0, G_KVH, G_ROW0, G_NROWS, G_NSPLIT, G_PART, G_STRIDE, G_PAD1,
  kGroupWords = 8
};

// pa_plan_info.variant: 0 float32 kernel; bf16 plans 1, plus 2 when some
// row item holds more than 16 rows (selects the wide row-item kernel), plus 4
// when the plan has tail lists (selects a kernel with wildcard workgroups).
constexpr int32_t kVariantBf16 = 1;
constexpr int32_t kVariantWideRows = 2;
constexpr int32_t kVariantTail = 4;

constexpr int32_t kTileRows = 128;    // rows per tile item (4 waves x 32)
constexpr int32_t kRowItemRows = 32;  // rows per single-wave item (two 16-column MFMA tiles)
constexpr int32_t kMergeRows = 4;     // rows per merge group (one wavefront each)
constexpr int32_t kRowSeqRows = 64;   // sequences with at most this many rows use row items
constexpr int32_t kKeyStep = 32;      // keys per row-item inner iteration
constexpr int32_t kRowItemBlocks = 64;  // most blocks (of 16 keys) one row item spans
constexpr int32_t kTileStep = 64;     // keys per tile-item inner iteration
constexpr int32_t kSharedChunk = 6144;  // most shared keys one cascade item covers
constexpr int32_t kSharedMinKeys = 256; // shorter shared prefixes are not split off

}  // namespace pa
