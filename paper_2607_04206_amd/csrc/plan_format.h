// Launch-plan blob shared by the host planner (plan.cpp) and the gfx950
// kernels (attn_fwd.hip). The blob is position independent: every array is
// addressed by a byte offset from the start of the blob, so the same bytes
// work in host memory and, after a plain copy, in device memory.
#pragma once

#include <stdint.h>

namespace sangam {

constexpr uint32_t kPlanMagic = 0x50414753u;  // "SGAP"
constexpr uint32_t kPlanVersion = 4;  // 4: prefill_rows may be the wide tile (256)

constexpr int kWaveRows = 32;       // query rows held by one wave (one decode block)
constexpr int kPrefillQWaves = 4;   // waves of a prefill-shaped work-group
constexpr int kPrefillQBlocks = 1;  // 32-row query blocks per prefill wave
constexpr int kPrefillRows = kWaveRows * kPrefillQBlocks * kPrefillQWaves;
// Wide prefill-shaped work-groups (head_dim 128, batches whose prefill
// launch holds no fused block decodes and only long prefill-shaped items):
// eight waves of 32 rows of one query head, 128-key stages, one work-group
// per CU; half the barriers per key of the four-wave tile.
constexpr int kWidePrefillQWaves = 8;
constexpr int kWidePrefillRows = kWaveRows * kWidePrefillQWaves;
constexpr int kWidePrefillMinRows = 1024;  // every prefill-shaped item at least this long
constexpr int kKeyAlign = 64;       // split boundaries are multiples of this many keys
constexpr int kForcedSplitLen = 8192;  // a decode context longer than this is always split
// Longest context range of one tile that reads cached (paged) rows: the
// kernel stages that range's page ids in LDS.
constexpr int kMaxCachedRange = 8192;

// One work item of the batch (a block decode or a whole prefill).
struct ItemRec {
    int32_t q_start;     // first packed query row
    int32_t n;           // query rows
    int32_t o;           // position of the first query row (block offset)
    int32_t L;           // context length
    int32_t page_start;  // first entry of the item in page_ids
    int32_t num_splits;  // context chunks (1 = written straight to out)
    int32_t split_len;   // keys per chunk (multiple of kKeyAlign), last may be shorter
    int32_t merge_base;  // first merge row of the item, -1 when not split
    int64_t ws_o;        // float offset of partial O  [num_splits][n][Hq][D]
    int64_t ws_lse;      // float offset of partial LSE [num_splits][n][Hq]
    int32_t flags;       // kItemPosList or 0
    int32_t pos_start;   // first entry of the item's positions (kItemPosList)
};

// ItemRec.flags: the rows sit at the listed positions (positions[pos_start +
// r]), not at o + r; page_info[page_start + k] describes the item's page k.
constexpr int32_t kItemPosList = 1;

// page_info entry of a page of a kItemPosList item: bit s (s < 16) is set when
// slot s holds a listed position; bits 16..31 count the listed positions on
// the item's earlier pages, so the fresh row of slot s is that count plus the
// set bits below s.
constexpr int kPageInfoRowShift = 16;

// TileRec.flags: the waves of a prefill-shaped work-group hold consecutive
// query heads (q_head0 + wave, those inside the tile's GQA group) of one
// block decode instead of consecutive 32-row blocks of one head.
constexpr int32_t kTileHeadsAcross = 1;

// One work-group of an attention launch.
struct TileRec {
    int32_t item;
    int32_t kv_head;
    int32_t q_head0;   // first query head of the tile
    int32_t row0;      // first query row (local to the item)
    int32_t kv_begin;  // context range [kv_begin, kv_end)
    int32_t kv_end;
    int32_t split;     // chunk index of the context
    int32_t flags;     // kTileHeadsAcross or 0
};

// One (item, row) whose split partial results the merge kernel combines.
struct MergeRow {
    int32_t item;
    int32_t row;
};

struct PlanHeader {
    uint32_t magic;
    uint32_t version;
    uint64_t total_bytes;

    int32_t num_items;
    int32_t hq;
    int32_t hkv;
    int32_t d;
    int32_t group;      // hq / hkv
    int32_t page_size;
    float sm_scale;
    float scale_log2;   // sm_scale * log2(e): scores enter exp2 in this scale
    int64_t num_pool_pages;
    int64_t total_q;
    int64_t total_pages;

    // decode-shaped launch: items with n <= kWaveRows; one work-group holds
    // decode_qw query heads (one per wave) x decode_kw context sub-ranges
    int32_t n_decode_tiles;
    int32_t decode_qw;
    int32_t decode_kw;
    int32_t decode_nb;   // 32-key blocks per wave per stage
    // prefill-shaped launch: items with n > kWaveRows; kPrefillQWaves waves
    // of 32 rows of one query head. In a batch that holds prefills (or a
    // small decode-only batch), block decodes whose GQA group spans at least
    // kPrefillQWaves query heads run in this launch too (kTileHeadsAcross
    // tiles, n_fused_decode_tiles of n_prefill_tiles), filling its tail
    // instead of a launch of their own.
    int32_t n_prefill_tiles;
    int32_t prefill_nb;
    int32_t n_merge_rows;
    int32_t num_split_items;
    int32_t max_splits;
    int32_t prefill_rows;  // query rows per prefill-shaped tile: kPrefillRows or kWidePrefillRows
    int32_t n_fused_decode_tiles;
    int32_t reserved;
    int64_t workspace_bytes;

    uint64_t off_items;
    uint64_t off_decode_tiles;
    uint64_t off_prefill_tiles;
    uint64_t off_merge;
    uint64_t off_positions;  // int32 positions of kItemPosList items
    uint64_t off_page_info;  // uint32 per page (page_indptr order), when any item is kItemPosList
};

static_assert(sizeof(ItemRec) == 56, "ItemRec layout is part of the blob format");
static_assert(sizeof(TileRec) == 32, "TileRec layout is part of the blob format");
static_assert(sizeof(MergeRow) == 8, "MergeRow layout is part of the blob format");
static_assert(sizeof(PlanHeader) == 176, "PlanHeader layout is part of the blob format");

}  // namespace sangam
