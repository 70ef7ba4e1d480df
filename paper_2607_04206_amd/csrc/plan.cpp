// Host-side planner of the mixed block-decode / prefill attention call.
//
// Host only: no HIP call is made here, so every descriptor check runs (and is
// testable) on a CPU. The planner validates the batch, cuts it into
// work-groups for the two launch shapes, splits long contexts, orders the
// work-groups longest first and sizes the split-KV workspace.
//
// Work-group shapes (the kernels in attn_fwd.hip hold the matching templates):
//   decode-shaped  (n_i <= 32, a block decode): one work-group per (item, KV
//                  head, context chunk); each wave holds the 32 block rows of
//                  one query head of the GQA group, so every K/V tile staged
//                  in LDS serves the whole group. With few query heads per
//                  group, extra waves split the chunk further.
//   prefill-shaped (n_i > 32, a whole prefill): one work-group per (item,
//                  query head, 128-row block); four waves of 32 rows share
//                  each staged K/V tile. At head_dim 128, when no block
//                  decode joins this launch and every such item is long, the
//                  wide shape instead: 256-row blocks on eight waves with
//                  128-key stages (one work-group per CU).
// In a batch that holds prefills, block decodes whose GQA group has at least
// four query heads are cut into prefill-shaped work-groups instead (one query
// head per wave, kTileHeadsAcross): they join the prefill launch, where the
// longest-first order puts them last, so they fill the tail of the prefill
// work rather than running after it, and they are split only where the
// context range limit requires (no split, no merge for typical contexts).
// A small decode-only batch of such groups takes the same tiles, with its
// contexts cut to fill the CUs.
#include <algorithm>
#include <cstring>
#include <numeric>
#include <string>
#include <vector>

#include "../../include/sangam_attn.h"
#include "page_check.h"
#include "plan_format.h"

namespace sangam {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }
void clear_error() { g_last_error.clear(); }

static sangam_status fail(sangam_status code, const std::string& msg) {
    set_error(msg);
    return code;
}

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
static inline uint64_t align256(uint64_t x) { return (x + 255u) & ~uint64_t(255); }

// Query heads per decode work-group: the whole GQA group when it fits in
// eight waves, else the largest divisor of the group that does.
static int decode_q_waves(int group) {
    if (group <= 8) return group;
    for (int w = 8; w >= 1; --w)
        if (group % w == 0) return w;
    return 1;
}

// Context sub-range waves of a decode work-group. MHA (one query head per
// work-group) measured fastest with two context-splitting waves and two
// work-groups per CU; pairs of query heads split two ways as well.
static int decode_kv_waves(int qw) {
    if (qw <= 2) return 2;
    return 1;
}

// Shortest context chunk the planner cuts for balance in a launch that fills
// the CUs (forced splits above kForcedSplitLen aside): a chunk must carry
// enough keys to amortize a work-group's prologue and its merge traffic. A
// GQA chunk also writes (and the merge reads back) a G x 32-row fp32 partial,
// about the bytes of 1024 keys of its K/V at G = 7, so GQA takes the same
// floor as MHA (measured on 96 Dream decodes of 28/4 heads: 79 us with 2048,
// 82-99 us with 1024, 102-135 us with no balance split).
static int64_t min_chunk(int /*qw*/) { return 2048; }
// the same floor while a decode launch leaves CUs idle (see below)
static int64_t min_chunk_idle(int qw) { return qw == 1 ? 256 : 512; }

// XCDs of the chip (each with its own L2), and the rounds of tiles per
// work-group slot from which a prefill-shaped launch takes the XCD-aware order
constexpr int kXcds = 8;
constexpr size_t kXcdOrderMinRounds = 8;

// Longest context an item may have: tile key ranges are int32, and a split's
// end (its start plus the chunk) must stay representable.
constexpr int64_t kMaxKvLen = int64_t(1) << 30;

const PlanHeader* check_plan(const void* plan) {
    if (!plan) return nullptr;
    const PlanHeader* h = static_cast<const PlanHeader*>(plan);
    if (h->magic != kPlanMagic || h->version != kPlanVersion) return nullptr;
    return h;
}

}  // namespace sangam

using namespace sangam;

extern "C" const char* sangam_last_error(void) { return g_last_error.c_str(); }

extern "C" int32_t sangam_version(void) { return 0x000100; }

extern "C" sangam_status sangam_attn_plan(const sangam_attn_desc* d, void* plan_buf, size_t cap,
                                          size_t* used) {
    clear_error();
    if (!d || !used) return fail(SANGAM_ERR_INVALID_ARG, "desc and used must not be NULL");
    *used = 0;
    const int n_items = d->num_items;
    if (n_items < 1) return fail(SANGAM_ERR_INVALID_ARG, "num_items must be >= 1");
    if (!d->q_indptr || !d->q_offset || !d->kv_len || !d->page_indptr || !d->page_ids)
        return fail(SANGAM_ERR_INVALID_ARG, "descriptor arrays must not be NULL");
    if (d->num_q_heads < 1 || d->num_kv_heads < 1)
        return fail(SANGAM_ERR_INVALID_ARG, "head counts must be >= 1");
    if (d->num_q_heads % d->num_kv_heads != 0)
        return fail(SANGAM_ERR_UNSUPPORTED, "num_q_heads must be a multiple of num_kv_heads");
    if (d->head_dim != 64 && d->head_dim != 128)
        return fail(SANGAM_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
    if (d->page_size != 16) return fail(SANGAM_ERR_UNSUPPORTED, "page_size must be 16");
    if (d->num_pool_pages < 1 || d->num_pool_pages > INT32_MAX)
        return fail(SANGAM_ERR_INVALID_ARG, "num_pool_pages must be in [1, 2^31)");
    if (!(d->sm_scale > 0.0f) || d->sm_scale != d->sm_scale || d->sm_scale > 1e30f)
        return fail(SANGAM_ERR_INVALID_ARG, "sm_scale must be a positive finite number");
    if (d->force_kv_splits < 0) return fail(SANGAM_ERR_INVALID_ARG, "force_kv_splits must be >= 0");
    if (d->num_cus < 0) return fail(SANGAM_ERR_INVALID_ARG, "num_cus must be >= 0");
    if (d->q_indptr[0] != 0 || d->page_indptr[0] != 0)
        return fail(SANGAM_ERR_INVALID_ARG, "q_indptr[0] and page_indptr[0] must be 0");

    const int hq = d->num_q_heads, hkv = d->num_kv_heads, D = d->head_dim;
    const int G = hq / hkv;
    const int num_cus = d->num_cus ? d->num_cus : 256;

    // ---- per-item validation. With a position list, an item whose rows sit
    // on one contiguous range is a block (offset = its first position); any
    // other is a per-token cached decode (kItemPosList).
    int64_t total_q = 0;
    std::vector<int32_t> offset(n_items);
    std::vector<char> listed(n_items, 0);
    for (int i = 0; i < n_items; ++i) {
        const int64_t n = int64_t(d->q_indptr[i + 1]) - d->q_indptr[i];
        const int64_t L = d->kv_len[i];
        if (n < 1)
            return fail(SANGAM_ERR_INVALID_ARG, "item " + std::to_string(i) + ": n_i must be >= 1");
        if (L < 1 || L > kMaxKvLen)
            return fail(SANGAM_ERR_INVALID_ARG, "item " + std::to_string(i) + ": kv_len must be in [1, 2^30]");
        int64_t o = d->q_offset[i];
        if (d->q_pos) {
            const int32_t* pp = d->q_pos + d->q_indptr[i];
            bool contiguous = true;
            for (int64_t r = 0; r < n; ++r) {
                if (pp[r] < 0 || pp[r] >= L || (r > 0 && pp[r] <= pp[r - 1]))
                    return fail(SANGAM_ERR_INVALID_ARG, "item " + std::to_string(i) +
                                                            ": positions must increase strictly inside [0, kv_len)");
                contiguous = contiguous && pp[r] == pp[0] + r;
            }
            o = pp[0];
            if (!contiguous) {
                if (n > kWaveRows || n == L)
                    return fail(SANGAM_ERR_INVALID_ARG,
                                "item " + std::to_string(i) + ": a non-contiguous position list holds at most " +
                                    std::to_string(kWaveRows) + " rows");
                listed[i] = 1;
            }
        }
        if (o < 0 || o + n > L)
            return fail(SANGAM_ERR_INVALID_ARG,
                        "item " + std::to_string(i) + ": need 0 <= q_offset and q_offset + n <= kv_len");
        offset[i] = int32_t(o);
        const int64_t np = int64_t(d->page_indptr[i + 1]) - d->page_indptr[i];
        if (np != ceil_div(L, d->page_size))
            return fail(SANGAM_ERR_INVALID_ARG,
                        "item " + std::to_string(i) + ": page count must be ceil(kv_len / page_size)");
        total_q += n;
    }
    if (total_q > INT32_MAX) return fail(SANGAM_ERR_INVALID_ARG, "too many query rows");
    const int64_t total_pages = d->page_indptr[n_items];

    // ---- page ids: in range and never shared within the batch (two items
    // writing into one page would race)
    {
        bool alias;
        const int64_t k = find_bad_page(d->page_ids, total_pages, d->num_pool_pages, &alias);
        if (k >= 0 && !alias)
            return fail(SANGAM_ERR_PAGE_RANGE, "page id " + std::to_string(d->page_ids[k]) + " at entry " +
                                                   std::to_string(k) + " is outside the pool");
        if (k >= 0)
            return fail(SANGAM_ERR_PAGE_ALIAS, "page id " + std::to_string(d->page_ids[k]) + " is listed twice");
    }

    // ---- splits: decode-shaped contexts longer than kForcedSplitLen are always
    // split; others are cut so that the decode launch has about four
    // work-groups per CU. Prefill-shaped items already give one work-group per
    // 128 rows and head, and block decodes fused into the prefill launch run
    // beside them, so both are split only on request (or where the context
    // range limit of cached rows requires it), except fused block decodes of
    // a small decode-only batch (below).
    const int qw = decode_q_waves(G);
    const int kw = decode_kv_waves(qw);
    const int heads_per_tile = qw;
    const int tiles_per_kv_head = G / heads_per_tile;
    bool has_prefill = false;
    for (int i = 0; i < n_items && !has_prefill; ++i)
        has_prefill = int64_t(d->q_indptr[i + 1]) - d->q_indptr[i] > kWaveRows;
    int64_t decode_keys = 0, decode_units = 0, decode_ctx = 0;
    for (int i = 0; i < n_items; ++i) {
        const int64_t n = int64_t(d->q_indptr[i + 1]) - d->q_indptr[i];
        if (n <= kWaveRows) {
            decode_keys += int64_t(hkv) * tiles_per_kv_head * d->kv_len[i];
            decode_units += int64_t(hkv) * tiles_per_kv_head;
            decode_ctx += d->kv_len[i];
        }
    }
    // Block decodes of a GQA group of >= kPrefillQWaves query heads run as
    // heads-across prefill-shaped tiles (one query head per wave, 4 waves on
    // 4 SIMDs) in a batch that holds prefills, and also in a small decode-only
    // batch: there a whole-group work-group (G waves on 4 SIMDs) leaves most
    // CUs idle and each runs its stages at the pace of its busiest SIMD, while
    // the heads-across tiles spread the group over ceil(G / 4) work-groups
    // (measured on 28/4 heads, 1 to 16 decodes of 1024 keys: 15-35 % faster).
    // Larger decode-only batches keep the whole-group tiles, which read each
    // K/V byte once per group rather than once per work-group.
    const int fused_tiles_per_kv_head = int(ceil_div(G, kPrefillQWaves));
    const bool fuse = G >= kPrefillQWaves && (has_prefill || 2 * decode_units < int64_t(num_cus));
    // a decode-only batch fused this way is still small: its contexts are cut
    // so that the launch has about two work-groups per CU
    int64_t fused_chunk = kForcedSplitLen;
    if (fuse && !has_prefill) {
        const int64_t units = decode_units / tiles_per_kv_head * fused_tiles_per_kv_head;
        const int64_t floor_keys = 4 * units <= int64_t(num_cus) ? 256 : 512;
        fused_chunk = std::min<int64_t>(
            kForcedSplitLen,
            std::max<int64_t>(floor_keys, round_up(ceil_div(int64_t(hkv) * fused_tiles_per_kv_head * decode_ctx,
                                                            2 * int64_t(num_cus)),
                                                   kKeyAlign)));
    }
    if (fuse) decode_keys = decode_units = 0;  // no decode-shaped work-group
    // prefill-shaped tiles: the wide (eight-wave, 128-key stage) shape when
    // the launch holds no fused block decodes (they take one query head per
    // wave of a four-wave tile) and every prefill-shaped item is long, so
    // that few of the 256-row tiles run part-empty
    bool wide = D == 128 && has_prefill;
    for (int i = 0; i < n_items && wide; ++i) {
        const int64_t n = int64_t(d->q_indptr[i + 1]) - d->q_indptr[i];
        if (n > kWaveRows ? n < kWidePrefillMinRows : fuse) wide = false;
    }
    const int prefill_rows = wide ? kWidePrefillRows : kPrefillRows;
    // While the unsplit decode work-groups would leave CUs idle (a small
    // batch: fewer than two MHA work-groups, or one GQA work-group, per CU),
    // a call is bound by the latency of each work-group's stage chain, not by
    // bandwidth: then chunks go down to min_chunk_idle keys, at a merge cost
    // that stays small in absolute terms.
    const bool underfilled = decode_units < int64_t(num_cus) * (qw == 1 ? 2 : 1);
    int64_t chunk = ceil_div(decode_keys, 4 * int64_t(num_cus));
    chunk = std::min<int64_t>(std::max<int64_t>(round_up(std::max<int64_t>(chunk, 1), kKeyAlign),
                                                underfilled ? min_chunk_idle(qw) : min_chunk(qw)),
                              kForcedSplitLen);
    if (underfilled) {
        // Cutting further than the work-groups the chip keeps resident (two
        // MHA or one GQA whole-group work-group per CU) only adds merge work
        // and per-tile start-up: the chunk is the shortest (from the floor
        // above, in kKeyAlign steps) whose tiles fit in those slots. A split
        // of a GQA block decode also writes partial O for all G query heads
        // of the group, about as many bytes as the chunk's K/V for the Dream
        // shape. (Measured: 6-15 LLaDA decodes of 1024 keys 17-30 % faster,
        // 48 Dream decodes 50 instead of 63 us, 1-4 and 32 decodes unchanged.)
        const int64_t slots = int64_t(num_cus) * (qw == 1 ? 2 : 1);
        auto tiles_at = [&](int64_t c) {
            int64_t n = 0;
            for (int i = 0; i < n_items; ++i)
                if (int64_t(d->q_indptr[i + 1]) - d->q_indptr[i] <= kWaveRows)
                    n += int64_t(hkv) * tiles_per_kv_head * ceil_div(d->kv_len[i], c);
            return n;
        };
        int64_t lo = chunk, hi = kForcedSplitLen;  // tiles_at(hi) <= slots: the launch is underfilled
        if (tiles_at(lo) > slots) {
            while (hi - lo > kKeyAlign) {  // invariant: tiles_at(lo) > slots >= tiles_at(hi)
                const int64_t mid = round_up((lo + hi) / 2, kKeyAlign);
                if (mid >= hi) break;
                if (tiles_at(mid) > slots) lo = mid;
                else hi = mid;
            }
            chunk = hi;
        }
    }

    std::vector<ItemRec> items(n_items);
    std::vector<int32_t> positions;    // rows of kItemPosList items
    std::vector<uint32_t> page_info;   // per page, when any item is kItemPosList
    if (std::find(listed.begin(), listed.end(), 1) != listed.end()) page_info.assign(total_pages, 0u);
    int64_t ws_floats = 0;
    int n_merge = 0, n_split_items = 0, max_splits = 1;
    for (int i = 0; i < n_items; ++i) {
        ItemRec& it = items[i];
        it.q_start = d->q_indptr[i];
        it.n = d->q_indptr[i + 1] - d->q_indptr[i];
        it.o = offset[i];
        it.L = d->kv_len[i];
        it.page_start = d->page_indptr[i];
        it.flags = listed[i] ? kItemPosList : 0;
        it.pos_start = int32_t(positions.size());
        if (listed[i]) {
            const int32_t* pp = d->q_pos + it.q_start;
            positions.insert(positions.end(), pp, pp + it.n);
            for (int r = 0; r < it.n; ++r) page_info[it.page_start + (pp[r] >> 4)] |= 1u << (pp[r] & 15);
            uint32_t before = 0;  // listed positions on earlier pages
            for (int64_t k = 0; k < ceil_div(it.L, d->page_size); ++k) {
                uint32_t& e = page_info[it.page_start + k];
                const uint32_t cnt = uint32_t(__builtin_popcount(e));
                e |= before << kPageInfoRowShift;
                before += cnt;
            }
        }
        int64_t S;
        if (d->force_kv_splits > 0) {
            S = std::min<int64_t>(d->force_kv_splits, ceil_div(it.L, kKeyAlign));
        } else if (it.n <= kWaveRows && !fuse) {
            S = std::max<int64_t>(ceil_div(it.L, kForcedSplitLen), ceil_div(it.L, chunk));
        } else if (it.n <= kWaveRows) {
            S = ceil_div(it.L, fused_chunk);
        } else {
            S = 1;
        }
        // a tile that reads cached rows stages its page ids in LDS, which
        // bounds its context range
        const bool all_fresh = it.o == 0 && it.n == it.L;
        if (!all_fresh) S = std::max<int64_t>(S, ceil_div(it.L, kMaxCachedRange));
        int64_t len = round_up(ceil_div(it.L, S), kKeyAlign);
        S = ceil_div(it.L, len);  // no empty chunk
        it.num_splits = int32_t(S);
        it.split_len = int32_t(len);
        it.merge_base = -1;
        it.ws_o = it.ws_lse = 0;
        if (S > 1) {
            it.merge_base = n_merge;
            n_merge += it.n;
            ++n_split_items;
            max_splits = std::max<int>(max_splits, int(S));
            it.ws_o = ws_floats;
            ws_floats += S * it.n * int64_t(hq) * D;
            ws_floats = round_up(ws_floats, 64);
            it.ws_lse = ws_floats;
            ws_floats += S * it.n * int64_t(hq);
            ws_floats = round_up(ws_floats, 64);
        }
    }

    // ---- tiles
    std::vector<TileRec> dec, pre;
    std::vector<int64_t> dec_cost, pre_cost;
    {
        int64_t nd = 0, np = 0;
        for (int i = 0; i < n_items; ++i) {
            const ItemRec& it = items[i];
            if (it.n <= kWaveRows && fuse) np += int64_t(it.num_splits) * hkv * fused_tiles_per_kv_head;
            else if (it.n <= kWaveRows) nd += int64_t(it.num_splits) * hkv * tiles_per_kv_head;
            else np += int64_t(it.num_splits) * hq * ceil_div(it.n, prefill_rows);
        }
        dec.reserve(size_t(nd)); dec_cost.reserve(size_t(nd));
        pre.reserve(size_t(np)); pre_cost.reserve(size_t(np));
    }
    int64_t n_fused = 0;  // (item, chunk) pairs cut into prefill-shaped tiles
    for (int i = 0; i < n_items; ++i) {
        const ItemRec& it = items[i];
        for (int s = 0; s < it.num_splits; ++s) {
            const int32_t kb = s * it.split_len;
            const int32_t ke = std::min<int32_t>(it.L, kb + it.split_len);
            if (it.n <= kWaveRows && fuse) {
                for (int g = 0; g < hkv; ++g)
                    for (int t = 0; t < fused_tiles_per_kv_head; ++t) {
                        TileRec tr{i, g, g * G + t * kPrefillQWaves, 0, kb, ke, s, kTileHeadsAcross};
                        pre.push_back(tr);
                        pre_cost.push_back(int64_t(ke - kb) * kPrefillQWaves);
                    }
                ++n_fused;
            } else if (it.n <= kWaveRows) {
                for (int g = 0; g < hkv; ++g)
                    for (int t = 0; t < tiles_per_kv_head; ++t) {
                        TileRec tr{i, g, g * G + t * heads_per_tile, 0, kb, ke, s, 0};
                        dec.push_back(tr);
                        dec_cost.push_back(int64_t(ke - kb));
                    }
            } else {
                const int nrb = int(ceil_div(it.n, prefill_rows));
                for (int h = 0; h < hq; ++h)
                    for (int rb = 0; rb < nrb; ++rb) {
                        TileRec tr{i, h / G, h, rb * prefill_rows, kb, ke, s, 0};
                        pre.push_back(tr);
                        const int rows = std::min(prefill_rows, it.n - rb * prefill_rows);
                        pre_cost.push_back(int64_t(ke - kb) * ((rows + kWaveRows - 1) / kWaveRows));
                    }
            }
        }
    }
    // longest first, ties in creation order: one sort of (-cost, index) pairs
    auto lpt = [](std::vector<TileRec>& v, const std::vector<int64_t>& c) {
        std::vector<std::pair<int64_t, size_t>> key(v.size());
        for (size_t k = 0; k < v.size(); ++k) key[k] = {-c[k], k};
        std::sort(key.begin(), key.end());
        std::vector<TileRec> out(v.size());
        for (size_t k = 0; k < key.size(); ++k) out[k] = v[key[k].second];
        v.swap(out);
    };
    lpt(dec, dec_cost);
    lpt(pre, pre_cost);
    // XCD-aware order of a long prefill-shaped launch. The dispatcher deals
    // work-groups to the kXcds XCDs in turn (block b to XCD b mod kXcds, up
    // to a fixed rotation), and each XCD has its own L2. Cut the
    // longest-first list into chunks of kXcds x C tiles (C = the launch's
    // slots per XCD) and give each XCD C consecutive tiles of every chunk:
    // they are row blocks of one query head, so the XCD's work-groups stream
    // the same K/V at once and share it in L2 (prefill-heavy: 46 % less
    // traffic beyond L2, time unchanged). Only with at least
    // kXcdOrderMinRounds rounds of tiles per slot: in a shorter launch the
    // chunks split the longest-first balance unevenly across XCDs.
    {
        const size_t C = size_t(std::max(1, num_cus / kXcds)) * (prefill_rows == kWidePrefillRows ? 1 : 2);
        const size_t C8 = C * kXcds;
        if (pre.size() >= kXcdOrderMinRounds * C8) {
            std::vector<TileRec> out(pre.size());
            for (size_t base = 0; base < pre.size(); base += C8) {
                const size_t M = std::min(C8, pre.size() - base);
                const size_t c = M / kXcds;  // a last, partial chunk keeps its remainder in order
                for (size_t q = 0; q < M; ++q) {
                    const size_t dst = q < c * kXcds ? base + kXcds * (q % c) + q / c : base + q;
                    out[dst] = pre[base + q];
                }
            }
            pre.swap(out);
        }
    }
    if (dec.size() > size_t(INT32_MAX) || pre.size() > size_t(INT32_MAX))
        return fail(SANGAM_ERR_INVALID_ARG, "batch too large");

    std::vector<MergeRow> merge;
    merge.reserve(n_merge);
    for (int i = 0; i < n_items; ++i)
        if (items[i].num_splits > 1)
            for (int r = 0; r < items[i].n; ++r) merge.push_back(MergeRow{i, r});

    // ---- layout of the blob
    uint64_t off = align256(sizeof(PlanHeader));
    const uint64_t off_items = off;
    off = align256(off + sizeof(ItemRec) * items.size());
    const uint64_t off_dec = off;
    off = align256(off + sizeof(TileRec) * dec.size());
    const uint64_t off_pre = off;
    off = align256(off + sizeof(TileRec) * pre.size());
    const uint64_t off_merge = off;
    off = align256(off + sizeof(MergeRow) * merge.size());
    const uint64_t off_pos = off;
    off = align256(off + sizeof(int32_t) * positions.size());
    const uint64_t off_pinfo = off;
    off = align256(off + sizeof(uint32_t) * page_info.size());
    const uint64_t total = off;

    *used = size_t(total);
    if (!plan_buf || cap < total)
        return fail(SANGAM_ERR_BUFFER, "plan buffer needs " + std::to_string(total) + " bytes");

    uint8_t* base = static_cast<uint8_t*>(plan_buf);
    std::memset(base, 0, total);
    PlanHeader h{};
    h.magic = kPlanMagic;
    h.version = kPlanVersion;
    h.total_bytes = total;
    h.num_items = n_items;
    h.hq = hq;
    h.hkv = hkv;
    h.d = D;
    h.group = G;
    h.page_size = d->page_size;
    h.sm_scale = d->sm_scale;
    h.scale_log2 = d->sm_scale * 1.44269504088896340736f;
    h.num_pool_pages = d->num_pool_pages;
    h.total_q = total_q;
    h.total_pages = total_pages;
    h.n_decode_tiles = int32_t(dec.size());
    h.decode_qw = qw;
    h.decode_kw = kw;
    h.decode_nb = qw == 1 ? 1 : 2;
    h.n_prefill_tiles = int32_t(pre.size());
    h.prefill_nb = wide ? 4 : 2;
    h.n_merge_rows = n_merge;
    h.num_split_items = n_split_items;
    h.max_splits = max_splits;
    h.prefill_rows = prefill_rows;
    h.n_fused_decode_tiles = int32_t(n_fused * hkv * fused_tiles_per_kv_head);
    h.workspace_bytes = ws_floats * int64_t(sizeof(float));
    h.off_items = off_items;
    h.off_decode_tiles = off_dec;
    h.off_prefill_tiles = off_pre;
    h.off_merge = off_merge;
    h.off_positions = off_pos;
    h.off_page_info = off_pinfo;
    std::memcpy(base, &h, sizeof h);
    if (!items.empty()) std::memcpy(base + off_items, items.data(), sizeof(ItemRec) * items.size());
    if (!dec.empty()) std::memcpy(base + off_dec, dec.data(), sizeof(TileRec) * dec.size());
    if (!pre.empty()) std::memcpy(base + off_pre, pre.data(), sizeof(TileRec) * pre.size());
    if (!merge.empty()) std::memcpy(base + off_merge, merge.data(), sizeof(MergeRow) * merge.size());
    if (!positions.empty()) std::memcpy(base + off_pos, positions.data(), sizeof(int32_t) * positions.size());
    if (!page_info.empty()) std::memcpy(base + off_pinfo, page_info.data(), sizeof(uint32_t) * page_info.size());
    return SANGAM_OK;
}

extern "C" size_t sangam_plan_workspace_bytes(const void* plan_buf) {
    const PlanHeader* h = check_plan(plan_buf);
    return h ? size_t(h->workspace_bytes) : 0;
}

extern "C" sangam_status sangam_plan_get_info(const void* plan_buf, sangam_plan_info* info) {
    clear_error();
    const PlanHeader* h = check_plan(plan_buf);
    if (!h) return fail(SANGAM_ERR_PLAN, "not a plan of this library version");
    if (!info) return fail(SANGAM_ERR_INVALID_ARG, "info must not be NULL");
    info->num_items = h->num_items;
    info->num_decode_tiles = h->n_decode_tiles;
    info->num_prefill_tiles = h->n_prefill_tiles;
    info->num_split_items = h->num_split_items;
    info->max_splits = h->max_splits;
    info->decode_q_waves = h->decode_qw;
    info->decode_kv_waves = h->decode_kw;
    info->num_fused_decode_tiles = h->n_fused_decode_tiles;
    info->total_q_rows = h->total_q;
    info->workspace_bytes = h->workspace_bytes;
    info->plan_bytes = int64_t(h->total_bytes);
    return SANGAM_OK;
}

extern "C" sangam_status sangam_plan_item_splits(const void* plan_buf, int32_t item, int32_t* num_splits,
                                                 int32_t* starts, int32_t cap) {
    clear_error();
    const PlanHeader* h = check_plan(plan_buf);
    if (!h) return fail(SANGAM_ERR_PLAN, "not a plan of this library version");
    if (item < 0 || item >= h->num_items || !num_splits)
        return fail(SANGAM_ERR_INVALID_ARG, "bad item or NULL num_splits");
    const ItemRec* items =
        reinterpret_cast<const ItemRec*>(static_cast<const uint8_t*>(plan_buf) + h->off_items);
    const ItemRec& it = items[item];
    *num_splits = it.num_splits;
    if (starts) {
        if (cap < it.num_splits + 1) return fail(SANGAM_ERR_BUFFER, "starts needs num_splits + 1 entries");
        for (int s = 0; s < it.num_splits; ++s) starts[s] = s * it.split_len;
        starts[it.num_splits] = it.L;
    }
    return SANGAM_OK;
}
