// Host-side plan of the paged-KV export / import: validates a batch of
// requests and lists, per page, where its slots go in the packed buffers.
// No HIP call is made here, so every check runs (and is testable) on a CPU.
#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/sangam_kv.h"
#include "kv_format.h"
#include "page_check.h"

namespace sangam {
void set_error(const std::string& msg);
void clear_error();

const KvPlanHeader* check_kv_plan(const void* plan) {
    if (!plan) return nullptr;
    const KvPlanHeader* h = static_cast<const KvPlanHeader*>(plan);
    if (h->magic != kKvPlanMagic || h->version != kKvPlanVersion) return nullptr;
    return h;
}
}  // namespace sangam

using namespace sangam;

static sangam_status kv_fail(sangam_status code, const std::string& msg) {
    set_error(msg);
    return code;
}

extern "C" sangam_status sangam_kv_plan(const sangam_kv_desc* d, void* plan_buf, size_t cap, size_t* used) {
    clear_error();
    if (!d || !used) return kv_fail(SANGAM_ERR_INVALID_ARG, "desc and used must not be NULL");
    *used = 0;
    const int n = d->num_items;
    if (n < 1) return kv_fail(SANGAM_ERR_INVALID_ARG, "num_items must be >= 1");
    if (!d->kv_len || !d->page_indptr || !d->page_ids)
        return kv_fail(SANGAM_ERR_INVALID_ARG, "kv_len, page_indptr and page_ids must not be NULL");
    if (d->num_kv_heads < 1) return kv_fail(SANGAM_ERR_INVALID_ARG, "num_kv_heads must be >= 1");
    if (d->head_dim != 64 && d->head_dim != 128)
        return kv_fail(SANGAM_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
    if (d->page_size != 16) return kv_fail(SANGAM_ERR_UNSUPPORTED, "page_size must be 16");
    if (d->num_pool_pages < 1) return kv_fail(SANGAM_ERR_INVALID_ARG, "num_pool_pages must be >= 1");
    if (d->page_indptr[0] != 0) return kv_fail(SANGAM_ERR_INVALID_ARG, "page_indptr[0] must be 0");
    int64_t rows = 0;
    for (int i = 0; i < n; ++i) {
        const int64_t L = d->kv_len[i];
        if (L < 1) return kv_fail(SANGAM_ERR_INVALID_ARG, "item " + std::to_string(i) + ": kv_len must be >= 1");
        const int64_t np = int64_t(d->page_indptr[i + 1]) - d->page_indptr[i];
        if (np != (L + 15) / 16)
            return kv_fail(SANGAM_ERR_INVALID_ARG, "item " + std::to_string(i) + ": lists " + std::to_string(np) +
                                                       " pages, its " + std::to_string(L) + " positions need " +
                                                       std::to_string((L + 15) / 16));
        rows += L;
    }
    if (rows > INT32_MAX) return kv_fail(SANGAM_ERR_INVALID_ARG, "more than 2^31 - 1 packed rows");
    const int64_t total_pages = d->page_indptr[n];
    // every page at most once: an import writes each listed page
    bool alias;
    const int64_t bad = find_bad_page(d->page_ids, total_pages, d->num_pool_pages, &alias);
    if (bad >= 0 && !alias)
        return kv_fail(SANGAM_ERR_PAGE_RANGE, "page id " + std::to_string(d->page_ids[bad]) + " outside [0, " +
                                                  std::to_string(d->num_pool_pages) + ")");
    if (bad >= 0) return kv_fail(SANGAM_ERR_PAGE_ALIAS, "page " + std::to_string(d->page_ids[bad]) + " listed twice");
    const uint64_t off_pages = (sizeof(KvPlanHeader) + 255u) & ~uint64_t(255);
    const uint64_t total = off_pages + uint64_t(total_pages) * sizeof(KvPageRec);
    *used = size_t(total);
    if (!plan_buf || cap < total) return kv_fail(SANGAM_ERR_BUFFER, "plan buffer needs " + std::to_string(total) + " bytes");
    uint8_t* base = static_cast<uint8_t*>(plan_buf);
    std::memset(base, 0, size_t(off_pages));
    KvPlanHeader* h = reinterpret_cast<KvPlanHeader*>(base);
    h->magic = kKvPlanMagic;
    h->version = kKvPlanVersion;
    h->total_bytes = total;
    h->num_items = n;
    h->hkv = d->num_kv_heads;
    h->d = d->head_dim;
    h->page_size = d->page_size;
    h->num_pool_pages = d->num_pool_pages;
    h->total_rows = rows;
    h->total_pages = total_pages;
    h->off_pages = off_pages;
    KvPageRec* recs = reinterpret_cast<KvPageRec*>(base + off_pages);
    int64_t row = 0;
    for (int i = 0; i < n; ++i) {
        const int L = d->kv_len[i];
        for (int k = 0; k * 16 < L; ++k) {
            KvPageRec& r = recs[d->page_indptr[i] + k];
            r.page = d->page_ids[d->page_indptr[i] + k];
            r.row0 = int32_t(row + 16 * k);
            r.nslots = L - 16 * k < 16 ? L - 16 * k : 16;
            r.item = i;
        }
        row += L;
    }
    return SANGAM_OK;
}

extern "C" int64_t sangam_kv_plan_rows(const void* plan_buf) {
    const KvPlanHeader* h = check_kv_plan(plan_buf);
    return h ? h->total_rows : 0;
}
