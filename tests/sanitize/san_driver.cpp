// Drives the host code of the library (planner, KV hand-off planner, deficit
// admission) and the C oracle over many random and malformed inputs, built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_sanitize.py. Any out-of-bounds access, leak, overflow or other
// undefined behaviour aborts the run; the driver also checks the documented
// size protocol of each planner (a too-small buffer is refused with the size
// it needs, the exact size is accepted).
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../include/sangam_attn.h"
#include "../../include/sangam_kv.h"
#include "../../include/sangam_sched.h"

extern "C" {
int oracle_attn(int32_t n_items, int32_t hq, int32_t hkv, int32_t d, float sm_scale, const int32_t* q_indptr,
                const int32_t* q_offset, const int32_t* q_pos, const int32_t* kv_len, const int64_t* ctx_indptr,
                const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new, const uint16_t* k_ctx,
                const uint16_t* v_ctx, const int64_t* sel, int64_t n_sel, double* out, double* lse);
int oracle_weights(int32_t n_items, int32_t hq, int32_t hkv, int32_t d, float sm_scale, const int32_t* q_indptr,
                   const int32_t* q_offset, const int32_t* q_pos, const int32_t* kv_len, const int64_t* ctx_indptr,
                   const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new, const uint16_t* k_ctx,
                   const uint16_t* v_ctx, int64_t row, int32_t head, double* w_out);
int oracle_expected_kv(int32_t n_items, int32_t hkv, int32_t d, const int32_t* q_indptr, const int32_t* q_offset,
                       const int32_t* q_pos, const int32_t* kv_len, const int64_t* ctx_indptr, const uint16_t* k_new,
                       const uint16_t* v_new, const uint16_t* k_ctx, const uint16_t* v_ctx, int32_t item,
                       uint16_t* k_out, uint16_t* v_out);
}

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static uint64_t next() {  // xorshift64*
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return g_state * 0x2545F4914F6CDD1Dull;
}
static int64_t rnd(int64_t lo, int64_t hi) { return lo + int64_t(next() % uint64_t(hi - lo + 1)); }
static bool chance(int pct) { return rnd(0, 99) < pct; }

static int failures = 0;
static int plans_ok = 0, kv_plans_ok = 0, oracle_ok = 0;
#define EXPECT(c)                                                          \
    do {                                                                   \
        if (!(c)) {                                                        \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            ++failures;                                                    \
        }                                                                  \
    } while (0)

struct Batch {
    std::vector<int32_t> q_indptr, q_offset, kv_len, page_indptr, page_ids, q_pos;
    int64_t pool = 0;
};

// a batch of block decodes, larger cached blocks, per-token position lists
// and whole prefills; with `bad`, one field is broken on purpose
static Batch make_batch(int n_items, bool bad) {
    Batch b;
    b.q_indptr.push_back(0);
    b.page_indptr.push_back(0);
    bool lists = chance(30);
    for (int i = 0; i < n_items; ++i) {
        int kind = int(rnd(0, 3));
        int32_t L = int32_t(chance(10) ? rnd(8193, 20000) : rnd(1, 3000));
        int32_t n, o;
        if (kind == 0) {  // block decode
            n = int32_t(std::min<int64_t>(rnd(1, 32), L));
            o = int32_t(rnd(0, L - n));
        } else if (kind == 1 && L > 33) {  // larger cached block
            n = int32_t(rnd(33, std::min<int64_t>(300, L)));
            o = int32_t(rnd(0, L - n));
        } else {  // whole prefill
            L = std::min<int32_t>(L, 3000);
            n = L;
            o = 0;
        }
        b.q_offset.push_back(o);
        b.kv_len.push_back(L);
        b.q_indptr.push_back(b.q_indptr.back() + n);
        b.page_indptr.push_back(b.page_indptr.back() + (L + 15) / 16);
        for (int r = 0; r < n; ++r) b.q_pos.push_back(o + r);
        if (lists && n <= 32 && n < L && chance(50)) {  // scattered positions instead
            std::vector<int32_t> all(L);
            for (int p = 0; p < L; ++p) all[p] = p;
            for (int k = 0; k < n; ++k) std::swap(all[k], all[k + int(rnd(0, L - 1 - k))]);
            std::vector<int32_t> pick(all.begin(), all.begin() + n);
            std::sort(pick.begin(), pick.end());
            std::copy(pick.begin(), pick.end(), b.q_pos.end() - n);
        }
    }
    if (!lists) b.q_pos.clear();
    const int32_t pages = b.page_indptr.back();
    b.pool = pages + rnd(0, pages + 3);
    std::vector<int32_t> perm(size_t(b.pool));
    for (int64_t k = 0; k < b.pool; ++k) perm[size_t(k)] = int32_t(k);
    for (int64_t k = 0; k < pages; ++k) std::swap(perm[size_t(k)], perm[size_t(k + rnd(0, b.pool - 1 - k))]);
    b.page_ids.assign(perm.begin(), perm.begin() + pages);
    if (bad) {
        switch (rnd(0, 6)) {
            case 0: if (pages) b.page_ids[size_t(rnd(0, pages - 1))] = int32_t(b.pool + rnd(0, 5)); break;
            case 1: if (pages > 1) b.page_ids[1] = b.page_ids[0]; break;
            case 2: b.q_offset[size_t(rnd(0, n_items - 1))] = -1; break;
            case 3: b.kv_len[size_t(rnd(0, n_items - 1))] += 17; break;
            case 4: b.page_indptr[0] = 1; break;
            case 5: b.kv_len[size_t(rnd(0, n_items - 1))] = 0; break;
            default: if (!b.q_pos.empty()) b.q_pos[0] = -3; break;
        }
    }
    return b;
}

static void fuzz_attn_plan(int iters) {
    for (int it = 0; it < iters; ++it) {
        const bool bad = chance(25);
        Batch b = make_batch(int(rnd(1, 24)), bad);
        const int hkv = int(rnd(1, 8));
        int hq = hkv * int(rnd(1, 8));
        if (chance(5)) hq += 1;  // not a multiple
        sangam_attn_desc d{};
        d.num_items = int32_t(b.kv_len.size());
        d.num_q_heads = hq;
        d.num_kv_heads = hkv;
        d.head_dim = chance(95) ? (chance(50) ? 64 : 128) : 96;
        d.page_size = chance(97) ? 16 : 8;
        d.force_kv_splits = int32_t(chance(70) ? 0 : rnd(1, 9));
        d.num_pool_pages = b.pool;
        d.sm_scale = chance(98) ? 0.0883883f : -1.0f;
        d.num_cus = int32_t(chance(50) ? 0 : rnd(1, 300));
        d.q_indptr = b.q_indptr.data();
        d.q_offset = b.q_offset.data();
        d.kv_len = b.kv_len.data();
        d.page_indptr = b.page_indptr.data();
        d.page_ids = b.page_ids.data();
        d.q_pos = b.q_pos.empty() ? nullptr : b.q_pos.data();
        size_t used = 0;
        sangam_status st = sangam_attn_plan(&d, nullptr, 0, &used);
        if (st != SANGAM_ERR_BUFFER) {
            EXPECT(st < 0 && st != SANGAM_OK);
            EXPECT(std::strlen(sangam_last_error()) > 0);
            continue;
        }
        EXPECT(used > 0);
        std::vector<uint8_t> small(used - 1);
        size_t used2 = 0;
        EXPECT(sangam_attn_plan(&d, small.data(), small.size(), &used2) == SANGAM_ERR_BUFFER && used2 == used);
        std::vector<uint8_t> buf(used);
        EXPECT(sangam_attn_plan(&d, buf.data(), buf.size(), &used2) == SANGAM_OK && used2 == used);
        sangam_plan_info info{};
        EXPECT(sangam_plan_get_info(buf.data(), &info) == SANGAM_OK);
        EXPECT(info.num_items == d.num_items);
        EXPECT(size_t(info.workspace_bytes) == sangam_plan_workspace_bytes(buf.data()));
        std::vector<int32_t> starts(size_t(info.max_splits) + 1);
        for (int i = 0; i < d.num_items; ++i) {
            int32_t ns = 0;
            EXPECT(sangam_plan_item_splits(buf.data(), i, &ns, starts.data(), int32_t(starts.size())) == SANGAM_OK);
            EXPECT(ns >= 1 && ns <= info.max_splits && starts[size_t(ns)] == b.kv_len[size_t(i)]);
        }
        int32_t ns = 0;
        EXPECT(sangam_plan_item_splits(buf.data(), d.num_items, &ns, nullptr, 0) == SANGAM_ERR_INVALID_ARG);
        ++plans_ok;
    }
    // malformed calls
    size_t used = 0;
    EXPECT(sangam_attn_plan(nullptr, nullptr, 0, &used) == SANGAM_ERR_INVALID_ARG);
    std::vector<uint8_t> junk(256, 0x5A);
    sangam_plan_info info{};
    EXPECT(sangam_plan_get_info(junk.data(), &info) == SANGAM_ERR_PLAN);
    EXPECT(sangam_plan_workspace_bytes(junk.data()) == 0);
}

static void fuzz_kv_plan(int iters) {
    for (int it = 0; it < iters; ++it) {
        Batch b = make_batch(int(rnd(1, 30)), chance(25));
        sangam_kv_desc d{};
        d.num_items = int32_t(b.kv_len.size());
        d.num_kv_heads = int32_t(rnd(1, 8));
        d.head_dim = chance(95) ? 128 : 80;
        d.page_size = 16;
        d.num_pool_pages = b.pool;
        d.kv_len = b.kv_len.data();
        d.page_indptr = b.page_indptr.data();
        d.page_ids = b.page_ids.data();
        size_t used = 0;
        sangam_status st = sangam_kv_plan(&d, nullptr, 0, &used);
        if (st != SANGAM_ERR_BUFFER) {
            EXPECT(st < 0);
            continue;
        }
        std::vector<uint8_t> buf(used);
        size_t used2 = 0;
        EXPECT(sangam_kv_plan(&d, buf.data(), buf.size(), &used2) == SANGAM_OK && used2 == used);
        int64_t rows = 0;
        for (int32_t L : b.kv_len) rows += L;
        EXPECT(sangam_kv_plan_rows(buf.data()) == rows);
        ++kv_plans_ok;
    }
}

static void fuzz_deficit(int iters) {
    for (int it = 0; it < iters; ++it) {
        std::vector<int64_t> waiting(size_t(rnd(0, 8)));
        for (auto& w : waiting) w = rnd(chance(3) ? 0 : 1, 6000);
        int64_t deficit = rnd(chance(3) ? -5 : 0, 6000);
        int32_t admitted = -1;
        const int64_t tau = rnd(chance(3) ? -1 : 0, 8192);
        sangam_status st = sangam_deficit_admit(tau, rnd(0, 4000), int32_t(rnd(0, 64)),
                                                waiting.empty() ? nullptr : waiting.data(),
                                                int32_t(waiting.size()), &deficit, &admitted);
        if (st == SANGAM_OK) EXPECT(admitted >= 0 && admitted <= int32_t(waiting.size()) && deficit >= 0);
    }
}

static void fuzz_oracle(int iters) {
    for (int it = 0; it < iters; ++it) {
        const int n_items = int(rnd(1, 4));
        const int hkv = int(rnd(1, 3)), hq = hkv * int(rnd(1, 3)), d = int(rnd(1, 3)) * 8;
        std::vector<int32_t> q_indptr{0}, q_offset, kv_len;
        std::vector<int64_t> ctx{0};
        for (int i = 0; i < n_items; ++i) {
            const int32_t L = int32_t(rnd(1, 40));
            const bool prefill = chance(40);
            const int32_t n = prefill ? L : int32_t(rnd(1, L));
            q_offset.push_back(prefill ? 0 : int32_t(rnd(0, L - n)));
            kv_len.push_back(L);
            q_indptr.push_back(q_indptr.back() + n);
            ctx.push_back(ctx.back() + (prefill ? 0 : L));
        }
        if (chance(10)) q_offset[0] = kv_len[0];  // invalid: rows past the context
        const int64_t T = q_indptr.back();
        auto fill = [](size_t cnt) {
            std::vector<uint16_t> v(cnt == 0 ? 1 : cnt);
            for (auto& x : v) x = uint16_t(0x3C00 + (next() % 0x0800)) ^ uint16_t((next() & 1) << 15);
            return v;
        };
        auto q = fill(size_t(T * hq * d)), kn = fill(size_t(T * hkv * d)), vn = fill(size_t(T * hkv * d));
        auto kc = fill(size_t(ctx.back() * hkv * d)), vc = fill(size_t(ctx.back() * hkv * d));
        std::vector<double> out(size_t(T * hq * d)), lse(size_t(T * hq));
        int rc = oracle_attn(n_items, hq, hkv, d, 0.125f, q_indptr.data(), q_offset.data(), nullptr, kv_len.data(),
                             ctx.data(), q.data(), kn.data(), vn.data(), kc.data(), vc.data(), nullptr, 0, out.data(),
                             lse.data());
        if (rc != 0) continue;
        ++oracle_ok;
        std::vector<int64_t> sel{0, T * hq - 1};
        std::vector<double> o2(2 * size_t(d)), l2(2);
        EXPECT(oracle_attn(n_items, hq, hkv, d, 0.125f, q_indptr.data(), q_offset.data(), nullptr, kv_len.data(),
                           ctx.data(), q.data(), kn.data(), vn.data(), kc.data(), vc.data(), sel.data(), 2, o2.data(),
                           l2.data()) == 0);
        std::vector<int64_t> badsel{T * hq};
        EXPECT(oracle_attn(n_items, hq, hkv, d, 0.125f, q_indptr.data(), q_offset.data(), nullptr, kv_len.data(),
                           ctx.data(), q.data(), kn.data(), vn.data(), kc.data(), vc.data(), badsel.data(), 1,
                           o2.data(), l2.data()) != 0);
        std::vector<double> w(static_cast<size_t>(kv_len[0]));
        EXPECT(oracle_weights(n_items, hq, hkv, d, 0.125f, q_indptr.data(), q_offset.data(), nullptr, kv_len.data(),
                              ctx.data(), q.data(), kn.data(), vn.data(), kc.data(), vc.data(), 0, 0, w.data()) == 0);
        for (int i = 0; i < n_items; ++i) {
            std::vector<uint16_t> ko(static_cast<size_t>(kv_len[size_t(i)]) * hkv * d), vo(ko.size());
            EXPECT(oracle_expected_kv(n_items, hkv, d, q_indptr.data(), q_offset.data(), nullptr, kv_len.data(),
                                      ctx.data(), kn.data(), vn.data(), kc.data(), vc.data(), i, ko.data(),
                                      vo.data()) == 0);
        }
    }
}

int main(int argc, char** argv) {
    if (argc > 1) g_state = std::strtoull(argv[1], nullptr, 10) | 1u;
    fuzz_attn_plan(400);
    fuzz_kv_plan(200);
    fuzz_deficit(5000);
    fuzz_oracle(200);
    std::printf("sanitized driver: %d plans, %d KV plans, %d oracle calls accepted; %d failed checks\n", plans_ok,
                kv_plans_ok, oracle_ok, failures);
    if (plans_ok < 100 || kv_plans_ok < 50 || oracle_ok < 50) {
        std::printf("too few accepted inputs to exercise the code\n");
        return 1;
    }
    return failures ? 1 : 0;
}
