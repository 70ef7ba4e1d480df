// Page-table checks shared by the host planners (plan.cpp, kv_plan.cpp).
#pragma once

#include <stdint.h>

#include <algorithm>
#include <vector>

namespace sangam {

// Checks that every id lies in [0, pool) and that no id is listed twice.
// Returns -1 when both hold; otherwise the entry of the first id out of range
// (*alias = false) or, all ids being in range, an entry whose id was already
// listed (*alias = true). A bitmap over the pool does the duplicate test in
// one pass; a pool far larger than the table falls back to sorting a copy.
inline int64_t find_bad_page(const int32_t* ids, int64_t n, int64_t pool, bool* alias) {
    *alias = false;
    for (int64_t k = 0; k < n; ++k)
        if (ids[k] < 0 || ids[k] >= pool) return k;
    *alias = true;
    if (pool <= std::max<int64_t>(int64_t(1) << 24, 64 * n)) {
        std::vector<uint64_t> seen(size_t((pool + 63) / 64), 0);
        for (int64_t k = 0; k < n; ++k) {
            const uint64_t bit = uint64_t(1) << (ids[k] & 63);
            uint64_t& w = seen[size_t(ids[k] >> 6)];
            if (w & bit) return k;
            w |= bit;
        }
        return -1;
    }
    std::vector<std::pair<int32_t, int64_t>> s(static_cast<size_t>(n));
    for (int64_t k = 0; k < n; ++k) s[size_t(k)] = {ids[k], k};
    std::sort(s.begin(), s.end());
    for (size_t k = 1; k < s.size(); ++k)
        if (s[k].first == s[k - 1].first) return std::max(s[k].second, s[k - 1].second);
    return -1;
}

}  // namespace sangam
