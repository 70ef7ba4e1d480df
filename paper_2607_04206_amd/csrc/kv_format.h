// Plan blob of the paged-KV export / import (kv_plan.cpp writes it,
// kv_copy.hip reads it). Position independent like the attention plan: the
// page records sit at a byte offset from the start of the blob, so the same
// bytes serve in host memory and, after a plain copy, in device memory.
#pragma once

#include <stdint.h>

namespace sangam {

constexpr uint32_t kKvPlanMagic = 0x5056474Bu;  // "KGVP"
constexpr uint32_t kKvPlanVersion = 1;

// One listed page: its slots [0, nslots) hold positions whose packed rows
// start at row0 (slot s <-> packed row row0 + s).
struct KvPageRec {
    int32_t page;
    int32_t row0;
    int32_t nslots;
    int32_t item;
};

struct KvPlanHeader {
    uint32_t magic;
    uint32_t version;
    uint64_t total_bytes;
    int32_t num_items;
    int32_t hkv;
    int32_t d;
    int32_t page_size;
    int64_t num_pool_pages;
    int64_t total_rows;   // sum of L_i: rows of the packed buffers
    int64_t total_pages;  // page records
    uint64_t off_pages;
};

static_assert(sizeof(KvPageRec) == 16, "KvPageRec layout is part of the blob format");
static_assert(sizeof(KvPlanHeader) == 64, "KvPlanHeader layout is part of the blob format");

}  // namespace sangam
