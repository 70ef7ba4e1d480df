// gfx950 kernels of the mixed block-decode / prefill attention call and the
// C-ABI forward entry point that launches them.
//
// What is computed (Sangam paper, Sec. 2.1 and Sec. 2.2): dLLM attention is
// bidirectional, so each query row of an item attends to all L positions of
// its sequence; a block decode recomputes only its 32 block rows and reuses
// the request's approximately cached KV for every other position, a prefill
// brings (and writes back) its whole sequence. Batches mix both kinds
// (Sec. 4.1, Alg. 1); the KV cache is paged with 16-token pages (Sec. 5,
// Sec. 6.1).
//
// Kernels:
//   attn_tiles_kernel one work-group per plan tile: a context range of one
//                     item and KV head against up to 8 x 32 query rows; one
//                     tile per item, KV head and row block also copies the
//                     fresh K/V rows into their cache pages.
//                     Per wave: S^T = K Q^T with v_mfma_f32_32x32x16_bf16
//                     (each lane holds the scores of one query, so row max /
//                     row sum need one cross-half exchange), online softmax
//                     in the exp2 domain, P^T rounded to bf16 feeds
//                     O^T += V^T P^T directly from the score registers.
//                     K/V stream global -> LDS with global_load_lds_dwordx4
//                     into XOR-swizzled tiles (double buffered); V^T operands
//                     come from ds_read_b64_tr_b16 transposing reads. Output
//                     rows leave through LDS, whole rows per 16 lanes.
//   merge_kernel      combines split-context partial (O, LSE) in split order.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/sangam_attn.h"
#include "plan_format.h"

namespace sangam {
void set_error(const std::string& msg);
void clear_error();
const PlanHeader* check_plan(const void* plan);
}  // namespace sangam

using namespace sangam;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define LDS __attribute__((address_space(3)))

struct AttnArgs {
    const TileRec* tiles;
    const ItemRec* items;
    const int32_t* page_ids;
    const uint16_t* q;
    const uint16_t* k_new;
    const uint16_t* v_new;
    uint16_t* k_cache;  // read (cached rows) and written (the fresh rows' pages)
    uint16_t* v_cache;
    uint16_t* out;
    float* lse;
    float* ws;
    const int32_t* positions;    // rows of per-token cached decodes (kItemPosList items)
    const uint32_t* page_info;   // per page of such items: listed slots and earlier rows
    int32_t hq;
    int32_t hkv;
    float scale_log2;
};

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Asynchronous copy of 16 bytes per lane from global memory into LDS
// (global_load_lds_dwordx4): lane l's bytes land at dst_wave + 16 l. Issued
// through inline assembly so that the compiler does not track the LDS write:
// it would otherwise wait for every copy in flight before any later LDS read,
// including the copies that prefetch the next stage into another buffer,
// which serialises the prefetch with the compute it should overlap. The
// kernels order the copies themselves: s_waitcnt vmcnt and a barrier before a
// staged buffer is read, a barrier before it is overwritten. M0 (the LDS
// base) is saved and restored around the copy, with the wait state the
// hardware needs between an M0 write and its use.
__device__ __forceinline__ uint32_t lds_wave_base(LDS void* p) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
}
__device__ __forceinline__ void lds_copy16(const void* src, LDS void* dst_wave) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
        "global_load_lds_dwordx4 %2, off\n\ts_nop 0\n\ts_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_wave_base(dst_wave)), "v"(src)
        : "memory");
}
// the same from a wave-uniform base plus a per-lane 32-bit byte offset
__device__ __forceinline__ void lds_copy16(const void* base, uint32_t off, LDS void* dst_wave) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
        "global_load_lds_dwordx4 %2, %3\n\ts_nop 0\n\ts_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_wave_base(dst_wave)), "v"(off), "s"(base)
        : "memory");
}

// Swizzle of 16-byte chunks inside a staged key row. K rows are read one key
// per lane (ds_read_b128), so consecutive keys rotate their chunks. V rows are
// read four keys at a time by ds_read_b64_tr_b16, so groups of four keys
// spread over the LDS banks.
template <int D>
__device__ __forceinline__ int swz_k(int r) {
    return r & (D / 8 - 1);
}
template <int D>
__device__ __forceinline__ int swz_v(int r) {
    return D == 128 ? ((r & 3) << 2) : (((r >> 1) & 1) << 2);
}

// Cross-half (lane l <-> l ^ 32) pair of a value: v_permlane32_swap with both
// operands x returns (x[l], x[l^32]) for the lower half and (x[l^32], x[l])
// for the upper half, so a symmetric combine of the two results is the pair's.
__device__ __forceinline__ float half_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// The running max moves only when a score exceeds it by more than this (log2
// units), so P <= 2^8 and O is rescaled rarely; the result is unchanged
// because O and l always share the same reference.
constexpr float kRescaleThreshold = 8.0f;

// Work-groups per CU the register budget is sized for: two waves per SIMD for
// four-wave work-groups whose staging fits twice in LDS and whose waves hold
// one query block; one wave per SIMD otherwise.
template <int D, int QW, int KW, int QB, int NB, int NSTAGE>
constexpr int min_blocks_per_cu() {
    return (QB == 1 && QW * KW == 4 && 2 * NSTAGE * (32 * NB * KW) * D * 2 <= 80 * 1024) ? 2 : 1;
}

// One work-group per plan tile: a context range [kv_begin, kv_end) of one
// item and KV head against QW query slots x QB blocks of 32 rows per slot.
//   D      head dim (64, 128)
//   QW     waves holding distinct query rows (query heads of a GQA group when
//          HEADS_ACROSS, else consecutive 32*QB-row blocks of one head)
//   KW     waves splitting each stage's keys (merged through LDS at the end)
//   QB     32-row query blocks per wave: every K and V fragment read from
//          LDS feeds QB MFMAs, so QB = 2 halves LDS traffic per flop
//   NB     32-key blocks per wave per stage
//   NSTAGE K/V stage buffers in LDS (NSTAGE - 1 stages in flight)
template <int D, int QW, int KW, int QB, int NB, int NSTAGE, bool HEADS_ACROSS, int MINB>
__global__ __launch_bounds__(64 * QW * KW, MINB) void attn_tiles_kernel(AttnArgs a) {
    constexpr int NT = 64 * QW * KW;     // threads
    constexpr int KT = 32 * NB;          // keys per wave per stage
    constexpr int STEP = KT * KW;        // keys per stage
    constexpr int NC = D / 8;            // 16-byte chunks per key row
    constexpr int ROWB = D * 2;          // bytes per key row
    constexpr int TILE = STEP * ROWB;    // bytes of one staged K (or V) tile
    constexpr int NCH = STEP * NC;       // 16-byte chunks of one staged tile
    constexpr int NJ = (NCH + NT - 1) / NT;  // chunk rounds per thread
    constexpr int DS = D / 16;           // k-steps of the QK^T contraction
    constexpr int MB = D / 32;           // 32-dim blocks of O^T
    static_assert(NCH % 64 == 0, "a wave moves whole 1 KiB rows of chunks");
    constexpr int MERGE_REGS = MB * 16 + 2;
    static_assert(KW == 1 || QB == 1, "context-splitting waves hold one query block");
    static_assert(!HEADS_ACROSS || QB == 1, "a decode block is 32 rows");
    static_assert(KW == 1 || (QW * (KW - 1) * MERGE_REGS * 64 * 4) <= 2 * NSTAGE * TILE,
                  "cross-wave merge must fit in the stage buffers");
    static_assert(NSTAGE >= 2 && NSTAGE <= 4, "2 to 4 stage buffers");
    // pages a tile's write-back range can touch: its rows at any offset
    constexpr int WPAGES = HEADS_ACROSS ? 16 : (32 * QB * QW + 15) / 16 + 1;
    static_assert(WPAGES <= NT, "one thread per write-back page id");
    // with more than two buffers the wait counts loads, so every wave must
    // issue the same number per stage
    static_assert(NSTAGE == 2 || NCH % NT == 0, "deeper pipelines need whole staging rounds");
    constexpr int MAX_PAGES = kMaxCachedRange / 16;

    __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * NSTAGE * TILE];
    __shared__ int32_t pages[MAX_PAGES];
    __shared__ uint32_t pinfo[MAX_PAGES];  // page_info of the tile's pages (kItemPosList items)
    __shared__ int32_t fpos[kWaveRows];    // the listed positions (kItemPosList items)
    __shared__ int32_t wpages[WPAGES];  // pages of the fresh rows this tile writes back

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = uniform(tid >> 6);
    const int qs = wave % QW;
    const int ks = wave / QW;
    const int qn = lane & 31;   // query (column) this lane holds in each block
    const int hh = lane >> 5;   // half-wave

    const TileRec t = a.tiles[blockIdx.x];
    const ItemRec it = a.items[t.item];
    // heads across the waves: a decode-shaped work-group, or a block decode
    // cut into a prefill-shaped one (whose last tile of a GQA group may hold
    // fewer heads than waves: the extra waves only stage K/V, write back and
    // meet the barriers; they compute and store nothing)
    const bool across = HEADS_ACROSS || (t.flags & kTileHeadsAcross);
    const int head_want = across ? t.q_head0 + qs : t.q_head0;
    const bool head_ok = head_want < (t.kv_head + 1) * (a.hq / a.hkv);
    const int head = head_ok ? head_want : t.q_head0;
    const int row_base = across ? t.row0 : t.row0 + 32 * QB * qs;
    const int kv_begin = t.kv_begin, kv_end = t.kv_end;
    const int nstages = (kv_end - kv_begin + STEP - 1) / STEP;
    // a whole prefill brings every position fresh: no page lookups
    const bool all_fresh = it.o == 0 && it.n == it.L;
    // a per-token cached decode: its rows sit at listed positions
    const bool plist = (it.flags & kItemPosList) != 0;
    const int pg0 = kv_begin >> 4;
    if (!all_fresh) {
        // the tile's page ids, once (the plan keeps such ranges <= kMaxCachedRange):
        // every load is issued before the first LDS store, so a long range
        // costs one memory round trip, not one per round of NT pages
        const int npg = ((kv_end + 15) >> 4) - pg0;
        constexpr int PR = (MAX_PAGES + NT - 1) / NT;  // rounds of the page table per thread
        int32_t pv[PR];
        uint32_t iv[PR];
#pragma unroll
        for (int r = 0; r < PR; ++r) {
            const int k = tid + r * NT;
            if (k < npg) {
                pv[r] = a.page_ids[it.page_start + pg0 + k];
                if (plist) iv[r] = a.page_info[it.page_start + pg0 + k];
            }
        }
#pragma unroll
        for (int r = 0; r < PR; ++r) {
            const int k = tid + r * NT;
            if (k < npg) {
                pages[k] = pv[r];
                if (plist) pinfo[k] = iv[r];
            }
        }
        if (plist && tid < it.n) fpos[tid] = a.positions[it.pos_start + tid];
    }

    // ---- Q fragments (B operand: k = dims, n = query), zero for rows past n
    bf16x8 qf[QB][DS];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int row = row_base + 32 * qb + qn;
        const bool ok = row < it.n;
        const uint16_t* qp = a.q + ((size_t)(it.q_start + (ok ? row : 0)) * a.hq + head) * D;
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            u32x4 v = *(const u32x4*)(qp + 16 * s + 8 * hh);
            if (!ok) v = u32x4{0, 0, 0, 0};
            qf[qb][s] = __builtin_bit_cast(bf16x8, v);
        }
    }

    // ---- stage-invariant staging offsets: thread chunk j of a stage is key
    // row r_j, source chunk (pos ^ swizzle(r_j)) of K and of V
    const size_t row_stride = (size_t)a.hkv * D;                       // elements between positions
    const uint16_t* kfresh = a.k_new + ((size_t)(it.q_start - it.o) * a.hkv + t.kv_head) * D;
    const uint16_t* vfresh = a.v_new + ((size_t)(it.q_start - it.o) * a.hkv + t.kv_head) * D;
    const size_t page_stride = (size_t)a.hkv * 16 * D;
    const uint16_t* kcache = a.k_cache + (size_t)t.kv_head * 16 * D;
    const uint16_t* vcache = a.v_cache + (size_t)t.kv_head * 16 * D;

    // per-thread byte offsets of its chunks within a stage of fresh rows
    // (whole prefills): key row r_j at row_stride, swizzled chunk
    uint32_t foff_k[NJ], foff_v[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int P = j * NT + tid;
        const int r = P / NC;
        const int pos = P % NC;
        foff_k[j] = uint32_t(r * row_stride * 2 + ((pos ^ swz_k<D>(r)) << 4));
        foff_v[j] = uint32_t(r * row_stride * 2 + ((pos ^ swz_v<D>(r)) << 4));
    }
    // the same within a 16-row page (K/V head chunk of the cache) for a stage
    // that starts on a page boundary: key row r_j sits in slot r_j mod 16 of
    // the stage's page r_j / 16
    uint32_t poff_k[NJ], poff_v[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int P = j * NT + tid;
        const int r = P / NC;
        const int pos = P % NC;
        poff_k[j] = uint32_t((r & 15) * ROWB + ((pos ^ swz_k<D>(r)) << 4));
        poff_v[j] = uint32_t((r & 15) * ROWB + ((pos ^ swz_v<D>(r)) << 4));
    }
    // A full stage with no fresh row reads only cached rows. When it starts
    // on a page boundary, each wave's copy instruction covers 64 / NC key rows
    // of one page, so the page base is wave-uniform (scalar registers) and
    // the lanes add the precomputed offsets: no per-lane page lookup,
    // freshness test or 64-bit address arithmetic on the common path.
    auto stage_all_cached = [&](int key0) -> bool {
        if (all_fresh || (kv_begin & 15) != 0) return false;
        if (plist) {
            uint32_t slots = 0;
#pragma unroll
            for (int k = 0; k < STEP / 16; ++k) slots |= pinfo[(key0 >> 4) - pg0 + k];
            return (uniform(int(slots & 0xFFFFu))) == 0;
        }
        return key0 + STEP <= it.o || key0 >= it.o + it.n;
    };

    auto issue_stage = [&](int st, int buf) __attribute__((always_inline)) {
        uint8_t* kb = smem + buf * 2 * TILE;
        uint8_t* vb = kb + TILE;
        const int key0 = kv_begin + st * STEP;
        const bool tail = key0 + STEP > kv_end;
        if (all_fresh && !tail) {
            // uniform base + precomputed 32-bit offsets
            const uint16_t* kbase = kfresh + (size_t)key0 * row_stride;
            const uint16_t* vbase = vfresh + (size_t)key0 * row_stride;
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                if ((NCH % NT) != 0 && j * NT + wave * 64 >= NCH) break;  // wave-uniform
                const int dst = (j * NT + wave * 64) * 16;
                lds_copy16(kbase, foff_k[j], (LDS void*)(kb + dst));
                lds_copy16(vbase, foff_v[j], (LDS void*)(vb + dst));
            }
            return;
        }
        if (!tail && stage_all_cached(key0)) {
            const int prel = (key0 >> 4) - pg0;  // the stage's first page among the tile's
            int pid[NJ];
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                pid[j] = 0;
                if ((NCH % NT) == 0 || j * NT + wave * 64 < NCH)
                    pid[j] = pages[prel + (((j * NT + wave * 64) / NC) >> 4)];
            }
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                if ((NCH % NT) != 0 && j * NT + wave * 64 >= NCH) break;  // wave-uniform
                const size_t off = (size_t)uniform(pid[j]) * page_stride;
                const int dst = (j * NT + wave * 64) * 16;
                lds_copy16(kcache + off, poff_k[j], (LDS void*)(kb + dst));
                lds_copy16(vcache + off, poff_v[j], (LDS void*)(vb + dst));
            }
            return;
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            if ((NCH % NT) != 0 && j * NT + wave * 64 >= NCH) break;  // wave-uniform
            const int P = j * NT + tid;
            const int r = P / NC;
            const int pos = P % NC;
            int p = key0 + r;
            if (tail) p = p < kv_end ? p : kv_begin;  // past the range: a valid row, masked later
            const int ck = (pos ^ swz_k<D>(r)) * 8;
            const int cv = (pos ^ swz_v<D>(r)) * 8;
            // fresh row holding position p, counted from position o (row r
            // sits at o + r in kfresh / vfresh), or -1 for a cached row
            int fr;
            if (all_fresh) {
                fr = p;
            } else if (plist) {
                const uint32_t inf = pinfo[(p >> 4) - pg0];
                const uint32_t below = inf & ((1u << (p & 15)) - 1u);
                fr = (inf >> (p & 15)) & 1u ? int(inf >> kPageInfoRowShift) + __builtin_popcount(below) + it.o : -1;
            } else {
                fr = unsigned(p - it.o) < unsigned(it.n) ? p : -1;
            }
            const uint16_t *ksrc, *vsrc;
            if (fr >= 0) {
                ksrc = kfresh + (size_t)fr * row_stride;
                vsrc = vfresh + (size_t)fr * row_stride;
            } else {
                const size_t off = (size_t)pages[(p >> 4) - pg0] * page_stride + (p & 15) * D;
                ksrc = kcache + off;
                vsrc = vcache + off;
            }
            const int dst = (j * NT + wave * 64) * 16;
            lds_copy16(ksrc + ck, (LDS void*)(kb + dst));
            lds_copy16(vsrc + cv, (LDS void*)(vb + dst));
        }
    };

    // ---- write-back of the fresh K/V rows into their cache pages. Per item
    // and KV head, the tiles of the group's first query head copy the fresh
    // rows they stage (a prefill tile its own row block, a block decode its
    // rows) from LDS, right after the stage lands: no second read of k_new /
    // v_new. Every fresh position lies in exactly one such tile's row block
    // and context range. No tile reads these cache rows (fresh positions come
    // from k_new / v_new, and the planner rejects pages shared between items),
    // so the copy needs no ordering with the attention. The pages of the
    // written range (at most 9) are staged in LDS once, right after the first
    // stage is issued (their wait overlaps that stage's), so the copy loop
    // issues no global load whose wait would also drain the prefetch.
    const int group = a.hq / a.hkv;
    const bool wb_head = across ? t.q_head0 == t.kv_head * group : t.q_head0 % group == 0;
    // positions written: [wb_lo, wb_hi) for a block; for a position list (a
    // decode, so heads-across), its listed positions inside the span from the
    // first to the last listed position
    const int last_pos = plist ? a.positions[it.pos_start + it.n - 1] : it.o + it.n - 1;
    const int wb_lo = max(kv_begin, it.o + (across ? 0 : t.row0));
    const int wb_hi = min(kv_end, across ? last_pos + 1 : it.o + min(it.n, t.row0 + 32 * QB * QW));
    const bool writer = wb_head && wb_lo < wb_hi;
    const int wpg0 = wb_lo >> 4;
    auto write_back = [&](int st) {
        const int key0 = kv_begin + st * STEP;
        const int lo = max(wb_lo, key0), hi = min(wb_hi, key0 + STEP);
        if (lo >= hi) return;
        const uint8_t* kb = smem + (st % NSTAGE) * 2 * TILE;
        const uint8_t* vb = kb + TILE;
        if (plist) {  // the listed positions inside [lo, hi); their pages are the tile's
            for (int cidx = tid; cidx < it.n * NC; cidx += NT) {
                const int p = fpos[cidx / NC], pos = cidx % NC;
                if (p < lo || p >= hi) continue;
                const int r = p - key0;
                const u32x4 kv = *(const LDS u32x4*)(kb + r * ROWB + ((pos ^ swz_k<D>(r)) << 4));
                const u32x4 vv = *(const LDS u32x4*)(vb + r * ROWB + ((pos ^ swz_v<D>(r)) << 4));
                const size_t dst = (((size_t)pages[(p >> 4) - pg0] * a.hkv + t.kv_head) * 16 + (p & 15)) * D + pos * 8;
                *(u32x4*)(a.k_cache + dst) = kv;
                *(u32x4*)(a.v_cache + dst) = vv;
            }
            return;
        }
        for (int cidx = tid; cidx < (hi - lo) * NC; cidx += NT) {
            const int p = lo + cidx / NC, pos = cidx % NC;
            const int r = p - key0;
            const u32x4 kv = *(const LDS u32x4*)(kb + r * ROWB + ((pos ^ swz_k<D>(r)) << 4));
            const u32x4 vv = *(const LDS u32x4*)(vb + r * ROWB + ((pos ^ swz_v<D>(r)) << 4));
            const size_t dst = (((size_t)wpages[(p >> 4) - wpg0] * a.hkv + t.kv_head) * 16 + (p & 15)) * D + pos * 8;
            *(u32x4*)(a.k_cache + dst) = kv;
            *(u32x4*)(a.v_cache + dst) = vv;
        }
    };

    // ---- stage-invariant LDS read offsets
    // K (A operand): lane reads key qn of each 32-key block, chunk 2k + hh
    int koff[DS];
#pragma unroll
    for (int k = 0; k < DS; ++k) koff[k] = qn * ROWB + (((2 * k + hh) ^ swz_k<D>(qn)) << 4);
    // V^T (A operand) via transposing reads: 16-lane group g16 covers dims
    // mb*32 + (g16&1)*16 .. +15; lane (r4, j4) points at key row 4hh + r4 (+8),
    // dims 4 j4 .. 4 j4 + 3 of that group
    const int g16 = lane >> 4;
    const int r4 = (lane >> 2) & 3;
    const int j4 = lane & 3;
    const int vrow = (4 * hh + r4) * ROWB;
    int voff[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        const int dim = mb * 32 + (g16 & 1) * 16 + 4 * j4;
        voff[mb] = vrow + (((dim >> 3) ^ swz_v<D>(4 * hh + r4)) << 4) + (dim & 7) * 2;
    }

    f32x16 o[QB][MB];
    float m_used[QB];  // reference max (log2 domain) of this lane's query, per block
    float l_run[QB];   // sum of rounded P over this lane's half of the keys
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        m_used[qb] = -INFINITY;
        l_run[qb] = 0.0f;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int i = 0; i < 16; ++i) o[qb][mb][i] = 0.0f;
    }
    const float c = a.scale_log2;

    if (!all_fresh) __syncthreads();  // page ids visible before the first loads

    // S^T = K Q^T for this wave's NB 32-key blocks of stage st: rows = keys,
    // columns = queries; each K fragment feeds the QB query blocks
    // The QK^T MFMAs run at raised wave priority: with two waves per SIMD,
    // the wave that reaches its QK^T chain keeps the matrix core fed while the
    // other works through its softmax (measured about 1 % faster on prefills).
    auto qk = [&](int st, f32x16 (&s)[QB][NB]) {
        const uint8_t* kb = smem + (st % NSTAGE) * 2 * TILE + ks * KT * ROWB;
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
#pragma unroll
                for (int i = 0; i < 16; ++i) s[qb][b][i] = 0.0f;
#pragma unroll
            for (int k = 0; k < DS; ++k) {
                const bf16x8 kf = *(const LDS bf16x8*)(kb + b * 32 * ROWB + koff[k]);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    s[qb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qb][k], s[qb][b], 0, 0, 0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
    };

    // Online softmax of stage st's scores (exp2 domain) and O^T += V^T P^T.
    // The reference max moves (and O, l are rescaled) only when a score
    // exceeds it by more than kRescaleThreshold, which is rare after the first
    // stage. tail: the stage may hold keys past the range (set to -inf).
    auto softmax_pv = [&](int st, f32x16 (&s)[QB][NB], bool tail) {
        const uint8_t* vb = smem + (st % NSTAGE) * 2 * TILE + TILE + ks * KT * ROWB;
        if (tail) {
            const int key0 = kv_begin + st * STEP + ks * KT;  // this wave's first key
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = key0 + b * 32 + 8 * (i >> 2) + 4 * hh + (i & 3);
#pragma unroll
                    for (int qb = 0; qb < QB; ++qb)
                        if (key >= kv_end) s[qb][b][i] = -INFINITY;
                }
        }
        float mx_s[QB];
        bool any_need = false;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            float mx = -INFINITY;
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[qb][b][i]);
            mx_s[qb] = half_max(mx) * c;
            any_need |= mx_s[qb] > m_used[qb] + kRescaleThreshold;
        }
        if (__builtin_amdgcn_ballot_w64(any_need)) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                const bool need = mx_s[qb] > m_used[qb] + kRescaleThreshold;
                const float alpha = need ? __builtin_amdgcn_exp2f(m_used[qb] - mx_s[qb]) : 1.0f;
                m_used[qb] = need ? mx_s[qb] : m_used[qb];
                l_run[qb] *= alpha;
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) o[qb][mb][i] *= alpha;
            }
        }

        // P = exp2(s c - m) rounded to bf16 (the PV operand); l += the rounded values
        bf16x8 pf[QB][NB][2];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            const float mref = m_used[qb] == -INFINITY ? 0.0f : m_used[qb];
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int i = 0; i < 16; i += 2) {
                    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[qb][b][i], c, -mref));
                    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[qb][b][i + 1], c, -mref));
                    const bf16x2 pp = {(__bf16)p0, (__bf16)p1};
                    l_run[qb] = __builtin_amdgcn_fdot2_f32_bf16(pp, bf16x2{(__bf16)1.0f, (__bf16)1.0f},
                                                                l_run[qb], false);
                    pf[qb][b][i >> 3][i & 7] = pp[0];
                    pf[qb][b][i >> 3][(i & 7) + 1] = pp[1];
                }
        }

        // lane slot j of P^T holds key 16kk + 8(j/4) + 4hh + j%4; each V
        // fragment feeds the QB query blocks
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    const uint8_t* vp = vb + (b * 32 + kk * 16) * ROWB + voff[mb];
                    const bf16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LDS bf16x4*)(vp));
                    const bf16x4 vc = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LDS bf16x4*)(vp + 8 * ROWB));
                    const bf16x8 vf = {va[0], va[1], va[2], va[3], vc[0], vc[1], vc[2], vc[3]};
#pragma unroll
                    for (int qb = 0; qb < QB; ++qb)
                        o[qb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[qb][b][kk], o[qb][mb], 0, 0, 0);
                }
    };

    // Stages st+1 .. st+NSTAGE-1 are in flight while stage st is computed.
    // Loads complete in order, so waiting for stage st leaves the later
    // stages outstanding.
    constexpr int LPS = 2 * NJ;  // loads per stage per thread (K and V)
    const int full_stages = (kv_end - kv_begin) / STEP;  // stages with no key past the range
    auto wait_stage = [&](int st) {
        const int later = min(NSTAGE - 2, nstages - 1 - st);  // stages issued after st
        if (NSTAGE >= 4 && later >= 2)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LPS) : "memory");
        else if (NSTAGE >= 3 && later >= 1)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPS) : "memory");
        else
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };
    for (int k = 0; k < NSTAGE - 1 && k < nstages; ++k) issue_stage(k, k);
    if (writer && !plist && tid < ((wb_hi + 15) >> 4) - wpg0) wpages[tid] = a.page_ids[it.page_start + wpg0 + tid];
    int st = 0;
    for (; st < full_stages; ++st) {
        wait_stage(st);
        __syncthreads();
        if (st + NSTAGE - 1 < nstages) issue_stage(st + NSTAGE - 1, (st + NSTAGE - 1) % NSTAGE);
        if (writer) write_back(st);
        if (head_ok) {  // a wave past its tile's GQA group only stages and writes back
            f32x16 sc[QB][NB];
            qk(st, sc);
            softmax_pv(st, sc, false);
        }
    }
    if (st < nstages) {  // the last, partial stage
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (writer) write_back(st);
        if (head_ok) {
            f32x16 sc[QB][NB];
            qk(st, sc);
            softmax_pv(st, sc, true);
        }
    }

    // ---- combine the context sub-ranges of the waves that share query rows
    if constexpr (KW > 1) {
        __syncthreads();
        float* mbuf = reinterpret_cast<float*>(smem);
        if (ks > 0) {
            float* dst = mbuf + (size_t)((qs * (KW - 1) + (ks - 1)) * MERGE_REGS) * 64;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 16; ++i) dst[(mb * 16 + i) * 64 + lane] = o[0][mb][i];
            dst[(MB * 16) * 64 + lane] = m_used[0];
            dst[(MB * 16 + 1) * 64 + lane] = l_run[0];
        }
        __syncthreads();
        if (ks > 0) return;
        float m_tot = m_used[0];
#pragma unroll
        for (int k = 1; k < KW; ++k) {
            const float* src = mbuf + (size_t)((qs * (KW - 1) + (k - 1)) * MERGE_REGS) * 64;
            m_tot = fmaxf(m_tot, src[(MB * 16) * 64 + lane]);
        }
        // wave ks = 0 always holds a valid key, so m_tot is finite
        const float sc0 = __builtin_amdgcn_exp2f(m_used[0] - m_tot);
        l_run[0] *= sc0;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int i = 0; i < 16; ++i) o[0][mb][i] *= sc0;
#pragma unroll
        for (int k = 1; k < KW; ++k) {
            const float* src = mbuf + (size_t)((qs * (KW - 1) + (k - 1)) * MERGE_REGS) * 64;
            const float sck = __builtin_amdgcn_exp2f(src[(MB * 16) * 64 + lane] - m_tot);
            l_run[0] += sck * src[(MB * 16 + 1) * 64 + lane];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 16; ++i) o[0][mb][i] += sck * src[(mb * 16 + i) * 64 + lane];
        }
        m_used[0] = m_tot;
    }

    // ---- epilogue
    // Rows written straight to `out` leave through LDS where it holds them:
    // each lane stages its query's dims in 8-byte pieces, then 16 consecutive
    // lanes store one whole row in 16-byte pieces (stored directly, one
    // instruction would leave 16-byte fragments of 32 rows).
    constexpr int EROW = D * 2 + 16;  // bytes per staged row: 16-byte aligned, shifted by four banks
    constexpr int EBASE = KW > 1 ? QW * (KW - 1) * MERGE_REGS * 64 * 4 : 0;  // past the merge data
    constexpr bool ESTAGE = EBASE + QW * QB * 32 * EROW <= 2 * NSTAGE * TILE;
    const bool split_out = it.num_splits > 1;  // split partials go to the workspace in fp32
    if constexpr (ESTAGE && KW == 1) {
        if (!split_out) __syncthreads();  // every wave is past its last stage's reads
    }
    uint8_t* ebuf = smem + EBASE + qs * (QB * 32 * EROW);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int row = row_base + 32 * qb + qn;
        const float l_tot = half_sum(l_run[qb]);
        const float inv = 1.0f / l_tot;
        const float lse_val = m_used[qb] * 0.69314718055994530942f + logf(l_tot);
        if (ESTAGE && !split_out) {
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int dim = mb * 32 + 8 * q4 + 4 * hh;
                    const bf16x4 v = {(__bf16)(o[qb][mb][4 * q4] * inv), (__bf16)(o[qb][mb][4 * q4 + 1] * inv),
                                      (__bf16)(o[qb][mb][4 * q4 + 2] * inv),
                                      (__bf16)(o[qb][mb][4 * q4 + 3] * inv)};
                    *(LDS u32x2*)(ebuf + (32 * qb + qn) * EROW + dim * 2) = __builtin_bit_cast(u32x2, v);
                }
            if (row < it.n && head_ok && hh == 0 && a.lse) a.lse[(size_t)(it.q_start + row) * a.hq + head] = lse_val;
            continue;
        }
        if (row >= it.n || !head_ok) continue;
        if (split_out) {
            const size_t prow = (size_t)(t.split * it.n + row) * a.hq + head;
            float* po = a.ws + it.ws_o + prow * D;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int dim = mb * 32 + 8 * q4 + 4 * hh;
                    float4 v = {o[qb][mb][4 * q4] * inv, o[qb][mb][4 * q4 + 1] * inv,
                                o[qb][mb][4 * q4 + 2] * inv, o[qb][mb][4 * q4 + 3] * inv};
                    *(float4*)(po + dim) = v;
                }
            if (hh == 0) a.ws[it.ws_lse + prow] = lse_val;
        } else {
            uint16_t* op = a.out + ((size_t)(it.q_start + row) * a.hq + head) * D;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int dim = mb * 32 + 8 * q4 + 4 * hh;
                    const bf16x4 v = {(__bf16)(o[qb][mb][4 * q4] * inv), (__bf16)(o[qb][mb][4 * q4 + 1] * inv),
                                      (__bf16)(o[qb][mb][4 * q4 + 2] * inv),
                                      (__bf16)(o[qb][mb][4 * q4 + 3] * inv)};
                    *(u32x2*)(op + dim) = __builtin_bit_cast(u32x2, v);
                }
            if (hh == 0 && a.lse) a.lse[(size_t)(it.q_start + row) * a.hq + head] = lse_val;
        }
    }
    if constexpr (ESTAGE) {
        if (!split_out && head_ok) {
            // the wave reads back only rows it staged itself
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            constexpr int CPR = D / 8;           // 16-byte pieces per row
            constexpr int NCE = QB * 32 * CPR;   // pieces per wave
            static_assert(NCE % 64 == 0, "whole rounds of 64 lanes");
#pragma unroll
            for (int j = 0; j < NCE / 64; ++j) {
                const int c = j * 64 + lane;
                const int r = c / CPR, col = c % CPR;  // staged row r is row row_base + r
                if (row_base + r < it.n) {
                    const u32x4 v = *(const LDS u32x4*)(ebuf + r * EROW + col * 16);
                    *(u32x4*)(a.out + ((size_t)(it.q_start + row_base + r) * a.hq + head) * D + col * 8) = v;
                }
            }
        }
    }
}

// --------------------------------------------------------------- split merge
struct MergeArgs {
    const MergeRow* rows;
    const ItemRec* items;
    const float* ws;
    uint16_t* out;
    float* lse;
    int32_t hq;
    int32_t d;
};

// grid: (merge row, 256-element slice of the row's Hq x D/4 float4 outputs);
// one thread per float4 of one head, so that every partial of a row is
// loaded by a different thread in parallel
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a) {
    const MergeRow mr = a.rows[blockIdx.x];
    const ItemRec it = a.items[mr.item];
    const int S = it.num_splits;
    const int d4n = a.d / 4;
    const int e = blockIdx.y * 256 + threadIdx.x;
    if (e >= a.hq * d4n) return;
    const int head = e / d4n;
    const int d4 = e - head * d4n;
    float mx = -INFINITY;
    for (int s = 0; s < S; ++s) mx = fmaxf(mx, a.ws[it.ws_lse + (size_t)(s * it.n + mr.row) * a.hq + head]);
    float tot = 0.0f;
    float4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int s = 0; s < S; ++s) {
        const size_t prow = (size_t)(s * it.n + mr.row) * a.hq + head;
        const float w = __expf(a.ws[it.ws_lse + prow] - mx);
        const float4 v = *(const float4*)(a.ws + it.ws_o + prow * a.d + 4 * d4);
        tot += w;
        acc.x += w * v.x;
        acc.y += w * v.y;
        acc.z += w * v.z;
        acc.w += w * v.w;
    }
    const float inv = 1.0f / tot;
    const bf16x4 v = {(__bf16)(acc.x * inv), (__bf16)(acc.y * inv), (__bf16)(acc.z * inv), (__bf16)(acc.w * inv)};
    const size_t orow = (size_t)(it.q_start + mr.row) * a.hq + head;
    *(u32x2*)(a.out + orow * a.d + 4 * d4) = __builtin_bit_cast(u32x2, v);
    if (d4 == 0 && a.lse) a.lse[orow] = mx + logf(tot);
}

// ------------------------------------------------------------------ launch
// Start / stop events attached to one launch (timed entry point), or none.
struct LaunchEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};

// A launch with events carries them in its dispatch (hipExtLaunchKernel), so
// their timestamps bracket the kernel itself, as a kernel trace does.
template <typename Args>
hipError_t launch(const void* fn, dim3 grid, unsigned threads, Args args, hipStream_t stream, LaunchEvents ev) {
    void* kargs[] = {&args};
    if (!ev.start && !ev.stop) return hipLaunchKernel(fn, grid, dim3(threads), kargs, 0, stream);
    return hipExtLaunchKernel(fn, grid, dim3(threads), kargs, 0, stream, ev.start, ev.stop, 0);
}

template <int D, int QW, int KW, int QB, int NB, bool HA, int NSTAGE = 2>
hipError_t launch_tiles(const AttnArgs& args, int n_tiles, hipStream_t stream, LaunchEvents ev) {
    constexpr int MINB = min_blocks_per_cu<D, QW, KW, QB, NB, NSTAGE>();
    return launch(reinterpret_cast<const void*>(&attn_tiles_kernel<D, QW, KW, QB, NB, NSTAGE, HA, MINB>),
                  dim3(unsigned(n_tiles)), unsigned(64 * QW * KW), args, stream, ev);
}

template <int D>
hipError_t launch_decode(const AttnArgs& args, int n_tiles, int qw, int kw, int nb, hipStream_t stream,
                         LaunchEvents ev, bool* supported) {
    *supported = true;
    if (qw == 1 && kw == 2 && nb == 1) return launch_tiles<D, 1, 2, 1, 1, true>(args, n_tiles, stream, ev);
    if (qw == 2 && kw == 2 && nb == 2) return launch_tiles<D, 2, 2, 1, 2, true>(args, n_tiles, stream, ev);
    if (kw == 1 && nb == 2) {
        switch (qw) {
            case 3: return launch_tiles<D, 3, 1, 1, 2, true>(args, n_tiles, stream, ev);
            case 4: return launch_tiles<D, 4, 1, 1, 2, true>(args, n_tiles, stream, ev);
            case 5: return launch_tiles<D, 5, 1, 1, 2, true>(args, n_tiles, stream, ev);
            case 6: return launch_tiles<D, 6, 1, 1, 2, true>(args, n_tiles, stream, ev);
            case 7: return launch_tiles<D, 7, 1, 1, 2, true>(args, n_tiles, stream, ev);
            case 8: return launch_tiles<D, 8, 1, 1, 2, true>(args, n_tiles, stream, ev);
            default: break;
        }
    }
    *supported = false;
    return hipSuccess;
}

sangam_status hip_fail(hipError_t e, const char* what) {
    set_error(std::string(what) + ": " + hipGetErrorString(e));
    return SANGAM_ERR_HIP;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

// ---------------------------------------------------------- allocation-free
// Split-KV partial results of sangam_attn_forward_noalloc live in this array
// instead of a caller workspace. Each GPU the library runs on holds its own
// copy for the life of the process. In host code the name is only a stand-in
// for the symbol: kernels receive the device address that hipGetSymbolAddress
// returns for the current device, cached per device below.
namespace {
constexpr size_t kScratchBytes = size_t(32) << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxScratchDevices] = {};

// the scratch array's address on the device that runs `stream`, which must
// be the current device (the symbol is resolved with that device current)
sangam_status scratch_address(hipStream_t stream, void** addr) {
    int cur = -1;
    if (hipError_t e = hipGetDevice(&cur); e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (stream) {
        hipDevice_t sd = -1;
        if (hipError_t e = hipStreamGetDevice(stream, &sd); e != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
        if (int(sd) != cur) {
            set_error("the stream belongs to device " + std::to_string(int(sd)) + ", the current device is " +
                      std::to_string(cur));
            return SANGAM_ERR_INVALID_ARG;
        }
    }
    if (cur < 0 || cur >= kMaxScratchDevices) {
        set_error("device ordinal " + std::to_string(cur) + " beyond the scratch table");
        return SANGAM_ERR_UNSUPPORTED;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[cur]) {
        void* p = nullptr;
        if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)); e != hipSuccess)
            return hip_fail(e, "hipGetSymbolAddress(scratch)");
        g_scratch_dev[cur] = p;
    }
    *addr = g_scratch_dev[cur];
    return SANGAM_OK;
}
}  // namespace

static sangam_status forward_impl(const void* plan_host, const void* plan_dev, const void* q,
                                  const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                                  int64_t pool_pages, const int32_t* page_ids_dev, int64_t num_page_ids,
                                  void* out, float* lse, void* workspace, size_t workspace_bytes,
                                  void* stream_ptr, void* const* events, bool use_scratch = false) {
    clear_error();
    const PlanHeader* h = check_plan(plan_host);
    if (!h) {
        set_error("plan_host is not a plan of this library version");
        return SANGAM_ERR_PLAN;
    }
    if (!plan_dev || !q || !k_new || !v_new || !k_cache || !v_cache || !page_ids_dev || !out) {
        set_error("plan_dev, q, k_new, v_new, k_cache, v_cache, page_ids_dev and out must not be NULL");
        return SANGAM_ERR_INVALID_ARG;
    }
    if (!aligned16(plan_dev) || !aligned16(q) || !aligned16(k_new) || !aligned16(v_new) ||
        !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out) ||
        (reinterpret_cast<uintptr_t>(page_ids_dev) & 3u) || (lse && (reinterpret_cast<uintptr_t>(lse) & 3u))) {
        set_error("tensors must be 16-byte aligned (page_ids and lse 4-byte aligned)");
        return SANGAM_ERR_ALIGN;
    }
    if (pool_pages < h->num_pool_pages) {
        set_error("the plan addresses " + std::to_string(h->num_pool_pages) + " pool pages, the cache holds " +
                  std::to_string(pool_pages));
        return SANGAM_ERR_BUFFER;
    }
    if (num_page_ids < h->total_pages) {
        set_error("the plan reads " + std::to_string(h->total_pages) + " page ids, page_ids_dev holds " +
                  std::to_string(num_page_ids));
        return SANGAM_ERR_BUFFER;
    }
    if (use_scratch && h->workspace_bytes > 0) {
        // the allocation-free entry point: split partials go to the scratch array
        if (size_t(h->workspace_bytes) > kScratchBytes) {
            set_error("the plan's split partials need " + std::to_string(h->workspace_bytes) +
                      " bytes; the allocation-free forward holds " + std::to_string(kScratchBytes));
            return SANGAM_ERR_BUFFER;
        }
        if (sangam_status st = scratch_address(static_cast<hipStream_t>(stream_ptr), &workspace); st != SANGAM_OK)
            return st;
        workspace_bytes = kScratchBytes;
    }
    if (h->workspace_bytes > 0) {
        if (!workspace || workspace_bytes < size_t(h->workspace_bytes)) {
            set_error("workspace needs " + std::to_string(h->workspace_bytes) + " bytes");
            return SANGAM_ERR_BUFFER;
        }
        if (!aligned16(workspace)) {
            set_error("workspace must be 16-byte aligned");
            return SANGAM_ERR_ALIGN;
        }
    }
    hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
    const uint8_t* pd = static_cast<const uint8_t*>(plan_dev);
    // events[2k], events[2k+1] bracket launch k (prefill-shaped, decode-shaped,
    // merge); a launch with no work records its pair back to back
    auto evs = [&](int k) {
        LaunchEvents ev;
        if (events) {
            ev.start = static_cast<hipEvent_t>(events[2 * k]);
            ev.stop = static_cast<hipEvent_t>(events[2 * k + 1]);
        }
        return ev;
    };
    auto mark_empty = [&](int k) -> hipError_t {
        const LaunchEvents ev = evs(k);
        for (hipEvent_t e : {ev.start, ev.stop})
            if (e)
                if (hipError_t r = hipEventRecord(e, stream); r != hipSuccess) return r;
        return hipSuccess;
    };
    const ItemRec* items = reinterpret_cast<const ItemRec*>(pd + h->off_items);

    AttnArgs args{nullptr,
                  items,
                  page_ids_dev,
                  static_cast<const uint16_t*>(q),
                  static_cast<const uint16_t*>(k_new),
                  static_cast<const uint16_t*>(v_new),
                  static_cast<uint16_t*>(k_cache),
                  static_cast<uint16_t*>(v_cache),
                  static_cast<uint16_t*>(out),
                  lse,
                  static_cast<float*>(workspace),
                  reinterpret_cast<const int32_t*>(pd + h->off_positions),
                  reinterpret_cast<const uint32_t*>(pd + h->off_page_info),
                  h->hq,
                  h->hkv,
                  h->scale_log2};

    // 1. attention: prefill-shaped tiles (compute-bound) first, then
    // decode-shaped tiles; both also write the fresh rows into their pages
    if (h->n_prefill_tiles > 0) {
        args.tiles = reinterpret_cast<const TileRec*>(pd + h->off_prefill_tiles);
        hipError_t e;
        if (h->prefill_rows == kWidePrefillRows && h->d == 128)
            e = launch_tiles<128, kWidePrefillQWaves, 1, 1, 4, false>(args, h->n_prefill_tiles, stream, evs(0));
        else if (h->prefill_rows == kPrefillRows)
            e = h->d == 128
                    ? launch_tiles<128, kPrefillQWaves, 1, kPrefillQBlocks, 2, false>(args, h->n_prefill_tiles, stream, evs(0))
                    : launch_tiles<64, kPrefillQWaves, 1, kPrefillQBlocks, 2, false>(args, h->n_prefill_tiles, stream, evs(0));
        else {
            set_error("no prefill kernel for this tile shape");
            return SANGAM_ERR_UNSUPPORTED;
        }
        if (e != hipSuccess) return hip_fail(e, "prefill attention launch");
    } else if (hipError_t e = mark_empty(0); e != hipSuccess) {
        return hip_fail(e, "event record");
    }
    if (h->n_decode_tiles > 0) {
        args.tiles = reinterpret_cast<const TileRec*>(pd + h->off_decode_tiles);
        bool ok = false;
        hipError_t e = h->d == 128 ? launch_decode<128>(args, h->n_decode_tiles, h->decode_qw, h->decode_kw,
                                                        h->decode_nb, stream, evs(1), &ok)
                                   : launch_decode<64>(args, h->n_decode_tiles, h->decode_qw, h->decode_kw,
                                                       h->decode_nb, stream, evs(1), &ok);
        if (!ok) {
            set_error("no decode kernel for this head grouping");
            return SANGAM_ERR_UNSUPPORTED;
        }
        if (e != hipSuccess) return hip_fail(e, "decode attention launch");
    } else if (hipError_t e = mark_empty(1); e != hipSuccess) {
        return hip_fail(e, "event record");
    }

    // 2. merge split contexts
    if (h->n_merge_rows > 0) {
        MergeArgs m{reinterpret_cast<const MergeRow*>(pd + h->off_merge),
                    items,
                    static_cast<const float*>(workspace),
                    static_cast<uint16_t*>(out),
                    lse,
                    h->hq,
                    h->d};
        const unsigned slices = unsigned((h->hq * (h->d / 4) + 255) / 256);
        hipError_t e = launch(reinterpret_cast<const void*>(&merge_kernel), dim3(unsigned(h->n_merge_rows), slices),
                              256u, m, stream, evs(2));
        if (e != hipSuccess) return hip_fail(e, "merge launch");
    } else if (hipError_t e = mark_empty(2); e != hipSuccess) {
        return hip_fail(e, "event record");
    }
    return SANGAM_OK;
}

extern "C" sangam_status sangam_attn_forward(const void* plan_host, const void* plan_dev, const void* q,
                                             const void* k_new, const void* v_new, void* k_cache,
                                             void* v_cache, int64_t pool_pages, const int32_t* page_ids_dev,
                                             int64_t num_page_ids, void* out, float* lse, void* workspace,
                                             size_t workspace_bytes, void* stream) {
    clear_error();
    return forward_impl(plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache, pool_pages, page_ids_dev,
                        num_page_ids, out, lse, workspace, workspace_bytes, stream, nullptr);
}

extern "C" size_t sangam_noalloc_scratch_bytes(void) { return kScratchBytes; }

extern "C" sangam_status sangam_attn_forward_noalloc(const void* plan_host, const void* plan_dev, const void* q,
                                                     const void* k_new, const void* v_new, void* k_cache,
                                                     void* v_cache, int64_t pool_pages,
                                                     const int32_t* page_ids_dev, int64_t num_page_ids,
                                                     void* out, float* lse, void* stream) {
    clear_error();
    return forward_impl(plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache, pool_pages, page_ids_dev,
                        num_page_ids, out, lse, nullptr, 0, stream, nullptr, true);
}

extern "C" sangam_status sangam_attn_forward_timed(const void* plan_host, const void* plan_dev,
                                                   const void* q, const void* k_new, const void* v_new,
                                                   void* k_cache, void* v_cache, int64_t pool_pages,
                                                   const int32_t* page_ids_dev, int64_t num_page_ids,
                                                   void* out, float* lse, void* workspace,
                                                   size_t workspace_bytes, void* stream, void* const* events) {
    clear_error();
    if (!events) {
        set_error("events must not be NULL");
        return SANGAM_ERR_INVALID_ARG;
    }
    return forward_impl(plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache, pool_pages, page_ids_dev,
                        num_page_ids, out, lse, workspace, workspace_bytes, stream, events);
}
