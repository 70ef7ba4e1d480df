/*
 * sangam_attn.h - C ABI of the mixed block-decode / prefill attention call of
 * cached diffusion-LLM serving, for AMD Instinct MI355X (gfx950).
 *
 * The operation (Sangam paper: Sec. 2.1 bidirectional attention, Sec. 2.2
 * blockwise approximate KV cache, Sec. 4.1 / Alg. 1 mixed microbatches of
 * in-flight decodes plus whole prefills, Sec. 5 paged KV cache, Sec. 6.1
 * page size 16, block size 32, bf16):
 *
 *   One call serves a ragged batch of work items. Item i has n_i query rows
 *   at sequence positions o_i .. o_i+n_i-1 (the block-offset table) and a
 *   context of L_i positions. A block decode has n_i = 32 rows (one response
 *   block) and reuses the request's cached KV; a prefill has o_i = 0,
 *   n_i = L_i and brings its whole sequence. A per-token cached decode
 *   (Sec. 2.2, the dKV-Cache-PD variant: prompt KV fixed, response tokens
 *   refreshed individually) recomputes up to 32 rows at arbitrary positions,
 *   given by the optional position list q_pos instead of o_i. For each item
 *   the call
 *     1. writes the fresh rows k_new / v_new into the paged cache at the rows'
 *        positions ([o_i, o_i+n_i), or the listed ones), and
 *     2. lets every query row attend, without a causal mask, to all positions
 *        [0, L_i) of the item's post-write sequence:
 *          out[r,h,:] = softmax_j(sm_scale * q[r,h,:] . K[j,g,:]) V[j,g,:]
 *          lse[r,h]   = ln sum_j exp(sm_scale * q[r,h,:] . K[j,g,:])
 *        with g = h / (Hq / Hkv) (contiguous GQA groups).
 *   Attention reads the item's own fresh rows from k_new / v_new, never from
 *   the cache, so the write and the reads of one launch never race.
 *
 * Layouts (row-major, contiguous, 16-byte aligned; bf16 = IEEE bfloat16 bits):
 *   q, out          [sum n_i, Hq, D]  bf16   (item i's rows start at q_indptr[i])
 *   k_new, v_new    [sum n_i, Hkv, D] bf16   (row t of item i = position o_i + t, or the
 *                                             t-th listed position)
 *   k_cache,v_cache [num_pool_pages, Hkv, page_size, D] bf16
 *                   position p of item i lives in page
 *                   page_ids[page_indptr[i] + p / page_size], slot p % page_size
 *   lse             [sum n_i, Hq] fp32 (natural log), may be NULL
 * Slots >= L_i of an item's last page are never read and never written.
 *
 * Ownership: the caller owns every host and device buffer, including the plan
 * buffer, its device copy and the workspace. The library allocates nothing,
 * holds no device state and keeps no pointer after a call returns.
 *
 * Errors: every entry point returns a sangam_status (0 = success, negative =
 * failure) and never throws or aborts; sangam_last_error() gives a message
 * for the calling thread's last failure.
 */
#ifndef SANGAM_ATTN_H
#define SANGAM_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t sangam_status;

#define SANGAM_OK 0
#define SANGAM_ERR_INVALID_ARG (-1) /* malformed descriptor or argument */
#define SANGAM_ERR_UNSUPPORTED (-2) /* head_dim not 64/128, page_size not 16, Hq % Hkv != 0 */
#define SANGAM_ERR_PAGE_RANGE (-3)  /* a page id outside [0, num_pool_pages) */
#define SANGAM_ERR_PAGE_ALIAS (-4)  /* a page listed twice in one batch */
#define SANGAM_ERR_BUFFER (-5)      /* plan buffer or workspace too small */
#define SANGAM_ERR_ALIGN (-6)       /* a tensor pointer not 16-byte aligned */
#define SANGAM_ERR_HIP (-7)         /* a HIP runtime error during launch */
#define SANGAM_ERR_PLAN (-8)        /* not a plan of this library version */

/* Batch descriptor. All arrays are host memory, read only during the call. */
typedef struct sangam_attn_desc {
    int32_t num_items;       /* number of work items, >= 1 */
    int32_t num_q_heads;     /* Hq >= 1 */
    int32_t num_kv_heads;    /* Hkv >= 1, Hq % Hkv == 0 */
    int32_t head_dim;        /* D: 64 or 128 */
    int32_t page_size;       /* tokens per KV page: 16 */
    int32_t force_kv_splits; /* 0: the plan chooses; k >= 1: cut every item's context into
                                chunks of one 64-aligned length, round_up(ceil(L_i / k'), 64)
                                with k' = min(k, ceil(L_i / 64)): at most k' chunks, at
                                least two when k' >= 2 (more only where a tile's range
                                limit of 8192 cached keys requires) (tests, tuning) */
    int64_t num_pool_pages;  /* pages in k_cache / v_cache */
    float sm_scale;          /* softmax scale, e.g. 1/sqrt(D) */
    int32_t num_cus;         /* compute units to balance over; 0 means 256 */
    const int32_t *q_indptr;    /* [num_items + 1], q_indptr[0] = 0, n_i = q_indptr[i+1]-q_indptr[i] >= 1 */
    const int32_t *q_offset;    /* [num_items] block-offset table o_i >= 0, o_i + n_i <= L_i */
    const int32_t *kv_len;      /* [num_items] 1 <= L_i <= 2^30 */
    const int32_t *page_indptr; /* [num_items + 1], page_indptr[i+1]-page_indptr[i] = ceil(L_i/page_size) */
    const int32_t *page_ids;    /* [page_indptr[num_items]], in range, no page twice */
    const int32_t *q_pos;       /* NULL, or [q_indptr[num_items]]: the sequence position of each
                                   query row (row r of item i at q_pos[q_indptr[i] + r]); then
                                   q_offset is ignored. Per item strictly increasing in [0, L_i).
                                   An item whose positions are not one contiguous range (a
                                   per-token cached decode) has n_i <= 32 and a cached context */
} sangam_attn_desc;

/*
 * Validate a batch and write its launch plan into plan_buf (host memory).
 * Host only: makes no HIP call. The plan is position independent; the caller
 * copies the same bytes to device memory (plan_dev below) before the forward.
 * If cap is too small, returns SANGAM_ERR_BUFFER with *used = bytes needed
 * (plan_buf may be NULL to query the size). On success *used = bytes written.
 * Errors: SANGAM_ERR_INVALID_ARG, _UNSUPPORTED, _PAGE_RANGE, _PAGE_ALIAS, _BUFFER.
 */
sangam_status sangam_attn_plan(const sangam_attn_desc *desc, void *plan_buf, size_t cap,
                               size_t *used);

/* Device workspace bytes the forward needs for split-KV partial results
 * (fp32 O and LSE); 0 when no item is split. Returns 0 for an invalid plan. */
size_t sangam_plan_workspace_bytes(const void *plan_buf);

/* Summary of a plan, for tests and tuning. */
typedef struct sangam_plan_info {
    int32_t num_items;
    int32_t num_decode_tiles;  /* work-groups of the decode-shaped launch (n_i <= 32) */
    int32_t num_prefill_tiles; /* work-groups of the prefill-shaped launch (n_i > 32, and
                                  the fused block decodes below) */
    int32_t num_split_items;   /* items whose context is split (merged afterwards) */
    int32_t max_splits;        /* largest split count of an item */
    int32_t decode_q_waves;    /* waves per decode work-group that hold query rows */
    int32_t decode_kv_waves;   /* waves per decode work-group that split the context */
    int32_t num_fused_decode_tiles; /* prefill-shaped work-groups that hold block decodes:
                                       in a batch with prefills, or a decode-only batch too
                                       small to fill the CUs, a GQA group of >= 4 query
                                       heads per KV head puts its block decodes there (one
                                       query head per wave); with prefills unsplit up to
                                       8192 keys */
    int64_t total_q_rows;      /* sum n_i */
    int64_t workspace_bytes;
    int64_t plan_bytes;
} sangam_plan_info;

sangam_status sangam_plan_get_info(const void *plan_buf, sangam_plan_info *info);

/* Split count and first context position of each split of item `item`.
 * starts must hold max_splits + 1 entries (the last one is L_i). */
sangam_status sangam_plan_item_splits(const void *plan_buf, int32_t item, int32_t *num_splits,
                                      int32_t *starts, int32_t cap);

/*
 * Run the call on `stream` (a hipStream_t; NULL is the default stream).
 * Asynchronous: it only enqueues kernels. It allocates nothing, never
 * synchronizes and copies nothing between host and device, so it may be
 * captured into a HIP graph. plan_host is the plan in host memory (launch
 * sizes are read from it); plan_dev is the same bytes in device memory.
 * k_cache / v_cache each hold pool_pages pages of [Hkv, 16, D] bf16; the
 * kernels address pages below the plan's num_pool_pages, so pool_pages must
 * be at least that. page_ids_dev holds desc->page_ids in device memory,
 * num_page_ids entries of it (at least page_indptr[num_items]). lse may be
 * NULL. workspace must hold sangam_plan_workspace_bytes(plan_host) bytes
 * (NULL when that is 0); workspace_bytes is its size.
 * Errors: SANGAM_ERR_PLAN, _INVALID_ARG (a NULL tensor), _ALIGN, _BUFFER
 * (workspace, pool or page table smaller than the plan addresses), _HIP
 * (launch failed; nothing is rolled back).
 */
sangam_status sangam_attn_forward(const void *plan_host, const void *plan_dev, const void *q,
                                  const void *k_new, const void *v_new, void *k_cache,
                                  void *v_cache, int64_t pool_pages, const int32_t *page_ids_dev,
                                  int64_t num_page_ids, void *out, float *lse, void *workspace,
                                  size_t workspace_bytes, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * call as sangam_attn_forward, with the split-KV partial results in a
 * library-owned device array instead of a caller workspace. It calls no
 * allocator. The array holds sangam_noalloc_scratch_bytes() bytes (32 MiB)
 * per GPU; each GPU the library runs on keeps its own copy until the process
 * ends. Its address is looked up once per device, on the first call with
 * that device current. `stream` must belong to the current device.
 * Every call on one GPU shares that GPU's array: two calls that overlap in
 * time on one GPU (different streams, or threads) race on it; serialize
 * them. The array keeps the last call's contents; nothing in it needs to
 * start at zero (each split's partials are written before they are read).
 * Errors: as sangam_attn_forward; SANGAM_ERR_BUFFER when the plan's
 * workspace (sangam_plan_workspace_bytes) exceeds the array;
 * SANGAM_ERR_INVALID_ARG when `stream` belongs to another device.
 */
sangam_status sangam_attn_forward_noalloc(const void *plan_host, const void *plan_dev, const void *q,
                                          const void *k_new, const void *v_new, void *k_cache,
                                          void *v_cache, int64_t pool_pages,
                                          const int32_t *page_ids_dev, int64_t num_page_ids,
                                          void *out, float *lse, void *stream);

/* Bytes of the device array that sangam_attn_forward_noalloc uses for split
 * partials (its largest plan workspace). */
size_t sangam_noalloc_scratch_bytes(void);

/*
 * sangam_attn_forward, plus HIP events carried by its launches, for measuring
 * each kernel in place: events[0] and [1] are the start and stop of the
 * prefill-shaped attention launch, [2] and [3] of the decode-shaped launch,
 * [4] and [5] of the split merge (the KV write-back runs inside the two
 * attention launches). The events travel in the kernel dispatch itself, so
 * their elapsed time is the kernel's execution time, as a kernel trace
 * reports it. A launch with no work records its two events back to back.
 * events holds six entries, each a hipEvent_t the caller created (and owns)
 * or NULL for no timestamp; otherwise identical to sangam_attn_forward.
 * Errors: as sangam_attn_forward, plus SANGAM_ERR_INVALID_ARG for a NULL
 * events array.
 */
sangam_status sangam_attn_forward_timed(const void *plan_host, const void *plan_dev,
                                        const void *q, const void *k_new, const void *v_new,
                                        void *k_cache, void *v_cache, int64_t pool_pages,
                                        const int32_t *page_ids_dev, int64_t num_page_ids,
                                        void *out, float *lse, void *workspace,
                                        size_t workspace_bytes, void *stream,
                                        void *const *events);

/* Message of the calling thread's last failure ("" if none). The pointer
 * stays valid until the thread's next call into the library. */
const char *sangam_last_error(void);

/* Library version, e.g. 0x000100 for 0.1.0. */
int32_t sangam_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SANGAM_ATTN_H */
