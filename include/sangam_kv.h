/*
 * sangam_kv.h - C ABI of the paged-KV export / import that hands a request's
 * KV cache from one worker to another in the hybrid configuration of the
 * Sangam paper (Sec. 4.2 and Alg. 2, Sec. 4.3 with its hybrid architecture
 * figure: dedicated prefill workers pass the KV they produce to decode-role
 * workers; Sec. 5: the KV cache is paged and the transfer streams over
 * torch.distributed; Sec. 6.3 measures its cost), for AMD Instinct MI355X
 * (gfx950).
 *
 * The point-to-point send / receive between two GPUs is the caller's (one
 * contiguous buffer per tensor, e.g. over RCCL). These calls do the two GPU
 * steps around it:
 *   export  packs positions [0, L_i) of a batch of requests out of one paged
 *           pool into contiguous buffers;
 *   import  unpacks such buffers into the pages of another pool, whose page
 *           table for the same requests may differ entirely.
 *
 * Layouts (row-major, contiguous, 16-byte aligned; bf16 = IEEE bfloat16 bits):
 *   k_cache, v_cache  [num_pool_pages, Hkv, page_size, D] bf16
 *                     position p of request i lives in page
 *                     page_ids[page_indptr[i] + p / page_size], slot p % page_size
 *                     (the layout of the attention call's cache)
 *   k_packed,v_packed [sum L_i, Hkv, D] bf16
 *                     position p of request i is row kv_indptr[i] + p, with
 *                     kv_indptr the exclusive prefix sum of kv_len (the layout
 *                     of the attention call's k_new / v_new for whole prefills)
 * Export reads only slots < L_i of a request's last page; import writes only
 * those, so the other slots of that page and every page not listed keep
 * their content.
 *
 * Ownership: the caller owns every buffer (plan blob, its device copy, pools,
 * packed buffers). The library allocates nothing and keeps no pointer after a
 * call returns. Errors: a sangam_status from sangam_attn.h; sangam_last_error()
 * gives the message. No call throws or aborts.
 */
#ifndef SANGAM_KV_H
#define SANGAM_KV_H

#include "sangam_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Batch of requests to move. Arrays are host memory, read during the call only. */
typedef struct sangam_kv_desc {
    int32_t num_items;          /* requests, >= 1 */
    int32_t num_kv_heads;       /* Hkv >= 1 */
    int32_t head_dim;           /* D: 64 or 128 */
    int32_t page_size;          /* 16 */
    int64_t num_pool_pages;     /* pages of the pool the plan addresses */
    const int32_t *kv_len;      /* [num_items] L_i >= 1 */
    const int32_t *page_indptr; /* [num_items + 1], page_indptr[0] == 0,
                                   page_indptr[i+1] - page_indptr[i] == ceil(L_i / 16) */
    const int32_t *page_ids;    /* [page_indptr[num_items]] in [0, num_pool_pages), no page twice */
} sangam_kv_desc;

/*
 * Host only (no HIP call). Validates the descriptor and writes a position
 * independent plan (one record per listed page) into plan_buf. Errors:
 * SANGAM_ERR_INVALID_ARG (NULL arrays, num_items < 1, L_i < 1, page counts
 * that do not match L_i, indptr not starting at 0), SANGAM_ERR_UNSUPPORTED
 * (head_dim, page_size), SANGAM_ERR_PAGE_RANGE, SANGAM_ERR_PAGE_ALIAS (an
 * import would write the page twice), SANGAM_ERR_BUFFER (cap too small:
 * *used holds the size needed; plan_buf may be NULL with cap 0 to ask).
 */
sangam_status sangam_kv_plan(const sangam_kv_desc *d, void *plan_buf, size_t cap, size_t *used);

/* Rows of the packed buffers (sum of L_i) of a plan; 0 if plan_buf is not a plan. */
int64_t sangam_kv_plan_rows(const void *plan_buf);

/*
 * Asynchronous on stream (a hipStream_t; NULL is the null stream): one kernel
 * launch, no allocation, no host synchronisation. plan_host is the blob of
 * sangam_kv_plan, plan_dev the same bytes already copied to device memory.
 * export: k_packed[kv_indptr[i] + p] = k_cache[page(i, p), :, slot(p), :] for
 * p < L_i, and the same for V. Errors: SANGAM_ERR_PLAN, SANGAM_ERR_INVALID_ARG
 * (NULL pointers), SANGAM_ERR_ALIGN, SANGAM_ERR_HIP.
 */
sangam_status sangam_kv_export(const void *plan_host, const void *plan_dev, const void *k_cache,
                               const void *v_cache, void *k_packed, void *v_packed, void *stream);

/* The inverse copy: k_cache[page(i, p), :, slot(p), :] = k_packed[kv_indptr[i] + p]
 * for p < L_i, and the same for V. Same contract as sangam_kv_export. */
sangam_status sangam_kv_import(const void *plan_host, const void *plan_dev, const void *k_packed,
                               const void *v_packed, void *k_cache, void *v_cache, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SANGAM_KV_H */
