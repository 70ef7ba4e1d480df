// Paged-KV export / import kernels for gfx950 and their C ABI entry points.
//
// One work-group per (listed page, tensor): grid.x walks the plan's page
// records, grid.y picks K (0) or V (1). A page's chunk of one KV head is 16
// slots x D contiguous in the pool; in the packed buffers slot s of that head
// is row row0 + s, Hkv x D elements apart. Thread t of a 256-thread group
// owns 16-byte piece t % (D / 8) of slot (t / (D / 8)) % 16 of head
// t / (16 D / 8) of each group of 256 / (16 D / 8) heads, so the pool side
// reads or writes whole 4 KiB (2 KiB at D = 64) head chunks and the packed
// side whole 256-byte (128-byte) rows. Four head groups are in flight per
// thread before the first store. Both directions move bytes only.
#include <hip/hip_runtime.h>

#include <string>

#include "../../include/sangam_kv.h"
#include "kv_format.h"

namespace sangam {
void set_error(const std::string& msg);
void clear_error();
const KvPlanHeader* check_kv_plan(const void* plan);
}  // namespace sangam

using namespace sangam;

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct KvCopyArgs {
    const KvPageRec* recs;
    const uint16_t* src[2];  // K, V (pool for export, packed for import)
    uint16_t* dst[2];
    int32_t hkv;
};

template <int D, bool EXPORT>
__global__ __launch_bounds__(256) void kv_copy_kernel(KvCopyArgs a) {
    constexpr int NC = D / 8;           // 16-byte pieces of a row
    constexpr int HPG = 256 / (16 * NC);  // heads per thread group round
    constexpr int U = 4;                // rounds in flight
    const KvPageRec r = a.recs[blockIdx.x];
    const int t = blockIdx.y;
    const uint16_t* __restrict__ src = a.src[t];
    uint16_t* __restrict__ dst = a.dst[t];
    const int tid = threadIdx.x;
    const int pos = tid % NC;
    const int s = (tid / NC) % 16;
    const int hsub = tid / (16 * NC);
    if (s >= r.nslots) return;  // no position in this slot (last page of an item)
    const int hkv = a.hkv;
    const size_t pool0 = ((size_t)r.page * hkv * 16 + s) * D + pos * 8;      // head 0 of the page
    const size_t pack0 = ((size_t)(r.row0 + s) * hkv) * D + pos * 8;         // head 0 of the row
    for (int h0 = hsub; h0 < hkv; h0 += HPG * U) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int h = h0 + u * HPG;
            if (h < hkv) {
                const size_t off = EXPORT ? pool0 + (size_t)h * 16 * D : pack0 + (size_t)h * D;
                v[u] = *(const u32x4*)(src + off);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int h = h0 + u * HPG;
            if (h < hkv) {
                const size_t off = EXPORT ? pack0 + (size_t)h * D : pool0 + (size_t)h * 16 * D;
                *(u32x4*)(dst + off) = v[u];
            }
        }
    }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

sangam_status run_copy(bool is_export, const void* plan_host, const void* plan_dev, const void* src_k,
                       const void* src_v, void* dst_k, void* dst_v, void* stream) {
    clear_error();
    const KvPlanHeader* h = check_kv_plan(plan_host);
    if (!h) {
        set_error("plan_host is not a KV transfer plan of this library version");
        return SANGAM_ERR_PLAN;
    }
    if (!plan_dev || !src_k || !src_v || !dst_k || !dst_v) {
        set_error("plan_dev and the K / V source and destination pointers must not be NULL");
        return SANGAM_ERR_INVALID_ARG;
    }
    if (!aligned16(plan_dev) || !aligned16(src_k) || !aligned16(src_v) || !aligned16(dst_k) || !aligned16(dst_v)) {
        set_error("plan_dev and the K / V buffers must be 16-byte aligned");
        return SANGAM_ERR_ALIGN;
    }
    KvCopyArgs args;
    args.recs = reinterpret_cast<const KvPageRec*>(static_cast<const uint8_t*>(plan_dev) + h->off_pages);
    args.src[0] = static_cast<const uint16_t*>(src_k);
    args.src[1] = static_cast<const uint16_t*>(src_v);
    args.dst[0] = static_cast<uint16_t*>(dst_k);
    args.dst[1] = static_cast<uint16_t*>(dst_v);
    args.hkv = h->hkv;
    const void* fn;
    if (h->d == 128)
        fn = is_export ? reinterpret_cast<const void*>(&kv_copy_kernel<128, true>)
                       : reinterpret_cast<const void*>(&kv_copy_kernel<128, false>);
    else
        fn = is_export ? reinterpret_cast<const void*>(&kv_copy_kernel<64, true>)
                       : reinterpret_cast<const void*>(&kv_copy_kernel<64, false>);
    void* kargs[] = {&args};
    const hipError_t e = hipLaunchKernel(fn, dim3(unsigned(h->total_pages), 2), dim3(256), kargs, 0,
                                         static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        set_error(std::string(is_export ? "kv export" : "kv import") + " launch: " + hipGetErrorString(e));
        return SANGAM_ERR_HIP;
    }
    return SANGAM_OK;
}

}  // namespace

extern "C" sangam_status sangam_kv_export(const void* plan_host, const void* plan_dev, const void* k_cache,
                                          const void* v_cache, void* k_packed, void* v_packed, void* stream) {
    return run_copy(true, plan_host, plan_dev, k_cache, v_cache, k_packed, v_packed, stream);
}

extern "C" sangam_status sangam_kv_import(const void* plan_host, const void* plan_dev, const void* k_packed,
                                          const void* v_packed, void* k_cache, void* v_cache, void* stream) {
    return run_copy(false, plan_host, plan_dev, k_packed, v_packed, k_cache, v_cache, stream);
}
