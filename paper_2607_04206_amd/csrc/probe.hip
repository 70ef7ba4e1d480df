// Ceiling probes of MI355X (gfx950): a streaming HBM read and an MFMA-only
// loop, timed by the caller beside the attention kernels so their rates can
// be reported against what the chip delivers as well as against the sheet.
#include <hip/hip_runtime.h>

#include <string>

#include "../../include/sangam_probe.h"

namespace sangam {
void set_error(const std::string& msg);
void clear_error();
}  // namespace sangam

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// grid-stride 16-byte loads, four in flight per thread per round
__global__ __launch_bounds__(256) void hbm_read_kernel(const u32x4* src, size_t n16, uint32_t* sink) {
    const size_t stride = size_t(gridDim.x) * 256;
    size_t i = size_t(blockIdx.x) * 256 + threadIdx.x;
    u32x4 acc = {0, 0, 0, 0};
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
        acc ^= a ^ b ^ c ^ d;
    }
    for (; i < n16; i += stride) acc ^= src[i];
    uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
    __shared__ uint32_t red[256];
    red[threadIdx.x] = x;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (int(threadIdx.x) < s) red[threadIdx.x] ^= red[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) sink[blockIdx.x] = red[0];
}

// 8 independent accumulator chains per wave: the matrix core never waits on
// a previous result, and no memory is touched inside the loop
__global__ __launch_bounds__(256) void mfma_kernel(float* sink, int iters) {
    const int lane = threadIdx.x & 63;
    bf16x8 a, b;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        a[k] = (__bf16)(0.001f * float((lane + k) & 15));
        b[k] = (__bf16)(0.002f * float((lane * 3 + k) & 15));
    }
    f32x16 acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[j][e] = 0.0f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) s += acc[j][e];
    __shared__ float red[256];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int k = 128; k > 0; k >>= 1) {
        if (int(threadIdx.x) < k) red[threadIdx.x] += red[threadIdx.x + k];
        __syncthreads();
    }
    if (threadIdx.x == 0) sink[blockIdx.x] = red[0];
}

sangam_status launched(hipError_t e, const char* what) {
    if (e == hipSuccess) return SANGAM_OK;
    sangam::set_error(std::string(what) + ": " + hipGetErrorString(e));
    return SANGAM_ERR_HIP;
}

}  // namespace

extern "C" sangam_status sangam_probe_hbm_read(const void* src, size_t bytes, uint32_t* sink, int32_t grid,
                                               void* stream) {
    sangam::clear_error();
    if (!src || !sink || (reinterpret_cast<uintptr_t>(src) & 15u) || (reinterpret_cast<uintptr_t>(sink) & 3u)) {
        sangam::set_error("src (16-byte aligned) and sink (4-byte aligned) must not be NULL");
        return SANGAM_ERR_INVALID_ARG;
    }
    if (bytes == 0 || bytes % 16 != 0 || grid < 1) {
        sangam::set_error("bytes must be a positive multiple of 16 and grid >= 1");
        return SANGAM_ERR_INVALID_ARG;
    }
    hipLaunchKernelGGL(hbm_read_kernel, dim3(unsigned(grid)), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<const u32x4*>(src), bytes / 16, sink);
    return launched(hipGetLastError(), "hbm read probe launch");
}

extern "C" sangam_status sangam_probe_mfma_bf16(float* sink, int32_t grid, int32_t iters, void* stream) {
    sangam::clear_error();
    if (!sink || (reinterpret_cast<uintptr_t>(sink) & 3u)) {
        sangam::set_error("sink must be a 4-byte aligned device buffer");
        return SANGAM_ERR_INVALID_ARG;
    }
    if (grid < 1 || iters < 1) {
        sangam::set_error("grid and iters must be >= 1");
        return SANGAM_ERR_INVALID_ARG;
    }
    hipLaunchKernelGGL(mfma_kernel, dim3(unsigned(grid)), dim3(256), 0, static_cast<hipStream_t>(stream), sink,
                       int(iters));
    return launched(hipGetLastError(), "mfma probe launch");
}
