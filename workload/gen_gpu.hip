// GPU copy of the seeded generator in gen.c: same counter-based bits, same
// Irwin-Hall construction, same fp32 rounding, so every value is
// bit-identical to the host generator (checked by a GPU test).  Holds no
// arithmetic of the verify method.
#include <hip/hip_runtime.h>
#include <stdint.h>

#define GOLDEN 0x9e3779b97f4a7c15ULL

__host__ __device__ static inline uint64_t fin64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

__host__ __device__ static inline uint64_t wl_key(uint64_t seed, uint64_t stream) {
    return fin64(fin64(seed + GOLDEN) ^ (stream * 0xd1b54a32d192ed03ULL + 0x2545f4914f6cdd1dULL));
}

__device__ static inline uint64_t wl_bits(uint64_t key, uint64_t i) { return fin64(key + (i + 1) * GOLDEN); }

__device__ static inline float ih4(uint64_t b, float scale) {
    int32_t s = (int32_t)(b & 0xffff) + (int32_t)((b >> 16) & 0xffff) +
                (int32_t)((b >> 32) & 0xffff) + (int32_t)((b >> 48) & 0xffff) - 131070;
    return __fmul_rn((float)s, scale);
}

__device__ static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffff) ? 0x40 : 0));
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__global__ void k_normal(void* out, int64_t n, uint64_t key, int64_t offset, float scale, int bf16) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const float v = ih4(wl_bits(key, (uint64_t)(offset + i)), scale);
        if (bf16) ((uint16_t*)out)[i] = f32_to_bf16_rne(v);
        else ((float*)out)[i] = v;
    }
}

__global__ void k_uniform(void* out, int64_t n, uint64_t key, int64_t offset, float lo, float hi,
                          int bf16) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const float u = __fmul_rn((float)(wl_bits(key, (uint64_t)(offset + i)) >> 40), 0x1.0p-24f);
        const float v = __fadd_rn(lo, __fmul_rn(__fsub_rn(hi, lo), u));
        if (bf16) ((uint16_t*)out)[i] = f32_to_bf16_rne(v);
        else ((float*)out)[i] = v;
    }
}

#define IH4_STD 37837.2270017029f

extern "C" int wlg_fill_normal(void* out, int64_t n, uint64_t seed, uint64_t stream, int64_t offset,
                               float std, int bf16, void* hip_stream) {
    if (n <= 0) return 0;
    const float scale = std / IH4_STD;
    const int64_t blocks = (n + 255) / 256 < 65536 ? (n + 255) / 256 : 65536;
    hipLaunchKernelGGL(k_normal, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)hip_stream, out,
                       n, wl_key(seed, stream), offset, scale, bf16);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

extern "C" int wlg_fill_uniform(void* out, int64_t n, uint64_t seed, uint64_t stream,
                                int64_t offset, float lo, float hi, int bf16, void* hip_stream) {
    if (n <= 0) return 0;
    const int64_t blocks = (n + 255) / 256 < 65536 ? (n + 255) / 256 : 65536;
    hipLaunchKernelGGL(k_uniform, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)hip_stream, out,
                       n, wl_key(seed, stream), offset, lo, hi, bf16);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}
