// Device helpers shared by the gfx950 kernels: element types, bf16
// conversion, wave64 reductions and the Philox-4x64-10 counter generator.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;  // storage type: raw bf16 bits
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace sdv {

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// round-to-nearest-even (inputs are finite in this library)
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<bf16_t>(u >> 16);
}

// load / store one element of the tensor type (float or bf16 bits)
template <typename T> __device__ __forceinline__ float ld(const T* p, size_t i);
template <> __device__ __forceinline__ float ld<float>(const float* p, size_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<bf16_t>(const bf16_t* p, size_t i) {
    return bf16_to_f32(p[i]);
}
template <typename T> __device__ __forceinline__ void st(T* p, size_t i, float v);
template <> __device__ __forceinline__ void st<float>(float* p, size_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st<bf16_t>(bf16_t* p, size_t i, float v) {
    p[i] = f32_to_bf16(v);
}

// Store of an activation that feeds a matrix product.  fp32 model: one
// plane.  bf16 model: two bf16 planes, hi = bf16(v) at p[i] and
// lo = bf16(v - hi) at p[plane + i]; the products consume both, so the
// activation keeps about 16 significant bits instead of 8.
template <typename T> __device__ __forceinline__ void st_act(T* p, size_t plane, size_t i, float v);
template <> __device__ __forceinline__ void st_act<float>(float* p, size_t, size_t i, float v) {
    p[i] = v;
}
template <> __device__ __forceinline__ void st_act<bf16_t>(bf16_t* p, size_t plane, size_t i, float v) {
    const bf16_t hi = f32_to_bf16(v);
    p[i] = hi;
    p[plane + i] = f32_to_bf16(v - bf16_to_f32(hi));
}

// four values as bf16 (8 bytes); the activation planes hi = bf16(v),
// lo = bf16(v - hi) of four consecutive columns
__device__ __forceinline__ uint2 pack_bf16x4(const float (&v)[4]) {
    return uint2{(uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16),
                 (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16)};
}
__device__ __forceinline__ void st_act4(bf16_t* p, size_t plane, size_t i, const float (&v)[4]) {
    float lo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) lo[e] = v[e] - bf16_to_f32(f32_to_bf16(v[e]));
    *(uint2*)(p + i) = pack_bf16x4(v);
    *(uint2*)(p + plane + i) = pack_bf16x4(lo);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

// Softmax statistics of a set of logits z: m = max z, s = sum exp(z - m),
// and the argmax (value v, index i, the lowest index on ties).  Merging two
// sets is exact in m, v and i and commutative bit for bit in s (the larger
// maximum's sum plus the other one rescaled), so a butterfly leaves every
// lane with the same result; only the grouping of the merges moves the
// rounding of s.
struct __attribute__((aligned(16))) VStat {
    float m, s, v;
    int i;
};
__device__ __forceinline__ VStat vstat_empty() { return VStat{-INFINITY, 0.f, -INFINITY, 0x7fffffff}; }
__device__ __forceinline__ void merge_ms(float& m, float& s, float m2, float s2) {
    if (m2 == -INFINITY) return;
    if (m == -INFINITY) { m = m2; s = s2; return; }
    if (m2 > m) { s = s * expf(m - m2) + s2; m = m2; }
    else s += s2 * expf(m2 - m);
}
__device__ __forceinline__ VStat vstat_merge(VStat a, const VStat& b) {
    merge_ms(a.m, a.s, b.m, b.s);
    if (b.v > a.v || (b.v == a.v && b.i < a.i)) { a.v = b.v; a.i = b.i; }
    return a;
}
__device__ __forceinline__ VStat vstat_shfl_xor(const VStat& a, int o) {
    return VStat{__shfl_xor(a.m, o, 64), __shfl_xor(a.s, o, 64), __shfl_xor(a.v, o, 64),
                 __shfl_xor(a.i, o, 64)};
}

// Block-wide sum for blockDim.x == 256 (4 waves); `red` holds 4 floats.
__device__ __forceinline__ float block_sum_256(float v, float* red) {
    v = wave_sum(v);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    float s = red[0] + red[1] + red[2] + red[3];
    __syncthreads();
    return s;
}

// s_waitcnt immediate for "vector memory counter <= N" (LGK counter <= 0
// when LGK0, else free)
template <int N, bool LGK0 = false>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | ((LGK0 ? 0 : 15) << 8));
}

// Workgroup barrier without the memory fence of __syncthreads(): the fence
// would wait for every outstanding load, including direct-to-LDS loads of
// later pipeline stages that are meant to stay in flight.  Callers wait for what
// must be complete themselves; the empty asm statements keep the compiler
// from moving memory accesses across the barrier.
__device__ __forceinline__ void barrier_nofence() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// ---------------------------------------------------------------------------
// Philox-4x64-10 (Salmon et al., SC'11).  Ten rounds of: multiply words 0 and
// 2 by the round multipliers, swap halves, xor in the round key; the key
// advances by the two Weyl constants between rounds.
// ---------------------------------------------------------------------------
struct u64x4 { uint64_t x, y, z, w; };

__device__ __forceinline__ u64x4 philox4x64_10(u64x4 c, uint64_t k0, uint64_t k1) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t lo0 = M0 * c.x, hi0 = __umul64hi(M0, c.x);
        const uint64_t lo1 = M1 * c.z, hi1 = __umul64hi(M1, c.z);
        u64x4 n;
        n.x = hi1 ^ c.y ^ k0;
        n.y = lo1;
        n.z = hi0 ^ c.w ^ k1;
        n.w = lo0;
        c = n;
        k0 += 0x9E3779B97F4A7C15ull;
        k1 += 0xBB67AE8584CAA73Bull;
    }
    return c;
}

// Sampler draw layout: counter (round, user, purpose << 32 | slot, k / 4),
// key (seed, 0); word k % 4.
enum { PURPOSE_ACCEPT = 1, PURPOSE_RACE = 2 };

__device__ __forceinline__ uint64_t word_of(const u64x4& v, int i) {
    return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
}

// u in [0, 1) on a 2^-24 grid
__device__ __forceinline__ float accept_uniform(uint64_t x) {
    return static_cast<float>(static_cast<uint32_t>(x >> 40)) * 0x1.0p-24f;
}

// V in [2^-64, 1): the 24 bits below the leading one, scaled by its position
__device__ __forceinline__ float race_uniform(uint64_t x) {
    if (x == 0) return 0.0f;
    const int lz = __clzll(static_cast<long long>(x));
    const uint32_t mant = static_cast<uint32_t>((x << lz) >> 40);
    return ldexpf(static_cast<float>(mant), -24 - lz);
}

// unit exponential -log(1 - V)
__device__ __forceinline__ float race_exponential(uint64_t x) {
    return -log1pf(-race_uniform(x));
}

}  // namespace sdv
