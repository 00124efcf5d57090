// Small per-token kernels of the verify forward: batch preparation (slot
// tokens, RoPE angles), embedding gather, RMSNorm, fused QK-norm + RoPE +
// KV-page append, and KV copies between caller buffers and the pages.
#include "sdv_device.h"
#include "sdv_internal.h"

namespace sdv {

// ---------------------------------------------------------------------------
// prepare: slot tokens (root at slot 0, drafts after it; Sec. II-A step 2) with
// range checks, and cos/sin of the RoPE angle pos * base^(-2a/hd) per slot,
// computed in double so that large positions keep full fp32 accuracy.
// ---------------------------------------------------------------------------
__global__ void k_prepare(BatchView bv, int32_t* tok, float* cs, int half, int V,
                          double log_base, int hd) {
    const int t = blockIdx.x;
    if (t >= bv.T) return;
    const int b = bv.slot_b[t], j = bv.slot_j[t];
    if (threadIdx.x == 0) {
        int v = (j == 0) ? bv.root[b] : bv.drafts[bv.draft_off[b] + j - 1];
        if (v < 0 || v >= V) {
            atomicOr(bv.flags, 1);
            v = 0;
        }
        tok[t] = v;
    }
    const double pos = (double)(bv.prefix[b] + j);
    for (int a = threadIdx.x; a < half; a += blockDim.x) {
        const double ang = pos * exp(-2.0 * a / hd * log_base);
        double sn, cn;
        sincos(ang, &sn, &cn);
        cs[((size_t)t * half + a) * 2 + 0] = (float)cn;
        cs[((size_t)t * half + a) * 2 + 1] = (float)sn;
    }
}

void launch_prepare(const Dims& D, const BatchView& bv, const SlotBufs& sb, hipStream_t s) {
    hipLaunchKernelGGL(k_prepare, dim3(bv.T), dim3(64), 0, s, bv, sb.tok, sb.cs, D.hd / 2, D.V,
                       log((double)D.rope_base), D.hd);
}

// ---------------------------------------------------------------------------
// embedding gather into the fp32 residual stream
// ---------------------------------------------------------------------------
template <typename TW>
__global__ void k_embed(const int32_t* tok, const TW* E, float* x, int d) {
    const int t = blockIdx.x;
    const size_t row = (size_t)tok[t] * d;
    for (int i = threadIdx.x; i < d; i += blockDim.x) x[(size_t)t * d + i] = ld(E, row + i);
}

void launch_embed(const Dims& D, const BatchView& bv, const void* embed, const SlotBufs& sb,
                  hipStream_t s) {
    if (D.bf16)
        hipLaunchKernelGGL(k_embed<bf16_t>, dim3(bv.T), dim3(256), 0, s, sb.tok,
                           (const bf16_t*)embed, sb.x, D.d);
    else
        hipLaunchKernelGGL(k_embed<float>, dim3(bv.T), dim3(256), 0, s, sb.tok,
                           (const float*)embed, sb.x, D.d);
}

// ---------------------------------------------------------------------------
// RMSNorm of one fp32 row, output in the GEMM input type.  The row is read
// once into registers (float4 loads, all issued before the reduction).
// ---------------------------------------------------------------------------
template <typename TA, int PER>  // PER: float4 loads per thread
__global__ __launch_bounds__(256) void k_rmsnorm(const float* x, const TA* gamma, TA* out, int d,
                                                 float eps) {
    __shared__ float red[4];
    const int t = blockIdx.x;
    const float4* xr = (const float4*)(x + (size_t)t * d);
    const int n4 = d >> 2;
    float4 v[PER];
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int k = threadIdx.x + i * 256;
        v[i] = k < n4 ? xr[k] : float4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    ss = block_sum_256(ss, red);
    const float r = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int k = threadIdx.x + i * 256;
        if (k < n4) {
            const size_t o = (size_t)t * d + 4 * k;
            st(out, o + 0, v[i].x * r * ld(gamma, 4 * k + 0));
            st(out, o + 1, v[i].y * r * ld(gamma, 4 * k + 1));
            st(out, o + 2, v[i].z * r * ld(gamma, 4 * k + 2));
            st(out, o + 3, v[i].w * r * ld(gamma, 4 * k + 3));
        }
    }
}

template <typename TA>
static void rmsnorm_dispatch(int T, const float* x, const TA* gamma, TA* out, int d, float eps,
                             hipStream_t s) {
    const int per = (d / 4 + 255) / 256;
    if (per <= 1) hipLaunchKernelGGL((k_rmsnorm<TA, 1>), dim3(T), dim3(256), 0, s, x, gamma, out, d, eps);
    else if (per <= 2) hipLaunchKernelGGL((k_rmsnorm<TA, 2>), dim3(T), dim3(256), 0, s, x, gamma, out, d, eps);
    else if (per <= 5) hipLaunchKernelGGL((k_rmsnorm<TA, 5>), dim3(T), dim3(256), 0, s, x, gamma, out, d, eps);
    else hipLaunchKernelGGL((k_rmsnorm<TA, 8>), dim3(T), dim3(256), 0, s, x, gamma, out, d, eps);
}

void launch_rmsnorm(const Dims& D, int T, const float* x, const void* gamma, void* out,
                    hipStream_t s) {
    if (D.bf16)
        rmsnorm_dispatch<bf16_t>(T, x, (const bf16_t*)gamma, (bf16_t*)out, D.d, D.eps, s);
    else
        rmsnorm_dispatch<float>(T, x, (const float*)gamma, (float*)out, D.d, D.eps, s);
}

// ---------------------------------------------------------------------------
// QK-norm + rotate-half RoPE + KV append.  One wave per (slot, head) where
// heads 0..hq-1 are query heads and hq..hq+hkv-1 are KV heads.  Lane a < hd/2
// owns the rotation pair (a, a + hd/2).  Query heads go to qbuf; key heads
// go (normed, rotated) into the K block of the slot's page and the matching
// value row (unrotated) into the V^T block.
// ---------------------------------------------------------------------------
template <typename TA>
__global__ __launch_bounds__(256) void k_qkrope(BatchView bv, const float* qkv, const float* cs,
                                                TA* qbuf, KVPool kv, int layer, const TA* qn,
                                                const TA* kn, int hq, int hkv, int hd, int qk_norm,
                                                float eps) {
    const int wave = (blockIdx.x * 4) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int nh = hq + hkv;
    const int t = wave / nh, h = wave % nh;
    if (t >= bv.T) return;
    const int half = hd >> 1;
    const int nqkv = (hq + 2 * hkv) * hd;
    const bool act = lane < half;
    const bool is_q = h < hq;
    const int col = is_q ? h * hd : hq * hd + (h - hq) * hd;
    const float* src = qkv + (size_t)t * nqkv + col;
    float x0 = act ? src[lane] : 0.f;
    float x1 = act ? src[lane + half] : 0.f;
    if (qk_norm) {
        const float ss = wave_sum(x0 * x0 + x1 * x1);
        const float r = 1.0f / sqrtf(ss / (float)hd + eps);
        const TA* g = is_q ? qn : kn;
        if (act) {
            x0 = x0 * r * ld(g, lane);
            x1 = x1 * r * ld(g, lane + half);
        }
    }
    if (!act) return;
    const float c = cs[((size_t)t * half + lane) * 2 + 0];
    const float sn = cs[((size_t)t * half + lane) * 2 + 1];
    const float y0 = x0 * c - x1 * sn;
    const float y1 = x1 * c + x0 * sn;
    if (is_q) {
        TA* dst = qbuf + (size_t)t * hq * hd + (size_t)h * hd;
        st(dst, lane, y0);
        st(dst, lane + half, y1);
        return;
    }
    const int g = h - hq;
    const int b = bv.slot_b[t];
    const int pos = bv.prefix[b] + bv.slot_j[t];
    const int page = bv.page_table[(size_t)b * bv.max_pages + pos / kPageTokens];
    const int off = pos % kPageTokens;
    TA* base = (TA*)kv.base;
    TA* kd = base + kv.k_off(layer, page, g) + (size_t)off * hd;
    st(kd, lane, y0);
    st(kd, lane + half, y1);
    const float* vs = qkv + (size_t)t * nqkv + (size_t)(hq + hkv) * hd + (size_t)g * hd;
    TA* vd = base + kv.v_off(layer, page, g);
    st(vd, (size_t)lane * kPageTokens + off, vs[lane]);
    st(vd, (size_t)(lane + half) * kPageTokens + off, vs[lane + half]);
}

void launch_qkrope(const Dims& D, const BatchView& bv, const SlotBufs& sb, const KVPool& kv,
                   int layer, const void* qn, const void* kn, hipStream_t s) {
    const int waves = bv.T * (D.hq + D.hkv);
    const int blocks = (waves + 3) / 4;
    if (D.bf16)
        hipLaunchKernelGGL(k_qkrope<bf16_t>, dim3(blocks), dim3(256), 0, s, bv, sb.qkv, sb.cs,
                           (bf16_t*)sb.qbuf, kv, layer, (const bf16_t*)qn, (const bf16_t*)kn, D.hq,
                           D.hkv, D.hd, D.qk_norm, D.eps);
    else
        hipLaunchKernelGGL(k_qkrope<float>, dim3(blocks), dim3(256), 0, s, bv, sb.qkv, sb.cs,
                           (float*)sb.qbuf, kv, layer, (const float*)qn, (const float*)kn, D.hq,
                           D.hkv, D.hd, D.qk_norm, D.eps);
}

// ---------------------------------------------------------------------------
// KV copy between a caller buffer [n][hkv][hd] and one user's pages
// ---------------------------------------------------------------------------
template <typename TA>
__global__ void k_kv_copy(KVPool kv, const int32_t* pages, int layer, int pos0, int n, TA* k,
                          TA* v, int to_pool) {
    const int i = blockIdx.x, g = blockIdx.y;
    if (i >= n) return;
    const int hd = kv.hd, hkv = kv.hkv;
    const int pos = pos0 + i;
    const int page = pages[pos / kPageTokens], off = pos % kPageTokens;
    TA* base = (TA*)kv.base;
    TA* kp = base + kv.k_off(layer, page, g) + (size_t)off * hd;
    TA* vp = base + kv.v_off(layer, page, g);
    TA* kc = k + ((size_t)i * hkv + g) * hd;
    TA* vc = v + ((size_t)i * hkv + g) * hd;
    for (int a = threadIdx.x; a < hd; a += blockDim.x) {
        if (to_pool) {
            kp[a] = kc[a];
            vp[(size_t)a * kPageTokens + off] = vc[a];
        } else {
            kc[a] = kp[a];
            vc[a] = vp[(size_t)a * kPageTokens + off];
        }
    }
}

void launch_kv_copy(const Dims& D, const KVPool& kv, const int32_t* pages_dev, int layer,
                    int pos0, int n, const void* k, const void* v, int to_pool, hipStream_t s) {
    if (n <= 0) return;
    if (D.bf16)
        hipLaunchKernelGGL(k_kv_copy<bf16_t>, dim3(n, D.hkv), dim3(128), 0, s, kv, pages_dev,
                           layer, pos0, n, (bf16_t*)k, (bf16_t*)v, to_pool);
    else
        hipLaunchKernelGGL(k_kv_copy<float>, dim3(n, D.hkv), dim3(128), 0, s, kv, pages_dev, layer,
                           pos0, n, (float*)k, (float*)v, to_pool);
}

}  // namespace sdv
