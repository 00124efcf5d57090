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
__global__ void k_prepare(BatchView bv, int32_t* tok, int32_t* dnext, float* cs, int half, int V,
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
        // the draft whose acceptance slot t decides (-1 after the last
        // draft; an out-of-range draft, flagged by slot t + 1, reads as 0)
        int dn = -1;
        if (j < bv.L[b]) {
            dn = bv.drafts[bv.draft_off[b] + j];
            if (dn < 0 || dn >= V) dn = 0;
        }
        dnext[t] = dn;
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
    hipLaunchKernelGGL(k_prepare, dim3(bv.T), dim3(64), 0, s, bv, sb.tok, sb.dnext, sb.cs, D.hd / 2, D.V,
                       log((double)D.rope_base), D.hd);
}

// ---------------------------------------------------------------------------
// Split-K reduction fused with the residual add and the next RMSNorm:
// x[t] += sum_s part[s][t] (split order, fixed), h[t] = x[t] * rstd * gamma
// (h as activation planes, see st_act).  One workgroup per slot row, the
// row held in registers.
// ---------------------------------------------------------------------------
template <typename TA, int PER>
__global__ __launch_bounds__(1024) void k_resid_norm(const float* part, int S, int T, float* x,
                                                     const TA* gamma, TA* h, int d, float eps) {
    __shared__ float red[16];
    const int t = blockIdx.x;
    const int n4 = d >> 2;
    float4* xr = (float4*)(x + (size_t)t * d);
    const size_t plane4 = (size_t)T * d / 4;
    const float4* pr = (const float4*)(part + (size_t)t * d);
    float4 v[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) v[i] = float4{0.f, 0.f, 0.f, 0.f};
    // partial planes in split order, four planes' loads in flight at a time
    int sp = 0;
    for (; sp + 4 <= S; sp += 4) {
        float4 b[4][PER];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int k = threadIdx.x + i * 1024;
                b[q][i] = k < n4 ? pr[(sp + q) * plane4 + k] : float4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                v[i].x += b[q][i].x; v[i].y += b[q][i].y; v[i].z += b[q][i].z; v[i].w += b[q][i].w;
            }
    }
    for (; sp < S; ++sp)
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int k = threadIdx.x + i * 1024;
            if (k < n4) {
                const float4 b = pr[sp * plane4 + k];
                v[i].x += b.x; v[i].y += b.y; v[i].z += b.z; v[i].w += b.w;
            }
        }
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int k = threadIdx.x + i * 1024;
        if (k < n4) {
            float4 r = xr[k];
            r.x += v[i].x; r.y += v[i].y; r.z += v[i].z; r.w += v[i].w;
            xr[k] = r;
            v[i] = r;
        }
        ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < 16; ++w) tot += red[w];
    const float rs = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int k = threadIdx.x + i * 1024;
        if (k < n4) {
            const size_t o = (size_t)t * d + 4 * k, pl = (size_t)T * d;
            st_act(h, pl, o + 0, v[i].x * rs * ld(gamma, 4 * k + 0));
            st_act(h, pl, o + 1, v[i].y * rs * ld(gamma, 4 * k + 1));
            st_act(h, pl, o + 2, v[i].z * rs * ld(gamma, 4 * k + 2));
            st_act(h, pl, o + 3, v[i].w * rs * ld(gamma, 4 * k + 3));
        }
    }
}

template <typename TA>
static void resid_norm_dispatch(int T, const float* part, int S, float* x, const TA* gamma, TA* h,
                                int d, float eps, hipStream_t s) {
    const int per = (d / 4 + 1023) / 1024;
    if (per <= 1) hipLaunchKernelGGL((k_resid_norm<TA, 1>), dim3(T), dim3(1024), 0, s, part, S, T, x, gamma, h, d, eps);
    else hipLaunchKernelGGL((k_resid_norm<TA, 2>), dim3(T), dim3(1024), 0, s, part, S, T, x, gamma, h, d, eps);
}

void launch_resid_norm(const Dims& D, int T, const float* part, int S, float* x,
                       const void* gamma, void* h, hipStream_t s) {
    if (D.bf16)
        resid_norm_dispatch<bf16_t>(T, part, S, x, (const bf16_t*)gamma, (bf16_t*)h, D.d, D.eps, s);
    else
        resid_norm_dispatch<float>(T, part, S, x, (const float*)gamma, (float*)h, D.d, D.eps, s);
}

// ---------------------------------------------------------------------------
// bf16 configuration: split-K reduction fused with the residual add and the
// elementwise half of the next RMSNorm.  x[t] += sum_s part[s][t] (split
// order, fixed); h[t] = x[t] * gamma as activation planes; and the sum of
// squares of each 1024-column block of the new x.  The row factor rstd(t)
// is applied by the consumers of h after their products (it commutes with
// them), so no workgroup needs a whole row: one workgroup per (slot row,
// column block), five per row of the 32B model, where one workgroup per row
// (the fused norm) is bound by what a single CU can pull.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_resid_reduce(const float* part, int S, int T, float* x,
                                                      const bf16_t* gamma, bf16_t* h, float* ssq,
                                                      int d, int nsq) {
    __shared__ float red[4];
    const int t = blockIdx.x, blk = blockIdx.y;
    const int k = blk * 256 + threadIdx.x;  // float4 column index
    const bool act = k < (d >> 2);
    float4* xr = (float4*)(x + (size_t)t * d);
    const size_t plane4 = (size_t)T * d / 4;
    const float4* pr = (const float4*)(part + (size_t)t * d);
    const float4 xv = act ? xr[k] : float4{0.f, 0.f, 0.f, 0.f};
    const uint2 gq = act ? *(const uint2*)(gamma + 4 * k) : uint2{0u, 0u};
    // partial planes added in split order, sixteen planes' loads in flight
    // (one memory round trip for the split counts the GEMMs choose)
    float4 v = float4{0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < S; sp += 16) {
        float4 b[16];
#pragma unroll
        for (int q = 0; q < 16; ++q)
            b[q] = act && sp + q < S ? pr[(sp + q) * plane4 + k] : float4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            v.x += b[q].x; v.y += b[q].y; v.z += b[q].z; v.w += b[q].w;
        }
    }
    float4 r = xv;
    r.x += v.x; r.y += v.y; r.z += v.z; r.w += v.w;
    if (act) {
        xr[k] = r;
        const size_t o = (size_t)t * d + 4 * k, pl = (size_t)T * d;
        const float hv[4] = {r.x * bf16_to_f32((bf16_t)(gq.x & 0xffffu)), r.y * bf16_to_f32((bf16_t)(gq.x >> 16)),
                             r.z * bf16_to_f32((bf16_t)(gq.y & 0xffffu)), r.w * bf16_to_f32((bf16_t)(gq.y >> 16))};
        st_act4(h, pl, o, hv);
    }
    float ss = act ? r.x * r.x + r.y * r.y + r.z * r.z + r.w * r.w : 0.f;
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    if (threadIdx.x == 0) ssq[(size_t)t * nsq + blk] = red[0] + red[1] + red[2] + red[3];
}

void launch_resid_reduce(const Dims& D, int T, const float* part, int S, float* x,
                         const void* gamma, void* h, float* ssq, int nsq, hipStream_t s) {
    hipLaunchKernelGGL(k_resid_reduce, dim3(T, nsq), dim3(256), 0, s, part, S, T, x,
                       (const bf16_t*)gamma, (bf16_t*)h, ssq, D.d, nsq);
}

// bf16 configuration: embedding gather into x, h = x * gamma (activation
// planes) and the block sums of squares (the first QKV GEMM's consumer
// applies rstd); iteration i of a thread covers column block i
template <int PER>
__global__ __launch_bounds__(256) void k_embed_ss(const int32_t* tok, const bf16_t* E,
                                                  const bf16_t* gamma, float* x, bf16_t* h,
                                                  float* ssq, int d, int nsq, int T) {
    __shared__ float red[PER][4];
    const int t = blockIdx.x;
    const size_t row = (size_t)tok[t] * d;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int k = threadIdx.x + i * 256;
        float v[4];
        float ss = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[e] = 4 * k < d ? ld(E, row + 4 * k + e) : 0.f;
            ss += v[e] * v[e];
        }
        if (4 * k < d) {
            *(float4*)(x + (size_t)t * d + 4 * k) = float4{v[0], v[1], v[2], v[3]};
#pragma unroll
            for (int e = 0; e < 4; ++e)
                st_act(h, (size_t)T * d, (size_t)t * d + 4 * k + e, v[e] * ld(gamma, 4 * k + e));
        }
        ss = wave_sum(ss);
        if ((threadIdx.x & 63) == 0) red[i][threadIdx.x >> 6] = ss;
    }
    __syncthreads();
    if ((int)threadIdx.x < nsq) ssq[(size_t)t * nsq + threadIdx.x] = red[threadIdx.x][0] +
                                                                  red[threadIdx.x][1] +
                                                                  red[threadIdx.x][2] +
                                                                  red[threadIdx.x][3];
}

// embedding gather fused with the first RMSNorm
template <typename TA, int PER>
__global__ __launch_bounds__(256) void k_embed_norm(const int32_t* tok, const TA* E,
                                                    const TA* gamma, float* x, TA* h, int d,
                                                    float eps, int T) {
    __shared__ float red[4];
    const int t = blockIdx.x;
    const size_t row = (size_t)tok[t] * d;
    float v[PER][4];
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int k = threadIdx.x + i * 256;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[i][e] = 4 * k < d ? ld(E, row + 4 * k + e) : 0.f;
            ss += v[i][e] * v[i][e];
        }
        if (4 * k < d)
            *(float4*)(x + (size_t)t * d + 4 * k) = float4{v[i][0], v[i][1], v[i][2], v[i][3]};
    }
    ss = block_sum_256(ss, red);
    const float rs = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int k = threadIdx.x + i * 256;
        if (4 * k < d)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                st_act(h, (size_t)T * d, (size_t)t * d + 4 * k + e, v[i][e] * rs * ld(gamma, 4 * k + e));
    }
}

void launch_embed_norm(const Dims& D, const BatchView& bv, const void* embed, const void* gamma,
                       const SlotBufs& sb, hipStream_t s) {
    const int per = (D.d / 4 + 255) / 256;
#define EN(TA, P) hipLaunchKernelGGL((k_embed_norm<TA, P>), dim3(bv.T), dim3(256), 0, s, sb.tok, \
                                     (const TA*)embed, (const TA*)gamma, sb.x, (TA*)sb.h, D.d, D.eps, bv.T)
    if (D.bf16) {
        // x, h = x * gamma and the block sums of squares
        const int nsq = sb.nsq;
#define ES(P) hipLaunchKernelGGL((k_embed_ss<P>), dim3(bv.T), dim3(256), 0, s, sb.tok, \
                                 (const bf16_t*)embed, (const bf16_t*)gamma, sb.x, (bf16_t*)sb.h, \
                                 sb.ssq, D.d, nsq, bv.T)
        if (nsq <= 1) ES(1); else if (nsq <= 2) ES(2); else if (nsq <= 4) ES(4); else ES(8);
#undef ES
    } else {
        if (per <= 1) EN(float, 1); else if (per <= 2) EN(float, 2); else if (per <= 5) EN(float, 5); else EN(float, 8);
    }
#undef EN
}

// ---------------------------------------------------------------------------
// QK-norm + rotate-half RoPE + KV append (fp32 configuration).  One wave
// per (slot, head) where heads 0..hq-1 are query heads and hq..hq+hkv-1 are
// KV heads.  Lane a < hd/2 owns the rotation pair (a, a + hd/2).  Query heads go to qbuf; key heads
// go (normed, rotated) into the K block of the slot's page and the matching
// value row (unrotated) into the V^T block.
// ---------------------------------------------------------------------------
template <typename TA>
__global__ __launch_bounds__(256) void k_qkrope(BatchView bv, const float* qkv, int S,
                                                const float* cs, TA* qbuf, KVPool kv, int layer,
                                                const TA* qn, const TA* kn, int hq, int hkv, int hd,
                                                int qk_norm, float eps, const float* nss, int nnb,
                                                int d) {
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
    // qkv holds S split-K partial planes [S][T][nqkv]; add them in order
    const size_t plane = (size_t)bv.T * nqkv;
    const float* src = qkv + (size_t)t * nqkv + col;
    // the input's RMSNorm row factor (bf16: the GEMM multiplied x * gamma);
    // its block sums are requested first
    float ssb[kNormKMax / kNormBlock];
#pragma unroll
    for (int b = 0; b < kNormKMax / kNormBlock; ++b)
        ssb[b] = nss != nullptr && b < nnb ? nss[(size_t)t * nnb + b] : 0.f;
    // partial planes added in split order, eight planes' loads in flight at
    // a time (key heads also fetch their value columns in the same batch)
    const float* vs = qkv + (size_t)t * nqkv + (size_t)(hq + hkv) * hd + (size_t)(is_q ? 0 : h - hq) * hd;
    float x0 = 0.f, x1 = 0.f, v0 = 0.f, v1 = 0.f;
    for (int sp = 0; sp < S; sp += 8) {
        float a0[8], a1[8], b0[8], b1[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const bool ok = act && sp + u < S;
            const size_t o = (size_t)(sp + u) * plane + lane;
            a0[u] = ok ? src[o] : 0.f;
            a1[u] = ok ? src[o + half] : 0.f;
            b0[u] = ok && !is_q ? vs[o] : 0.f;
            b1[u] = ok && !is_q ? vs[o + half] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            x0 += a0[u];
            x1 += a1[u];
            v0 += b0[u];
            v1 += b1[u];
        }
    }
    float rt = 1.0f;
    if (nss != nullptr) {
        float ssx = 0.f;
#pragma unroll
        for (int b = 0; b < kNormKMax / kNormBlock; ++b) ssx += ssb[b];
        rt = 1.0f / sqrtf(ssx / (float)d + eps);
        x0 *= rt;
        x1 *= rt;
    }
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
        const size_t q0 = ((size_t)t * hq + h) * hd, pl = (size_t)bv.T * hq * hd;
        st_act(qbuf, pl, q0 + lane, y0);
        st_act(qbuf, pl, q0 + lane + half, y1);
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
    v0 *= rt;
    v1 *= rt;
    TA* vd = base + kv.v_off(layer, page, g);
    st(vd, (size_t)lane * kPageTokens + off, v0);
    st(vd, (size_t)(lane + half) * kPageTokens + off, v1);
}

// bf16 configuration (head_dim 128): the same steps with 16 lanes per head
// and four heads of one slot per wave.  Lane l of a head owns dims 4l..4l+3
// and their rotation partners 64+4l..64+4l+3, so every partial-plane read is
// a 16-byte load (a wave reads 1 KB per instruction instead of 256 B) and
// the query and key rows leave as 8-byte stores.  Value heads take lanes of
// their own (they are only summed, scaled and appended), so every wave
// carries the same loads.  One wave per workgroup, so that few waves (small
// batches) still spread over the CUs.
__global__ __launch_bounds__(64) void k_qkrope_bf16(BatchView bv, const float* qkv, int S,
                                                     const float* cs, bf16_t* qbuf, KVPool kv,
                                                     int layer, const bf16_t* qn, const bf16_t* kn,
                                                     int hq, int hkv, int qk_norm, float eps,
                                                     const float* nss, int nnb, int d) {
    constexpr int HD = 128, HALF = 64;
    const int wave = blockIdx.x;
    const int lane = threadIdx.x, l = lane & 15;
    // q, k and v heads (contiguous in the QKV output), four per wave
    const int nh = hq + 2 * hkv, ng = (nh + 3) >> 2;
    const int t = wave / ng;
    if (t >= bv.T) return;
    const int h = (wave % ng) * 4 + (lane >> 4);
    const bool act = h < nh;
    const bool is_q = h < hq, is_v = h >= hq + hkv;
    const int nqkv = nh * HD;
    const size_t plane = (size_t)bv.T * nqkv;
    const float* src = qkv + (size_t)t * nqkv + (size_t)h * HD + 4 * l;
    float ssb[kNormKMax / kNormBlock];
#pragma unroll
    for (int b = 0; b < kNormKMax / kNormBlock; ++b)
        ssb[b] = nss != nullptr && b < nnb ? nss[(size_t)t * nnb + b] : 0.f;
    // partial planes added in split order, eight planes' loads in flight
    f32x4 xa = f32x4{0.f, 0.f, 0.f, 0.f}, xb = xa;
    for (int sp = 0; sp < S; sp += 8) {
        f32x4 a0[8], a1[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const bool ok = act && sp + u < S;
            const size_t o = (size_t)(sp + u) * plane;
            const f32x4 z = f32x4{0.f, 0.f, 0.f, 0.f};
            a0[u] = ok ? *(const f32x4*)(src + o) : z;
            a1[u] = ok ? *(const f32x4*)(src + o + HALF) : z;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            xa += a0[u];
            xb += a1[u];
        }
    }
    if (nss != nullptr) {
        float ssx = 0.f;
#pragma unroll
        for (int b = 0; b < kNormKMax / kNormBlock; ++b) ssx += ssb[b];
        const float rt = 1.0f / sqrtf(ssx / (float)d + eps);
        xa *= rt;
        xb *= rt;
    }
    const int b = bv.slot_b[t];
    const int pos = bv.prefix[b] + bv.slot_j[t];
    if (is_v) {
        if (!act) return;
        const int g = h - hq - hkv;
        const int page = bv.page_table[(size_t)b * bv.max_pages + pos / kPageTokens];
        const int off = pos % kPageTokens;
        bf16_t* vd = (bf16_t*)kv.base + kv.v_off(layer, page, g);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            vd[(size_t)(4 * l + e) * kPageTokens + off] = f32_to_bf16(xa[e]);
            vd[(size_t)(HALF + 4 * l + e) * kPageTokens + off] = f32_to_bf16(xb[e]);
        }
        return;
    }
    if (qk_norm) {
        float ss = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) ss += xa[e] * xa[e] + xb[e] * xb[e];
#pragma unroll
        for (int o = 8; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 16);
        const float r = 1.0f / sqrtf(ss / (float)HD + eps);
        const bf16_t* g = is_q ? qn : kn;
        if (act) {
            const uint2 ga = *(const uint2*)(g + 4 * l), gb = *(const uint2*)(g + HALF + 4 * l);
            const uint32_t gw[4] = {ga.x, ga.y, gb.x, gb.y};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t wa = gw[e >> 1], wb = gw[2 + (e >> 1)];
                xa[e] = xa[e] * r * bf16_to_f32((bf16_t)((e & 1) ? wa >> 16 : wa & 0xffffu));
                xb[e] = xb[e] * r * bf16_to_f32((bf16_t)((e & 1) ? wb >> 16 : wb & 0xffffu));
            }
        }
    }
    if (!act) return;
    const f32x4 c0 = *(const f32x4*)(cs + ((size_t)t * HALF + 4 * l) * 2);
    const f32x4 c1 = *(const f32x4*)(cs + ((size_t)t * HALF + 4 * l) * 2 + 4);
    const float cv[4] = {c0[0], c0[2], c1[0], c1[2]}, sv[4] = {c0[1], c0[3], c1[1], c1[3]};
    float ya[4], yb[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        ya[e] = xa[e] * cv[e] - xb[e] * sv[e];
        yb[e] = xb[e] * cv[e] + xa[e] * sv[e];
    }
    if (is_q) {
        const size_t q0 = ((size_t)t * hq + h) * HD + 4 * l, pl = (size_t)bv.T * hq * HD;
        st_act4(qbuf, pl, q0, ya);
        st_act4(qbuf, pl, q0 + HALF, yb);
        return;
    }
    const int g = h - hq;
    const int page = bv.page_table[(size_t)b * bv.max_pages + pos / kPageTokens];
    const int off = pos % kPageTokens;
    bf16_t* kd = (bf16_t*)kv.base + kv.k_off(layer, page, g) + (size_t)off * HD + 4 * l;
    *(uint2*)kd = pack_bf16x4(ya);
    *(uint2*)(kd + HALF) = pack_bf16x4(yb);
}

void launch_qkv_finish(const Dims& D, const BatchView& bv, const SlotBufs& sb, const KVPool& kv,
                       int layer, const float* part, int S, const void* qn, const void* kn,
                       hipStream_t s) {
    if (D.bf16) {
        // head_dim 128 (checked at init): four heads per wave
        const int waves = bv.T * ((D.hq + 2 * D.hkv + 3) / 4);
        hipLaunchKernelGGL(k_qkrope_bf16, dim3(waves), dim3(64), 0, s, bv, part, S, sb.cs,
                           (bf16_t*)sb.qbuf, kv, layer, (const bf16_t*)qn, (const bf16_t*)kn, D.hq,
                           D.hkv, D.qk_norm, D.eps, sb.ssq, sb.nsq, D.d);
        return;
    }
    const int waves = bv.T * (D.hq + D.hkv);
    hipLaunchKernelGGL(k_qkrope<float>, dim3((waves + 3) / 4), dim3(256), 0, s, bv, part, S, sb.cs,
                       (float*)sb.qbuf, kv, layer, (const float*)qn, (const float*)kn, D.hq, D.hkv,
                       D.hd, D.qk_norm, D.eps, (const float*)nullptr, 0, D.d);
}

// ---------------------------------------------------------------------------
// KV copy between a caller buffer [n][hkv][hd] and one user's pages.  The
// pages of one launch travel in its kernel arguments (at most kKVCopyPages
// of them, starting at the user's page index page0), so a copy needs no
// device staging buffer and no host wait.
// ---------------------------------------------------------------------------
template <typename TA>
__global__ void k_kv_copy(KVPool kv, KVCopyPages pages, int layer, int pos0, int n, TA* k,
                          TA* v, int to_pool) {
    const int i = blockIdx.x, g = blockIdx.y;
    if (i >= n) return;
    const int hd = kv.hd, hkv = kv.hkv;
    const int pos = pos0 + i;
    const int page = pages.id[pos / kPageTokens - pages.page0], off = pos % kPageTokens;
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

void launch_kv_copy(const Dims& D, const KVPool& kv, const KVCopyPages& pages, int layer,
                    int pos0, int n, const void* k, const void* v, int to_pool, hipStream_t s) {
    if (n <= 0) return;
    if (D.bf16)
        hipLaunchKernelGGL(k_kv_copy<bf16_t>, dim3(n, D.hkv), dim3(128), 0, s, kv, pages,
                           layer, pos0, n, (bf16_t*)k, (bf16_t*)v, to_pool);
    else
        hipLaunchKernelGGL(k_kv_copy<float>, dim3(n, D.hkv), dim3(128), 0, s, kv, pages, layer,
                           pos0, n, (float*)k, (float*)v, to_pool);
}

}  // namespace sdv
