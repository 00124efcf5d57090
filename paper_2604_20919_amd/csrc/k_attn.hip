// Ragged paged causal attention with grouped query heads.
//
// For user b and KV head g the query rows are the (l_b + 1) slots times the
// G query heads sharing g; slot j sits at position i_b + j and attends to
// positions 0 .. i_b + j (cached prefix plus the batch's own earlier slots,
// whose keys the QK-norm/RoPE kernel has already appended to the pages).
//
// bf16 path (MFMA): a workgroup takes one work item (b, g, context chunk of
// up to 256 tokens); its 4 waves take interleaved 32-token blocks.  Per
// block, for up to 4 tiles of 16 query rows:
//   S^T = K Q^T   with K as the A operand (16 tokens x 32 dims) and Q^T as
//                 the B operand; the K rows are loaded in the token order
//                 (0-3, 8-11, 16-19, 24-27 | 4-7, 12-15, 20-23, 28-31) so that
//                 each lane ends up holding 8 consecutive tokens of one query
//                 row -- exactly the B-operand layout of the next product;
//   O^T += V^T P^T with V^T fragments read straight from the dim-major V
//                 page blocks and P^T taken from registers (no LDS transpose).
// The softmax is online in fp32 (exp2 domain).  Each wave writes its partial
// (row max, row sum, unnormalised output); a combine kernel merges the
// partials of all chunks in a fixed order, so results are deterministic.
//
// fp32 path: one wave per (slot, query head), plain loop over the context.
#include "sdv_device.h"
#include "sdv_internal.h"

namespace sdv {

struct AttnP {
    BatchView bv;
    const bf16_t* q;   // [T][hq][hd]
    KVPool kv;
    int layer;
    int hq, hkv, G;
    float scale_log2;  // log2(e) / sqrt(hd)
    float* apart;      // [items*4][rows_max][hd]
    float* aml;        // [items*4][rows_max][2]
};

constexpr int HD = 128;

template <int RT>
__global__ __launch_bounds__(256) void k_attn_bf16(AttnP p) {
    const int item = blockIdx.x;
    const int4 it = p.bv.items[item];
    const int b = it.x, g = it.y, c0 = it.z, c1 = it.w;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int lr = lane & 15, lg = lane >> 4;
    const int G = p.G;
    const int nslot = p.bv.L[b] + 1;
    const int R = nslot * G;
    const int prefix = p.bv.prefix[b];
    const int tbase = p.bv.slot_off[b];
    const int32_t* pt = p.bv.page_table + (size_t)b * p.bv.max_pages;
    const bf16_t* kvb = (const bf16_t*)p.kv.base;
    const int nblk = (c1 - c0 + 31) >> 5;
    const int pidx = item * 4 + wave;
    // token order of the K rows this lane loads (A operand row lr)
    const int pi0 = 8 * (lr >> 2) + (lr & 3);
    const int pi1 = pi0 + 4;

    for (int rp0 = 0; rp0 < R; rp0 += 16 * RT) {
        bf16x8 qf[RT][4];
        int lim[RT];
        float m[RT], l[RT];
        f32x4 o[RT][8];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const int row = rp0 + rt * 16 + lr;
            const bool ok = row < R;
            const int j = ok ? row / G : 0, hh = ok ? row % G : 0;
            const bf16_t* qs = p.q + ((size_t)(tbase + j) * p.hq + g * G + hh) * HD + 8 * lg;
#pragma unroll
            for (int ds = 0; ds < 4; ++ds) {
                if (ok)
                    qf[rt][ds] = *(const bf16x8*)(qs + ds * 32);
                else
                    qf[rt][ds] = bf16x8{};
            }
            lim[rt] = prefix + j;
            m[rt] = -INFINITY;
            l[rt] = 0.f;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) o[rt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        const int rt_act = min(RT, (R - rp0 + 15) >> 4);

        for (int blk = wave; blk < nblk; blk += 4) {
            const int t0 = c0 + blk * 32;
            // K fragments of the two 16-token tiles
            bf16x8 ka[4], kb[4];
            {
                const int ta = t0 + pi0, tb = t0 + pi1;
                const bf16_t* pa = kvb + p.kv.k_off(p.layer, ta < c1 ? pt[ta >> 4] : 0, g) +
                                   (size_t)(ta & 15) * HD + 8 * lg;
                const bf16_t* pb = kvb + p.kv.k_off(p.layer, tb < c1 ? pt[tb >> 4] : 0, g) +
                                   (size_t)(tb & 15) * HD + 8 * lg;
#pragma unroll
                for (int ds = 0; ds < 4; ++ds) {
                    ka[ds] = ta < c1 ? *(const bf16x8*)(pa + ds * 32) : bf16x8{};
                    kb[ds] = tb < c1 ? *(const bf16x8*)(pb + ds * 32) : bf16x8{};
                }
            }
            // V^T fragments: dims dt*16 + lr, tokens t0 + 8*lg .. +7
            bf16x8 vf[8];
            {
                const int tv = t0 + 8 * lg;
                const int page = tv < c1 ? pt[tv >> 4] : 0;
                const bf16_t* pv = kvb + p.kv.v_off(p.layer, page, g) + (tv & 15);
                const int nvalid = c1 - tv;  // tokens of this group inside the chunk
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) {
                    if (nvalid >= 8) {
                        vf[dt] = *(const bf16x8*)(pv + (size_t)(dt * 16 + lr) * kPageTokens);
                    } else {
                        bf16x8 v = bf16x8{};
                        for (int e = 0; e < nvalid; ++e)
                            v[e] = *(const __bf16*)(pv + (size_t)(dt * 16 + lr) * kPageTokens + e);
                        vf[dt] = v;
                    }
                }
            }
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                if (rt >= rt_act) continue;
                f32x4 sa = f32x4{0.f, 0.f, 0.f, 0.f}, sb = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ds = 0; ds < 4; ++ds) {
                    sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[ds], qf[rt][ds], sa, 0, 0, 0);
                    sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb[ds], qf[rt][ds], sb, 0, 0, 0);
                }
                // lane holds scores of query row (rp0 + rt*16 + lr) at tokens
                // t0 + 8*lg + e, e = 0..7 (sa: e < 4, sb: e >= 4)
                float s[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    s[e] = sa[e];
                    s[4 + e] = sb[e];
                }
                float bm = -INFINITY;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int tok = t0 + 8 * lg + e;
                    s[e] = (tok < c1 && tok <= lim[rt]) ? s[e] * p.scale_log2 : -INFINITY;
                    bm = fmaxf(bm, s[e]);
                }
                bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
                bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
                const float mn = fmaxf(m[rt], bm);
                if (mn == -INFINITY) continue;  // nothing visible yet for this row
                const float alpha = exp2f(m[rt] - mn);
                float rs = 0.f;
                bf16x8 pb8;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float pe = exp2f(s[e] - mn);
                    rs += pe;
                    pb8[e] = (__bf16)pe;
                }
                rs += __shfl_xor(rs, 16, 64);
                rs += __shfl_xor(rs, 32, 64);
                l[rt] = l[rt] * alpha + rs;
                m[rt] = mn;
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) {
                    o[rt][dt] *= alpha;
                    o[rt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[dt], pb8, o[rt][dt], 0, 0, 0);
                }
            }
        }
        // partial of this wave: lane holds O^T[d = dt*16 + 4*lg + r][row lr]
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const int row = rp0 + rt * 16 + lr;
            if (row >= R) continue;
            const size_t pr = (size_t)pidx * p.bv.rows_max + row;
            if (lg == 0) {
                p.aml[pr * 2 + 0] = m[rt];
                p.aml[pr * 2 + 1] = l[rt];
            }
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
                *(f32x4*)(p.apart + pr * HD + dt * 16 + 4 * lg) = o[rt][dt];
        }
    }
}

// Merge the partials of all chunks and waves of (b, g) for one query row in
// a fixed order; one wave per (slot, query head).
template <typename TA>
__global__ __launch_bounds__(256) void k_attn_combine(BatchView bv, const float* apart,
                                                      const float* aml, TA* out, int hq, int hkv,
                                                      int hd) {
    const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int t = wave / hq, h = wave % hq;
    if (t >= bv.T) return;
    const int G = hq / hkv, g = h / G, hh = h % G;
    const int b = bv.slot_b[t], j = bv.slot_j[t];
    const int row = j * G + hh;
    const int i0 = bv.item_off[b], nch = (bv.item_off[b + 1] - i0) / hkv;
    const int p0 = (i0 + g * nch) * 4, p1 = p0 + nch * 4;
    float M = -INFINITY;
    for (int pi = p0; pi < p1; ++pi) M = fmaxf(M, aml[((size_t)pi * bv.rows_max + row) * 2]);
    float Ls = 0.f, acc0 = 0.f, acc1 = 0.f;
    for (int pi = p0; pi < p1; ++pi) {
        const size_t pr = (size_t)pi * bv.rows_max + row;
        const float mi = aml[pr * 2];
        if (mi == -INFINITY) continue;
        const float w = exp2f(mi - M);
        Ls += aml[pr * 2 + 1] * w;
        acc0 += apart[pr * hd + lane] * w;
        if (lane + 64 < hd) acc1 += apart[pr * hd + lane + 64] * w;
    }
    const float inv = 1.0f / Ls;
    TA* dst = out + (size_t)t * hq * hd + (size_t)h * hd;
    if (lane < hd) st(dst, lane, acc0 * inv);
    if (lane + 64 < hd) st(dst, lane + 64, acc1 * inv);
}

// fp32 path: one wave per (slot, query head); lanes split head_dim
__global__ __launch_bounds__(256) void k_attn_f32(BatchView bv, const float* q, KVPool kv,
                                                  int layer, float* out, int hq, int hkv, int hd,
                                                  float scale) {
    const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int t = wave / hq, h = wave % hq;
    if (t >= bv.T) return;
    const int G = hq / hkv, g = h / G;
    const int b = bv.slot_b[t];
    const int n = bv.prefix[b] + bv.slot_j[t] + 1;
    const int32_t* pt = bv.page_table + (size_t)b * bv.max_pages;
    const float* base = (const float*)kv.base;
    const float* qv = q + ((size_t)t * hq + h) * hd;
    float m = -INFINITY, l = 0.f, a0 = 0.f, a1 = 0.f;
    const float q0 = lane < hd ? qv[lane] : 0.f, q1 = lane + 64 < hd ? qv[lane + 64] : 0.f;
    for (int tok = 0; tok < n; ++tok) {
        const int page = pt[tok >> 4], off = tok & 15;
        const float* kr = base + kv.k_off(layer, page, g) + (size_t)off * hd;
        const float* vb = base + kv.v_off(layer, page, g);
        float d = (lane < hd ? q0 * kr[lane] : 0.f) + (lane + 64 < hd ? q1 * kr[lane + 64] : 0.f);
        d = wave_sum(d) * scale;
        const float mn = fmaxf(m, d);
        const float al = expf(m - mn), pe = expf(d - mn);
        l = l * al + pe;
        if (lane < hd) a0 = a0 * al + pe * vb[(size_t)lane * kPageTokens + off];
        if (lane + 64 < hd) a1 = a1 * al + pe * vb[(size_t)(lane + 64) * kPageTokens + off];
        m = mn;
    }
    float* dst = out + ((size_t)t * hq + h) * hd;
    if (lane < hd) dst[lane] = a0 / l;
    if (lane + 64 < hd) dst[lane + 64] = a1 / l;
}

void launch_attention(const Dims& D, const BatchView& bv, const SlotBufs& sb, const KVPool& kv,
                      int layer, hipStream_t s) {
    const int waves = bv.T * D.hq;
    const int blocks = (waves + 3) / 4;
    if (!D.bf16) {
        hipLaunchKernelGGL(k_attn_f32, dim3(blocks), dim3(256), 0, s, bv, (const float*)sb.qbuf,
                           kv, layer, (float*)sb.attn, D.hq, D.hkv, D.hd,
                           1.0f / sqrtf((float)D.hd));
        return;
    }
    AttnP p;
    p.bv = bv;
    p.q = (const bf16_t*)sb.qbuf;
    p.kv = kv;
    p.layer = layer;
    p.hq = D.hq;
    p.hkv = D.hkv;
    p.G = D.G();
    p.scale_log2 = 1.4426950408889634f / sqrtf((float)D.hd);
    p.apart = sb.apart;
    p.aml = sb.aml;
    const int rtiles = (bv.rows_max + 15) / 16;
    if (rtiles <= 1)
        hipLaunchKernelGGL(k_attn_bf16<1>, dim3(bv.n_items), dim3(256), 0, s, p);
    else if (rtiles <= 2)
        hipLaunchKernelGGL(k_attn_bf16<2>, dim3(bv.n_items), dim3(256), 0, s, p);
    else if (rtiles <= 3)
        hipLaunchKernelGGL(k_attn_bf16<3>, dim3(bv.n_items), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL(k_attn_bf16<4>, dim3(bv.n_items), dim3(256), 0, s, p);
    hipLaunchKernelGGL(k_attn_combine<bf16_t>, dim3(blocks), dim3(256), 0, s, bv, sb.apart, sb.aml,
                       (bf16_t*)sb.attn, D.hq, D.hkv, D.hd);
}

}  // namespace sdv
