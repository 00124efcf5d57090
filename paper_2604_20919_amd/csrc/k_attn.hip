// Ragged paged causal attention with grouped query heads.
//
// For user b and KV head g the query rows are the (l_b + 1) slots times the
// G query heads sharing g; slot j sits at position i_b + j and attends to
// positions 0 .. i_b + j (cached prefix plus the batch's own earlier slots,
// whose keys the QK-norm/RoPE kernel has already appended to the pages).
//
// bf16 path (MFMA).  A workgroup takes one work item (b, g, context chunk);
// the host sizes chunks so that a batch has about 512 items of equal length.
// The chunk is streamed in 32-token blocks (two KV pages, 16 KB of K and V)
// through double-buffered LDS; the blocks are written to LDS in MFMA
// fragment order, so every operand read is one contiguous 1 KB wave read.
// Wave w owns query-row tiles w, w+4, ... (16 rows each) and, per block:
//   S^T = K Q^T   K rows as the A operand (16 tokens x 32 dims), in the token
//                 order (0-3, 8-11, 16-19, 24-27 | 4-7, 12-15, 20-23, 28-31)
//                 so that each lane ends up with 8 consecutive tokens of one
//                 query row -- the B-operand layout of the next product;
//   O^T += V^T P^T with V^T fragments from the dim-major V page blocks and
//                 P^T taken from registers (no transpose).
// The softmax is online in fp32 (exp2 domain).  Each item writes one partial
// (row max, row sum, unnormalised output); a combine kernel merges the
// partials of a row's chunks in chunk order, so results are deterministic.
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
    float* apart;      // [items][rows_max][hd]
    float* aml;        // [items][rows_max][2]
};

constexpr int HD = 128;
constexpr int RT_MAX = 2;  // row tiles per wave and pass

// LDS fragment index of K element (token t of the block, 16-byte dim piece j)
__device__ __forceinline__ int k_frag_slot(int t, int j) {
    const int tt = (t >> 2) & 1, lr = 4 * (t >> 3) + (t & 3);
    const int ds = j >> 2, lg = j & 3;
    return (tt * 4 + ds) * 64 + lr + 16 * lg;
}
// LDS fragment index of V^T piece (dim d, tokens 8h..8h+7 of page pg)
__device__ __forceinline__ int v_frag_slot(int d, int pg, int h) {
    return (d >> 4) * 64 + (d & 15) + 16 * (pg * 2 + h);
}

__global__ __launch_bounds__(256) void k_attn_bf16(AttnP p) {
    __shared__ __attribute__((aligned(16))) uint4 kvs[2][1024];  // [buf][K 512 | V 512] x 16 B
    const int item = blockIdx.x;
    const int4 it = p.bv.items[item];
    const int b = it.x, g = it.y, c0 = it.z, c1 = it.w;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int lr = lane & 15, lg = lane >> 4;
    const int G = p.G;
    const int R = (p.bv.L[b] + 1) * G;
    const int prefix = p.bv.prefix[b];
    const int tbase = p.bv.slot_off[b];
    const int32_t* pt = p.bv.page_table + (size_t)b * p.bv.max_pages;
    const char* kvb = (const char*)p.kv.base;
    const int nblk = (c1 - c0 + 31) >> 5;

    // staging: thread i moves K piece (token i/16, dims 8*(i%16)) and V^T
    // piece (dim i/2, tokens 8*(i%2)) of both pages of the block
    const int tid = threadIdx.x;
    const int kt = tid >> 4, kj = tid & 15;   // K: token 0..15 of a page, piece
    const int vd = tid >> 1, vh = tid & 1;    // V: dim 0..127, token half
    uint4 st[4];
    auto load_blk = [&](int blk) {
        const int t0 = c0 + blk * 32;
#pragma unroll
        for (int pg = 0; pg < 2; ++pg) {
            // clamp to the last valid token: masked tokens only need finite data
            const int tok = min(t0 + pg * 16, c1 - 1);
            const int page = pt[tok >> 4];
            const char* kp = kvb + (p.kv.k_off(p.layer, page, g) * 2);
            const char* vp = kvb + (p.kv.v_off(p.layer, page, g) * 2);
            st[pg * 2 + 0] = *(const uint4*)(kp + (kt * HD + kj * 8) * 2);
            uint4 v = *(const uint4*)(vp + (vd * kPageTokens + vh * 8) * 2);
            // value slots past the chunk end may hold stale bits (even NaN):
            // zero them so that p = 0 times v stays 0 (masked keys are
            // handled by the score mask)
            const int vt = t0 + pg * 16 + vh * 8;  // token of element 0
            uint32_t* w = (uint32_t*)&v;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t lo = vt + 2 * e < c1 ? 0x0000ffffu : 0u;
                const uint32_t hi = vt + 2 * e + 1 < c1 ? 0xffff0000u : 0u;
                w[e] &= lo | hi;
            }
            st[pg * 2 + 1] = v;
        }
    };
    auto store_blk = [&](int buf) {
#pragma unroll
        for (int pg = 0; pg < 2; ++pg) {
            kvs[buf][k_frag_slot(pg * 16 + kt, kj)] = st[pg * 2 + 0];
            kvs[buf][512 + v_frag_slot(vd, pg, vh)] = st[pg * 2 + 1];
        }
    };

    const int ntiles = (R + 15) >> 4;
    for (int rp = 0; rp < ntiles; rp += 4 * RT_MAX) {
        // this wave's row tiles in this pass: rp + wave + 4*i
        bf16x8 qf[RT_MAX][4];
        int lim[RT_MAX];
        float m[RT_MAX], l[RT_MAX];
        f32x4 o[RT_MAX][8];
        bool act[RT_MAX];
#pragma unroll
        for (int i = 0; i < RT_MAX; ++i) {
            const int tile = rp + wave + 4 * i;
            act[i] = tile < ntiles;
            const int row = tile * 16 + lr;
            const bool ok = act[i] && row < R;
            const int j = ok ? row / G : 0, hh = ok ? row % G : 0;
            const bf16_t* qs = p.q + ((size_t)(tbase + j) * p.hq + g * G + hh) * HD + 8 * lg;
#pragma unroll
            for (int ds = 0; ds < 4; ++ds) qf[i][ds] = ok ? *(const bf16x8*)(qs + ds * 32) : bf16x8{};
            lim[i] = prefix + j;
            m[i] = -INFINITY;
            l[i] = 0.f;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) o[i][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }

        auto compute = [&](int buf, int blk) {
            const int t0 = c0 + blk * 32;
            const uint4* kb = kvs[buf];
            const uint4* vb = kvs[buf] + 512;
#pragma unroll
            for (int i = 0; i < RT_MAX; ++i) {
                if (!act[i]) continue;
                f32x4 sa = f32x4{0.f, 0.f, 0.f, 0.f}, sb = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ds = 0; ds < 4; ++ds) {
                    const bf16x8 ka = __builtin_bit_cast(bf16x8, kb[(0 * 4 + ds) * 64 + lane]);
                    const bf16x8 kk = __builtin_bit_cast(bf16x8, kb[(1 * 4 + ds) * 64 + lane]);
                    sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[i][ds], sa, 0, 0, 0);
                    sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qf[i][ds], sb, 0, 0, 0);
                }
                // lane holds the scores of its query row at tokens t0 + 8*lg + e
                float sc[8];
                float bm = -INFINITY;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int tok = t0 + 8 * lg + e;
                    const float v = e < 4 ? sa[e] : sb[e - 4];
                    sc[e] = (tok < c1 && tok <= lim[i]) ? v * p.scale_log2 : -INFINITY;
                    bm = fmaxf(bm, sc[e]);
                }
                bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
                bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
                const float mn = fmaxf(m[i], bm);
                const bool live = mn != -INFINITY;  // something visible for this row
                const float alpha = live ? exp2f(m[i] - mn) : 1.f;
                float rs = 0.f;
                bf16x8 pb;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float pe = live ? exp2f(sc[e] - mn) : 0.f;
                    rs += pe;
                    pb[e] = (__bf16)pe;
                }
                rs += __shfl_xor(rs, 16, 64);
                rs += __shfl_xor(rs, 32, 64);
                l[i] = l[i] * alpha + rs;
                m[i] = live ? mn : m[i];
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) {
                    const bf16x8 vf = __builtin_bit_cast(bf16x8, vb[dt * 64 + lane]);
                    o[i][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb, o[i][dt] * alpha, 0, 0, 0);
                }
            }
        };

        // ping-pong over blocks: prefetch block k+1 while computing block k;
        // the prefetch index is clamped so the loads stay unconditional
        const int last = nblk - 1;
        load_blk(0);
        store_blk(0);
        __syncthreads();
        for (int k = 0; k < nblk; k += 2) {
            load_blk(min(k + 1, last));
            __builtin_amdgcn_sched_barrier(0);
            compute(0, k);
            __builtin_amdgcn_sched_barrier(0);
            store_blk(1);
            __syncthreads();
            if (k + 1 >= nblk) break;
            load_blk(min(k + 2, last));
            __builtin_amdgcn_sched_barrier(0);
            compute(1, k + 1);
            __builtin_amdgcn_sched_barrier(0);
            store_blk(0);
            __syncthreads();
        }

        // partial of this item: lane holds O^T[d = dt*16 + 4*lg + r][row lr]
#pragma unroll
        for (int i = 0; i < RT_MAX; ++i) {
            if (!act[i]) continue;
            const int row = (rp + wave + 4 * i) * 16 + lr;
            if (row >= R) continue;
            const size_t pr = (size_t)item * p.bv.rows_max + row;
            if (lg == 0) {
                p.aml[pr * 2 + 0] = m[i];
                p.aml[pr * 2 + 1] = l[i];
            }
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
                *(f32x4*)(p.apart + pr * HD + dt * 16 + 4 * lg) = o[i][dt];
        }
        __syncthreads();  // the LDS buffers are reused by the next row pass
    }
}

// Merge the partials of the chunks of (b, g) for one query row in chunk
// order; one wave per (slot, query head).
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
    const int p0 = i0 + g * nch, p1 = p0 + nch;
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
    hipLaunchKernelGGL(k_attn_bf16, dim3(bv.n_items), dim3(256), 0, s, p);
    hipLaunchKernelGGL(k_attn_combine<bf16_t>, dim3(blocks), dim3(256), 0, s, bv, sb.apart, sb.aml,
                       (bf16_t*)sb.attn, D.hq, D.hkv, D.hd);
}

}  // namespace sdv
