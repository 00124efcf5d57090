// Accept/reject and resampling over the full vocabulary (DiP-SD Sec. II-A,
// step 2: stop at the first rejected draft, emit one bonus or corrected
// token).  Two kernels, both split over vocab chunks so that every row is
// read by many workgroups at once:
//   phase A, per query slot: row max, sum of exp(z - max) and argmax (lowest
//     index on ties) per vocab chunk -- or, in the verify pass of the bf16
//     configuration, per lm_head workgroup, written by the lm_head
//     epilogue together with the logit of the slot's next draft, so the
//     logits need not be read back; a second kernel merges the partials of
//     a slot in a fixed order and takes the slot's accept decision:
//     greedy: draft == argmax; stochastic: u < p(d)/q(d) as an fp32
//     division, u from the caller or from Philox;
//   phase B, per user: a = number of leading accepts; greedy/force emit the
//     argmax of slot a (force: slot l); stochastic runs an exponential race
//     argmax_k w_k / E_k with w = max(0, p - q) at slot a (p itself when all
//     drafts passed, or when the residual is empty), E_k unit exponentials
//     from Philox keyed by (round, user, slot, k).  Chunk winners are merged
//     in chunk order (ties to the lowest index) by a second kernel.
// Merges run in separate launches (stream order makes the partials visible),
// so no device-scope fence is needed.
#include "sdv_device.h"
#include "sdv_internal.h"

namespace sdv {
static_assert(kVocabChunks <= 64, "chunk partials are merged by one wave");

struct SampP {
    BatchView bv;
    const float* logits;  // [T][V]
    int V, cw;            // vocab, chunk width (multiple of 4)
    float* sstat;         // [T][4]
    float* spartA;        // [T][kVocabChunks][4]
    float* spartB;        // [B][kVocabChunks][4]
    int32_t* result;      // n_acc [Bmax], token [Bmax], flags
    int bmax;
    // statistics of the lm_head epilogue: groups partials per slot
    // ([groups][T]) and the logit of each slot's next draft
    const VStat* lstat;
    const float* zd;
    int groups;
};

// A1: per (slot, vocab chunk): max, sum of exp(z - max), argmax (lowest index)
__global__ __launch_bounds__(256) void k_samp_a1(SampP p) {
    __shared__ float sm[4], ss[4], sv[4];
    __shared__ int si[4];
    const int t = blockIdx.x, c = blockIdx.y;
    const float* z = p.logits + (size_t)t * p.V;
    const int k0 = c * p.cw, k1 = min(p.V, k0 + p.cw);
    float m = -INFINITY, s = 0.f, bv = -INFINITY;
    int bi = 0x7fffffff;
    auto add = [&](float v, int k) {
        if (v > bv) { bv = v; bi = k; }  // increasing k per thread: first max kept
        if (v > m) { s = (m == -INFINITY ? 0.f : s * expf(m - v)) + 1.f; m = v; }
        else if (v != -INFINITY) s += expf(v - m);
    };
    if ((p.V & 3) == 0) {
        // four float4 loads per thread in flight, then the elements in
        // increasing k order (chunk bounds are multiples of 4)
        for (int k4 = k0 + 4 * threadIdx.x; k4 < k1; k4 += 4 * 1024) {
            float4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int k = k4 + u * 1024;
                v[u] = k < k1 ? *(const float4*)(z + k) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int k = k4 + u * 1024;
                if (k < k1) {
                    add(v[u].x, k);
                    add(v[u].y, k + 1);
                    add(v[u].z, k + 2);
                    add(v[u].w, k + 3);
                }
            }
        }
    } else {
        for (int k = k0 + threadIdx.x; k < k1; k += 256) add(z[k], k);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float m2 = __shfl_xor(m, o, 64), s2 = __shfl_xor(s, o, 64);
        merge_ms(m, s, m2, s2);
        const float v2 = __shfl_xor(bv, o, 64);
        const int i2 = __shfl_xor(bi, o, 64);
        if (v2 > bv || (v2 == bv && i2 < bi)) { bv = v2; bi = i2; }
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) { sm[w] = m; ss[w] = s; sv[w] = bv; si[w] = bi; }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int i = 1; i < 4; ++i) {
            merge_ms(m, s, sm[i], ss[i]);
            if (sv[i] > bv || (sv[i] == bv && si[i] < bi)) { bv = sv[i]; bi = si[i]; }
        }
        float* dst = p.spartA + ((size_t)t * kVocabChunks + c) * 4;
        dst[0] = m; dst[1] = s; dst[2] = bv; dst[3] = __int_as_float(bi);
    }
}

// A2: merge a slot's partials and take its accept decision for the draft
// that follows it.  Unfused: one wave per slot, lane i holding vocab chunk
// i's partial.  FUSED: one workgroup per slot over the lm_head workgroups'
// records ([T][groups]); thread i merges records i, i + 256, ... in that
// order, then the lanes and the four waves are merged.  Ties of the argmax
// go to the lowest index either way.
template <bool FUSED>
__global__ __launch_bounds__(256) void k_samp_a2(SampP p, int chunks) {
    __shared__ VStat wst[4];
    const int lane = threadIdx.x & 63;
    const BatchView& bv = p.bv;
    int t;
    float M = -INFINITY, S = 0.f;
    int BI = 0x7fffffff;
    if (FUSED) {
        t = blockIdx.x;
        const VStat* rec = p.lstat + (size_t)t * p.groups;
        VStat a = vstat_empty();
        for (int g0 = 0; g0 < p.groups; g0 += 4 * 256) {
            VStat r[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int g = g0 + (int)threadIdx.x + u * 256;
                r[u] = g < p.groups ? rec[g] : vstat_empty();
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) a = vstat_merge(a, r[u]);
        }
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) a = vstat_merge(a, vstat_shfl_xor(a, o));
        if (lane == 0) wst[threadIdx.x >> 6] = a;
        __syncthreads();
        if (threadIdx.x >= 64) return;
        a = wst[0];
#pragma unroll
        for (int w = 1; w < 4; ++w) a = vstat_merge(a, wst[w]);
        M = a.m; S = a.s; BI = a.i;
    } else {
        t = blockIdx.x * 4 + (threadIdx.x >> 6);
        if (t >= bv.T) return;
        float BV = -INFINITY;
        if (lane < chunks) {
            const float4 e = *(const float4*)(p.spartA + ((size_t)t * kVocabChunks + lane) * 4);
            M = e.x; S = e.y; BV = e.z; BI = __float_as_int(e.w);
        }
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const float m2 = __shfl_xor(M, o, 64), s2 = __shfl_xor(S, o, 64);
            const float v2 = __shfl_xor(BV, o, 64);
            const int i2 = __shfl_xor(BI, o, 64);
            merge_ms(M, S, m2, s2);
            if (v2 > BV || (v2 == BV && i2 < BI)) { BV = v2; BI = i2; }
        }
    }
    if (BI == 0x7fffffff) BI = 0;  // a row of -inf logits only
    const int b = bv.slot_b[t], j = bv.slot_j[t];
    // sparse q: q(d) of the draft that follows this slot, looked up by the
    // whole wave (token ids of a row are distinct, so at most one lane hits)
    float qsp = -1.f;
    if (bv.qk > 0 && bv.mode == 1 && j < bv.L[b]) {
        const int di = bv.draft_off[b] + j;
        const int d = bv.drafts[di];
        for (int e = lane; e < bv.qk; e += 64)
            if (bv.q_idx[(size_t)di * bv.qk + e] == d) qsp = bv.q_val[(size_t)di * bv.qk + e];
        qsp = wave_max(qsp);
        if (qsp < 0.f) qsp = bv.q_rest[di];
    }
    if (lane != 0) return;
    float acc = 0.f;
    if (j < bv.L[b]) {
        const int di = bv.draft_off[b] + j;
        int d = bv.drafts[di];
        if (d < 0 || d >= p.V) d = 0;  // flagged by the prepare kernel
        if (bv.mode == 0) acc = (d == BI) ? 1.f : 0.f;
        else if (bv.mode == 2) acc = 1.f;
        else {
            const float zdv = FUSED ? p.zd[t] : p.logits[(size_t)t * p.V + d];
            const float pd = expf(zdv - M) / S;
            const float qd = bv.qk > 0 ? qsp : bv.q[(size_t)di * p.V + d];
            const float r = pd / qd;
            float u;
            if (bv.accept_u) u = bv.accept_u[di];
            else {
                const u64x4 ctr = {bv.round, (uint64_t)bv.user_id[b],
                                   ((uint64_t)PURPOSE_ACCEPT << 32) | (uint64_t)j, 0ull};
                u = accept_uniform(philox4x64_10(ctr, bv.seed, 0ull).x);
            }
            acc = (u < r) ? 1.f : 0.f;
        }
    }
    float* st4 = p.sstat + (size_t)t * 4;
    st4[0] = M; st4[1] = S; st4[2] = __int_as_float(BI); st4[3] = acc;
}

__device__ __forceinline__ int leading_accepts(const SampP& p, int b) {
    const int Lb = p.bv.L[b], so = p.bv.slot_off[b];
    if (p.bv.mode == 2) return Lb;
    int a = 0;
    while (a < Lb && p.sstat[(size_t)(so + a) * 4 + 3] != 0.f) ++a;
    return a;
}

// B1 (stochastic): per (user, vocab chunk): best race keys of the residual
// max(0, p - q) at the stop slot and of p itself (the bonus draw, and the
// fallback when the residual is empty); both use the same unit exponentials
template <bool SPARSE>
__global__ __launch_bounds__(256) void k_samp_b1(SampP p) {
    __shared__ float sk[2][4];
    __shared__ int sidx[2][4];
    __shared__ float qloc[SPARSE ? kSparseChunkMax : 1];  // sparse q over this chunk
    const int b = blockIdx.x, c = blockIdx.y;
    const BatchView& bv = p.bv;
    const int Lb = bv.L[b];
    const int a = leading_accepts(p, b);
    const int row = bv.slot_off[b] + a;
    const float* st4 = p.sstat + (size_t)row * 4;
    const float M = st4[0], S = st4[1];
    const float* z = p.logits + (size_t)row * p.V;
    const bool resid = a < Lb;
    const int k0 = c * p.cw, k1 = min(p.V, k0 + p.cw);
    const float* qr = nullptr;
    if (SPARSE) {
        // the stop slot's q on [k0, k1): the remainder probability, then the
        // listed tokens that fall into the chunk
        if (resid) {
            const size_t di = (size_t)bv.draft_off[b] + a;
            const float rest = bv.q_rest[di];
            for (int k = threadIdx.x; k < k1 - k0; k += 256) qloc[k] = rest;
            __syncthreads();
            for (int e = threadIdx.x; e < bv.qk; e += 256) {
                const int tk = bv.q_idx[di * bv.qk + e];
                if (tk >= k0 && tk < k1) qloc[tk - k0] = bv.q_val[di * bv.qk + e];
            }
            __syncthreads();
        }
    } else {
        qr = resid ? bv.q + (size_t)(bv.draft_off[b] + a) * p.V : nullptr;
    }
    const uint64_t user = (uint64_t)bv.user_id[b];
    float br = -1.f, bp = -1.f;
    int ir = 0x7fffffff, ip = 0x7fffffff;
    for (int k4 = k0 + 4 * threadIdx.x; k4 < k1; k4 += 4 * 256) {
        const u64x4 ctr = {bv.round, user, ((uint64_t)PURPOSE_RACE << 32) | (uint64_t)a,
                           (uint64_t)(k4 >> 2)};
        const u64x4 rnd = philox4x64_10(ctr, bv.seed, 0ull);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int k = k4 + e;
            if (k >= k1) break;
            const float pk = expf(z[k] - M) / S;
            const float E = race_exponential(word_of(rnd, e));
            if (pk > 0.f) {
                const float kp = pk / E;
                if (kp > bp) { bp = kp; ip = k; }
            }
            if (resid) {
                const float wk = fmaxf(pk - (SPARSE ? qloc[k - k0] : qr[k]), 0.f);
                if (wk > 0.f) {
                    const float kr = wk / E;
                    if (kr > br) { br = kr; ir = k; }
                }
            }
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float b2 = __shfl_xor(br, o, 64);
        const int i2 = __shfl_xor(ir, o, 64);
        if (b2 > br || (b2 == br && i2 < ir)) { br = b2; ir = i2; }
        const float p2 = __shfl_xor(bp, o, 64);
        const int j2 = __shfl_xor(ip, o, 64);
        if (p2 > bp || (p2 == bp && j2 < ip)) { bp = p2; ip = j2; }
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) { sk[0][w] = br; sidx[0][w] = ir; sk[1][w] = bp; sidx[1][w] = ip; }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int i = 1; i < 4; ++i) {
            if (sk[0][i] > br || (sk[0][i] == br && sidx[0][i] < ir)) { br = sk[0][i]; ir = sidx[0][i]; }
            if (sk[1][i] > bp || (sk[1][i] == bp && sidx[1][i] < ip)) { bp = sk[1][i]; ip = sidx[1][i]; }
        }
        float* dst = p.spartB + ((size_t)b * kVocabChunks + c) * 4;
        dst[0] = br; dst[1] = __int_as_float(ir); dst[2] = bp; dst[3] = __int_as_float(ip);
    }
}

// B2: one thread per user: the stop slot a, then the token -- argmax of that
// slot (greedy / force), or the race winner merged over chunks in chunk
// order (ties to the lowest index)
__global__ __launch_bounds__(256) void k_samp_b2(SampP p, int chunks) {
    const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const BatchView& bv = p.bv;
    if (b == 0 && lane == 0) p.result[2 * p.bmax] = *bv.flags;
    if (b >= bv.B) return;
    const int a = leading_accepts(p, b);
    int tok;
    if (bv.mode != 1) {
        tok = __float_as_int(p.sstat[(size_t)(bv.slot_off[b] + a) * 4 + 2]);
    } else {
        // lane i holds chunk i's two race winners; the best key wins, ties to
        // the lowest token index (the chunk-order result)
        float BR = -1.f, BP = -1.f;
        int IR = 0x7fffffff, IP = 0x7fffffff;
        if (lane < chunks) {
            const float4 e = *(const float4*)(p.spartB + ((size_t)b * kVocabChunks + lane) * 4);
            BR = e.x; IR = __float_as_int(e.y); BP = e.z; IP = __float_as_int(e.w);
        }
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const float r2 = __shfl_xor(BR, o, 64), p2 = __shfl_xor(BP, o, 64);
            const int ir2 = __shfl_xor(IR, o, 64), ip2 = __shfl_xor(IP, o, 64);
            if (r2 > BR || (r2 == BR && ir2 < IR)) { BR = r2; IR = ir2; }
            if (p2 > BP || (p2 == BP && ip2 < IP)) { BP = p2; IP = ip2; }
        }
        tok = (a < bv.L[b] && BR > 0.f) ? IR : IP;
    }
    if (lane != 0) return;
    p.result[b] = a;
    p.result[p.bmax + b] = tok;
}

// Decode-step output: the target distribution p of every slot, written
// with the expression phase B's race evaluates, so a token drawn by the
// race is a draw from exactly these rows.  One thread per four entries.
__global__ __launch_bounds__(256) void k_probs(BatchView bv, const float* logits, const float* sstat,
                                               float* probs, int V) {
    const int t = blockIdx.y;
    const int k = (blockIdx.x * 256 + threadIdx.x) * 4;
    if (k >= V) return;
    const float M = sstat[(size_t)t * 4 + 0], S = sstat[(size_t)t * 4 + 1];
    const float* z = logits + (size_t)t * V;
    float* o = probs + (size_t)bv.prow[bv.slot_b[t]] * V;
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if (k + e < V) o[k + e] = expf(z[k + e] - M) / S;
}

void launch_probs(const Dims& D, const BatchView& bv, const SlotBufs& sb, const float* logits,
                  float* probs, hipStream_t s) {
    const int blocks = ((D.V + 3) / 4 + 255) / 256;
    hipLaunchKernelGGL(k_probs, dim3(blocks, bv.T), dim3(256), 0, s, bv, logits, sb.sstat, probs, D.V);
}

// Batch tables of the context-free sampler call, built on the device from
// the kernel argument (nothing is copied from the host): user ids and draft
// lengths as given, slot and draft offsets, the (user, slot) of every slot;
// the error flags are cleared and every draft token is range-checked.  One
// workgroup of 1024 threads.
__global__ __launch_bounds__(1024) void k_noalloc_stage(NoallocMeta m, NoallocTables t,
                                                        const int32_t* drafts) {
    const int tid = threadIdx.x;
    if (tid < m.B) {
        t.user_id[tid] = m.user_id[tid];
        t.L[tid] = m.L[tid];
    }
    if (tid == 0) {
        int so = 0, dof = 0;
        for (int b = 0; b < m.B; ++b) {
            t.slot_off[b] = so;
            t.draft_off[b] = dof;
            so += m.L[b] + 1;
            dof += m.L[b];
        }
        t.slot_off[m.B] = so;
        t.draft_off[m.B] = dof;
        *t.flags = 0;
    }
    __syncthreads();
    const int T = t.slot_off[m.B], nd = t.draft_off[m.B];
    for (int i = tid; i < T; i += blockDim.x) {
        int b = 0;
        while (t.slot_off[b + 1] <= i) ++b;
        t.slot_b[i] = b;
        t.slot_j[i] = i - t.slot_off[b];
    }
    __syncthreads();  // flags cleared above before any thread sets a bit
    for (int i = tid; i < nd; i += blockDim.x) {
        const int d = drafts[i];
        if (d < 0 || d >= m.V) atomicOr(t.flags, 1);
    }
}

void launch_noalloc_stage(const NoallocMeta& m, const NoallocTables& t, const int32_t* drafts,
                          hipStream_t s) {
    hipLaunchKernelGGL(k_noalloc_stage, dim3(1), dim3(1024), 0, s, m, t, drafts);
}

void launch_sampler(const Dims& D, const BatchView& bv, const SlotBufs& sb, const float* logits,
                    hipStream_t s, int groups) {
    SampP p;
    p.bv = bv;
    p.logits = logits;
    p.V = D.V;
    p.cw = ((D.V + kVocabChunks - 1) / kVocabChunks + 3) & ~3;
    p.sstat = sb.sstat;
    p.spartA = sb.spart;
    p.spartB = sb.spartB;
    p.result = sb.result;
    p.bmax = sb.bmax;
    p.lstat = reinterpret_cast<const VStat*>(sb.lstat);
    p.zd = sb.zd;
    p.groups = groups;
    const int chunks = (D.V + p.cw - 1) / p.cw;
    if (groups > 0) {
        hipLaunchKernelGGL(k_samp_a2<true>, dim3(bv.T), dim3(256), 0, s, p, chunks);
    } else {
        hipLaunchKernelGGL(k_samp_a1, dim3(bv.T, chunks), dim3(256), 0, s, p);
        hipLaunchKernelGGL(k_samp_a2<false>, dim3((bv.T + 3) / 4), dim3(256), 0, s, p, chunks);
    }
    if (bv.mode == 1) {
        if (bv.qk > 0)
            hipLaunchKernelGGL(k_samp_b1<true>, dim3(bv.B, chunks), dim3(256), 0, s, p);
        else
            hipLaunchKernelGGL(k_samp_b1<false>, dim3(bv.B, chunks), dim3(256), 0, s, p);
    }
    hipLaunchKernelGGL(k_samp_b2, dim3((bv.B + 3) / 4), dim3(256), 0, s, p, chunks);
}

}  // namespace sdv
