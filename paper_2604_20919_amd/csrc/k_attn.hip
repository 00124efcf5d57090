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
// with direct global-to-LDS loads (one buffer resource over the layer's
// pages, 32-bit offsets) into a ring of LDS buffers, so the next block is in
// flight while one is multiplied, without staging registers.  The block's
// fragments are read from LDS by ds_read instructions issued in inline
// assembly: for reads the compiler sees, it cannot tell a ring buffer from
// the one being loaded and waits for every direct-to-LDS load in flight,
// which leaves nothing in flight during the products (C4 attention 6.1 ->
// 5.5 ms per step); their completion is waited for explicitly.  Each lane
// gathers the piece that belongs to its LDS slot, which leaves the block in
// MFMA fragment order: every operand read is one contiguous 1 KB wave read.
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
    const bf16_t* q;   // [2][T][hq][hd]: hi and lo planes
    KVPool kv;
    int layer;
    int hq, hkv, G;
    float scale_log2;  // log2(e) / sqrt(hd)
    float* apart;      // [items][rows_max][hd]
    float* aml;        // [items][rows_max][2]
};

constexpr int HD = 128;
constexpr int RT_MAX = 2;  // row tiles per wave and pass

// Gather map of the direct-to-LDS block loads.  A block is 32 tokens (two
// pages) of K and V for one KV head, 16 KB, held in LDS as 1024 16-byte
// slots in MFMA fragment order: K slots 0..511, V^T slots 512..1023.  Slot
// s is filled by thread s % 256 of load instruction s / 256, and since a
// wave's direct load writes its 64 lanes to 64 consecutive slots, each lane
// gathers the global piece that belongs to its slot:
//   K slot s: fragment q = s/64 (token half tt = q/4, dim step ds = q%4),
//     lane r = s%64 (lr = r%16, lg = r/16) holds token
//     t = 8*(lr/4) + 4*tt + lr%4 of the block, dims 32*ds + 8*lg .. +7;
//     this token order makes each lane of S^T = K Q^T end up with 8
//     consecutive tokens of one query row (the B layout of O^T += V^T P^T);
//   V slot s: dim tile dt = s/64, r = s%64: dim 16*dt + r%16, tokens
//     8*(r/16 % 2) .. +7 of page r/32 (V pages are dim-major, so this is
//     16 contiguous bytes).
// Returns the page (0/1) of the block and the byte offset inside that
// page's K or V block.
__device__ __forceinline__ void k_slot_src(int s, int& pg, int& off) {
    const int q = s >> 6, r = s & 63;
    const int tt = q >> 2, ds = q & 3, lr = r & 15, lg = r >> 4;
    const int t = 8 * (lr >> 2) + 4 * tt + (lr & 3);
    pg = t >> 4;
    off = ((t & 15) * HD + 32 * ds + 8 * lg) * 2;
}
__device__ __forceinline__ void v_slot_src(int s, int& pg, int& off) {
    const int dt = s >> 6, r = s & 63;
    const int d = 16 * dt + (r & 15), x = r >> 4;
    pg = x >> 1;
    off = (d * kPageTokens + 8 * (x & 1)) * 2;
}

typedef __attribute__((address_space(4))) const int32_t cint32_t;

// Reductions over the four lanes l, l^16, l^32, l^48 that hold one query
// row: each cross-lane swap returns the row halves exchanged between its two
// operands, so combining both results with the own value pairs every lane
// with its partner 16 (then 32) lanes away.
__device__ __forceinline__ float row_max4(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float row_sum4(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Eight 16-byte LDS reads of consecutive 1 KB fragments starting at LDS
// byte address `a` (this lane's slot), issued without a wait.
__device__ __forceinline__ void lds_read8(bf16x8 (&f)[8], uint32_t a) {
    asm volatile(
        "ds_read_b128 %0, %8\n\t"
        "ds_read_b128 %1, %8 offset:1024\n\t"
        "ds_read_b128 %2, %8 offset:2048\n\t"
        "ds_read_b128 %3, %8 offset:3072\n\t"
        "ds_read_b128 %4, %8 offset:4096\n\t"
        "ds_read_b128 %5, %8 offset:5120\n\t"
        "ds_read_b128 %6, %8 offset:6144\n\t"
        "ds_read_b128 %7, %8 offset:7168"
        : "=&v"(f[0]), "=&v"(f[1]), "=&v"(f[2]), "=&v"(f[3]), "=&v"(f[4]), "=&v"(f[5]), "=&v"(f[6]),
          "=&v"(f[7])
        : "v"(a)
        : "memory");
}

// Per-item constants of the ring and the per-pass state of a wave's row tiles.
struct AttnItem {
    int c0, c1, nblk, prefix, wave, lane, lg, g;
    const cint32_t* pt;
    int kpg0, koff0, kpg1, koff1, vpg0, voff0, vpg1, voff1;  // this thread's gather sources
};
struct AttnState {
    bf16x8 qf[RT_MAX][4], ql[RT_MAX][4];  // query hi / lo planes
    int lim[RT_MAX];
    float m[RT_MAX], l[RT_MAX];
    f32x4 o[RT_MAX][8];
    bool act[RT_MAX];
};

// The chunk's blocks through the LDS ring (buffers r0..r3) for one pass of
// row tiles.
template <int NBUF>
__device__ __forceinline__ void attn_ring(const AttnP& p, const AttnItem& ac, AttnState& st, uint4* r0,
                                          uint4* r1, uint4* r2, uint4* r3) {
    constexpr int PD = NBUF - 1;  // blocks in flight
    static_assert(NBUF >= 2 && NBUF <= 4, "the ring's tail waits cover up to three blocks in flight");
    const int c0 = ac.c0, c1 = ac.c1, nblk = ac.nblk, prefix = ac.prefix, wave = ac.wave;
    const int lane = ac.lane, lg = ac.lg, g = ac.g;
    const int kpg0 = ac.kpg0, koff0 = ac.koff0, kpg1 = ac.kpg1, koff1 = ac.koff1;
    const int vpg0 = ac.vpg0, voff0 = ac.voff0, vpg1 = ac.vpg1, voff1 = ac.voff1;
    const cint32_t* pt = ac.pt;
    auto& qf = st.qf;
    auto& ql = st.ql;
    auto& lim = st.lim;
    auto& m = st.m;
    auto& l = st.l;
    auto& o = st.o;
    auto& act = st.act;
    // One buffer resource over this layer's pages (the host keeps a layer's
    // pages below 4 GB); per lane a 32-bit offset: page * page bytes + the
    // KV head's block + the piece.
    const uint32_t page_bytes = (uint32_t)(p.kv.page_elems() * 2);
    const uint32_t gk = (uint32_t)(p.kv.k_off(0, 0, g) * 2);  // K block of head g
    const uint32_t gv = (uint32_t)(p.kv.v_off(0, 0, g) * 2);  // V block of head g
    const __amdgpu_buffer_rsrc_t kres = __builtin_amdgcn_make_buffer_rsrc(
        (void*)((const char*)p.kv.base + p.kv.k_off(p.layer, 0, 0) * 2), (short)0,
        (int)(uint32_t)((uint64_t)p.kv.n_pages * page_bytes), 0x00020000);
    typedef __attribute__((address_space(3))) void lds_void;
    // Requests block blk into LDS buffer buf: four 16-byte direct loads per
    // thread.  Tokens past the chunk end are read from the chunk's last page
    // (the page index is clamped); their scores are masked, and V there is
    // finite (pool zeroed at init, later only model values), so p = 0
    // contributes exactly 0.
    auto issue = [&](int blk, uint4* buf) __attribute__((always_inline)) {
        const int t0 = c0 + blk * 32;
        const uint32_t pb0 = (uint32_t)pt[min(t0, c1 - 1) >> 4] * page_bytes;
        const uint32_t pb1 = (uint32_t)pt[min(t0 + 16, c1 - 1) >> 4] * page_bytes;
        uint4* dst = buf + wave * 64;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(kres, (lds_void*)dst, 16, (int)((kpg0 ? pb1 : pb0) + gk + koff0), 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(kres, (lds_void*)(dst + 256), 16, (int)((kpg1 ? pb1 : pb0) + gk + koff1), 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(kres, (lds_void*)(dst + 512), 16, (int)((vpg0 ? pb1 : pb0) + gv + voff0), 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(kres, (lds_void*)(dst + 768), 16, (int)((vpg1 ? pb1 : pb0) + gv + voff1), 0, 0, 0);
    };

        // One 32-token block for this wave's row tiles.  Scores stay in the
    // raw (unscaled) domain until the exponent, which folds the scale in:
    // p = 2^(s*c - m*c) with c = log2(e)/sqrt(hd).  Blocks that every
    // row sees completely skip the causal/chunk mask; the running output
    // is rescaled only when some row's maximum grew; the row sum stays
    // per lane until the end of the chunk.
    auto compute = [&](const uint4* buf, int blk) __attribute__((always_inline)) {
        const int t0 = c0 + blk * 32;
        const bool full = t0 + 32 <= c1 && t0 + 31 <= prefix;
        // The block's 16 fragments (8 K, 8 V^T; shared by the wave's row
        // tiles) are read by ds_read instructions the compiler does not see:
        // it cannot tell these reads apart from the direct-to-LDS loads into
        // the other ring buffers and would make them wait for every load in
        // flight.  The reads' completion is waited for explicitly below (the
        // waits take the fragments as operands, so nothing that uses a
        // fragment can be scheduled before its wait).
        bf16x8 kfr[8], vfr[8];
        const uint32_t la = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint4*)buf + lane * 16u;
        lds_read8(kfr, la);
        lds_read8(vfr, la + 512u * 16u);
        asm volatile("s_waitcnt lgkmcnt(8)"
                     : "+v"(kfr[0]), "+v"(kfr[1]), "+v"(kfr[2]), "+v"(kfr[3]), "+v"(kfr[4]),
                       "+v"(kfr[5]), "+v"(kfr[6]), "+v"(kfr[7]));
#pragma unroll
        for (int i = 0; i < RT_MAX; ++i) {
            if (!act[i]) continue;
            // S^T = K (Q_hi + Q_lo)^T
            f32x4 sa = f32x4{0.f, 0.f, 0.f, 0.f}, sb = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ds = 0; ds < 4; ++ds) {
                const bf16x8 ka = kfr[ds];
                const bf16x8 kk = kfr[4 + ds];
                sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[i][ds], sa, 0, 0, 0);
                sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, ql[i][ds], sa, 0, 0, 0);
                sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qf[i][ds], sb, 0, 0, 0);
                sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, ql[i][ds], sb, 0, 0, 0);
            }
            // lane holds the scores of its query row at tokens t0 + 8*lg + e
            float sc[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                sc[e] = sa[e];
                sc[4 + e] = sb[e];
            }
            if (!full) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int tok = t0 + 8 * lg + e;
                    sc[e] = (tok < c1 && tok <= lim[i]) ? sc[e] : -INFINITY;
                }
            }
            float bm = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                             fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
            bm = row_max4(bm);
            const float mn = fmaxf(m[i], bm);
            const bool live = mn != -INFINITY;  // something visible for this row
            const float ms = live ? mn * p.scale_log2 : 0.f;
            const float alpha = live ? __builtin_amdgcn_exp2f((m[i] - mn) * p.scale_log2) : 1.f;
            // P as hi + lo bf16 pair (about 16 significant bits)
            float rs = 0.f;
            bf16x8 pb, pl;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float pe = __builtin_amdgcn_exp2f(fmaf(sc[e], p.scale_log2, -ms));
                rs += pe;
                pb[e] = (__bf16)pe;
                pl[e] = (__bf16)(pe - (float)pb[e]);
            }
            l[i] = fmaf(l[i], alpha, rs);
            m[i] = mn;
            if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) o[i][dt] *= alpha;
            }
            if (i == 0)
                asm volatile("s_waitcnt lgkmcnt(0)"
                             : "+v"(vfr[0]), "+v"(vfr[1]), "+v"(vfr[2]), "+v"(vfr[3]), "+v"(vfr[4]),
                               "+v"(vfr[5]), "+v"(vfr[6]), "+v"(vfr[7]));
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) {
                const bf16x8 vf = vfr[dt];
                o[i][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb, o[i][dt], 0, 0, 0);
                o[i][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl, o[i][dt], 0, 0, 0);
            }
        }
    };

    // Ring pipeline over NBUF LDS buffers.  Iteration k waits for its own
    // loads of block k (the loads of the blocks issued after it may stay
    // in flight: 4*(PD-1), or 4*(last-k) in the tail) and its LDS reads,
    // then a barrier makes every wave's loads of block k visible and
    // retires every wave's reads of block k-1, whose buffer then
    // receives block k+PD while there is one.  Loads retire in issue
    // order, so the counts are exact; the prologue clamps its block
    // indices (a chunk shorter than PD blocks re-reads its last one,
    // which only makes the waits stricter).
    const int last = nblk - 1;
#pragma unroll
    for (int u = 0; u < PD; ++u) issue(min(u, last), u == 0 ? r0 : u == 1 ? r1 : r2);
    for (int k0 = 0; k0 < nblk; k0 += NBUF) {
#pragma unroll
        for (int u = 0; u < NBUF; ++u) {
            const int k = k0 + u;
            if (k >= nblk) break;
            if (k + PD <= last) {
                wait_vm<4 * (PD - 1), true>();
                barrier_nofence();
                const int nb = (u + PD) % NBUF;
                issue(k + PD, nb == 0 ? r0 : nb == 1 ? r1 : nb == 2 ? r2 : r3);
            } else {
                // tail: blocks k..last are the only ones in flight
                if (last - k >= 2) wait_vm<8, true>();
                else if (last - k == 1) wait_vm<4, true>();
                else wait_vm<0, true>();
                barrier_nofence();
            }
            compute(u == 0 ? r0 : u == 1 ? r1 : u == 2 ? r2 : r3, k);
        }
    }
    // drain the tail loads before the buffers are reused or released
    wait_vm<0>();

}

template <int NBUF>
__device__ __forceinline__ void attn_bf16_body(const AttnP& p, uint4* r0, uint4* r1, uint4* r2, uint4* r3) {
    // The batch metadata is read-only while the kernel runs: reading it
    // through the constant address space gives scalar loads, which keep the
    // vector memory counter (waited on below) free of anything but KV.
    const cint32_t* items = (const cint32_t*)p.bv.items;
    const int item = blockIdx.x;
    const int b = items[4 * item + 0], g = items[4 * item + 1];
    const int c0 = items[4 * item + 2], c1 = items[4 * item + 3];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int lr = lane & 15, lg = lane >> 4;
    const int G = p.G;
    const int R = (((const cint32_t*)p.bv.L)[b] + 1) * G;
    const int prefix = ((const cint32_t*)p.bv.prefix)[b];
    const int tbase = ((const cint32_t*)p.bv.slot_off)[b];
    const cint32_t* pt = (const cint32_t*)p.bv.page_table + (size_t)b * p.bv.max_pages;
    const int nblk = (c1 - c0 + 31) >> 5;

    // this thread's four gather sources (page of the block, byte offset)
    int kpg0, koff0, kpg1, koff1, vpg0, voff0, vpg1, voff1;
    k_slot_src(threadIdx.x, kpg0, koff0);
    k_slot_src(256 + threadIdx.x, kpg1, koff1);
    v_slot_src(threadIdx.x, vpg0, voff0);
    v_slot_src(256 + threadIdx.x, vpg1, voff1);
    AttnItem ac;
    ac.c0 = c0;
    ac.c1 = c1;
    ac.nblk = nblk;
    ac.prefix = prefix;
    ac.wave = wave;
    ac.lane = lane;
    ac.lg = lg;
    ac.g = g;
    ac.pt = pt;
    ac.kpg0 = kpg0; ac.koff0 = koff0; ac.kpg1 = kpg1; ac.koff1 = koff1;
    ac.vpg0 = vpg0; ac.voff0 = voff0; ac.vpg1 = vpg1; ac.voff1 = voff1;
    const int ntiles = (R + 15) >> 4;
    for (int rp = 0; rp < ntiles; rp += 4 * RT_MAX) {
        // this wave's row tiles in this pass: rp + wave + 4*i
        AttnState st;
        auto& qf = st.qf;  // query hi / lo planes
        auto& ql = st.ql;
        auto& lim = st.lim;
        auto& m = st.m;
        auto& l = st.l;
        auto& o = st.o;
        auto& act = st.act;
#pragma unroll
        for (int i = 0; i < RT_MAX; ++i) {
            const int tile = rp + wave + 4 * i;
            act[i] = tile < ntiles;
            const int row = tile * 16 + lr;
            const bool ok = act[i] && row < R;
            const int j = ok ? row / G : 0, hh = ok ? row % G : 0;
            const bf16_t* qs = p.q + ((size_t)(tbase + j) * p.hq + g * G + hh) * HD + 8 * lg;
            const size_t qpl = (size_t)p.bv.T * p.hq * HD;
#pragma unroll
            for (int ds = 0; ds < 4; ++ds) {
                qf[i][ds] = ok ? *(const bf16x8*)(qs + ds * 32) : bf16x8{};
                ql[i][ds] = ok ? *(const bf16x8*)(qs + qpl + ds * 32) : bf16x8{};
            }
            lim[i] = prefix + j;
            m[i] = -INFINITY;
            l[i] = 0.f;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) o[i][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        // the query loads must not be counted by the block waits below
        wait_vm<0>();

        attn_ring<NBUF>(p, ac, st, r0, r1, r2, r3);

        // partial of this item: lane holds O^T[d = dt*16 + 4*lg + r][row lr]
#pragma unroll
        for (int i = 0; i < RT_MAX; ++i) {
            if (!act[i]) continue;
            const int row = (rp + wave + 4 * i) * 16 + lr;
            const float lsum = row_sum4(l[i]);  // all lanes take part in the swaps
            if (row >= R) continue;
            const size_t pr = (size_t)item * p.bv.rows_max + row;
            if (lg == 0) {
                p.aml[pr * 2 + 0] = m[i] == -INFINITY ? -INFINITY : m[i] * p.scale_log2;
                p.aml[pr * 2 + 1] = lsum;
            }
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
                *(f32x4*)(p.apart + pr * HD + dt * 16 + 4 * lg) = o[i][dt];
        }
        __syncthreads();  // the LDS buffers are reused by the next row pass
    }
}

template <int NBUF>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_attn_bf16(AttnP p) {
    __shared__ __attribute__((aligned(16))) uint4 kv0[1024];
    __shared__ __attribute__((aligned(16))) uint4 kv1[1024];
    __shared__ __attribute__((aligned(16))) uint4 kv2[NBUF > 2 ? 1024 : 1];
    __shared__ __attribute__((aligned(16))) uint4 kv3[NBUF > 3 ? 1024 : 1];
    attn_bf16_body<NBUF>(p, kv0, kv1, kv2, kv3);
}

// Merge the partials of the chunks of (b, g) for one query row in chunk
// order; half a wave per (slot, query head), lane l of it holding dims
// 4l..4l+3 (16-byte partial loads, 8-byte stores of the two output planes).
// Chunks are taken eight at a time with all their loads issued before the
// merge (online maximum: the running sums are rescaled when a group raises
// it).
__global__ __launch_bounds__(256) void k_attn_combine(BatchView bv, const float* apart,
                                                      const float* aml, bf16_t* out, int hq, int hkv) {
    const int rid = blockIdx.x * 8 + (threadIdx.x >> 5);  // (slot, query head)
    const int l = threadIdx.x & 31;
    const int t = rid / hq, h = rid % hq;
    if (t >= bv.T) return;
    const int G = hq / hkv, g = h / G, hh = h % G;
    const int b = bv.slot_b[t], j = bv.slot_j[t];
    const int row = j * G + hh;
    const int i0 = bv.item_off[b], nch = (bv.item_off[b + 1] - i0) / hkv;
    const int p0 = i0 + g * nch, p1 = p0 + nch;
    float M = -INFINITY, Ls = 0.f;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int pg = p0; pg < p1; pg += 8) {
        float mi[8], li[8];
        f32x4 a[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const bool ok = pg + u < p1;
            const size_t pr = (size_t)(ok ? pg + u : p0) * bv.rows_max + row;
            mi[u] = ok ? aml[pr * 2] : -INFINITY;
            li[u] = ok ? aml[pr * 2 + 1] : 0.f;
            a[u] = ok ? *(const f32x4*)(apart + pr * HD + 4 * l) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        float mg = M;
#pragma unroll
        for (int u = 0; u < 8; ++u) mg = fmaxf(mg, mi[u]);
        if (mg == -INFINITY) continue;  // no key of these chunks is visible to the row
        const float sc = exp2f(M - mg);  // 0 while M is still -inf
        Ls *= sc;
        acc *= sc;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (mi[u] == -INFINITY) continue;
            const float w = exp2f(mi[u] - mg);
            Ls += li[u] * w;
            acc += a[u] * w;
        }
        M = mg;
    }
    const float inv = 1.0f / Ls;
    const float o[4] = {acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv};
    st_act4(out, (size_t)bv.T * hq * HD, ((size_t)t * hq + h) * HD + 4 * l, o);
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
    hipLaunchKernelGGL(k_attn_bf16<kAttnBuffers>, dim3(bv.n_items), dim3(256), 0, s, p);
    // half a wave per (slot, query head)
    hipLaunchKernelGGL(k_attn_combine, dim3((bv.T * D.hq + 7) / 8), dim3(256), 0, s, bv, sb.apart,
                       sb.aml, (bf16_t*)sb.attn, D.hq, D.hkv);
}

}  // namespace sdv
