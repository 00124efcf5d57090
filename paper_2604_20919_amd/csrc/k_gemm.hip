// Skinny GEMMs of the verify forward: Y[t][n] = sum_k X[t][k] W[n][k] for
// T = sum(l_m + 1) query slots (tens to a few hundred) against weight
// matrices of thousands of rows.  At these shapes the work is bound by
// streaming the weights from HBM once, so the kernels are built around that
// stream:
//   * weights are repacked once (at init) into fragment order: the A operand
//     of v_mfma_f32_16x16x32_bf16 for 16 weight rows x 32 k is one 1 KB block
//     laid out lane by lane (lane l: row l % 16, k 8*(l/16)..+7), and the
//     blocks of a 16-row group follow each other along k, so a wave-wide
//     weight load reads 1 KB (or, for the 32x32 form, two 512-byte runs)
//     contiguously;
//   * two MFMA forms share that layout: 16x16x32 tiles (16 slots per tile)
//     for small slot counts, where their finer slot padding wins, and
//     32x32x16 tiles (32 slots per tile) above, where the form's higher
//     rate (measured 2.1 vs 1.2 PFLOP/s) wins; every product runs twice, once
//     per activation plane, so the MFMA rate matters even here;
//   * the activation chunk X[0:T][k0:k0+KC] is staged in LDS (double
//     buffered) and read by all waves of the workgroup as the B operand;
//     activations come as two bf16 planes (hi, lo = x - hi) that are
//     multiplied separately, which carries them at about 16 significant bits;
//   * software pipeline per chunk: the loads of X(c+1) are issued before the
//     weight loads of chunk c+1, so storing X(c+1) to LDS after computing
//     chunk c waits for X only and the weight prefetch stays in flight;
//   * each wave owns a fixed set of weight rows and all T slots, so every
//     weight byte is read once per call;
//   * when there are too few column tiles to fill the GPU the k range is
//     split over S workgroups; partial sums are written to a workspace and a
//     second kernel (or a fused consumer) adds them in split order and
//     applies the epilogue (no device-wide fences, deterministic results);
//   * epilogues: fp32 store, residual add into the fp32 stream, or SwiGLU
//     silu(g) * u with gate/up rows interleaved per 16-row group.
// An fp32 fallback (plain FMA loop) serves the fp32 model configuration.
#include <algorithm>

#include "sdv_device.h"
#include "sdv_internal.h"

namespace sdv {

// Cache policy of the two operand streams (the aux word of the buffer
// loads): weights are read once per pass, so they are fetched nontemporal
// (nt), which measured 6.8 TB/s for the bare weight stream against 6.2 TB/s
// with the default policy; the activation chunks, which every workgroup
// re-reads from L2, take sc0.  Together: gate/up at T = 80 104-109 us
// against 117 us in isolation.
constexpr int kWeightAux = 2;
constexpr int kActAux = 1;

struct GemmP {
    const bf16_t* X;
    const bf16_t* Wp;  // packed weights: [vcols/16][K/32][64 lanes][8]
    int K, KT, T, S, kchunks, tiles;  // KT = K / 32 fragments per 16-row group
    // Work split: a wave unit is the row block one wave multiplies (NSUB
    // 16-row groups, or NS 32-row groups); G units in total.  Each k split
    // has WPS workgroups; workgroup w of a split takes units
    // [w*G/WPS, (w+1)*G/WPS), one per wave, so G need not be a multiple of
    // the waves per workgroup (waves past the range load nothing).
    int G, WPS;
    float* part;     // [S][T][vcols] when S > 1
    int vcols;
    void* out;
    int ldo;
    size_t oplane;  // SwiGLU: elements between the hi and lo output planes
    // RMSNorm applied after the product: when nss is set the input planes
    // hold x * gamma (not normalised) and every output of slot t is scaled
    // by rstd(t) = 1 / sqrt(sum_b nss[t][b] / K + eps), which commutes with
    // the product (one factor per slot row)
    const float* nss;
    int nnb;
    float eps;
    // EPI_LMSTAT: per (slot, workgroup) statistics [T][tiles], the logit of
    // each slot's next draft, that draft per slot (-1: none)
    VStat* lstat;
    float* zd;
    const int32_t* dnext;
    // stream-K (unsplit column-split GEMMs that leave CUs idle): the tiles x
    // kchunks (row tile, chunk) pairs are dealt out in tile-major order as
    // sk_nwg contiguous ranges of equal length, one per workgroup; a piece
    // that does not end its tile leaves its sums in partial slot (tile,
    // piece) of `part` and counts itself in sk_cnt[tile]; the tile's last
    // piece waits for that count, adds the earlier pieces in order and runs
    // the epilogue (sk_nwg = 0: off)
    // the piece waits for at most sk_polls polls of the count
    int sk_nwg, sk_maxp, sk_polls;
    // column-split form at 225-240 slots: the last slot tile holds the hi
    // rows of slots 224-239 in its rows 0-15 and their lo rows in rows 16-31
    // (one tile-plane instead of two); 0: off
    int pkl;
    int* sk_cnt;
    int32_t* flags;  // device error bits (bit 2: a stream-K wait gave up)
};

// stream-K: first pair of workgroup w's range, and the workgroup whose range
// holds pair i
__host__ __device__ __forceinline__ int sk_begin(int w, int total, int nwg) {
    return (int)((long long)w * total / nwg);
}
__host__ __device__ __forceinline__ int sk_owner(int i, int total, int nwg) {
    return (int)(((long long)(i + 1) * nwg - 1) / total);
}
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// lm_head epilogue, the part common to both MFMA forms: the per-wave
// statistics of every slot (staged in LDS as [wave][slot]) are merged over
// the workgroup's waves in wave order, i.e. in increasing vocab rows, and
// leave as one 16-byte record per (workgroup, slot)
template <int NTH, int NW, int NSLOT>
__device__ __forceinline__ void lmstat_merge_waves(const GemmP& p, const VStat* stg, int wgi) {
    for (int i = threadIdx.x; i < NSLOT && i < p.T; i += NTH) {
        VStat st = stg[i];
#pragma unroll
        for (int w = 1; w < NW; ++w) st = vstat_merge(st, stg[w * NSLOT + i]);
        p.lstat[(size_t)i * p.tiles + wgi] = st;
    }
}

// statistics of the n logits one lane holds for one slot (rows in
// increasing order); the draft's logit goes to zd when its row is here
template <int N>
__device__ __forceinline__ VStat lane_stat(const float (&z)[N], const int (&row)[N], int d, float* zd) {
    VStat st = vstat_empty();
#pragma unroll
    for (int e = 0; e < N; ++e) {
        if (z[e] > st.v) { st.v = z[e]; st.i = row[e]; }
        if (row[e] == d) *zd = z[e];
    }
    st.m = st.v;
    if (st.m != -INFINITY) {
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < N; ++e) sum += expf(z[e] - st.m);
        st.s = sum;
    }
    return st;
}

// block sums of one slot row, all loads issued before the sum (at most
// kNormKMax / kNormBlock blocks)
__device__ __forceinline__ void load_row_ss(const GemmP& p, int t, bool on, float (&v)[kNormKMax / kNormBlock]) {
#pragma unroll
    for (int b = 0; b < kNormKMax / kNormBlock; ++b)
        v[b] = on && b < p.nnb ? p.nss[(size_t)t * p.nnb + b] : 0.f;
}
__device__ __forceinline__ float rstd_of(const GemmP& p, const float (&v)[kNormKMax / kNormBlock]) {
    float ss = 0.f;
#pragma unroll
    for (int b = 0; b < kNormKMax / kNormBlock; ++b) ss += v[b];
    return 1.0f / sqrtf(ss / (float)p.K + p.eps);
}
__device__ __forceinline__ float row_rstd(const GemmP& p, int t) {
    if (p.nss == nullptr) return 1.0f;
    float v[kNormKMax / kNormBlock];
    load_row_ss(p, t, true, v);
    return rstd_of(p, v);
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }

template <int EPI>
__device__ __forceinline__ void epi_store4(const GemmP& p, int t, int col, f32x4 v, float sc) {
    v *= sc;
    float* o = (float*)p.out + (size_t)t * p.ldo + col;
    if (EPI == EPI_RESID) {
        f32x4 x = *(f32x4*)o;
        x += v;
        *(f32x4*)o = x;
    } else {
        *(f32x4*)o = v;
    }
}

// SwiGLU output as the next GEMM's activation planes: hi = bf16(a) at out,
// lo = bf16(a - hi) one plane (oplane elements) further
__device__ __forceinline__ void swiglu_store4(const GemmP& p, int t, int col, f32x4 g, f32x4 u,
                                              float sc) {
    g *= sc;
    u *= sc;
    bf16_t* o = (bf16_t*)p.out + (size_t)t * p.ldo + col;
    uint32_t hi[4], lo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float a = silu(g[e]) * u[e];
        hi[e] = f32_to_bf16(a);
        lo[e] = f32_to_bf16(a - bf16_to_f32((bf16_t)hi[e]));
    }
    *(uint2*)o = uint2{hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16)};
    *(uint2*)(o + p.oplane) = uint2{lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16)};
}

// Split-K partial sums of the 32x32 form leave through LDS: the
// workgroup's waves hold consecutive weight rows for every slot, staged as
// [slot][row] (row stride ldr floats), so that each 64-lane store writes
// 1 KB of one partial-sum row instead of 32-byte pieces of 32 rows.  Writes
// nsl slot rows starting at slot t0; only the first nrow rows are the
// workgroup's.  (Kernel traces on one machine at 80 slots: QKV / O / down
// 31.0 / 25.0 / 55.9 -> 29.8 / 23.7 / 53.5 us.)
template <int NTH, int WR>
__device__ __forceinline__ void store_partial_rows(const GemmP& p, const float* stg, int ldr, int split,
                                                   int t0, int nsl, int col0, int nrow) {
    constexpr int P4 = WR / 4;  // 16-byte pieces per staged slot row
    float* base = p.part + ((size_t)split * p.T + t0) * p.vcols + col0;
    for (int i = threadIdx.x; i < nsl * P4; i += NTH) {
        const int sl = i / P4, c4 = (i % P4) * 4;
        if (c4 < nrow) *(f32x4*)(base + (size_t)sl * p.vcols + c4) = *(const f32x4*)(stg + sl * ldr + c4);
    }
}

// 16x16x32 form.  MT: 16-slot tiles; NSUB: 16-row weight groups per wave;
// KC: k per chunk (a multiple of 32); NW: waves per workgroup; PL:
// activation planes; PD: chunks of prefetch.
// XPAD: bf16 elements of padding per staged row.  With 16 (a row stride of
// an odd multiple of 32 bytes) the B-fragment reads of 32 lanes (16 rows at
// two k offsets) hit distinct banks of the 128-bank LDS, and the staging
// stores are ordered so that the rows written together sit 16/R rows apart
// (R rows per 32 lanes), which also spreads them over every bank.  With 8
// (stride 272 or 144 bytes) rows 0 and 15 of a read share banks.
// LA (split SwiGLU product reduced by its last split): the S workgroups of
// a row tile each take a k range, store their sums and count themselves;
// the one that counts last adds every split's sums in split order and
// runs the SwiGLU epilogue, so no separate reduction kernel is needed.
template <int MT, int NSUB, int KC, int EPI, bool SPLIT, int NW, int PL, int PD, int XPAD = 16, bool LA = false>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(1, 2)))
void k_gemm16(GemmP p) {
    constexpr int NTH = 64 * NW;         // threads per workgroup
    constexpr int ROWS_PER_TILE = 16;
    constexpr int KS = KC / 32;          // MFMA k-steps per chunk
    constexpr int LDX = KC + XPAD;       // padded LDS row (bf16 elements)
    constexpr int PPR = KC / 8;          // 16-byte pieces per staged row
    constexpr int RPP = PPR >= 32 ? 1 : 32 / PPR;  // staged rows per 32 lanes
    constexpr int NPP = MT * 16 * PPR;   // pieces per staged plane
    constexpr int NPC = PL * NPP;        // pieces per staged chunk (all planes)
    constexpr int XPT = (NPC + NTH - 1) / NTH;  // X pieces per thread
    constexpr bool XEVEN = NPC % NTH == 0;
    constexpr int PLANE = MT * 16 * LDX;  // LDS elements per plane
    static_assert(EPI != EPI_SWIGLU || NSUB % 2 == 0, "SwiGLU pairs gate/up sub-tiles");
    static_assert(2 * PL * PLANE * 2 <= 160 * 1024, "X staging exceeds LDS");
    static_assert(!LA || (!SPLIT && EPI == EPI_SWIGLU), "last-split reduction: the SwiGLU product");
    __shared__ __attribute__((aligned(16))) bf16_t xs[2][PL * PLANE];
    __shared__ float rsl[SPLIT ? 1 : MT * ROWS_PER_TILE];  // per-slot RMSNorm factor
    __shared__ int la_count;  // LA: splits of this tile counted before this one

    // k split of this workgroup (consecutive workgroups take consecutive
    // splits, so with S a divisor of 8 every XCD works on one k range) and
    // its range of wave units
    constexpr bool KSPLIT = SPLIT || LA;
    const int split = KSPLIT ? blockIdx.x % p.S : 0;
    const int wgi = KSPLIT ? blockIdx.x / p.S : blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int lr = lane & 15, lg = lane >> 4;
    const int mt_act = (p.T + 15) >> 4;

    // Buffer resources: one uniform resource per operand, fixed 32-bit
    // per-lane offsets, uniform chunk offsets.  Out-of-range reads return 0
    // (and fetch nothing: a wave without a unit points past the buffer).
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const int unit = wgi * p.G / p.WPS + wv;
    const bool has_unit = unit < (wgi + 1) * p.G / p.WPS;
    const uint64_t wbytes = (uint64_t)p.vcols * (uint64_t)p.K * 2u;
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        (void*)p.Wp, (short)0, (int)(wbytes > 0x7fffffffu ? 0x7fffffffu : wbytes), 0x00020000);
    uint32_t woff[NSUB];
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
        const uint32_t vs = (uint32_t)(unit * NSUB + s);  // 16-row group
        woff[s] = has_unit ? vs * (uint32_t)p.KT * 1024u + (uint32_t)lane * 16u : 0x80000000u;
    }
    const __amdgpu_buffer_rsrc_t xres =
        __builtin_amdgcn_make_buffer_rsrc((void*)p.X, (short)0, PL * p.T * p.K * 2, 0x00020000);

    f32x4 acc[NSUB][MT];
#pragma unroll
    for (int s = 0; s < NSUB; ++s)
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[s][m] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int c_begin = split * p.kchunks / p.S;
    const int c_end = (split + 1) * p.kchunks / p.S;

    // Register-ring pipeline with prefetch distance PD chunks: while chunk c
    // is multiplied (X from LDS buffer c&1, W from ring set c % NB), X and W
    // of chunk c+PD are requested into ring set (c+PD) % NB, and X(c+1),
    // requested PD-1 chunks earlier, is stored to the other LDS buffer.  The
    // loop is unrolled by NB so that ring indices are compile-time constants
    // (register copies would force waits on loads still in flight), the
    // loads are unconditional (the chunk index is clamped; the last steps
    // re-read a cached chunk) and scheduling barriers keep the order issue
    // loads -> multiply -> store X.  X rows >= T are read as row T-1: they
    // only feed output slots >= T, which are never stored.
    constexpr int NB = PD + 1;
    uint4 xr[NB][XPT];
    bf16x8 wr[NB][KS][NSUB];
    uint32_t xoff[XPT];
    // staging order q -> LDS row (a permutation within each block of 16
    // rows; the identity for XPAD != 16)
    auto staged_row = [](int q) {
        if constexpr (XPAD != 16 || RPP == 1) return q;
        else return (q & ~15) | ((q % RPP) * (16 / RPP)) | ((q / RPP) % (16 / RPP));
    };
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
        const int idx = min((int)threadIdx.x + i * NTH, NPC - 1);
        const int pl = idx / NPP, pi = idx % NPP;
        const int r = min(staged_row(pi / PPR), p.T - 1), cc = pi % PPR;
        xoff[i] = (((uint32_t)pl * (uint32_t)p.T + (uint32_t)r) * (uint32_t)p.K + (uint32_t)cc * 8u) * 2u;
    }
    auto load_x = [&](uint4 (&x)[XPT], int c) {
        const int so = c * KC * 2;
#pragma unroll
        for (int i = 0; i < XPT; ++i)
            x[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xres, xoff[i], so, kActAux));
    };
    auto store_x = [&](const uint4 (&x)[XPT], int buf) {
#pragma unroll
        for (int i = 0; i < XPT; ++i) {
            const int idx = threadIdx.x + i * NTH;
            const int pl = idx / NPP, pi = idx % NPP;
            if (XEVEN || idx < NPC)
                *(uint4*)(&xs[buf][pl * PLANE + staged_row(pi / PPR) * LDX + (pi % PPR) * 8]) = x[i];
        }
    };
    auto load_w = [&](bf16x8 (&w)[KS][NSUB], int c) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int s = 0; s < NSUB; ++s)
                w[ks][s] = __builtin_bit_cast(
                    bf16x8, __builtin_amdgcn_raw_buffer_load_b128(wres, woff[s], (c * KS + ks) * 1024, kWeightAux));
    };
    // The X fragments of a group of slot tiles are read before their MFMAs
    // (all tiles of the k-step up to 8 tiles, groups of 4 above), and every
    // slot tile of the class is computed (tiles past T multiply clamped
    // copies of row T-1 and are never stored): a per-tile branch would
    // serialise LDS latency and MFMAs tile by tile.
    constexpr int MG = MT <= 8 ? MT : 4;
    // all slot tiles' B fragments of one k-step
    auto read_x = [&](bf16x8 (&xf)[PL][MT], const bf16_t* xb, int ks) {
#pragma unroll
        for (int pl = 0; pl < PL; ++pl)
#pragma unroll
            for (int g = 0; g < MT; ++g)
                xf[pl][g] = *(const bf16x8*)(xb + pl * PLANE + (g * 16 + lr) * LDX + ks * 32 + 8 * lg);
    };
    auto compute = [&](int buf, const bf16x8 (&w)[KS][NSUB]) {
        const bf16_t* xb = xs[buf];
        if constexpr (MT <= 8 && NW == 8) {
            // The next k-step's fragments are requested before this k-step's
            // MFMAs (scheduling barriers keep the order), so the LDS latency
            // hides under the matrix work instead of stalling each MFMA pair
            // (gate/up at T = 80: 112 -> 102 us).  Eight-wave tiles only: the
            // second fragment set would cost the four-wave tiles (lm_head)
            // their second wave per SIMD.
            bf16x8 xf[2][PL][MT];
            read_x(xf[0], xb, 0);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                if (ks + 1 < KS) read_x(xf[(ks + 1) & 1], xb, ks + 1);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int g = 0; g < MT; ++g)
#pragma unroll
                    for (int pl = 0; pl < PL; ++pl)
#pragma unroll
                        for (int s = 0; s < NSUB; ++s)
                            acc[s][g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[ks][s], xf[ks & 1][pl][g],
                                                                                acc[s][g], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
            return;
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
            for (int m0 = 0; m0 < MT; m0 += MG) {
                bf16x8 xf[PL][MG];
#pragma unroll
                for (int pl = 0; pl < PL; ++pl)
#pragma unroll
                    for (int g = 0; g < MG; ++g)
                        if (m0 + g < MT)
                            xf[pl][g] = *(const bf16x8*)(xb + pl * PLANE + ((m0 + g) * 16 + lr) * LDX +
                                                         ks * 32 + 8 * lg);
#pragma unroll
                for (int g = 0; g < MG; ++g)
                    if (m0 + g < MT)
#pragma unroll
                        for (int pl = 0; pl < PL; ++pl)
#pragma unroll
                            for (int s = 0; s < NSUB; ++s)
                                acc[s][m0 + g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    w[ks][s], xf[pl][g], acc[s][m0 + g], 0, 0, 0);
            }
        }
    };

    const int c_last = c_end - 1;
    // RMSNorm row factors of the tile's slots (epilogues that scale by
    // them): loads issued ahead of the pipeline prologue, the factors go to
    // LDS before the first barrier
    constexpr int NSL = MT * ROWS_PER_TILE;
    constexpr int NSPT = SPLIT ? 1 : (NSL + NTH - 1) / NTH;  // slots per thread
    float ssv[NSPT][kNormKMax / kNormBlock];
    if constexpr (!SPLIT) {
#pragma unroll
        for (int i = 0; i < NSPT; ++i) {
            const int sl = threadIdx.x + i * NTH;
            load_row_ss(p, min(sl, p.T - 1), p.nss != nullptr && sl < NSL, ssv[i]);
        }
    }
#pragma unroll
    for (int u = 0; u < PD; ++u) {
        load_x(xr[u], min(c_begin + u, c_last));
        load_w(wr[u], min(c_begin + u, c_last));
    }
    if constexpr (!SPLIT) {
#pragma unroll
        for (int i = 0; i < NSPT; ++i) {
            const int sl = threadIdx.x + i * NTH;
            if (sl < NSL) rsl[sl] = p.nss != nullptr ? rstd_of(p, ssv[i]) : 1.0f;
        }
    }
    store_x(xr[0], 0);
    __syncthreads();
    for (int c0 = c_begin; c0 < c_end; c0 += NB) {
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const int c = c0 + u;
            if (c >= c_end) break;
            load_x(xr[(u + PD) % NB], min(c + PD, c_last));
            load_w(wr[(u + PD) % NB], min(c + PD, c_last));
            __builtin_amdgcn_sched_barrier(0);
            compute((c - c_begin) & 1, wr[u]);
            __builtin_amdgcn_sched_barrier(0);
            store_x(xr[(u + 1) % NB], ((c - c_begin) & 1) ^ 1);
            __syncthreads();
        }
    }

    if constexpr (LA) {
        // The tile's splits exchange their sums through memory at system
        // scope (written through, read past the caches), ordered by the
        // count: each split stores into a slot of its own, waits for the
        // stores, passes a barrier and counts; the split that counts last
        // (no waiting anywhere: every split goes on or leaves at once)
        // resets the count and loads the other slots.  Slot layout: piece
        // j = s * MT + m of thread i at j * NTH + i (16 bytes, coalesced).
        constexpr int PER = NSUB * MT;  // 16-byte accumulator pieces per thread
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(p.part + (size_t)wgi * p.S * (size_t)(NTH * PER * 4)), (short)0, p.S * NTH * PER * 16,
            0x00020000);
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
            for (int m = 0; m < MT; ++m)
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[s][m]), r,
                                                       ((split * PER + s * MT + m) * NTH + (int)threadIdx.x) * 16,
                                                       0, 17);
        wait_vm<0>();
        __syncthreads();
        if (threadIdx.x == 0)
            la_count = __hip_atomic_fetch_add(p.sk_cnt + wgi, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        __syncthreads();
        if (la_count < p.S - 1) return;
        // every split has counted: back to zero for the next launch
        if (threadIdx.x == 0) __hip_atomic_store(p.sk_cnt + wgi, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        // all splits' sums in split order (this split's from its registers)
        f32x4 tot[NSUB][MT];
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
            for (int m = 0; m < MT; ++m) tot[s][m] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int sp = 0; sp < p.S; ++sp) {
            if (sp == split) {
#pragma unroll
                for (int s = 0; s < NSUB; ++s)
#pragma unroll
                    for (int m = 0; m < MT; ++m) tot[s][m] += acc[s][m];
                continue;
            }
            u32x4 v[NSUB][MT];
#pragma unroll
            for (int s = 0; s < NSUB; ++s)
#pragma unroll
                for (int m = 0; m < MT; ++m)
                    v[s][m] = __builtin_amdgcn_raw_buffer_load_b128(
                        r, ((sp * PER + s * MT + m) * NTH + (int)threadIdx.x) * 16, 0, 17);
#pragma unroll
            for (int s = 0; s < NSUB; ++s)
#pragma unroll
                for (int m = 0; m < MT; ++m) tot[s][m] += __builtin_bit_cast(f32x4, v[s][m]);
        }
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
            for (int m = 0; m < MT; ++m) acc[s][m] = tot[s][m];
    }

    if constexpr (EPI == EPI_LMSTAT) {
        // lane holds D[n = 4*lg + r][t = lr]: a slot's 16 rows of a group sit
        // in lanes lr, lr + 16, lr + 32, lr + 48
        static_assert(!SPLIT, "the lm_head statistics need whole k sums");
        constexpr int NSLOT = MT * 16;
        static_assert(NW * NSLOT * (int)sizeof(VStat) <= (int)sizeof(xs), "statistics staging exceeds LDS");
        VStat* stg = reinterpret_cast<VStat*>(&xs[0][0]);
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            const int t = m * 16 + lr;
            VStat st = vstat_empty();
            if (has_unit && m < mt_act && t < p.T) {
                const float sc = rsl[t];
                float z[NSUB * 4];
                int row[NSUB * 4];
#pragma unroll
                for (int s = 0; s < NSUB; ++s) {
                    const int r0 = (unit * NSUB + s) * 16 + 4 * lg;
                    f32x4 v = acc[s][m] * sc;
                    if (p.out) *(f32x4*)((float*)p.out + (size_t)t * p.ldo + r0) = v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        z[s * 4 + e] = v[e];
                        row[s * 4 + e] = r0 + e;
                    }
                }
                st = lane_stat(z, row, p.dnext[t], p.zd + t);
            }
            st = vstat_merge(st, vstat_shfl_xor(st, 16));
            st = vstat_merge(st, vstat_shfl_xor(st, 32));
            if (lg == 0) stg[wv * NSLOT + t] = st;
        }
        __syncthreads();
        lmstat_merge_waves<NTH, NW, NSLOT>(p, stg, wgi);
        return;
    }
    // lane holds D[n = 4*lg + r][t = lr] of each (sub-tile, slot tile)
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const int t = m * 16 + lr;
        if (!(has_unit && m < mt_act && t < p.T)) continue;
        const float sc = SPLIT ? 1.0f : rsl[t];
        if (SPLIT) {
#pragma unroll
            for (int s = 0; s < NSUB; ++s) {
                const int v = (unit * NSUB + s) * 16 + 4 * lg;
                *(f32x4*)(p.part + ((size_t)split * p.T + t) * p.vcols + v) = acc[s][m];
            }
        } else if (EPI == EPI_SWIGLU) {
            // groups 2j / 2j+1 hold gate / up rows 16j..16j+15
#pragma unroll
            for (int s = 0; s < NSUB; s += 2)
                swiglu_store4(p, t, (unit * NSUB + s) / 2 * 16 + 4 * lg, acc[s][m], acc[s + 1][m], sc);
        } else {
#pragma unroll
            for (int s = 0; s < NSUB; ++s)
                epi_store4<EPI>(p, t, (unit * NSUB + s) * 16 + 4 * lg, acc[s][m], sc);
        }
    }
}

typedef float f32x16 __attribute__((ext_vector_type(16)));

// 32x32x16 form.  MT: 32-slot tiles; NS: 32-row weight groups (pairs of
// 16-row groups) per wave; KC: k per chunk (a multiple of 16); NW: waves per
// workgroup; PL: activation planes; PD: chunks of prefetch.
// PK (two planes packed, for 32a < T <= 32a + 16): the B operand's columns
// are (slot, plane) pairs instead of slots, MT = 2a + 1 tiles in one staged
// plane: tiles 0..a-1 the hi plane of slots 0..32a-1, tile a the hi plane of
// slots 32a.. in columns 0-15 and their lo plane in columns 16-31, tiles
// a+1..2a the lo plane of slots 0..32a-1.  That is one tile fewer than two
// planes of a + 1 tiles each; the epilogue adds each slot's hi and lo sums
// (same lane of tiles m and m + a + 1, or lanes l and l ^ 16 of tile a).
//
// CS (column split): CS waves share one row unit and each multiplies MT/CS
// of the slot tiles.  With NS = 2 (64 weight rows per wave) every B
// fragment read from LDS then feeds two MFMAs instead of one: four SIMDs
// issuing 32-cycle MFMAs ask for 64 bytes per clock of LDS reads instead
// of 128, at the same accumulator count per wave.
// SKF: stream-K (unsplit column-split GEMMs, see GemmP).
template <int MT, int NS, int KC, int EPI, bool SPLIT, int NW, int PL, int PD, bool PK = false, int CS = 1,
          bool SKF = false>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(NW > 8 ? NW / 4 : 1, NW > 8 ? NW / 4 : 2)))
void k_gemm32(GemmP p) {
    static_assert(!PK || (PL == 2 && MT % 2 == 1), "packed planes: two planes, 2a + 1 tiles");
    static_assert(MT % CS == 0 && NW % CS == 0 && (CS == 1 || !PK),
                  "column split: whole tiles per wave, no packed planes");
    static_assert(!SKF || (CS > 1 && !SPLIT && EPI == EPI_SWIGLU), "stream-K: the unsplit SwiGLU product");
    constexpr int MTW = MT / CS;         // slot tiles per wave
    constexpr int PLS = PK ? 1 : PL;     // staged (and multiplied) planes
    constexpr int PA = MT / 2;           // packed: full tiles per plane
    constexpr int NTH = 64 * NW;         // threads per workgroup
    constexpr int ROWS_PER_TILE = 32;
    constexpr int KS = KC / 16;          // MFMA k-steps per chunk
    constexpr int LDX = KC + 8;          // padded LDS row (bf16 elements)
    constexpr int PPR = KC / 8;          // 16-byte pieces per staged row
    constexpr int NPP = MT * 32 * PPR;   // pieces per staged plane
    constexpr int NPC = PLS * NPP;       // pieces per staged chunk (all planes)
    constexpr int XPT = (NPC + NTH - 1) / NTH;  // X pieces per thread
    constexpr bool XEVEN = NPC % NTH == 0;
    constexpr int PLANE = MT * 32 * LDX;  // LDS elements per plane
    // NXB X staging buffers of XBUF elements (padded rows; the column-split
    // form keeps two unpadded chunks in the same array); the split epilogue
    // stages its partial sums in the same memory, which may need more
    constexpr int XBUF = PLS * PLANE;
    constexpr int NXB = 2;
    constexpr int STG_BYTES = SPLIT ? CS * 32 * (NW / CS * NS * 32 + 4) * 4 : 0;
    constexpr int XS_ELEMS = 2 * NXB * XBUF >= STG_BYTES ? NXB * XBUF : STG_BYTES / 2;
    static_assert(XS_ELEMS * 2 <= 160 * 1024, "staging exceeds LDS");
    __shared__ __attribute__((aligned(16))) bf16_t xs[XS_ELEMS];
    __shared__ float rsl[SPLIT ? 1 : MT * ROWS_PER_TILE];  // per-slot RMSNorm factor

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int lc = lane & 31, lh = lane >> 5;
    // Stream-K: the workgroup's range of (row tile, chunk) pairs is shorter
    // than a tile, so it is one piece of a tile or two: the head of the last
    // tile and the tail of the first, taken in that order (k increasing, so
    // all workgroups walk the activation chunks nearly together and share
    // them in L2).  Otherwise one piece: the whole k range of a split.
    int sk_np = 1, sk_t[2] = {0, 0}, sk_b[2] = {0, 0}, sk_e[2] = {0, 0};
    if constexpr (SKF) {
        const int total = p.tiles * p.kchunks;
        const int wb = sk_begin(blockIdx.x, total, p.sk_nwg), we = sk_begin(blockIdx.x + 1, total, p.sk_nwg);
        const int t0 = wb / p.kchunks, t1 = (we - 1) / p.kchunks;
        if (t0 == t1) {
            sk_t[0] = t0; sk_b[0] = wb - t0 * p.kchunks; sk_e[0] = we - t0 * p.kchunks;
        } else {
            sk_np = 2;
            sk_t[0] = t1; sk_b[0] = 0; sk_e[0] = we - t1 * p.kchunks;
            sk_t[1] = t0; sk_b[1] = wb - t0 * p.kchunks; sk_e[1] = p.kchunks;
        }
    }
    for (int piece = 0; piece < sk_np; ++piece) {
    const int split = SPLIT ? blockIdx.x % p.S : 0;
    const int wgi = SKF ? (piece == 0 ? sk_t[0] : sk_t[1]) : (SPLIT ? blockIdx.x / p.S : blockIdx.x);

    // Buffer resources: one uniform resource per operand, fixed 32-bit
    // per-lane offsets, uniform chunk offsets.  Out-of-range reads return 0
    // (and fetch nothing: a wave without a unit points past the buffer).
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const int half = CS == 1 ? 0 : wv % CS;   // which MT/CS slot tiles
    const int m0 = half * MTW;
    const int unit = wgi * p.G / p.WPS + wv / CS;
    const bool has_unit = unit < (wgi + 1) * p.G / p.WPS;
    const uint64_t wbytes = (uint64_t)p.vcols * (uint64_t)p.K * 2u;
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        (void*)p.Wp, (short)0, (int)(wbytes > 0x7fffffffu ? 0x7fffffffu : wbytes), 0x00020000);
    // The A operand of a 16-k step (lane l: row l % 32, k 8*(l/32)..+7)
    // taken from the 16-row fragments: rows 0-15 / 16-31 are 16-row groups
    // 2g / 2g+1; k-step j sits in fragment j/2 at k 16*(j%2), i.e. lane slot
    // (l % 16) + 16*(l/32) + 32*(j%2).  Per lane that is a fixed offset plus
    // a uniform 512*j.
    uint32_t woff[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const uint32_t g16 = (uint32_t)((unit * NS + s) * 2 + (lc >> 4));
        woff[s] = has_unit ? g16 * (uint32_t)p.KT * 1024u + (uint32_t)((lane & 15) + 16 * lh) * 16u
                           : 0x80000000u;
    }
    const __amdgpu_buffer_rsrc_t xres =
        __builtin_amdgcn_make_buffer_rsrc((void*)p.X, (short)0, PL * p.T * p.K * 2, 0x00020000);

    f32x16 acc[NS][MTW];
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int m = 0; m < MTW; ++m)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[s][m][e] = 0.f;

    const int c_begin = SKF ? (piece == 0 ? sk_b[0] : sk_b[1]) : split * p.kchunks / p.S;
    const int c_end = SKF ? (piece == 0 ? sk_e[0] : sk_e[1]) : (split + 1) * p.kchunks / p.S;

    // Register-ring pipeline with prefetch distance PD chunks (the form
    // without column split; the column-split form below stages X by direct
    // loads): while chunk c is multiplied (X from LDS buffer c&1, W from
    // ring set c % NB), X and W of chunk c+PD are requested into ring set
    // (c+PD) % NB, and X(c+1), requested PD-1 chunks earlier, is stored to
    // the other LDS buffer.  The
    // loop is unrolled by NB so that ring indices are compile-time constants
    // (register copies would force waits on loads still in flight), the
    // loads are unconditional (the chunk index is clamped; the last steps
    // re-read a cached chunk) and scheduling barriers keep the order issue
    // loads -> multiply -> store X.  X rows >= T are read as row T-1: they
    // only feed output slots >= T, which are never stored.
    constexpr int NB = PD + 1;
    uint4 xr[NB][XPT];
    bf16x8 wr[NB][KS][NS];
    uint32_t xoff[XPT];
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
        const int idx = min((int)threadIdx.x + i * NTH, NPC - 1);
        int pl = idx / NPP, row = (idx % NPP) / PPR;
        const int cc = idx % PPR;
        if (PK) {
            // staged row -> (plane, slot) of the packed layout
            const int v = row;
            pl = v < 32 * PA + 16 ? 0 : 1;
            row = v < 32 * PA + 16 ? v : v < 32 * PA + 32 ? v - 16 : v - 32 * (PA + 1);
        }
        const int r = min(row, p.T - 1);
        xoff[i] = (((uint32_t)pl * (uint32_t)p.T + (uint32_t)r) * (uint32_t)p.K + (uint32_t)cc * 8u) * 2u;
    }
    auto load_x = [&](uint4 (&x)[XPT], int c) {
        const int so = c * KC * 2;
#pragma unroll
        for (int i = 0; i < XPT; ++i)
            x[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xres, xoff[i], so, kActAux));
    };
    auto store_x = [&](const uint4 (&x)[XPT], int buf) {
#pragma unroll
        for (int i = 0; i < XPT; ++i) {
            const int idx = threadIdx.x + i * NTH;
            const int pl = idx / NPP, pi = idx % NPP;
            if (XEVEN || idx < NPC)
                *(uint4*)(&xs[buf * XBUF + pl * PLANE + (pi / PPR) * LDX + (pi % PPR) * 8]) = x[i];
        }
    };
    auto load_w = [&](bf16x8 (&w)[KS][NS], int c) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int s = 0; s < NS; ++s)
                w[ks][s] = __builtin_bit_cast(
                    bf16x8, __builtin_amdgcn_raw_buffer_load_b128(wres, woff[s], (c * KS + ks) * 512, kWeightAux));
    };
    // The B fragments of a k-step (lane l: slot l % 32 of the tile, k
    // 8*(l/32)..+7) are read for all tiles before their MFMAs, one k-step
    // ahead, and every slot tile of the class is computed (tiles past T
    // multiply clamped copies of row T-1 and are never stored).  MFMAs on one
    // accumulator are MT*NS instructions apart (planes outermost).
    auto read_x = [&](bf16x8 (&xf)[PLS][MT], const bf16_t* xb, int ks) {
#pragma unroll
        for (int pl = 0; pl < PLS; ++pl)
#pragma unroll
            for (int m = 0; m < MT; ++m)
                xf[pl][m] = *(const bf16x8*)(xb + pl * PLANE + (m * 32 + lc) * LDX + ks * 16 + 8 * lh);
    };
    auto compute = [&](int buf, const bf16x8 (&w)[KS][NS]) {
        if constexpr (CS == 1) {
            const bf16_t* xb = xs + buf * XBUF;
            bf16x8 xf[2][PLS][MT];
            read_x(xf[0], xb, 0);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                if (ks + 1 < KS) read_x(xf[(ks + 1) & 1], xb, ks + 1);
#pragma unroll
                for (int pl = 0; pl < PLS; ++pl)
#pragma unroll
                    for (int m = 0; m < MT; ++m)
#pragma unroll
                        for (int s = 0; s < NS; ++s)
                            acc[s][m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w[ks][s], xf[ks & 1][pl][m],
                                                                                 acc[s][m], 0, 0, 0);
            }
        }
    };

    const int c_last = c_end - 1;
    // RMSNorm row factors of the tile's slots (epilogues that scale by
    // them): loads issued ahead of the pipeline prologue, the factors go to
    // LDS before the first barrier
    constexpr int NSL = MT * ROWS_PER_TILE;
    constexpr int NSPT = SPLIT ? 1 : (NSL + NTH - 1) / NTH;  // slots per thread
    float ssv[NSPT][kNormKMax / kNormBlock];
    if constexpr (!SPLIT) {
#pragma unroll
        for (int i = 0; i < NSPT; ++i) {
            const int sl = threadIdx.x + i * NTH;
            load_row_ss(p, min(sl, p.T - 1), p.nss != nullptr && sl < NSL, ssv[i]);
        }
    }
#pragma unroll
    for (int u = 0; u < PD; ++u) {
        if constexpr (CS == 1) load_x(xr[u], min(c_begin + u, c_last));
        load_w(wr[u], min(c_begin + u, c_last));
    }
    if constexpr (!SPLIT) {
#pragma unroll
        for (int i = 0; i < NSPT; ++i) {
            const int sl = threadIdx.x + i * NTH;
            if (sl < NSL) rsl[sl] = p.nss != nullptr ? rstd_of(p, ssv[i]) : 1.0f;
        }
    }
    if constexpr (CS > 1) {
        // Two X buffers; per chunk c: the direct loads of X(c + 1) into the
        // other buffer are issued first; phases (k-step, plane) follow, the
        // next phase's fragments requested before this phase's NS * MTW
        // MFMAs; after the last plane of a k-step its weight registers are
        // reloaded with the same k-step of chunk c + 1 (one register set,
        // each fragment requested about a chunk ahead); the wave then waits
        // for its direct loads and the barrier publishes the buffer.
        constexpr int NPH = KS * PLS;
        static_assert(NPH % 2 == 0, "phase fragments alternate between two register sets");
        // X is staged by direct global-to-LDS loads: a chunk is 64 blocks of
        // 1 KB, block (plane, tile, row group of 8) holding 8 rows of 64 k
        // (128 B each) whose 16-byte pieces are XOR-swizzled by the row
        // (piece q at position q ^ ((row >> 1) & 7), row within the tile), so
        // that the fragment reads of 16 rows hit 16 different bank groups.
        // A wave's direct load fills one block (lane l: row l / 8, position
        // l % 8), so each lane fetches the piece that belongs to its
        // position; each wave loads eight blocks per chunk.
        static_assert(MT == 8 && KC == 64 && PLS == 2 && NW == 8 && MTW == 4,
                      "direct X staging: 64 blocks per chunk, 8 per wave");
        constexpr int DBUF = PLS * MT * 32 * KC;  // bf16 elements per staged chunk
        static_assert(2 * DBUF <= XS_ELEMS, "two staged chunks fit the staging array");
        typedef __attribute__((address_space(3))) void lds_void;
        uint32_t doff[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int blk = wv * 8 + i, pl = blk >> 5, mt = (blk >> 2) & 7, rb = blk & 3;
            const int lrow = rb * 8 + (lane >> 3);
            const int pc = (lane & 7) ^ ((lrow >> 1) & 7);
            // packed last tile: rows 0-15 from the hi plane, 16-31 from the lo
            // plane, of the same 16 slots
            const bool pk = p.pkl && pl == 0 && mt == MT - 1;
            const int spl = pk ? lrow >> 4 : pl;
            const int row = min(mt * 32 + (pk ? lrow & 15 : lrow), p.T - 1);
            doff[i] = (((uint32_t)spl * (uint32_t)p.T + (uint32_t)row) * (uint32_t)p.K + (uint32_t)pc * 8u) * 2u;
        }
        auto dma_x = [&](int c, int buf) {
            bf16_t* base = xs + buf * DBUF + wv * 8 * 512;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(xres, (lds_void*)(base + i * 512), 16, (int)doff[i],
                                                         c * KC * 2, 0, kActAux);
        };
        // fragment reads in inline assembly: the compiler cannot tell them from
        // the direct loads into the other buffer and would wait for every
        // load in flight before them; their completion is waited for
        // explicitly, with the fragments as operands
        const uint32_t xs_addr = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16_t*)xs;
        const bool pkl_half = p.pkl && half == CS - 1;  // this wave holds the packed tile
        uint32_t loff[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            loff[ks] = (uint32_t)((lc >> 3) * 1024 + (lc & 7) * 128 + (((2 * ks + lh) ^ ((lc >> 1) & 7)) * 16));
        bf16x8 xq[2][MTW];
        auto read_phase = [&](bf16x8 (&xf)[MTW], int buf, int ph) {
            const int ks = ph / PLS, pl = ph % PLS;
            const uint32_t a = xs_addr + (uint32_t)(buf * DBUF * 2) + loff[ks] + (uint32_t)((pl * MT + m0) * 4096);
            asm volatile(
                "ds_read_b128 %0, %4\n\t"
                "ds_read_b128 %1, %4 offset:4096\n\t"
                "ds_read_b128 %2, %4 offset:8192\n\t"
                "ds_read_b128 %3, %4 offset:12288"
                : "=&v"(xf[0]), "=&v"(xf[1]), "=&v"(xf[2]), "=&v"(xf[3])
                : "v"(a)
                : "memory");
        };
        auto load_w_ks = [&](bf16x8 (&w)[NS], int c, int ks) {
#pragma unroll
            for (int s = 0; s < NS; ++s)
                w[s] = __builtin_bit_cast(
                    bf16x8, __builtin_amdgcn_raw_buffer_load_b128(wres, woff[s], (c * KS + ks) * 512, kWeightAux));
        };
        dma_x(c_begin, 0);
        __syncthreads();
        read_phase(xq[0], 0, 0);
        for (int c = c_begin; c < c_end; ++c) {
            const int b = (c - c_begin) & 1;
            const int cn = min(c + 1, c_last);
            dma_x(cn, b ^ 1);
#pragma unroll
            for (int ph = 0; ph < NPH; ++ph) {
                if (ph + 1 < NPH) {
                    read_phase(xq[(ph + 1) & 1], b, ph + 1);
                    asm volatile("s_waitcnt lgkmcnt(4)"
                                 : "+v"(xq[ph & 1][0]), "+v"(xq[ph & 1][1]), "+v"(xq[ph & 1][2]), "+v"(xq[ph & 1][3]));
                } else {
                    asm volatile("s_waitcnt lgkmcnt(0)"
                                 : "+v"(xq[ph & 1][0]), "+v"(xq[ph & 1][1]), "+v"(xq[ph & 1][2]), "+v"(xq[ph & 1][3]));
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int m = 0; m < MTW; ++m)
#pragma unroll
                    for (int s = 0; s < NS; ++s)
                        if (!(m == MTW - 1 && ph % PLS == 1 && pkl_half))  // packed tile: one plane-phase
                            acc[s][m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wr[0][ph / PLS][s], xq[ph & 1][m],
                                                                                 acc[s][m], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
                if (ph % PLS == PLS - 1) load_w_ks(wr[0][ph / PLS], cn, ph / PLS);
            }
            // this wave's direct loads of chunk cn precede the NS * KS weight
            // loads issued since; the barrier then publishes every wave's
            // block (all reads of the other buffer were waited for above)
            wait_vm<NS * KS>();
            barrier_nofence();
            if (c + 1 < c_end) read_phase(xq[0], b ^ 1, 0);
        }
    } else {
    store_x(xr[0], 0);
    __syncthreads();
    for (int c0 = c_begin; c0 < c_end; c0 += NB) {
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const int c = c0 + u;
            if (c >= c_end) break;
            load_x(xr[(u + PD) % NB], min(c + PD, c_last));
            load_w(wr[(u + PD) % NB], min(c + PD, c_last));
            __builtin_amdgcn_sched_barrier(0);
            compute((c - c_begin) & 1, wr[u]);
            __builtin_amdgcn_sched_barrier(0);
            store_x(xr[(u + 1) % NB], ((c - c_begin) & 1) ^ 1);
            __syncthreads();
        }
    }
    }

    int sk_ord = 0;  // earlier pieces of this tile to add (the tile's last piece)
    if constexpr (SKF) {
        // Partial sums travel through memory at system scope (written
        // through, read past the caches), ordered by the count: stores, wait
        // for them, barrier, then the count; the reader polls the count
        // before it loads.  Slot layout: element j of thread i at j * NTH + i
        // (16-byte pieces, coalesced).
        constexpr int PER4 = NS * MTW * 4;  // 16-byte accumulator pieces per thread
        const int total = p.tiles * p.kchunks;
        const int ord = (int)blockIdx.x - sk_owner(wgi * p.kchunks, total, p.sk_nwg);
        auto slot_rsrc = [&](int o) {
            return __builtin_amdgcn_make_buffer_rsrc(
                (void*)(p.part + ((size_t)wgi * p.sk_maxp + o) * (size_t)(NTH * PER4 * 4)), (short)0,
                NTH * PER4 * 16, 0x00020000);
        };
        if (c_end < p.kchunks) {
            const __amdgpu_buffer_rsrc_t r = slot_rsrc(ord);
#pragma unroll
            for (int s = 0; s < NS; ++s)
#pragma unroll
                for (int m = 0; m < MTW; ++m)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int j = (s * MTW + m) * 4 + q;
                        const f32x4 v = f32x4{acc[s][m][4 * q], acc[s][m][4 * q + 1], acc[s][m][4 * q + 2],
                                              acc[s][m][4 * q + 3]};
                        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r,
                                                               (j * NTH + (int)threadIdx.x) * 16, 0, 17);
                    }
            wait_vm<0>();
            __syncthreads();
            if (threadIdx.x == 0)
                __hip_atomic_fetch_add(p.sk_cnt + wgi, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            continue;
        }
        if (ord > 0) {
            if (threadIdx.x == 0) {
                for (int polls = 0;; ++polls) {
                    if (polls >= p.sk_polls) {
                        atomicOr(p.flags, 4);
                        break;
                    }
                    if (__hip_atomic_load(p.sk_cnt + wgi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) >= ord)
                        break;
                    __builtin_amdgcn_s_sleep(2);
                }
                // back to zero once every earlier piece has counted, also
                // after a wait that gave up (the stream runs the next launch
                // only when all of this one's workgroups have ended)
                __hip_atomic_fetch_sub(p.sk_cnt + wgi, ord, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            }
            __syncthreads();
            sk_ord = ord;  // added tile by tile in the epilogue (fewer live registers)
        }
    }
    // Packed last tile of the column-split form (its wave's tile MTW - 1):
    // slot 224 + i's sums are those of lanes l and l ^ 16 (i = l % 16),
    // added by v_permlane16_swap; run after the earlier stream-K pieces'
    // sums are in
    const bool pkl_fold = CS > 1 && p.pkl && half == CS - 1;
    auto fold_last = [&]() {
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const auto pr = __builtin_amdgcn_permlane16_swap(__float_as_uint(acc[s][MTW - 1][e]),
                                                                 __float_as_uint(acc[s][MTW - 1][e]), false, false);
                acc[s][MTW - 1][e] = __uint_as_float(pr[0]) + __uint_as_float(pr[1]);
            }
    };
    // Accumulator layout: lane l holds slot t = 32*m + l % 32 and, in
    // registers 4q..4q+3, weight rows 8q + 4*(l/32) + 0..3 of its group.
    // Packed planes: slot t's sums are those of tile m and tile m + a + 1
    // (t < 32a), or of lanes l and l ^ 16 of tile a, swapped in by
    // v_permlane16_swap, which hands each lane the pair (own, partner).
    if constexpr (PK) {
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const auto pr = __builtin_amdgcn_permlane16_swap(__float_as_uint(acc[s][PA][e]),
                                                                 __float_as_uint(acc[s][PA][e]), false, false);
                acc[s][PA][e] = __uint_as_float(pr[0]) + __uint_as_float(pr[1]);
#pragma unroll
                for (int m = 0; m < PA; ++m) acc[s][m][e] += acc[s][m + PA + 1][e];
            }
    }
    if constexpr (EPI == EPI_LMSTAT) {
        // lane l holds slot 32m + l % 32 and rows 8q + 4(l/32) + 0..3 of its
        // 32-row group: a slot's rows sit in lanes l and l ^ 32
        static_assert(!SPLIT, "the lm_head statistics need whole k sums");
        // (column split: the NW / CS row units each stage every slot once)
        constexpr int MTO = PK ? PA + 1 : MTW;
        constexpr int NSLOT = (PK ? PA + 1 : MT) * 32;
        constexpr int NU = NW / CS;  // row units per workgroup
        static_assert(NU * NSLOT * (int)sizeof(VStat) <= (int)sizeof(xs), "statistics staging exceeds LDS");
        VStat* stg = reinterpret_cast<VStat*>(xs);
        if (pkl_fold) fold_last();
#pragma unroll
        for (int m = 0; m < MTO; ++m) {
            const int t = (m0 + m) * 32 + lc;
            VStat st = vstat_empty();
            if (has_unit && t < p.T && !(PK && m == PA && lc >= 16)) {
                const float sc = rsl[t];
                float z[NS * 16];
                int row[NS * 16];
#pragma unroll
                for (int s = 0; s < NS; ++s)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int r0 = (unit * NS + s) * 32 + 8 * q + 4 * lh;
                        const f32x4 v = f32x4{acc[s][m][4 * q], acc[s][m][4 * q + 1], acc[s][m][4 * q + 2],
                                              acc[s][m][4 * q + 3]} * sc;
                        if (p.out) *(f32x4*)((float*)p.out + (size_t)t * p.ldo + r0) = v;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            z[s * 16 + 4 * q + e] = v[e];
                            row[s * 16 + 4 * q + e] = r0 + e;
                        }
                    }
                st = lane_stat(z, row, p.dnext[t], p.zd + t);
            }
            st = vstat_merge(st, vstat_shfl_xor(st, 32));
            if (lh == 0) stg[(wv / CS) * NSLOT + t] = st;
        }
        __syncthreads();
        lmstat_merge_waves<NTH, NU, NSLOT>(p, stg, wgi);
        return;
    }
    if constexpr (SPLIT) {
        // slot tiles m0 + m of every column half at a time through the (now
        // idle) staging buffer, staged as [half][slot][row]
        constexpr int WR = NW / CS * NS * 32;  // weight rows of the workgroup
        constexpr int LDR = WR + 4;
        static_assert(CS * 32 * LDR * 4 <= (int)sizeof(xs), "partial staging exceeds the X buffer");
        float* stg = reinterpret_cast<float*>(xs);
        const int u0 = wgi * p.G / p.WPS;
        const int nrow = ((wgi + 1) * p.G / p.WPS - u0) * NS * 32;
        const int wrow = wv / CS;  // row unit within the workgroup
        if (pkl_fold) fold_last();
#pragma unroll
        for (int m = 0; m < (PK ? PA + 1 : MTW); ++m) {
            if (m * 32 >= p.T) break;  // so are the other halves' tiles m + MTW * h
            if (has_unit) {
#pragma unroll
                for (int s = 0; s < NS; ++s)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        *(f32x4*)(stg + (half * 32 + lc) * LDR + (wrow * NS + s) * 32 + 8 * q + 4 * lh) =
                            f32x4{acc[s][m][4 * q], acc[s][m][4 * q + 1], acc[s][m][4 * q + 2], acc[s][m][4 * q + 3]};
            }
            __syncthreads();
#pragma unroll
            for (int h = 0; h < CS; ++h) {
                const int tile = h * MTW + m;
                const int nsl = min(PK && m == PA ? 16 : 32, p.T - tile * 32);
                if (nsl > 0)
                    store_partial_rows<NTH, WR>(p, stg + h * 32 * LDR, LDR, split, tile * 32, nsl, u0 * NS * 32,
                                                nrow);
            }
            __syncthreads();
        }
        return;
    }
#pragma unroll
    for (int m = 0; m < (PK ? PA + 1 : MTW); ++m) {
        if constexpr (SKF) {
            // the earlier pieces' sums of this slot tile, in piece order
            for (int o = 0; o < sk_ord; ++o) {
                const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
                    (void*)(p.part + ((size_t)wgi * p.sk_maxp + o) * (size_t)(NTH * NS * MTW * 16)), (short)0,
                    NTH * NS * MTW * 64, 0x00020000);
                u32x4 v[NS][4];
#pragma unroll
                for (int s = 0; s < NS; ++s)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        v[s][q] = __builtin_amdgcn_raw_buffer_load_b128(
                            r, (((s * MTW + m) * 4 + q) * NTH + (int)threadIdx.x) * 16, 0, 17);
#pragma unroll
                for (int s = 0; s < NS; ++s)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const f32x4 f = __builtin_bit_cast(f32x4, v[s][q]);
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc[s][m][4 * q + e] += f[e];
                    }
            }
        }
        if (m == MTW - 1 && pkl_fold) fold_last();
        const int t = (m0 + m) * 32 + lc;
        if (!has_unit || t >= p.T || (PK && m == PA && lc >= 16)) continue;
        const float sc = rsl[t];
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int grp = unit * NS + s;
            if (EPI == EPI_SWIGLU) {
                // rows 0-15 of the group are gate rows 16*grp.., 16-31 the
                // matching up rows; both sit in the same lane
#pragma unroll
                for (int q = 0; q < 2; ++q)
                    swiglu_store4(p, t, grp * 16 + 8 * q + 4 * lh,
                                  f32x4{acc[s][m][4 * q], acc[s][m][4 * q + 1], acc[s][m][4 * q + 2], acc[s][m][4 * q + 3]},
                                  f32x4{acc[s][m][4 * q + 8], acc[s][m][4 * q + 9], acc[s][m][4 * q + 10], acc[s][m][4 * q + 11]},
                                  sc);
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    epi_store4<EPI>(p, t, grp * 32 + 8 * q + 4 * lh,
                                    f32x4{acc[s][m][4 * q], acc[s][m][4 * q + 1], acc[s][m][4 * q + 2], acc[s][m][4 * q + 3]},
                                    sc);
            }
        }
    }
    }
}

// Sum of the S split-K partials (in split order) plus the epilogue; one
// thread per 4 output columns of one slot.
template <int EPI>
__global__ __launch_bounds__(256) void k_splitk_reduce(GemmP p) {
    const int ncols = EPI == EPI_SWIGLU ? p.vcols / 2 : p.vcols;
    const int per_row = ncols / 4;
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= p.T * per_row) return;
    const int t = idx / per_row, c = (idx % per_row) * 4;
    const size_t stride = (size_t)p.T * p.vcols;
    const float* base = p.part + (size_t)t * p.vcols;
    if (EPI == EPI_SWIGLU) {
        const int vg = (c / 16) * 32 + (c % 16);  // gate group 2j, up group 2j+1
        f32x4 g = f32x4{0.f, 0.f, 0.f, 0.f}, u = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < p.S; ++s) {
            g += *(const f32x4*)(base + s * stride + vg);
            u += *(const f32x4*)(base + s * stride + vg + 16);
        }
        swiglu_store4(p, t, c, g, u, row_rstd(p, t));
    } else {
        f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < p.S; ++s) v += *(const f32x4*)(base + s * stride + c);
        epi_store4<EPI>(p, t, c, v, row_rstd(p, t));
    }
}

// Weight repack into fragment order.  One wave per (16-row group, 32-k step)
// fragment; lane (r, g) = (lane % 16, lane / 16) copies row r, k 8g..8g+7.
// mode 0: virtual rows are the concatenation of up to three row-major
// segments (QKV); mode 1: groups 2j / 2j+1 are rows 16j.. of src0 / src1
// (SwiGLU gate / up).
__global__ __launch_bounds__(256) void k_pack(const bf16_t* src0, const bf16_t* src1,
                                              const bf16_t* src2, int seg1, int seg2, int mode,
                                              int K, int groups, bf16_t* dst) {
    const int KT = K / 32;
    const long long f = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (f >= (long long)groups * KT) return;
    const int lane = threadIdx.x & 63;
    const int vs = (int)(f / KT), ks = (int)(f % KT);
    const int r = lane & 15, g = lane >> 4;
    const bf16_t* row;
    if (mode == 1) {
        row = ((vs & 1) ? src1 : src0) + (size_t)((vs >> 1) * 16 + r) * K;
    } else {
        const int v = vs * 16 + r;
        row = v < seg1 ? src0 + (size_t)v * K
              : v < seg2 ? src1 + (size_t)(v - seg1) * K : src2 + (size_t)(v - seg2) * K;
    }
    *(uint4*)(dst + ((size_t)f * 64 + lane) * 8) = *(const uint4*)(row + ks * 32 + 8 * g);
}

void launch_pack(const void* s0, const void* s1, const void* s2, int seg1, int seg2, int mode,
                 int K, int vrows, void* dst, hipStream_t s) {
    const long long frags = (long long)(vrows / 16) * (K / 32);
    hipLaunchKernelGGL(k_pack, dim3((unsigned)((frags + 3) / 4)), dim3(256), 0, s,
                       (const bf16_t*)s0, (const bf16_t*)s1, (const bf16_t*)s2, seg1, seg2, mode, K,
                       vrows / 16, (bf16_t*)dst);
}

// ---------------------------------------------------------------------------
// fp32 fallback: one thread per output, plain k loop
// ---------------------------------------------------------------------------
struct GemmF {
    const float* X;
    const float* W0;
    const float* W1;
    const float* W2;
    int seg1, seg2, N, K, T, epi;
    float* out;
    int ldo;
};

__global__ void k_gemm_f32(GemmF p) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= p.T * p.N) return;
    const int t = idx / p.N, c = idx % p.N;
    const float* x = p.X + (size_t)t * p.K;
    if (p.epi == EPI_SWIGLU) {
        const float* wg = p.W0 + (size_t)c * p.K;
        const float* wu = p.W1 + (size_t)c * p.K;
        float g = 0.f, u = 0.f;
        for (int k = 0; k < p.K; ++k) {
            g = fmaf(x[k], wg[k], g);
            u = fmaf(x[k], wu[k], u);
        }
        p.out[(size_t)t * p.ldo + c] = silu(g) * u;
        return;
    }
    const float* w = c < p.seg1 ? p.W0 + (size_t)c * p.K
                     : c < p.seg2 ? p.W1 + (size_t)(c - p.seg1) * p.K
                                  : p.W2 + (size_t)(c - p.seg2) * p.K;
    float a = 0.f;
    for (int k = 0; k < p.K; ++k) a = fmaf(x[k], w[k], a);
    if (p.epi == EPI_RESID)
        p.out[(size_t)t * p.ldo + c] += a;
    else
        p.out[(size_t)t * p.ldo + c] = a;
}

// ---------------------------------------------------------------------------
// host-side configuration
// ---------------------------------------------------------------------------

// Tile shape per slot-count class: form F (16: 16x16x32 MFMA, 16-slot
// tiles, NSUB = 2 row groups of 16 per wave; 32: 32x32x16 MFMA, 32-slot
// tiles, one 32-row group per wave), MT slot tiles, KC k elements per
// pipeline chunk, PD chunks of prefetch, NW waves per workgroup.  Measured
// on the 32B shapes (two activation planes):
//   * eight waves (256 weight rows) share one staged X chunk where the row
//     count allows; it halves the X staging per weight byte;
//   * up to 96 slots the 16x16 form (128-k chunks, one chunk of prefetch)
//     wins: at T = 80 its 5 slot tiles pad nothing, where the 32x32 form
//     computes 96 slots (gate/up 113 vs 119 us in the full step);
//   * above, the 32x32 form wins by its MFMA rate: gate/up at T = 128 / 176
//     / 240 takes 141 / 188 / 390 us against 181 / 237 / 509 us;
//   * 225..256 slots: eight waves with 32-k chunks (gate/up at T = 240
//     292 us against 392 us for four waves with 64-k chunks);
//   * above 256 slots tiles need the register budget of one wave per SIMD
//     (four waves) and shorter chunks so that a double-buffered two-plane
//     chunk fits in LDS.
// FILL: choose the k splits to fill one wave of workgroups (the eight-wave
// rule of choose_splits) even for four-wave tiles.
// F: MFMA form (16 or 32 rows); MT: slot tiles; NSUB: 16- or 32-row groups
// per wave; KC: k per chunk; NW: waves per workgroup; PD: prefetch depth;
// PK: packed planes; FILL: split policy of eight-wave tiles; CS: column
// split (waves per row unit)
struct GemmShape { int F, MT, NSUB, KC, NW, PD, PK, FILL = 0, CS = 1; };

constexpr int kT32 = 97;  // first slot count served by the 32x32 form

static int cu_count();

static GemmShape shape_for(int T, int vcols, bool raw, int K) {
    const bool wide = vcols % 256 == 0;
    // packed planes (2a + 1 tiles for 32a < T <= 32a + 16): split-K
    // partial GEMMs at 65..80 slots (QKV / O / down at T = 80: 29.5 / 23.7
    // / 53 us against 32.4 / 25.3 / 54 us for the 16x16 form), and every
    // GEMM at 97..112 slots (gate/up at T = 112: 147-175 us against 167-194)
    if (wide && raw && T > 64 && T <= 80) return {32, 5, 1, 64, 8, 2, 1};
    if (wide && T > 96 && T <= 112) return {32, 7, 1, 64, 8, 1, 1};
    if (T < kT32) {
        const int mt = std::max(2, (T + 15) / 16);
        // split-K partial GEMMs with few weight rows (the Qwen3-1.7B shapes):
        // when eight-wave tiles with at least two 128-k chunks per split
        // cannot fill 90% of the CUs, four-wave tiles with 64-k chunks give
        // twice the workgroups (QKV / O / down at T = 60: 7.9 / 6.5 / 9.4 us
        // against 10.2 / 8.9 / 11.6 us)
        if (raw && wide) {
            const int tiles8 = vcols / 256;
            const int s8 = std::min(std::max(1, K / 128 / 2), std::max(1, cu_count() / tiles8));
            if (10 * tiles8 * s8 < 9 * cu_count()) return GemmShape{16, mt, 2, 64, 4, 2, 0, 1};
        }
        // SwiGLU products of fewer than a quarter as many 256-row tiles as
        // CUs (the Qwen3-1.7B gate/up: 48): four-wave 128-row tiles, split
        // as the eight-wave ones are (two splits, 192 workgroups; one
        // machine at T = 60, then with a separate reduction kernel: gate/up
        // 25.7 -> 24.2 us per layer, the step 2.45-2.47 -> 2.42-2.43 ms;
        // four splits 26.4 us, three 28.3 us, unsplit 28.7 us).  The split
        // is now reduced by its last split (launch_gemm): 23.1 us.
        if (!raw && wide && vcols / 256 * 4 < cu_count()) return GemmShape{16, mt, 2, 64, 4, 2, 0, 1};
        // an lm_head over a short k (the Qwen3-1.7B one: 151936 x 2048,
        // weight-bound at these slot counts) on four-wave 128-row tiles:
        // 1187 shorter workgroups leave a shorter tail than 594 eight-wave
        // ones at one per CU (one machine at T = 60: 158 -> 143-148 us; the
        // Qwen3-32B lm_head at T = 80, MFMA-heavier, is slower that way:
        // 338-350 -> 359-363 us)
        if (!raw && !wide && vcols % 32 == 0 && K <= 2048) return GemmShape{16, mt, 2, 64, 4, 2, 0};
        // the lm_head (151936 rows: not a multiple of 256) takes the
        // eight-wave tiles too; its last workgroup has fewer units
        if (wide || (!raw && vcols % 32 == 0)) return GemmShape{16, mt, 2, 128, 8, 1, 0};
        return GemmShape{16, mt, 2, 64, 4, 2, 0};
    }
    const int mt = (T + 31) / 32;
    // eight-wave workgroups also for the lm_head, whose row count is not a
    // multiple of 256 (the workgroups then take 7 or 8 row units each)
    const bool w8 = wide || (!raw && vcols % 32 == 0);
    if (mt <= 4) return w8 ? GemmShape{32, mt, 1, 64, 8, 2, 0} : GemmShape{32, mt, 1, 64, 4, 2, 0};
    if (mt <= 7) return w8 ? GemmShape{32, mt, 1, 64, 8, 1, 0} : GemmShape{32, mt, 1, 64, 4, 1, 0};
    // 225..256 slots: eight waves with 32-k chunks (double-buffered staging
    // of 2 x 256 rows then fits one workgroup of 256 weight rows per CU);
    // probe on one machine at T = 240: gate/up 292 vs 392 us, QKV 63 vs 99, O 51
    // vs 93, down 143 vs 210 us against four waves with 64-k chunks
    if (mt <= 8) {
        // 64-row units shared by two waves (four slot tiles each) with 64-k
        // chunks: every B fragment feeds two MFMAs.  Timing on one machine of the
        // 32B shapes at T = 229 in isolation: gate/up 263 vs 293 us, QKV 57
        // vs 59, O 52 vs 56, down 121 vs 137 us against 32-row units
        if (vcols % 64 == 0) return GemmShape{32, 8, 2, 64, 8, 1, 0, 0, 2};
        return w8 ? GemmShape{32, 8, 1, 32, 8, 1, 0} : GemmShape{32, 8, 1, 64, 4, 1, 0};
    }
    if (mt <= 10) return {32, 10, 1, 32, 4, 1, 0};
    if (mt <= 13) return {32, 13, 1, 16, 4, 1, 0};
    return {0, 0, 0, 0, 0, 0, 0};
}

typedef void (*GemmFn)(GemmP);
typedef void (*ReduceFn)(GemmP);

// Activations always come as two planes (hi, lo); split-K kernels write raw
// partial planes and the epilogue runs in the reducer.
template <int F, int MT, int NW, int KC, int PD, bool SPLIT, bool PK = false, int CS = 1, int NS = 1>
static GemmFn pick_epi(int epi, bool skf = false) {
    if constexpr (F == 16) {
        if (SPLIT) return k_gemm16<MT, 2, KC, EPI_STORE, true, NW, 2, PD>;
        switch (epi) {
            case EPI_RESID: return k_gemm16<MT, 2, KC, EPI_RESID, false, NW, 2, PD>;
            case EPI_SWIGLU: return k_gemm16<MT, 2, KC, EPI_SWIGLU, false, NW, 2, PD>;
            case EPI_LMSTAT: return k_gemm16<MT, 2, KC, EPI_LMSTAT, false, NW, 2, PD>;
            default: return k_gemm16<MT, 2, KC, EPI_STORE, false, NW, 2, PD>;
        }
    } else {
        if constexpr (CS > 1 && !SPLIT)
            if (skf) return epi == EPI_SWIGLU ? k_gemm32<MT, NS, KC, EPI_SWIGLU, false, NW, 2, PD, PK, CS, true> : nullptr;
        if (SPLIT) return k_gemm32<MT, NS, KC, EPI_STORE, true, NW, 2, PD, PK, CS>;
        switch (epi) {
            case EPI_RESID: return k_gemm32<MT, NS, KC, EPI_RESID, false, NW, 2, PD, PK, CS>;
            case EPI_SWIGLU: return k_gemm32<MT, NS, KC, EPI_SWIGLU, false, NW, 2, PD, PK, CS>;
            case EPI_LMSTAT: return k_gemm32<MT, NS, KC, EPI_LMSTAT, false, NW, 2, PD, PK, CS>;
            default: return k_gemm32<MT, NS, KC, EPI_STORE, false, NW, 2, PD, PK, CS>;
        }
    }
}

template <int NW, bool SPLIT>
static GemmFn pick_nw(const GemmShape& sh, int epi) {
    constexpr int KC16 = NW == 8 ? 128 : 64, PD16 = NW == 8 ? 1 : 2;
    if (sh.F == 16) {
        switch (sh.MT) {
            case 2: return pick_epi<16, 2, NW, KC16, PD16, SPLIT>(epi);
            case 3: return pick_epi<16, 3, NW, KC16, PD16, SPLIT>(epi);
            case 4: return pick_epi<16, 4, NW, KC16, PD16, SPLIT>(epi);
            case 5: return pick_epi<16, 5, NW, KC16, PD16, SPLIT>(epi);
            case 6: return pick_epi<16, 6, NW, KC16, PD16, SPLIT>(epi);
        }
        return nullptr;
    }
    switch (sh.MT) {
        case 4: return pick_epi<32, 4, NW, 64, 2, SPLIT>(epi);
        case 5: return pick_epi<32, 5, NW, 64, 1, SPLIT>(epi);
        case 6: return pick_epi<32, 6, NW, 64, 1, SPLIT>(epi);
        case 7: return pick_epi<32, 7, NW, 64, 1, SPLIT>(epi);
    }
    return nullptr;
}

template <bool SPLIT>
static GemmFn pick(const GemmShape& sh, int epi, bool skf = false) {
    if (sh.PK) {
        if (sh.MT == 5) return SPLIT ? pick_epi<32, 5, 8, 64, 2, true, true>(epi) : nullptr;
        if (sh.MT == 7) return pick_epi<32, 7, 8, 64, 1, SPLIT, true>(epi);
        return nullptr;
    }
    if (sh.F == 32 && sh.MT == 8) {
        if (sh.CS == 2) return pick_epi<32, 8, 8, 64, 1, SPLIT, false, 2, 2>(epi, skf);
        return sh.NW == 8 ? pick_epi<32, 8, 8, 32, 1, SPLIT>(epi) : pick_epi<32, 8, 4, 64, 1, SPLIT>(epi);
    }
    if (sh.F == 32 && sh.MT == 10) return pick_epi<32, 10, 4, 32, 1, SPLIT>(epi);
    if (sh.F == 32 && sh.MT == 13) return pick_epi<32, 13, 4, 16, 1, SPLIT>(epi);
    return sh.NW == 8 ? pick_nw<8, SPLIT>(sh, epi) : pick_nw<4, SPLIT>(sh, epi);
}

// the last-split SwiGLU product on the four-wave 16x16 tiles
static GemmFn pick_la(const GemmShape& sh) {
    if (sh.F != 16 || sh.NW != 4 || sh.NSUB != 2 || sh.KC != 64 || sh.PD != 2) return nullptr;
    switch (sh.MT) {
        case 2: return k_gemm16<2, 2, 64, EPI_SWIGLU, false, 4, 2, 2, 16, true>;
        case 3: return k_gemm16<3, 2, 64, EPI_SWIGLU, false, 4, 2, 2, 16, true>;
        case 4: return k_gemm16<4, 2, 64, EPI_SWIGLU, false, 4, 2, 2, 16, true>;
        case 5: return k_gemm16<5, 2, 64, EPI_SWIGLU, false, 4, 2, 2, 16, true>;
        case 6: return k_gemm16<6, 2, 64, EPI_SWIGLU, false, 4, 2, 2, 16, true>;
    }
    return nullptr;
}

static ReduceFn pick_reduce(int epi) {
    switch (epi) {
        case EPI_RESID: return k_splitk_reduce<EPI_RESID>;
        case EPI_SWIGLU: return k_splitk_reduce<EPI_SWIGLU>;
        default: return k_splitk_reduce<EPI_STORE>;
    }
}

static int cu_count() {  // cached
    static int n = 0;
    if (n == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
            n = 256;
    }
    return n;
}

// k splits.  Four-wave tiles (a divisor of kchunks): the largest count
// giving 1.25 to 1.75 workgroups per CU, else the smallest giving at least
// 1.25.  Eight-wave tiles (one workgroup per CU fits in LDS): the largest
// count keeping the grid within one wave of workgroups, splits of unequal
// chunk counts allowed, at least two chunks per split (measured on the 32B
// shapes at T = 80: QKV 40 tiles x 6 = 240 workgroups 27.2 us vs x 5
// 30.7 us, O 20 x 12 23.9 vs x 8 27.4, down 20 x 12 52.6 vs x 10 57.1; the
// extra partial sums cost the consumers less than the idle CUs cost the
// GEMM.  On the 1.7B shapes one-chunk splits lose to pipeline start-up and
// partial-sum traffic: the step goes from 2.99 to 2.77 ms with two).
static int choose_splits(int tiles, int kchunks, int nw) {
    if (nw == 8) {
        const int hi = cu_count();
        if (tiles * 2 > hi) return 1;
        return std::max(1, std::min(std::max(1, kchunks / 2), hi / tiles));
    }
    const int lo = cu_count() * 5 / 4, hi = cu_count() * 7 / 4;
    if (tiles >= lo) return 1;
    int best = 0;
    for (int s = 2; s <= kchunks; ++s)
        if (kchunks % s == 0 && tiles * s >= lo && tiles * s <= hi) best = s;
    if (best) return best;
    for (int s = 2; s <= kchunks; ++s)
        if (kchunks % s == 0 && tiles * s >= lo) return s;
    return kchunks;
}

size_t gemm_partial_floats(const Dims& D, int Tmax) {
    // fp32 path: one plane of the widest raw output
    if (!D.bf16) return (size_t)Tmax * (size_t)std::max(D.nqkv(), D.d);
    // the split count is bounded by the CU count over the tile count, so
    // S * vcols <= ~2 * (CUs * NT) for every call; reserve generously
    // (three planes' worth also holds the stream-K partial slots of the
    // gate/up product at 225-256 slots: 200 tiles x 2 x 65536 floats on the
    // Qwen3-32B shape)
    const size_t widest = (size_t)std::max(std::max(D.nqkv(), D.d), 2 * D.F);
    return (size_t)Tmax * std::max<size_t>(widest * 3, (size_t)65536);
}


int launch_gemm(const Dims& D, const GemmCall& g, const SlotBufs& sb, hipStream_t s) {
    if (!D.bf16) {
        GemmF p;
        p.X = (const float*)g.X;
        p.W0 = (const float*)g.W[0];
        p.W1 = (const float*)(g.nseg > 1 ? g.W[1] : g.W[0]);
        p.W2 = (const float*)(g.nseg > 2 ? g.W[2] : g.W[0]);
        p.seg1 = g.nseg > 1 ? g.seg[1] : (1 << 30);
        p.seg2 = g.nseg > 2 ? g.seg[2] : (1 << 30);
        p.N = g.N;
        p.K = g.K;
        p.T = g.T;
        p.epi = g.raw ? EPI_STORE : g.epi;
        p.out = g.raw ? sb.gpart : (float*)g.out;
        p.ldo = g.raw ? g.N : g.ldo;
        const int n = g.T * g.N;
        hipLaunchKernelGGL(k_gemm_f32, dim3((n + 255) / 256), dim3(256), 0, s, p);
        return 1;
    }
    const int vcols = g.epi == EPI_SWIGLU ? 2 * g.N : g.N;
    const GemmShape sh = shape_for(g.T, vcols, g.raw != 0, g.K);
    const int unit_rows = sh.F * sh.NSUB;  // weight rows of one row unit
    GemmP p;
    p.X = (const bf16_t*)g.X;
    p.Wp = (const bf16_t*)g.Wp;
    p.K = g.K;
    p.KT = g.K / 32;
    p.T = g.T;
    p.kchunks = g.K / sh.KC;
    p.vcols = vcols;
    // workgroups of NW waves; a last partial workgroup when the row count is
    // not a multiple of NW units (its surplus waves load and store nothing)
    const int units = p.vcols / unit_rows;
    const int upw = sh.NW / sh.CS;  // row units per workgroup
    p.tiles = (units + upw - 1) / upw;
    int S = g.epi == EPI_LMSTAT ? 1 : choose_splits(p.tiles, p.kchunks, sh.FILL ? 8 : sh.NW);
    // four-wave split-K tiles over a short k (the Qwen3-1.7B QKV and O
    // projections, k = 2048): half the splits, so each split keeps four
    // 64-k chunks and the consumer reads half the partial planes (one
    // machine at T = 60, each with its consumer: QKV 18.8 -> 18.4 us, O
    // 14.3 -> 14.0 us per layer; the down projection, k = 6144, is slower
    // so: 19.4 -> 20.0 us)
    if (g.raw && sh.NW == 4 && sh.FILL && g.K <= 2048) S = std::max(1, S / 2);
    while (S > 1 && (size_t)S * g.T * p.vcols > sb.gpart_floats) {
        int t = S - 1;
        while (t > 1 && p.kchunks % t) --t;
        S = t;
    }
    p.S = S;
    p.G = units;
    p.WPS = p.tiles;
    p.part = sb.gpart;
    p.out = g.out;
    p.ldo = g.ldo;
    p.oplane = (size_t)g.T * g.ldo;  // SwiGLU output planes are [2][T][ldo]
    p.nss = g.norm_ss;
    p.nnb = g.norm_nb;
    p.eps = D.eps;
    p.lstat = reinterpret_cast<VStat*>(g.lstat);
    p.zd = g.zd;
    p.dnext = g.dnext;
    if (g.groups_out) *g.groups_out = p.tiles;
    // Stream-K for an unsplit column-split SwiGLU product that leaves CUs
    // idle (gate/up at 225-256 slots: 200 row tiles of 256 rows on 256 CUs)
    p.sk_nwg = 0;
    p.sk_maxp = 0;
    p.pkl = sh.CS > 1 && sh.MT == 8 && g.T > 224 && g.T <= 240;
    p.sk_polls = g.sk_polls;
    p.sk_cnt = g.sk_cnt;
    p.flags = g.flags;
    if (!g.raw && g.epi == EPI_SWIGLU && sh.CS > 1 && S == 1 && g.sk_cnt && g.flags &&
        p.tiles < cu_count() && p.tiles <= kSkCounters) {
        const int total = p.tiles * p.kchunks, nwg = std::min(cu_count(), total);
        int maxp = 0;  // most pieces of a tile before its last
        for (int t = 0; t < p.tiles; ++t)
            maxp = std::max(maxp, sk_owner(t * p.kchunks + p.kchunks - 1, total, nwg) -
                                      sk_owner(t * p.kchunks, total, nwg));
        const size_t slot_floats = (size_t)64 * sh.NW * sh.NSUB * (sh.MT / sh.CS) * 16;
        if (maxp >= 1 && (size_t)p.tiles * maxp * slot_floats <= sb.gpart_floats) {
            p.sk_nwg = nwg;
            p.sk_maxp = maxp;
            hipLaunchKernelGGL(pick<false>(sh, g.epi, true), dim3(nwg), dim3(64 * sh.NW), 0, s, p);
            return 1;
        }
    }
    if (g.raw) {
        // S partial planes [S][T][N] for a fused consumer to reduce
        hipLaunchKernelGGL(pick<true>(sh, EPI_STORE), dim3(p.tiles * S), dim3(64 * sh.NW), 0, s, p);
    } else if (S == 1) {
        hipLaunchKernelGGL(pick<false>(sh, g.epi), dim3(p.tiles), dim3(64 * sh.NW), 0, s, p);
    } else {
        // a split SwiGLU product on four-wave tiles: its last split adds the
        // others' sums (slots of NTH x NSUB x MT x 4 floats per split and
        // tile) and runs the epilogue, no reduction kernel
        const size_t la_floats = (size_t)p.tiles * S * (64 * sh.NW) * sh.NSUB * sh.MT * 4;
        const GemmFn la = g.epi == EPI_SWIGLU && g.sk_cnt && p.tiles <= kSkCounters && la_floats <= sb.gpart_floats
                              ? pick_la(sh)
                              : nullptr;
        if (la) {
            hipLaunchKernelGGL(la, dim3(p.tiles * S), dim3(64 * sh.NW), 0, s, p);
            return S;
        }
        hipLaunchKernelGGL(pick<true>(sh, g.epi), dim3(p.tiles * S), dim3(64 * sh.NW), 0, s, p);
        const int ncols = g.epi == EPI_SWIGLU ? p.vcols / 2 : p.vcols;
        const int n = g.T * (ncols / 4);
        hipLaunchKernelGGL(pick_reduce(g.epi), dim3((n + 255) / 256), dim3(256), 0, s, p);
    }
    return S;
}

}  // namespace sdv
