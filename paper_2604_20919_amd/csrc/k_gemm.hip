// Skinny GEMMs of the verify forward: Y[t][n] = sum_k X[t][k] W[n][k] for
// T = sum(l_m + 1) query slots (tens to a few hundred) against weight
// matrices of thousands of rows.  At these shapes the work is bound by
// streaming the weights from HBM once, so the kernel is built around that
// stream:
//   * weights are read in place, row-major [out][in]; each lane loads 16
//     contiguous bytes (8 bf16 along k) straight into the A operand of
//     v_mfma_f32_16x16x32_bf16 (16 weight rows x 32 k);
//   * the activation chunk X[0:T][k0:k0+KC] is staged once per workgroup in
//     LDS and read by the 4 waves as the B operand (32 k x 16 slots);
//   * each wave owns NSUB groups of 16 weight rows and all T slots, so every
//     weight byte is read exactly once per call;
//   * the k range is split over S workgroups when there are too few column
//     tiles to fill the GPU; partial sums go to a workspace and the last
//     workgroup of a tile (atomic arrival counter) adds them in split order,
//     so results are bit-identical from run to run;
//   * the epilogue is fused: plain fp32 store, residual add into the fp32
//     stream, or SwiGLU silu(g) * u with gate/up rows interleaved per wave.
// An fp32 fallback (plain FMA loop) serves the fp32 model configuration.
#include <map>
#include <tuple>

#include "sdv_device.h"
#include "sdv_internal.h"

namespace sdv {

struct GemmP {
    const bf16_t* X;
    const bf16_t* W0;
    const bf16_t* W1;
    const bf16_t* W2;
    int seg1, seg2;  // first virtual column of segments 1 and 2
    int K, T, S, kchunks, tiles;
    float* part;
    int32_t* cnt;
    void* out;
    int ldo;
};

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }

template <int MT, int NSUB, int KC, int EPI>
__global__ __launch_bounds__(256) void k_gemm_bf16(GemmP p) {
    constexpr int NT = 4 * NSUB * 16;  // virtual columns per tile
    constexpr int KS = KC / 32;        // MFMA k-steps per chunk
    constexpr int LDX = KC + 8;        // padded LDS row (bf16 elements)
    __shared__ __attribute__((aligned(16))) bf16_t xs[MT * 16 * LDX];
    __shared__ int last_flag;

    const int tile = blockIdx.x / p.S, split = blockIdx.x % p.S;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int lr = lane & 15, lg = lane >> 4;
    const int mt_act = (p.T + 15) >> 4;

    // weight row of this lane for each sub-tile
    const bf16_t* wrow[NSUB];
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
        if (EPI == EPI_SWIGLU) {
            const int col = tile * (NT / 2) + (wave * (NSUB / 2) + s / 2) * 16 + lr;
            wrow[s] = ((s & 1) ? p.W1 : p.W0) + (size_t)col * p.K;
        } else {
            const int v = tile * NT + (wave * NSUB + s) * 16 + lr;
            const bf16_t* w = v < p.seg1 ? p.W0 + (size_t)v * p.K
                              : v < p.seg2 ? p.W1 + (size_t)(v - p.seg1) * p.K
                                           : p.W2 + (size_t)(v - p.seg2) * p.K;
            wrow[s] = w;
        }
        wrow[s] += 8 * lg;
    }

    f32x4 acc[NSUB][MT];
#pragma unroll
    for (int s = 0; s < NSUB; ++s)
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[s][m] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int c_begin = split * p.kchunks / p.S;
    const int c_end = (split + 1) * p.kchunks / p.S;

    bf16x8 wcur[KS][NSUB], wnxt[KS][NSUB];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
            wcur[ks][s] = *(const bf16x8*)(wrow[s] + (size_t)c_begin * KC + ks * 32);

    constexpr int PIECES = MT * 16 * (KC / 8);
    for (int c = c_begin; c < c_end; ++c) {
        if (c + 1 < c_end) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                for (int s = 0; s < NSUB; ++s)
                    wnxt[ks][s] = *(const bf16x8*)(wrow[s] + (size_t)(c + 1) * KC + ks * 32);
        }
        // stage X[0:16*mt_act][c*KC : (c+1)*KC] (rows >= T are zero)
        for (int i = threadIdx.x; i < mt_act * 16 * (KC / 8); i += 256) {
            const int r = i / (KC / 8), cc = i % (KC / 8);
            uint4 v = {0u, 0u, 0u, 0u};
            if (r < p.T) v = *(const uint4*)(p.X + (size_t)r * p.K + (size_t)c * KC + cc * 8);
            *(uint4*)(xs + r * LDX + cc * 8) = v;
        }
        (void)PIECES;
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                if (m < mt_act) {
                    const bf16x8 xf = *(const bf16x8*)(xs + (m * 16 + lr) * LDX + ks * 32 + 8 * lg);
#pragma unroll
                    for (int s = 0; s < NSUB; ++s)
                        acc[s][m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wcur[ks][s], xf,
                                                                             acc[s][m], 0, 0, 0);
                }
            }
        }
        __syncthreads();
        if (c + 1 < c_end) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                for (int s = 0; s < NSUB; ++s) wcur[ks][s] = wnxt[ks][s];
        }
    }

    // lane holds D[n = 4*lg + r][t = lr] of each (sub-tile, slot tile)
    if (p.S > 1) {
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const int t = m * 16 + lr;
                if (m < mt_act && t < p.T) {
                    float* dst = p.part + ((size_t)(tile * p.S + split) * p.T + t) * NT +
                                 (wave * NSUB + s) * 16 + 4 * lg;
                    *(f32x4*)dst = acc[s][m];
                }
            }
        __threadfence();
        __syncthreads();
        if (threadIdx.x == 0) last_flag = (atomicAdd(p.cnt + tile, 1) == p.S - 1);
        __syncthreads();
        if (!last_flag) return;
        __threadfence();
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const int t = m * 16 + lr;
                if (m < mt_act && t < p.T) {
                    f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
                    for (int sp = 0; sp < p.S; ++sp)
                        sum += *(const f32x4*)(p.part + ((size_t)(tile * p.S + sp) * p.T + t) * NT +
                                               (wave * NSUB + s) * 16 + 4 * lg);
                    acc[s][m] = sum;
                }
            }
        if (threadIdx.x == 0) p.cnt[tile] = 0;
    }

#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const int t = m * 16 + lr;
        if (!(m < mt_act && t < p.T)) continue;
        if (EPI == EPI_SWIGLU) {
#pragma unroll
            for (int s = 0; s < NSUB; s += 2) {
                const int col = tile * (NT / 2) + (wave * (NSUB / 2) + s / 2) * 16 + 4 * lg;
                bf16_t* o = (bf16_t*)p.out + (size_t)t * p.ldo + col;
                const f32x4 g = acc[s][m], u = acc[s + 1][m];
                uint2 pk;
                pk.x = (uint32_t)f32_to_bf16(silu(g[0]) * u[0]) |
                       ((uint32_t)f32_to_bf16(silu(g[1]) * u[1]) << 16);
                pk.y = (uint32_t)f32_to_bf16(silu(g[2]) * u[2]) |
                       ((uint32_t)f32_to_bf16(silu(g[3]) * u[3]) << 16);
                *(uint2*)o = pk;
            }
        } else {
#pragma unroll
            for (int s = 0; s < NSUB; ++s) {
                const int col = tile * NT + (wave * NSUB + s) * 16 + 4 * lg;
                float* o = (float*)p.out + (size_t)t * p.ldo + col;
                if (EPI == EPI_RESID) {
                    f32x4 v = *(f32x4*)o;
                    v += acc[s][m];
                    *(f32x4*)o = v;
                } else {
                    *(f32x4*)o = acc[s][m];
                }
            }
        }
    }
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
namespace {

constexpr int kNSub = 2;
constexpr int kNT = 4 * kNSub * 16;

struct Shape { int MT, KC; };

Shape shape_for(int T) {
    const int mt = (T + 15) / 16;
    static const int classes[] = {2, 4, 6, 8, 12, 16, 20, 26};
    for (int c : classes)
        if (mt <= c) return {c, c <= 8 ? 256 : (c <= 16 ? 128 : 64)};
    return {0, 0};
}

typedef void (*GemmFn)(GemmP);

template <int MT, int KC>
GemmFn pick_epi(int epi) {
    switch (epi) {
        case EPI_RESID: return k_gemm_bf16<MT, kNSub, KC, EPI_RESID>;
        case EPI_SWIGLU: return k_gemm_bf16<MT, kNSub, KC, EPI_SWIGLU>;
        default: return k_gemm_bf16<MT, kNSub, KC, EPI_STORE>;
    }
}

GemmFn pick(const Shape& sh, int epi) {
    switch (sh.MT) {
        case 2: return pick_epi<2, 256>(epi);
        case 4: return pick_epi<4, 256>(epi);
        case 6: return pick_epi<6, 256>(epi);
        case 8: return pick_epi<8, 256>(epi);
        case 12: return pick_epi<12, 128>(epi);
        case 16: return pick_epi<16, 128>(epi);
        case 20: return pick_epi<20, 64>(epi);
        case 26: return pick_epi<26, 64>(epi);
    }
    return nullptr;
}

int resident_blocks(GemmFn fn) {
    static std::map<GemmFn, int> cache;
    auto it = cache.find(fn);
    if (it != cache.end()) return it->second;
    int per_cu = 1, cus = 256, dev = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)fn, 256, 0) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    if (hipGetDevice(&dev) == hipSuccess)
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int n = per_cu * cus;
    cache[fn] = n;
    return n;
}

// number of k splits: the largest divisor of kchunks that keeps every
// workgroup resident at once (so all of them stream weights concurrently)
int choose_splits(int tiles, int kchunks, int capacity) {
    int best = 1;
    for (int s = 1; s <= kchunks; ++s)
        if (kchunks % s == 0 && (long)tiles * s <= capacity) best = s;
    return best;
}

}  // namespace

size_t gemm_partial_floats(const Dims& D, int Tmax) {
    if (!D.bf16) return 0;
    // worst case: every call uses at most 32 splits of the widest non-SwiGLU output
    const int nmax = D.nqkv() > D.d ? D.nqkv() : D.d;
    return (size_t)32 * Tmax * nmax;
}

int gemm_counter_count(const Dims& D) {
    const int v = 2 * D.F > D.nqkv() ? 2 * D.F : D.nqkv();
    return (v > D.V ? v : D.V) / 16 + 64;
}

void launch_gemm(const Dims& D, const GemmCall& g, const SlotBufs& sb, hipStream_t s) {
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
        p.epi = g.epi;
        p.out = (float*)g.out;
        p.ldo = g.ldo;
        const int n = g.T * g.N;
        hipLaunchKernelGGL(k_gemm_f32, dim3((n + 255) / 256), dim3(256), 0, s, p);
        return;
    }
    const Shape sh = shape_for(g.T);
    GemmFn fn = pick(sh, g.epi);
    const int vcols = g.epi == EPI_SWIGLU ? 2 * g.N : g.N;
    GemmP p;
    p.X = (const bf16_t*)g.X;
    p.W0 = (const bf16_t*)g.W[0];
    p.W1 = (const bf16_t*)(g.nseg > 1 ? g.W[1] : g.W[0]);
    p.W2 = (const bf16_t*)(g.nseg > 2 ? g.W[2] : g.W[0]);
    p.seg1 = g.nseg > 1 ? g.seg[1] : (1 << 30);
    p.seg2 = g.nseg > 2 ? g.seg[2] : (1 << 30);
    p.K = g.K;
    p.T = g.T;
    p.kchunks = g.K / sh.KC;
    p.tiles = vcols / kNT;
    int S = 1;
    if (g.epi != EPI_SWIGLU || true) S = choose_splits(p.tiles, p.kchunks, resident_blocks(fn));
    // the partial buffer bounds the split count
    while (S > 1 && (size_t)S * g.T * (size_t)p.tiles * kNT > sb.gpart_floats) {
        int t = S - 1;
        while (t > 1 && p.kchunks % t) --t;
        S = t;
    }
    p.S = S;
    p.part = sb.gpart;
    p.cnt = sb.gcount;
    p.out = g.out;
    p.ldo = g.ldo;
    hipLaunchKernelGGL(fn, dim3(p.tiles * S), dim3(256), 0, s, p);
}

// shape checks used by the runtime before anything is enqueued
bool gemm_shape_ok(const Dims& D, int T, int K, int N, int epi) {
    if (!D.bf16) return true;
    const Shape sh = shape_for(T);
    if (sh.MT == 0) return false;
    const int vcols = epi == EPI_SWIGLU ? 2 * N : N;
    return K % sh.KC == 0 && vcols % kNT == 0;
}

}  // namespace sdv
