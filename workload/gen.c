/*
 * Seeded synthetic inputs for the speculative-verify workloads.
 *
 * This module holds no arithmetic of the verify method: it only produces
 * weights, cached keys/values, token ids, draft distributions and uniforms.
 * Both the CPU oracle and the GPU path consume what it writes, so neither
 * side generates its own inputs.
 *
 * Every value is a pure function of (seed, stream, index): stream names the
 * tensor (layer, kind), index is the flat row-major element index.  The
 * bit source is the splitmix64 sequence (Steele, Lea, Flood, OOPSLA 2014)
 * started at a per-(seed, stream) state, so results do not depend on thread
 * count or chunking.
 *
 * "Normal" values are an Irwin-Hall sum of four 16-bit uniforms, centred and
 * scaled to the requested standard deviation.  The construction is integer
 * arithmetic plus one correctly rounded fp32 multiply, so it is bit-identical
 * on every IEEE machine; bf16 outputs are the round-to-nearest-even of that
 * fp32 value.
 */
#include <stdint.h>
#include <stddef.h>
#include <math.h>

#define GOLDEN 0x9e3779b97f4a7c15ULL

static inline uint64_t fin64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

/* state for (seed, stream) */
static inline uint64_t wl_key(uint64_t seed, uint64_t stream) {
    return fin64(fin64(seed + GOLDEN) ^ (stream * 0xd1b54a32d192ed03ULL + 0x2545f4914f6cdd1dULL));
}

/* i-th output of the splitmix64 sequence started at state `key` */
static inline uint64_t wl_bits(uint64_t key, uint64_t i) {
    return fin64(key + (i + 1) * GOLDEN);
}

uint64_t wl_raw(uint64_t seed, uint64_t stream, uint64_t i) {
    return wl_bits(wl_key(seed, stream), i);
}

/* std of (sum of four U{0..65535}) - 131070 is sqrt((2^32-1)/3) */
#define IH4_STD 37837.2270017029f

static inline float ih4(uint64_t b, float scale) {
    int32_t s = (int32_t)(b & 0xffff) + (int32_t)((b >> 16) & 0xffff) +
                (int32_t)((b >> 32) & 0xffff) + (int32_t)((b >> 48) & 0xffff) - 131070;
    return (float)s * scale; /* |s| < 2^18: exact in fp32, one rounding in the multiply */
}

static inline uint16_t f32_to_bf16_rne(float f) {
    union { float f; uint32_t u; } v = { f };
    uint32_t u = v.u;
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffff) ? 0x40 : 0));
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

void wl_fill_normal_f32(float* out, int64_t n, uint64_t seed, uint64_t stream,
                        int64_t offset, float std) {
    const uint64_t key = wl_key(seed, stream);
    const float scale = std / IH4_STD;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = ih4(wl_bits(key, (uint64_t)(offset + i)), scale);
}

void wl_fill_normal_bf16(uint16_t* out, int64_t n, uint64_t seed, uint64_t stream,
                         int64_t offset, float std) {
    const uint64_t key = wl_key(seed, stream);
    const float scale = std / IH4_STD;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = f32_to_bf16_rne(ih4(wl_bits(key, (uint64_t)(offset + i)), scale));
}

/* uniform in [lo, hi) as fp32, 24-bit grid */
void wl_fill_uniform_f32(float* out, int64_t n, uint64_t seed, uint64_t stream,
                         int64_t offset, float lo, float hi) {
    const uint64_t key = wl_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        float u = (float)(wl_bits(key, (uint64_t)(offset + i)) >> 40) * 0x1.0p-24f;
        out[i] = lo + (hi - lo) * u;
    }
}

/* bf16 version of the above (norm gains in tests) */
void wl_fill_uniform_bf16(uint16_t* out, int64_t n, uint64_t seed, uint64_t stream,
                          int64_t offset, float lo, float hi) {
    const uint64_t key = wl_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        float u = (float)(wl_bits(key, (uint64_t)(offset + i)) >> 40) * 0x1.0p-24f;
        out[i] = f32_to_bf16_rne(lo + (hi - lo) * u);
    }
}

/* integers uniform in [lo, hi] (inclusive), multiply-shift range reduction */
void wl_fill_int(int32_t* out, int64_t n, uint64_t seed, uint64_t stream, int64_t offset,
                 int32_t lo, int32_t hi) {
    const uint64_t key = wl_key(seed, stream);
    const uint64_t span = (uint64_t)((int64_t)hi - (int64_t)lo + 1);
    for (int64_t i = 0; i < n; ++i) {
        uint64_t b = wl_bits(key, (uint64_t)(offset + i)) >> 32;
        out[i] = lo + (int32_t)((b * span) >> 32);
    }
}

/*
 * Draft distributions: for each of `rows` rows, q = mix * softmax(sa * g_a)
 * + (1 - mix) * softmax(sb * g_b) with g_a, g_b the normal streams
 * (stream_a, stream_b) at row offset r * vocab.  mix = 1 gives a single
 * softmax.  Then one draft token per row is drawn from q by inverse CDF with
 * a 53-bit uniform from stream_u.  Computed in double, q stored as fp32.
 */
void wl_draft_rows(float* q, int32_t* tok, int64_t rows, int64_t vocab, uint64_t seed,
                   uint64_t stream_a, float sa, uint64_t stream_b, float sb, float mix,
                   uint64_t stream_u, int64_t row_offset) {
    const uint64_t ka = wl_key(seed, stream_a), kb = wl_key(seed, stream_b);
    const uint64_t ku = wl_key(seed, stream_u);
    const float scale = 1.0f / IH4_STD;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < rows; ++r) {
        float* qr = q + r * vocab;
        const uint64_t base = (uint64_t)((r + row_offset) * vocab);
        double ma = -INFINITY, mb = -INFINITY;
        for (int64_t k = 0; k < vocab; ++k) {
            double a = (double)sa * ih4(wl_bits(ka, base + k), scale);
            if (a > ma) ma = a;
            if (mix < 1.0f) {
                double b = (double)sb * ih4(wl_bits(kb, base + k), scale);
                if (b > mb) mb = b;
            }
        }
        double za = 0.0, zb = 0.0;
        for (int64_t k = 0; k < vocab; ++k) {
            za += exp((double)sa * ih4(wl_bits(ka, base + k), scale) - ma);
            if (mix < 1.0f) zb += exp((double)sb * ih4(wl_bits(kb, base + k), scale) - mb);
        }
        double cum = 0.0;
        const double u = (double)(wl_bits(ku, (uint64_t)(r + row_offset)) >> 11) * 0x1.0p-53;
        int32_t pick = -1;
        for (int64_t k = 0; k < vocab; ++k) {
            double v = (double)mix * exp((double)sa * ih4(wl_bits(ka, base + k), scale) - ma) / za;
            if (mix < 1.0f)
                v += (1.0 - (double)mix) *
                     exp((double)sb * ih4(wl_bits(kb, base + k), scale) - mb) / zb;
            qr[k] = (float)v;
            cum += v;
            if (pick < 0 && u < cum && qr[k] > 0.0f) pick = (int32_t)k;
        }
        if (pick < 0) { /* u fell in the rounding gap at the top: last nonzero entry */
            for (int64_t k = vocab - 1; k >= 0; --k)
                if (qr[k] > 0.0f) { pick = (int32_t)k; break; }
        }
        tok[r] = pick;
    }
}
