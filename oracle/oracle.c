/*
 * oracle.c -- plain CPU reference for the batched speculative-verify pass.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or helper with
 * the GPU library.
 *
 * What it computes (DiP-SD, arXiv 2604.20919):
 *   - the verification step of one speculative-decoding round (Sec. II-A,
 *     step 2): one target-model forward over every user's root token plus
 *     its l_m draft tokens, then the first-mismatch rule with one bonus token
 *     per user;
 *   - the accept/resample rule itself is the standard speculative sampling
 *     the paper builds on (Sec. I, the accept/reject-and-resample procedures
 *     that preserve the target distribution): accept draft d with probability
 *     min(1, p(d)/q(d)); on the first rejection draw from norm(max(0, p - q));
 *     if every draft is accepted draw the bonus token from p.
 *
 * The forward is a pre-RMSNorm decoder with grouped-query attention, optional
 * per-head QK-RMSNorm, rotate-half RoPE and a SwiGLU FFN (the Qwen3 shape the
 * paper evaluates in Sec. IV-A, Table II).  Dot products and softmax sums are
 * accumulated in double and activations are kept in double.  When kv_bf16
 * is set (bf16 models) the keys and values of the new slots are rounded to
 * bf16 after QK-norm and RoPE, because that is what a bf16 KV cache stores and
 * what later slots of the same batch read back; the cached prefix is given
 * in bf16 already.  The paper fixes no precision; weights and the KV cache
 * are the only bf16 quantities of this reading.
 *
 * Sampler decisions are taken in fp32 (the precision of the GPU sampler):
 * r = p(d)/q(d) is an fp32 division compared with an fp32 uniform, and race
 * keys w/E are fp32 divisions.  Probabilities are computed in double and
 * rounded to fp32 once.
 *
 * Random draws use Philox-4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11),
 * written here from the paper's definition.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* threads the OpenMP loops of this file run on */
int or_omp_threads(void) { return omp_get_max_threads(); }

/* ------------------------------------------------------------------ */
/* Philox-4x64-10                                                      */
/* ------------------------------------------------------------------ */

static inline void mulhilo64(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo) {
    unsigned __int128 p = (unsigned __int128)a * b;
    *lo = (uint64_t)p;
    *hi = (uint64_t)(p >> 64);
}

/* One Philox-4x64 bijection with 10 rounds.  Each round multiplies words 0
 * and 2 by the two round constants, swaps the halves and xors in the round
 * key; the key advances by the Weyl constants between rounds. */
void or_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ULL, M1 = 0xCA5A826395121157ULL;
    const uint64_t W0 = 0x9E3779B97F4A7C15ULL, W1 = 0xBB67AE8584CAA73BULL;
    uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) { k0 += W0; k1 += W1; }
        uint64_t hi0, lo0, hi1, lo1;
        mulhilo64(M0, c0, &hi0, &lo0);
        mulhilo64(M1, c2, &hi1, &lo1);
        uint64_t n0 = hi1 ^ c1 ^ k0;
        uint64_t n1 = lo1;
        uint64_t n2 = hi0 ^ c3 ^ k1;
        uint64_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Counter layout for the sampler's draws: (round, user, purpose<<32 | slot,
 * k/4), key (seed, 0); word k%4 of the output block. */
enum { OR_PURPOSE_ACCEPT = 1, OR_PURPOSE_RACE = 2 };

static uint64_t draw64(uint64_t seed, uint64_t round, uint64_t user, uint64_t purpose,
                       uint64_t slot, uint64_t k) {
    uint64_t ctr[4] = { round, user, (purpose << 32) | slot, k >> 2 };
    uint64_t key[2] = { seed, 0 };
    uint64_t out[4];
    or_philox4x64_10(ctr, key, out);
    return out[k & 3];
}

/* accept uniform: top 24 bits, u in [0, 1) */
float or_accept_uniform(uint64_t x) { return (float)(x >> 40) * 0x1.0p-24f; }

/* race uniform: 24 significant bits below the leading one, V in [2^-64, 1) */
float or_race_uniform(uint64_t x) {
    if (x == 0) return 0.0f;
    int lz = __builtin_clzll(x);
    uint64_t mant = (x << lz) >> 40;
    return ldexpf((float)mant, -24 - lz);
}

/* unit exponential E = -log(1 - V), rounded to fp32 */
float or_race_exponential(uint64_t x) {
    double v = (double)or_race_uniform(x);
    return (float)(-log1p(-v));
}

/* ------------------------------------------------------------------ */
/* numerics helpers                                                    */
/* ------------------------------------------------------------------ */

static inline float bf16_bits_to_f32(uint16_t h) {
    union { uint32_t u; float f; } v = { (uint32_t)h << 16 };
    return v.f;
}

/* round to fp32, then to bf16 with round-to-nearest-even */
double or_round_bf16(double x) {
    union { float f; uint32_t u; } v = { (float)x };
    if ((v.u & 0x7f800000u) == 0x7f800000u) return (double)v.f;
    v.u = (v.u + 0x7fffu + ((v.u >> 16) & 1u)) & 0xffff0000u;
    return (double)v.f;
}

/* element i of a weight array stored as fp32 (dt 0) or bf16 (dt 1) */
static inline double wget(const void* p, size_t i, int dt) {
    return dt ? (double)bf16_bits_to_f32(((const uint16_t*)p)[i]) : (double)((const float*)p)[i];
}

/* y = x / sqrt(mean(x^2) + eps) * gamma  (gamma == NULL means 1) */
void or_rmsnorm(const double* x, int n, const void* gamma, int gdt, double eps, double* y) {
    double ss = 0.0;
    for (int i = 0; i < n; ++i) ss += x[i] * x[i];
    double r = 1.0 / sqrt(ss / n + eps);
    for (int i = 0; i < n; ++i) y[i] = x[i] * r * (gamma ? wget(gamma, i, gdt) : 1.0);
}

/* rotate-half RoPE on one head vector v[hd] at absolute position pos:
 * for a < hd/2, angle = pos * base^(-2a/hd); the pair (v[a], v[a+hd/2]) is
 * rotated by that angle. */
void or_rope(double* v, int hd, double pos, double base) {
    int h = hd / 2;
    for (int a = 0; a < h; ++a) {
        double ang = pos * pow(base, -2.0 * a / hd);
        double c = cos(ang), s = sin(ang);
        double x0 = v[a], x1 = v[a + h];
        v[a] = x0 * c - x1 * s;
        v[a + h] = x1 * c + x0 * s;
    }
}

/* single-head attention: o = sum_t softmax(q.k_t * scale)_t v_t over n rows
 * of k and v (row stride ld).  Plain two-pass softmax in double. */
void or_attend(const double* q, const double* k, const double* v, int n, int hd, long ld,
               double scale, double* o) {
    double* s = (double*)malloc(sizeof(double) * (n > 0 ? n : 1));
    double mx = -INFINITY;
    for (int t = 0; t < n; ++t) {
        double acc = 0.0;
        for (int d = 0; d < hd; ++d) acc += q[d] * k[t * ld + d];
        s[t] = acc * scale;
        if (s[t] > mx) mx = s[t];
    }
    double z = 0.0;
    for (int t = 0; t < n; ++t) { s[t] = exp(s[t] - mx); z += s[t]; }
    for (int d = 0; d < hd; ++d) o[d] = 0.0;
    for (int t = 0; t < n; ++t) {
        double w = s[t] / z;
        for (int d = 0; d < hd; ++d) o[d] += w * v[t * ld + d];
    }
    free(s);
}

static inline double silu(double g) { return g / (1.0 + exp(-g)); }

/* ------------------------------------------------------------------ */
/* forward                                                             */
/* ------------------------------------------------------------------ */

typedef struct {
    int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab;
    int32_t qk_norm;  /* per-head RMSNorm on q and k before RoPE */
    int32_t kv_bf16;  /* new keys / values rounded to bf16 (bf16 KV cache) */
    int32_t wdtype;   /* weight arrays: 0 = fp32, 1 = bf16 bits */
    double rope_base, rms_eps;
} or_model;

/* weights of one layer, each [out][in] row-major, y = W x */
typedef struct {
    const void *wq, *wk, *wv, *wo, *wg, *wu, *wd;
    const void *norm1, *norm2, *qnorm, *knorm;
} or_layer;

/* fills the weights of layer `layer`; returns 0 on success */
typedef int (*or_layer_fn)(void* cb, int32_t layer, or_layer* out);
/* cached keys/values of batch user b at layer `layer`: positions [0, prefix)
 * as [prefix][n_kv_heads][head_dim] fp32 arrays; returns 0 on success */
typedef int (*or_kv_fn)(void* cb, int32_t layer, int32_t b, float* k, float* v);

static double kvr(const or_model* m, double x) { return m->kv_bf16 ? or_round_bf16(x) : x; }

/* y[t][o] = sum_i x[t][i] * W[o][i] for t < rows, o < nout */
static void matmul_rows(const double* x, int rows, int nin, const void* w, int dt, int nout,
                        double* y) {
#pragma omp parallel for schedule(static)
    for (int o = 0; o < nout; ++o) {
        const size_t base = (size_t)o * nin;
        for (int t = 0; t < rows; ++t) {
            const double* xr = x + (size_t)t * nin;
            double acc = 0.0;
            for (int i = 0; i < nin; ++i) acc += xr[i] * wget(w, base + i, dt);
            y[(size_t)t * nout + o] = acc;
        }
    }
}

/*
 * Logits of the verify forward for a batch of users.
 *   prefix_len[b]: cached context length i_m of user b (keys at 0..i_m-1)
 *   n_slots[b]:    query slots of user b (root + l_m drafts = l_m + 1)
 *   tokens:        slot tokens, users in order, slots in order (T total)
 *   slot j of user b sits at absolute position prefix_len[b] + j and attends
 *   to every position <= its own.
 * Outputs logits [T][vocab] (fp32) and, if k_new/v_new are given, the new
 * slots' keys/values [n_layers][T][n_kv_heads][head_dim].
 */
int or_forward(const or_model* m, int32_t n_users, const int32_t* prefix_len,
               const int32_t* n_slots, const int32_t* tokens, const void* embed,
               const void* norm_f, const void* lm_head, or_layer_fn lf, or_kv_fn kf, void* cb,
               float* logits, float* k_new, float* v_new) {
    const int d = m->d_model, hq = m->n_q_heads, hkv = m->n_kv_heads, hd = m->head_dim;
    const int F = m->d_ffn, V = m->vocab, dt = m->wdtype, G = hq / hkv;
    const int nq = hq * hd, nk = hkv * hd;
    int T = 0;
    int* off = (int*)malloc(sizeof(int) * (n_users + 1));
    off[0] = 0;
    for (int b = 0; b < n_users; ++b) { off[b + 1] = off[b] + n_slots[b]; }
    T = off[n_users];
    int max_ctx = 0;
    for (int b = 0; b < n_users; ++b)
        if (prefix_len[b] + n_slots[b] > max_ctx) max_ctx = prefix_len[b] + n_slots[b];

    double* x = (double*)malloc(sizeof(double) * (size_t)T * d);
    double* h = (double*)malloc(sizeof(double) * (size_t)T * (d > F ? d : F));
    double* q = (double*)malloc(sizeof(double) * (size_t)T * nq);
    double* kk = (double*)malloc(sizeof(double) * (size_t)T * nk);
    double* vv = (double*)malloc(sizeof(double) * (size_t)T * nk);
    double* att = (double*)malloc(sizeof(double) * (size_t)T * nq);
    double* y = (double*)malloc(sizeof(double) * (size_t)T * (2 * F > d ? 2 * F : d));
    double* g = (double*)malloc(sizeof(double) * (size_t)T * F);
    double* Kc = (double*)malloc(sizeof(double) * (size_t)n_users * max_ctx * nk);
    double* Vc = (double*)malloc(sizeof(double) * (size_t)n_users * max_ctx * nk);
    float* kbuf = (float*)malloc(sizeof(float) * (size_t)max_ctx * nk + 1);
    float* vbuf = (float*)malloc(sizeof(float) * (size_t)max_ctx * nk + 1);
    int rc = 0;

    /* embedding */
    for (int t = 0; t < T; ++t)
        for (int i = 0; i < d; ++i) x[(size_t)t * d + i] = wget(embed, (size_t)tokens[t] * d + i, dt);

    for (int l = 0; l < m->n_layers && rc == 0; ++l) {
        or_layer w;
        if (lf(cb, l, &w) != 0) { rc = -1; break; }

        /* attention block */
        for (int t = 0; t < T; ++t) {
            or_rmsnorm(x + (size_t)t * d, d, w.norm1, dt, m->rms_eps, h + (size_t)t * d);
        }
        matmul_rows(h, T, d, w.wq, dt, nq, q);
        matmul_rows(h, T, d, w.wk, dt, nk, kk);
        matmul_rows(h, T, d, w.wv, dt, nk, vv);
        for (int b = 0; b < n_users; ++b) {
            for (int j = 0; j < n_slots[b]; ++j) {
                const int t = off[b] + j;
                const double pos = (double)(prefix_len[b] + j);
                double tmp[1024];
                for (int hh = 0; hh < hq; ++hh) {
                    double* v = q + (size_t)t * nq + (size_t)hh * hd;
                    if (m->qk_norm) { or_rmsnorm(v, hd, w.qnorm, dt, m->rms_eps, tmp); memcpy(v, tmp, sizeof(double) * hd); }
                    or_rope(v, hd, pos, m->rope_base);
                }
                for (int hh = 0; hh < hkv; ++hh) {
                    double* v = kk + (size_t)t * nk + (size_t)hh * hd;
                    if (m->qk_norm) { or_rmsnorm(v, hd, w.knorm, dt, m->rms_eps, tmp); memcpy(v, tmp, sizeof(double) * hd); }
                    or_rope(v, hd, pos, m->rope_base);
                    for (int i = 0; i < hd; ++i) v[i] = kvr(m, v[i]);
                    double* u = vv + (size_t)t * nk + (size_t)hh * hd;
                    for (int i = 0; i < hd; ++i) u[i] = kvr(m, u[i]);
                }
            }
        }
        /* per-user context: cached prefix then the new slots */
        for (int b = 0; b < n_users; ++b) {
            const int P = prefix_len[b];
            double* Kb = Kc + (size_t)b * max_ctx * nk;
            double* Vb = Vc + (size_t)b * max_ctx * nk;
            if (P > 0) {
                if (kf(cb, l, b, kbuf, vbuf) != 0) { rc = -2; break; }
                for (size_t i = 0; i < (size_t)P * nk; ++i) { Kb[i] = kbuf[i]; Vb[i] = vbuf[i]; }
            }
            memcpy(Kb + (size_t)P * nk, kk + (size_t)off[b] * nk, sizeof(double) * (size_t)n_slots[b] * nk);
            memcpy(Vb + (size_t)P * nk, vv + (size_t)off[b] * nk, sizeof(double) * (size_t)n_slots[b] * nk);
        }
        if (rc) break;
        if (k_new) {
            for (size_t i = 0; i < (size_t)T * nk; ++i) {
                k_new[(size_t)l * T * nk + i] = (float)kk[i];
                v_new[(size_t)l * T * nk + i] = (float)vv[i];
            }
        }
        const double scale = 1.0 / sqrt((double)hd);
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
        for (int t = 0; t < T; ++t) {
            for (int hh = 0; hh < hq; ++hh) {
                int b = 0;
                while (t >= off[b + 1]) ++b;
                const int j = t - off[b];
                const int n = prefix_len[b] + j + 1; /* causal: positions 0..i_m+j */
                const int kvh = hh / G;
                const double* Kb = Kc + (size_t)b * max_ctx * nk + (size_t)kvh * hd;
                const double* Vb = Vc + (size_t)b * max_ctx * nk + (size_t)kvh * hd;
                or_attend(q + (size_t)t * nq + (size_t)hh * hd, Kb, Vb, n, hd, nk, scale,
                          att + (size_t)t * nq + (size_t)hh * hd);
            }
        }
        matmul_rows(att, T, nq, w.wo, dt, d, y);
        for (size_t i = 0; i < (size_t)T * d; ++i) x[i] += y[i];

        /* FFN block */
        for (int t = 0; t < T; ++t) {
            or_rmsnorm(x + (size_t)t * d, d, w.norm2, dt, m->rms_eps, h + (size_t)t * d);
        }
        matmul_rows(h, T, d, w.wg, dt, F, g);
        matmul_rows(h, T, d, w.wu, dt, F, y);
        for (size_t i = 0; i < (size_t)T * F; ++i) g[i] = silu(g[i]) * y[i];
        matmul_rows(g, T, F, w.wd, dt, d, y);
        for (size_t i = 0; i < (size_t)T * d; ++i) x[i] += y[i];
    }

    if (rc == 0) {
        for (int t = 0; t < T; ++t) {
            or_rmsnorm(x + (size_t)t * d, d, norm_f, dt, m->rms_eps, h + (size_t)t * d);
        }
#pragma omp parallel for schedule(static)
        for (int o = 0; o < V; ++o) {
            for (int t = 0; t < T; ++t) {
                const double* xr = h + (size_t)t * d;
                double acc = 0.0;
                for (int i = 0; i < d; ++i) acc += xr[i] * wget(lm_head, (size_t)o * d + i, dt);
                logits[(size_t)t * V + o] = (float)acc;
            }
        }
    }
    free(off); free(x); free(h); free(q); free(kk); free(vv); free(att); free(y); free(g);
    free(Kc); free(Vc); free(kbuf); free(vbuf);
    return rc;
}

/* ------------------------------------------------------------------ */
/* sampler                                                             */
/* ------------------------------------------------------------------ */

enum { OR_GREEDY = 0, OR_STOCHASTIC = 1, OR_FORCE = 2 };

/* row statistics: max, sum of exp(z - max) (double), argmax (lowest index) */
static void row_stats(const float* z, long V, float* mx, double* sum, int* amax) {
    float m = -INFINITY;
    int a = 0;
    for (long k = 0; k < V; ++k)
        if (z[k] > m) { m = z[k]; a = (int)k; }
    double s = 0.0;
    for (long k = 0; k < V; ++k) s += exp((double)z[k] - (double)m);
    *mx = m; *sum = s; *amax = a;
}

/* p_k = exp(z_k - max) / sum, rounded once to fp32 */
static inline float prob32(float zk, float mx, double sum) {
    return (float)(exp((double)zk - (double)mx) / sum);
}

/* Exponential race over weights w_k >= 0 (w == NULL slot-wise computed by
 * the caller's mode): winner = argmax w_k / E_k, E_k unit exponentials,
 * ties to the lowest index, zero weights excluded.  Returns -1 if every
 * weight is zero.  gap = relative distance between the two best keys. */
static int race(const float* w, long V, uint64_t seed, uint64_t round, uint64_t user,
                uint64_t slot, double* gap) {
    float best = -1.0f, second = -1.0f;
    int win = -1;
    for (long k = 0; k < V; ++k) {
        if (!(w[k] > 0.0f)) continue;
        float e = or_race_exponential(draw64(seed, round, user, OR_PURPOSE_RACE, slot, (uint64_t)k));
        float key = w[k] / e;
        if (key > best) { second = best; best = key; win = (int)k; }
        else if (key > second) second = key;
    }
    if (gap) *gap = (win >= 0 && second >= 0.0f && isfinite(best)) ? (double)(best - second) / best : INFINITY;
    return win;
}

/*
 * Verify decisions for a batch.  For user b with L = L[b] drafts, logits rows
 * are z_0..z_L (slot j predicts the token after slot j's token); draft j+1 is
 * drafts[doff + j] with draft distribution q row doff + j.
 *   greedy:     accept draft iff it equals argmax z_j; correction/bonus =
 *               argmax at the stop slot.
 *   stochastic: accept iff u_j < p_j(d)/q_j(d) (fp32 division); on the first
 *               rejection race over max(0, p - q) (fallback p if that is all
 *               zero); if all L accepted race over p at slot L.
 *   force:      accept all, token = argmax at slot L (teacher forcing).
 * Outputs n_acc[b], token[b]; optional diagnostics ratio/u per draft,
 * race_gap per user (INFINITY when no race ran) and race_w [n_users][V], the
 * weights the stop slot's race ran over (zeros when no race ran), so that a
 * test can compute the law of the emitted token exactly.
 */
int or_sample(int32_t mode, int32_t n_users, const int32_t* user_ids, const int32_t* L,
              int64_t V, const float* logits, const int32_t* drafts, const float* q,
              const float* accept_u, uint64_t seed, uint64_t round, int32_t* n_acc,
              int32_t* token, float* ratio, float* u_used, double* race_gap, float* race_w) {
    long toff = 0, doff = 0;
    float* w = (float*)malloc(sizeof(float) * (size_t)V);
    for (int b = 0; b < n_users; ++b) {
        const int Lb = L[b];
        const uint64_t user = (uint64_t)user_ids[b];
        int a = 0;
        int stopped = 0;
        for (int j = 0; j < Lb; ++j) {
            const float* z = logits + (size_t)(toff + j) * V;
            const int d = drafts[doff + j];
            float mx; double sum; int amax;
            row_stats(z, V, &mx, &sum, &amax);
            int acc;
            float r = NAN, u = NAN;
            if (mode == OR_GREEDY) acc = (d == amax);
            else if (mode == OR_FORCE) acc = 1;
            else {
                const float pd = prob32(z[d], mx, sum);
                const float qd = q[(size_t)(doff + j) * V + d];
                r = pd / qd;
                u = accept_u ? accept_u[doff + j]
                             : or_accept_uniform(draw64(seed, round, user, OR_PURPOSE_ACCEPT, (uint64_t)j, 0));
                acc = (u < r);
            }
            if (ratio) ratio[doff + j] = r;
            if (u_used) u_used[doff + j] = u;
            if (!stopped) {
                if (acc) ++a;
                else stopped = 1;
            }
        }
        const float* z = logits + (size_t)(toff + a) * V;
        float mx; double sum; int amax;
        row_stats(z, V, &mx, &sum, &amax);
        double gap = INFINITY;
        int tok;
        if (mode != OR_STOCHASTIC) {
            tok = amax;
        } else {
            for (long k = 0; k < V; ++k) w[k] = prob32(z[k], mx, sum);
            if (a < Lb) {
                const float* qr = q + (size_t)(doff + a) * V;
                int any = 0;
                for (long k = 0; k < V; ++k) {
                    float pk = w[k];
                    float wk = pk - qr[k];
                    w[k] = wk > 0.0f ? wk : 0.0f;
                    any |= (w[k] > 0.0f);
                }
                if (!any)
                    for (long k = 0; k < V; ++k) w[k] = prob32(z[k], mx, sum);
            }
            tok = race(w, V, seed, round, user, (uint64_t)a, &gap);
        }
        if (race_w) {
            float* rw = race_w + (size_t)b * V;
            for (long k = 0; k < V; ++k) rw[k] = mode == OR_STOCHASTIC ? w[k] : 0.0f;
        }
        n_acc[b] = a;
        token[b] = tok;
        if (race_gap) race_gap[b] = gap;
        toff += Lb + 1;
        doff += Lb;
    }
    free(w);
    return 0;
}
