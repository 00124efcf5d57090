// Internal interfaces between the host runtime and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace sdv {

constexpr int kPageTokens = 16;   // tokens per KV page
constexpr int kAttnItemsMax = 1024;  // attention work items per batch (beyond one per (user, KV head))
constexpr int kAttnWGsPerCU = 2;     // co-resident attention workgroups per CU (register bound)
constexpr int kAttnBuffers = 2;      // LDS ring of the attention kernel (buffers - 1 blocks in flight)
constexpr int kVocabChunks = 64;  // vocab split of the sampler kernels (at most 64: one wave merges)
constexpr int kNormBlock = 1024;   // columns per sum-of-squares block of x
constexpr int kNormKMax = 8192;    // widest model dimension the GEMM can normalise on load
constexpr int kMaxPending = 8;
constexpr int kSparseChunkMax = 4096;  // largest vocab chunk of the sparse-q race (vocab <= 64 * 4096)
constexpr int kSparseKMax = 4096;      // most listed tokens per sparse draft row

// Model dimensions as the kernels see them.
struct Dims {
    int L, d, hq, hkv, hd, F, V, qk_norm, bf16;
    float rope_base, eps;
    int nq() const { return hq * hd; }
    int nkv() const { return hkv * hd; }
    int nqkv() const { return (hq + 2 * hkv) * hd; }
    int G() const { return hq / hkv; }
};

// Paged KV pool: [layer][page][K | V][kv_head] blocks; a K block is
// [page_tokens][head_dim] (token-major), a V block is [head_dim][page_tokens]
// (dim-major, so attention reads V^T fragments contiguously).
struct KVPool {
    void* base;
    int n_pages;
    int hkv, hd, esize;  // esize: bytes per element
    __host__ __device__ size_t block_elems() const { return (size_t)kPageTokens * hd; }
    __host__ __device__ size_t page_elems() const { return 2 * (size_t)hkv * block_elems(); }
    __host__ __device__ size_t k_off(int layer, int page, int g) const {
        return ((size_t)layer * n_pages + page) * page_elems() + (size_t)g * block_elems();
    }
    __host__ __device__ size_t v_off(int layer, int page, int g) const {
        return k_off(layer, page, g) + (size_t)hkv * block_elems();
    }
};

// Device view of one staged batch (all pointers into the workspace slot).
struct BatchView {
    int B, T, nd, mode;
    uint64_t seed, round;
    int max_pages;     // page-table row length
    int n_items;       // attention work items
    int rows_max;      // (max l_m + 1) * G, rows of an attention partial
    const int32_t* user_id;    // [B] global user id
    const int32_t* prefix;     // [B] i_m
    const int32_t* L;          // [B] l_m
    const int32_t* root;       // [B] root token
    const int32_t* slot_off;   // [B+1]
    const int32_t* draft_off;  // [B+1]
    const int32_t* slot_b;     // [T] user index of slot
    const int32_t* slot_j;     // [T] slot index within the user
    const int32_t* page_table; // [B][max_pages]
    const int4* items;         // [n_items] (b, g, c0, c1)
    const int32_t* item_off;   // [B+1]
    const int32_t* drafts;     // device input [nd]
    const float* q;            // device input [nd][V]
    const float* accept_u;     // device input [nd] or null
    // sparse draft distributions (qk > 0; q is then unused): row r lists qk
    // tokens q_idx[r][.] with probabilities q_val[r][.]; every other token
    // has probability q_rest[r]
    const int32_t* q_idx;      // device input [nd][qk]
    const float* q_val;        // device input [nd][qk]
    const float* q_rest;       // device input [nd]
    int qk;
    int32_t* flags;            // [1] device error bits, zeroed by the staging copy
    const int32_t* prow;       // [B] decode steps: output row of each user's probabilities
};

// Workspace buffers of one batch slot.
struct SlotBufs {
    int32_t* tok;     // [Tmax]
    float* cs;        // [Tmax][hd/2][2]
    float* x;         // [Tmax][d]
    float* ssq;       // [Tmax][nsq] sums of squares of x per 1024-column block
                      // (bf16 configuration: h holds x * gamma and the
                      // consumers of RMSNorm(x) scale their outputs by rstd)
    int nsq;
    // activations feeding matrix products; bf16 configuration: [2][T][...]
    // hi and lo planes of the batch's T slots (plane stride T * width)
    void* h;          // [T][d] GEMM input: RMSNorm(x) * gamma (fp32), x * gamma (bf16)
    void* ffn;        // [T][F] SwiGLU output
    void* qbuf;       // [T][nq] rotated queries
    void* attn;       // [T][nq] attention output
    float* apart;     // [max_items][rows_max][hd] attention chunk partials
    float* aml;       // [max_items][rows_max][2]
    float* gpart;     // GEMM split-K partials
    size_t gpart_floats;
    float* logits;    // [Tmax][V]
    float* sstat;     // [Tmax][4] per-slot max, sum, argmax, accept
    float* spart;     // [Tmax * kVocabChunks][4] phase-A vocab-chunk partials
    float* spartB;    // [Bmax * kVocabChunks][4] phase-B partials
    // phase-A statistics from the lm_head epilogue (bf16 configuration):
    // per (slot, workgroup) row max, sum of exp(z - max), argmax value and
    // index over the workgroup's vocab rows, [T][groups][4]; the logit of
    // the draft that follows each slot; that draft token per slot (-1: none)
    float* lstat;
    float* zd;        // [Tmax]
    int32_t* dnext;   // [Tmax]
    int* skcnt;       // [kSkCounters] stream-K piece counters, zero between launches
    int32_t* result;  // [2*Bmax + 4]: n_acc, token, flags
    int bmax;
};

// ---- launchers (all enqueue on `s`, no synchronisation) ----
void launch_prepare(const Dims& D, const BatchView& bv, const SlotBufs& sb, hipStream_t s);
void launch_attention(const Dims& D, const BatchView& bv, const SlotBufs& sb, const KVPool& kv,
                      int layer, hipStream_t s);

// EPI_LMSTAT (lm_head): phase-A statistics per (workgroup, slot) into
// lstat, the logit of each slot's next draft into zd, and the logits
// themselves into out when out is set; never split over k.
enum GemmEpi { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LMSTAT = 3 };
struct GemmCall {
    const void* X;    // [T][K] act type
    const void* Wp;   // bf16: packed weights (fragment order, virtual rows)
    const void* W[3]; // fp32: weight segments, rows [out][K]
    int seg[3];       // first virtual column of each segment (seg[0] = 0)
    int nseg;
    int N;            // output columns (real); SWIGLU: F, with W[0]=gate, W[1]=up
    int K, T;
    int epi;
    void* out;        // EPI_STORE: float [T][ldo]; EPI_RESID: float x [T][ldo]; SWIGLU: act [T][ldo]
    int ldo;
    int raw;          // 1: write split-K partial planes [S][T][N] to the slot's
                      //    partial buffer and leave the reduction to the consumer
    // bf16 configuration, RMSNorm after the product: when norm_ss is set, X
    // holds x * gamma and each output of slot t is scaled by
    // rstd(t) = 1 / sqrt(sum_b norm_ss[t][b] / K + eps)
    const float* norm_ss;
    int norm_nb;
    // EPI_LMSTAT outputs (see SlotBufs) and the number of statistic groups
    // (workgroups) the launch writes
    float* lstat;
    float* zd;
    const int32_t* dnext;
    int* groups_out;
    // stream-K of the gate/up product (see k_gemm.hip): per-tile piece
    // counters (kSkCounters, zero between launches), the device error bits
    // and the polls of a wait before it gives up
    int* sk_cnt;
    int32_t* flags;
    int sk_polls;
};
constexpr int kSkCounters = 4096;
// polls of a stream-K wait before it gives up (a fraction of a second)
constexpr int kSkPollsDefault = 1 << 18;
// Upper bound of the statistic groups of an lm_head of V rows (workgroups
// of at least 128 rows, one more for rounding)
inline int lm_stat_groups_max(int V) { return (V + 127) / 128 + 1; }
// Returns the number of partial planes S (raw mode), else the splits used.
int launch_gemm(const Dims& D, const GemmCall& g, const SlotBufs& sb, hipStream_t s);
// bf16 configuration: x[t] += sum_s part[s][t] (split order), h = x * gamma
// (activation planes) and the block sums of squares of the new x; the
// consumers of h scale by rstd
void launch_resid_reduce(const Dims& D, int T, const float* part, int S, float* x,
                         const void* gamma, void* h, float* ssq, int nsq, hipStream_t s);
// x[t] += sum_s part[s][t] (split order); h[t] = RMSNorm(x[t]) * gamma
void launch_resid_norm(const Dims& D, int T, const float* part, int S, float* x,
                       const void* gamma, void* h, hipStream_t s);
// embedding gather into x and h = RMSNorm(x) * gamma (fp32 configuration),
// or into x, h = x * gamma and the block sums of squares (bf16)
void launch_embed_norm(const Dims& D, const BatchView& bv, const void* embed, const void* gamma,
                       const SlotBufs& sb, hipStream_t s);
// QKV partial reduction fused with QK-norm, RoPE, query store and KV append
// (bf16: the summed partials are first scaled by the slot's rstd)
void launch_qkv_finish(const Dims& D, const BatchView& bv, const SlotBufs& sb, const KVPool& kv,
                       int layer, const float* part, int S, const void* qn, const void* kn,
                       hipStream_t s);
size_t gemm_partial_floats(const Dims& D, int Tmax);
void launch_pack(const void* s0, const void* s1, const void* s2, int seg1, int seg2, int mode,
                 int K, int vrows, void* dst, hipStream_t s);

// Accept/resample of a batch.  groups = 0: phase A over the logits; groups
// > 0: phase A from the lm_head epilogue's statistics (sb.lstat, groups
// partials per slot, and sb.zd); logits then only feed phase B (stochastic).
void launch_sampler(const Dims& D, const BatchView& bv, const SlotBufs& sb, const float* logits,
                    hipStream_t s, int groups = 0);
// probs[t][k] = exp(z[t][k] - m_t) / S_t from the sampler's per-slot
// statistics (the same expression the race uses for p)
void launch_probs(const Dims& D, const BatchView& bv, const SlotBufs& sb, const float* logits,
                  float* probs, hipStream_t s);

// Page ids of one KV copy launch: pages page0 .. page0 + kKVCopyPages - 1
// of a user (a by-value kernel argument of 1 KB).
constexpr int kKVCopyPages = 256;
struct KVCopyPages {
    int32_t page0;
    int32_t id[kKVCopyPages];
};

// Context-free sampler call: per-batch tables in a fixed scratch array.
constexpr int kNoallocUsers = 64;
constexpr int kNoallocSlots = 1024;
struct NoallocMeta {  // kernel argument (520 bytes)
    int32_t B, V;
    int32_t user_id[kNoallocUsers];
    int32_t L[kNoallocUsers];
};
struct NoallocTables {  // device pointers into the scratch array
    int32_t *user_id, *L, *slot_off, *draft_off, *slot_b, *slot_j, *flags;
};
void launch_noalloc_stage(const NoallocMeta& m, const NoallocTables& t, const int32_t* drafts,
                          hipStream_t s);

void launch_kv_copy(const Dims& D, const KVPool& kv, const KVCopyPages& pages, int layer,
                    int pos0, int n, const void* k, const void* v, int to_pool, hipStream_t s);

}  // namespace sdv
