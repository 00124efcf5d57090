// Host runtime and C ABI of the batched speculative-verify library.
//
// The host side owns user state (cached length i_m, root token, KV pages),
// the page free list, per-batch staging and the launch sequence of one verify
// pass.  All device memory (weights, KV pool, workspace) belongs to the
// caller; this file never allocates device memory.  Batches are validated and
// planned on the host before anything is enqueued, so an error return leaves
// every state untouched.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/sd_verify.h"
#include "sdv_internal.h"

using namespace sdv;

namespace sdv {
}

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

int ceil_div(long a, long b) { return (int)((a + b - 1) / b); }

// Byte layout of one workspace slot and of the staging block inside it.
struct Layout {
    // staging block (int32 offsets within the block)
    size_t st_user, st_prefix, st_L, st_root, st_soff, st_doff, st_sb, st_sj, st_pt, st_items,
        st_ioff, st_flags, st_prow, st_bytes;
    // slot buffers (byte offsets within the slot)
    size_t stage, tok, cs, x, ssq, h, ffn, qbuf, attn, apart, aml, gpart, logits, sstat, spart,
        spartB, lstat, zd, dnext, skcnt, result, slot_bytes;
    size_t gpart_floats;
    int nsq;
    // global region after the slots
    size_t total;
    int max_pages, max_items, rows_max, Tmax, Bmax;
};

Dims dims_of(const sd_config& c) {
    Dims D;
    D.L = c.n_layers;
    D.d = c.d_model;
    D.hq = c.n_q_heads;
    D.hkv = c.n_kv_heads;
    D.hd = c.head_dim;
    D.F = c.d_ffn;
    D.V = c.vocab;
    D.qk_norm = c.qk_norm;
    D.bf16 = c.dtype == SD_BF16;
    D.rope_base = c.rope_base;
    D.eps = c.rms_eps;
    return D;
}

sd_status validate_config(const sd_config* c) {
    if (!c) return SD_EINVAL;
    if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 ||
        c->head_dim < 2 || c->d_ffn < 1 || c->vocab < 2)
        return SD_EINVAL;
    if (c->n_q_heads % c->n_kv_heads) return SD_EINVAL;
    if (c->head_dim % 2 || c->head_dim > 128) return SD_EINVAL;
    if (c->d_model % 4 || c->d_model > 8192) return SD_ENOTIMPL;
    if (c->dtype != SD_F32 && c->dtype != SD_BF16) return SD_EINVAL;
    if (c->page_tokens != kPageTokens) return SD_EINVAL;
    if (c->n_pages < 1 || c->max_users < 1 || c->max_draft < 1 || c->max_draft > 64) return SD_EINVAL;
    if (c->max_batch_users < 1 || c->max_batch_tokens < 2 || c->max_ctx < 2) return SD_EINVAL;
    if (c->max_pending < 1 || c->max_pending > kMaxPending) return SD_EINVAL;
    if (!(c->rope_base > 1.0f) || !(c->rms_eps >= 0.0f)) return SD_EINVAL;
    if (c->qk_norm != 0 && c->qk_norm != 1) return SD_EINVAL;
    if (c->logits_out < SD_LOGITS_AS_NEEDED || c->logits_out > SD_LOGITS_UNFUSED) return SD_EINVAL;
    if (c->dtype == SD_BF16) {
        // MFMA kernels: 128-wide heads, k dimensions in whole LDS chunks and
        // output widths in whole 128-column tiles
        if (c->head_dim != 128) return SD_ENOTIMPL;
        const Dims D = dims_of(*c);
        if (D.d % 256 || D.nq() % 256 || D.F % 256) return SD_ENOTIMPL;
        if (D.nqkv() % 128 || D.d % 128 || (2 * D.F) % 128 || D.V % 128) return SD_ENOTIMPL;
        if (D.hq * D.hd % 16 || D.hkv * D.hd % 16) return SD_ENOTIMPL;
        if (c->max_batch_tokens > 416) return SD_ENOTIMPL;
        // the attention kernel addresses one layer's pages with 32-bit
        // offsets: below 4 GB per layer (65535 pages of the 32B shape)
        const uint64_t page_bytes = 2ull * D.hkv * kPageTokens * D.hd * 2;
        if ((uint64_t)c->n_pages * page_bytes >= (1ull << 32)) return SD_ENOTIMPL;
    } else {
        if (c->head_dim > 128) return SD_ENOTIMPL;
    }
    return SD_OK;
}

Layout plan(const sd_config& c) {
    const Dims D = dims_of(c);
    Layout L;
    L.Tmax = c.max_batch_tokens;
    L.Bmax = c.max_batch_users;
    L.max_pages = ceil_div(c.max_ctx, kPageTokens);
    // the chunk lengths are chosen per batch so that there are at most
    // max(kAttnItemsMax, users * kv heads) work items
    L.max_items = std::max(kAttnItemsMax, L.Bmax * D.hkv);
    L.rows_max = (c.max_draft + 1) * D.G();
    const size_t es = D.bf16 ? 2 : 4;
    // staging block
    size_t o = 0;
    auto take_i = [&](size_t n) { size_t r = o; o = align_up(o + n * 4); return r; };
    L.st_user = take_i(L.Bmax);
    L.st_prefix = take_i(L.Bmax);
    L.st_L = take_i(L.Bmax);
    L.st_root = take_i(L.Bmax);
    L.st_soff = take_i(L.Bmax + 1);
    L.st_doff = take_i(L.Bmax + 1);
    L.st_sb = take_i(L.Tmax);
    L.st_sj = take_i(L.Tmax);
    L.st_pt = take_i((size_t)L.Bmax * L.max_pages);
    L.st_items = take_i((size_t)L.max_items * 4);
    L.st_ioff = take_i(L.Bmax + 1);
    L.st_flags = take_i(4);
    L.st_prow = take_i(L.Bmax);
    L.st_bytes = o;
    // slot
    size_t s = 0;
    auto take = [&](size_t bytes) { size_t r = s; s = align_up(s + bytes); return r; };
    L.stage = take(L.st_bytes);
    L.tok = take((size_t)L.Tmax * 4);
    L.cs = take((size_t)L.Tmax * (D.hd / 2) * 2 * 4);
    L.x = take((size_t)L.Tmax * D.d * 4);
    L.nsq = (D.d + kNormBlock - 1) / kNormBlock;
    L.ssq = take((size_t)L.Tmax * L.nsq * 4);
    // activations that feed matrix products: two bf16 planes (hi, lo) each
    // in the bf16 configuration, one fp32 plane otherwise
    const size_t ap = D.bf16 ? 2 : 1;
    L.h = take(ap * L.Tmax * D.d * es);
    L.ffn = take(ap * L.Tmax * D.F * es);
    L.qbuf = take(ap * L.Tmax * D.nq() * es);
    L.attn = take(ap * L.Tmax * D.nq() * es);
    const size_t nparts = D.bf16 ? (size_t)L.max_items * L.rows_max : 1;
    L.apart = take(nparts * D.hd * 4);
    L.aml = take(nparts * 2 * 4);
    L.gpart_floats = gemm_partial_floats(D, L.Tmax);
    L.gpart = take(std::max<size_t>(L.gpart_floats, 1) * 4);
    L.logits = take((size_t)L.Tmax * D.V * 4);
    L.sstat = take((size_t)L.Tmax * 4 * 4);
    L.spart = take((size_t)L.Tmax * kVocabChunks * 4 * 4);
    L.spartB = take((size_t)L.Bmax * kVocabChunks * 4 * 4);
    L.lstat = take(D.bf16 ? (size_t)lm_stat_groups_max(D.V) * L.Tmax * 4 * 4 : 16);
    L.zd = take((size_t)L.Tmax * 4);
    L.dnext = take((size_t)L.Tmax * 4);
    L.skcnt = take((size_t)kSkCounters * 4);
    L.result = take((size_t)(2 * L.Bmax + 4) * 4);
    L.slot_bytes = s;
    L.total = align_up(L.slot_bytes * (size_t)c.max_pending);
    return L;
}

// Element offsets of the packed GEMM weights (bf16): per layer QKV, O,
// gate/up (interleaved), down; then lm_head.
struct PackLayout {
    size_t qkv, o, gu, down, layer, lm, total;
};

PackLayout pack_layout(const Dims& D) {
    PackLayout P;
    P.qkv = 0;
    P.o = P.qkv + (size_t)D.nqkv() * D.d;
    P.gu = P.o + (size_t)D.d * D.nq();
    P.down = P.gu + (size_t)2 * D.F * D.d;
    P.layer = P.down + (size_t)D.d * D.F;
    P.lm = P.layer * D.L;
    P.total = P.lm + (size_t)D.V * D.d;
    return P;
}

struct User {
    bool active = false;
    int prefix = 0;
    int root = 0;
    std::vector<int> pages;
    int pending_slot = -1;
};

struct Slot {
    bool pending = false;
    bool sample_only = false;
    bool logits_ok = false;  // the pending pass stored every slot's logits
    int batch = -1;
    int B = 0, T = 0, nd = 0;
    std::vector<int> users;  // global ids in batch order
    std::vector<int> L;
    std::vector<int> prow;   // decode steps: destination row of each user's probabilities
    hipEvent_t done = nullptr;
    char* stage_host = nullptr;  // pinned
    int32_t* result_host = nullptr;  // pinned
    char* base = nullptr;        // device slot base
    SlotBufs bufs{};
    // graph of the slot's last captured pass and the launch signature it
    // was captured for (sd_verify_batch_graph)
    hipGraphExec_t gexec = nullptr;
    std::vector<int64_t> gkey;
};

}  // namespace

struct sd_ctx {
    sd_config cfg{};
    Dims D{};
    Layout lay{};
    sd_weights w{};
    std::vector<sd_layer_weights> layers;
    KVPool kv{};
    char* ws = nullptr;
    char* wpack = nullptr;  // packed GEMM weights (bf16 configurations)
    PackLayout pl{};
    std::vector<User> users;
    std::vector<int> free_pages;  // stack: back is allocated first
    Slot slots[kMaxPending];
    int device = 0;
    int attn_cap = 512;  // attention work items that run in one wave of workgroups
    int sk_polls = kSkPollsDefault;  // bound of the stream-K waits
    // diagnostic timing of one kernel class
    int prof_class = 0;
    int prof_used = 0;
    std::vector<hipEvent_t> prof_ev;  // pairs (start, end)
};

namespace {

sd_status hip_status(hipError_t e) { return e == hipSuccess ? SD_OK : SD_EHIP; }

#define SD_HIP(expr)                                            \
    do {                                                        \
        hipError_t _e = (expr);                                 \
        if (_e != hipSuccess) return SD_EHIP;                   \
    } while (0)

int pages_for(int tokens) { return ceil_div(tokens, kPageTokens); }

void release_to(sd_ctx* c, User& u, int keep) {
    while ((int)u.pages.size() > keep) {
        c->free_pages.push_back(u.pages.back());
        u.pages.pop_back();
    }
}

bool reserve_to(sd_ctx* c, User& u, int want) {
    const int need = want - (int)u.pages.size();
    if (need <= 0) return true;
    if ((int)c->free_pages.size() < need) return false;
    for (int i = 0; i < need; ++i) {
        u.pages.push_back(c->free_pages.back());
        c->free_pages.pop_back();
    }
    return true;
}

BatchView make_view(sd_ctx* c, Slot& s) {
    const Layout& L = c->lay;
    char* st = s.base + L.stage;
    BatchView v{};
    v.user_id = (const int32_t*)(st + L.st_user);
    v.prefix = (const int32_t*)(st + L.st_prefix);
    v.L = (const int32_t*)(st + L.st_L);
    v.root = (const int32_t*)(st + L.st_root);
    v.slot_off = (const int32_t*)(st + L.st_soff);
    v.draft_off = (const int32_t*)(st + L.st_doff);
    v.slot_b = (const int32_t*)(st + L.st_sb);
    v.slot_j = (const int32_t*)(st + L.st_sj);
    v.page_table = (const int32_t*)(st + L.st_pt);
    v.items = (const int4*)(st + L.st_items);
    v.item_off = (const int32_t*)(st + L.st_ioff);
    v.flags = (int32_t*)(st + L.st_flags);
    v.prow = (const int32_t*)(st + L.st_prow);
    v.max_pages = L.max_pages;
    return v;
}

// Collect the users of batch `batch` and validate every argument that does
// not need the device.  Fills users / Ls / T / nd.
// draft_len == NULL: a decode step, every batch user contributes its root
// alone (l_m = 0, one query slot).
sd_status collect_batch(sd_ctx* c, int32_t batch, int32_t n_users, const int32_t* assign,
                        const int32_t* draft_len, bool need_active, std::vector<int>& users,
                        std::vector<int>& Ls, int& T, int& nd) {
    if (batch < 0 || n_users < 1 || n_users > c->cfg.max_users || !assign) return SD_EINVAL;
    users.clear();
    Ls.clear();
    T = 0;
    nd = 0;
    for (int m = 0; m < n_users; ++m) {
        if (assign[m] != batch) continue;
        const int L = draft_len ? draft_len[m] : 0;
        if (draft_len && (L < 1 || L > c->cfg.max_draft)) return SD_EINVAL;
        const User& u = c->users[m];
        if (need_active) {
            if (!u.active) return SD_EINVAL;
            if (u.prefix + L + 1 > c->cfg.max_ctx) return SD_EINVAL;
        }
        if (u.pending_slot >= 0) return SD_ESTATE;
        users.push_back(m);
        Ls.push_back(L);
        T += L + 1;
        nd += L;
    }
    if (users.empty()) return SD_EINVAL;  // eq. (10): a declared batch is active
    if ((int)users.size() > c->cfg.max_batch_users || T > c->cfg.max_batch_tokens) return SD_EINVAL;
    return SD_OK;
}

// Write the staging block for the batch into the slot's pinned buffer.
void build_stage(sd_ctx* c, Slot& s, int mode, bool with_items, int* n_items, int* rows_max) {
    const Layout& L = c->lay;
    char* st = s.stage_host;
    int32_t* user = (int32_t*)(st + L.st_user);
    int32_t* prefix = (int32_t*)(st + L.st_prefix);
    int32_t* Lb = (int32_t*)(st + L.st_L);
    int32_t* root = (int32_t*)(st + L.st_root);
    int32_t* soff = (int32_t*)(st + L.st_soff);
    int32_t* doff = (int32_t*)(st + L.st_doff);
    int32_t* sb = (int32_t*)(st + L.st_sb);
    int32_t* sj = (int32_t*)(st + L.st_sj);
    int32_t* pt = (int32_t*)(st + L.st_pt);
    int32_t* items = (int32_t*)(st + L.st_items);
    int32_t* ioff = (int32_t*)(st + L.st_ioff);
    int32_t* flags = (int32_t*)(st + L.st_flags);
    (void)mode;
    soff[0] = 0;
    doff[0] = 0;
    int maxL = 0, ni = 0;
    ioff[0] = 0;
    // Attention work items: each (user, KV head) context is cut into chunks
    // (multiples of 32 tokens, the kernel's block) so that the whole batch
    // has at most attn_cap items -- one wave of co-resident workgroups, so
    // no workgroup waits for a second round -- and each user's chunks are
    // of equal length.  Fewer, longer items also keep the partial-sum
    // traffic (one [rows][head_dim] fp32 partial per item) small.
    const int hkv = c->D.hkv;
    const int cap = std::max(c->attn_cap, s.B * hkv);
    long total = 0;
    for (int b = 0; b < s.B; ++b) total += c->users[s.users[b]].prefix + s.L[b] + 1;
    // A token costs its share of the KV stream plus the products of the wave
    // with the most 16-row query tiles (the four waves take tiles w, w+4,
    // ...): a user whose (l+1)*G rows need two tiles per wave costs about
    // 1.3x per token (measured: the products add ~6 us to the ~14 us KV
    // stream of a one-tile layer at 80 slots), so its chunks are shortened
    // in proportion and the items end together.
    const int G = c->D.G();
    auto weight = [&](int b) {  // cost per token in tenths
        const int tiles = ceil_div((s.L[b] + 1) * G, 16);
        return 10 + 3 * (ceil_div(tiles, 4) - 1);
    };
    auto user_chunk = [&](int b, int ch) {  // chunk length of user b for base length ch
        return std::max(32, (int)((long)ch * 10 / weight(b)) & ~31);
    };
    auto n_items_for = [&](int ch) {
        long n = 0;
        for (int b = 0; b < s.B; ++b)
            n += ceil_div(c->users[s.users[b]].prefix + s.L[b] + 1, user_chunk(b, ch));
        return n * hkv;
    };
    // (ends: once every user's chunk holds its whole context there are
    // B * hkv <= cap items)
    int chunk = (int)std::max<long>(32, ((total * hkv + cap - 1) / cap + 31) & ~31L);
    while (n_items_for(chunk) > cap) chunk += 32;
    for (int b = 0; b < s.B; ++b) {
        const User& u = c->users[s.users[b]];
        user[b] = s.users[b];
        prefix[b] = u.prefix;
        Lb[b] = s.L[b];
        root[b] = u.root;
        soff[b + 1] = soff[b] + s.L[b] + 1;
        doff[b + 1] = doff[b] + s.L[b];
        for (int j = 0; j <= s.L[b]; ++j) {
            sb[soff[b] + j] = b;
            sj[soff[b] + j] = j;
        }
        for (int i = 0; i < L.max_pages; ++i)
            pt[(size_t)b * L.max_pages + i] = i < (int)u.pages.size() ? u.pages[i] : 0;
        maxL = std::max(maxL, s.L[b]);
        if (with_items) {
            const int ctx = u.prefix + s.L[b] + 1;
            // equal chunks for this user: as many as its chunk length needs,
            // evened out
            const int ub = user_chunk(b, chunk);
            const int cb = (ceil_div(ctx, ceil_div(ctx, ub)) + 31) & ~31;
            const int nch = ceil_div(ctx, cb);
            for (int g = 0; g < hkv; ++g)
                for (int ch = 0; ch < nch; ++ch) {
                    items[ni * 4 + 0] = b;
                    items[ni * 4 + 1] = g;
                    items[ni * 4 + 2] = ch * cb;
                    items[ni * 4 + 3] = std::min(ctx, (ch + 1) * cb);
                    ++ni;
                }
        }
        ioff[b + 1] = ni;
    }
    flags[0] = flags[1] = flags[2] = flags[3] = 0;
    int32_t* prow = (int32_t*)(st + L.st_prow);
    for (int b = 0; b < s.B; ++b) prow[b] = s.prow.empty() ? b : s.prow[b];
    *n_items = ni;
    *rows_max = (maxL + 1) * c->D.G();
}

// Records a start event before a launch group of class k and an end event
// after it when that class is being profiled.
struct ProfScope {
    sd_ctx* c;
    hipStream_t st;
    int idx = -1;
    ProfScope(sd_ctx* c_, int k, hipStream_t s) : c(c_), st(s) {
        if (c->prof_class == k && 2 * (c->prof_used + 1) <= (int)c->prof_ev.size()) {
            idx = c->prof_used++;
            (void)hipEventRecord(c->prof_ev[2 * idx], st);
        }
    }
    ~ProfScope() {
        if (idx >= 0) (void)hipEventRecord(c->prof_ev[2 * idx + 1], st);
    }
};

// write_logits: store the fp32 logits of every slot; *groups receives the
// number of phase-A statistic records per slot the lm_head writes (0: the
// sampler computes phase A from the logits)
sd_status enqueue_forward(sd_ctx* c, Slot& s, const BatchView& bv, hipStream_t st, bool write_logits,
                          int* groups) {
    const Dims& D = c->D;
    const SlotBufs& sb = s.bufs;
    const int T = bv.T;
    {
        ProfScope ps(c, SD_K_SMALL, st);
        launch_prepare(D, bv, sb, st);
        // x = E[tok]; h = RMSNorm(x) with the first layer's pre-attention
        // gain (bf16: h = x * gain and the block sums of squares)
        launch_embed_norm(D, bv, c->w.embed, c->layers[0].norm1, sb, st);
    }
    // GEMM input RMSNorm(x) * gamma: h = RMSNorm(x) * gamma (fp32), or
    // h = x * gamma with the rstd factor applied to the GEMM's outputs (bf16:
    // the norm's row reduction then needs no single-workgroup pass)
    auto normed_input = [&](GemmCall& g) {
        g.X = sb.h;
        if (D.bf16) {
            g.norm_ss = sb.ssq;
            g.norm_nb = sb.nsq;
        }
    };
    // x += partial sums; then h = x * gamma plus the block sums of squares
    // (bf16) or h = RMSNorm(x) * gamma (fp32)
    auto residual = [&](int S, const void* gamma) {
        if (D.bf16)
            launch_resid_reduce(D, T, sb.gpart, S, sb.x, gamma, sb.h, sb.ssq, sb.nsq, st);
        else
            launch_resid_norm(D, T, sb.gpart, S, sb.x, gamma, sb.h, st);
    };
    for (int l = 0; l < D.L; ++l) {
        const sd_layer_weights& w = c->layers[l];
        const size_t lbase = (size_t)l * c->pl.layer * 2;
        {
            // QKV projection (split-K partials), then their reduction fused
            // with QK-norm, RoPE, the query store and the KV append
            ProfScope ps(c, SD_K_QKV, st);
            GemmCall g{};
            normed_input(g);
            g.Wp = c->wpack + lbase + c->pl.qkv * 2;
            g.W[0] = w.wq; g.W[1] = w.wk; g.W[2] = w.wv;
            g.seg[0] = 0; g.seg[1] = D.nq(); g.seg[2] = D.nq() + D.nkv();
            g.nseg = 3;
            g.N = D.nqkv();
            g.K = D.d;
            g.T = T;
            g.epi = EPI_STORE;
            g.raw = 1;
            const int S = launch_gemm(D, g, sb, st);
            launch_qkv_finish(D, bv, sb, c->kv, l, sb.gpart, S, w.qnorm, w.knorm, st);
        }
        {
            ProfScope ps(c, SD_K_ATTN, st);
            launch_attention(D, bv, sb, c->kv, l, st);
        }
        {
            // output projection, then residual add fused with the pre-FFN norm
            ProfScope ps(c, SD_K_O, st);
            GemmCall o{};
            o.X = sb.attn;
            o.Wp = c->wpack + lbase + c->pl.o * 2;
            o.W[0] = w.wo;
            o.nseg = 1;
            o.N = D.d;
            o.K = D.nq();
            o.T = T;
            o.epi = EPI_STORE;
            o.raw = 1;
            const int S = launch_gemm(D, o, sb, st);
            residual(S, w.norm2);
        }
        {
            ProfScope ps(c, SD_K_GATEUP, st);
            GemmCall gu{};
            normed_input(gu);
            gu.Wp = c->wpack + lbase + c->pl.gu * 2;
            gu.W[0] = w.wg; gu.W[1] = w.wu;
            gu.nseg = 2;
            gu.seg[1] = D.F;
            gu.N = D.F;
            gu.K = D.d;
            gu.T = T;
            gu.epi = EPI_SWIGLU;
            gu.out = sb.ffn;
            gu.ldo = D.F;
            gu.sk_cnt = sb.skcnt;
            gu.flags = bv.flags;
            gu.sk_polls = c->sk_polls;
            launch_gemm(D, gu, sb, st);
        }
        {
            // down projection, then residual add fused with the next norm
            // (next layer's pre-attention gain, or the final norm)
            ProfScope ps(c, SD_K_DOWN, st);
            GemmCall dn{};
            dn.X = sb.ffn;
            dn.Wp = c->wpack + lbase + c->pl.down * 2;
            dn.W[0] = w.wd;
            dn.nseg = 1;
            dn.N = D.d;
            dn.K = D.F;
            dn.T = T;
            dn.epi = EPI_STORE;
            dn.raw = 1;
            const int S = launch_gemm(D, dn, sb, st);
            const void* gnext = l + 1 < D.L ? c->layers[l + 1].norm1 : c->w.norm_f;
            residual(S, gnext);
        }
    }
    ProfScope ps_lm(c, SD_K_LMHEAD, st);
    GemmCall lm{};
    normed_input(lm);
    lm.Wp = c->wpack + c->pl.lm * 2;
    lm.W[0] = c->w.lm_head;
    lm.nseg = 1;
    lm.N = D.V;
    lm.K = D.d;
    lm.T = T;
    lm.ldo = D.V;
    *groups = 0;
    if (D.bf16 && c->cfg.logits_out != SD_LOGITS_UNFUSED) {
        // phase-A statistics from the epilogue; logits only when asked for
        lm.epi = EPI_LMSTAT;
        lm.out = write_logits ? sb.logits : nullptr;
        lm.lstat = sb.lstat;
        lm.zd = sb.zd;
        lm.dnext = sb.dnext;
        lm.groups_out = groups;
    } else {
        lm.epi = EPI_STORE;
        lm.out = sb.logits;
    }
    launch_gemm(D, lm, sb, st);
    return hip_status(hipGetLastError());
}

}  // namespace

// ---------------------------------------------------------------------------
// Scratch of sd_sample_logits_noalloc: one fixed array per GPU (each device
// the library runs on holds its own copy until the process ends).  Layout:
// the batch tables, then the sampler's per-slot statistics and vocab-chunk
// partials, each section 256-byte aligned.  Host code never uses the name
// `scratch` as an address: it takes the device address from
// hipGetSymbolAddress, once per device, and passes that to the kernels.
// ---------------------------------------------------------------------------
namespace {
constexpr size_t na_align(size_t x) { return (x + 255) & ~(size_t)255; }
constexpr size_t kNaTables = na_align((size_t)(4 * kNoallocUsers + 2 + 2 * kNoallocSlots + 1) * 4);
constexpr size_t kNaSstat = na_align((size_t)kNoallocSlots * 4 * 4);
constexpr size_t kNaSpart = na_align((size_t)kNoallocSlots * kVocabChunks * 4 * 4);
constexpr size_t kNaSpartB = na_align((size_t)kNoallocUsers * kVocabChunks * 4 * 4);
constexpr size_t kNaBytes = kNaTables + kNaSstat + kNaSpart + kNaSpartB;
static_assert(kNaBytes <= SD_NOALLOC_SCRATCH_BYTES, "scratch layout exceeds the declared size");
static_assert(kNoallocUsers == SD_NOALLOC_MAX_USERS && kNoallocSlots == SD_NOALLOC_MAX_SLOTS,
              "limits of the header and the kernels differ");
}  // namespace

static __device__ __align__(256) unsigned char scratch[SD_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kNaMaxDevices = 64;
std::mutex g_na_mutex;
unsigned char* g_na_ptr[kNaMaxDevices] = {};

// Device address of this GPU's scratch array (looked up on the first call
// on the device, with that device current).
sd_status na_scratch(unsigned char** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return SD_EHIP;
    if (dev >= kNaMaxDevices) return SD_ENODEV;
    std::lock_guard<std::mutex> lock(g_na_mutex);
    if (!g_na_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return SD_EHIP;
        g_na_ptr[dev] = (unsigned char*)ptr;
    }
    *out = g_na_ptr[dev];
    return SD_OK;
}
}  // namespace

extern "C" {

const char* sd_status_str(sd_status s) {
    switch (s) {
        case SD_OK: return "ok";
        case SD_EINVAL: return "invalid argument";
        case SD_ENOMEM: return "out of KV pages or workspace";
        case SD_EHIP: return "HIP runtime error";
        case SD_ESTATE: return "call out of order";
        case SD_EDEVICE: return "device reported bad input data";
        case SD_ENOTIMPL: return "configuration not supported";
        case SD_ENODEV: return "no gfx950 device";
        case SD_ELIMIT: return "input exceeds the fixed limits of this call";
    }
    return "unknown status";
}

sd_status sd_verify_query_sizes(const sd_config* cfg, uint64_t* kv_pool_bytes,
                                uint64_t* workspace_bytes, uint64_t* weight_pack_bytes) {
    sd_status r = validate_config(cfg);
    if (r != SD_OK) return r;
    if (!kv_pool_bytes || !workspace_bytes || !weight_pack_bytes) return SD_EINVAL;
    const Dims D = dims_of(*cfg);
    const size_t es = D.bf16 ? 2 : 4;
    *kv_pool_bytes = (uint64_t)D.L * cfg->n_pages * 2 * D.hkv * kPageTokens * D.hd * es;
    *workspace_bytes = plan(*cfg).total;
    *weight_pack_bytes = D.bf16 ? (uint64_t)pack_layout(D).total * 2 : 0;
    return SD_OK;
}

sd_status sd_verify_init(const sd_config* cfg, const sd_weights* w, void* kv_pool, void* workspace,
                         void* weight_pack, sd_ctx** out) {
    if (!out) return SD_EINVAL;
    *out = nullptr;
    sd_status r = validate_config(cfg);
    if (r != SD_OK) return r;
    if (!w || !w->embed || !w->lm_head || !w->norm_f || !w->layers || !kv_pool || !workspace)
        return SD_EINVAL;
    if (cfg->dtype == SD_BF16 && !weight_pack) return SD_EINVAL;
    if (((uintptr_t)kv_pool | (uintptr_t)workspace | (uintptr_t)weight_pack) & (kAlign - 1))
        return SD_EINVAL;
    for (int l = 0; l < cfg->n_layers; ++l) {
        const sd_layer_weights& lw = w->layers[l];
        if (!lw.wq || !lw.wk || !lw.wv || !lw.wo || !lw.wg || !lw.wu || !lw.wd || !lw.norm1 ||
            !lw.norm2)
            return SD_EINVAL;
        if (cfg->qk_norm && (!lw.qnorm || !lw.knorm)) return SD_EINVAL;
        // gains are read four elements (8 bytes in bf16) at a time
        uintptr_t g = (uintptr_t)lw.norm1 | (uintptr_t)lw.norm2;
        if (cfg->qk_norm) g |= (uintptr_t)lw.qnorm | (uintptr_t)lw.knorm;
        if (g & 7) return SD_EINVAL;
    }
    if ((uintptr_t)w->norm_f & 7) return SD_EINVAL;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return SD_ENODEV;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return SD_ENODEV;
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) return SD_ENODEV;

    sd_ctx* c = new (std::nothrow) sd_ctx();
    if (!c) return SD_ENOMEM;
    c->cfg = *cfg;
    c->D = dims_of(*cfg);
    c->lay = plan(*cfg);
    c->w = *w;
    c->layers.assign(w->layers, w->layers + cfg->n_layers);
    c->w.layers = nullptr;
    c->device = dev;
    c->attn_cap = std::min(kAttnItemsMax, kAttnWGsPerCU * std::max(prop.multiProcessorCount, 1));
    c->kv.base = kv_pool;
    c->kv.n_pages = cfg->n_pages;
    c->kv.hkv = c->D.hkv;
    c->kv.hd = c->D.hd;
    c->kv.esize = c->D.bf16 ? 2 : 4;
    c->ws = (char*)workspace;
    c->wpack = (char*)weight_pack;
    c->pl = pack_layout(c->D);
    c->users.resize(cfg->max_users);
    c->free_pages.reserve(cfg->n_pages);
    for (int p = cfg->n_pages - 1; p >= 0; --p) c->free_pages.push_back(p);
    const Layout& L = c->lay;
    bool ok = true;
    for (int i = 0; i < cfg->max_pending && ok; ++i) {
        Slot& s = c->slots[i];
        s.base = c->ws + (size_t)i * L.slot_bytes;
        ok &= hipHostMalloc((void**)&s.stage_host, L.st_bytes, hipHostMallocDefault) == hipSuccess;
        ok &= hipHostMalloc((void**)&s.result_host, (size_t)(2 * L.Bmax + 4) * 4,
                            hipHostMallocDefault) == hipSuccess;
        ok &= hipEventCreateWithFlags(&s.done, hipEventDisableTiming) == hipSuccess;
        SlotBufs& b = s.bufs;
        b.tok = (int32_t*)(s.base + L.tok);
        b.cs = (float*)(s.base + L.cs);
        b.x = (float*)(s.base + L.x);
        b.ssq = (float*)(s.base + L.ssq);
        b.nsq = L.nsq;
        b.h = s.base + L.h;
        b.ffn = s.base + L.ffn;
        b.qbuf = s.base + L.qbuf;
        b.attn = s.base + L.attn;
        b.apart = (float*)(s.base + L.apart);
        b.aml = (float*)(s.base + L.aml);
        b.gpart = (float*)(s.base + L.gpart);
        b.gpart_floats = L.gpart_floats;
        b.logits = (float*)(s.base + L.logits);
        b.sstat = (float*)(s.base + L.sstat);
        b.spart = (float*)(s.base + L.spart);
        b.spartB = (float*)(s.base + L.spartB);
        b.lstat = (float*)(s.base + L.lstat);
        b.zd = (float*)(s.base + L.zd);
        b.dnext = (int32_t*)(s.base + L.dnext);
        b.skcnt = (int*)(s.base + L.skcnt);
        b.result = (int32_t*)(s.base + L.result);
        b.bmax = L.Bmax;
    }
    if (ok) {
        // The attention kernel reads whole 32-token blocks and multiplies the
        // value rows past a user's context by an exact 0; zeroing the pool
        // once keeps never-written rows finite (0 * NaN would not be 0).
        const Dims& D = c->D;
        const size_t kv_bytes = (size_t)D.L * cfg->n_pages * 2 * D.hkv * kPageTokens * D.hd * c->kv.esize;
        ok &= hipMemset(kv_pool, 0, kv_bytes) == hipSuccess;
        // the stream-K piece counters start at zero (each launch leaves them so)
        for (int i = 0; ok && i < cfg->max_pending; ++i)
            ok &= hipMemset(c->slots[i].bufs.skcnt, 0, (size_t)kSkCounters * 4) == hipSuccess;
    }
    if (ok && c->D.bf16) {
        // repack the projection matrices and the lm_head into fragment order
        const Dims& D = c->D;
        const PackLayout& P = c->pl;
        for (int l = 0; l < D.L; ++l) {
            const sd_layer_weights& lw = c->layers[l];
            char* base = c->wpack + (size_t)l * P.layer * 2;
            launch_pack(lw.wq, lw.wk, lw.wv, D.nq(), D.nq() + D.nkv(), 0, D.d, D.nqkv(),
                        base + P.qkv * 2, nullptr);
            launch_pack(lw.wo, nullptr, nullptr, 1 << 30, 1 << 30, 0, D.nq(), D.d, base + P.o * 2,
                        nullptr);
            launch_pack(lw.wg, lw.wu, nullptr, 0, 0, 1, D.d, 2 * D.F, base + P.gu * 2, nullptr);
            launch_pack(lw.wd, nullptr, nullptr, 1 << 30, 1 << 30, 0, D.F, D.d, base + P.down * 2,
                        nullptr);
        }
        launch_pack(c->w.lm_head, nullptr, nullptr, 1 << 30, 1 << 30, 0, D.d, D.V,
                    c->wpack + P.lm * 2, nullptr);
        ok = hipGetLastError() == hipSuccess;
    }
    ok = ok && hipDeviceSynchronize() == hipSuccess;
    if (!ok) {
        sd_verify_destroy(c);
        return SD_EHIP;
    }
    *out = c;
    return SD_OK;
}

sd_status sd_verify_destroy(sd_ctx* c) {
    if (!c) return SD_EINVAL;
    for (int i = 0; i < kMaxPending; ++i) {
        Slot& s = c->slots[i];
        if (s.done) {
            (void)hipEventSynchronize(s.done);
            (void)hipEventDestroy(s.done);
        }
        if (s.gexec) (void)hipGraphExecDestroy(s.gexec);
        if (s.stage_host) (void)hipHostFree(s.stage_host);
        if (s.result_host) (void)hipHostFree(s.result_host);
    }
    for (hipEvent_t e : c->prof_ev) (void)hipEventDestroy(e);
    delete c;
    return SD_OK;
}

sd_status sd_user_reset(sd_ctx* c, int32_t user, int32_t prefix_len, int32_t root_token) {
    if (!c || user < 0 || user >= c->cfg.max_users) return SD_EINVAL;
    if (prefix_len < 0 || prefix_len + 2 > c->cfg.max_ctx) return SD_EINVAL;
    if (root_token < 0 || root_token >= c->cfg.vocab) return SD_EINVAL;
    User& u = c->users[user];
    if (u.pending_slot >= 0) return SD_ESTATE;
    const int want = pages_for(prefix_len);
    if (want > (int)u.pages.size() &&
        want - (int)u.pages.size() > (int)c->free_pages.size())
        return SD_ENOMEM;
    release_to(c, u, std::max(want, 0));
    reserve_to(c, u, want);
    u.active = true;
    u.prefix = prefix_len;
    u.root = root_token;
    return SD_OK;
}

sd_status sd_user_release(sd_ctx* c, int32_t user) {
    if (!c || user < 0 || user >= c->cfg.max_users) return SD_EINVAL;
    User& u = c->users[user];
    if (u.pending_slot >= 0) return SD_ESTATE;
    release_to(c, u, 0);
    u.active = false;
    u.prefix = 0;
    u.root = 0;
    return SD_OK;
}

sd_status sd_user_state(sd_ctx* c, int32_t user, int32_t* prefix_len, int32_t* root_token) {
    if (!c || user < 0 || user >= c->cfg.max_users || !prefix_len || !root_token) return SD_EINVAL;
    const User& u = c->users[user];
    if (!u.active) return SD_EINVAL;
    *prefix_len = u.prefix;
    *root_token = u.root;
    return SD_OK;
}

static sd_status kv_copy(sd_ctx* c, int32_t user, int32_t layer, int32_t pos0, int32_t n,
                         const void* k, const void* v, sd_stream stream, int to_pool) {
    if (!c || user < 0 || user >= c->cfg.max_users || layer < 0 || layer >= c->cfg.n_layers ||
        pos0 < 0 || n < 0 || (n > 0 && (!k || !v)))
        return SD_EINVAL;
    User& u = c->users[user];
    if (!u.active) return SD_EINVAL;
    const int limit = to_pool ? u.prefix : (int)u.pages.size() * kPageTokens;
    if (pos0 + n > limit) return SD_EINVAL;
    if (n == 0) return SD_OK;
    if (to_pool && u.pending_slot >= 0) return SD_ESTATE;
    hipStream_t st = (hipStream_t)stream;
    // one launch per kKVCopyPages pages; the page ids ride in the kernel
    // arguments, so nothing is staged and the call does not wait
    const size_t row = (size_t)c->D.hkv * c->D.hd * (c->D.bf16 ? 2 : 4);
    const int end = pos0 + n;
    for (int p0 = pos0; p0 < end;) {
        KVCopyPages pg;
        pg.page0 = p0 / kPageTokens;
        const int pmax = std::min((int)u.pages.size(), pg.page0 + kKVCopyPages);
        for (int j = pg.page0; j < pmax; ++j) pg.id[j - pg.page0] = u.pages[j];
        const int p1 = std::min(end, pmax * kPageTokens);
        launch_kv_copy(c->D, c->kv, pg, layer, p0, p1 - p0, (const char*)k + (size_t)(p0 - pos0) * row,
                       (const char*)v + (size_t)(p0 - pos0) * row, to_pool, st);
        SD_HIP(hipGetLastError());
        p0 = p1;
    }
    return SD_OK;
}

sd_status sd_kv_write(sd_ctx* c, int32_t user, int32_t layer, int32_t pos0, int32_t n,
                      const void* k, const void* v, sd_stream stream) {
    return kv_copy(c, user, layer, pos0, n, k, v, stream, 1);
}

sd_status sd_kv_read(sd_ctx* c, int32_t user, int32_t layer, int32_t pos0, int32_t n, void* k,
                     void* v, sd_stream stream) {
    return kv_copy(c, user, layer, pos0, n, k, v, stream, 0);
}

// Whether a verify pass stores the fp32 logits of every slot: always with
// SD_LOGITS_ALL / SD_LOGITS_UNFUSED or the fp32 configuration; otherwise
// only when something reads them after phase A -- the stochastic race of
// phase B (the stop slot is known only once every slot's statistics are
// complete) or the probabilities of a decode step.
static bool pass_writes_logits(const sd_ctx* c, int mode, const float* probs) {
    return !c->D.bf16 || c->cfg.logits_out != SD_LOGITS_AS_NEEDED || mode == SD_STOCHASTIC ||
           probs != nullptr;
}

// Device work of one pass: staging upload, forward + sampler (or the
// sampler alone on caller logits), result download.  No allocation, no
// memset: the whole sequence can be captured into a graph.
static sd_status enqueue_pass(sd_ctx* c, Slot& s, const BatchView& bv, const float* logits,
                              hipStream_t st, float* probs = nullptr) {
    sd_status rs = hip_status(hipMemcpyAsync(s.base + c->lay.stage, s.stage_host, c->lay.st_bytes,
                                             hipMemcpyHostToDevice, st));
    if (rs == SD_OK) {
        if (logits) {
            launch_prepare(c->D, bv, s.bufs, st);
            launch_sampler(c->D, bv, s.bufs, logits, st);
            rs = hip_status(hipGetLastError());
        } else {
            int groups = 0;
            rs = enqueue_forward(c, s, bv, st, pass_writes_logits(c, bv.mode, probs), &groups);
            if (rs == SD_OK) {
                ProfScope ps(c, SD_K_SAMPLER, st);
                launch_sampler(c->D, bv, s.bufs, s.bufs.logits, st, groups);
                if (probs) launch_probs(c->D, bv, s.bufs, s.bufs.logits, probs, st);
                rs = hip_status(hipGetLastError());
            }
        }
    }
    if (rs == SD_OK)
        rs = hip_status(hipMemcpyAsync(s.result_host, s.bufs.result,
                                       (size_t)(2 * c->lay.Bmax + 4) * 4, hipMemcpyDeviceToHost, st));
    return rs;
}

// Everything the launch shapes and kernel arguments of a pass depend on,
// apart from the staged tables (which the graph's upload re-reads from the
// pinned staging buffer at every launch).
static std::vector<int64_t> launch_key(sd_ctx* c, const Slot& s, const BatchView& bv,
                                       hipStream_t st) {
    std::vector<int64_t> k = {bv.B, bv.T, bv.nd, bv.mode, (int64_t)bv.seed, (int64_t)bv.round,
                              bv.n_items, bv.rows_max, (int64_t)(intptr_t)bv.drafts,
                              (int64_t)(intptr_t)bv.q, (int64_t)(intptr_t)bv.accept_u,
                              (int64_t)(intptr_t)st, c->sk_polls};
    for (int b = 0; b < s.B; ++b) {
        k.push_back(s.users[b]);
        k.push_back(s.L[b]);
        k.push_back(c->users[s.users[b]].prefix);
    }
    return k;
}

// Graph path: replay the slot's graph when the signature matches, else
// capture the pass on `st` (thread-local capture mode), instantiate it and
// launch it.  A stream the caller is already capturing gets the plain
// launches (they become part of the caller's graph).
static sd_status enqueue_graph(sd_ctx* c, Slot& s, const BatchView& bv, hipStream_t st) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    SD_HIP(hipStreamIsCapturing(st, &cs));
    if (cs != hipStreamCaptureStatusNone) return enqueue_pass(c, s, bv, nullptr, st);
    std::vector<int64_t> key = launch_key(c, s, bv, st);
    if (!s.gexec || s.gkey != key) {
        if (s.gexec) {
            (void)hipGraphExecDestroy(s.gexec);
            s.gexec = nullptr;
            s.gkey.clear();
        }
        SD_HIP(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal));
        const sd_status rs = enqueue_pass(c, s, bv, nullptr, st);
        hipGraph_t g = nullptr;
        const hipError_t e = hipStreamEndCapture(st, &g);
        if (rs != SD_OK || e != hipSuccess || !g) {
            if (g) (void)hipGraphDestroy(g);
            return rs != SD_OK ? rs : SD_EHIP;
        }
        hipGraphExec_t ex = nullptr;
        const hipError_t ei = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
        (void)hipGraphDestroy(g);
        if (ei != hipSuccess) return SD_EHIP;
        s.gexec = ex;
        s.gkey = std::move(key);
    }
    return hip_status(hipGraphLaunch(s.gexec, st));
}

// draft_len == NULL: decode step of sd_draft_batch (no drafts, one slot per
// user); probs, if set, receives softmax of each slot's logits.
// Sparse draft distributions of sd_verify_batch_sparse (k == 0: dense q).
struct SparseQ {
    const int32_t* idx = nullptr;
    const float* val = nullptr;
    const float* rest = nullptr;
    int32_t k = 0;
};

static sd_status submit(sd_ctx* c, int32_t batch, int32_t n_users, const int32_t* assign,
                        const int32_t* draft_len, const int32_t* draft_tokens, const float* q,
                        const float* logits, int32_t mode, uint64_t seed, uint64_t round,
                        const float* accept_u, sd_stream stream, bool graph = false,
                        float* probs = nullptr, const int32_t* probs_row = nullptr,
                        SparseQ sq = SparseQ{}) {
    if (!c) return SD_EINVAL;
    if (graph && (stream == nullptr || logits != nullptr)) return SD_EINVAL;
    if (mode != SD_GREEDY && mode != SD_STOCHASTIC && mode != SD_FORCE) return SD_EINVAL;
    const bool need_q = mode == SD_STOCHASTIC && sq.k == 0;
    if (draft_len && (!draft_tokens || (need_q && !q))) return SD_EINVAL;
    const bool sample_only = logits != nullptr;
    if (batch < 0) return SD_EINVAL;
    Slot& s = c->slots[batch % c->cfg.max_pending];
    if (s.pending) return SD_ESTATE;
    std::vector<int> users, Ls;
    int T = 0, nd = 0;
    sd_status r = collect_batch(c, batch, n_users, assign, draft_len, !sample_only, users, Ls, T, nd);
    if (r != SD_OK) return r;
    if (!sample_only) {
        // page reservation for i_m + l_m + 1 tokens per user, all or nothing
        int need = 0;
        for (size_t b = 0; b < users.size(); ++b) {
            const User& u = c->users[users[b]];
            need += std::max(0, pages_for(u.prefix + Ls[b] + 1) - (int)u.pages.size());
        }
        if (need > (int)c->free_pages.size()) return SD_ENOMEM;
        for (size_t b = 0; b < users.size(); ++b) {
            User& u = c->users[users[b]];
            reserve_to(c, u, pages_for(u.prefix + Ls[b] + 1));
        }
    }
    if (probs_row) {
        for (int m : users)
            if (probs_row[m] < 0) {
                if (!sample_only)
                    for (int m2 : users) release_to(c, c->users[m2], pages_for(c->users[m2].prefix));
                return SD_EINVAL;
            }
    }
    s.users = users;
    s.L = Ls;
    s.prow.clear();
    if (probs_row)
        for (int m : users) s.prow.push_back(probs_row[m]);
    s.B = (int)users.size();
    s.T = T;
    s.nd = nd;
    s.batch = batch;
    s.sample_only = sample_only;
    s.logits_ok = sample_only || pass_writes_logits(c, mode, probs);
    int n_items = 0, rows_max = 0;
    build_stage(c, s, mode, !sample_only, &n_items, &rows_max);
    BatchView bv = make_view(c, s);
    bv.B = s.B;
    bv.T = T;
    bv.nd = nd;
    bv.mode = mode;
    bv.seed = seed;
    bv.round = round;
    bv.n_items = n_items;
    bv.rows_max = rows_max;
    bv.drafts = draft_tokens;
    bv.q = q;
    bv.accept_u = accept_u;
    bv.q_idx = sq.idx;
    bv.q_val = sq.val;
    bv.q_rest = sq.rest;
    bv.qk = sq.k;
    hipStream_t st = (hipStream_t)stream;
    // an open profiling window records events between launches: eager path
    sd_status rs = graph && c->prof_class == 0 ? enqueue_graph(c, s, bv, st)
                                               : enqueue_pass(c, s, bv, logits, st, probs);
    if (rs == SD_OK) rs = hip_status(hipEventRecord(s.done, st));
    if (rs != SD_OK) {
        if (!sample_only)
            for (size_t b = 0; b < users.size(); ++b) {
                User& u = c->users[users[b]];
                release_to(c, u, pages_for(u.prefix));
            }
        return rs;
    }
    s.pending = true;
    const int slot_index = (int)(&s - c->slots);
    for (int m : users) c->users[m].pending_slot = slot_index;
    return SD_OK;
}

sd_status sd_verify_batch(sd_ctx* c, int32_t batch, int32_t n_users, const int32_t* assign,
                          const int32_t* draft_len, const int32_t* draft_tokens, const float* q,
                          int32_t mode, uint64_t seed, uint64_t round, const float* accept_u,
                          sd_stream stream) {
    return submit(c, batch, n_users, assign, draft_len, draft_tokens, q, nullptr, mode, seed, round,
                  accept_u, stream);
}

sd_status sd_verify_batch_graph(sd_ctx* c, int32_t batch, int32_t n_users, const int32_t* assign,
                                const int32_t* draft_len, const int32_t* draft_tokens, const float* q,
                                int32_t mode, uint64_t seed, uint64_t round, const float* accept_u,
                                sd_stream stream) {
    return submit(c, batch, n_users, assign, draft_len, draft_tokens, q, nullptr, mode, seed, round,
                  accept_u, stream, true);
}

sd_status sd_verify_batch_sparse(sd_ctx* c, int32_t batch, int32_t n_users, const int32_t* assign,
                                 const int32_t* draft_len, const int32_t* draft_tokens,
                                 const int32_t* q_idx, const float* q_val, const float* q_rest,
                                 int32_t q_k, int32_t mode, uint64_t seed, uint64_t round,
                                 const float* accept_u, sd_stream stream) {
    if (!c || q_k < 1 || q_k > kSparseKMax || !q_idx || !q_val || !q_rest) return SD_EINVAL;
    // the race kernel holds one vocab chunk of q in LDS
    const int cw = ((c->D.V + kVocabChunks - 1) / kVocabChunks + 3) & ~3;
    if (cw > kSparseChunkMax) return SD_ENOTIMPL;
    SparseQ sq;
    sq.idx = q_idx;
    sq.val = q_val;
    sq.rest = q_rest;
    sq.k = q_k;
    return submit(c, batch, n_users, assign, draft_len, draft_tokens, nullptr, nullptr, mode, seed,
                  round, accept_u, stream, false, nullptr, nullptr, sq);
}

sd_status sd_draft_batch(sd_ctx* c, int32_t batch, int32_t n_users, const int32_t* assign,
                         int32_t mode, uint64_t seed, uint64_t round, float* probs,
                         const int32_t* probs_row, sd_stream stream) {
    if (mode == SD_FORCE || (probs_row && !probs)) return SD_EINVAL;
    return submit(c, batch, n_users, assign, nullptr, nullptr, nullptr, nullptr, mode, seed, round,
                  nullptr, stream, false, probs, probs_row);
}

sd_status sd_sample_logits(sd_ctx* c, int32_t batch, int32_t n_users, const int32_t* assign,
                           const int32_t* draft_len, const int32_t* draft_tokens, const float* q,
                           const float* logits, int32_t mode, uint64_t seed, uint64_t round,
                           const float* accept_u, sd_stream stream) {
    if (!logits) return SD_EINVAL;
    return submit(c, batch, n_users, assign, draft_len, draft_tokens, q, logits, mode, seed, round,
                  accept_u, stream);
}

sd_status sd_accept(sd_ctx* c, int32_t batch, int32_t* n_accepted, int32_t* out_token,
                    int32_t commit) {
    if (!c || batch < 0 || !n_accepted || !out_token) return SD_EINVAL;
    Slot& s = c->slots[batch % c->cfg.max_pending];
    if (!s.pending || s.batch != batch) return SD_ESTATE;
    if (hipEventSynchronize(s.done) != hipSuccess) return SD_EHIP;
    const int Bmax = c->lay.Bmax;
    const int flags = s.result_host[2 * Bmax];
    const bool ok = flags == 0;
    for (int b = 0; b < s.B; ++b) {
        User& u = c->users[s.users[b]];
        if (ok) {
            n_accepted[s.users[b]] = s.result_host[b];
            out_token[s.users[b]] = s.result_host[Bmax + b];
        }
        if (!s.sample_only) {
            if (ok && commit) {
                u.prefix += 1 + s.result_host[b];
                u.root = s.result_host[Bmax + b];
            }
            release_to(c, u, pages_for(u.prefix));
        }
        u.pending_slot = -1;
    }
    s.pending = false;
    return ok ? SD_OK : SD_EDEVICE;
}

sd_status sd_debug_logits(sd_ctx* c, int32_t batch, float* dst, sd_stream stream) {
    if (!c || batch < 0 || !dst) return SD_EINVAL;
    Slot& s = c->slots[batch % c->cfg.max_pending];
    if (!s.pending || s.batch != batch || s.sample_only || !s.logits_ok) return SD_ESTATE;
    hipStream_t st = (hipStream_t)stream;
    SD_HIP(hipStreamWaitEvent(st, s.done, 0));
    SD_HIP(hipMemcpyAsync(dst, s.bufs.logits, (size_t)s.T * c->D.V * 4, hipMemcpyDeviceToDevice, st));
    return SD_OK;
}

sd_status sd_debug_wait_limit(sd_ctx* c, int32_t max_polls) {
    if (!c) return SD_EINVAL;
    c->sk_polls = max_polls < 0 ? kSkPollsDefault : max_polls;
    return SD_OK;
}

sd_status sd_profile_begin(sd_ctx* c, int32_t kclass, int32_t max_launches) {
    if (!c || kclass < SD_K_QKV || kclass > SD_K_SMALL || max_launches < 1 || max_launches > 65536)
        return SD_EINVAL;
    if (c->prof_class) return SD_ESTATE;
    while ((int)c->prof_ev.size() < 2 * max_launches) {
        hipEvent_t e;
        SD_HIP(hipEventCreate(&e));
        c->prof_ev.push_back(e);
    }
    c->prof_used = 0;
    c->prof_class = kclass;
    return SD_OK;
}

sd_status sd_profile_end(sd_ctx* c, double* total_ms, int32_t* launches) {
    if (!c || !total_ms || !launches) return SD_EINVAL;
    if (!c->prof_class) return SD_ESTATE;
    double tot = 0.0;
    for (int i = 0; i < c->prof_used; ++i) {
        SD_HIP(hipEventSynchronize(c->prof_ev[2 * i + 1]));
        float ms = 0.f;
        SD_HIP(hipEventElapsedTime(&ms, c->prof_ev[2 * i], c->prof_ev[2 * i + 1]));
        tot += ms;
    }
    *total_ms = tot;
    *launches = c->prof_used;
    c->prof_class = 0;
    c->prof_used = 0;
    return SD_OK;
}

sd_status sd_sample_logits_noalloc(int32_t n_users, const int32_t* user_ids, const int32_t* draft_len,
                                   int32_t vocab, const int32_t* draft_tokens, const float* q,
                                   const float* logits, int32_t mode, uint64_t seed, uint64_t round,
                                   const float* accept_u, int32_t* result, sd_stream stream) {
    if (mode != SD_GREEDY && mode != SD_STOCHASTIC && mode != SD_FORCE) return SD_EINVAL;
    if (n_users < 1 || !user_ids || !draft_len || !draft_tokens || !logits || !result || vocab < 1)
        return SD_EINVAL;
    if (mode == SD_STOCHASTIC && !q) return SD_EINVAL;
    if (n_users > SD_NOALLOC_MAX_USERS || vocab > SD_NOALLOC_MAX_VOCAB) return SD_ELIMIT;
    NoallocMeta meta;
    meta.B = n_users;
    meta.V = vocab;
    int T = 0, nd = 0;
    for (int b = 0; b < n_users; ++b) {
        if (user_ids[b] < 0 || draft_len[b] < 1) return SD_EINVAL;
        if (draft_len[b] >= SD_NOALLOC_MAX_SLOTS) return SD_ELIMIT;
        meta.user_id[b] = user_ids[b];
        meta.L[b] = draft_len[b];
        T += draft_len[b] + 1;
        nd += draft_len[b];
        if (T > SD_NOALLOC_MAX_SLOTS) return SD_ELIMIT;
    }
    unsigned char* sp = nullptr;
    sd_status r = na_scratch(&sp);
    if (r != SD_OK) return r;
    int32_t* tab = (int32_t*)sp;
    NoallocTables t;
    t.user_id = tab;
    t.L = t.user_id + kNoallocUsers;
    t.slot_off = t.L + kNoallocUsers;
    t.draft_off = t.slot_off + kNoallocUsers + 1;
    t.slot_b = t.draft_off + kNoallocUsers + 1;
    t.slot_j = t.slot_b + kNoallocSlots;
    t.flags = t.slot_j + kNoallocSlots;
    BatchView bv{};
    bv.B = n_users;
    bv.T = T;
    bv.nd = nd;
    bv.mode = mode;
    bv.seed = seed;
    bv.round = round;
    bv.user_id = t.user_id;
    bv.L = t.L;
    bv.slot_off = t.slot_off;
    bv.draft_off = t.draft_off;
    bv.slot_b = t.slot_b;
    bv.slot_j = t.slot_j;
    bv.drafts = draft_tokens;
    bv.q = q;
    bv.accept_u = accept_u;
    bv.qk = 0;
    bv.flags = t.flags;
    SlotBufs sb{};
    sb.sstat = (float*)(sp + kNaTables);
    sb.spart = (float*)(sp + kNaTables + kNaSstat);
    sb.spartB = (float*)(sp + kNaTables + kNaSstat + kNaSpart);
    sb.result = result;  // the caller's output: n_acc [B], token [B], flags
    sb.bmax = n_users;
    Dims D{};
    D.V = vocab;
    hipStream_t st = (hipStream_t)stream;
    launch_noalloc_stage(meta, t, draft_tokens, st);
    launch_sampler(D, bv, sb, logits, st);
    return hip_status(hipGetLastError());
}

}  // extern "C"
