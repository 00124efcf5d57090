/*
 * sd_verify.h -- C ABI of the batched speculative-verify library (gfx950).
 *
 * The library runs the edge server's verification step of distributed
 * speculative decoding (DiP-SD, arXiv 2604.20919, Sec. II-A step 2): one
 * target-model forward over a batch of users, each bringing its cached
 * prefix plus l_m drafted tokens, then per-user accept/reject with one bonus
 * or resampled token.  A batch is one column n of the user-to-batch
 * assignment x_mn (eq. 7-8), every user in it has an integer draft length
 * l_m >= 1 (eq. 9), and a declared batch is never empty (eq. 10).
 *
 * Conventions for every entry point:
 *   - Every call returns an sd_status (0 = SD_OK, negative = error).  No call
 *     throws or aborts.  On any error return nothing has changed: no user
 *     state, page, or pending batch is modified and nothing was enqueued.
 *   - "device" pointers are HIP device allocations on the context's device;
 *     "host" pointers are ordinary host memory.  The caller owns every buffer
 *     it passes; the library keeps device pointers (weights, KV pool,
 *     workspace) until sd_verify_destroy and never allocates or frees device
 *     memory itself.
 *   - Streams are hipStream_t values passed as sd_stream (NULL = the null
 *     stream).  Work is enqueued asynchronously; sd_accept is the only call
 *     that waits for the GPU.
 *   - One context must not be used from two host threads at once.
 *   - The tensor element type is set by sd_config.dtype: SD_BF16 (bf16
 *     weights, bf16 KV cache, bf16 GEMM inputs, fp32 residual stream) or
 *     SD_F32 (everything fp32).  Norm gains use the same type.
 */
#ifndef SD_VERIFY_H
#define SD_VERIFY_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t sd_status;
enum {
    SD_OK = 0,
    SD_EINVAL = -1,   /* bad argument (range, shape, unknown user, empty batch) */
    SD_ENOMEM = -2,   /* KV page pool exhausted or workspace too small */
    SD_EHIP = -3,     /* a HIP runtime call failed */
    SD_ESTATE = -4,   /* call out of order (batch pending / not pending) */
    SD_EDEVICE = -5,  /* the GPU found bad input data (token id out of range), or a
                         bounded wait of one workgroup for another gave up */
    SD_ENOTIMPL = -6, /* configuration the library does not implement */
    SD_ENODEV = -7,   /* no usable gfx950 device */
    SD_ELIMIT = -8    /* input beyond the fixed limits of sd_sample_logits_noalloc */
};

enum { SD_F32 = 0, SD_BF16 = 1 };

/* verification modes */
enum {
    SD_GREEDY = 0,     /* accept a draft iff it is the target's argmax; the
                          correction / bonus token is the argmax */
    SD_STOCHASTIC = 1, /* speculative sampling: accept iff u < p(d)/q(d); on the
                          first rejection draw from norm(max(0, p - q)); if all
                          drafts pass draw the bonus token from p */
    SD_FORCE = 2       /* teacher forcing: every draft is accepted; the returned
                          token is the argmax after the last draft (prefill) */
};

typedef void* sd_stream; /* a hipStream_t */

typedef struct sd_config {
    int32_t n_layers;     /* J */
    int32_t d_model;      /* h1 */
    int32_t n_q_heads;
    int32_t n_kv_heads;   /* n_q_heads must be a multiple */
    int32_t head_dim;     /* 64 or 128 */
    int32_t d_ffn;        /* h2 (SwiGLU width) */
    int32_t vocab;
    int32_t qk_norm;      /* 1: per-head RMSNorm on q and k before RoPE */
    int32_t dtype;        /* SD_BF16 or SD_F32 */
    int32_t page_tokens;  /* KV page size in tokens; must be 16 */
    int32_t n_pages;      /* pages in the KV pool */
    int32_t max_users;    /* user ids are 0 .. max_users-1 */
    int32_t max_draft;    /* largest l_m accepted (<= 64) */
    int32_t max_batch_users;  /* most users in one batch */
    int32_t max_batch_tokens; /* most query slots sum(l_m + 1) in one batch */
    int32_t max_ctx;      /* largest i_m + l_m + 1 of any user */
    int32_t max_pending;  /* batches that may be in flight at once (1..8) */
    float rope_base;      /* RoPE base (1e6 for Qwen3 shapes) */
    float rms_eps;        /* RMSNorm epsilon */
    int32_t logits_out;   /* SD_LOGITS_AS_NEEDED (0), SD_LOGITS_ALL or SD_LOGITS_UNFUSED */
} sd_config;

/* Where the accept step of Sec. II-A step 2 gets each slot's softmax
 * statistics (row max, sum of exp(z - max), argmax, logit of the next
 * draft) and which passes store the fp32 logits [sum(l_m+1)][vocab].
 * bf16 configuration:
 *   SD_LOGITS_AS_NEEDED  the lm_head product emits the statistics from its
 *                        epilogue; logits are stored only when a later step
 *                        reads them: SD_STOCHASTIC (the resampling race at
 *                        the stop slot, which is known only after every
 *                        slot's statistics) and decode steps with probs.
 *                        SD_GREEDY / SD_FORCE passes store none, and
 *                        sd_debug_logits returns SD_ESTATE for them;
 *   SD_LOGITS_ALL        statistics from the epilogue, logits stored by
 *                        every pass;
 *   SD_LOGITS_UNFUSED    logits stored by every pass and the statistics
 *                        computed from them by separate kernels (the
 *                        sd_sample_logits path).  Decisions and tokens equal
 *                        the fused modes' except where u lies within a few
 *                        fp32 ulps of p(d)/q(d) or two race keys do: the
 *                        exp-sum is added up in another grouping.
 * The fp32 configuration always stores logits and ignores this field. */
enum { SD_LOGITS_AS_NEEDED = 0, SD_LOGITS_ALL = 1, SD_LOGITS_UNFUSED = 2 };

/* Device pointers of one decoder layer, each row-major [out][in] so that
 * y = W x; element type sd_config.dtype.  The gain vectors (norm1, norm2,
 * qnorm, knorm and sd_weights.norm_f) must be 8-byte aligned: they are read
 * four bf16 at a time (sd_verify_init returns SD_EINVAL otherwise). */
typedef struct sd_layer_weights {
    const void* wq;     /* [n_q_heads*head_dim][d_model] */
    const void* wk;     /* [n_kv_heads*head_dim][d_model] */
    const void* wv;     /* [n_kv_heads*head_dim][d_model] */
    const void* wo;     /* [d_model][n_q_heads*head_dim] */
    const void* wg;     /* [d_ffn][d_model]  (SwiGLU gate) */
    const void* wu;     /* [d_ffn][d_model]  (SwiGLU up) */
    const void* wd;     /* [d_model][d_ffn]  (down) */
    const void* norm1;  /* [d_model] pre-attention RMSNorm gain */
    const void* norm2;  /* [d_model] pre-FFN RMSNorm gain */
    const void* qnorm;  /* [head_dim] (ignored unless qk_norm) */
    const void* knorm;  /* [head_dim] (ignored unless qk_norm) */
} sd_layer_weights;

typedef struct sd_weights {
    const void* embed;    /* device [vocab][d_model] */
    const void* lm_head;  /* device [vocab][d_model] (untied) */
    const void* norm_f;   /* device [d_model] final RMSNorm gain */
    const sd_layer_weights* layers; /* host array of n_layers entries (copied) */
} sd_weights;

typedef struct sd_ctx sd_ctx;

/* Device memory the caller must provide for `cfg`.
 * kv_pool_bytes: the paged KV cache, n_pages pages of page_tokens tokens for
 *   every layer and KV head (K and V), in dtype.
 * workspace_bytes: activations, logits and per-batch staging for max_pending
 *   batches of up to max_batch_tokens slots.
 * weight_pack_bytes: the library's copy of the projection matrices and the
 *   lm_head in its streaming layout (SD_BF16; 0 for SD_F32).
 * Returns SD_EINVAL if cfg is inconsistent, SD_ENOTIMPL for shapes the
 * kernels do not cover (SD_BF16: head_dim 128, widths in whole tiles, at most
 * 416 slots per batch, one layer's pages below 4 GB). Host-only; needs no
 * device. */
sd_status sd_verify_query_sizes(const sd_config* cfg, uint64_t* kv_pool_bytes,
                                uint64_t* workspace_bytes, uint64_t* weight_pack_bytes);

/* Create a context on the current HIP device.
 * w: weights as above (device pointers).  With SD_BF16 the projection
 *   matrices (wq, wk, wv, wo, wg, wu, wd) and lm_head are copied here into
 *   weight_pack in the order the GEMM kernels stream them (16-row x 32-column
 *   fragments, each 1 KB contiguous); after this call returns they are no
 *   longer read and the caller may free them.  embed and the norm gains are
 *   read in place until destroy.  With SD_F32 every pointer is kept.
 * kv_pool / workspace / weight_pack: device buffers of at least the queried
 *   sizes, 256-byte aligned, owned by the caller, kept until destroy
 *   (weight_pack may be NULL when its size is 0).  The KV pool is zero-filled
 *   here (attention reads whole blocks past a context's end and needs those
 *   rows finite); KV contents written later must be finite too.
 *   Initialisation work runs on the null stream and is synchronised before
 *   returning.
 * out: receives the context.  Errors: SD_EINVAL (cfg, NULL pointer),
 * SD_ENODEV (current device is not gfx950), SD_EHIP. */
sd_status sd_verify_init(const sd_config* cfg, const sd_weights* w, void* kv_pool,
                         void* workspace, void* weight_pack, sd_ctx** out);

/* Destroy a context (waits for pending work; frees host state only). */
sd_status sd_verify_destroy(sd_ctx* ctx);

/* Start (or restart) user `user` with a cached context of prefix_len tokens
 * i_m (positions 0..i_m-1, Sec. II-A: the prompt plus accepted tokens) and
 * root token root_token (the last emitted token, not yet in the cache; it is
 * query slot 0 of the next verify).  Reserves ceil(i_m / page_tokens) pages;
 * pages the user already held are kept in order, so re-calling with a
 * shorter or equal length keeps the cached entries.  New pages hold
 * undefined data until written with sd_kv_write.
 * Errors: SD_EINVAL (user, length or token out of range), SD_ESTATE (user is
 * in a pending batch), SD_ENOMEM (pool exhausted). */
sd_status sd_user_reset(sd_ctx* ctx, int32_t user, int32_t prefix_len, int32_t root_token);

/* Drop user `user` and return its pages. SD_ESTATE if it is in a pending batch. */
sd_status sd_user_release(sd_ctx* ctx, int32_t user);

/* Read a user's state: cached length i_m and root token (host out-params). */
sd_status sd_user_state(sd_ctx* ctx, int32_t user, int32_t* prefix_len, int32_t* root_token);

/* Copy keys/values of positions pos0..pos0+n-1 of `user`, layer `layer`, into
 * the paged cache.  k, v: device [n][n_kv_heads][head_dim] in dtype (k after
 * QK-norm and RoPE, as the forward stores it).  Requires pos0 + n <= the
 * user's prefix_len.  Enqueued on `stream` without waiting: the page ids
 * travel in the kernel arguments (one launch per 256 pages), so back-to-back
 * writes need no host synchronisation and the call can be captured into a
 * graph.  The page mapping is the one at the time of the call; the data must
 * stay valid until the stream reaches the copy. */
sd_status sd_kv_write(sd_ctx* ctx, int32_t user, int32_t layer, int32_t pos0, int32_t n,
                      const void* k, const void* v, sd_stream stream);

/* Inverse of sd_kv_write (for tests): k, v device [n][n_kv_heads][head_dim];
 * positions may reach prefix_len + l_m + 1 of the user's pending batch.
 * Enqueued on `stream` without waiting, like sd_kv_write. */
sd_status sd_kv_read(sd_ctx* ctx, int32_t user, int32_t layer, int32_t pos0, int32_t n,
                     void* k, void* v, sd_stream stream);

/*
 * Enqueue the verification of batch `batch` on `stream`.
 *   n_users:      M, the length of assign / draft_len
 *   assign:       host [M], batch index of each user (x_mn as one index per
 *                 user); users m with assign[m] == batch form the batch, in
 *                 ascending m.  User ids are 0..M-1 and must have been started
 *                 with sd_user_reset.
 *   draft_len:    host [M], l_m for users in the batch (1..max_draft)
 *   draft_tokens: device int32 [sum l_m], the batch users' drafts in order
 *   q:            device fp32 [sum l_m][vocab], the draft distribution each
 *                 draft was sampled from (dense rows; read only in
 *                 SD_STOCHASTIC mode; may be NULL otherwise)
 *   mode:         SD_GREEDY, SD_STOCHASTIC or SD_FORCE
 *   seed, round:  key of the Philox-4x64-10 stream for this round's draws
 *   accept_u:     device fp32 [sum l_m] accept uniforms, or NULL to draw them
 *                 from Philox
 * For every user the forward covers l_m + 1 query slots: the root token at
 * position i_m followed by the drafts at i_m+1 .. i_m+l_m; their keys and
 * values are written into the user's pages (reserved here).  Device inputs
 * must stay valid until sd_accept(batch) returns.  The call does not wait for
 * the GPU and allocates nothing; the launch shapes depend only on the batch
 * composition (users, l_m, i_m), so a captured graph of it can be replayed
 * while those are unchanged.
 * Errors (nothing enqueued): SD_EINVAL (empty batch, l_m out of range, user
 * not started, sum l_m+1 > max_batch_tokens, i_m+l_m+1 > max_ctx),
 * SD_ESTATE (the batch's workspace slot batch % max_pending is busy, or a
 * user is already pending), SD_ENOMEM (no pages left).
 */
sd_status sd_verify_batch(sd_ctx* ctx, int32_t batch, int32_t n_users, const int32_t* assign,
                          const int32_t* draft_len, const int32_t* draft_tokens, const float* q,
                          int32_t mode, uint64_t seed, uint64_t round, const float* accept_u,
                          sd_stream stream);

/*
 * sd_verify_batch with the device work of the pass replayed from a HIP graph.
 * Same arguments, validation, errors and completion (sd_accept) as
 * sd_verify_batch; `stream` must not be NULL (the null stream cannot be
 * captured).  The batch's workspace slot (batch % max_pending) keeps one
 * graph: the first call captures the pass (staging upload, every kernel,
 * result download) on `stream`, instantiates it and launches it; a later
 * call whose launch signature is unchanged -- the same users with the same
 * l_m and i_m, mode, seed, round, input pointers and stream -- only re-plans
 * the host side (page reservation, staged tables, which the graph's upload
 * reads from the slot's pinned staging buffer at launch time) and launches
 * the graph once.  Any other signature re-captures (so a serving loop whose
 * i_m advance every round re-captures every round; repeated verification of
 * an unchanged batch replays).  The graph holds no memset nodes.  If the
 * caller is itself capturing `stream`, the launches are enqueued into the
 * caller's capture instead.  While a profiling window (sd_profile_begin) is
 * open the pass runs eagerly.  Graphs are released by sd_verify_destroy.
 * Errors as sd_verify_batch, plus SD_EINVAL for a NULL stream and SD_EHIP if
 * capture or instantiation fails (nothing is left pending then).
 */
sd_status sd_verify_batch_graph(sd_ctx* ctx, int32_t batch, int32_t n_users, const int32_t* assign,
                                const int32_t* draft_len, const int32_t* draft_tokens,
                                const float* q, int32_t mode, uint64_t seed, uint64_t round,
                                const float* accept_u, sd_stream stream);

/*
 * sd_verify_batch with sparse draft distributions, the compact payload of
 * Sec. II-A (drafted tokens plus a little probability information per draft).
 * Draft row r (the batch's drafts in order, as for q) is given by q_k token
 * ids q_idx[r][0..q_k-1] (device int32 [sum l_m][q_k], distinct, in
 * 0..vocab-1), their probabilities q_val[r][.] (device fp32 [sum l_m][q_k])
 * and the probability q_rest[r] (device fp32 [sum l_m]) that every token not
 * listed carries:  q_r(k) = q_val[r][i] if k == q_idx[r][i], else q_rest[r].
 * Verification is exact for drafts drawn from that distribution (a device
 * that drafts from its top-q_k tokens plus a uniform remainder, say): the
 * accept ratio uses q_r(d) and the residual at the stop slot uses q_r over
 * the whole vocabulary, exactly as with the equivalent dense row, and the
 * decisions equal those of sd_verify_batch given that dense row.  The rows
 * are read, not checked: they must describe a distribution (the caller's
 * contract, as for dense q).  The sparse rows matter only in SD_STOCHASTIC
 * mode.  Completion and other rules as sd_verify_batch.
 * Errors: SD_EINVAL (q_k outside 1..4096, a NULL row pointer, or the
 * sd_verify_batch conditions), SD_ENOTIMPL (vocab above 262144).
 */
sd_status sd_verify_batch_sparse(sd_ctx* ctx, int32_t batch, int32_t n_users,
                                 const int32_t* assign, const int32_t* draft_len,
                                 const int32_t* draft_tokens, const int32_t* q_idx,
                                 const float* q_val, const float* q_rest, int32_t q_k,
                                 int32_t mode, uint64_t seed, uint64_t round,
                                 const float* accept_u, sd_stream stream);

/*
 * One decode step of a drafting model (Sec. II-A step 1 and eq. 13: each
 * device generates its l_m drafts one token at a time and sends each with
 * its probability; here the drafting model runs in its own context on the
 * GPU).  For every user m with assign[m] == batch (ascending m) the forward
 * covers one query slot, the root token at position i_m; its key and value
 * are written into the user's pages.  The token is then drawn from the
 * slot's distribution p = softmax(z) at temperature 1 -- exponential race
 * keyed by (seed, round, user, slot 0) in SD_STOCHASTIC mode, argmax
 * (lowest index on ties) in SD_GREEDY -- which is the bonus draw of
 * sd_verify_batch with l_m = 0.
 *   probs: device fp32 [rows][vocab], or NULL.  Receives p of each user's
 *          slot, evaluated with the same expression the race uses, so the
 *          drawn token is a draw from exactly these rows; pass them as
 *          sd_verify_batch's q.
 *   probs_row: host int32 [n_users] or NULL: the row of `probs` that
 *          receives user m's distribution (entries of users outside the
 *          batch are ignored; the caller guarantees the rows exist and are
 *          distinct).  NULL: row b for the b-th batch user.  A drafting loop
 *          points step j of user m at row draft_off[m] + j - 1 of the q array
 *          it will pass to sd_verify_batch.  Negative rows: SD_EINVAL.
 * Complete with sd_accept(batch, n_accepted, out_token, commit): every user
 * gets a_m = 0 and out_token = the drawn token; commit = 1 advances the user
 * by one position (i_m += 1, root := token), ready for the next step.
 * Draws of one call are keyed by (seed, round): give every step of a
 * drafting loop its own round value.  SD_FORCE is rejected (SD_EINVAL).
 * SD_EINVAL also for probs_row without probs.  Other errors as
 * sd_verify_batch (max_batch_tokens bounds the batch's user count here).
 */
sd_status sd_draft_batch(sd_ctx* ctx, int32_t batch, int32_t n_users, const int32_t* assign,
                         int32_t mode, uint64_t seed, uint64_t round, float* probs,
                         const int32_t* probs_row, sd_stream stream);

/*
 * Wait for batch `batch` and return its decisions (Sec. II-A steps 2-3):
 *   n_accepted: host [M] (M of the sd_verify_batch call); entry m of every
 *               batch user receives a_m, the number of leading drafts accepted
 *   out_token:  host [M]; entry m receives the resampled token (a_m < l_m) or
 *               the bonus token (a_m == l_m)
 *   commit:     1 = advance each user (Sec. II-A step 4): i_m += 1 + a_m, root
 *               := out_token, pages trimmed to the new length; 0 = leave the
 *               user state unchanged (repeatable measurements)
 * Entries of users outside the batch are not touched.  Returns SD_EDEVICE,
 * without committing, if the GPU saw a token id >= vocab, or if a workgroup
 * of the split gate/up product stopped waiting for the partial sums of
 * another (a bounded wait, well under a second); the results are
 * then not written.
 */
sd_status sd_accept(sd_ctx* ctx, int32_t batch, int32_t* n_accepted, int32_t* out_token,
                    int32_t commit);

/* Diagnostic: run only the accept/resample step of sd_verify_batch on
 * caller-supplied logits (device fp32 [sum(l_m+1)][vocab], slot rows of the
 * batch users in order).  Same arguments and rules otherwise; the batch is
 * then completed with sd_accept(batch, ..., commit = 0). */
sd_status sd_sample_logits(sd_ctx* ctx, int32_t batch, int32_t n_users, const int32_t* assign,
                           const int32_t* draft_len, const int32_t* draft_tokens, const float* q,
                           const float* logits, int32_t mode, uint64_t seed, uint64_t round,
                           const float* accept_u, sd_stream stream);

/* Diagnostic: copy the logits of pending batch `batch` (device fp32
 * [sum(l_m+1)][vocab]) into dst (device), ordered after the batch on
 * `stream`.  SD_ESTATE if the batch is not pending or its pass stored no
 * logits (sd_config.logits_out). */
sd_status sd_debug_logits(sd_ctx* ctx, int32_t batch, float* dst, sd_stream stream);

/* Diagnostic: bound of the waits in the split gate/up product of passes
 * enqueued after this call.  When the product is split over more
 * workgroups than its row tiles, the workgroup that finishes a tile polls a
 * counter until every earlier workgroup of the tile has left its partial
 * sums; after max_polls polls it gives up, and sd_accept of that batch
 * returns SD_EDEVICE.  max_polls = 0 gives up at once (to test that error
 * path); a negative value restores the default (2^18 polls).  Passes whose
 * product takes no split are not affected. */
sd_status sd_debug_wait_limit(sd_ctx* ctx, int32_t max_polls);

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the
 * accept/resample step of sd_sample_logits with no context, no workspace
 * and no allocation of any kind.  Its scratch (batch tables, per-slot
 * statistics, vocab-chunk partials) is a fixed array in the library's
 * device memory, SD_NOALLOC_SCRATCH_BYTES on every GPU the library runs on,
 * held until the process ends; the caller passes only inputs and outputs.
 *   n_users:      B, 1..SD_NOALLOC_MAX_USERS users, in the order the rows
 *                 below follow (any order; no user state is involved)
 *   user_ids:     host [B], ids >= 0 that key the Philox draws (as the
 *                 global user ids of sd_sample_logits do)
 *   draft_len:    host [B], l_m >= 1; T = sum(l_m + 1) <= SD_NOALLOC_MAX_SLOTS
 *   vocab:        V, 1..SD_NOALLOC_MAX_VOCAB
 *   draft_tokens: device [sum l_m] int32, users in order
 *   q:            device [sum l_m][V] fp32 (stochastic mode; else may be NULL)
 *   logits:       device [T][V] fp32, rows user by user, slot 0 first
 *   mode, seed, round, accept_u: as for sd_verify_batch
 *   result:       device int32 [2*B + 1], written on `stream`: n_acc[B],
 *                 then token[B], then a flag word (nonzero: a draft token
 *                 was outside [0, V); n_acc and token are then undefined)
 * Decisions and tokens are those of sd_sample_logits on the same inputs
 * (the same kernels).  Asynchronous on `stream`; nothing waits.  Every call
 * on a GPU uses that GPU's one scratch array, so calls that overlap on one
 * GPU (two streams, two host threads) race and must be ordered by the
 * caller.  The array keeps the last call's contents; everything a call
 * reads from it is written earlier in the same call (the error flag is
 * cleared by its first kernel).
 * Errors (nothing enqueued): SD_EINVAL (bad argument), SD_ELIMIT (more
 * users, slots or vocabulary than the fixed scratch holds), SD_EHIP.
 */
#define SD_NOALLOC_MAX_USERS 64
#define SD_NOALLOC_MAX_SLOTS 1024
#define SD_NOALLOC_MAX_VOCAB (1 << 20)
#define SD_NOALLOC_SCRATCH_BYTES 1179648
sd_status sd_sample_logits_noalloc(int32_t n_users, const int32_t* user_ids, const int32_t* draft_len,
                                   int32_t vocab, const int32_t* draft_tokens, const float* q,
                                   const float* logits, int32_t mode, uint64_t seed, uint64_t round,
                                   const float* accept_u, int32_t* result, sd_stream stream);

/* Kernel classes for sd_profile_begin. */
enum {
    SD_K_QKV = 1,      /* QKV projection GEMM + fused QK-norm/RoPE/KV append */
    SD_K_ATTN = 2,     /* paged attention + chunk combine */
    SD_K_O = 3,        /* output projection GEMM + fused residual/RMSNorm */
    SD_K_GATEUP = 4,   /* gate/up GEMM with the SwiGLU epilogue */
    SD_K_DOWN = 5,     /* down projection GEMM + fused residual/RMSNorm */
    SD_K_LMHEAD = 6,   /* lm_head GEMM */
    SD_K_SAMPLER = 7,  /* accept/resample kernels */
    SD_K_SMALL = 8     /* batch preparation, embedding + first RMSNorm */
};

/* Diagnostic timing: until sd_profile_end, every sd_verify_batch records a
 * pair of HIP events around each launch of kernel class `kclass`, on the
 * stream the kernels run on (up to max_launches pairs; later launches are
 * not timed).  Host-side event creation happens here, not per batch. */
sd_status sd_profile_begin(sd_ctx* ctx, int32_t kclass, int32_t max_launches);

/* Wait for the recorded launches and return their summed duration in
 * milliseconds and their count; stops profiling.  SD_ESTATE if not active. */
sd_status sd_profile_end(sd_ctx* ctx, double* total_ms, int32_t* launches);

/*
 * Achievable peaks of this GPU, for quoting kernel rates against what the
 * chip delivers as well as against its published peaks.  Measurement
 * helpers only: no context is needed and nothing of the verification state
 * is touched.  Both calls are synchronous (they wait for their own events on
 * `stream`) and allocate no device memory.
 *
 * sd_calib_hbm: HBM bandwidth over the caller's device buffer `buf` (16-byte
 * aligned, `bytes` >= 1 MiB and a multiple of 32; its contents are
 * overwritten).  mode 0: device-to-device copy of the first half onto the
 * second; mode 1: read-only stream of the whole buffer.  One warm-up, then
 * `reps` (>= 1) timed launches; *gbs = bytes read plus bytes written per
 * second / 1e9.
 *
 * sd_calib_mfma: dense bf16 matrix-core rate: every SIMD runs independent
 * chains of v_mfma_f32_32x32x16_bf16 (2*32*32*16 FLOPs each) for `iters`
 * (>= 1) rounds with no memory traffic; *tflops = FLOPs per second / 1e12.
 * `sink` is a device float the kernel may write.
 *
 * Errors: SD_EINVAL (bad arguments), SD_ENODEV (current device is not
 * gfx950), SD_EHIP.
 */
sd_status sd_calib_hbm(void* buf, size_t bytes, int32_t mode, int32_t reps, double* gbs,
                       sd_stream stream);
sd_status sd_calib_mfma(float* sink, int32_t iters, double* tflops, sd_stream stream);

/* Static description of a status code. */
const char* sd_status_str(sd_status s);

#ifdef __cplusplus
}
#endif

#endif /* SD_VERIFY_H */
