/*
 * dels.h -- C ABI of the DeLS-Spec block-drafting library (libdels.so), MI355X / gfx950.
 *
 * The library drafts one block of B tokens per sequence the way DeLS-Spec does
 * (Sec. 4.3, Algorithm 1): at each draft position a local head is stepped on the
 * tokens drafted so far, its short-context logits are fused with fixed long-context
 * (DFlash) logits and an optional log unigram prior,
 *
 *     l_v = w_long * l_L,v + alpha * l_S,v - beta * l_P,v          (Sec. 4.3 fusion)
 *
 * and the greedy (argmax) token is taken.  The local head is the paper's RNN head
 * (App. A): a bias-free one-layer GRU over the frozen target embedding, a SiLU
 * projection to rank r and a vocabulary head,
 *
 *     h' = GRU(E[u], h),   rho = SiLU(W_rank h'),   l_S = W_vocab rho.
 *
 * GRU gates use the (r, z, n) row order: r = sigmoid(W_ir x + W_hr h),
 * z = sigmoid(W_iz x + W_hz h), n = tanh(W_in x + r * (W_hn h)),
 * h' = (1 - z) * n + z * h, and h = 0 at the start of every block.
 *
 * Conventions shared by every entry point
 *  - All tensor pointers are DEVICE pointers owned by the caller and must stay
 *    valid until the work queued on `stream` has completed.  Tensors are dense and
 *    row-major.  Bulk tensors (logits, weights, scores, workspace) must be 16-byte
 *    aligned; int32/float vectors 4-byte aligned.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).  Every
 *    call only enqueues work; nothing is synchronised.  Outputs are valid once the
 *    caller has synchronised the stream.
 *  - The library never allocates device memory in a call.  Scratch memory is the
 *    caller's `workspace`; one workspace must not be used by two calls that may run
 *    concurrently.  The only mutable global state is the per-GPU scratch array of
 *    dls_draft_block_noalloc.
 *  - Arguments are checked on the host before any HIP call.  A failed check returns
 *    DLS_ERR_ARG / DLS_ERR_SHAPE / DLS_ERR_DTYPE / DLS_ERR_WORKSPACE and enqueues
 *    nothing.  No usable GPU gives DLS_ERR_DEVICE; a HIP failure gives DLS_ERR_HIP.
 *    dls_last_error() returns a message for the last failure on the calling thread.
 *  - Not checked (that would need a device sync): token ids lie in [0, V); logits
 *    and weights are finite.  -inf is allowed in long logits (a masked token); NaN
 *    gives unspecified results.
 *  - Empty work (rows == 0, batch == 0 or B == 0) returns DLS_OK and enqueues nothing.
 *  - Greedy decoding takes the lowest index among equal fused values.  All
 *    arithmetic is float32; bf16 inputs are widened exactly.
 */
#ifndef DELS_H
#define DELS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DLS_ABI_VERSION 4

typedef enum dls_status {
  DLS_OK = 0,
  DLS_ERR_ARG = 1,        /* NULL or misaligned pointer, non-finite weight argument */
  DLS_ERR_SHAPE = 2,      /* size outside the documented limits */
  DLS_ERR_DTYPE = 3,      /* unknown or inconsistent element type */
  DLS_ERR_WORKSPACE = 4,  /* workspace smaller than the size query returned */
  DLS_ERR_DEVICE = 5,     /* no usable gfx950 device */
  DLS_ERR_HIP = 6         /* a HIP runtime call or kernel launch failed */
} dls_status;

typedef enum dls_dtype { DLS_F32 = 0, DLS_BF16 = 1 } dls_dtype;

/* dls_fusion.flags */
#define DLS_FIRST_ROW_LONG_ONLY 0x1u  /* Algorithm 1 literally: draft position 0 is decoded
                                         from the long logits alone (no short logits, no
                                         prior) and the head only consumes drafted tokens;
                                         the last accepted token is then unused. */
#define DLS_EXCLUSIVE_DEVICE 0x2u     /* The caller guarantees that no other kernel runs on the
                                         device during the call.  The persistent drafting kernel
                                         is then launched as an ordinary dispatch rather than a
                                         cooperative one, which on MI355X saves about 17 us of
                                         dispatch time per call.  If other work does hold compute
                                         units, workgroups wait for them; a wait longer than the
                                         hand-off spin budget (a fraction of a second) sets the
                                         workspace error word.  Ignored by the per-position path
                                         and by dls_combine_logits. */

/* Fusion weights (Sec. 4.3).  The paper uses w_long = 1 and alpha = beta = 0.3;
   alpha = beta = 0 is the DFlash baseline (Sec. 5.6). */
typedef struct dls_fusion {
  float w_long;    /* weight on the long logits                       */
  float alpha;     /* weight on the short (local-head) logits         */
  float beta;      /* weight subtracted on the log unigram prior      */
  uint32_t flags;  /* DLS_FIRST_ROW_LONG_ONLY | DLS_EXCLUSIVE_DEVICE, or 0 */
} dls_fusion;

/* Per-row statistics of the fused distribution, for the decoded token t.
 *   score     = l_t - (w_long * lse_long + alpha * lse_short)
 *             = w_long*log softmax(l_L)_t + alpha*log softmax(l_S)_t - beta*l_P,t
 *   logprob   = l_t - lse_fused = log softmax(l)_t (the distribution Algorithm 1 decodes)
 *   gap       = top-1 minus top-2 fused value (+inf when V == 1)
 *   lse_*     = log-sum-exp over the vocabulary of l_L, l_S and l
 * A row without short logits (DLS_FIRST_ROW_LONG_ONLY, position 0) has
 * lse_short = NaN and score = l_t - w_long * lse_long. */
typedef struct dls_row_stats {
  float score;
  float logprob;
  float gap;
  float lse_long;
  float lse_short;
  float lse_fused;
} dls_row_stats;

/* The two local heads of App. A. */
typedef enum dls_head_kind {
  DLS_HEAD_RNN = 0,     /* rho_i = SiLU(W_rank GRU(E_tgt(z_i))),  l_S = W_vocab rho_i */
  DLS_HEAD_MARKOV = 1   /* rho_i = E_M(x_{i-1}),                  l_S = W_M rho_i     */
} dls_head_kind;

/* Local head (App. A).  All tensors share `dtype` (DLS_BF16 or DLS_F32).
 * kind DLS_HEAD_RNN:
 *   emb     [V, d]   frozen target embedding E_tgt
 *   w_ih    [3H, d]  GRU input weights, rows (r, z, n)
 *   w_hh    [3H, H]  GRU recurrent weights, rows (r, z, n)
 *   w_rank  [r, H]   low-rank projection (followed by SiLU)
 *   w_vocab [V, r]   vocabulary head
 * kind DLS_HEAD_MARKOV (d and H are ignored, w_ih, w_hh and w_rank may be NULL):
 *   emb     [V, r]   E_M, the low-rank state of each previous token
 *   w_vocab [V, r]   W_M, the low-rank vocabulary head
 * prepared  NULL, or a device buffer filled by dls_prepare_head from these same tensors;
 *           it enables the persistent drafting kernel (see below)
 * prepared_bytes  the size of that buffer in bytes (0 when prepared is NULL).  A drafting
 *           call checks on the host that it is at least dls_prepare_head_size(head)
 *           (DLS_ERR_WORKSPACE otherwise); the persistent kernel checks the buffer's header,
 *           written by dls_prepare_head, against the head's shapes and tensor pointers and
 *           fails with DLS_DRAFT_ERR_PREPARED (see dls_draft_block_error) if they differ
 * Limits: 1 <= V <= 2^24; d, H, r multiples of 8 with 8 <= d <= 16384,
 * 8 <= H <= 4096, 8 <= r <= 512 (RNN); 8 <= r <= 512, r a multiple of 8 (Markov). */
typedef struct dls_local_head {
  int32_t V, d, H, r;
  dls_dtype dtype;
  const void *emb;
  const void *w_ih;
  const void *w_hh;
  const void *w_rank;
  const void *w_vocab;
  const void *prepared;
  int32_t kind;        /* dls_head_kind */
  int32_t reserved;    /* 0 */
  size_t prepared_bytes;
} dls_local_head;

/* ---------------------------------------------------------------------------------
 * One-time preparation of a bf16 head for the persistent drafting kernel (App. A head,
 * rearranged; nothing of the method changes):
 *  - RNN: the GRU input projection is folded into a table T[u] = W_ih E[u] of [V, 3H]
 *    float32 values (E is frozen and the GRU has no bias, so the input term depends on
 *    the token only); T is accumulated in float32 from exact bf16 products;
 *  - W_vocab (W_M) and, for the RNN head, W_hh are copied into the operand order of the
 *    bf16 matrix cores.
 * The buffer needs dls_prepare_head_size(head) bytes (RNN: V*3H*4 + V*r*2 + 3H*H*2 +
 * small, 1.98 GB for V = 151,936, H = 1024, r = 256; Markov: V*r*2 + small) and stays
 * valid while the head tensors are unchanged.  Requirements: dtype DLS_BF16, r in {32,
 * 64, 128, 256}, and H a multiple of 32 for the RNN head; otherwise DLS_ERR_SHAPE /
 * DLS_ERR_DTYPE, and dls_prepare_head_size returns 0.  Asynchronous on `stream`. */
size_t dls_prepare_head_size(const dls_local_head *head);
dls_status dls_prepare_head(const dls_local_head *head, void *prepared, size_t bytes, void *stream);

/* ---------------------------------------------------------------------------------
 * Fused combine + greedy argmax over independent rows (Sec. 4.3 fusion and the
 * decode step of Algorithm 1), with the short logits given.
 *   long_logits, short_logits  [rows, V] of `dtype`
 *   prior        [V] float32 log unigram prior l_P, or NULL (then beta is ignored)
 *   out_token    [rows] int32, the argmax of the fused logits
 *   out_stats    [rows] dls_row_stats, or NULL
 *   out_scores   [rows, V] float32, the full row of scores c_v (see dls_row_stats), or NULL
 *   workspace    at least dls_combine_logits_workspace_size(rows, V) bytes (may be
 *                NULL when that size is 0)
 * Limits: 1 <= V <= 2^24, 0 <= rows <= 2^20.  The DLS_FIRST_ROW_LONG_ONLY flag is
 * not used here. */
size_t dls_combine_logits_workspace_size(int64_t rows, int32_t V);
dls_status dls_combine_logits(const void *long_logits, const void *short_logits,
                              dls_dtype dtype, const float *prior, int64_t rows, int32_t V,
                              dls_fusion fusion, int32_t *out_token, dls_row_stats *out_stats,
                              float *out_scores, void *workspace, size_t ws_bytes,
                              void *stream);

/* ---------------------------------------------------------------------------------
 * One draft block per sequence (Algorithm 1, the decoding loop).
 * Two implementations share this entry point.  With head->prepared set and a supported
 * shape (bf16 head, H/16 <= number of CUs, r divisible by H/16 with at most 16 rank rows
 * per group, and the per-CU share of W_vocab fitting in AGPRs + LDS) one persistent kernel
 * keeps the head weights on chip for the whole block, for at most 64 sequences per launch
 * (a larger batch runs as consecutive launches of 64 on the same workspace and stream;
 * sampling keys its noise by each sequence's index in the whole call, so the split does not
 * change a draw); otherwise each position is a sequence of kernel launches.
 * dls_draft_block_path tells which is used.
 * The workspace must be zero-filled before its first use; the library keeps it
 * consistent afterwards.  A persistent call that fails sets the workspace's error word
 * (read it with dls_draft_block_error; the call itself has returned DLS_OK long before,
 * since it only enqueues work).  A failed call writes token -1 at every position it did
 * not finish drafting (all positions unless only the statistics failed) and NaN into
 * every statistics row it could not merge, so that no stale output passes for a draft.
 * Later persistent calls on a workspace whose error word is set do nothing but write
 * the same sentinels, until the workspace is zero-filled again.
 *   head         RNN or Markov local head (see dls_local_head); device pointers
 *   long_logits  [batch, B, V] of `long_dtype`; row j is the long logits of draft
 *                position j
 *   last_token   [batch] int32, the last accepted token; it is the head's first input
 *                (unused with DLS_FIRST_ROW_LONG_ONLY).  Values must lie in [0, V); one
 *                outside is read as token 0 (no fault, but a meaningless draft)
 *   prior        [V] float32 or NULL
 *   out_tokens   [batch, B] int32 drafted tokens; token j feeds the head at j + 1
 *   out_stats    [batch, B] dls_row_stats, or NULL
 *   workspace    at least dls_draft_block_workspace_size(head, batch, B) bytes
 * Limits: 1 <= batch <= 256, 1 <= B <= 64 (0 is a no-op), the head limits above,
 * long_dtype F32 or BF16. */
size_t dls_draft_block_workspace_size(const dls_local_head *head, int32_t batch, int32_t B);
/* 1: the persistent kernel would be used for these arguments, 0: per-position launches,
 * negative: the arguments are invalid.  Needs the device (it counts its CUs). */
int dls_draft_block_path(const dls_local_head *head, int32_t batch, int32_t B, dls_dtype long_dtype,
                         int has_prior);
dls_status dls_draft_block(const dls_local_head *head, const void *long_logits,
                           dls_dtype long_dtype, const int32_t *last_token, const float *prior,
                           int32_t batch, int32_t B, dls_fusion fusion, int32_t *out_tokens,
                           dls_row_stats *out_stats, void *workspace, size_t ws_bytes,
                           void *stream);

/* Error word of a drafting workspace (0 when every persistent call on it succeeded). */
#define DLS_DRAFT_ERR_STALLED 1   /* a hand-off between workgroups did not arrive within the spin
                                     budget (about a second): typically other kernels held compute
                                     units during a DLS_EXCLUSIVE_DEVICE call */
#define DLS_DRAFT_ERR_PREPARED 2  /* head->prepared holds the prepared form of another head (its
                                     header's shapes or tensor pointers differ from head's) */
/* Copy the error word of `workspace` (a drafting workspace of ws_bytes >= 256 bytes, as
 * passed to dls_draft_block) into *out_error, asynchronously on `stream` after the work
 * already queued there: one int32 in memory the device can write (device memory, or host
 * memory from hipHostMalloc).  With workspace == NULL it reads the error word of the
 * current device's scratch used by dls_draft_block_noalloc.  Nothing is synchronised. */
dls_status dls_draft_block_error(const void *workspace, size_t ws_bytes, int32_t *out_error,
                                 void *stream);

/* Per-position fusion weights (Sec. 5.6 learns one alpha_j and one beta_j for each
 * draft position; App. C lists them): host arrays of B values that replace fusion.alpha
 * and fusion.beta at position j.  NULL keeps the scalar for every position.  Values must
 * be finite.  Otherwise dls_draft_block_scheduled is dls_draft_block. */
typedef struct dls_fusion_schedule {
  const float *alpha;   /* [B] host, or NULL */
  const float *beta;    /* [B] host, or NULL */
} dls_fusion_schedule;
dls_status dls_draft_block_scheduled(const dls_local_head *head, const void *long_logits,
                                     dls_dtype long_dtype, const int32_t *last_token,
                                     const float *prior, int32_t batch, int32_t B, dls_fusion fusion,
                                     dls_fusion_schedule schedule, int32_t *out_tokens,
                                     dls_row_stats *out_stats, void *workspace, size_t ws_bytes,
                                     void *stream);

/* Temperature sampling (the Decode step of Algorithm 1 at temperature T; the paper
 * reports T = 0 and T = 1).  temperature = 0 is greedy decoding, exactly as in
 * dls_draft_block.  A finite T > 0 draws each drafted token from softmax(l / T) by the
 * Gumbel-max rule: the token is the argmax over v of l_v / T + g_v, with g_v standard
 * Gumbel noise -log(-log u_v).  u_v of row (sequence b, position j) is word v mod 4 of
 * Philox4x32-10 (Salmon et al., SC 2011) at counter (v / 4, j, b, 0) under the key
 * (seed mod 2^32, seed / 2^32), mapped as ((x >> 9) + 1/2) / 2^23; the draws therefore
 * depend on (seed, b, j, v) only, not on the batch size, the path or the launch shape.
 * With T > 0 the row statistics refer to the sampled distribution: logprob =
 * l_t / T - lse_fused, lse_fused = log-sum-exp of l / T, gap = top-1 minus top-2 of
 * l / T + g; score keeps its definition (it does not depend on T). */
typedef struct dls_sampling {
  float temperature;   /* 0 (greedy) or finite > 0 */
  uint32_t reserved;   /* 0 */
  uint64_t seed;
} dls_sampling;
dls_status dls_draft_block_sampled(const dls_local_head *head, const void *long_logits,
                                   dls_dtype long_dtype, const int32_t *last_token,
                                   const float *prior, int32_t batch, int32_t B, dls_fusion fusion,
                                   dls_fusion_schedule schedule, dls_sampling sampling,
                                   int32_t *out_tokens, dls_row_stats *out_stats, void *workspace,
                                   size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------------------
 * Adaptive fusion.  Sec. 7 proposes adjusting the local-head and prior weights by the
 * token-level entropy or confidence of the long logits, without a rule; the library's
 * rule, per row (sequence b, position j) of long logits l_L with p = softmax(l_L):
 *   u = H(p) / log V               DLS_UNC_ENTROPY  (H = -sum_v p_v log p_v, in nats)
 *   u = (1 - max_v p_v) / (1 - 1/V)  DLS_UNC_MAXPROB
 *   (u = 0 when V = 1; u = 1 when the row has no finite entry)
 *   g = min(1, max(0, (u - h_lo) / (h_hi - h_lo)))
 * and the row fuses with alpha_j * g and beta_j * g: no local terms while the long
 * logits are confident (u <= h_lo), the full weights once they are uncertain
 * (u >= h_hi); h_lo < 0 keeps a floor.  -inf entries (masked tokens) have p = 0. */
typedef enum dls_uncertainty_measure {
  DLS_UNC_ENTROPY = 0,
  DLS_UNC_MAXPROB = 1
} dls_uncertainty_measure;
typedef struct dls_adaptive {
  int32_t measure;    /* dls_uncertainty_measure */
  float h_lo, h_hi;   /* finite, h_lo < h_hi */
  uint32_t reserved;  /* 0 */
} dls_adaptive;
/* What the pre-pass reports for a row.  entropy and max_prob are NaN for a row without a
 * finite entry. */
typedef struct dls_row_uncertainty {
  float entropy;   /* H(p), nats */
  float max_prob;  /* max_v p_v */
  float u;         /* the rule's measure, in [0, 1] up to rounding */
  float gate;      /* g */
} dls_row_uncertainty;

/* Uncertainty and gate of every row of long logits [rows, V] (device memory, float32 or
 * bfloat16, 16-byte aligned, finite values or -inf) into out[rows] (device memory).  The
 * workspace (device, 16-byte aligned; NULL when its size is 0) holds per-range partials when
 * rows are too few to cover the GPU.  Limits: 0 <= rows <= 2^24, 1 <= V <= 2^24. */
size_t dls_long_uncertainty_workspace_size(int64_t rows, int32_t V);
dls_status dls_long_uncertainty(const void *long_logits, dls_dtype dtype, int64_t rows, int32_t V,
                                dls_adaptive rule, dls_row_uncertainty *out, void *workspace,
                                size_t ws_bytes, void *stream);

/* dls_draft_block_sampled with adaptive fusion: the rule's pre-pass over the batch * B
 * rows of long_logits writes out_uncertainty ([batch, B] device memory, required: the
 * drafting kernels read their gates there), then every row (b, j) fuses with
 * alpha_j * g[b, j] and beta_j * g[b, j] (w_long unchanged).  The first row of
 * DLS_FIRST_ROW_LONG_ONLY stays long-only.  The workspace is the drafting workspace of
 * dls_draft_block_workspace_size, which includes the pre-pass partials. */
dls_status dls_draft_block_adaptive(const dls_local_head *head, const void *long_logits,
                                    dls_dtype long_dtype, const int32_t *last_token,
                                    const float *prior, int32_t batch, int32_t B, dls_fusion fusion,
                                    dls_fusion_schedule schedule, dls_sampling sampling,
                                    dls_adaptive rule, dls_row_uncertainty *out_uncertainty,
                                    int32_t *out_tokens, dls_row_stats *out_stats, void *workspace,
                                    size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------------------
 * Allocation-free drafting.  For callers that cannot allocate device memory or own a
 * workspace: code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  dls_draft_block without the workspace arguments: the call runs in a scratch
 * array that the library holds in device memory, one per GPU, of
 * DLS_NOALLOC_SCRATCH_BYTES (32 MiB, reserved on every GPU the library runs on until the
 * process ends).  Calls whose dls_draft_block_workspace_size(head, batch, B) exceeds it
 * return DLS_ERR_WORKSPACE; the Qwen3-shaped heads (H = 1024, r = 256) fit up to batch 64
 * at B = 16.  The call allocates nothing and calls no allocating routine.  Every call on a
 * GPU uses that GPU's one scratch array, which keeps the state of the previous call:
 * calls that may overlap on one GPU (two streams, two threads) race and must be ordered
 * by the caller.  Each call first enqueues a one-workgroup check that zero-fills the
 * scratch when the previous call left its error word set, so a failed call (read its
 * error with dls_draft_block_error(NULL, 0, ...)) does not affect the next one.
 * Otherwise identical to dls_draft_block. */
#define DLS_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
dls_status dls_draft_block_noalloc(const dls_local_head *head, const void *long_logits,
                                   dls_dtype long_dtype, const int32_t *last_token,
                                   const float *prior, int32_t batch, int32_t B, dls_fusion fusion,
                                   int32_t *out_tokens, dls_row_stats *out_stats, void *stream);

/* ---------------------------------------------------------------------------------
 * Prefix-acceptance length (verification step of Algorithm 1): out_len[b] is the
 * number of leading positions j with draft[b, j] == target[b, j], in [0, B].  The
 * paper's acceptance length tau counts the bonus token too: tau = out_len + 1.
 *   draft, target [batch, B] int32;  out_len [batch] int32.
 * Limits: 0 <= batch <= 2^24, 0 <= B <= 4096. */
dls_status dls_accept_len(const int32_t *draft, const int32_t *target, int32_t batch,
                          int32_t B, int32_t *out_len, void *stream);

/* ---------------------------------------------------------------------------------
 * Unigram log-prior (App. A, prior estimation): the counts c(v) of the tokens that lie
 * in [0, V) (others are skipped), then
 *   out_log_prior[v] = log((c(v) + smoothing) / (N + smoothing * V)),
 * N the number of counted tokens, evaluated in float64 and rounded to float32.  The
 * result is the `prior` argument of dls_combine_logits and dls_draft_block.
 *   tokens         [n] int32 (device); the caller selects which tokens count (the paper
 *                  counts the loss-masked response tokens of the training data)
 *   out_counts     [V + 1] uint64 (device, caller-owned): c(0..V-1), then N; overwritten
 *   out_log_prior  [V] float32 (device)
 *   smoothing      the paper's lambda (1.0 by default); > 0, or 0 (then unseen tokens
 *                  get -inf)
 * Limits: 0 <= n <= 2^40, 1 <= V <= 2^24.  Asynchronous on `stream`. */
dls_status dls_unigram_log_prior(const int32_t *tokens, int64_t n, int32_t V, float smoothing,
                                 uint64_t *out_counts, float *out_log_prior, void *stream);

/* ---------------------------------------------------------------------------------
 * Measurement helpers.  They compute nothing of the method: they measure the device's
 * attainable peaks, which benchmarks report beside the vendor figures (8 TB/s HBM,
 * 2.5 PFLOP/s dense bf16) that rooflines are quoted against.  Asynchronous on `stream`;
 * time them with events on it.
 *
 * dls_measure_read streams `bytes` of `buf` once with 16-byte non-temporal loads and
 *   writes one checksum word per workgroup (the XOR of every 32-bit word it read) into
 *   `out`, so that no load is dropped; the XOR of the DLS_MEASURE_READ_WORDS words is
 *   the XOR of the whole buffer.  bytes / duration is the attainable HBM read bandwidth
 *   when the buffer is much larger than the caches (>= 2 GB).
 *   buf  device, 16-byte aligned, bytes a multiple of 16 (> 0)
 *   out  device, DLS_MEASURE_READ_WORDS uint32
 * dls_measure_mfma runs `iters` rounds of 4 independent v_mfma_f32_32x32x16_bf16
 *   products (32768 flops each) in every wave of `groups` workgroups of 256 threads
 *   (4 waves): groups * 4 * iters * 131072 flops.  Every input element is x (a power of
 *   two, exact in bf16), so out[t] (one float per thread, groups * 256 of them) is
 *   exactly iters * 1024 * x^2 (the iteration limit keeps every partial sum below 2^24
 *   units of 16 x^2).
 *   Limits: 1 <= groups <= 65536, 1 <= iters <= 2^18, groups * iters <= 2^24 (at most
 *   8.8 TFLOP, a few milliseconds); x a power of two in [2^-20, 1].
 * Errors: DLS_ERR_ARG for NULL or misaligned pointers, DLS_ERR_SHAPE for sizes outside
 * the limits, DLS_ERR_DEVICE without a device. */
#define DLS_MEASURE_READ_WORDS 8192
dls_status dls_measure_read(const void *buf, size_t bytes, uint32_t *out, void *stream);
dls_status dls_measure_mfma(int32_t groups, int32_t iters, float x, float *out, void *stream);

/* Names and messages. */
const char *dls_status_string(dls_status status);
const char *dls_last_error(void);
int dls_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* DELS_H */
