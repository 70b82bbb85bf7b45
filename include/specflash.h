/*
 * specflash.h -- C ABI of the SpecFLASH draft-verify hot path on MI355X (gfx950).
 *
 * SpecFLASH (arXiv 2505.12728) speeds up large multimodal models with
 * speculative decoding.  One draft-verify round needs three data-parallel
 * operations, exported here:
 *
 *   sd_latent_compress   learned latent queries attend over the visual
 *                        features (Sec. 3.2, Eq. 3; Algorithm 1, Appendix B)
 *   sd_verify_attention  the target model's attention for the K drafted
 *                        positions, scored in one parallel pass over the KV
 *                        cache (Sec. 3.1)
 *   sd_spec_accept       token-wise acceptance / rejection with residual
 *                        resampling (Sec. 3.1, Sec. 3.3), or greedy
 *                        verification for temperature 0 (Sec. 4.2)
 *
 * and, on either side of the acceptance, the steps that produce its inputs:
 *
 *   sd_lm_head_probs     the LM head: hidden states to token distributions
 *                        p = softmax(h W^T / tau) (Sec. 3.1; Sec. 3.3 and
 *                        Algorithm 1 for the draft's P'; tau of Sec. 4.2)
 *   sd_sample_tokens     drafts drawn from their distributions,
 *                        T' ~ Categorical(P') (Algorithm 1)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every tensor pointer is DEVICE memory on the current HIP device, owned by
 *   the caller, dense and row-major in the layout given at each call.  The
 *   library never allocates, frees or keeps device memory.  Its only global
 *   state is a per-device cache of the compute-unit count (filled on the
 *   first call on a device with the value the runtime reports, never
 *   changed afterwards); calls are thread-safe.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   Work is enqueued asynchronously; no call synchronises the host.
 * - Return value: an sd_status.  Arguments are validated on the host before
 *   anything is enqueued; a non-SD_OK status means nothing was launched.
 *   Data-dependent conditions (finite values, ids in range) are
 *   preconditions that the device cannot report; kernels clamp every index
 *   they read so that a violated precondition yields an unspecified result,
 *   never an out-of-bounds access.
 * - dtype: SD_F32 (float32 storage) or SD_BF16 (bfloat16 storage).  All
 *   arithmetic accumulates in float32 and all floating outputs are float32.
 * - Workspace: a caller-owned device buffer of at least the size returned by
 *   the matching *_workspace_size function for the same shape arguments
 *   (NULL is allowed when that size is 0).  Two calls in flight at the
 *   same time must not share a workspace.  Entry points marked "zeroed
 *   workspace" below keep arrival counters in it (the last work-group of a
 *   group of partial results to finish does the combining step, so no
 *   second launch is needed): such a workspace must be all zero before its
 *   first use and again whenever the shape arguments change; every call
 *   returns the counters to zero, so later calls of the same shape reuse
 *   it without clearing.  Other workspaces need no initialisation, and all
 *   other workspace contents are garbage after a call.
 */
#ifndef SPECFLASH_H
#define SPECFLASH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sd_status {
  SD_OK = 0,
  SD_ERR_INVALID_ARG = 1,   /* null pointer, non-positive or inconsistent size */
  SD_ERR_UNSUPPORTED = 2,   /* valid but not implemented: head size, dtype, ... */
  SD_ERR_WORKSPACE = 3,     /* workspace missing or smaller than required */
  SD_ERR_HIP = 4            /* the HIP runtime reported an error at launch */
} sd_status;

typedef enum sd_dtype { SD_F32 = 0, SD_BF16 = 1 } sd_dtype;

typedef enum sd_accept_mode {
  SD_ACCEPT_GREEDY = 0,     /* temperature 0: longest prefix equal to the target argmax */
  SD_ACCEPT_SAMPLED = 1     /* min(1, p/q) acceptance and residual resampling */
} sd_accept_mode;

/* Human-readable name of a status code (static storage, never NULL). */
const char* sd_status_string(int status);

/* Library ABI version, (major << 16) | minor. */
int sd_version(void);

/* ------------------------------------------------------------------------
 * Latent-guided visual-token compression (Sec. 3.2, Eq. 3).
 *
 * The learned query set Cq [C, d] attends over the visual features F_V of
 * each sequence; F_V is both key and value.  With H = num_heads the width d
 * is cut into H contiguous slices of width dh = d / H and, for every
 * sequence b, head h and latent c,
 *
 *   out[b, c, h*dh:(h+1)*dh] =
 *     sum_n softmax_n(scale * Cq[c, hs] . feats[b, n, hs]) * feats[b, n, hs]
 *
 * (H = 1 and scale = 1 is Eq. 3 literally.)  The query set is shared by all
 * sequences.
 *
 *   latents  [C, d]     dtype   learned queries
 *   feats    [B, N, d]  dtype   visual features F_V, token-major
 *   out      [B, C, d]  float32 compressed features
 *   scale               score multiplier (finite)
 * Requirements: B, N, C >= 1; d % num_heads == 0; dh in {64, 128, 256};
 * N <= 2^24; C <= 2^20; d <= 2^22.
 * SD_F32, and SD_BF16 with dh = 256, run scores, softmax and aggregation in
 * float64 on the vector units (bf16 values widened exactly).
 * For SD_BF16 with dh in {64, 128} both products run on float16 matrix
 * cores with the inputs
 * converted exactly (fp16 holds zero and every bf16 magnitude in 2^-17 ..
 * 65280 exactly).  Larger magnitudes convert to inf; each group of 32
 * latents of one head whose results then come out non-finite, or all below
 * 2^-12 in magnitude (inputs far below fp16's normal range), is recomputed
 * in float64 from the bf16 values, so every finite input is handled (such
 * calls are slower).
 * When the tokens are split across work-groups, the workspace holds one
 * partial result per split; for SD_BF16 the split count follows the
 * compute units of the current device, so query
 * sd_latent_compress_workspace_size with the device the call will run on
 * current (a smaller workspace is rejected with SD_ERR_WORKSPACE).
 * ---------------------------------------------------------------------- */
size_t sd_latent_compress_workspace_size(int B, int N, int C, int d,
                                         int num_heads, int dtype);

int sd_latent_compress(const void* latents, const void* feats, float* out,
                       int B, int N, int C, int d, int num_heads, float scale,
                       int dtype, void* workspace, size_t workspace_bytes,
                       void* stream);

/* ------------------------------------------------------------------------
 * Latent compression of the int8 draft (Eq. 3 with the draft quantised to
 * int8, Appendix A; the paper names no scheme).  The learned queries and the
 * visual features are int8 rows, each row with its own power-of-two scale:
 * latent c stands for latents_q[c, :] * 2^latent_exp[c], token n of sequence
 * b for feats_q[b, n, :] * 2^feat_exp[b, n].  The result is
 * sd_latent_compress on those values (same heads, scale and output).
 *
 *   latents_q  [C, d]     int8     latent_exp [C]     int8
 *   feats_q    [B, N, d]  int8     feat_exp   [B, N]  int8
 *   out        [B, C, d]  float32
 *   workspace  sd_latent_compress_q8_workspace_size(...) bytes (token-split
 *              partials; depends on the current device like the bf16 path's)
 * Every q * 2^e with |q| <= 127 and e in [-14, 9] is a normal fp16 (or
 * zero), so the kernel forms the values exactly and runs both products on
 * fp16 matrix cores; exponents outside [-14, 9] are clamped to it (a
 * precondition).  Half the feature bytes of the bf16 path.
 * Requirements: those of sd_latent_compress for SD_BF16 with dh = 128;
 * latents_q, feats_q and out 16-byte aligned.  Errors as there.
 * ---------------------------------------------------------------------- */
size_t sd_latent_compress_q8_workspace_size(int B, int N, int C, int d, int num_heads);

int sd_latent_compress_q8(const int8_t* latents_q, const int8_t* latent_exp,
                          const int8_t* feats_q, const int8_t* feat_exp, float* out,
                          int B, int N, int C, int d, int num_heads, float scale,
                          void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Average pooling of the visual tokens, the non-parametric compressor the
 * compression ablation compares against (Sec. 4.3): the N tokens of each
 * sequence form C contiguous groups, group c holding tokens
 * floor(c N / C) .. floor((c + 1) N / C) - 1, and
 *
 *   out[b, c, :] = mean of feats[b, t, :] over the tokens t of group c
 *
 * (summed in float64).  C = 1 is Eq. 3 with zero queries.
 *
 *   feats  [B, N, d]  dtype    visual features, token-major
 *   out    [B, C, d]  float32  pooled features
 * Requirements: 1 <= C <= N; B, C <= 65535; N <= 2^24; d <= 2^20.  No
 * workspace.  Errors: SD_ERR_INVALID_ARG (sizes, NULL or misaligned
 * pointers, dtype), SD_ERR_UNSUPPORTED (limits above).
 * ---------------------------------------------------------------------- */
int sd_avg_pool_compress(const void* feats, float* out, int B, int N, int C, int d, int dtype,
                         void* stream);

/* ------------------------------------------------------------------------
 * Verification attention of the drafted block (Sec. 3.1).
 *
 * The target scores the k drafted tokens in one pass; per layer that is
 * attention of the k block queries over the KV cache, causal inside the
 * block, with grouped-query heads.  kv_len[b] counts every cache entry of
 * sequence b including the k block entries, which are its last k.  For
 * block row j, query head h and g = Hq / Hkv:
 *
 *   visible keys t = 0 .. kv_len[b] - k + j,
 *   s_t = scale * q[b, j, h] . K[b, t, h / g],
 *   out[b, j, h] = sum_t softmax(s)_t V[b, t, h / g],
 *   lse[b, j, h] = log sum_t exp(s_t)            (natural log)
 *
 * A row with no visible key gets out = 0 and lse = -inf.
 *
 *   q           [B, k, Hq, D]    dtype  queries of the block (after RoPE)
 *   k_cache,    contiguous (page_table == NULL): [B, Lmax, Hkv, D] dtype
 *   v_cache     paged: page pools [num_pages, Hkv, 16, D] dtype; token t of
 *               sequence b lives in page page_table[b, t / 16], slot t % 16
 *   kv_len      [B] int32, device; values are clamped to [0, capacity] with
 *               capacity = Lmax (contiguous) or 16 * max_pages (paged)
 *   page_table  [B, max_pages] int32, device, or NULL for contiguous caches;
 *               page ids outside [0, num_pages) are a precondition violation
 *   out         [B, k, Hq, D] float32
 *   lse         [B, k, Hq] float32, or NULL when not wanted
 * Requirements: 1 <= k <= 16; Hq % Hkv == 0; k * (Hq / Hkv) <= 256;
 * D in {64, 128}; Lmax >= 1 (contiguous) or max_pages, num_pages >= 1
 * (paged); scale finite.  bf16: B * Hkv * ceil(capacity / 32) * ceil(k *
 * (Hq / Hkv) / 64) < 2^30; fp32: B * Hkv * (key splits of at least 8
 * keys) < 2^31, which B * Hkv * ceil(capacity / 8) < 2^31 guarantees;
 * else SD_ERR_UNSUPPORTED (the workspace size is then 0).
 * The bf16 workspace holds partial results per work-group, and the
 * work-group count follows the compute units of the current device: query
 * sd_verify_workspace_size with the device the call will run on current
 * (a smaller workspace is rejected with SD_ERR_WORKSPACE, never overrun).
 * ---------------------------------------------------------------------- */
size_t sd_verify_workspace_size(int B, int k, int Hq, int Hkv, int D,
                                int capacity, int dtype);

int sd_verify_attention(const void* q, const void* k_cache, const void* v_cache,
                        const int32_t* kv_len, const int32_t* page_table,
                        int max_pages, int num_pages, int Lmax,
                        float* out, float* lse,
                        int B, int k, int Hq, int Hkv, int D, float scale,
                        int dtype, void* workspace, size_t workspace_bytes,
                        void* stream);

/* ------------------------------------------------------------------------
 * Speculative acceptance (Sec. 3.1, Sec. 3.3; greedy at temperature 0,
 * Sec. 4.2).  Per sequence b, drafted ids x_i = draft[b, i] (i < k):
 *
 * SD_ACCEPT_SAMPLED: accept position i iff u[b,i] * q[b,i,x_i] < p[b,i,x_i]
 *   (exact float64 test, i.e. u < min(1, p/q)); ids outside [0, V) are
 *   rejected.  n = number of leading accepted positions.  The extra token
 *   is drawn with a = floor(u[b,k] * 2^24) by inverse CDF over integer
 *   weights R_v = floor(r_v * 2^40): r = max(0, p[b,n] - q[b,n]) (float32
 *   subtraction) when n < k, r = p[b,k] when n == k; T = floor(a * S / 2^24)
 *   with S = sum R; the token is the smallest j whose inclusive prefix sum
 *   of R exceeds T.  If S == 0, R = floor(p[b,n] * 2^40) is used; if that
 *   is 0 too, the token is argmax p[b,n].  The result is bit-exact and
 *   independent of summation order.
 * SD_ACCEPT_GREEDY: g_i = argmax_v p[b,i,v] (lowest index on ties);
 *   n = longest prefix with x_i == g_i; the extra token is g_n.  q and u
 *   are not read (may be NULL).
 *
 * Temperature is the caller's: p and q are already softmax(logits / tau).
 *
 *   p           [B, k+1, V] float32  target probabilities
 *   q           [B, k, V]   float32  draft probabilities
 *   draft       [B, k]      int32    drafted ids
 *   u           [B, k+1]    float32  uniforms in [0, 1) (multiples of 2^-24)
 *   n_accepted  [B]         int32    out: accepted drafts per sequence
 *   tokens      [B, k+1]    int32    out: draft[0..n-1], the extra token,
 *                                    then -1 padding
 *   workspace   sd_spec_accept_workspace_size(B, k, V, mode) bytes, zeroed
 *               workspace (one arrival counter per sequence, then the
 *               per-chunk partial sums or maxima of the vocabulary pass)
 * Requirements: 1 <= B <= 2^22; 1 <= k <= 16; 1 <= V <= 2^18; p, q in [0, 1]
 * (values outside are clamped when forming the weights).
 * ---------------------------------------------------------------------- */
size_t sd_spec_accept_workspace_size(int B, int k, int V, int mode);

int sd_spec_accept(const float* p, const float* q, const int32_t* draft,
                   const float* u, int32_t* n_accepted, int32_t* tokens,
                   int B, int k, int V, int mode,
                   void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * sd_spec_accept without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same rule, arguments, outputs and
 * bit-exact results as sd_spec_accept; its counters and partials live in a
 * fixed device array of the library (4 MiB on each device it runs on, held
 * until the process ends): arrival counters of up to 1024 sequences, then
 * the chunk partials.  It calls no allocating routine.  On its first call
 * on a device it looks up that array's address and clears the counters (a
 * kernel on `stream`); every call returns them to zero.
 * All calls on one device share the array: calls that overlap in time on
 * one device (different streams or host threads) race and give undefined
 * results; calls ordered on one stream are safe.
 * Requirements: those of sd_spec_accept, plus B <= 1024 and a partial size
 * (per sequence 16 * ceil(V / 1024) bytes sampled, 8 * (k+1) * ceil(V /
 * 1024) greedy) of at most 4 MiB - 4 KiB in total; larger calls return
 * SD_ERR_WORKSPACE without launching anything.
 * ---------------------------------------------------------------------- */
int sd_spec_accept_noalloc(const float* p, const float* q, const int32_t* draft,
                           const float* u, int32_t* n_accepted, int32_t* tokens,
                           int B, int k, int V, int mode, void* stream);

/* ------------------------------------------------------------------------
 * Speculative acceptance from logits (the same rule as sd_spec_accept,
 * Sec. 3.1 and Sec. 3.3, with the temperature softmax of Sec. 4.2 and the
 * uniforms produced on the device).
 *
 * SD_ACCEPT_SAMPLED: p = softmax(target_logits / tau) and q =
 *   softmax(draft_logits / tau) per row, in float32 (p(v) = 2^(z(v) s - M)
 *   / L with s = log2(e) / tau and the row's max M and sum L), and u[b, i] =
 *   the Philox uniform of sd_philox_uniforms(seed, offset); then the rule
 *   of sd_spec_accept exactly as stated there, applied to these float32
 *   values.
 * SD_ACCEPT_GREEDY: g_i = argmax_v target_logits[b, i, v] (lowest index on
 *   ties); temperature, seed, offset and draft_logits are not used
 *   (draft_logits may be NULL).
 *
 *   target_logits [B, k+1, V] dtype (SD_F32 or SD_BF16)
 *   draft_logits  [B, k, V]   dtype (sampled mode)
 *   draft         [B, k]      int32 drafted ids
 *   seed, offset              key and stream offset of the uniforms
 *   temperature               tau > 0, finite (sampled mode)
 *   n_accepted, tokens        as for sd_spec_accept
 *   workspace   sd_spec_accept_logits_workspace_size(B, k, V, mode) bytes,
 *               zeroed workspace (row statistics of the logits, then the
 *               rule's counters and partials)
 * Requirements: as for sd_spec_accept, with B <= 2^19; logits finite (others give an
 * unspecified result, never an out-of-bounds access).
 * ---------------------------------------------------------------------- */
size_t sd_spec_accept_logits_workspace_size(int B, int k, int V, int mode);

int sd_spec_accept_logits(const void* target_logits, const void* draft_logits,
                          const int32_t* draft, uint64_t seed, uint64_t offset,
                          float temperature, int32_t* n_accepted,
                          int32_t* tokens, int B, int k, int V, int dtype,
                          int mode, void* workspace, size_t workspace_bytes,
                          void* stream);

/* ------------------------------------------------------------------------
 * Counter-based uniforms for the acceptance (Philox-4x64-10 of Salmon,
 * Moraes, Dror and Shaw, SC'11).  u[b, i] for b < B, i < n: the block
 * at counter (i / 4, b, offset, 0) under key (seed, 0), its word i % 4
 * as (word >> 40) * 2^-24, a multiple of 2^-24 in [0, 1).  Any (b, i) is
 * computed alone, so the same values arise wherever they are needed.
 *
 *   u   [B, n] float32, device, out
 * Requirements: B >= 1, 1 <= n <= 2^16, B * n <= 2^31 - 1.
 * ---------------------------------------------------------------------- */
int sd_philox_uniforms(uint64_t seed, uint64_t offset, float* u, int B,
                       int n, void* stream);

/* ------------------------------------------------------------------------
 * LM head with temperature softmax (Sec. 3.1: the head maps a feature to a
 * distribution over the vocabulary; Sec. 3.3 and Algorithm 1: the draft's K
 * hidden states go through the target's frozen head to give P'; Sec. 4.2:
 * temperature tau).  For every row r and vocabulary entry v,
 *
 *   probs[r, v] = exp(z[r, v] / tau) / sum_u exp(z[r, u] / tau),
 *   z[r, v]     = hidden[r] . weight[v]
 *
 * (a bias-free linear head; normalisation before it belongs to the model).
 * Greedy decoding (tau = 0) uses the argmax of the logits, which any
 * positive tau preserves: pass tau = 1 and take the argmax of probs.
 *
 *   hidden  [R, d] dtype    hidden states (target rows, or the draft's rows)
 *   weight  [V, d] dtype    head weight (nn.Linear layout: one row per entry)
 *   probs   [R, V] float32  out
 *   workspace  sd_lm_head_workspace_size(R, d, V, dtype) bytes (the rows'
 *              partial softmax statistics, one (max, sum) pair per
 *              16-entry block or per work-group of the logits pass)
 * Requirements: R, d, V >= 1; temperature > 0 and finite; V <= 2^24;
 * SD_BF16: R <= 256, d % 64 == 0, 16-byte aligned hidden and weight (the
 * weight is streamed from HBM once); SD_F32 (float64 dot products, for
 * accuracy checks rather than speed): R <= 4096, any d.
 * ---------------------------------------------------------------------- */
size_t sd_lm_head_workspace_size(int R, int d, int V, int dtype);

int sd_lm_head_probs(const void* hidden, const void* weight, float* probs,
                     int R, int d, int V, float temperature, int dtype,
                     void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Categorical sampling of the drafts (Algorithm 1: T'_i ~ Categorical(P'_i)).
 * Per row r, with the exact fixed-point inverse CDF of sd_spec_accept's
 * final draw: weights R_v = floor(probs[r, v] * 2^40) (values clamped to
 * [0, 1]), a = floor(u[r] * 2^24), T = floor(a * S / 2^24) with S = sum R;
 * tokens[r] = the smallest v whose inclusive prefix sum of R exceeds T.
 * All-zero weights give argmax probs[r] (lowest index).  Bit-exact and
 * independent of summation order.
 *
 *   probs   [R, V] float32  distributions
 *   u       [R]    float32  uniforms in [0, 1) (multiples of 2^-24)
 *   tokens  [R]    int32    out
 *   workspace  sd_sample_workspace_size(R, V) bytes, zeroed workspace
 * Requirements: R >= 1; 1 <= V <= 2^18.
 * ---------------------------------------------------------------------- */
size_t sd_sample_workspace_size(int R, int V);

int sd_sample_tokens(const float* probs, const float* u, int32_t* tokens, int R, int V,
                     void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Skinny projection y = x W^T (+ bias) (+ residual) for few input rows, the
 * shape of every projection of a drafting step (Sec. 3.1: the fully
 * connected fusion of feature and embedding; Sec. 3.3: the draft layer).
 *
 *   x         [R, K] bf16     input rows (row-major)
 *   w         [N, K] bf16     weight (row n holds output column n)
 *   bias      [N]    float32  or NULL
 *   residual  [R, N] float32  or NULL (may alias y)
 *   y         [R, N] float32  out
 *   workspace sd_linear_workspace_size(R, K, N) bytes (fp32 partial sums of
 *             the reduction splits; the split count follows the compute units
 *             of the current device, so size it on the device of the call)
 * Accumulation in fp32 on bf16 matrix cores; the weight is read once per
 * pass of up to 128 input rows.
 * Requirements: 1 <= R <= 65535; K a multiple of 256 (at most 2^20); N >= 1;
 * R * N <= 2^31; x and w 16-byte aligned.  Errors: SD_ERR_INVALID_ARG (NULL or
 * misaligned pointers), SD_ERR_UNSUPPORTED (shape outside the
 * requirements), SD_ERR_WORKSPACE (missing or short workspace).
 * ---------------------------------------------------------------------- */
size_t sd_linear_workspace_size(int R, int K, int N);

int sd_linear(const void* x, const void* w, const float* bias, const float* residual, float* y,
              int R, int K, int N, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * One step of the draft's semi-autoregressive layer over its cached context
 * (Sec. 3.1 and Algorithm 1: textual input FC(concat(F_T, E)); Sec. 3.3:
 * one pass of the layer gives the states of the K placeholder positions;
 * Sec. 4.3: one layer, 32 heads).  For the r new rows of each sequence b
 * (the last K of them placeholders), at positions pos[b] .. pos[b] + r - 1:
 *
 *   x0  = u W_fc^T + b_fc
 *   q, k, v = RoPE(RMSNorm(x0; ln1) Wqkv^T)     (k, v written to the cache)
 *   x1  = x0 + Attn(q; cache positions 0 .. pos[b] + r - 1) Wo^T
 *   out = x1 + (silu(h Wg^T) * (h Wu^T)) Wdown^T,  h = RMSNorm(x1; ln2)
 *
 * RMSNorm(x; w) = x / sqrt(mean(x^2) + eps) * w.  RoPE turns the pairs
 * (i, i + D/2) of every head by the angle p * theta^(-2i/D).  Attention:
 * scale 1/sqrt(D), query head h reads KV head h / (Hq / Hkv), row j of a
 * sequence sees cache positions 0 .. pos[b] + j (causal inside the new
 * rows); D = d / Hq.
 *
 *   u        [B r, 2d] bf16     concat(F_T, E) of the new rows (a
 *                                placeholder row carries its own input)
 *   fc_w     [d, 2d] bf16, fc_b [d] float32
 *   ln1, ln2 [d] float32        RMSNorm weights
 *   wqkv     [(Hq + 2 Hkv) D, d] bf16   query heads, key heads, value heads
 *   wo       [d, Hq D] bf16
 *   wgu      [2I, d] bf16       gate rows, then up rows
 *   wdown    [d, I] bf16
 *   k_cache, v_cache [B, Lmax, Hkv, D] bf16  the draft cache (post-RoPE
 *            keys); positions pos[b] .. pos[b] + r - 1 are overwritten
 *   pos      [B] int32 (device)  first new position of each sequence; rows
 *            whose position falls outside 0 .. Lmax - 1 are not written to
 *            the cache and attend over what the cache holds (unspecified
 *            output, no out-of-range access)
 *   out      [B r, d] float32   the layer's outputs (placeholder rows: the
 *            draft states for the LM head)
 *   workspace  sd_semi_ar_layer_workspace_size(...) bytes, 256-byte aligned
 *            (device-dependent like sd_linear's)
 * Requirements: d = Hq * D with D in {64, 128}; Hq % Hkv == 0; 1 <= r <= 16;
 * r * (Hq / Hkv) <= 256; d and I multiples of 256; Lmax >= r; B * r <=
 * 65535; eps >= 0; theta > 0.  Errors as for sd_linear.
 * ---------------------------------------------------------------------- */
size_t sd_semi_ar_layer_workspace_size(int B, int r, int d, int num_q_heads, int num_kv_heads,
                                       int I, int Lmax);

int sd_semi_ar_layer(const void* u, const void* fc_w, const float* fc_b, const float* ln1,
                     const void* wqkv, const void* wo, const float* ln2, const void* wgu,
                     const void* wdown, void* k_cache, void* v_cache, const int32_t* pos,
                     float* out, int B, int r, int d, int num_q_heads, int num_kv_heads, int I,
                     int Lmax, float eps, float theta, void* workspace, size_t workspace_bytes,
                     void* stream);

/* ------------------------------------------------------------------------
 * The int8 draft (the quantised drafts of Appendix A; weight-only): every
 * projection row n holds int8 values wq[n, :] and one fp32 scale, the
 * weight it stands for being scale[n] * wq[n, :].  Activations, norms and
 * the FC bias are as in the bf16 draft; the int8 x bf16 products are exact
 * in the fp32 accumulation and each output is scaled once, so the results
 * match the bf16 path on the dequantised weights to the same tolerance
 * while every weight byte read is halved.
 *
 * sd_linear_q8: y = x (scale * wq)^T (+ bias) (+ residual); wq [N, K] int8,
 *   scale [N] float32; other arguments, requirements, errors and workspace
 *   (sd_linear_workspace_size) as for sd_linear.
 * sd_semi_ar_layer_q8: sd_semi_ar_layer with int8 fc_w, wqkv, wo, wgu,
 *   wdown and their scales fc_s [d], wqkv_s [(Hq + 2 Hkv) D], wo_s [d],
 *   wgu_s [2I], wdown_s [d]; workspace sd_semi_ar_layer_workspace_size.
 * ---------------------------------------------------------------------- */
int sd_linear_q8(const void* x, const int8_t* wq, const float* scale, const float* bias,
                 const float* residual, float* y, int R, int K, int N, void* workspace,
                 size_t workspace_bytes, void* stream);

int sd_semi_ar_layer_q8(const void* u, const int8_t* fc_w, const float* fc_s, const float* fc_b,
                        const float* ln1, const int8_t* wqkv, const float* wqkv_s,
                        const int8_t* wo, const float* wo_s, const float* ln2,
                        const int8_t* wgu, const float* wgu_s, const int8_t* wdown,
                        const float* wdown_s, void* k_cache, void* v_cache, const int32_t* pos,
                        float* out, int B, int r, int d, int num_q_heads, int num_kv_heads, int I,
                        int Lmax, float eps, float theta, void* workspace, size_t workspace_bytes,
                        void* stream);

/* ------------------------------------------------------------------------
 * K drafts in K / k' passes of the semi-autoregressive layer, k' per pass
 * (the group size k' of the paper's ablation, Appendix E: the draft emits k'
 * tokens per forward pass and feeds them back for the next k').
 *
 * Pass 0 is sd_semi_ar_layer on u0 [B, r0, 2d] at positions pos[b] ..
 * pos[b] + r0 - 1, the last k' rows being placeholders.  After each pass the
 * placeholder rows' states, rounded to bf16, go through the frozen LM head
 * (softmax(h lm_w^T / temperature)) and one token per row is drawn with
 * sd_sample_tokens' exact inverse CDF and the uniform u[b][t k' + j] (pass t,
 * row j).  Pass t + 1 runs on 2k' rows: the k' drafted tokens, with input
 * concat(bf16(state of the placeholder that drafted it), emb[token]), at
 * that placeholder's position, then k' placeholder rows with input ph.
 *
 *   u0       [B, r0, 2d] bf16; weights as for sd_semi_ar_layer
 *   lm_w     [V, d] bf16     frozen LM head
 *   emb      [V, d] bf16     token embeddings
 *   ph       [2d] bf16       input of a placeholder row
 *   k_cache, v_cache, pos    as for sd_semi_ar_layer (the caches gain every
 *            pass's rows; pos is not modified)
 *   u        [B, K] float32  uniforms in [0, 1) (multiples of 2^-24)
 *   tokens   [B, K] int32    out: the drafts
 *   q        [B, K, V] float32  out: their distributions (the q of the
 *            acceptance rule)
 *   workspace  sd_semi_ar_draft_workspace_size(...) bytes, 256-byte aligned
 *            (device-dependent), zeroed workspace (the draws' counters)
 * Requirements: those of sd_semi_ar_layer for r0 and, when K > k', for
 * 2k' rows; 1 <= k' <= min(r0, 8); K % k' == 0; B * k' <= 256;
 * 1 <= V <= 2^18; temperature > 0.  Errors as for sd_linear.
 * ---------------------------------------------------------------------- */
size_t sd_semi_ar_draft_workspace_size(int B, int r0, int d, int num_q_heads, int num_kv_heads,
                                       int I, int Lmax, int V, int K, int k_prime);

int sd_semi_ar_draft(const void* u0, const void* fc_w, const float* fc_b, const float* ln1,
                     const void* wqkv, const void* wo, const float* ln2, const void* wgu,
                     const void* wdown, const void* lm_w, const void* emb, const void* ph,
                     void* k_cache, void* v_cache, const int32_t* pos, const float* u,
                     int32_t* tokens, float* q, int B, int r0, int d, int num_q_heads,
                     int num_kv_heads, int I, int Lmax, int V, int K, int k_prime, float eps,
                     float theta, float temperature, void* workspace, size_t workspace_bytes,
                     void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPECFLASH_H */
