/*
 * hspec.h - C ABI of the MI355X (gfx950) block-drafting step of H-Spec
 * ("Parallel Speculative Decoding Without a Drafter-Side KV Cache").
 *
 * One drafting step of the hybrid drafter has two layers:
 *   (a) a Mamba-2 mixer run over the k-token draft block with a chunked parallel scan, its
 *       per-head state initialised from a projection of the target model's last-position
 *       hidden state (Sec. 3.3.1, the cross-layer fusion equation and "Parallel-drafting
 *       compatibility");
 *   (b) an attention layer whose k block queries attend, in place, over one target layer's
 *       paged GQA K/V cache plus the block's own K/V, with RoPE positions continuing the
 *       prefix (Sec. 3.3.2: "KV dimension", "Attention mask", "Positional alignment").
 *
 * Conventions shared by every entry point
 *   - Memory: every tensor pointer is device memory owned by the caller; the library never
 *     allocates, frees, or keeps a pointer after returning.  Tensors are dense row-major.
 *   - Storage dtype (hspec_dtype): block/hidden inputs, weight matrices, conv weights and the
 *     K/V cache use the configuration's dtype (bf16 or fp32).  Per-head and norm parameters
 *     (dt_bias, A_log, D, norm gains) are always fp32.  Every output is fp32.
 *   - Asynchrony: work is enqueued on `stream` (a hipStream_t, NULL = default stream) and the
 *     call returns without synchronising.  Calls on different streams with disjoint
 *     workspaces may run concurrently.
 *   - Workspace: caller-provided device scratch of at least the size returned by the matching
 *     *_workspace() query; 256-byte aligned.  Its first 256 bytes are reserved: the first
 *     int32 is a device status word that the call resets and the kernels OR bits into
 *     (HSPEC_DEV_*), read it after the stream completes with hspec_read_status(); the rest
 *     holds the work-queue counters of the attention sweep.
 *   - Errors: host-checkable problems (NULL pointers, non-positive or inconsistent sizes,
 *     unsupported dimensions, a too-small workspace) return an error before anything is
 *     enqueued.  A failed launch returns HSPEC_ERR_LAUNCH.  hspec_last_error() gives a
 *     thread-local message for the last failing call.
 *   - Device-resident page tables and context lengths are validated on the device: a page id
 *     outside [0, num_pages) is read as zeros and sets HSPEC_DEV_BAD_PAGE; a context length
 *     below 0 or above min(max_ctx_len, max_pages * page_size) is clamped and sets
 *     HSPEC_DEV_BAD_CTX_LEN.  No out-of-bounds access happens in either case.
 */
#ifndef HSPEC_H
#define HSPEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HSPEC_OK = 0,
  HSPEC_ERR_NULL = 1,        /* a required pointer is NULL */
  HSPEC_ERR_SHAPE = 2,       /* a size is non-positive or sizes disagree */
  HSPEC_ERR_DTYPE = 3,       /* unknown storage dtype, or dtypes of two configs differ */
  HSPEC_ERR_UNSUPPORTED = 4, /* a dimension this build has no kernel for */
  HSPEC_ERR_WORKSPACE = 5,   /* workspace NULL, misaligned or smaller than required */
  HSPEC_ERR_LAUNCH = 6       /* the HIP runtime rejected a launch */
} hspec_status;

typedef enum { HSPEC_BF16 = 0, HSPEC_F32 = 1 } hspec_dtype;

/* hspec_attn_cfg.flags */
enum {
  HSPEC_BLOCK_CAUSAL = 1u << 0, /* block keys s visible to block query j only if s <= j
                                   (default: the whole block is visible to every query) */
  HSPEC_ATTN_PRECISE_IO = 1u << 1 /* the layer's normalised input enters W_q/W_k/W_v, and its
                                     attention output enters W_o, as bf16 hi/lo planes (two
                                     products each) instead of one bf16 plane: for stacks of
                                     attention layers (hspec_drafter_forward sets it) */
};

/* Device status bits (first int32 of the workspace). */
enum { HSPEC_DEV_BAD_PAGE = 1, HSPEC_DEV_BAD_CTX_LEN = 2, HSPEC_DEV_BAD_TOKEN = 4, HSPEC_DEV_NONFINITE = 8 };

/*
 * Mamba layer configuration (Sec. 3.3.1; sizes of App. B.1 "Mamba").
 *   B requests, k draft positions, d_model hidden size, d_h = |M| * target hidden size
 *   (the concatenated last-position hidden states), r fusion rank, H heads of P channels
 *   (P must be 64), N = d_state (16, 32, 64 or 128), G groups of B/C (H % G == 0),
 *   chunk = SSD chunk length (1..16), conv_w = causal conv width (1..8), eps of every RMSNorm.
 *   d_inner = H*P, d_S = H*P*N.  d_h, r, d_model must be multiples of 8.
 *   flags: HSPEC_W_DS_PACKED when hspec_mamba_w.W_dS points at the packed layout written by
 *   hspec_pack_w_ds (bf16 storage, r a multiple of 64, d_h a multiple of 32);
 *   HSPEC_MAMBA_PRECISE_IO (below).
 */
typedef struct {
  int B, k, d_model, d_h, r, H, P, N, G, chunk, conv_w;
  unsigned flags;
  hspec_dtype dtype;
  float eps;
} hspec_mamba_cfg;

/* hspec_mamba_cfg.flags */
enum {
  HSPEC_W_DS_PACKED = 1u << 0,
  HSPEC_MAMBA_PRECISE_IO = 1u << 1 /* with bf16 storage, the Mamba layer's normalised input enters
                                      W_in, and its gated-norm output enters W_out, as bf16 hi/lo
                                      planes (two products each) instead of one bf16 plane, as fp32
                                      storage always does, and F = W_r h_last enters a packed W_dS
                                      as fp16 hi/lo planes instead of one fp16 plane: for stacks of
                                      layers (hspec_drafter_forward sets it) */
};

/*
 * Mamba weights.  Matrices are [out, in] row-major in the storage dtype:
 *   W_r [r, d_h] (Proj_r), W_dS [d_S, r] (Proj_dS; row (h*P + p)*N + n is state element
 *   [h, p, n]), W_in [2*d_inner + 2*G*N + H, d_model] with output order (z, x, B, C, dt),
 *   conv_w [d_inner + 2*G*N, conv_w] and conv_b [d_inner + 2*G*N] (storage dtype),
 *   W_out [d_model, d_inner].  fp32: dt_bias [H], A_log [H] (A = -exp(A_log)), D [H],
 *   gnorm_w [d_inner] (gain of the gated RMSNorm, normalised within each of the G groups).
 */
typedef struct {
  const void *W_r, *W_dS, *W_in, *conv_w, *conv_b;
  const float *dt_bias, *A_log, *D, *gnorm_w;
  const void *W_out;
} hspec_mamba_w;

/*
 * Attention layer configuration (Sec. 3.3.2; App. B.2 "Unified attention implementation").
 *   Hq query heads, Hkv KV heads (Hq % Hkv == 0, query head q reads KV head q / (Hq/Hkv)),
 *   D head dim (64 or 128), k * Hq/Hkv <= 128, B <= 32767, page_size a power of two >= 16.
 *   The target cache is two pools
 *   [num_pages, page_size, Hkv, D] (K stored after RoPE; Hkv_cache heads per slot, below), addressed through page_table
 *   [B, max_pages] int32 and ctx_lens [B] int32: cache position i of request b lives in
 *   slot page_table[b, i / page_size] * page_size + i % page_size.  Block position j sits at
 *   RoPE position ctx_lens[b] + j.  window > 0 hides cache position p from the query at
 *   position pos when pos - p >= window (sliding window; requires k <= window).
 *   The sweep reads, for each request, the cache positions some block query can see: all
 *   of [0, ctx_len), or [ctx_len - window + 1, ctx_len) under a window; the swept length is
 *   at most max_ctx_len, or window - 1 with a window.
 *   split_tokens: cache positions per split of the KV sweep (multiple of 64, at most 8192,
 *   and at least the swept length / 256 so that no request has more than 256 splits),
 *   0 = automatic.
 *   A setting outside these limits returns HSPEC_ERR_UNSUPPORTED.
 *   scale: softmax scale, 0 = 1/sqrt(D).  rope_theta: RoPE base (rotate-half pairing).
 *   Partial target-KV-head reuse (Sec. 3.3.2 "KV dimension": reusing only a subset of the
 *   target's KV heads, left to future work in Sec. 5): Hkv_cache is the number of KV heads per
 *   slot of the target cache (0 = Hkv), and kv_heads (host array of Hkv entries, or NULL for
 *   0 .. Hkv-1) names the cache head each of the drafter's Hkv KV heads reads; the drafter's
 *   W_k, W_v and block K/V have Hkv heads, its queries Hq.  Hkv <= Hkv_cache <= 16 and every
 *   entry in [0, Hkv_cache), else HSPEC_ERR_SHAPE / HSPEC_ERR_UNSUPPORTED.  The cache pools are
 *   then [num_pages, page_size, Hkv_cache, D] and only the named heads are read.
 */
typedef struct {
  int B, k, d_model, Hq, Hkv, D, page_size, max_pages, num_pages, window, split_tokens;
  unsigned flags;
  hspec_dtype dtype;
  float eps, scale;
  double rope_theta;
  int Hkv_cache;
  const int32_t* kv_heads;
} hspec_attn_cfg;

/*
 * Attention weights: W_q [Hq*D, d_model], W_k and W_v [Hkv*D, d_model], W_o [d_model, Hq*D]
 * (storage dtype); q_norm_w, k_norm_w [D] fp32 gains of the per-head RMSNorm of q and k.
 */
typedef struct {
  const void *W_q, *W_k, *W_v, *W_o;
  const float *q_norm_w, *k_norm_w;
} hspec_attn_w;

/* ------------------------------------------------------------------ layer-level calls */

/*
 * Mamba layer from the injected state (Sec. 3.3.1).
 *   S0 = reshape(W_dS (W_r h_last), [H, P, N]) per request;
 *   [z | xBC | dt_raw] = u W_in^T;  x, B, C = SiLU(causal_conv(xBC)) (zero left state);
 *   dt = softplus(dt_raw + dt_bias);  y = selective scan of (x, dt, A, B, C, D) from S0;
 *   out = W_out (RMSNorm_G(y * SiLU(z)) * gnorm_w).   No residual, no pre-norm.
 * h_last [B, d_h], block_hidden u [B, k, d_model] (storage dtype); out [B, k, d_model] fp32;
 * S_final [B, H, P, N] fp32 or NULL (the state after the last draft position).
 */
hspec_status hspec_mamba_block_scan(const hspec_mamba_cfg* cfg, const hspec_mamba_w* w,
                                    const void* h_last, const void* block_hidden, float* out,
                                    float* S_final, void* workspace, size_t ws_bytes, void* stream);
size_t hspec_mamba_block_scan_workspace(const hspec_mamba_cfg* cfg);

/*
 * Attention layer over the target's paged K/V, in place (Sec. 3.3.2).
 *   q = RMSNorm_D(x W_q^T) q_norm_w, k_b = RMSNorm_D(x W_k^T) k_norm_w, v_b = x W_v^T;
 *   q, k_b rotated at positions ctx_len + j;  o = softmax over (visible cache keys, block keys);
 *   out = o W_o^T.   No residual, no pre-norm.
 * x [B, k, d_model] (storage dtype); k_cache, v_cache [num_pages, page_size, Hkv, D];
 * page_table [B, max_pages], ctx_lens [B] (device int32); max_ctx_len: host upper bound of
 * ctx_lens (sizes the launch; larger lengths are clamped and flagged); out [B, k, d_model] fp32.
 */
hspec_status hspec_target_kv_block_attn(const hspec_attn_cfg* cfg, const hspec_attn_w* w, const void* x,
                                        const void* k_cache, const void* v_cache,
                                        const int32_t* page_table, const int32_t* ctx_lens,
                                        int max_ctx_len, float* out, void* workspace, size_t ws_bytes,
                                        void* stream);
size_t hspec_target_kv_block_attn_workspace(const hspec_attn_cfg* cfg, int max_ctx_len);

/*
 * One drafting step (Sec. 3.3 architecture: Mamba then attention):
 *   x1 = e + Mamba(RMSNorm(e) norm1_w; S0(h_last));   out = x1 + Attn(RMSNorm(x1) norm2_w).
 * The two configs must agree on B, k, d_model and dtype.  block_emb e [B, k, d_model]
 * (storage dtype); norm1_w, norm2_w [d_model] fp32; other arguments as in the layer calls.
 */
hspec_status hspec_draft_step(const hspec_mamba_cfg* mcfg, const hspec_mamba_w* mw, const float* norm1_w,
                              const hspec_attn_cfg* acfg, const hspec_attn_w* aw, const float* norm2_w,
                              const void* h_last, const void* block_emb, const void* k_cache,
                              const void* v_cache, const int32_t* page_table, const int32_t* ctx_lens,
                              int max_ctx_len, float* out, void* workspace, size_t ws_bytes, void* stream);
size_t hspec_draft_step_workspace(const hspec_mamba_cfg* mcfg, const hspec_attn_cfg* acfg, int max_ctx_len);

/*
 * Whole drafter forward over the block (Sec. 3.3; App. B.1 "Number of drafter layers", "MLP",
 * "Target-layer mapping"):
 *   S0 = reshape(W_dS (W_r h_last)), once, given to every layer's Mamba (h_last [B, d_h]: the
 *   |M| fused target layers' last hidden states, d_h = |M| * target hidden size);
 *   x = block_emb;  for each layer:
 *     x += Mamba(RMSNorm(x) norm1_w; S0)
 *     x += Attn(RMSNorm(x) norm2_w) over the layer's own target cache   (layers with attention)
 *     x += W_down (SiLU(W_gate RMSNorm(x) norm3_w) * (W_up RMSNorm(x) norm3_w))
 *   out [B, k, d_model] fp32 = x.
 * mcfg.d_h and mcfg.r size W_r [r, d_h] and W_dS [d_S, r] (packed with HSPEC_W_DS_PACKED); the
 * layers' mamba weights (their W_r and W_dS are not read) and attention weights are as in the
 * layer calls; all attention layers share acfg, page_table and ctx_lens and read their own
 * k_cache/v_cache.  ff: MLP hidden size (multiple of 8); W_gate, W_up [ff, d_model] and W_down
 * [d_model, ff] in the storage dtype.  layers: host array of n_layers (>= 1) entries.
 */
typedef struct {
  const hspec_mamba_w* mamba; /* W_in .. W_out of this layer; NULL: no Mamba (a block-diffusion
                                 layer; with no Mamba in any layer, W_r and W_dS are not read) */
  const float* norm1_w;       /* pre-Mamba RMSNorm gain [d_model] */
  const hspec_attn_w* attn;   /* NULL: the layer has no attention */
  const float* norm2_w;       /* pre-attention gain (layers with attention) */
  const void *k_cache, *v_cache; /* the target layer this attention reads */
  const float* norm3_w;       /* pre-MLP gain */
  const void *W_gate, *W_up, *W_down;
} hspec_layer_w;

hspec_status hspec_drafter_forward(const hspec_mamba_cfg* mcfg, const hspec_attn_cfg* acfg, int ff, int n_layers,
                                   const void* W_r, const void* W_dS, const hspec_layer_w* layers,
                                   const void* h_last, const void* block_emb, const int32_t* page_table,
                                   const int32_t* ctx_lens, int max_ctx_len, float* out, void* workspace,
                                   size_t ws_bytes, void* stream);
size_t hspec_drafter_forward_workspace(const hspec_mamba_cfg* mcfg, const hspec_attn_cfg* acfg, int ff,
                                       int max_ctx_len);

/*
 * Drafter-side KV injection, the per-step cost of block-diffusion drafters that H-Spec removes
 * (Sec. 2, "KV injection in block drafting"; Fig. 3), for comparison: the n = cfg->k new
 * positions of every request (h_new [B, n, d_h], the |M| target layers' hidden states,
 * storage dtype) are fused, f = h_new W_fc^T (W_fc [d_model, d_h]), and for each drafter layer
 * l projected into k = RoPE(RMSNorm_D(f W_k[l]^T) k_norm_w[l]) and v = f W_v[l]^T
 * (W_k[l], W_v[l] [Hkv*D, d_model]), which are written at slot(ctx_lens[b] + i) of that
 * layer's paged cache k_cache[l], v_cache[l] [num_pages, page_size, Hkv, D] (storage dtype,
 * updated in place).  W_k, W_v, k_norm_w, k_cache, v_cache are host arrays of n_layers device
 * pointers.  The page table must map positions up to ctx_len + n - 1; unmapped positions set
 * HSPEC_DEV_BAD_CTX_LEN and page ids outside the pool HSPEC_DEV_BAD_PAGE, and are skipped.
 * Uses cfg B, k, d_model, Hkv, D, page_size, max_pages, num_pages, dtype, eps, rope_theta.
 */
hspec_status hspec_kv_inject(const hspec_attn_cfg* cfg, int d_h, int n_layers, const void* h_new, const void* W_fc,
                             const void* const* W_k, const void* const* W_v, const float* const* k_norm_w,
                             void* const* k_cache, void* const* v_cache, const int32_t* page_table,
                             const int32_t* ctx_lens, void* workspace, size_t ws_bytes, void* stream);
size_t hspec_kv_inject_workspace(const hspec_attn_cfg* cfg, int d_h);

/*
 * Draft head (Sec. 3.3.3 "Causal correction"; App. B.1 "Markov rank"; App. B.2 "Pruned drafter
 * vocabulary"): from the block's last hidden states to k draft tokens per request.
 *   logits_j = RMSNorm(hidden_j) norm_f_w W_lm^T                 (V pruned-vocabulary columns)
 *   l'_j[v]  = logits_j[v] + sum_r U_M[v, r] E_M[t_{j-1}, r]     (first-order Markov term, rank R)
 *   t_j      = argmax_v l'_j[v]                                   (gumbel == NULL: greedy)
 *            = argmax_v (l'_j[v] / temperature + gumbel[b, j, v])  (Gumbel-max sampling)
 * with t_{-1} = prev_tok[b], the request's last committed token; a tie goes to the lowest index.
 *   hidden [B, k, d_model] fp32 (e.g. the drafting step's output); norm_f_w [d_model] fp32;
 *   W_lm [V, d_model], E_M [V, R], U_M [V, R] bf16 (V = vocab, R = rank);
 *   prev_tok [B] int32 in [0, V); gumbel [B, k, V] fp32 or NULL (the caller draws the noise);
 *   forced [B, k] int32 or NULL: when given, the Markov term of position j uses forced[b, j-1]
 *   as t_{j-1} (teacher forcing, to score a given continuation) and tokens still receive each
 *   position's argmax; tokens [B, k] int32 out; logits [B, k, V] fp32 out (the corrected l') or
 *   NULL.  The normalised hidden state enters the LM head as one bf16 plane.
 * d_model % 8 == 0 and R % 32 == 0, else HSPEC_ERR_UNSUPPORTED; temperature > 0 when gumbel is
 * given, else HSPEC_ERR_SHAPE.  Token ids outside [0, V) in prev_tok or forced are read as 0 and
 * set HSPEC_DEV_BAD_TOKEN; a NaN score counts as -inf and sets HSPEC_DEV_NONFINITE.
 */
typedef struct {
  int B, k, d_model, vocab, rank;
  float eps, temperature;
} hspec_head_cfg;

typedef struct {
  const float* norm_f_w;
  const void *W_lm, *E_M, *U_M;
} hspec_head_w;

hspec_status hspec_draft_head(const hspec_head_cfg* cfg, const hspec_head_w* w, const float* hidden,
                              const int32_t* prev_tok, const float* gumbel, const int32_t* forced,
                              int32_t* tokens, float* logits, void* workspace, size_t ws_bytes, void* stream);
size_t hspec_draft_head_workspace(const hspec_head_cfg* cfg);

/* ------------------------------------------------------------- weight preparation */

/*
 * Packed layout of W_dS for the state projection (Sec. 3.3.1, Proj_dS), written once when
 * the weights are loaded, never per step.  The projection streams W_dS from HBM once per
 * step; this layout lets every wave read whole 1 KB blocks that are already MFMA operand
 * fragments, and every workgroup one contiguous run of blocks.  Block (s, t) holds rows
 * 16t..16t+15 and columns 32s..32s+31 of W_dS; the 16-row tiles form groups of 32
 * (g = t / 32, the last group holding gs = min(32, d_S/16 - 32g) tiles), and block (s, t)
 * starts at byte (32 g (r/32) + s gs + t mod 32) * 1024; inside it, the 8 consecutive columns
 * 32s + 8c .. +7 of row 16t + i are the 16 bytes at (i + 16c) * 16.  Every element is the
 * fp16 value of 256 x W_dS (exact for bf16 weights of magnitude 2^-25 .. 255.875; smaller
 * magnitudes round to fp16 subnormals in steps of 2^-32 of W_dS, bf16 subnormals become 0,
 * larger magnitudes become +-inf and inf/NaN stay; the projection divides the 256 back out),
 * so that the projection runs as one fp16 product with F as one fp16 plane (hi/lo fp16
 * planes with HSPEC_MAMBA_PRECISE_IO).
 * W_dS [d_S, r] row-major bf16 in, W_packed (hspec_pack_w_ds_bytes bytes) out, both device
 * memory; d_S % 16 == 0 and r % 64 == 0, else HSPEC_ERR_UNSUPPORTED.  Asynchronous on stream.
 */
size_t hspec_pack_w_ds_bytes(int d_S, int r);
hspec_status hspec_pack_w_ds(int d_S, int r, const void* W_dS, void* W_packed, void* stream);

/* --------------------------------------------------- primitives (same kernels as above) */

/*
 * Fusion + state projection only (Sec. 3.3.1 equation): S0 [B, H, P, N] fp32 =
 * reshape(W_dS (W_r h_last)).  Uses cfg B, d_h, r, H, P, N, dtype.
 */
hspec_status hspec_state_init(const hspec_mamba_cfg* cfg, const hspec_mamba_w* w, const void* h_last,
                              float* S0, void* workspace, size_t ws_bytes, void* stream);
size_t hspec_state_init_workspace(const hspec_mamba_cfg* cfg);

/*
 * Selective scan (Sec. 3.3.1 recurrence), chunked: per head h of group g = h / (H/G),
 *   S_t = exp(dt_t A_h) S_{t-1} + dt_t x_t (outer) B_t,   y_t = S_t C_t + D_h x_t,
 * from S_{-1} = S0.  x [B, T, H, P], Bm, Cm [B, T, G, N], S0 [B, H, P, N] or NULL (zeros) in
 * the storage dtype; dt [B, T, H] (already softplus-ed), A [H], Dskip [H] fp32;
 * y [B, T, H, P] fp32; S_final [B, H, P, N] fp32 or NULL.  P must be 64, 1 <= chunk <= 16.
 */
hspec_status hspec_ssd_scan(int B, int T, int H, int P, int N, int G, int chunk, hspec_dtype dtype,
                            const void* x, const float* dt, const float* A, const void* Bm, const void* Cm,
                            const float* Dskip, const void* S0, float* y, float* S_final,
                            void* workspace, size_t ws_bytes, void* stream);
size_t hspec_ssd_scan_workspace(int B, int T, int H, int P, int N, int G, hspec_dtype dtype);

/*
 * Attention core (the KV sweep and its split reduction) on given post-norm, post-RoPE
 * q [B, k, Hq, D], k_blk, v_blk [B, k, Hkv, D] (storage dtype): o [B, k, Hq, D] fp32.
 * Sec. 3.3.2 ("KV dimension", "Attention mask", "Positional alignment"): block query j of
 * request b attends, with softmax scale 1/sqrt(D), to the target's cached keys of positions
 * [lo_j, ctx_lens[b]) read in place through page_table (lo_j = 0, or ctx_len + j - window + 1
 * under a sliding window, App. B.2), plus the block's own keys (all k of them, or s <= j under
 * HSPEC_BLOCK_CAUSAL); query head hq reads KV head hq / (Hq / Hkv).  The caches and the page
 * table are those of hspec_target_kv_block_attn.  All pointers are caller-owned device memory;
 * host-checkable errors return before any launch; out-of-pool page ids and out-of-range
 * lengths set bits of the workspace status word (hspec_read_status).
 */
hspec_status hspec_paged_attn(const hspec_attn_cfg* cfg, const void* q, const void* k_blk, const void* v_blk,
                              const void* k_cache, const void* v_cache, const int32_t* page_table,
                              const int32_t* ctx_lens, int max_ctx_len, float* o, void* workspace,
                              size_t ws_bytes, void* stream);
size_t hspec_paged_attn_workspace(const hspec_attn_cfg* cfg, int max_ctx_len);

/*
 * hspec_paged_attn for callers that cannot allocate device memory (code under graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same kernels, in the same order,
 * with the same results, but no workspace argument.  The workspace is a fixed array of
 * HSPEC_STATIC_WS_BYTES inside the library's device code object; each GPU the library runs on
 * holds its own copy until the process ends.  A call whose hspec_paged_attn_workspace exceeds
 * that size returns HSPEC_ERR_WORKSPACE before any launch.  All calls on one GPU share its
 * array: calls that overlap on one GPU (different streams, or unordered threads) race and
 * give undefined results.  status: a device int32 that receives the call's device status word
 * (HSPEC_DEV_* bits), or NULL.  The call allocates nothing (no hipMalloc, no hipFree).
 * Other arguments and errors as hspec_paged_attn.
 */
#define HSPEC_STATIC_WS_BYTES (64u << 20)
hspec_status hspec_paged_attn_static(const hspec_attn_cfg* cfg, const void* q, const void* k_blk, const void* v_blk,
                                     const void* k_cache, const void* v_cache, const int32_t* page_table,
                                     const int32_t* ctx_lens, int max_ctx_len, float* o, int32_t* status,
                                     void* stream);

/*
 * hspec_paged_attn in separately launched phases, for timing one kernel at a time: the work
 * list (which also clears the workspace status words), the KV sweep (with any fp32 -> bf16
 * plane conversion of its inputs), and the cross-split reduction.  `phases` is an OR of the
 * flags below; a call with all three is hspec_paged_attn.  The phases of one attention must
 * run in this order, on one stream, with the same arguments and workspace: a sweep or a
 * reduction whose predecessors have not run on this workspace reads an undefined work list
 * or undefined partials, and its behaviour is undefined.  Unknown bits: HSPEC_ERR_UNSUPPORTED.
 */
enum { HSPEC_PHASE_WORKLIST = 1u << 0, HSPEC_PHASE_SWEEP = 1u << 1, HSPEC_PHASE_REDUCE = 1u << 2 };
hspec_status hspec_paged_attn_phase(const hspec_attn_cfg* cfg, const void* q, const void* k_blk, const void* v_blk,
                                    const void* k_cache, const void* v_cache, const int32_t* page_table,
                                    const int32_t* ctx_lens, int max_ctx_len, float* o, void* workspace,
                                    size_t ws_bytes, unsigned phases, void* stream);

/*
 * Physical slot of every logical cache position: slots [B, max_ctx_len] int32, -1 at and past
 * ctx_lens[b] (and for out-of-pool page ids, which also set HSPEC_DEV_BAD_PAGE in *status).
 * slot(b, i) = page_table[b, i / page_size] * page_size + i % page_size: the paged layout
 * through which the target's cache is reused in place (Sec. 3.3.2, "Layer-wise KV mapping" and
 * in-place reuse; Sec. 4.2 serves through vLLM's paged cache).  The KV sweep addresses the
 * cache with the same device functions.  page_table [B, max_pages] and ctx_lens [B] are device
 * int32; page_size must be a power of two >= 16 (else HSPEC_ERR_UNSUPPORTED); status: device
 * int32 or NULL.  Caller-owned device memory; asynchronous on `stream`.
 */
hspec_status hspec_gather_slots(int B, int max_pages, int page_size, int num_pages, const int32_t* page_table,
                                const int32_t* ctx_lens, int max_ctx_len, int32_t* slots, int32_t* status,
                                void* stream);

/*
 * Plain projection C [M, N] fp32 = A [M, K] W [N, K]^T (+ R [M, N] fp32 if R != NULL), A and W
 * in the storage dtype (the GEMM used by every projection above: Proj_r and Proj_dS of the
 * Sec. 3.3.1 fusion equation, and the bias-free linear maps of the Mamba and attention modules
 * of Sec. 3.3.1-3.3.2).  Row-major, caller-owned device memory; K must be a multiple of 8
 * (else HSPEC_ERR_UNSUPPORTED); the workspace comes from hspec_linear_workspace and must be
 * 256-byte aligned (else HSPEC_ERR_WORKSPACE).
 */
hspec_status hspec_linear(hspec_dtype dtype, int M, int N, int K, const void* A, const void* W,
                          const float* R, float* C, void* workspace, size_t ws_bytes, void* stream);
size_t hspec_linear_workspace(hspec_dtype dtype, int M, int N, int K);

/* ------------------------------------------------------------------------- utilities */

/* Copies the device status word of `workspace` to *status after synchronising `stream`. */
hspec_status hspec_read_status(const void* workspace, int32_t* status, void* stream);
const char* hspec_status_string(hspec_status s);
/* Message of the last failing call on this thread ("" if none). */
const char* hspec_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HSPEC_H */
