/*
 * dcl.h — C ABI of the MI355X (gfx950) DC-Leap denoising-iteration library (libdcl.so).
 *
 * One denoising iteration of a masked-diffusion LM under DC-Leap ("Draft-guided
 * Contiguous Leaping", Algorithm 1 in Appendix A of the paper) is
 *   (ii)  Forward(p_theta, x): a bidirectional transformer over every position, then the
 *         per-position softmax over the vocabulary at the masked positions (Section 2.1, Eq. 2),
 *         reduced to the top-1 token, its probability c_i (Eq. threshold_pd) and the runner-up
 *         (the top-1/top-2 gap of Section 2.2)            -> dcl_denoise_step
 *   (iii) the contiguous window length K (Section 3.2, Eq. compute_k),
 *   (iv)  commit x[p, p+K), update drafts (Section 3.3, Eq. draft_update), advance p, and
 *   (i)   re-mask the next window (Eq. remasking)          -> dcl_select_contiguous
 *
 * Conventions for every call:
 *  - Pointers are DEVICE pointers unless a comment says "host".
 *  - Every GPU call is asynchronous on `stream` (0 = the null stream). Argument checks are
 *    synchronous, happen on the host before anything is launched, and never touch device memory.
 *  - The caller owns every buffer (weights, tokens, p, statistics, KV cache, workspace). The
 *    library allocates only the host-side model handle (and, inside dcl_load_weights only, a
 *    temporary device staging buffer that it frees before returning). dcl_denoise_step and
 *    dcl_select_contiguous never allocate.
 *  - bfloat16 tensors are passed as raw 16-bit patterns (round-to-nearest-even bfloat16).
 *  - Token ids are int32. Positions inside `tokens` are half-open ranges [a, b).
 *  - A failed check returns a non-zero dcl_status and leaves a message for dcl_last_error();
 *    no C++ exception crosses this interface. A device-side fault surfaces at the caller's next
 *    synchronisation of `stream`.
 *  - One model handle may be used from one stream at a time; concurrent steps need their own
 *    workspaces.
 */
#ifndef DCL_H_
#define DCL_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DCL_OK = 0,
  DCL_E_ARG = 1,          /* null pointer, size or range outside the documented domain */
  DCL_E_UNSUPPORTED = 2,  /* geometry the library has no kernels for */
  DCL_E_WORKSPACE = 3,    /* workspace or weight buffer smaller than required */
  DCL_E_HIP = 4,          /* a HIP runtime call or kernel launch failed */
  DCL_E_STATE = 5         /* object used in the wrong state (e.g. step before weights load) */
} dcl_status;

/* Model geometry: a pre-norm bidirectional transformer with RMSNorm, rotate-half RoPE, SwiGLU
 * (the LLaDA / Dream base models of Section 4 setup). Host struct. Supported: head_dim 64 or
 * 128; n_heads % n_kv_heads == 0; d_model, d_ffn multiples of 16 (d_model <= 8192); vocab >= 2;
 * 0 <= mask_id < vocab; rms_eps > 0; rope_base > 1; 1 <= max_positions <= 65536. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab, mask_id;
  float rms_eps;          /* RMSNorm epsilon */
  float rope_base;        /* RoPE theta base */
  int32_t qkv_bias;       /* 1: q/k/v projections carry a bias (Dream / Qwen2.5 geometry) */
  int32_t rope_enabled;   /* 1 normally; 0 turns RoPE off (test support: permutation checks) */
  int32_t max_positions;  /* largest absolute position + 1 that a step may use */
} dcl_config;

typedef struct dcl_model_s* dcl_model_t;

/* Per-position prediction statistics, each array [B, S] (row b*S + i), device memory.
 * Scored rows: top1 = argmax_v P(x_i = v), top2 = best other id (ties to the lowest id),
 * conf = P(top1) (the confidence c_i), p2 = P(top2), lse = log sum_v exp(logit_v),
 * entropy = H(x_i) = -sum_v P log P = lse - sum_v P logit_v (the marginal entropy of the error
 * bound in Section 2.2); conf - p2 is the top-1/top-2 margin.
 * Rows that are not scored: top1 = top2 = -1, conf = p2 = -1, lse = 0, entropy = -1.
 * entropy may be NULL (not written); the other arrays are required. */
typedef struct {
  int32_t* top1;
  int32_t* top2;
  float* conf;
  float* p2;
  float* lse;
  float* entropy;
} dcl_row_stats;

/* Cached prefix for the KV-cache step (dLLM-Cache combination, Section 4 "Scalability and
 * Extension"): per layer l, k[l] -> bf16 [B, n_kv_heads, capacity, head_dim] keys AFTER RoPE,
 * v[l] -> bf16 [B, n_kv_heads, head_dim, capacity] values (key index contiguous); positions
 * [0, prefix_len) are in use. capacity = 0 means capacity = prefix_len.
 * `k` and `v` themselves are HOST arrays of n_layers device pointers (writable buffers for
 * dcl_kv_append). prefix_len >= 0, capacity % 8 == 0, prefix_len <= capacity. A prefix length that is not
 * a multiple of 8 (for example after appending the K_eff tokens one iteration committed) is supported:
 * the step carries the last prefix_len % 8 cached keys and values next to its fresh ones. */
typedef struct {
  const void* const* k;
  const void* const* v;
  int32_t prefix_len;
  int32_t capacity;
} dcl_kv;

enum { DCL_DTYPE_F32 = 0, DCL_DTYPE_BF16 = 1 };

/* dcl_denoise_step flags */
#define DCL_SCORE_ALL_UNCOMMITTED 0x1u  /* score every position p <= i < gen_end, not only masks */
#define DCL_SCORE_SUPPRESS_MASK 0x2u    /* leave the [MASK] id out of the vocabulary: it takes no
                                           probability mass and is never top-1 or top-2 */
/* dcl_select_contiguous flags */
#define DCL_SEL_NO_PROGRESS_GUARD 0x1u  /* literal K: a step with K = 0 commits nothing */
#define DCL_SEL_SCORE_ALL 0x2u          /* drafts may overwrite non-mask positions (pairs with
                                           DCL_SCORE_ALL_UNCOMMITTED) */
#define DCL_SEL_NONCONTIGUOUS 0x4u      /* the independent threshold rule (Eq. threshold_pd) in the
                                           window instead of Dynamic Contiguous Verification */
#define DCL_SEL_CONTIGUOUS_DRAFTS 0x8u  /* drafts only along the leading chain (Appendix E) */
#define DCL_SEL_MARGIN 0x10u            /* accept on the margin conf - p2 instead of conf (commit
                                           and draft thresholds alike) */

/* Text for a status code; never NULL. */
const char* dcl_status_string(dcl_status s);

/* Detail of the last non-OK status returned on this thread (empty string if none). */
const char* dcl_last_error(void);

/* Validate `cfg` (host) and create a handle. *out receives the handle (host). Every weight matrix
 * (vocab x d_model, (n_heads + 2*n_kv_heads)*head_dim x d_model, 2*d_ffn x d_model, ...) must hold
 * fewer than 2^31 elements (DCL_E_UNSUPPORTED otherwise). */
dcl_status dcl_model_create(const dcl_config* cfg, dcl_model_t* out);

/* Release the handle (host memory only; the weight buffer stays the caller's). NULL is a no-op. */
void dcl_model_destroy(dcl_model_t model);

/* Bytes of the packed device weight buffer for `cfg`; 0 if `cfg` is invalid. */
size_t dcl_weights_bytes(const dcl_config* cfg);

/* Pack the model's weights into `dev_buf` (device, `bytes` >= dcl_weights_bytes, 256-byte
 * aligned). `src` is a HOST array of `n_src` pointers (host or device memory) in this order:
 *   embed [vocab, d];
 *   per layer: wq [H*dh, d], wk [Hkv*dh, d], wv [Hkv*dh, d], bq [H*dh], bk [Hkv*dh], bv [Hkv*dh],
 *              wo [d, H*dh], wgate [F, d], wup [F, d], wdown [d, F], g_attn [d], g_ffn [d];
 *   g_final [d]; lm_head [vocab, d]
 * (nn.Linear [out, in] row-major; bias entries may be NULL when qkv_bias = 0), so
 * n_src = 1 + 12 * n_layers + 2. Elements are `src_dtype` (DCL_DTYPE_F32 or DCL_DTYPE_BF16);
 * float32 matrices are rounded to bfloat16 (nearest even), vectors are kept in float32.
 * The handle borrows `dev_buf`, which must outlive it. Synchronises `stream` before returning. */
dcl_status dcl_load_weights(dcl_model_t model, void* dev_buf, size_t bytes, const void* const* src,
                            int32_t n_src, int32_t src_dtype, hipStream_t stream);

/* Workspace bytes for a step over B sequences of S tokens (kv_prefix = cached prefix length,
 * 0 for a full forward); 0 if the arguments are invalid. */
size_t dcl_workspace_bytes(dcl_model_t model, int32_t B, int32_t S, int32_t kv_prefix);

/* Steps (ii) of the iteration: forward over tokens [B, S] (device) and the vocabulary reduction
 * at the scored rows of each sequence b: x[b,i] == mask_id and p[b] <= i < gen_end (Section 2.1:
 * probabilities are defined at masked positions), or every p[b] <= i < gen_end with
 * DCL_SCORE_ALL_UNCOMMITTED. p: device [B]; 0 <= gen_end <= S. Logits are never written to
 * memory. Token i is at absolute position kv_prefix + i; with kv == NULL the forward covers the
 * S tokens alone, otherwise they also attend to the cached prefix. Token ids outside
 * [0, vocab) read an all-zero embedding row. Writes `out` (all B*S rows). ws: device,
 * ws_bytes >= dcl_workspace_bytes(model, B, S, prefix), 256-byte aligned. Sizes: B*S <= 2^22
 * (DCL_E_ARG otherwise), B*(S+8)*(n_heads + 2*n_kv_heads)*head_dim < 2^31 (S+16 with a prefix length
 * that is not a multiple of 8) and
 * B*S*max(d_model, n_heads*head_dim, d_ffn) < 2^31 (DCL_E_UNSUPPORTED otherwise: the kernels
 * address q/k/v^T and the GEMM operands with 32-bit offsets). */
dcl_status dcl_denoise_step(dcl_model_t model, const int32_t* tokens, int32_t B, int32_t S,
                            const int32_t* p, int32_t gen_end, const dcl_kv* kv, uint32_t flags,
                            dcl_row_stats out, void* ws, size_t ws_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): dcl_denoise_step with its workspace taken from a static scratch
 * array of DCL_NOALLOC_SCRATCH_BYTES bytes inside the library, one per device, held until the process
 * ends. The call allocates nothing (no hipMalloc / hipFree, no allocating library routine); the first
 * call on a device looks up that device's scratch address (hipGetSymbolAddress) and keeps it. Steps
 * whose workspace (dcl_workspace_bytes) exceeds the scratch are rejected with DCL_E_WORKSPACE before
 * anything is launched (the LLaDA-8B geometry fits B*S = 384 tokens, and B = 8 x 64 tokens after a
 * cached prefix). Every call on a device shares that device's scratch: calls that overlap in time on
 * one device (two streams, two threads) race and give undefined results; calls ordered on one stream
 * are safe. Nothing in the scratch needs to start at zero (every step writes what it reads). Uses the
 * current device; `stream` must belong to it. Other arguments, results and errors as dcl_denoise_step. */
#define DCL_NOALLOC_SCRATCH_BYTES ((size_t)96 << 20)
dcl_status dcl_denoise_step_noalloc(dcl_model_t model, const int32_t* tokens, int32_t B, int32_t S,
                                    const int32_t* p, int32_t gen_end, const dcl_kv* kv, uint32_t flags,
                                    dcl_row_stats out, hipStream_t stream);

/* Steps (iii), (iv) and (i) for every sequence b with p[b] < gen_end, in place on tokens [B, S]
 * and p [B] (device), using statistics `in` of a dcl_denoise_step on the same tokens:
 *   end(q) = gen_end, or with semi-autoregressive blocks (block_len > 0; Section 4 setup, blocks of 32)
 *   the end of the block holding position q, blocks of block_len positions tiling the line from
 *   block_origin (normally the prompt length), capped at gen_end;
 *   L_eff = min(L, end(p) - p);  K = number of leading window rows with conf > tau_commit
 *   (Eq. compute_k);  K_eff = max(K, 1) unless DCL_SEL_NO_PROGRESS_GUARD (K = 0 would stall
 *   Algorithm 1; committing the top-1 at p is one sequential step);  x[p, p+K_eff) = top1;
 *   for j in [p+L, gen_end) with x[j] == mask_id (any x[j] with DCL_SEL_SCORE_ALL) and
 *   conf[j] > tau_draft: x[j] = top1[j] (Eq. draft_update);  p += K_eff;
 *   x[p, min(p+L, end(p))) = mask_id with the new p (Eq. remasking for the next iteration).
 * The window thus never crosses a block end, while drafts still look ahead over [p+L, gen_end).
 * A window start whose row was not scored (top1 < 0) is never committed. Sequences with
 * p >= gen_end (or p < 0) are untouched (K_raw = K_eff = 0). K_raw, K_eff: device [B] outputs (may be
 * NULL). 1 <= L; block_len >= 0 (0: no blocks); with blocks 0 <= block_origin <= S; 0 <= tau_commit <= 1;
 * tau_draft >= 0 (values > 1 disable drafts).
 * DCL_SEL_CONTIGUOUS_DRAFTS (the variant of Appendix E): only the leading chain of the draft
 *   region is drafted; it ends at the first eligible position (as above) with conf <= tau_draft,
 *   and positions that already hold a token keep it without ending the chain.
 * DCL_SEL_NONCONTIGUOUS (the baseline of Eq. threshold_pd, in the same window): every masked,
 *   scored position j of [p, p + L_eff) with conf[j] > tau_commit is committed independently; if
 *   none is and DCL_SEL_NO_PROGRESS_GUARD is off, the most confident one is (lowest j on ties);
 *   p moves to the first position >= p still holding mask_id (gen_end if none); there are no
 *   drafts and no remasking. K_raw = number above tau_commit, K_eff = number committed.
 * DCL_SEL_MARGIN: every comparison above uses conf - p2 (float32) in place of conf. */
dcl_status dcl_select_contiguous(int32_t* tokens, int32_t B, int32_t S, int32_t* p, int32_t gen_end,
                                 int32_t L, int32_t block_origin, int32_t block_len, float tau_commit,
                                 float tau_draft, int32_t mask_id, dcl_row_stats in, int32_t* K_raw,
                                 int32_t* K_eff, uint32_t flags, hipStream_t stream);

/* Algorithm 1 (Section 3, Appendix A) end to end on the device: Eq. remasking of the first window,
 * then repeated iterations of dcl_denoise_step (flags `score_flags`) followed by
 * dcl_select_contiguous (L, block_origin, block_len, tau_commit, tau_draft, `select_flags`, mask_id of
 * the model; block_len > 0 gives the semi-autoregressive block decoding of Section 4), until every
 * sequence has p >= gen_end or max_steps iterations ran. tokens [B, S] and p [B] (device) hold the
 * state in and out; stats, K_raw, K_eff and ws are as for the two calls above (K_raw, K_eff may be
 * NULL). k_hist (device int32 [L + 1], may be NULL) is incremented at K_eff once per sequence and
 * iteration in which the sequence was unfinished; the caller clears it.
 * p is copied to the host every `check_every` iterations (and after the last) to test for
 * completion; iterations that run after every sequence finished change nothing. *steps_out (host)
 * receives the number of iterations run. The first iteration is launched directly; the others
 * replay one iteration captured into a HIP graph on a stream the call creates (the caller's stream
 * may be the legacy null stream); with kernel-class profiling on, all run directly. The call
 * returns after the device finished; the caller's stream is ordered after the work. It allocates
 * only that stream, one event and the graph, and releases them before returning. With `kv` the
 * loop runs over the tokens after a cached prefix (the prefix-KV decode mode): every iteration
 * reads the cache, none writes it (dcl_kv_append does).
 * 1 <= max_steps, 1 <= check_every; other argument rules as for the two calls. */
dcl_status dcl_generate(dcl_model_t model, int32_t* tokens, int32_t B, int32_t S, int32_t* p,
                        int32_t gen_end, const dcl_kv* kv, uint32_t score_flags, int32_t L,
                        int32_t block_origin, int32_t block_len, float tau_commit, float tau_draft,
                        uint32_t select_flags, int32_t max_steps,
                        int32_t check_every, dcl_row_stats stats, int32_t* K_raw, int32_t* K_eff,
                        int32_t* k_hist, void* ws, size_t ws_bytes, int32_t* steps_out,
                        hipStream_t stream);

/* KV-cache write-back (the cache maintenance of the dLLM-Cache combination, Section 4): the forward
 * of the S tokens [B, S] (device) at positions prefix_len + i over the cached prefix `kv`, as in
 * dcl_denoise_step, writing every layer's keys (after RoPE) and values of those tokens into the
 * cache at positions [prefix_len, prefix_len + S). The caller then uses prefix_len + S (for
 * example after the block's tokens are committed). With prefix_len = 0 over a whole sequence it
 * is the periodic refresh: every cached position is recomputed with the full context. No LM head
 * runs; the last layer stops after its keys and values. Needs prefix_len + S <= capacity and a
 * workspace of dcl_workspace_bytes(model, B, S, prefix_len) bytes; the cache is read at positions
 * [0, prefix_len) and written at [prefix_len, prefix_len + S). */
dcl_status dcl_kv_append(dcl_model_t model, const int32_t* tokens, int32_t B, int32_t S,
                         const dcl_kv* kv, void* ws, size_t ws_bytes, hipStream_t stream);

/* Workspace bytes for dcl_score_hidden over n rows; 0 if the arguments are invalid. */
size_t dcl_score_workspace_bytes(dcl_model_t model, int32_t n);

/* The vocabulary reduction alone (the LM head and softmax statistics of Section 2.1, Eq. 2 and
 * Eq. threshold_pd) on given final hidden states: hidden bf16 [n, d_model] (device, 16-byte
 * aligned), already final-normalised. Writes statistics for rows 0..n-1 into `out` (each array
 * has n entries). Logits are never written to memory. ws: device, 256-byte aligned,
 * ws_bytes >= dcl_score_workspace_bytes(model, n). Sizes: 1 <= n <= 2^22 (DCL_E_ARG otherwise)
 * and n*d_model < 2^31 (DCL_E_UNSUPPORTED otherwise). */
dcl_status dcl_score_hidden(dcl_model_t model, const void* hidden, int32_t n, dcl_row_stats out,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* Test support: the same forward as dcl_denoise_step, then float32 logits of the rows listed in
 * `rows` (device [n_rows], flat indices b*S + i; an index outside [0, B*S) gives a zero hidden
 * row) into out (device [n_rows, vocab]); if hidden_out is not NULL it also receives those rows'
 * final hidden states (bf16 [n_rows, d_model]). */
dcl_status dcl_debug_logits(dcl_model_t model, const int32_t* tokens, int32_t B, int32_t S,
                            const dcl_kv* kv, const int32_t* rows, int32_t n_rows, float* out,
                            void* hidden_out, void* ws, size_t ws_bytes, hipStream_t stream);

/* Test support: the intermediate tensors of one transformer layer, each a device buffer of the stated
 * layout or NULL (not written). T = B*S. */
typedef struct {
  void* u;       /* bf16 [T, d_model]: bf16(RMSNorm(r_in) * g_attn) */
  void* q;       /* bf16 [B, n_heads, S, head_dim]: queries after bias and RoPE */
  void* k;       /* bf16 [B, n_kv_heads, c + S, head_dim]: keys after bias and RoPE, token s in slot c + s,
                    where c = prefix_len % 8 (slots [0, c) hold the newest cached keys) */
  void* v;       /* bf16 [B, n_kv_heads, head_dim, Sp]: values, key index contiguous in the same slots,
                    Sp = c + S rounded up to 8 (slots >= c + S are 0) */
  void* o;       /* bf16 [T, n_heads * head_dim]: attention output (softmax(q k^T / sqrt(dh)) v, no mask) */
  float* r_mid;  /* [T, d_model]: r_in + o W_o^T */
  void* u2;      /* bf16 [T, d_model]: bf16(RMSNorm(r_mid) * g_ffn) */
  void* a;       /* bf16 [T, d_ffn]: bf16(silu(u2 W_gate^T) * (u2 W_up^T)) */
  float* r_out;  /* [T, d_model]: r_mid + a W_down^T, the next layer's input */
} dcl_layer_taps;

/* Test support: layer `layer` of the forward of dcl_denoise_step (Algorithm 1, Forward) run alone on the
 * float32 residual stream r_in (device [B*S, d_model], the layer's input), with the same kernels, tile
 * plans and split-K folding as a step over B sequences of S tokens (tokens at positions
 * kv->prefix_len + i, attending to the cached prefix when kv != NULL). Every non-NULL tap receives
 * that intermediate; chaining r_out into the next call from the embedding rows reproduces the step's
 * residual stream bit for bit. ws as for dcl_denoise_step (its contents are overwritten). */
dcl_status dcl_debug_layer(dcl_model_t model, int32_t B, int32_t S, const dcl_kv* kv, int32_t layer,
                           const float* r_in, dcl_layer_taps taps, void* ws, size_t ws_bytes, hipStream_t stream);

/* Test support (host only): the tile plan a GEMM of Nw weight rows, T tokens and depth K runs with.
 * lm_head = 1 asks for the fused LM-head plan (vocabulary tiles of 128 ids), otherwise the plan of a
 * residual GEMM allowed max_split (1..4) K-split slices. info (host int32[8]) receives
 * {configuration index, K-split slices, weight rows, tokens, K depth per stage, stages, waves along
 * the weight rows, waves along the tokens}; an LM-head plan whose weight rows per wave equal 128 has
 * every wave own a whole vocabulary tile. */
dcl_status dcl_debug_gemm_plan(int32_t Nw, int32_t T, int32_t K, int32_t lm_head, int32_t max_split, int32_t* info);

/* Kernel-class timing (profiling support for benchmarks). While enabled, every kernel launch
 * made by dcl_denoise_step / dcl_score_hidden / dcl_select_contiguous is bracketed by a pair of
 * hipEvents recorded on the caller's stream (this adds a little host work per launch; leave it
 * off for throughput runs). dcl_profile_read synchronises the recorded events and returns, per
 * kernel class, the number of launches and the summed GPU time between each pair. Classes:
 * 0 embed, 1 rmsnorm, 2 gemm_qkv_rope, 3 attention, 4 gemm_o_residual, 5 gemm_gate_up_swiglu,
 * 6 gemm_down_residual, 7 compact_rows, 8 gemm_lm_head_top2, 9 merge_partials, 10 select.
 * Host-side state, per process; not thread-safe. */
enum { DCL_PROF_CLASSES = 11 };
typedef struct {
  int64_t launches[DCL_PROF_CLASSES];
  double ms[DCL_PROF_CLASSES];
} dcl_profile;

/* on = 1 starts recording (and clears previous totals), on = 0 stops. */
dcl_status dcl_profile_enable(int32_t on);
/* Totals since the last enable (host struct). Blocks until every recorded event has completed. */
dcl_status dcl_profile_read(dcl_profile* out);

#ifdef __cplusplus
}
#endif

#endif /* DCL_H_ */
