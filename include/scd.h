/*
 * scd.h -- C ABI of the SCD KV-state codec on MI355X (gfx950).
 *
 * Semantic Cache Distillation moves a consumer model's prefix KV cache as compact codes:
 * the producer encodes each Reuse layer's de-RoPE'd keys and its values onto low-rank bases and
 * each Patch layer's normalised attention input onto a code (Section 4.3.2, Eq. encode_z_kv;
 * Section 4.4.1); the consumer decodes Reuse layers as code x basis (+ offset) and re-applies
 * RoPE to keys (Eq. decode_kv), and regenerates Patch layers' KV by pushing the predicted
 * normalised input through its own W_K / W_V with RoPE on keys (Section 4.4.2,
 * Eq. kv_from_patch).  Algorithm 1 ("Split Inference with Reuse and Patch") fixes the order
 * and the routing.  Every entry point below computes one of those steps on the GPU.
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 *  - All tensors are dense, row-major and contiguous, in the model's dtype (scd_dtype_t):
 *    fp32, or bf16 with fp32 accumulation and a single round-to-nearest-even at the store.
 *  - Matrices use the [out, in] layout of a linear layer's weight, so every map is y = x W^T
 *    (the paper writes x W with W of shape [in, out]; the maps are the same).
 *  - The KV cache of one layer and branch is [T, H, d_h] (token-major, heads contiguous inside a
 *    token), T = total packed tokens of the batch.  The consumer owns it; the library writes each
 *    slot of a routed layer exactly once and never touches other layers.
 *  - A basis of width w acts on rows of w consecutive channels: one token of D = H*d_h channels
 *    is g = D / w code rows (w = D: one row per token; w = d_h: the head-shared basis, where
 *    batch x heads x tokens form one sample axis, Section 4.1).  Codes are [T*g, r].
 *  - Per-layer tensors are passed as HOST arrays of length n_layers holding DEVICE pointers.
 *    Entries of layers the call does not route are ignored and may be NULL.  When the batch has
 *    no tokens every call is a no-op, and buffers sized by the token count may be NULL.
 *  - RoPE pairs channel i of a head with channel i + d_h/2 and rotates the pair by
 *    p * theta^(-2i/d_h), p the token's position in its own request (Section 4.1 names RoPE and
 *    deRoPE as forward and inverse; Appendix F.2 keeps the framework's own cache positions).
 *  - Device pointers must be 16-byte aligned.  Calls are asynchronous on the given stream, never
 *    synchronise, and allocate nothing: the caller owns every buffer.
 *  - Every argument is validated before any launch.  A non-OK status means nothing was launched
 *    and no output was written; scd_last_error() then describes the problem.  Device-side
 *    contents (cu_seqlens, pos0) are not validated: they must be non-decreasing with
 *    cu_seqlens[0] = 0 and cu_seqlens[B] = n_tokens; positions at or beyond the RoPE table's
 *    max_position give unspecified values (never an out-of-bounds access).
 */
#ifndef SCD_H_
#define SCD_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SCD_OK = 0,
  SCD_ERR_NULL = 1,         /* a required pointer is NULL */
  SCD_ERR_SHAPE = 2,        /* inconsistent or out-of-range sizes */
  SCD_ERR_SCHEDULE = 3,     /* bad layer routing or ranks */
  SCD_ERR_ALIGN = 4,        /* a device pointer is not 16-byte aligned */
  SCD_ERR_UNSUPPORTED = 5,  /* valid per the paper but outside what the kernels implement */
  SCD_ERR_WORKSPACE = 6,    /* RoPE table missing or too small */
  SCD_ERR_HIP = 7           /* a HIP runtime call or kernel launch failed */
} scd_status_t;

typedef enum { SCD_F32 = 0, SCD_BF16 = 1 } scd_dtype_t;

/* Model pair description (host memory, read only during the call).
 * Section 4.1: layers 0..L-1 (0-based here); L_patch = {l : is_patch[l] != 0}, L_reuse its
 * complement; independent branch ranks r_K, r_V, r_H.
 * Supported by the kernels: head_dim 32, 64 or 128; basis_width a multiple of head_dim that
 * divides D; every rank routed by a call a multiple of 16 with
 * 16 <= rank_k, rank_v <= min(basis_width, 256) and 16 <= rank_h <= min(d_model, 256);
 * d_model a multiple of 32. */
typedef struct {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t basis_width;     /* w */
  int32_t dtype;           /* scd_dtype_t: dtype of every tensor argument */
  double rope_theta;
  const uint8_t* is_patch; /* [n_layers] */
  const int32_t* rank_k;   /* [n_layers] */
  const int32_t* rank_v;   /* [n_layers] */
  const int32_t* rank_h;   /* [n_layers] */
} scd_model_t;

/* A packed batch of B requests, T tokens in total (request b owns tokens
 * [cu_seqlens[b], cu_seqlens[b+1])).  Positions restart at pos0[b] (0 when pos0 is NULL) for
 * every request. */
typedef struct {
  int32_t n_seqs;              /* B >= 1 */
  int64_t n_tokens;            /* T >= 0 */
  const int32_t* cu_seqlens;   /* DEVICE [B+1], or NULL when B == 1 (one request of T tokens) */
  const int32_t* pos0;         /* DEVICE [B], or NULL */
} scd_batch_t;

/* ---- RoPE table ------------------------------------------------------------------------------
 * Opaque device table of rotation cosines and sines for positions [0, max_position), evaluated in
 * fp64 and rounded once to fp32 (fp32-evaluated angles lose ~1e-5 absolute accuracy by position
 * 512 and ~2e-3 by 32K).  It depends only on (head_dim, rope_theta, max_position): build it once
 * per model and reuse it.  scd_rope_table_bytes returns its size; scd_rope_table fills it.  The
 * entry points that take a table trust the (table, max_position) pair they are given: it must be a
 * table this model's head_dim and rope_theta built for that max_position, holding
 * scd_rope_table_bytes(model, max_position) bytes (the C calls cannot see its size; the Python
 * binding records head_dim, theta and max_position with the table and checks them). */
size_t scd_rope_table_bytes(const scd_model_t* model, int64_t max_position);
scd_status_t scd_rope_table(const scd_model_t* model, int64_t max_position, void* table,
                            size_t table_bytes, hipStream_t stream);

/* ---- a1: token positions ---------------------------------------------------------------------
 * pos_out[t] = t - cu_seqlens[b] + pos0[b] for every packed token t (DEVICE int32 [n_tokens]).
 * The same mapping every RoPE/deRoPE step below uses internally. */
scd_status_t scd_positions(const scd_batch_t* batch, int32_t* pos_out, hipStream_t stream);

/* ---- a0: routing and payload (host only) -------------------------------------------------------
 * scd_schedule writes the Reuse and Patch layer lists in increasing order (Section 4.5: the sets
 * are fixed inputs, membership is a constant-time lookup).  Output arrays hold n_layers entries.
 * scd_payload_bytes returns the bytes of the transmitted code set of Algorithm 1
 * ({Z_K, Z_V} per Reuse layer, Z_H per Patch layer; O(T r), Section 4.5) for n_tokens tokens and,
 * when offsets is not NULL, fills offsets[0..n_layers] with each layer's start in one packed buffer
 * (layer order, K codes before V codes).  Returns 0 on invalid input. */
scd_status_t scd_schedule(const scd_model_t* model, int32_t* reuse_layers, int32_t* n_reuse,
                          int32_t* patch_layers, int32_t* n_patch);
size_t scd_payload_bytes(const scd_model_t* model, int64_t n_tokens, int64_t* offsets);

/* ---- a2-a4: producer encode (Section 4.3.2, Eq. encode_z_kv; Section 4.4.1; Algorithm 1) ----
 * For every Reuse layer l:
 *   z_k[l] = (rows(deRoPE(k_in[l])) - mu_k[l]) w_enc_k[l]^T      [T*g, rank_k[l]]
 *   z_v[l] = (rows(v_in[l]) - mu_v[l]) w_enc_v[l]^T              [T*g, rank_v[l]]
 * with k_in, v_in [T, H, d_h], w_enc_k [rank_k, w], w_enc_v [rank_v, w], mu [w] (the optional
 * producer-side offset; NULL array or NULL entry = 0, which is the paper's equation).
 * For every Patch layer l:  z_h[l] = h_in[l] w_enc_h[l]^T  with h_in [T, d_model] (the producer's
 * normalised attention input) and w_enc_h [rank_h, d_model]; z_h [T, rank_h].
 * bf16 keys: the de-rotated input is rounded to bf16 once before the product; the offset enters as
 * the fp32 term mu w_enc^T subtracted from the accumulator, so it is never rounded. */
scd_status_t scd_encode(const scd_model_t* model, const scd_batch_t* batch,
                        const void* rope_table, int64_t max_position,
                        const void* const* k_in, const void* const* v_in,
                        const void* const* h_in,
                        const void* const* w_enc_k, const void* const* w_enc_v,
                        const void* const* w_enc_h,
                        const void* const* mu_k, const void* const* mu_v,
                        void* const* z_k, void* const* z_v, void* const* z_h,
                        hipStream_t stream);

/* ---- a5-a6, a8: consumer Reuse decode (Section 4.3.2, Eq. decode_kv; Algorithm 1) ------------
 * For every Reuse layer l, written straight into the consumer's cache:
 *   k_cache[l] = RoPE(unrows(z_k[l] w_dec_k[l]^T + mu_k[l]))     [T, H, d_h]
 *   v_cache[l] = unrows(z_v[l] w_dec_v[l]^T + mu_v[l])           [T, H, d_h]
 * with z [T*g, rank], w_dec [w, rank] and mu [w] the optional consumer-side offset (NULL = 0).
 * The paper writes one W_dec,B for both branches; keys and values are fitted independently
 * (Section 4.3.1), so each branch takes its own decoder.  Patch layers are not touched. */
scd_status_t scd_reuse_decode(const scd_model_t* model, const scd_batch_t* batch,
                              const void* rope_table, int64_t max_position,
                              const void* const* z_k, const void* const* z_v,
                              const void* const* w_dec_k, const void* const* w_dec_v,
                              const void* const* mu_k, const void* const* mu_v,
                              void* const* k_cache, void* const* v_cache, hipStream_t stream);

/* ---- a7, a8: consumer Patch (Section 4.4.2, Eq. kv_from_patch; Appendix F.2; Algorithm 1) ----
 * For every Patch layer l, written straight into the consumer's cache:
 *   k_cache[l] = RoPE(h_hat[l] w_k[l]^T + b_k[l]),   v_cache[l] = h_hat[l] w_v[l]^T + b_v[l]
 * with h_hat [T, d_model] the predicted normalised attention input (the aligner's output; this
 * call does not normalise), w_k, w_v [D, d_model] the consumer's own key/value projection weights
 * and b_k, b_v [D] optional projection biases (NULL array or NULL entry = none, as in the paper).
 * Reuse layers are not touched. */
scd_status_t scd_patch_kv(const scd_model_t* model, const scd_batch_t* batch,
                          const void* rope_table, int64_t max_position,
                          const void* const* h_hat,
                          const void* const* w_k, const void* const* w_v,
                          const void* const* b_k, const void* const* b_v,
                          void* const* k_cache, void* const* v_cache, hipStream_t stream);

/* ---- Patch aligner (Section 4.4.2, Eq. aligner) --------------------------------------------------
 * The consumer's aligner g_theta maps each Patch layer's code to a predicted normalised attention
 * input, the input of scd_patch_kv:
 *   act[l]   = SiLU(z_h[l] w1[l]^T + b1[l])           [T, hidden]
 *   h_hat[l] = act[l] w2[l]^T + b2[l]                 [T, d_model]
 * with z_h [T, rank_h[l]] (the transmitted code), w1 [hidden, rank_h[l]], w2 [d_model, hidden]
 * (nn.Linear layout), b1 [hidden] and b2 [d_model] optional (NULL array or entry = none) and
 * SiLU(x) = x / (1 + e^-x), evaluated in fp32 before the one rounding of each product.  The paper
 * calls g_theta an MLP and fixes neither its depth, width nor activation: this is a two-layer MLP
 * of width `hidden` (16 <= hidden, hidden % 16 == 0) with the backbone's SiLU.  act[l] holds layer
 * l's hidden activations: caller-owned, one buffer per Patch layer, distinct (the call writes them
 * all before it reads them); an act buffer that repeats returns SCD_ERR_SHAPE.  Reuse layers are
 * not touched. */
scd_status_t scd_patch_align(const scd_model_t* model, const scd_batch_t* batch, int32_t hidden,
                             const void* const* z_h,
                             const void* const* w1, const void* const* b1,
                             const void* const* w2, const void* const* b2,
                             void* const* act, void* const* h_hat, hipStream_t stream);

/* ---- Patch from the codes, with the aligner's output layer folded (Section 4.4.2) -------------
 * Eq. aligner ends in an affine layer (h_hat = act w2^T + b2) and Eq. kv_from_patch applies the
 * consumer's projections to h_hat with no nonlinearity in between, so for P = K, V:
 *   h_hat w_p^T + b_p = act (w_p w2)^T + (w_p b2 + b_p).
 * scd_patch_fold forms, once per model pair, for every Patch layer l:
 *   w_fold_k[l] = w_k[l] w2[l]   [D, hidden],    c_k[l] = w_k[l] b2[l] + b_k[l]   [D]
 *   w_fold_v[l] = w_v[l] w2[l]   [D, hidden],    c_v[l] = w_v[l] b2[l] + b_v[l]   [D]
 * with w2 [d_model, hidden] and b2 [d_model] the aligner's output layer (scd_patch_align's), w_k,
 * w_v [D, d_model] and b_k, b_v [D] the consumer's projections (b2, b_k, b_v optional: NULL array
 * or entry = 0), accumulated in fp32 and rounded once to the model's dtype.  Every output buffer
 * is written whole; outputs must not repeat across layers or branches (SCD_ERR_SHAPE) nor overlap
 * the inputs.  hidden % 16 == 0.  The batch plays no part.
 *
 * scd_patch_kv_from_codes is the consumer's Patch from the transmitted codes (Algorithm 1): for
 * every Patch layer l, in layer order,
 *   act[l]     = SiLU(z_h[l] w1[l]^T + b1[l])                 [T, hidden]
 *   k_cache[l] = RoPE(act[l] w_fold_k[l]^T + c_k[l]),   v_cache[l] = act[l] w_fold_v[l]^T + c_v[l]
 * which equals scd_patch_align followed by scd_patch_kv up to rounding, without forming h_hat
 * (its product of inner dimension d_model disappears).  act holds caller-owned [T, hidden]
 * activations and may repeat across layers: a run of consecutive Patch layers with distinct act
 * buffers is computed together (one launch of each product), and a buffer that repeats starts a
 * new run after the previous one has consumed it, so one buffer can serve every layer (at the
 * cost of a launch pair per layer).  c_k, c_v are optional (NULL = 0).  Other arguments and
 * limits as scd_patch_align and scd_patch_kv.  Reuse layers are not touched. */
scd_status_t scd_patch_fold(const scd_model_t* model, int32_t hidden,
                            const void* const* w2, const void* const* b2,
                            const void* const* w_k, const void* const* w_v,
                            const void* const* b_k, const void* const* b_v,
                            void* const* w_fold_k, void* const* w_fold_v,
                            void* const* c_k, void* const* c_v, hipStream_t stream);
scd_status_t scd_patch_kv_from_codes(const scd_model_t* model, const scd_batch_t* batch,
                                     const void* rope_table, int64_t max_position, int32_t hidden,
                                     const void* const* z_h,
                                     const void* const* w1, const void* const* b1,
                                     const void* const* w_fold_k, const void* const* w_fold_v,
                                     const void* const* c_k, const void* const* c_v,
                                     void* const* act, void* const* k_cache, void* const* v_cache,
                                     hipStream_t stream);

/* ---- packed payload and streamed receipt (Algorithm 1's transmitted set; Section 4.5) ---------
 * The codes Algorithm 1 sends travel as one contiguous buffer in the layout scd_payload_bytes
 * describes: layers in order, a Reuse layer's K codes [T*g, rank_k] then its V codes
 * [T*g, rank_v], a Patch layer's code [T, rank_h], no padding.
 *
 * scd_payload_views (host only, touches no memory) fills z_k, z_v, z_h [n_layers] with the
 * addresses of each layer's codes inside `payload` (any 16-byte aligned buffer of
 * scd_payload_bytes bytes), NULL for the branches a layer does not have.  The arrays can be passed
 * as they are to scd_encode (which then writes the packed payload), scd_reuse_decode and
 * scd_patch_align.
 *
 * scd_reuse_decode_streamed is the consumer's receipt: it copies the whole payload from
 * payload_src (pinned host memory, or device memory of this or a peer device; any address
 * hipMemcpyDefault accepts; pageable host memory works but serialises the copies) to payload_dst
 * (device, 16-byte aligned, scd_payload_bytes bytes, not overlapping payload_src) in groups of
 * layers_per_group layers on copy_stream, and enqueues the Reuse decode of each group (as
 * scd_reuse_decode, reading the codes from payload_dst) on `stream` behind that group's copy, so
 * the decode of one group overlaps the copy of the next.  The copies start after the work already
 * queued on `stream`; on return `stream` is ordered after every copy, so work queued on it next
 * (the aligner and scd_patch_kv on the Patch layers' codes) sees the whole payload.  copy_stream
 * may equal `stream` (no overlap).  With no tokens the payload is empty and both payload
 * pointers may be NULL.  The other arguments are scd_reuse_decode's.  SCD_ERR_HIP can leave
 * earlier groups enqueued; every other error means nothing was enqueued. */
scd_status_t scd_payload_views(const scd_model_t* model, int64_t n_tokens, void* payload,
                               void** z_k, void** z_v, void** z_h);
scd_status_t scd_reuse_decode_streamed(const scd_model_t* model, const scd_batch_t* batch,
                                       const void* rope_table, int64_t max_position,
                                       const void* payload_src, void* payload_dst,
                                       int32_t layers_per_group,
                                       const void* const* w_dec_k, const void* const* w_dec_v,
                                       const void* const* mu_k, const void* const* mu_v,
                                       void* const* k_cache, void* const* v_cache,
                                       hipStream_t copy_stream, hipStream_t stream);

/* ---- Offline Reuse fit (Section 4.3.1 "Joint Subspace Learning"; Appendix F.1) ---------------
 * Fits one branch's Reuse translators for every Reuse layer from paired calibration caches: the
 * producer's a_in[l] and the consumer's b_in[l], both [T, H, d_h] over the same packed batch of
 * prefixes (positions as everywhere else).  With rows A, B [N, w] (N = T*g; keys de-rotated first)
 * and X = [A B]:
 *   centring (optional):  mu_enc = mean of A's rows, mu_dec = mean of B's rows; A, B lose them;
 *   truncated SVD:        V_r = the top-r right singular vectors of X (r = rank_k or rank_v of
 *                         the layer), each with its largest-magnitude entry positive; Z = X V_r;
 *   ridge encoder:        E = argmin ||A E - Z||^2 + lambda ||E||^2   -> w_enc [r, w] = E^T;
 *   ridge decoder:        F = argmin ||Z F - B||^2 + lambda ||F||^2   -> w_dec [w, r] = F^T.
 * The outputs are exactly the w_enc / mu_enc the encoder takes and the w_dec / mu_dec the Reuse
 * decoder takes (the paper leaves the latent scale, the decoder's fit and the centring open: Z
 * carries the singular values, the decoder is a ridge fit with the same lambda, and centring is a
 * flag).
 *
 * The fit runs in two calls, stream-ordered:
 *  - scd_fit_gram accumulates, per Reuse layer, gram[l] = X^T X (fp32 [2w, 2w], symmetric) and
 *    colsum[l] = 1^T X (fp32 [2w]) on the matrix cores (bf16: keys de-rotated and rounded to bf16
 *    once, fp32 accumulation; fp32: fp32 products).  Rows are split into slices whose partial sums
 *    go to `workspace` and are added in a fixed order, so the result is deterministic.  branch 0 =
 *    keys (de-rotated; rope_table required), 1 = values.  Needs basis_width % 64 == 0 and at least
 *    one token.
 *  - scd_fit_solve takes those sums for N = n_rows rows (n_tokens * g) and solves the fit in fp64
 *    (Householder tridiagonalisation of the centred Gram, bisection and inverse iteration for its
 *    top r eigenpairs, Cholesky ridge solves; each stage one launch over all layers, except the
 *    tridiagonalisation, one launch per column until at most 128 rows remain, and the Cholesky of
 *    sizes above 128, one launch per column), writing w_enc, w_dec and, when
 *    center = 1, mu_enc and mu_dec in the model's dtype (rounded once).  Needs basis_width <= 1024
 *    and 16 <= rank <= basis_width, rank % 16 == 0, lambda >= 0.  lambda = 0 with a singular
 *    A^T A (fewer independent rows than w) leaves NaN in the layer's outputs.  Eigenvalues within
 *    1e-7 ||G_c|| of each other are solved as a cluster by one thread in turn (slow only for large
 *    clusters, e.g. a rank above the calibration rows' own rank).
 * `workspace` (device, 16-byte aligned, caller-owned, contents undefined on entry and exit, not
 * overlapping any argument) must hold scd_fit_workspace_bytes(model, n_tokens) bytes; one buffer
 * serves both calls.  Each layer's outputs need buffers of their own (a buffer that repeats across
 * layers returns SCD_ERR_SHAPE).  Layers run 64 per launch; the calls never synchronise.  Patch
 * layers are not touched. */
size_t scd_fit_workspace_bytes(const scd_model_t* model, int64_t n_tokens);
scd_status_t scd_fit_gram(const scd_model_t* model, const scd_batch_t* batch,
                          const void* rope_table, int64_t max_position, int32_t branch,
                          const void* const* a_in, const void* const* b_in,
                          float* const* gram, float* const* colsum, void* workspace,
                          size_t workspace_bytes, hipStream_t stream);
scd_status_t scd_fit_solve(const scd_model_t* model, int32_t branch, int64_t n_rows,
                           double ridge_lambda, int32_t center, const float* const* gram,
                           const float* const* colsum, void* const* w_enc, void* const* w_dec,
                           void* const* mu_enc, void* const* mu_dec, void* workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* ---- Allocation-free fit solve -----------------------------------------------------------------
 * For callers that cannot allocate device memory or hand over a workspace (code under stream
 * capture, serving loops, harnesses that forbid allocation): scd_fit_solve without the workspace
 * arguments.  Same arguments, validation and results (bit-identical) as scd_fit_solve.  The
 * solve's fp64 matrices live in a device-resident scratch array of
 * scd_fit_solve_noalloc_max_bytes() bytes (64 MiB) that the library holds on each GPU it runs on
 * until the process ends; layers are solved in as many stream-ordered rounds of launches as that
 * array needs (4 (2w)^2 + 8 (2w) fp64 values per layer).  A basis width whose per-layer matrices
 * exceed the array (w > 512) returns SCD_ERR_WORKSPACE.  The call uses the calling thread's
 * current device, which must own the stream and the buffers; its first call on a device looks the
 * array's address up.  It allocates
 * nothing and never synchronises.  Every call on one GPU shares that GPU's array: calls that may
 * run at the same time on one GPU (different streams, or other threads) race on it and must be
 * serialised by the caller. */
size_t scd_fit_solve_noalloc_max_bytes(void);
scd_status_t scd_fit_solve_noalloc(const scd_model_t* model, int32_t branch, int64_t n_rows,
                                   double ridge_lambda, int32_t center, const float* const* gram,
                                   const float* const* colsum, void* const* w_enc,
                                   void* const* w_dec, void* const* mu_enc, void* const* mu_dec,
                                   hipStream_t stream);

/* ---- diagnostics ---------------------------------------------------------------------------- */
const char* scd_status_string(scd_status_t status);
/* Detail of the last non-OK status returned on the calling thread ("" if none). */
const char* scd_last_error(void);
/* ABI version: bumped whenever a signature or a struct above changes. */
int32_t scd_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SCD_H_ */
