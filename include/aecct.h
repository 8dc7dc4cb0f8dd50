/*
 * aecct.h -- C ABI of the MI355X (gfx950) AECCT inference library.
 *
 * AECCT (Levy, Choukroun, Wolf, "Accelerating Error Correction Code
 * Transformers") decodes a binary linear code with a transformer encoder.
 * This library runs its batched inference forward pass: channel words y in,
 * bit decisions out.
 *
 * What one decode computes, per received word (Section 3, "Problem Settings"
 * and "Error Correction Code Transformer"; Section 4; Section 6):
 *   1. h(y) = [|y|, 1 - 2 s(y)] with s(y) = H bin(y) mod 2: 2n-k tokens, the n
 *      variable nodes first, then the n-k check nodes of the Tanner graph;
 *   2. each token scalar times its row of the embedding table (plus an
 *      optional fixed positional table, the inference form of the spectral
 *      positional encoding of Section 4.3);
 *   3. N Post-LN encoder blocks (Section 6).  Each block applies head
 *      partitioned self-attention (Section 4.2: the first h_f heads attend
 *      over Tanner neighbours, the rest over nodes two steps away, self
 *      included), then a ReLU feed-forward block (Section 4, item 4); every
 *      in-block linear map is an AAP linear layer (Section 4.1, Eq. 2-3):
 *      per-token absmax int8 activations times ternary weights, int32
 *      accumulation, dequantised by (weight scale) * alpha / 127 before the
 *      fp32 bias;
 *   4. the output head of Section 3: z = W_{d->1} x + b1 per token, then
 *      f = W_o^T z + b_o over tokens, and the hard decision
 *      bit = bin(y * f) = [y < 0] xor [f < 0].
 * The fp32 arithmetic follows one fixed evaluation order, so results are
 * reproducible bit for bit between runs, batch sizes and kernel paths.
 *
 * Conventions for every entry point:
 *   - The return value is the only error channel; no global state is kept.
 *   - "device" pointers are HIP device memory (or managed memory) of the GPU
 *     that was current at aecct_create; "host" pointers are ordinary memory.
 *   - stream is a hipStream_t passed as void* (NULL = the default stream).
 *     Entry points that take a stream only enqueue work on it; they neither
 *     allocate nor synchronise.  Results are ready once the stream is.
 *   - A model is immutable after create: concurrent calls with the same model
 *     on different streams are safe if their outputs and workspaces differ.
 */
#ifndef AECCT_H
#define AECCT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum aecct_status {
  AECCT_OK = 0,
  AECCT_ERR_INVALID_ARG = 1,          /* null pointer, bad size, non-ternary weight, bad H ... */
  AECCT_ERR_UNSUPPORTED = 2,          /* valid model outside the shapes the kernels implement */
  AECCT_ERR_OUT_OF_MEMORY = 3,        /* host or device allocation failed */
  AECCT_ERR_DEVICE = 4,               /* a HIP call or kernel launch failed */
  AECCT_ERR_WORKSPACE_TOO_SMALL = 5
} aecct_status;

/* Kernel path.  Both give identical results (same evaluation order). */
typedef enum aecct_path {
  AECCT_PATH_AUTO = 0,     /* fused when a word fits in on-chip memory, else layered */
  AECCT_PATH_LAYERED = 1,  /* one kernel per stage, intermediates in device memory */
  AECCT_PATH_FUSED = 2     /* whole words resident in LDS, all layers in one launch */
} aecct_path;

/* The six in-block linear maps, in the order used by `scale` and `aecct_ternary_gemm`. */
typedef enum aecct_linear {
  AECCT_LIN_Q = 0, AECCT_LIN_K = 1, AECCT_LIN_V = 2, AECCT_LIN_O = 3, AECCT_LIN_FF1 = 4,
  AECCT_LIN_FF2 = 5
} aecct_linear;

/*
 * Model parameters, all HOST pointers, row-major, read (and copied) by
 * aecct_create only; the caller keeps ownership.  L = n + m tokens.
 * Linear weights are stored [in][out] (x W, Section 4.1) with entries in
 * {-1, 0, +1}; scale[l][k] is the per-matrix weight scale gamma*delta of Eq. 3.
 */
typedef struct aecct_weights {
  const float *embed;                         /* [L][d] token embedding rows */
  const float *pos;                           /* [L][d] fixed positional rows, or NULL */
  const int8_t *w_q, *w_k, *w_v, *w_o;        /* [N][d][d] */
  const int8_t *w_ff1;                        /* [N][d][d_ff] */
  const int8_t *w_ff2;                        /* [N][d_ff][d] */
  const float *scale;                         /* [N][6] in aecct_linear order */
  const float *b_q, *b_k, *b_v, *b_o;         /* [N][d] */
  const float *b_ff1;                         /* [N][d_ff] */
  const float *b_ff2;                         /* [N][d] */
  const float *ln1_g, *ln1_b, *ln2_g, *ln2_b; /* [N][d] LayerNorm gain / offset */
  const float *head_w1;                       /* [d]   W_{d->1} */
  float head_b1;
  const float *head_wo;                       /* [L][n] W_o */
  const float *head_bo;                       /* [n] */
} aecct_weights;

/* Attention masks of the heads. */
typedef enum aecct_attention {
  AECCT_ATTN_HPSA = 0,  /* head partitioning (Section 4.2): heads 0..h_f-1 over the first-ring
                           mask (Tanner neighbours), the rest over the second-ring mask (nodes two
                           steps away, the node itself included) */
  AECCT_ATTN_CASA = 1   /* the ECCT mask for every head (Section 3, code-aware self attention): the
                           union of the two rings, nodes at most two steps away; h_f is ignored */
} aecct_attention;

/* How the layered path computes a layer's queries, keys, values (Eq. 3) and attention
   (Section 4.2); every form gives the same results bit for bit. */
typedef enum aecct_layered_attention {
  AECCT_LAYERED_ATTN_AUTO = -1,    /* the fastest form the shape allows (the default) */
  AECCT_LAYERED_ATTN_UNFUSED = 0,  /* ternary GEMM to Q, K, V in device memory, then attention */
  AECCT_LAYERED_ATTN_LDS_F32 = 1,  /* fused per word and 16-dimension head group, K and V in
                                      LDS as fp32 (d = 64, 128, short words) */
  AECCT_LAYERED_ATTN_LDS_I16 = 2,  /* fused, V (and, on the longest words or with 8-dimension
                                      heads, K too) in LDS as int16 accumulators with per-token
                                      scales, the rest as fp32 (d = 64, 128, longer words) */
  AECCT_LAYERED_ATTN_LDS_SPLIT = 3 /* fused, each head's rows one node type at a time (Section 4.2:
                                      under head partitioning a row reads keys of one node type),
                                      that type's keys and values in LDS as fp32 (d = 128,
                                      16-dimension heads, HPSA, the larger node type within LDS) */
} aecct_layered_attention;

/* Granularity of the Eq. 2 activation scale alpha = ||x||_inf (Section 4.1).  The paper calls
   every scaling factor a scalar and leaves open over which part of a layer input x it is taken. */
typedef enum aecct_act_scale {
  AECCT_ACT_SCALE_TOKEN = 0,  /* one alpha per token row of x (the default) */
  AECCT_ACT_SCALE_WORD = 1    /* one alpha per received word: the maximum over all of its tokens'
                                 features at that quantisation point (every word of a batch keeps
                                 its own, so words stay independent) */
} aecct_act_scale;

/* Every field is read; -1 selects the default where a field allows it.  A NULL options pointer
   is the same as { -1, -1, 0, AUTO, HPSA, AUTO, TOKEN }. */
typedef struct aecct_options {
  int32_t first_ring_heads;   /* h_f, 0..heads; -1 = heads / 2 (the paper's default split) */
  int32_t d_ff;               /* feed-forward width; -1 = 4 d */
  float ln_eps;               /* LayerNorm epsilon; <= 0 = 1e-5 */
  int32_t path;               /* aecct_path */
  int32_t attention;          /* aecct_attention */
  int32_t layered_attention;  /* aecct_layered_attention (the layered path's form); a form the
                                 shape does not allow gives AECCT_ERR_UNSUPPORTED.  AUTO takes the
                                 first that fits of LDS_F32, LDS_I16, LDS_SPLIT, UNFUSED */
  int32_t act_scale_mode;     /* aecct_act_scale.  WORD runs on the layered path in its unfused
                                 form with natural activation layouts (path AUTO resolves to it;
                                 FUSED or a fused layered form gives AECCT_ERR_UNSUPPORTED) */
} aecct_options;

typedef struct aecct_model aecct_model;   /* opaque */

/*
 * Build a model on the current HIP device.
 *   H    host [m][n] parity-check matrix (Section 3), entries 0/1, no
 *        all-zero row or column (such a node would have an empty attention
 *        row); the HPSA masks of Section 4.2 are derived from it here;
 *   w    parameters as above; d model width, n_layers >= 1, heads >= 1;
 *   opt  may be NULL (defaults).
 * Supported shapes: d in {32, 64, 128}, d / heads in {4, 8, 16}, d_ff = 4 d,
 * n + m <= 4096; anything else valid returns AECCT_ERR_UNSUPPORTED.
 * All arguments are validated before any HIP call.  The model's tables are sized
 * for the current device's compute units and LDS per workgroup, and the kernels'
 * launch limits are set for it.  On success *out owns device memory until
 * aecct_destroy.  Errors: INVALID_ARG, UNSUPPORTED, OUT_OF_MEMORY, DEVICE (no
 * GPU, or a HIP allocation, copy or attribute call failed).
 */
aecct_status aecct_create(const uint8_t *H, int32_t m, int32_t n, const aecct_weights *w, int32_t d,
                          int32_t n_layers, int32_t heads, const aecct_options *opt, aecct_model **out);

/*
 * Ternary weights and weight scale of one AAP linear layer from its trained
 * fp32 weights (Section 4.1, Eq. 1): the step that turns a checkpoint into
 * the `aecct_weights` above.  Host call, no GPU work.
 *   gamma    = Percentile(|W|, p): the p-quantile of the `count` absolute
 *              values, interpolated linearly between the order statistics
 *              floor(pos) and floor(pos) + 1 at pos = p (count - 1) (zero
 *              based), evaluated in double and rounded once to fp32; the
 *              paper's p is 0.5, the median;
 *   *scale   = fp32(gamma * delta), the matrix scale gamma*delta of Eq. 3;
 *   ternary  = RoundClip(W / (scale + eps), -1, 1): the fp32 quotient by
 *              fp32(scale + eps), rounded to the nearest integer (ties to
 *              even) and clipped; if scale + eps is 0 the quotient of a
 *              nonzero weight counts as +-infinity (ternary = its sign) and a
 *              zero weight gives 0.
 *   w          host fp32 [count], any layout (only the multiset of |w|
 *              matters for gamma); must be finite;
 *   percentile p in [0, 1]; delta the learned factor, finite and > 0;
 *   eps        the paper's epsilon, finite and >= 0 (1e-8 is usual);
 *   ternary    host int8 [count] out, entry i from w[i]; scale host fp32 out.
 * count >= 1.  Errors: INVALID_ARG (and OUT_OF_MEMORY for the copy of |w|).
 */
aecct_status aecct_aap_ternarize(const float *w, int64_t count, float percentile, float delta, float eps,
                                 int8_t *ternary, float *scale);

/*
 * Spectral positional encoding of the Tanner graph (Section 4.3, the SPE
 * equations and Fig. 4): a create-time step whose output is the fixed
 * positional table `aecct_weights.pos`.
 *
 * Graph: L = n + m nodes, variable nodes 0..n-1 then checks; node i and node
 * n + j are joined where H[j][i] = 1.  Laplacian: D - A.
 *
 * Canonical eigenbasis (the paper leaves signs and bases of repeated
 * eigenvalues open): eigenvalues ascending; consecutive ones closer than
 * 1e-8 * max(1, max |lambda|) form one cluster; a cluster's basis is built from
 * the columns P e_c of its eigenspace projector P in ascending c, each with the
 * components along the vectors already taken removed, taken (normalised) when
 * its squared norm exceeds 1e-6, until the cluster's dimension is reached.  It
 * depends on the eigenspaces only, and gives a simple eigenvalue's vector the
 * sign that makes its first entry of squared size above 1e-6 positive.
 *
 * aecct_tanner_spectrum: host call, no GPU work, float64 (Householder
 * tridiagonalisation, then implicit QR steps with Wilkinson shifts).
 *   H        host uint8 [m][n], 0/1 (zero rows or columns allowed);
 *   eigvals  host double [L] out, ascending;
 *   eigvecs  host double [L][L] out, row i = canonical unit eigenvector i.
 * 1 <= m, 1 <= n, L <= 4096.  Errors: INVALID_ARG, OUT_OF_MEMORY,
 * UNSUPPORTED (the iteration did not converge; not expected).
 */
aecct_status aecct_tanner_spectrum(const uint8_t *H, int32_t m, int32_t n, double *eigvals, double *eigvecs);

/*
 * Parameters of the SPE network, host fp32, row-major, [in][out]:
 *   for node j, Phi_j in R^{L x 2} has row i = (lambda_i, phi_i[j]);
 *   Z = Phi_j w_in + b_in                      (W_{2->d_PE}, [2][d_pe]);
 *   multi-head self-attention over the L rows with Q = K = V = Z:
 *     head h of `heads` uses columns h*dk..h*dk+dk-1, dk = d_pe / heads, of
 *     Z w_q + b_q, Z w_k + b_k, Z w_v + b_v; softmax(Q_h K_h^T / sqrt(dk)) V_h;
 *     heads concatenated, then w_o + b_o -> U in R^{L x d_pe};
 *   SPE_j = w_red^T U + b_red                  (W_{(2n-k)->1} over the L rows).
 * Bias pointers may be NULL (zero).
 */
typedef struct aecct_spe_params {
  int32_t d_pe;                       /* width of the encoding */
  int32_t heads;                      /* heads of its attention; d_pe % heads == 0 */
  const float *w_in, *b_in;           /* [2][d_pe], [d_pe] */
  const float *w_q, *w_k, *w_v, *w_o; /* [d_pe][d_pe] each */
  const float *b_q, *b_k, *b_v, *b_o; /* [d_pe] each */
  const float *w_red;                 /* [L] */
  float b_red;
} aecct_spe_params;

/*
 * The positional table from a given spectrum (any orthonormal eigenvectors;
 * the table depends on the basis).  Runs the attention on the current HIP
 * device (fp32, exp2 on the hardware unit), synchronously; the rest on the host
 * in float64.
 *   eigvals  host double [L]; eigvecs host double [L][L], row i = eigenvector i;
 *   pos      host fp32 [L][d] out: row j = zeros in columns 0..d-d_pe-1, SPE_j
 *            in the last d_pe columns, so that with an embedding whose last d_pe
 *            columns are zero, t_j E_j + P_j is the concatenation [t_j E_j, SPE_j].
 * 1 <= L <= 4096, 1 <= heads <= d_pe <= d, d_pe % heads == 0, every value
 * finite.  Errors: INVALID_ARG, OUT_OF_MEMORY, DEVICE (no GPU, or a HIP
 * allocation, copy or launch failed).
 */
aecct_status aecct_spe_table_from_spectrum(const double *eigvals, const double *eigvecs, int32_t L,
                                           const aecct_spe_params *p, int32_t d, float *pos);

/* aecct_tanner_spectrum followed by aecct_spe_table_from_spectrum; same
 * arguments and errors. */
aecct_status aecct_spe_table(const uint8_t *H, int32_t m, int32_t n, const aecct_spe_params *p, int32_t d,
                             float *pos);

/* Release a model (NULL is a no-op).  No call may still be running on it. */
void aecct_destroy(aecct_model *model);

/* Static description of a built model (host call, no GPU work). */
typedef struct aecct_model_info {
  int32_t n, m, L, d, n_layers, heads, first_ring_heads, d_ff;
  int32_t path;              /* resolved aecct_path (never AUTO) */
  int64_t nnz_first_ring;    /* allowed (query, key) pairs of the first-ring mask */
  int64_t nnz_second_ring;   /* same for the second-ring mask (diagonal included) */
  size_t device_bytes;       /* device memory held by the model */
  int32_t attention;         /* aecct_attention (first_ring_heads reads 0 under CASA) */
  int32_t layered_attention; /* resolved aecct_layered_attention (never AUTO): how the layered
                                path runs a layer's projection and attention (reported whatever
                                path resolved) */
  int32_t act_scale_mode;    /* aecct_act_scale */
  int32_t device;            /* HIP device the model lives on */
  int32_t compute_units;     /* its compute units, and the LDS bytes one workgroup may use on it: */
  int64_t lds_bytes;         /* the persistent grids and LDS layouts are sized from these */
} aecct_model_info;
aecct_status aecct_get_info(const aecct_model *model, aecct_model_info *info);

/*
 * Bytes of device workspace aecct_decode needs for `batch` words (host call).
 * The fused path needs none (0).  Errors: INVALID_ARG.
 */
aecct_status aecct_workspace_size(const aecct_model *model, int64_t batch, size_t *bytes);

/*
 * Decode `batch` received words.
 *   y          device fp32 [batch][n], channel output y = x_s + noise (Section 3);
 *   bits       device uint8 [batch][n], 0/1 hard decisions bin(y * f);
 *   logits     device fp32 [batch][n] noise estimate f = f_theta(h(y)), or NULL;
 *   workspace  device scratch of at least aecct_workspace_size bytes (may be
 *              NULL when that size is 0); 256-byte aligned.
 * batch == 0 is a no-op.  Non-finite y is not checked.  The current HIP device
 * must be the one the model was created on.  Errors: INVALID_ARG (also for
 * another current device), WORKSPACE_TOO_SMALL, DEVICE (launch failure
 * reported by HIP).
 */
aecct_status aecct_decode(const aecct_model *model, const float *y, int64_t batch, uint8_t *bits,
                          float *logits, void *workspace, size_t workspace_bytes, void *stream);

/*
 * aecct_decode without a workspace argument and without any allocation, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments and results as aecct_decode (y, bits, logits are the
 * caller's device buffers, bits and logits bit-identical to aecct_decode's).
 * The layered path's activations live in one static 256 MiB device array per GPU, which the
 * library holds from its first model on that GPU until the process ends; the batch runs in
 * chunks of as many words as the array holds (the fused path needs none).  Every call on a GPU
 * shares that GPU's array and leaves its contents behind; no part of it has to start cleared.
 * Calls that overlap in time on one GPU (on different streams or host threads) race on the
 * array: the caller must order them.  Enqueues only; never allocates or synchronises.
 * Errors: INVALID_ARG (as aecct_decode, or another current device), WORKSPACE_TOO_SMALL (one
 * word's activations exceed 256 MiB; no shape aecct_create accepts needs that much), DEVICE
 * (the array's address could not be obtained at create, or a launch failed).
 */
aecct_status aecct_decode_static(const aecct_model *model, const float *y, int64_t batch, uint8_t *bits,
                                 float *logits, void *stream);

/*
 * Device arithmetic self-check (for tests and bring-up; decoding does not need it).  The kernels
 * compute three quantities with gfx950 instructions whose results the oracle states in IEEE
 * terms; this compares the two on the current device over every fp32 operand of the ranges the
 * kernels use and writes, per quantity, the number of operands that differ (0 on a conforming
 * device):
 *   counts[0]  the split of 2^x (softmax, Sections 3 and 4.2): v_fract_f32(x) against
 *              min(x - floor(x), 1 - 2^-24) and v_cvt_flr_i32_f32(x) against floor(x), for x in
 *              [-126, 129];
 *   counts[1]  the softmax normaliser: reciprocal plus one fused correction against the IEEE
 *              quotient 1 / s, for s in [2^-64, 2^64];
 *   counts[2]  the Eq. 2 scale 127 / alpha (0 for alpha = 0) against the IEEE quotient, for every
 *              finite alpha >= 0, denormals included.
 * counts: host uint64_t[3].  Allocates a few bytes of device memory and synchronises the device
 * (about a second of GPU time).  Errors: INVALID_ARG (NULL counts), DEVICE (no GPU, HIP failure).
 */
aecct_status aecct_check_device_arith(uint64_t *counts);

/* ------------------------------------------------------------------------------------------
 * Quantisation-aware training step (Section 6, second phase; Section 4.1 Eq. 1-3): the forward
 * pass of a model whose in-block linear maps are AAP linear layers over latent fp32 weights, the
 * loss of the multiplicative noise, and the gradients of every parameter.  No optimiser: the
 * caller applies the gradients.
 *
 * Forward, per word: the inference model's steps, with each map's ternary weights and scale
 * recomputed from its current latent weights W and factor delta (Eq. 1: gamma = the 0.5 quantile
 * of |W| with linear interpolation, evaluated in double and rounded to fp32; s = fp32(gamma
 * delta); T = RoundClip(W / fp32(s + aap_eps), -1, 1), rounding half to even), int8 absmax codes
 * per token for every map input (Eq. 2), Y = (Xhat T) s + b with Xhat = q alpha / 127 (Eq. 3),
 * and the natural-base softmax of q.k / sqrt(d_h) over the same masks as inference.
 * Loss: the mean over words and bits of BCE-with-logits(-f, z), z = [y x_s < 0]: f is the logit of
 * "the sign of y is right", as bin(y f) is the decision.
 * Backward: Eq. 1 and Eq. 2 pass gradients straight through their rounding; alpha and gamma are
 * constants of the step; delta receives the gradient of s and of the division inside Eq. 1:
 *   dW = s / (s + eps) Xhat^T dY,  d delta = gamma sum(G T) - s gamma / (s + eps)^2 sum(G W),
 * with G = Xhat^T dY; dXhat = s dY T^T.
 * fp32 throughout, deterministic (fixed reduction order).
 * ---------------------------------------------------------------------------------------- */

/* Parameters of a training step: DEVICE fp32 pointers, the layouts of aecct_weights, latent
 * weights in place of the ternary ones.  Read only. */
typedef struct aecct_train_params {
  const float *embed;                       /* [L][d] */
  const float *pos;                         /* [L][d] fixed positional rows (not trained), or NULL */
  const float *w_q, *w_k, *w_v, *w_o;       /* [N][d][d] latent weights */
  const float *w_ff1, *w_ff2;               /* [N][d][d_ff], [N][d_ff][d] */
  const float *delta;                       /* [N][6] factors of Eq. 1's scale, aecct_linear order */
  const float *b_q, *b_k, *b_v, *b_o, *b_ff1, *b_ff2;
  const float *ln1_g, *ln1_b, *ln2_g, *ln2_b;
  const float *head_w1;                     /* [d] */
  const float *head_b1;                     /* [1] */
  const float *head_wo;                     /* [L][n] */
  const float *head_bo;                     /* [n] */
} aecct_train_params;

/* Gradients: DEVICE fp32 outputs of the same shapes (every one written; no pos). */
typedef struct aecct_train_grads {
  float *embed;
  float *w_q, *w_k, *w_v, *w_o, *w_ff1, *w_ff2;
  float *delta;
  float *b_q, *b_k, *b_v, *b_o, *b_ff1, *b_ff2;
  float *ln1_g, *ln1_b, *ln2_g, *ln2_b;
  float *head_w1, *head_b1, *head_wo, *head_bo;
} aecct_train_grads;

typedef struct aecct_trainer aecct_trainer;   /* opaque: the code's masks on the current device */

/* Host H [m][n] as for aecct_create; d, n_layers, heads and the options first_ring_heads, d_ff,
 * ln_eps and attention as there (path and layered_attention are ignored); act_scale_mode must be
 * TOKEN.  aap_eps: the epsilon of Eq. 1, finite and >= 0.  Shapes as aecct_create.  Errors:
 * INVALID_ARG, UNSUPPORTED, OUT_OF_MEMORY, DEVICE. */
aecct_status aecct_train_create(const uint8_t *H, int32_t m, int32_t n, int32_t d, int32_t n_layers, int32_t heads,
                                const aecct_options *opt, float aap_eps, aecct_trainer **out);
/* Device workspace bytes of a step on `batch` words (host call). */
aecct_status aecct_train_workspace_size(const aecct_trainer *tr, int64_t batch, size_t *bytes);
/* One step on `batch` >= 1 words: y device fp32 [batch][n] channel outputs; xs device fp32
 * [batch][n] transmitted +-1 words, or NULL for the all-zero codeword (the paper's training
 * data); loss device fp32 [1]; grads written; workspace as sized above.  Asynchronous on stream,
 * never allocates.  The current device must be the trainer's.  Errors: INVALID_ARG,
 * WORKSPACE_TOO_SMALL, DEVICE. */
aecct_status aecct_train_grad(const aecct_trainer *tr, const aecct_train_params *params, const float *y,
                              const float *xs, int64_t batch, const aecct_train_grads *grads, float *loss,
                              void *workspace, size_t workspace_bytes, void *stream);
void aecct_train_destroy(aecct_trainer *tr);

/* Human-readable name of a status code (static string). */
const char *aecct_status_string(aecct_status status);

/* ------------------------------------------------------------------------------------------
 * Stage entry points: the steps of the layered path, one launch each, on
 * caller-provided device buffers of `words` whole words (rows = words * L).
 * aecct_decode(path = LAYERED) is exactly embed, then per layer qkv ->
 * attention -> oproj_ln -> ffn1 -> ffn2_ln, then head.  They let a caller run, time or
 * check one step on inputs of its choice.  Layout of every activation: row r
 * of word b at index b * L + r, features contiguous.  The current device must be
 * the model's.  Errors: INVALID_ARG; UNSUPPORTED from the steps that quantise
 * (embed, attention, oproj_ln, ffn1, ffn2_ln) on a model with one alpha per
 * word, where a row's codes depend on the whole word.
 * ---------------------------------------------------------------------------------------- */

/* Section 3 pre-processing + embedding + Eq. 2 quantisation of layer 0's input.
 * y [words][n] -> x fp32 [rows][d], xq int8 [rows][d], ax fp32 [rows]. */
aecct_status aecct_stage_embed(const aecct_model *model, const float *y, int64_t words, float *x,
                               int8_t *xq, float *ax, void *stream);

/* Eq. 3 for the query, key and value maps of `layer`:
 * xq, ax -> qkv fp32 [rows][3d] (Q | K | V per row). */
aecct_status aecct_stage_qkv(const aecct_model *model, int32_t layer, const int8_t *xq,
                             const float *ax, int64_t words, float *qkv, void *stream);

/* Section 4.2 head-partitioned attention and Eq. 2 quantisation of its output:
 * qkv -> oq int8 [rows][d], ao fp32 [rows]; o fp32 [rows][d] also written when non-NULL. */
aecct_status aecct_stage_attention(const aecct_model *model, const float *qkv, int64_t words,
                                   float *o, int8_t *oq, float *ao, void *stream);

/* Output projection (Eq. 3), residual and LN1 (Post-LN, Section 6), then Eq. 2:
 * oq, ao, x -> x1 fp32 [rows][d], x1q int8 [rows][d], a1 fp32 [rows]. */
aecct_status aecct_stage_oproj_ln(const aecct_model *model, int32_t layer, const int8_t *oq,
                                  const float *ao, const float *x, int64_t words, float *x1,
                                  int8_t *x1q, float *a1, void *stream);

/* First feed-forward map (Eq. 3), ReLU (Section 4, item 4) and Eq. 2 on the hidden row:
 * x1q, a1 -> gq int8 [rows][d_ff], ag fp32 [rows]. */
aecct_status aecct_stage_ffn1(const aecct_model *model, int32_t layer, const int8_t *x1q, const float *a1,
                              int64_t words, int8_t *gq, float *ag, void *stream);

/* Second feed-forward map (Eq. 3), residual and LN2 (Post-LN, Section 6), then Eq. 2:
 * gq, ag, x1 -> x fp32 [rows][d], xq int8 [rows][d], ax fp32 [rows]. */
aecct_status aecct_stage_ffn2_ln(const aecct_model *model, int32_t layer, const int8_t *gq, const float *ag,
                                 const float *x1, int64_t words, float *x, int8_t *xq, float *ax,
                                 void *stream);

/* Output head and hard decision (Section 3): x [rows][d], y [words][n] ->
 * bits uint8 [words][n], logits fp32 [words][n] (may be NULL). */
aecct_status aecct_stage_head(const aecct_model *model, const float *x, const float *y, int64_t words,
                              uint8_t *bits, float *logits, void *stream);

/* The int8 x ternary product of one AAP linear map alone (Eq. 3 before the
 * dequantisation): a int8 [rows][in] -> acc int32 [rows][out] exactly, for
 * matrix `kind` (aecct_linear) of `layer`.  Any rows >= 0. */
aecct_status aecct_ternary_gemm(const aecct_model *model, int32_t layer, int32_t kind, const int8_t *a,
                                int64_t rows, int32_t *acc, void *stream);

#ifdef __cplusplus
}
#endif
#endif
