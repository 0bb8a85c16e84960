/*
 * sdattn.h -- C ABI of libsdattn, the attention of Stable Diffusion 1.4's
 * UNet transformer blocks as hand-written HIP kernels for AMD MI355X (gfx950).
 *
 * The operation is the one stated in Sec. 3.2.1 ("Partially Fused Softmax")
 * of "Speed Is All You Need: On-Device Acceleration of Large Diffusion Models
 * via GPU-Aware Optimizations" (Chen et al., 2023):
 *
 *   Eq. 3   Attention(Q, K, V) = softmax(Q K^T / sqrt(d)) V,
 *           Q in R^{N x d}, K, V in R^{M x d}
 *   Eq. 4   L = [max_j a_ij],  S = [sum_j exp(a_ij - max_k a_ik)]   for A = Q K^T / sqrt(d)
 *
 * followed by the element-wise normalisation exp(a_ij - L_i) / S_i.  Here N is
 * Lq (latent tokens), M is Lk (latent tokens for self-attention, text tokens
 * for cross-attention) and d is D, applied independently to each of B*H
 * (batch, head) pairs.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.    Every tensor argument is a device pointer owned by the caller.
 *            The library allocates nothing, frees nothing and keeps no state
 *            beyond a thread-local copy of the last HIP error.
 * Layout.    Dense row-major, innermost dimension last, no strides.
 * Streams.   `stream` is a hipStream_t (NULL = the default stream).  Work is
 *            enqueued on it and the call returns at once; a fault on the
 *            device shows up at the caller's next synchronisation.
 * Errors.    Arguments are checked before anything is enqueued.  On any
 *            nonzero status nothing was launched and no output was written.
 * Values.    Inputs are not scanned: NaN or Inf inputs give unspecified
 *            (NaN/Inf) outputs.
 * Rounding.  fp16/bf16 inputs, fp32 accumulation, probabilities rounded to
 *            the input type before the product with V, outputs rounded to
 *            nearest even.
 */
#ifndef SDATTN_H
#define SDATTN_H

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SDATTN_OK = 0,
    SDATTN_ERR_INVALID_ARG = 1,  /* NULL pointer, size < 1, non-finite scale, overlap, bad dtype */
    SDATTN_ERR_UNSUPPORTED = 2,  /* D not a multiple of 8, D > 256, or a grid too large */
    SDATTN_ERR_MISALIGNED = 3,   /* a pointer is not aligned as documented */
    SDATTN_ERR_HIP = 4,          /* a HIP runtime call failed; see sdattn_last_hip_error() */
    SDATTN_ERR_SCRATCH = 5       /* more workspace than SDATTN_STATIC_SCRATCH_BYTES */
} sdattn_status;

typedef enum {
    SDATTN_F16 = 0,              /* IEEE binary16 */
    SDATTN_BF16 = 1,             /* bfloat16 */
    SDATTN_F32 = 2               /* IEEE binary32 (logit matrices only) */
} sdattn_dtype;

/*
 * Eq. 3 for fp16 tensors.
 *
 *   q   [B, H, Lq, D] fp16     queries
 *   k   [B, H, Lk, D] fp16     keys
 *   v   [B, H, Lk, D] fp16     values
 *   out [B, H, Lq, D] fp16     out[b,h,i,:] = sum_j softmax_j(scale * q_i . k_j) v_j
 *
 * scale multiplies every logit; SD uses 1/sqrt(D) with the true head width
 * (any finite value is accepted, including 0 and negative values).
 * Requirements: q, k, v, out 16-byte aligned; B, H, Lq, Lk >= 1;
 * 8 <= D <= 256 with D % 8 == 0; out must not overlap q, k or v.
 * Returns an sdattn_status.
 */
int sdattn_forward(const void *q, const void *k, const void *v, void *out,
                   int B, int H, int Lq, int Lk, int D, float scale, void *stream);

/*
 * sdattn_forward for fp16 or bf16 (`dtype`, all four tensors alike), with an
 * optional per-row output of Eq. 4's statistics:
 *
 *   ls  NULL, or fp32 [B, H, Lq, 2]: ls[..., 0] = L_i = max_j scale * q_i . k_j,
 *       ls[..., 1] = S_i = sum_j exp(scale * q_i . k_j - L_i) (S_i >= 1).
 *       8-byte aligned, must not overlap any other argument.
 *
 * SDATTN_F32 is rejected with SDATTN_ERR_UNSUPPORTED.
 */
int sdattn_forward_ex(const void *q, const void *k, const void *v, void *out, float *ls,
                      int B, int H, int Lq, int Lk, int D, float scale,
                      sdattn_dtype dtype, void *stream);

/*
 * The reduction step of Eq. 4 (and, optionally, the element-wise step) on a
 * given matrix, as one kernel launch with a multi-stage (block-wise) reduction
 * of each row (Sec. 3.2.1, the paragraph after Eq. 4).
 *
 *   a   [rows, cols] of `dtype` (fp16, bf16 or fp32), with a_rj = scale * a[r, j]
 *   ls  fp32 [rows, 2]: ls[r, 0] = L_r = max_j a_rj, ls[r, 1] = S_r = sum_j exp(a_rj - L_r)
 *   p   NULL, or [rows, cols] of `dtype`: p[r, j] = exp(a_rj - L_r) / S_r
 *
 * Requirements: a and p 16-byte aligned, ls 8-byte aligned; rows, cols >= 1;
 * rows * cols < 2^62; no output may overlap another argument; finite scale.
 */
int sdattn_softmax_rows(const void *a, float *ls, void *p, long long rows, long long cols,
                        float scale, sdattn_dtype dtype, void *stream);

/*
 * The partially fused softmax of Sec. 3.2.1 as separate launches: the logit
 * matrix A = scale Q K^T is written to memory, Eq. 4's (L, S) is taken per
 * row with sdattn_softmax_rows (A viewed as [B*H*Lq, Lk], scale 1), and the
 * element-wise normalisation exp(a_ij - L_i) / S_i is fused with the product
 * by V.  The three calls compute Eq. 3 (the rounding of A aside) and let the
 * caller compare the method with the single-pass sdattn_forward.
 *
 * Logits:
 *   q   [B, H, Lq, D] of `dtype` (fp16 or bf16)
 *   k   [B, H, Lk, D] of `dtype`
 *   a   [B, H, Lq, Lk] of `a_dtype` (fp16, bf16 or fp32):
 *       a[b,h,i,j] = scale * q_i . k_j, accumulated in fp32, rounded to nearest even
 *
 * Requirements: q, k, a 16-byte aligned; B, H, Lq, Lk >= 1; 8 <= D <= 256
 * with D % 8 == 0; finite scale; a must not overlap q or k.
 */
int sdattn_logits(const void *q, const void *k, void *a, int B, int H, int Lq, int Lk, int D,
                  float scale, sdattn_dtype dtype, sdattn_dtype a_dtype, void *stream);

/*
 * Normalise and multiply by V:
 *   a   [B, H, Lq, Lk] of `a_dtype` (fp16, bf16 or fp32), the scale already applied
 *   ls  fp32 [B, H, Lq, 2]: (L_i, S_i) of each row of a, as sdattn_softmax_rows writes them
 *   v   [B, H, Lk, D] of `dtype` (fp16 or bf16)
 *   out [B, H, Lq, D] of `dtype`: out[b,h,i,:] = sum_j exp(a_ij - L_i) / S_i * v_j
 *
 * p = exp(a_ij - L_i) is rounded to `dtype` before the product with V, as in
 * sdattn_forward; S_i is used as given.  Requirements: a, v, out 16-byte
 * aligned, ls 8-byte aligned; sizes as for sdattn_logits; out must not
 * overlap a, ls or v.  Fastest when Lk % 8 == 0.
 */
int sdattn_softmax_pv(const void *a, const float *ls, const void *v, void *out, int B, int H,
                      int Lq, int Lk, int D, sdattn_dtype a_dtype, sdattn_dtype dtype,
                      void *stream);

/*
 * The steps either side of Eq. 3 in SD's transformer blocks: the Q, K, V and
 * output projections, and the split of their channels into heads.  A tensor
 * of token rows (B batches x L tokens, C channels) is stored in one of two
 * layouts:
 *   SDATTN_ROWS   [B, L, C]
 *   SDATTN_HEADS  [B, H, L, C/H]: channel c = h*(C/H) + d of token l at
 *                 ((b*H + h)*L + l)*(C/H) + d -- the layout the attention
 *                 entry points take, so a projection written in it is the
 *                 head split, and one read from it is the head merge.
 */
typedef enum {
    SDATTN_ROWS = 0,
    SDATTN_HEADS = 1
} sdattn_layout;

/*
 * Linear layer with weights stored [out, in]:
 *   y[m, n] = sum_k x[m, k] * w[n, k] + bias[n]     for the B*L token rows m = b*L + l
 *
 *   x     token rows of K channels in `x_layout`, `dtype` (fp16 or bf16)
 *   w     [N, K] of `dtype`; bias [N] of `dtype` or NULL
 *   y     token rows of N channels in `y_layout`, `dtype`, accumulated in fp32
 *         and rounded to nearest even
 *   H     heads of a SDATTN_HEADS side (ignored when neither side uses it)
 *
 * Requirements: x, w, y 16-byte aligned, bias 8-byte aligned; B, L, K, N >= 1;
 * K and N multiples of 8, at most 65536; on a SDATTN_HEADS side H >= 1 divides that side's channels into
 * widths that are multiples of 8; y must not overlap x, w or bias.
 */
int sdattn_linear(const void *x, const void *w, const void *bias, void *y, int B, int L, int K,
                  int N, int H, sdattn_layout x_layout, sdattn_layout y_layout, sdattn_dtype dtype,
                  void *stream);

/*
 * SD's attention block around Eq. 3 (multi-head attention of latent tokens x
 * over context tokens ctx; ctx = x for self-attention):
 *   Q = x wq^T, K = ctx wk^T, V = ctx wv^T, split into H heads of D = C/H;
 *   O_h = softmax(scale Q_h K_h^T) V_h;  out = [O_0 | ... | O_{H-1}] wo^T + bo
 *
 *   x [B, Lq, C], ctx [B, Lk, Cc], out [B, Lq, C]; wq, wo [C, C]; wk, wv [C, Cc];
 *   bo [C] or NULL; all of `dtype`.
 *   workspace: device memory of at least sdattn_attention_block_workspace(B, Lq, Lk, C)
 *   bytes, 16-byte aligned, owned by the caller; it receives Q, K, V and O
 *   (with Lk = 0 the size covers Q and O only, as sdattn_attention_block_kv needs).
 *
 * Three launches on `stream`: the Q, K and V projections together (heads
 * layout out), the attention forward (writing O with the heads merged, as
 * [B, Lq, C]), and the output projection.  Requirements: those of sdattn_linear for each projection and of
 * sdattn_forward_ex for the attention (D % 8 == 0, D <= 256); no argument may
 * overlap out or the workspace.
 */
long long sdattn_attention_block_workspace(int B, int Lq, int Lk, int C);
int sdattn_attention_block(const void *x, const void *ctx, const void *wq, const void *wk,
                           const void *wv, const void *wo, const void *bo, void *out,
                           void *workspace, long long workspace_bytes, int B, int Lq, int Lk,
                           int C, int Cc, int H, float scale, sdattn_dtype dtype, void *stream);

/*
 * sdattn_attention_block without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc): Q, K, V and O go through a static scratch
 * of SDATTN_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs
 * on until the process ends.  The call allocates nothing; its first call on a
 * device looks up that device's scratch address (no launch).
 *
 * Arguments as for sdattn_attention_block, minus the workspace; the scratch
 * belongs to the current device, so `stream` must belong to it too.
 * Returns SDATTN_ERR_SCRATCH, before any HIP call, when
 * sdattn_attention_block_workspace(B, Lq, Lk, C) exceeds the scratch (every
 * SD1.4 block at B = 2 fits: 21 MB at the 64x64 level).  Every call on one
 * GPU shares that GPU's scratch: calls that may overlap on one GPU (other
 * streams, other host threads) race and must be ordered by the caller.
 */
#define SDATTN_STATIC_SCRATCH_BYTES (32LL << 20)
int sdattn_attention_block_static(const void *x, const void *ctx, const void *wq, const void *wk,
                                  const void *wv, const void *wo, const void *bo, void *out, int B,
                                  int Lq, int Lk, int C, int Cc, int H, float scale,
                                  sdattn_dtype dtype, void *stream);

/*
 * The context side of a cross-attention block: K = ctx wk^T and V = ctx wv^T,
 * written split into H heads (SDATTN_HEADS layout, [B, H, Lk, C/H]).  The text
 * context is the same at every denoising step (Sec. 3, denoising network), so
 * a caller computes K and V once per prompt and hands them to
 * sdattn_attention_block_kv at each step.  One launch on `stream`.
 *
 *   ctx [B, Lk, Cc]; wk, wv [C, Cc]; k, v [B, H, Lk, C/H]; all of `dtype`.
 * Requirements: those of sdattn_linear for both products; k and v must not
 * overlap each other, ctx or the weights.
 */
int sdattn_project_kv(const void *ctx, const void *wk, const void *wv, void *k, void *v, int B,
                      int Lk, int Cc, int C, int H, sdattn_dtype dtype, void *stream);

/*
 * sdattn_attention_block with K and V given (from sdattn_project_kv):
 *   Q = x wq^T split into H heads; O_h = softmax(scale Q_h K_h^T) V_h;
 *   out = [O_0 | ... | O_{H-1}] wo^T + bo
 *
 *   x, out [B, Lq, C]; wq, wo [C, C]; k, v [B, H, Lk, C/H]; bo [C] or NULL.
 *   workspace: at least sdattn_attention_block_workspace(B, Lq, 0, C) bytes,
 *   16-byte aligned; it receives Q and O.
 * Three launches on `stream` (Q projection, attention, output projection);
 * requirements as for sdattn_attention_block.
 */
int sdattn_attention_block_kv(const void *x, const void *wq, const void *k, const void *v,
                              const void *wo, const void *bo, void *out, void *workspace,
                              long long workspace_bytes, int B, int Lq, int Lk, int C, int H,
                              float scale, sdattn_dtype dtype, void *stream);

/*
 * Group normalisation, Sec. 3.1 Eq. 1, in one launch with no intermediate
 * tensor, with the epsilon and per-channel affine terms of the networks that
 * use it (Eq. 1 itself is eps = 0, gamma = NULL, beta = NULL):
 *   y = (x - mu_g) / sqrt(var_g + eps) * gamma_c + beta_c
 * over feature maps x [B, C, HW] (channel-major: the C channels of batch b,
 * each a contiguous run of HW pixels); group g is channels g*C/G ..
 * (g+1)*C/G - 1, mu_g and var_g its mean and mean square deviation
 * (population variance).  fp32 arithmetic, output rounded to nearest even.
 *
 *   x, y [B, C, HW] of `dtype` (fp16 or bf16), 16-byte aligned; y may be x
 *   (in place) but must not overlap it otherwise; gamma, beta [C] of `dtype`
 *   or NULL (for 1 and 0).  Requirements: C % G == 0; eps finite and >= 0.
 */
int sdattn_group_norm(const void *x, const void *gamma, const void *beta, void *y, int B, int C,
                      long long HW, int G, float eps, sdattn_dtype dtype, void *stream);

/*
 * GELU, Sec. 3.1 Eq. 2, fused with the split and multiply around it (the gated
 * feed-forward of the transformer block):
 *   out[m, f] = h[m, f] * GELU(h[m, F + f]),  GELU(x) = x/2 (1 + erf(x / sqrt 2))
 * for h [M, 2F] (value half, then gate half) -> out [M, F]; fp32 arithmetic
 * (erf to within 3e-7), output rounded to nearest even.
 *
 *   h, out of `dtype` (fp16 or bf16), 16-byte aligned, not overlapping;
 *   F % 8 == 0.
 */
int sdattn_geglu(const void *h, void *out, long long M, int F, sdattn_dtype dtype, void *stream);

/*
 * 3x3 convolution, stride 1, zero padding 1, by Winograd's F(4x4, 3x3)
 * algorithm (Sec. 3.3, the 4x4 tile of Table 2):
 *   y[b, o, i, j] = bias[o] + sum_{c, u, v} w[o, c, u, v] x[b, c, i + u - 1, j + v - 1]
 * on channel-major maps x [B, Ci, H, W] -> y [B, Co, H, W].
 *
 * sdattn_winograd_weights transforms the kernels w [Co, Ci, 3, 3] once per
 * layer into u [36, Co, Ci] (sdattn_winograd_weights_elems(Co, Ci) elements,
 * 4x the kernels, Table 2's weight factor; u 16-byte aligned).
 * sdattn_conv3x3 then runs the input transform, 36 matrix products on the
 * matrix cores and the output transform (three launches on `stream`) through
 * a caller-owned workspace of sdattn_conv3x3_workspace(B, Ci, Co, H, W) bytes
 * (the transformed input, 2.25x the input -- Table 2's tensor factor -- and
 * the 36 products).  The transformed values are stored in `dtype` (fp16 or
 * bf16) with fp32 arithmetic inside each step, so the error exceeds a direct
 * convolution's by the transforms' growth (tested bound in the tests).
 *
 * Requirements: Ci and Co multiples of 8, at most 65536; H*W at most 2^25;
 * x, u, y, workspace
 * 16-byte aligned; bias [Co] of `dtype` or NULL; y must not overlap any input
 * or the workspace, nor the workspace an input.
 */
long long sdattn_winograd_weights_elems(int Co, int Ci);
int sdattn_winograd_weights(const void *w, void *u, int Co, int Ci, sdattn_dtype dtype,
                            void *stream);
long long sdattn_conv3x3_workspace(int B, int Ci, int Co, int H, int W);
int sdattn_conv3x3(const void *x, const void *u, const void *bias, void *y, void *workspace,
                   long long workspace_bytes, int B, int Ci, int Co, int H, int W,
                   sdattn_dtype dtype, void *stream);

/* Static English text for a status code (never NULL). */
const char *sdattn_status_str(int status);

/* hipError_t of the last failed HIP call on this thread (0 if none). */
int sdattn_last_hip_error(void);

/* Static version string of the library. */
const char *sdattn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SDATTN_H */
