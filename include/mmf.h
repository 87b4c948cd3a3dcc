/*
 * mmf.h -- C ABI of the MI355X (gfx950) fused BitLinear library.
 *
 * The library computes the forward pass of the BitLinear layer of "Scalable
 * MatMul-free Language Modeling" (arXiv 2406.02528): RMSNorm of each token,
 * per-token absmax int8 quantisation, ternary accumulation against weights in
 * {-1, 0, +1} with int32 sums, and dequantisation by the activation and weight
 * scales (Algorithm 1, "Fused RMSNorm and BitLinear Algorithm with
 * Quantization", forward_pass with bias 0; Sec. "MatMul-free Dense Layers with
 * Ternary Weights" for the ternary sum).
 *
 * Conventions for every entry point
 *  - Array arguments are DEVICE pointers on the current HIP device, owned by
 *    the caller; the library keeps no pointer after a call returns.
 *  - Work is enqueued on `stream` (NULL = the null stream) and is
 *    asynchronous: results are valid once the stream has been synchronised.
 *    No entry point synchronises the device.
 *  - Arguments are checked on the host before anything is enqueued; on any
 *    error nothing is enqueued and no output is touched.
 *  - Every pointer to an array must be 16-byte aligned (MMF_ERR_ALIGN).
 *  - K (in-features) must be a positive multiple of 16 and at most 2^20
 *    (MMF_ERR_SHAPE); M (tokens) and N (out-features) may be any value in
 *    [0, 2^31 - 1]; M == 0 or N == 0 is a successful no-op.  A call whose
 *    shape the contraction kernel it would run cannot address with its
 *    32-bit offsets returns MMF_ERR_SHAPE before anything is enqueued: the
 *    int8 MFMA kernel needs (K/16) * N * 4 < 2^31, N <= 2^24 and row slices
 *    of at least 256 tokens whose q and output stay below 2^31 bytes (so
 *    N < 2^21); the decode kernel needs (K/16 + 8) * N * 4 < 2^32.
 *  - Entry points with an `x_is_f32` argument take 0 (bfloat16 x) or 1
 *    (float32 x); any other value returns MMF_ERR_DTYPE.
 *  - Outputs must not alias inputs.
 *  - Calls on different streams may run concurrently.
 *  - Return value: an mmf_status code.
 *
 * Shapes and layouts (row-major, sizes in elements)
 *  - x        [M][K]  activations, bfloat16 (uint16 bit patterns) or float32
 *                     for the _f32 variants.
 *  - gamma    [K]     float32 RMSNorm scale; NULL means all ones.
 *  - W        [N][K]  float32 latent weights (out x in).
 *  - Wpacked  [K/16][N] uint32 ternary weights, 2 bits each (see below).
 *  - w_scale  [1]     float32 weight dequantisation multiplier, mean|W|.
 *  - q        [M][K]  int8 quantised activations.
 *  - a_scale  [M]     float32 per-token dequantisation multiplier, absmax/127.
 *  - q_rowsum [M]     int32 sum over k of q[m][k].
 *  - y        [M][N]  float32 output.
 *
 * Packed weight format.  Word (j, n) = Wpacked[j * N + n] holds the ternary
 * weights t[n][16j .. 16j + 15].  For k = 16j + 4i + b (i, b in 0..3) the code
 * c = t + 1 in {0, 1, 2} sits in bits 8b + 2i and 8b + 2i + 1, so that
 * (word >> 2i) & 0x03030303 holds the codes of k = 16j + 4i .. 16j + 4i + 3 in
 * byte order.  A word of zero weights is 0x55555555.  Code 3 never appears in
 * what mmf_ternarize_weights writes; a word containing it gives an
 * unspecified (memory-safe) result.
 */
#ifndef MMF_H
#define MMF_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define MMF_OK 0
#define MMF_ERR_NULL 1      /* a required pointer is NULL                      */
#define MMF_ERR_SHAPE 2     /* a size is out of range (K % 16, K == 0, a       */
                            /* shape past a kernel's 32-bit offsets, ...)      */
#define MMF_ERR_ALIGN 3     /* an array pointer is not 16-byte aligned         */
#define MMF_ERR_DTYPE 4     /* an activation dtype selector is not 0 or 1      */
#define MMF_ERR_HIP 5       /* a HIP runtime call or a kernel launch failed    */
#define MMF_ERR_WORKSPACE 6 /* the caller's workspace is too small or          */
                            /* misaligned                                      */
#define MMF_ERR_ARG 7       /* another argument is invalid (e.g. path value)   */

/* Activation dtype selector of the entry points that take either form
 * (the `x_is_f32` arguments below). */
#define MMF_DTYPE_BF16 0
#define MMF_DTYPE_F32 1

/* Human-readable name of a status code (static storage; never NULL). */
const char *mmf_status_string(int status);

/* Library ABI version, incremented on any incompatible change. */
int mmf_version(void);

/* Bytes of the packed weight array for N out-features and K in-features,
 * (K / 16) * N * 4.  Returns 0 for invalid shapes. */
size_t mmf_packed_weight_bytes(int64_t N, int64_t K);

/*
 * Weight ternarisation and packing (Algorithm 1, weight_quant; offline, once
 * per weight tensor).
 *   w_scale = max(mean over all N*K entries of |W|, 1e-5), the mean summed in
 *             fp64 and rounded to fp32;
 *   t[n][k] = clamp(round_half_even(W[n][k] * (1 / w_scale)), -1, 1), the
 *             reciprocal and product in fp32;
 * written to Wpacked in the format above and to w_scale[0].
 * W: [N][K] float32 in; Wpacked: [K/16][N] uint32 out; w_scale: 1 float out.
 * Allocates a small stream-ordered scratch buffer (hipMallocAsync).
 */
int mmf_ternarize_weights(const float *W, int64_t N, int64_t K,
                          uint32_t *Wpacked, float *w_scale, hipStream_t stream);

/*
 * Fused RMSNorm + per-token absmax int8 quantisation (Algorithm 1,
 * rms_norm_fwd and activation_quant; RMSNorm with the mean of squares,
 * eps = 1e-6, learned scale gamma, as in the RMSNorm equation of the
 * Loihi-methods section).  For each token m:
 *   r        = fp32(1 / sqrt(sum_k x^2 / K + 1e-6))      (sum and root in fp64)
 *   y_k      = (x_k * r) * gamma_k                         (fp32)
 *   a        = max(max_k |y_k|, 1e-5)
 *   q_k      = clamp(round_half_even(y_k * (127 / a)), -128, 127)
 *   a_scale  = a / 127,   q_rowsum = sum_k q_k.
 * x: [M][K] bf16 bits; gamma: [K] or NULL; q: [M][K] out; a_scale: [M] out.
 */
int mmf_act_quant(const uint16_t *x, const float *gamma, int8_t *q,
                  float *a_scale, int64_t M, int64_t K, hipStream_t stream);
/* The same for float32 activations. */
int mmf_act_quant_f32(const float *x, const float *gamma, int8_t *q,
                      float *a_scale, int64_t M, int64_t K, hipStream_t stream);
/* The same with the activation dtype as an argument (x_is_f32: 0 = bf16,
 * 1 = float32, else MMF_ERR_DTYPE) and the row sums q_rowsum [M] (int32,
 * may be NULL) that the contraction-stage entry points below take. */
int mmf_act_quant_ex(const void *x, int x_is_f32, const float *gamma, int8_t *q,
                     float *a_scale, int32_t *q_rowsum, int64_t M, int64_t K,
                     hipStream_t stream);

/*
 * The fused BitLinear forward (Algorithm 1, forward_pass, bias 0):
 *   y[m][n] = a_scale[m] * w_scale * sum_k q[m][k] t[n][k]
 * with q, a_scale from the act-quant step above and t from Wpacked.  The
 * integer sum is exact; the product is fp32 (a_scale[m] * w_scale first).
 * Up to 32 tokens (K <= 2048) or 64 (larger K) take the decode kernel in
 * launches of at most 16 tokens (16x16x64 int8 MFMA over 16 columns by the
 * token rows; weights streamed once per launch), larger M the int8 MFMA GEMM
 * kernel.  Allocates its M*K + 8*M byte scratch stream-ordered
 * (hipMallocAsync); mmf_bitlinear_fwd_ws takes caller scratch instead.
 * x: [M][K] bf16 bits; gamma: [K] or NULL; Wpacked: [K/16][N]; w_scale: [1];
 * y: [M][N] float32 out.
 */
int mmf_bitlinear_fwd(const uint16_t *x, const float *gamma,
                      const uint32_t *Wpacked, const float *w_scale, float *y,
                      int64_t M, int64_t K, int64_t N, hipStream_t stream);
/* The same for float32 activations. */
int mmf_bitlinear_fwd_f32(const float *x, const float *gamma,
                          const uint32_t *Wpacked, const float *w_scale,
                          float *y, int64_t M, int64_t K, int64_t N,
                          hipStream_t stream);

/* Bytes of caller scratch the _ws variants need for M tokens of K features. */
size_t mmf_bitlinear_workspace_bytes(int64_t M, int64_t K);

/* mmf_bitlinear_fwd with caller-provided scratch `workspace` of
 * `workspace_bytes` bytes (device memory, 256-byte aligned, at least
 * mmf_bitlinear_workspace_bytes(M, K); MMF_ERR_WORKSPACE otherwise).  The
 * scratch must not be used by other work on another stream meanwhile.
 * x_is_f32 selects float32 (1) or bf16 (0) activations. */
int mmf_bitlinear_fwd_ws(const void *x, int x_is_f32, const float *gamma,
                         const uint32_t *Wpacked, const float *w_scale,
                         float *y, int64_t M, int64_t K, int64_t N,
                         void *workspace, size_t workspace_bytes,
                         hipStream_t stream);

/*
 * mmf_bitlinear_fwd for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and results as mmf_bitlinear_fwd_ws, with the
 * scratch (q, a_scale, q_rowsum: mmf_bitlinear_workspace_bytes(M, K) bytes)
 * in a static device array of mmf_bitlinear_noalloc_max_bytes() = 64 MiB
 * that each GPU the library runs on holds until the process ends.  No call
 * allocates or frees memory; the array's address is looked up once per
 * device, on the first call there.  Calls that need more scratch than the
 * array holds return MMF_ERR_WORKSPACE before anything is enqueued (the
 * fused decode kernel, up to 32 tokens at K <= 2048 and 64 beyond, needs
 * none).  Every call on a GPU shares that
 * GPU's array: calls that overlap on one GPU (on different streams, or from
 * different host threads) race; serialise them.  The array keeps the last
 * call's contents, which every call overwrites before reading.
 * x_is_f32: 0 = bf16 x, 1 = float32 x (MMF_ERR_DTYPE otherwise).
 */
size_t mmf_bitlinear_noalloc_max_bytes(void);
int mmf_bitlinear_fwd_noalloc(const void *x, int x_is_f32, const float *gamma,
                              const uint32_t *Wpacked, const float *w_scale,
                              float *y, int64_t M, int64_t K, int64_t N,
                              hipStream_t stream);

/*
 * Ternary accumulation and dequantisation from already-quantised activations
 * (the contraction stage of the forward on its own; Sec. "MatMul-free Dense
 * Layers with Ternary Weights" and Algorithm 1):
 *   y[m][n] = (q_rowsum-corrected int32 sum_k q[m][k] t[n][k]) * (a_scale[m] * w_scale)
 * q: [M][K]; a_scale: [M]; q_rowsum: [M] = sum_k q[m][k] (as written by
 * mmf_act_quant; a wrong value shifts every output of that row);
 * Wpacked: [K/16][N]; w_scale: [1]; y: [M][N] out.  Allocates nothing.
 */
int mmf_ternary_gemm_dequant(const int8_t *q, const float *a_scale,
                             const int32_t *q_rowsum, const uint32_t *Wpacked,
                             const float *w_scale, float *y, int64_t M,
                             int64_t K, int64_t N, hipStream_t stream);

/*
 * Raw ternary accumulation, acc[m][n] = sum_{k: t=+1} q[m][k] -
 * sum_{k: t=-1} q[m][k], exact int32 (Sec. "MatMul-free Dense Layers with
 * Ternary Weights").  Runs the same contraction kernels as the forward, with
 * an integer epilogue.  q: [M][K]; Wpacked: [K/16][N]; acc: [M][N] int32 out.
 * Allocates a 4*M byte stream-ordered scratch buffer (hipMallocAsync).
 */
int mmf_ternary_gemm_i32(const int8_t *q, const uint32_t *Wpacked,
                         int32_t *acc, int64_t M, int64_t K, int64_t N,
                         hipStream_t stream);

/*
 * GLU channel mixer, up-projections and gate (Sec. "MatMul-free Channel
 * Mixer": g = x (*) W_g, u = x (*) W_u, p = SiLU(g) (.) u, SiLU(v) =
 * v / (1 + e^-v)), fused into one contraction.
 *
 * Both projections see the same RMSNorm (one gamma) and the same int8
 * activations, as the concatenated gate|up projection of the BitLinear above;
 * each keeps its own weight scale.  For token m and channel i:
 *   g = fp32(acc_g) * (a_scale[m] * w_scales[0])     (as y of mmf_bitlinear_fwd)
 *   u = fp32(acc_u) * (a_scale[m] * w_scales[1])
 * with acc_g, acc_u the exact ternary sums of the gate and up channel i.
 *   p[m][i] = (g * s) * u,  s = 1 / (1 + e^-g)           (fp32)
 * with s from the hardware base-2 exponential and reciprocal, e^-g taken as
 * 2^(-g log2 e) (1 ulp each; the rounded argument adds about |g| u of
 * relative error for large |g|, u = 2^-24).
 *
 * mmf_glu_pack interleaves the packed gate and up projections, [K/16][L]
 * words each (as written by mmf_ternarize_weights for [L][K] latent
 * weights), into Wgu_packed [K/16][2L]: blocks of 16 columns, gate channels
 * 16b .. 16b + 15, then the up channels with the same indices, in turn.
 * L must be a multiple of 16 (MMF_ERR_SHAPE otherwise).
 *
 * mmf_glu_fwd: x [M][K] bf16 bits (mmf_glu_fwd_f32: float32); gamma [K] or
 * NULL; Wgu_packed [K/16][2L] from mmf_glu_pack; w_scales [2] = gate, up;
 * p [M][L] float32 out.  Up to 32 tokens (K <= 2048) or 64 (larger K) run
 * the fused decode kernel with the same SiLU(g) * u epilogue (launches of at
 * most 16 tokens; the result is bit-identical to the GEMM kernel's), larger M
 * the int8 MFMA GEMM kernel.  Allocates the
 * same stream-ordered scratch as mmf_bitlinear_fwd; mmf_glu_fwd_ws takes
 * caller scratch of mmf_bitlinear_workspace_bytes(M, K) bytes instead.
 */
int mmf_glu_pack(const uint32_t *Wg_packed, const uint32_t *Wu_packed, int64_t L,
                 int64_t K, uint32_t *Wgu_packed, hipStream_t stream);
int mmf_glu_fwd(const uint16_t *x, const float *gamma, const uint32_t *Wgu_packed,
                const float *w_scales, float *p, int64_t M, int64_t K, int64_t L,
                hipStream_t stream);
int mmf_glu_fwd_f32(const float *x, const float *gamma, const uint32_t *Wgu_packed,
                    const float *w_scales, float *p, int64_t M, int64_t K, int64_t L,
                    hipStream_t stream);
int mmf_glu_fwd_ws(const void *x, int x_is_f32, const float *gamma,
                   const uint32_t *Wgu_packed, const float *w_scales, float *p,
                   int64_t M, int64_t K, int64_t L, void *workspace,
                   size_t workspace_bytes, hipStream_t stream);
/* The contraction stage of mmf_glu_fwd on its own, from quantised
 * activations (q, a_scale, q_rowsum as written by mmf_act_quant); always the
 * int8 MFMA kernel.  Allocates nothing. */
int mmf_ternary_gemm_glu(const int8_t *q, const float *a_scale, const int32_t *q_rowsum,
                         const uint32_t *Wgu_packed, const float *w_scales, float *p,
                         int64_t M, int64_t K, int64_t L, hipStream_t stream);

/*
 * Dense layer with bias (Algorithm 1, forward_pass: the ternary product plus
 * b): y = mmf_bitlinear_fwd's output + bias[n], the add in fp32 after the
 * dequantisation:  y[m][n] = fp32(acc) * (a_scale[m] * w_scale[0]) + bias[n].
 * x [M][K] bf16 bits (x_is_f32 = 0) or float32 (x_is_f32 = 1); bias [N]
 * float32; N must be a multiple of 4 (MMF_ERR_SHAPE).  Same kernels and
 * scratch as mmf_bitlinear_fwd.
 */
int mmf_bitlinear_fwd_bias(const void *x, int x_is_f32, const float *gamma,
                           const uint32_t *Wpacked, const float *w_scale, const float *bias,
                           float *y, int64_t M, int64_t K, int64_t N, hipStream_t stream);

/*
 * MLGRU token mixer (Sec. "MatMul-free Language Model Architecture",
 * paragraph "MatMul-free Linear Gated Recurrent Unit" and its equations),
 * with (*) the BitLinear above:
 *   f_t  = lb + (1 - lb) (.) sigmoid(x_t (*) W_f + b_f)    forget gate
 *   c_t  = SiLU(x_t (*) W_c + b_c)                         candidate
 *   h_t  = f_t (.) h_{t-1} + (1 - f_t) (.) c_t             state, h_0 given or 0
 *   g_t  = x_t (*) W_g + b_g                               output gate
 *   o'_t = g_t (.) sigmoid(h_t)
 *   o_t  = o'_t (*) W_o + b_o
 * lb [d] is the forget-gate lower bound of HGRN that the paper keeps for
 * deeper layers (NULL: no bound, the equations as printed); biases may be
 * NULL (zero).
 *
 * Layout: B sequences of T tokens, token t of sequence b in row b*T + t of
 * x, fcg, o_prime and o; states h0, h_last [B][d] float32.  d must be a
 * positive multiple of 16 (MMF_ERR_SHAPE).  The three input projections are
 * one packed matrix Wfcg [K/16][3d] (columns f | c | g: mmf_ternarize_weights
 * of the stacked [3d][K] latent weights, or three packs side by side) behind
 * one RMSNorm gamma and one activation quantisation; w_scales [3] scales the
 * three column blocks (three equal values when ternarised together).
 *
 * Workspace: every MLGRU entry point takes `workspace` of at least the bytes
 * its _workspace_bytes function returns (256-byte aligned,
 * MMF_ERR_WORKSPACE), or NULL, in which case it allocates that scratch
 * stream-ordered on `stream` and frees it there.
 */

/* Input projections and gate activations: fcg [M][3d] float32 with, for
 * column n of segment s = n / d (channel i = n % d),
 *   z = fp32(acc) * (a_scale[m] * w_scales[s]) + bias[n]      (fp32)
 *   f = (1 - lb[i]) * s + lb[i],  c = z * s,  g = z,   s = 1 / (1 + e^-z)
 * with s evaluated as for the GLU gate (hardware exp2 and reciprocal). The
 * recurrence's output gate o' = g * s(h) uses the same s.
 * x [M][K] bf16 bits or float32 (x_is_f32); bias [3d] or NULL; lb [d] or
 * NULL.  M <= 32 (K <= 2048) or 64 (larger K) runs the fused decode kernel
 * (launches of at most 16 tokens), larger M the int8 MFMA GEMM kernel. */
size_t mmf_mlgru_proj_workspace_bytes(int64_t M, int64_t K, int64_t d);
int mmf_mlgru_proj(const void *x, int x_is_f32, const float *gamma, const uint32_t *Wfcg,
                   const float *w_scales, const float *bias, const float *lb, float *fcg,
                   int64_t M, int64_t K, int64_t d, void *workspace, size_t workspace_bytes,
                   hipStream_t stream);

/* The contraction stage of mmf_mlgru_proj on its own, from quantised
 * activations (q, a_scale, q_rowsum as written by mmf_act_quant); always the
 * int8 MFMA kernel.  Allocates nothing. */
int mmf_mlgru_proj_q(const int8_t *q, const float *a_scale, const int32_t *q_rowsum,
                     const uint32_t *Wfcg, const float *w_scales, const float *bias,
                     const float *lb, float *fcg, int64_t M, int64_t K, int64_t d,
                     hipStream_t stream);

/* Recurrence and output gate from fcg [B*T][3d]: o_prime [B*T][d] float32,
 * the state after the last token in h_last [B][d] (NULL: not stored).  h0
 * NULL means h_0 = 0; h_last may be the same array as h0 (the state is then
 * updated in place), no other overlap is allowed.  In fp32, token by token
 * within chunks of tokens, the chunks joined through their products of
 * forget gates. */
size_t mmf_mlgru_scan_workspace_bytes(int64_t B, int64_t T, int64_t d);
int mmf_mlgru_scan(const float *fcg, const float *h0, float *o_prime, float *h_last,
                   int64_t B, int64_t T, int64_t d, void *workspace, size_t workspace_bytes,
                   hipStream_t stream);

/* The whole mixer: mmf_mlgru_proj (K = d), mmf_mlgru_scan, then
 * mmf_bitlinear_fwd_bias of o' (float32) with gamma_o, Wo [d/16][d],
 * w_scale_o [1] and b_o [d] (NULL: zero) into o [B*T][d] float32.  The same
 * kernels as those three calls, so the results are identical to them. */
size_t mmf_mlgru_workspace_bytes(int64_t B, int64_t T, int64_t d);
int mmf_mlgru_fwd(const void *x, int x_is_f32, const float *gamma, const uint32_t *Wfcg,
                  const float *w_scales, const float *bias, const float *lb, const float *h0,
                  float *h_last, const float *gamma_o, const uint32_t *Wo,
                  const float *w_scale_o, const float *b_o, float *o, int64_t B, int64_t T,
                  int64_t d, void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Training forward (Algorithm 1, forward_pass: the latent weights are
 * quantised on every call; the RMSNorm statistic r is kept for the
 * backward).  From latent float32 weights W [N][K]:
 *   Wpacked [K/16][N], w_scale [1]   as mmf_ternarize_weights(W)
 *   q [M][K], a_scale [M], rstd [M]  as mmf_act_quant(x), rstd[m] =
 *                                    1/sqrt(mean_k x^2 + 1e-6) (float32)
 *   y [M][N]                         as mmf_bitlinear_fwd(_bias) with them
 * (bias [N] or NULL; with a bias N must be a multiple of 4).  rstd may be
 * NULL.  Every M runs the int8 MFMA kernel; K/16 * N * 4 must stay below
 * 2^31 and N at most 2^24 (MMF_ERR_SHAPE).  Wpacked, w_scale, q, a_scale
 * and rstd are what mmf_bitlinear_bwd takes.  Workspace as for the MLGRU
 * entry points (NULL: allocated stream-ordered).
 */
size_t mmf_bitlinear_train_workspace_bytes(int64_t M, int64_t K, int64_t N);
int mmf_bitlinear_train_fwd(const void *x, int x_is_f32, const float *gamma, const float *W,
                            const float *bias, float *y, uint32_t *Wpacked, float *w_scale,
                            int8_t *q, float *a_scale, float *rstd, int64_t M, int64_t K,
                            int64_t N, void *workspace, size_t workspace_bytes,
                            hipStream_t stream);

/*
 * Backward of the BitLinear (Algorithm 1, backward_pass and rms_norm_bwd;
 * the straight-through estimator of Sec. "Surrogate Gradient" passes the
 * gradient through both quantisers unchanged), in the RMSNorm reading
 * (no mean subtracted) with y = (x r) gamma:
 *   dY = dO Wt^T,  Wt = t * w_scale (the ternary weights the forward used)
 *   dx = r g - (r^3 / K) x s,  g = gamma (.) dY,  s = sum_k g_k x_k
 *   dW = dO^T Yq,  Yq = q * a_scale stored as bfloat16 (the gradient of the
 *        latent weights through the straight-through weight quantiser)
 *   db = sum over tokens of dO;  dgamma = sum over tokens of dY (.) x r
 * dO [M][N] bfloat16 bits; x [M][K] bf16 bits or float32 (x_is_f32); gamma
 * [K] or NULL (ones); rstd, q, a_scale, Wpacked, w_scale from
 * mmf_bitlinear_train_fwd.  Outputs float32: dx [M][K], dW [N][K], db [N]
 * (NULL: not computed), dgamma [K] (NULL: not computed).  The two products
 * run on the matrix cores with bf16 operands and fp32 accumulation: dY reads
 * the packed codes (re-packed once per call with the contraction index
 * inside the word) and expands them in registers, with gamma, rstd and the
 * row sums of the RMSNorm backward in its epilogue; dW reads q and a_scale
 * and forms Yq while staging them.  s, db and dgamma are summed in fp64;
 * when the dW output has few tiles its contraction over tokens is split into
 * parts added in fp64.  Shapes whose dO rows, re-packed codes or dW exceed
 * 32-bit offsets ((N + 7) / 8 * 16 * 128 bytes of dO per 128 rows, K * 4 *
 * ceil(N / 16) bytes of codes, N * K * 4 bytes of dW, each below 2^31)
 * return MMF_ERR_SHAPE.  M == 0 or N == 0 is a no-op.  Workspace as above.
 */
size_t mmf_bitlinear_bwd_workspace_bytes(int64_t M, int64_t K, int64_t N);
int mmf_bitlinear_bwd(const uint16_t *dO, const void *x, int x_is_f32, const float *gamma,
                      const float *rstd, const int8_t *q, const float *a_scale,
                      const uint32_t *Wpacked, const float *w_scale, float *dx, float *dW,
                      float *db, float *dgamma, int64_t M, int64_t K, int64_t N,
                      void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Kernel selection for the contraction: MMF_PATH_AUTO (decode kernel for
 * M <= 32 at K <= 2048 and M <= 64 beyond, in launches of at most 16
 * tokens; the GEMM kernel otherwise),
 * MMF_PATH_GEMV or MMF_PATH_GEMM force one kernel for every M (the decode
 * kernel handles at most 16 tokens per launch and is launched once per
 * 16-token slice when forced).  Process-wide; returns
 * the previous setting, or -MMF_ERR_ARG for an unknown value.
 */
#define MMF_PATH_AUTO 0
#define MMF_PATH_GEMV 1
#define MMF_PATH_GEMM 2
int mmf_set_path(int path);

/*
 * The workgroup tile of the prefill (MFMA) contraction for an M x K x N
 * problem on `cus` compute units, as the library plans it for its launches
 * (host only: no device call, nothing enqueued; for problems split into row
 * slices by the 32-bit offset limit, the first slice's plan).  For callers
 * sizing their own work and for tests that must know which kernel form a
 * shape exercises.  `epilogue` is one of MMF_EPILOGUE_*; for the GLU, N is
 * the interleaved width 2 L (a multiple of 32).  Returns one of MMF_TILE_*:
 * 128 x 512 tiles with one 8-wave workgroup per CU; the same area as two
 * 128 x 256 workgroups of 4 waves per CU (K <= 4096, not the affine
 * epilogue, more than one round of wide tiles or most of one at K <= 2048);
 * 64 x 512 or 64 x 256 tiles for problems with few wide tiles; 256 x 256
 * when N % 4 != 0.  Errors as negative status: -MMF_ERR_SHAPE for a shape the
 * contraction rejects or cus < 1, -MMF_ERR_ARG for an unknown epilogue.
 */
#define MMF_EPILOGUE_DEQUANT 0
#define MMF_EPILOGUE_RAW_I32 1
#define MMF_EPILOGUE_GLU 2
#define MMF_EPILOGUE_AFFINE 3
#define MMF_TILE_128x512 0
#define MMF_TILE_128x256_PAIRED 1
#define MMF_TILE_64x512 2
#define MMF_TILE_64x256 3
#define MMF_TILE_256x256 4
int mmf_prefill_tile_plan(int64_t M, int64_t K, int64_t N, int epilogue, int cus);

#ifdef __cplusplus
}
#endif

#endif /* MMF_H */
