/*
 * ot.h -- C ABI of libot, OutlierTune's per-channel-quantized linear layer
 * for AMD Instinct MI355X (gfx950).
 *
 * The library implements the inference path of OutlierTune (Wang et al.,
 * 2024): static per-channel calibration of the activations with a
 * symmetrization shift (Sec. 3.2, App. A), the offline fold of the
 * activation scale into the weights and of the shift into the bias
 * (Sec. 3.1 Eq. (e), Eq. (f), Sec. 3.2 Eq. (g)), runtime per-channel
 * quantization of the activations (Eq. (g)), and the integer GEMM with a
 * dequantizing epilogue (Eq. (f) right-hand side, Eq. (g)).
 *
 * Conventions shared by every entry point
 *  - Tensors are dense and row-major (leading dimension = inner size).
 *    X is [M x K] (tokens x input channels); the weight W is [N x K], the
 *    layout of a PyTorch nn.Linear weight, so the paper's W^T is its
 *    transpose.
 *  - Every tensor pointer is a DEVICE pointer owned by the caller.  The
 *    library never allocates, frees or retains caller memory and keeps no
 *    global state (apart from ot_qlinear_noalloc's fixed scratch array);
 *    calls on different streams are independent.
 *  - fp16 tensors are passed as uint16_t IEEE binary16 bit patterns.
 *  - bits is in [2, 8]; the quantizer is symmetric and signed with largest
 *    code q(bits) = 2^(bits-1) - 1 (127 for 8 bits, 31 for 6 bits).  Codes
 *    are stored in int8 whatever the bit-width.  Rounding is round half to
 *    even throughout.
 *  - stream is a hipStream_t passed as void* (NULL = the default stream).
 *  - Every argument check happens on the host before any launch: on an
 *    error status no kernel runs and no output is written, except where an
 *    entry point says otherwise.  A fault inside an asynchronous kernel
 *    surfaces as OT_EHIP from a later synchronous call or from the caller's
 *    own stream synchronization.
 */
#ifndef OT_H_
#define OT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum ot_status {
  OT_OK = 0,
  OT_EINVAL = 1,     /* null pointer, bits outside [2, 8], negative size     */
  OT_ESHAPE = 2,     /* K not a multiple of 16, zero-sized where disallowed  */
  OT_ERANGE = 3,     /* K * qa * qw >= 2^31: the int32 accumulator could wrap */
  OT_ENONFINITE = 4, /* NaN or infinity in calibration data or weights       */
  OT_EHIP = 5,       /* a HIP runtime call failed                            */
  OT_ENOSCRATCH = 6  /* ot_qlinear_noalloc: the sizes need more scratch than  */
                     /* the library's fixed array holds                      */
} ot_status;

/* Static, human-readable description of a status code. */
const char *ot_strerror(int status);

/* Version of this ABI (bumped on any incompatible change). */
int ot_abi_version(void);

/* Static description of this build, "key=value" fields separated by ';':
 *   sources_sha256  SHA-256 of the sources and the release compiler flags
 *                   it was built from ("unknown" when built without the
 *                   recipe that computes it), so that a loaded library can
 *                   be matched against a source tree;
 *   arch            the GPU architecture of its device code;
 *   hip             the HIP version it was compiled against.
 * Never NULL; owned by the library. */
const char *ot_build_info(void);

/*
 * ot_calibrate -- static min-max calibration and symmetrization factors.
 * Sec. 3.2 (z = (max + min) / 2 per channel, X_hat = X - z) and App. A
 * (min-max calibration of the activations, done offline).
 *
 *   x       [rows x K] fp16 calibration activations (device).
 *   rows    >= 1.   K >= 1.
 *   a_bits  activation bit-width, in [2, 8]; qa = 2^(a_bits-1) - 1.
 *   first   nonzero: reset the running state before folding this batch in;
 *           zero: accumulate into the state left by earlier calls.
 *   minmax  [2K] fp32 running state (device): the K per-channel minima then
 *           the K maxima.  -0 is recorded as +0.
 *   z, s, inv_s  [K] fp32 outputs (device), rewritten from the running state
 *           on every call, so they are final after the last batch:
 *             z_k     = fp32((hi_k + lo_k) / 2)
 *             s_k     = fp32(((hi_k - lo_k) / 2) / qa), 1 if that is 0
 *             inv_s_k = fp32(1 / s_k)
 *           (fp64 arithmetic, each result rounded once to fp32).
 *
 * Synchronous: waits for the stream.  Returns OT_ENONFINITE if the running
 * state holds a NaN or an infinity (then z, s, inv_s are not written; the
 * state stays poisoned until a call with first != 0).
 */
ot_status ot_calibrate(const uint16_t *x, int64_t rows, int64_t K, int a_bits,
                       int first, float *minmax, float *z, float *s,
                       float *inv_s, void *stream);

/*
 * ot_scales_from_minmax -- z, s, 1/s from a calibration state (the minmax
 * that ot_calibrate keeps), for any bit-width, with or without the
 * symmetrization of Sec. 3.2 (the ablation of Sec. 4.4, Table 6):
 *   symmetrize != 0:  z_k = (hi_k + lo_k)/2,  s_k = ((hi_k - lo_k)/2)/qa
 *   symmetrize == 0:  z_k = 0,                s_k = max(|lo_k|, |hi_k|)/qa
 * fp64 math, fp32 storage, s_k = 1 where it would be 0, inv_s_k =
 * fp32(1/s_k).  With symmetrize != 0 and the calibration's own a_bits this
 * reproduces ot_calibrate's outputs exactly.
 *   minmax [2K] fp32 (device; the K minima then the K maxima, finite).
 *   z, s, inv_s [K] fp32 outputs (device).
 * Asynchronous on stream.
 */
ot_status ot_scales_from_minmax(const float *minmax, int64_t K, int a_bits,
                                int symmetrize, float *z, float *s,
                                float *inv_s, void *stream);

/*
 * ot_fold_weights -- the offline weight and bias transform.
 * Sec. 3.1 Eq. (e) (W_s = W scaled by s along the input channels), Eq. (f)
 * (per-output-channel quantization of W_s), Sec. 3.2 Eq. (g) (the shift z
 * moves into the bias, b' = z W^T + b), Implementation paragraph (the
 * weight quantization is done once, offline).
 *
 *   W       [N x K] fp16 weight (device).      b [N] fp16 bias or NULL.
 *   w_bits  weight bit-width in [2, 8]; qw = 2^(w_bits-1) - 1.
 *   z, s    [K] fp32 from ot_calibrate (device).
 *   Wq      [N x K] int8 output: clip(rne(W[n,k] s_k / sW_n), -qw, qw).
 *   sW      [N] fp32 output: fp32(max_k |W[n,k] s_k| / qw), 1 for a zero row.
 *   bprime  [N] fp32 output: fp32(sum_k z_k W[n,k] + b_n), summed in fp64
 *           (the summation order is unspecified, so it can differ from a
 *           sequential sum in the last fp32 place).
 *   The products W[n,k] s_k are exact in fp64, the division by sW_n is a
 *   correctly rounded fp64 division.
 *
 * Synchronous.  OT_ENONFINITE if W or b holds a NaN or an infinity; then
 * the contents of Wq, sW and bprime are unspecified.
 */
ot_status ot_fold_weights(const uint16_t *W, const uint16_t *b, int64_t N,
                          int64_t K, int w_bits, const float *z, const float *s,
                          int8_t *Wq, float *sW, float *bprime, void *stream);

/*
 * ot_quantize_act -- runtime symmetrize + per-channel quantize, Eq. (g):
 *   Xq[m,k] = clip(rne(fp32(fp32(x[m,k]) - z_k) * inv_s_k), -qa, qa)
 * with both fp32 operations rounded to nearest even (no fused multiply-add).
 * Values outside the calibrated range clip; NaN input gives unspecified
 * codes.
 *
 *   x      [M x K] fp16 (device).  M >= 0 (0 is a no-op), K >= 16, K % 16 == 0.
 *   z, inv_s  [K] fp32 (device).    Xq [M x K] int8 output (device).
 *
 * Asynchronous on stream.
 */
ot_status ot_quantize_act(const uint16_t *x, int64_t M, int64_t K, int a_bits,
                          const float *z, const float *inv_s, int8_t *Xq,
                          void *stream);

/*
 * ot_ln_quantize_act -- LayerNorm fused with symmetrization and Eq. (g)'s
 * per-channel quantization (Sec. 3.2: z is taken into the LayerNorm's bias,
 * Implementation paragraph: the quantization is fused with the LayerNorm
 * that precedes the linear).  Per row of h, with a_k = h_k 2^24 (an exact
 * integer for every fp16 value), S1 = sum_k a_k and S2 = sum_k a_k^2
 * (exact integers) and each float64 step rounded to nearest:
 *   mean = fl(fl(S1) / K) 2^-24
 *   var  = fl(fl(K S2 - S1^2) / K^2) 2^-48       (population variance)
 *   rstd = fl(1 / fl(sqrt(fl(var + eps))))
 * and per element, in fp32 rounded to nearest even (no fused multiply-add):
 *   Xq[m,k] = clip(rne((((h - fp32(mean)) * fp32(rstd)) * gamma_k
 *                       + (beta_k - z_k)) * inv_s_k), -qa, qa)
 * The codes are exactly these.  The kernel reaches fp32(mean) and
 * fp32(rstd) through float64 sums with a proven error bound, and through
 * the exact integer sums for the rows that bound cannot settle (a mean or
 * rstd within the bound of an fp32 rounding boundary, e.g. a mean of 0), so
 * such rows cost more.
 * The normalized fp16 activation is never written.
 *
 *   h      [M x K] fp16 LayerNorm input (device).  M >= 0 (0 is a no-op),
 *          16 <= K <= 65536, K % 16 == 0.  Finite values; a row of equal
 *          values with eps == 0 (and NaN or infinity anywhere in a row)
 *          gives unspecified codes for that row.
 *   gamma, beta  [K] fp16 LayerNorm weight and bias (device).
 *   eps    the LayerNorm epsilon, finite and >= 0.
 *   z, inv_s     [K] fp32 from ot_calibrate on the LayerNorm's output.
 *   Xq     [M x K] int8 output (device).
 *
 * Asynchronous on stream.
 */
ot_status ot_ln_quantize_act(const uint16_t *h, int64_t M, int64_t K,
                             const uint16_t *gamma, const uint16_t *beta,
                             float eps, int a_bits, const float *z,
                             const float *inv_s, int8_t *Xq, void *stream);

/*
 * ot_qlinear -- the quantized linear: integer GEMM (Eq. (f) right-hand side)
 * with the fused dequantizing epilogue of Eq. (g):
 *   acc[m,n] = sum_k Xq[m,k] Wq[n,k]                       (exact int32)
 *   Y[m,n]   = fp16(fp32(fp32(acc[m,n]) * sW_n) + bprime_n)
 * every conversion and operation rounded to nearest even, no fused
 * multiply-add.  Prefill shapes run on the int8 matrix cores; M <= 64 runs
 * a weight-streaming decode kernel.  Both give bit-identical results.
 *
 *   Xq [M x K] int8, Wq [N x K] int8, sW [N] fp32, bprime [N] fp32 (device).
 *   M >= 0 (0 is a no-op), N >= 1, K >= 16 with K % 16 == 0.
 *   a_bits, w_bits  the bit-widths the codes were made with; they bound the
 *           codes (|Xq| <= qa, |Wq| <= qw) and so the accumulator:
 *           OT_ERANGE if K * qa * qw >= 2^31.  Codes outside those bounds
 *           give unspecified results.
 *   Y      [M x N] fp16 output (device).
 *   acc_out  NULL, or [M x N] int32 (device) that also receives acc (for
 *           testing; costs extra memory traffic).
 *   workspace  NULL, or at least ot_qlinear_workspace_size(M, N, K) bytes of
 *           16-byte-aligned device memory the call may use as scratch; with
 *           NULL the call uses no scratch memory.  Results do not depend on
 *           it.  For 17..64 tokens, where the launch plan finds it faster
 *           (layers with few output channels per compute unit and long K),
 *           the call then splits K over more workgroups and adds their int32
 *           partial sums in a second kernel (the sums are exact, so the
 *           outputs are identical); ot_qlinear_workspace_size returns 0
 *           where it does not.  The contents need no initialization and
 *           are left unspecified; calls that overlap in time must not share
 *           a workspace.
 *
 * Asynchronous on stream; no synchronization, no allocation.
 */
ot_status ot_qlinear(const int8_t *Xq, const int8_t *Wq, const float *sW,
                     const float *bprime, int64_t M, int64_t N, int64_t K,
                     int a_bits, int w_bits, uint16_t *Y, int32_t *acc_out,
                     void *workspace, void *stream);

/*
 * Asymmetric weights, the paper's "Int8" setting (Sec. 4.1, App. A):
 * per-output-channel asymmetric quantization of W_s = W diag(s), Eq. (a)
 * with a zero point.  With L = 2^w_bits - 1, per output channel n:
 *   lo, hi = min(min_k W_s[n,k], 0), max(max_k W_s[n,k], 0)
 *   sW[n]  = fp32((hi - lo) / L)  (1 where 0);  zp = clip(rne(-lo/sW), 0, L)
 *   c[n,k] = clip(rne(W_s[n,k] / sW[n]) + zp, 0, L)   (fp64, correctly rounded)
 * stored shifted so that they fit int8: Wq = c - 2^(w_bits-1),
 * zW[n] = zp - 2^(w_bits-1).  bprime as for ot_fold_weights.
 *
 * ot_fold_weights_asym -- arguments as ot_fold_weights plus zW [N] int32
 * output.  Synchronous; OT_ENONFINITE as ot_fold_weights.
 */
ot_status ot_fold_weights_asym(const uint16_t *W, const uint16_t *b, int64_t N,
                               int64_t K, int w_bits, const float *z,
                               const float *s, int8_t *Wq, float *sW,
                               int32_t *zW, float *bprime, void *stream);

/*
 * ot_qlinear_asym -- the quantized linear with asymmetric weights:
 *   acc[m,n] = sum_k Xq[m,k] (Wq[n,k] - zW[n])   exact in int32
 *   Y[m,n]   = fp16(fp32(fp32(acc[m,n]) * sW[n]) + bprime[n])
 * The kernels compute sum_k Xq Wq and subtract zW[n] times the token's code
 * sum, which they take from the token fragments they already hold.
 * Arguments as ot_qlinear plus zW [N] int32 (device); acc_out receives acc.
 * OT_ERANGE when K * qa * 2^w_bits >= 2^31.
 */
ot_status ot_qlinear_asym(const int8_t *Xq, const int8_t *Wq, const float *sW,
                          const int32_t *zW, const float *bprime, int64_t M,
                          int64_t N, int64_t K, int a_bits, int w_bits,
                          uint16_t *Y, int32_t *acc_out, void *workspace,
                          void *stream);

/*
 * Per-token path.  The paper keeps the linears without activation outliers
 * (out and fc2, whose inputs are not LayerNorm outputs) on per-token
 * symmetric activation quantization, Eq. (c), and carries a symmetrized
 * residual stream back through their bias, Eq. (h) (Sec. 3.2, Sec. 4.1).
 *
 * ot_quantize_act_per_token -- dynamic per-token scales and codes:
 *   sX[m]    = fp32(max_k |x[m,k]| / qa)   (fp64 division; 1 for a zero row)
 *   Xq[m,k]  = clip(rne(fp32(x[m,k]) * fp32(1 / sX[m])), -qa, qa)
 *   x   [M x K] fp16 (device), finite.  M >= 0 (0 is a no-op),
 *       16 <= K <= 65536, K % 16 == 0.
 *   Xq  [M x K] int8 output, sX [M] fp32 output (device).
 * Asynchronous on stream.
 */
ot_status ot_quantize_act_per_token(const uint16_t *x, int64_t M, int64_t K,
                                    int a_bits, int8_t *Xq, float *sX,
                                    void *stream);

/*
 * ot_fold_weights_per_token -- offline weights of a per-token linear: no
 * activation scale is folded in (Eq. (c)).
 *   sW[n]     = fp32(max_k |W[n,k]| / qw)   (1 for a zero row)
 *   Wq[n,k]   = clip(rne(W[n,k] / sW[n]), -qw, qw)  (correctly rounded fp64)
 *   bprime[n] = fp32(b[n] + zres[n])        (fp64 sum; Eq. (h))
 *   W [N x K] fp16, b [N] fp16 or NULL, zres [N] fp32 or NULL: the shift z
 *   of the symmetrized residual stream that this linear's output is added
 *   to (NULL when the residual stream is not symmetrized).
 * Synchronous.  OT_ENONFINITE if W, b or zres hold a NaN or an infinity.
 */
ot_status ot_fold_weights_per_token(const uint16_t *W, const uint16_t *b,
                                    const float *zres, int64_t N, int64_t K,
                                    int w_bits, int8_t *Wq, float *sW,
                                    float *bprime, void *stream);

/*
 * ot_qlinear_per_token -- the quantized linear of Eq. (c) with the bias:
 *   Y[m,n] = fp16(fp32(fp32(fp32(acc[m,n]) * sX[m]) * sW[n]) + bprime[n])
 * with acc = Xq Wq^T exact in int32, each fp32 operation rounded to nearest
 * even.  Arguments as for ot_qlinear, plus sX [M] fp32 (device) from
 * ot_quantize_act_per_token; same kernels, same error codes.
 */
ot_status ot_qlinear_per_token(const int8_t *Xq, const int8_t *Wq,
                               const float *sX, const float *sW,
                               const float *bprime, int64_t M, int64_t N,
                               int64_t K, int a_bits, int w_bits, uint16_t *Y,
                               int32_t *acc_out, void *workspace, void *stream);

/*
 * ot_qlinear_noalloc -- ot_qlinear for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, checks and results as ot_qlinear
 * without the workspace argument: where ot_qlinear would use a workspace
 * (split-K decode, 17..64 tokens), this call uses a fixed device array of
 * OT_NOALLOC_SCRATCH_BYTES that the library holds on every device it runs
 * on until the process ends (its address is looked up on the first call on
 * each device).  It calls no allocation routine.  OT_ENOSCRATCH if
 * ot_qlinear_workspace_size(M, N, K) exceeds OT_NOALLOC_SCRATCH_BYTES
 * (then nothing runs; ot_qlinear with a workspace serves such sizes).  On
 * a 256-CU device that cannot happen: a split plan runs at most one
 * workgroup per CU, runs x ceil(N / rows) <= 256 with rows <= 128, so it
 * needs at most 64 x 4 x (32768 + 8) bytes (8.0 MiB).
 * Calls that overlap in time on one device share the array and race:
 * serialize them (one stream, or events).  Asynchronous on stream.
 */
#define OT_NOALLOC_SCRATCH_BYTES (9u << 20)
ot_status ot_qlinear_noalloc(const int8_t *Xq, const int8_t *Wq,
                             const float *sW, const float *bprime, int64_t M,
                             int64_t N, int64_t K, int a_bits, int w_bits,
                             uint16_t *Y, int32_t *acc_out, void *stream);

/* Bytes of optional scratch that ot_qlinear, ot_qlinear_per_token,
 * ot_qlinear_asym and ot_qlinear_packed can use for these sizes on the
 * current device (0 if none; also 0 for sizes the calls reject).
 * Synchronous, no device work. */
size_t ot_qlinear_workspace_size(int64_t M, int64_t N, int64_t K);

/*
 * ot_qlinear_plan -- which kernel configuration the quantized-linear calls
 * (ot_qlinear and its per-token and asymmetric variants, or, with
 * packed != 0, ot_qlinear_packed) launch for these sizes on the current
 * device, given a workspace (with_workspace != 0) or not.  Writes a
 * NUL-terminated description into buf (at most len bytes, truncated if
 * longer): "none" for M == 0; "prefill 256x256", "prefill 320x256",
 * "prefill 256x128" or "prefill 192x256" (output channels x tokens per
 * workgroup) above 64
 * tokens; "decode <layout> <R>-row tiles", with " split-K <runs>" where K
 * is split, up to 64 tokens.  OT_EINVAL for a NULL buf or len 0, OT_ESHAPE
 * for sizes the calls reject.  Synchronous, no device work; for
 * introspection and tests (the results never depend on the plan).
 */
ot_status ot_qlinear_plan(int64_t M, int64_t N, int64_t K, int packed,
                          int with_workspace, char *buf, size_t len);

/*
 * Packed weights for decode.  The folded codes (Eq. (f) right-hand side,
 * fixed offline like the fold itself, Sec. 3.2) re-laid so that each 1 KiB
 * is one matrix-instruction operand of a wave, which the weight-streaming
 * kernel loads straight into registers: micro-tiles of 16 output channels
 * by 64 input channels,
 *   Wp[g][s][l][b] = Wq[16 g + (l mod 16)][64 s + 16 (l / 16) + b]
 * for g < ceil(N/16), s < ceil(K/64), lane l < 64, byte b < 16, and 0 where
 * the row is >= N or the column >= K (the lane order of the A operand of
 * the 16x16x64 int8 matrix instruction).  The codes are unchanged, so
 * ot_qlinear_packed gives ot_qlinear's results bit for bit.
 *
 * ot_packed_weights_size -- bytes of Wp: ceil(N/16) ceil(K/64) 1024 (0 for
 *   sizes ot_pack_weights rejects).  No device work.
 * ot_pack_weights -- Wq [N x K] int8 (device) -> Wp (device, 16-byte
 *   aligned, ot_packed_weights_size bytes).  N >= 1, K >= 16, K % 16 == 0.
 *   Asynchronous on stream.
 * ot_qlinear_packed -- ot_qlinear for M <= 64 tokens (OT_ESHAPE beyond)
 *   with Wp from ot_pack_weights for the same N and K; the other arguments,
 *   the workspace and the results as for ot_qlinear.
 */
size_t ot_packed_weights_size(int64_t N, int64_t K);
ot_status ot_pack_weights(const int8_t *Wq, int64_t N, int64_t K, int8_t *Wp,
                          void *stream);
ot_status ot_qlinear_packed(const int8_t *Xq, const int8_t *Wp, const float *sW,
                            const float *bprime, int64_t M, int64_t N, int64_t K,
                            int a_bits, int w_bits, uint16_t *Y,
                            int32_t *acc_out, void *workspace, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* OT_H_ */
