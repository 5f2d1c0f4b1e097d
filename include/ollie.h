/*
 * ollie.h -- C ABI of the MI355X (gfx950) derived-operator library.
 *
 * The library executes the tensor-algebra expressions that the derivation method
 * reaches for three convolution operators and a banded batched matmul:
 *
 *   convolution-family operator  =  GEMM stage  +  eOperator stage
 *     GEMM stage   Y[m][n] = sum_c A'[m][c] * K'[c][n]   (the matched Matmul scope,
 *                  section 4.3.1; operand layouts of Eq. (3) and Eq. (4))
 *     eOperator    out[p][k] = sum over taps (r,s) of Y[m(p,r,s)][(r*S+s)*K + k]
 *                  (OffsetAdd of section 2 for convolutions, the selective add of
 *                  section 6.3 for the strided transposed convolution)
 *
 *   banded_bmm   S = G2BMM(Q, K) on the dilated band (Table 2), P = softmax(S),
 *                O = P * V on the same band; the dilation is removed by splitting
 *                rows by residue (section 6.4).
 *
 * Every tensor pointer is a HIP device pointer.  Every call only enqueues work on
 * `stream` (a hipStream_t; NULL means the default stream) and returns at once;
 * results are ready when the stream reaches that point.  The library allocates
 * nothing and frees nothing: the caller owns every buffer, including workspaces.
 * No call synchronises the device.
 *
 * Errors: each entry point returns an ollie_status.  All argument checks happen on
 * the host before any HIP call, so a non-zero status other than OLLIE_EHIP means
 * nothing was enqueued.  OLLIE_EHIP means a HIP launch failed; earlier launches of
 * the same call may have been enqueued.  ollie_last_error() gives a message for the
 * last failure on the calling thread.
 *
 * Common buffer rules: tensors are dense and row-major in the layouts stated below;
 * pointers must be 16-byte aligned (else OLLIE_EALIGN); outputs must not overlap
 * inputs or the workspace (else OLLIE_EINVAL; one stated exception: a fused residual
 * that is the output buffer itself, see ollie_conv_epilogue).
 */
#ifndef OLLIE_H
#define OLLIE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    OLLIE_OK = 0,
    OLLIE_EINVAL = 1,       /* bad shape, geometry, flag or null pointer        */
    OLLIE_EDTYPE = 2,       /* unsupported dtype or dtype combination           */
    OLLIE_EWORKSPACE = 3,   /* workspace smaller than the *_workspace_bytes size */
    OLLIE_EALIGN = 4,       /* a pointer or a row is not 16-byte aligned         */
    OLLIE_EHIP = 5          /* a HIP launch failed                              */
} ollie_status;

typedef enum {
    OLLIE_F32 = 0,          /* IEEE binary32                                     */
    OLLIE_BF16 = 1          /* bfloat16; conversions round to nearest even       */
} ollie_dtype;

/* flags */
#define OLLIE_FUSE_EPILOGUE     (1u << 0)  /* conv: fused GEMM + eOperator, no Y (see below)   */
#define OLLIE_Y_BF16            (1u << 1)  /* conv: hold the GEMM scope Y in bf16 (default fp32) */
#define OLLIE_BAND_STAGED       (1u << 2)  /* band: three kernels through S and P in the workspace */
#define OLLIE_BAND_MASK_INVALID (1u << 3)  /* band: keys outside [0,l) are left out of the softmax */
#define OLLIE_DILATED_RESIDUES  (1u << 4)  /* dilated conv: as non-dilated convs over residue sub-images */
#define OLLIE_CONV_SPLIT_3X3    (1u << 5)  /* conv: as a 3x3 convolution over kernel blocks + OffsetAdd */

/* Tile-configuration overrides, for tuning sweeps and tests (these bits zero = the
 * library's automatic choice, which is what every other caller should use).  They
 * change which kernel instance evaluates the expression, never what it computes.
 *   OLLIE_FUSED_TILE(n), n in 0..14: tile shape of the fused GEMM + eOperator kernel
 *     (conv entry points; ignored when the call takes the two-stage path).
 *   OLLIE_GEMM_TILE(n), n in 0..4: tile shape of the GEMM stage kernel (conv entry
 *     points on the two-stage path; ignored on the fused path).
 *   OLLIE_BAND_SHAPE(n), n in 0..3: wave shape of the fused band kernel (banded_bmm
 *     without OLLIE_BAND_STAGED).
 * An n outside its range gives OLLIE_EINVAL. */
#define OLLIE_FUSED_TILE(n)     ((uint32_t)(((n) + 1) & 0xff) << 16)
#define OLLIE_GEMM_TILE(n)      ((uint32_t)(((n) + 1) & 0xf) << 24)
#define OLLIE_BAND_SHAPE(n)     ((uint32_t)(((n) + 1) & 0xff) << 16)

/* Geometry of a convolution-family operator.
 *   X   [n][h][w][c]   input (NHWC).  As a GEMM operand it is A'[m][c] with
 *                      m = (n*h + hi)*w + wi, i.e. Eq. (3) with a batch dimension:
 *                      the identity eOperator of section 5.4, no copy is made.
 *   Wt  [r][s][k][c]   weight (the paper's K[r,s,f,c] with f = k).  Row-major it is
 *                      the [R*S*K][C] matrix K'^T of Eq. (4), column n = (r*S+s)*k + k.
 *                      From a torch conv2d weight [K][C][R][S] use permute(2,3,0,1);
 *                      from a conv_transpose2d weight [C][K][R][S] use permute(2,3,1,0).
 *                      This layout change depends on weights only and is done once,
 *                      ahead of time (compile-time evaluation, section 5.4).
 *   out [n][ho][wo][k] output (NHWC).
 *   stride, pad, dil >= 1, >= 0, >= 1 per axis; out_pad only for the transposed
 *   operator (0 <= out_pad < max(stride, dil)), 0 otherwise.
 *   in_dtype: dtype of X and Wt (F32 or BF16); accumulation is always fp32.
 *   out_dtype: dtype of out (F32 or BF16). */
typedef struct {
    int64_t n, c, h, w;
    int64_t k, r, s;
    int32_t stride_h, stride_w;
    int32_t pad_h, pad_w;
    int32_t dil_h, dil_w;
    int32_t out_pad_h, out_pad_w;
    int32_t in_dtype;      /* ollie_dtype */
    int32_t out_dtype;     /* ollie_dtype */
} ollie_conv_desc;

/* Element-wise tail of a convolution-family operator, evaluated inside its eOperator
 * (or inside the fused expression) right before the store -- the fusion of OffsetAdd
 * with the element-wise operators that follow it (section 6.3):
 *   out[n][ho][wo][k] = act( conv[n][ho][wo][k] + bias[k] + residual[n][ho][wo][k] )
 * with act = ReLU (max(., 0)) when relu != 0, the identity otherwise.  conv is the
 * operator's fp32 accumulation; the additions and the ReLU run in fp32 in this order,
 * then the result is converted to out_dtype.
 *   bias      [k] in bias_dtype, or NULL (no bias term)
 *   residual  [n][ho][wo][k] (the layout of out) in residual_dtype, or NULL; it may be
 *             the same buffer as out (each element is read before it is overwritten,
 *             by the same thread), but may not overlap it otherwise.
 * Both pointers must be 16-byte aligned; dtypes are OLLIE_F32 or OLLIE_BF16. */
typedef struct {
    const void* bias;
    const void* residual;
    int32_t bias_dtype;      /* ollie_dtype */
    int32_t residual_dtype;  /* ollie_dtype */
    int32_t relu;            /* 0 or 1 */
} ollie_conv_epilogue;

/* Geometry of banded_bmm.
 *   Q, K, V [b][l][d] bf16, O [b][l][d] (out_dtype F32 or BF16).
 *   Band entry j in [0, 2w] of row i reads key/value row t = i + (j - w) * dilation;
 *   rows outside [0, l) read as zero (section 3 padding).
 *   d must be 64. */
typedef struct {
    int64_t b, l, d, w;
    int32_t dilation;
    float scale;           /* multiplies Q.K before the softmax                    */
    int32_t in_dtype;      /* ollie_dtype, must be OLLIE_BF16                      */
    int32_t out_dtype;     /* ollie_dtype of O                                     */
} ollie_band_desc;

/* ------------------------------------------------------------------ helpers */

/* Output extent of the operator (transposed = 0: conv2d / dilated conv2d,
 * 1: conv_transpose2d), the traversal range of the output scope of the convolution
 * expression (section 3, section 4.2 with zero padding; the transposed operator as
 * the adjoint of the convolution, section 6.3):
 *   forward    ho = floor((h + 2*pad_h - dil_h*(r-1) - 1) / stride_h) + 1
 *   transposed ho = (h-1)*stride_h - 2*pad_h + dil_h*(r-1) + out_pad_h + 1
 * and likewise for wo.  Returns OLLIE_EINVAL on invalid geometry or an empty output. */
int ollie_conv_out_hw(const ollie_conv_desc* desc, int transposed, int64_t* ho, int64_t* wo);

/* Bytes of workspace that derived_conv2d / derived_dilated_conv2d /
 * derived_conv_transpose2d need: the instantiated scope Y [n*h*w][r*s*k] of the
 * matched Matmul (section 4.3.1, the scope instantiation of Eq. (3) and (4)) in fp32
 * (or bf16 with OLLIE_Y_BF16); 0 when OLLIE_FUSE_EPILOGUE is set and the fused kernel
 * covers the shape.  With OLLIE_CONV_SPLIT_3X3 (derived_conv2d): the split weights,
 * the 3x3 stage Z and that stage's own workspace (see derived_conv2d).  Returns 0 for
 * invalid geometry. */
size_t ollie_conv_workspace_bytes(const ollie_conv_desc* desc, int transposed, uint32_t flags);

/* Bytes of workspace banded_bmm needs: 0 for the fused path; with OLLIE_BAND_STAGED,
 * the G2BMM output scope (Table 2: iterators b, i in every tensor, the band offset j
 * in weight and output) S [b][l][2w+1] fp32 followed (at a 256-byte aligned offset) by P [b][l][2w+1] bf16.
 * Returns 0 for a descriptor banded_bmm rejects (invalid geometry, or a staged band
 * wider than 1024 entries). */
size_t ollie_band_workspace_bytes(const ollie_band_desc* desc, uint32_t flags);

/* Message for the last failure on this thread ("" if none); valid until the next
 * library call on this thread.  (Error reporting of the library; no passage of the
 * paper defines it.) */
const char* ollie_last_error(void);

/* Library version string, e.g. "ollie-mi355x 0.2.0 (gfx950)".  (Not defined by the
 * paper.) */
const char* ollie_version(void);

/* ------------------------------------------------------------- entry points */

/* Convolution (cross-correlation, section 4.2 expression E1) with stride and zero
 * padding, dilation 1, as a GEMM over all input pixels followed by the OffsetAdd
 * eOperator (section 2, Fig. "optimization found"):
 *   Y[m][(r*S+s)*K+k] = sum_c X[m][c] * Wt[r][s][k][c]
 *   out[n][ho][wo][k] = sum_{r,s} [0 <= hi < h][0 <= wi < w] Y[(n*h+hi)*w+wi][(r*S+s)*K+k]
 *   with hi = ho*stride_h - pad_h + r, wi = wo*stride_w - pad_w + s.
 * x: X, wt: Wt, out: out (layouts above).  ws: workspace of at least
 * ollie_conv_workspace_bytes(desc, 0, flags) bytes (holds Y).  flags: OLLIE_Y_BF16,
 * OLLIE_FUSE_EPILOGUE.
 * Rejects dil != 1 (OLLIE_EINVAL; use derived_dilated_conv2d).
 *
 * OLLIE_FUSE_EPILOGUE evaluates the expression obtained by fusing the GEMM scope into
 * the eOperator (expression fusion, section 4.1): one contraction over (tap, c) per
 * output element, so Y is never formed and ws may be NULL.  It covers bf16 inputs with
 * c % 64 == 0, r <= 64 and s <= 64 and at most 16 output residue classes (the
 * transposed operator has stride_h*stride_w classes, the residue form dil_h*dil_w, the
 * plain convolution one); other shapes take the two-stage path, which needs the
 * workspace.  ollie_conv_workspace_bytes returning 0 for these flags is the test for
 * the fused path.
 * Summation order differs from the two-stage path, so fp32 results agree to rounding
 * (integer-valued inputs agree exactly).
 *
 * OLLIE_CONV_SPLIT_3X3 evaluates the derived form that turns an R x S convolution into
 * a 3x3 one (the Conv5x5 -> Conv3x3 transformation of section 6, Table 3), stride 1
 * only.  Boundary relaxing extends the kernel to 3*nbr x 3*nbs taps (nbr = ceil(R/3),
 * nbs = ceil(S/3)) with zero weights; variable substitution writes r = 3*a + r',
 * s = 3*b + s'; summation splitting instantiates the inner sum over (r', s', c) as a
 * 3x3 convolution with nbr*nbs*K output channels,
 *   W3[r'][s'][(a*nbs + b)*K + k][c] = Wt[3a + r'][3b + s'][k][c]  (0 outside R x S)
 *   Z[n][i][j][(a*nbs + b)*K + k] = sum_{r',s',c} X0[n][i - ph - er + r'][j - pw - es + s'][c]
 *                                                 * W3[r'][s'][(a*nbs + b)*K + k][c]
 * (X0: X zero outside the image; er = 3*nbr - R, es = 3*nbs - S; Z is that
 * convolution with padding ph + er, pw + es, so i < h + 2(ph + er) - 2), and the outer
 * sum over the kernel blocks is an OffsetAdd with offset step 3:
 *   out[n][ho][wo][k] = sum_{a < nbr, b < nbs} Z[n][ho + er + 3a][wo + es + 3b][(a*nbs + b)*K + k].
 * Kernels: the weight split, then either
 *   - with OLLIE_FUSE_EPILOGUE where the fused kernel covers the 3x3 stage: that stage
 *     as the fused kernel into Z, and the block OffsetAdd over Z; or
 *   - otherwise: the 3x3 stage's GEMM into its scope
 *     Y[m][(r'*3 + s')*nbr*nbs*K + (a*nbs + b)*K + k] (fp32, or bf16 with OLLIE_Y_BF16),
 *     and its two consecutive eOperators (the 3x3 OffsetAdd, then the block OffsetAdd)
 *     fused into one (eOperator fusion, section 5.4):
 *       out[n][ho][wo][k] = sum_{r<R, s<S} [0 <= hi < h][0 <= wi < w]
 *           Y[(n*h + hi)*w + wi][((r%3)*3 + s%3)*nbr*nbs*K + ((r/3)*nbs + s/3)*K + k]
 *       with hi = ho - ph + r, wi = wo - pw + s (the relaxed taps carry zero weights and
 *       are not read), so Z is never formed.
 * The last kernel takes the element-wise tail.  ws holds W3 [3][3][nbr*nbs*K][c] in
 * in_dtype, then (at the next 256-byte aligned offset) Z in fp32 or the scope Y.
 * Needs stride 1 and dilation 1, else OLLIE_EINVAL. */
int derived_conv2d(const ollie_conv_desc* desc, const void* x, const void* wt, void* out,
                   void* ws, size_t ws_bytes, uint32_t flags, void* stream);

/* derived_conv2d for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same operator,
 * arguments and flags as derived_conv2d, with the workspace taken from the library's
 * own static device array instead of a caller buffer.  The call allocates nothing (no
 * hipMalloc, hipFree or allocating library routine); x, wt and out are still the
 * caller's.
 *   Limit: ollie_conv_workspace_bytes(desc, 0, flags) <= 64 MiB (67108864 bytes), else
 *   OLLIE_EWORKSPACE and nothing is enqueued.  (The fused path needs no workspace.)
 *   The array is one per GPU (64 MiB held on every GPU the library runs on, until the
 *   process ends), shared by every call on that GPU and left holding the last call's
 *   partials; no kernel reads a byte of it that the same call has not written first.
 *   Calls on one GPU whose executions overlap (other streams, other threads) race on
 *   it: serialise them.
 *   The first call on a device looks up the array's device address once
 *   (hipGetSymbolAddress; a failure gives OLLIE_EHIP). */
int ollie_derived_conv2d_noalloc(const ollie_conv_desc* desc, const void* x, const void* wt,
                                 void* out, uint32_t flags, void* stream);

/* Dilated convolution as the same GEMM plus the dilated OffsetAdd: taps are spaced by
 * the dilation, hi = ho*stride_h - pad_h + r*dil_h, wi = wo*stride_w - pad_w + s*dil_w;
 * taps outside the image read the zero padding and are skipped (boundary tightening,
 * section 4.2).  Same arguments as derived_conv2d; any dil >= 1.
 *
 * OLLIE_DILATED_RESIDUES (with OLLIE_FUSE_EPILOGUE) evaluates instead the derived form
 * of section 6.2: for stride 1, the outputs of residue (a, b) = (ho % dil_h,
 * wo % dil_w) are a non-dilated convolution over the input sub-image
 * X[n][dil_h*i + rho_h][dil_w*j + rho_w], read as a strided view (no copy), so the
 * operator becomes dil_h*dil_w non-dilated convolutions.  Needs stride 1,
 * dil_h*dil_w <= 16 and a shape the fused expression covers; else OLLIE_EINVAL. */
int derived_dilated_conv2d(const ollie_conv_desc* desc, const void* x, const void* wt,
                           void* out, void* ws, size_t ws_bytes, uint32_t flags,
                           void* stream);

/* Transposed convolution (section 6.3): the GEMM runs on the unpadded input, then
 * each output sums only the partials that land on it (selective add):
 *   out[n][ho][wo][k] = sum_{r,s} [th >= 0, th % stride_h == 0, th/stride_h < h]
 *                               [tw >= 0, tw % stride_w == 0, tw/stride_w < w]
 *                       Y[(n*h + th/stride_h)*w + tw/stride_w][(r*S+s)*K+k]
 *   with th = ho + pad_h - r*dil_h, tw = wo + pad_w - s*dil_w.
 * Here c is the operator's input channel count and k its output channel count.
 * Same arguments as derived_conv2d; ws sized with transposed = 1. */
int derived_conv_transpose2d(const ollie_conv_desc* desc, const void* x, const void* wt,
                             void* out, void* ws, size_t ws_bytes, uint32_t flags,
                             void* stream);

/* The three operators above with an element-wise tail (ollie_conv_epilogue) fused
 * into their last kernel, for both the two-stage and the fused path: the fusion of
 * the eOperator with the element-wise operators after it (section 6.3, and the
 * expression fusion of section 5.4).  epi == NULL is the plain operator.  Extra
 * checks: relu not in {0, 1} -> OLLIE_EINVAL; a bias/residual pointer that is not
 * 16-byte aligned -> OLLIE_EALIGN; an unknown bias_dtype/residual_dtype of a non-NULL
 * tensor -> OLLIE_EDTYPE; a bias overlapping out, or a residual overlapping out
 * other than exactly (same pointer) -> OLLIE_EINVAL. */
int ollie_derived_conv2d_ex(const ollie_conv_desc* desc, const void* x, const void* wt,
                            void* out, void* ws, size_t ws_bytes, uint32_t flags,
                            const ollie_conv_epilogue* epi, void* stream);
int ollie_derived_dilated_conv2d_ex(const ollie_conv_desc* desc, const void* x,
                                    const void* wt, void* out, void* ws, size_t ws_bytes,
                                    uint32_t flags, const ollie_conv_epilogue* epi,
                                    void* stream);
int ollie_derived_conv_transpose2d_ex(const ollie_conv_desc* desc, const void* x,
                                      const void* wt, void* out, void* ws, size_t ws_bytes,
                                      uint32_t flags, const ollie_conv_epilogue* epi,
                                      void* stream);

/* Banded dilated batched matmul with row softmax (Longformer-style sliding window):
 *   S[b][i][j] = scale * sum_e Q[b][i][e] * K0[b][t][e],  t = i + (j-w)*dilation
 *   P[b][i][:] = softmax_j S[b][i][:]
 *   O[b][i][e] = sum_j P[b][i][j] * V0[b][t][e]
 * K0, V0 are K, V with rows outside [0,l) reading zero.  By default such entries keep
 * S = 0 and take part in the softmax (zero mode); with OLLIE_BAND_MASK_INVALID they
 * are left out (P = 0).  The dilated band is evaluated as `dilation` non-dilated bands
 * over the row subsequences i = dilation*i' + rho (section 6.4).
 * Default: one fused kernel, S and P never leave the chip, ws may be NULL and
 * s_out must be NULL.  With OLLIE_BAND_STAGED: three kernels (G2BMM -> softmax
 * eOperator -> band-times-dense) through fp32 S and bf16 P in ws; if s_out is not
 * NULL, S [b][l][2w+1] fp32 is written there instead of into ws. */
int banded_bmm(const ollie_band_desc* desc, const void* q, const void* k, const void* v,
               void* o, float* s_out, void* ws, size_t ws_bytes, uint32_t flags,
               void* stream);

/* ------------------------------------------------- stage entry points (same kernels) */

/* GEMM stage alone, the matched Matmul of the derived convolution forms (section 4.3.1;
 * operand layouts of Eq. (3) and Eq. (4)):
 *   Y[m][n] = sum_kk A[m][kk] * B[n][kk]   (A [m][k], B [n][k], Y [m][n], row-major).
 * in_dtype F32 or BF16 (A and B); y_dtype F32 or BF16 (bf16 Y rounds the fp32 sum to
 * nearest even).  BF16 needs k % 8 == 0 (else OLLIE_EALIGN).  y must not overlap a or b
 * (OLLIE_EINVAL). */
int ollie_gemm_nt(int64_t m, int64_t n, int64_t k, const void* a, const void* b, void* y,
                  int32_t in_dtype, int32_t y_dtype, void* stream);

/* OffsetAdd eOperator alone (section 2; taps spaced by the dilation, out-of-image taps
 * never read, section 4.2 boundary tightening): y is the scope Y [n*h*w][r*s*k] in
 * y_dtype, out [n][ho][wo][k] in desc->out_dtype,
 *   out[n][ho][wo][k] = sum_{r,s} [0 <= hi < h][0 <= wi < w] Y[(n*h+hi)*w+wi][(r*S+s)*K+k]
 *   hi = ho*stride_h - pad_h + r*dil_h, wi = wo*stride_w - pad_w + s*dil_w.
 * out must not overlap y (OLLIE_EINVAL). */
int ollie_eop_offset_sum(const ollie_conv_desc* desc, const void* y, int32_t y_dtype,
                         void* out, void* stream);

/* Selective-add eOperator of the transposed convolution alone (section 6.3): the same
 * arguments, with the tap rule of derived_conv_transpose2d
 *   th = ho + pad_h - r*dil_h, th >= 0, th % stride_h == 0, hi = th / stride_h < h. */
int ollie_eop_convt_gather(const ollie_conv_desc* desc, const void* y, int32_t y_dtype,
                           void* out, void* stream);

/* Band stages alone (layouts as in banded_bmm):
 *   g2bmm:   the G2BMM of Table 2, S fp32 [b][l][2w+1] from Q, K (dilated band evaluated
 *            per residue subsequence, section 6.4);
 *   softmax: the row softmax eOperator, P bf16 [b][l][2w+1] from S (flags:
 *            OLLIE_BAND_MASK_INVALID); 2w+1 <= 1024 (else OLLIE_EINVAL);
 *   gbmm:    the band-times-dense product, O [b][l][d] (out_dtype) from P and V.
 * Outputs must not overlap inputs (OLLIE_EINVAL). */
int ollie_band_g2bmm(const ollie_band_desc* desc, const void* q, const void* k, float* s,
                     void* stream);
int ollie_band_softmax(const ollie_band_desc* desc, const float* s, void* p, uint32_t flags,
                       void* stream);
int ollie_band_gbmm(const ollie_band_desc* desc, const void* p, const void* v, void* o,
                    void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OLLIE_H */
