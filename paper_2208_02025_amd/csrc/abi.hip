// Host side of the C ABI declared in include/ollie.h: argument validation, output and
// workspace sizing, and kernel launches on the caller's stream.  Every check runs
// before the first HIP call, so invalid arguments never reach the device.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>

#include "../../include/ollie.h"
#include "common.h"

using namespace ollie;

namespace {

thread_local char g_err[512];

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(OLLIE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Whether the byte ranges [a, a + na) and [b, b + nb) share a byte (null or empty
// ranges share none).
bool overlap(const void* a, size_t na, const void* b, size_t nb) {
    if (!a || !b || na == 0 || nb == 0) return false;
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

// Tile-configuration override bits of the flags (0 = automatic, else config + 1).
constexpr uint32_t kFusedTileBits = 0xffu << 16, kGemmTileBits = 0xfu << 24;
constexpr uint32_t kBandShapeBits = 0xffu << 16;
constexpr int kFusedTiles = 15, kGemmTiles = 5, kBandShapes = 4;
int fused_tile(uint32_t flags) { return (int)((flags & kFusedTileBits) >> 16) - 1; }
int gemm_tile(uint32_t flags) { return (int)((flags & kGemmTileBits) >> 24) - 1; }
int band_shape(uint32_t flags) { return (int)((flags & kBandShapeBits) >> 16) - 1; }

bool dtype_ok(int32_t d) { return d == OLLIE_F32 || d == OLLIE_BF16; }

size_t dsize(int32_t d) { return d == OLLIE_BF16 ? 2 : 4; }

constexpr int64_t kMaxElems = (int64_t)1 << 31;   // per-tensor element bound for 32-bit index math

// Overflow-checked product of non-negative values; -1 if it exceeds 2^62.
int64_t mul(int64_t a, int64_t b) {
    if (a < 0 || b < 0) return -1;
    if (a != 0 && b > ((int64_t)1 << 62) / a) return -1;
    return a * b;
}

int check_conv_geom(const ollie_conv_desc* d, int transposed, int64_t* ho, int64_t* wo) {
    if (!d) return fail(OLLIE_EINVAL, "desc is NULL");
    if (d->n < 1 || d->c < 1 || d->h < 1 || d->w < 1 || d->k < 1 || d->r < 1 || d->s < 1)
        return fail(OLLIE_EINVAL, "n, c, h, w, k, r, s must all be >= 1");
    if (d->stride_h < 1 || d->stride_w < 1) return fail(OLLIE_EINVAL, "stride must be >= 1");
    if (d->dil_h < 1 || d->dil_w < 1) return fail(OLLIE_EINVAL, "dilation must be >= 1");
    if (d->pad_h < 0 || d->pad_w < 0) return fail(OLLIE_EINVAL, "padding must be >= 0");
    if (transposed) {
        int mh = d->stride_h > d->dil_h ? d->stride_h : d->dil_h;
        int mw = d->stride_w > d->dil_w ? d->stride_w : d->dil_w;
        if (d->out_pad_h < 0 || d->out_pad_w < 0 || d->out_pad_h >= mh || d->out_pad_w >= mw)
            return fail(OLLIE_EINVAL, "out_pad must satisfy 0 <= out_pad < max(stride, dilation)");
    } else if (d->out_pad_h != 0 || d->out_pad_w != 0) {
        return fail(OLLIE_EINVAL, "out_pad is only meaningful for conv_transpose2d");
    }
    int64_t oh, ow;
    if (transposed) {
        oh = (d->h - 1) * d->stride_h - 2 * (int64_t)d->pad_h + (int64_t)d->dil_h * (d->r - 1) +
             d->out_pad_h + 1;
        ow = (d->w - 1) * d->stride_w - 2 * (int64_t)d->pad_w + (int64_t)d->dil_w * (d->s - 1) +
             d->out_pad_w + 1;
    } else {
        int64_t sh = d->h + 2 * (int64_t)d->pad_h - (int64_t)d->dil_h * (d->r - 1) - 1;
        int64_t sw = d->w + 2 * (int64_t)d->pad_w - (int64_t)d->dil_w * (d->s - 1) - 1;
        oh = sh < 0 ? 0 : sh / d->stride_h + 1;
        ow = sw < 0 ? 0 : sw / d->stride_w + 1;
    }
    if (oh < 1 || ow < 1) return fail(OLLIE_EINVAL, "output would be empty (ho=%lld, wo=%lld)",
                                      (long long)oh, (long long)ow);
    int64_t m = mul(mul(d->n, d->h), d->w);
    int64_t nc = mul(mul(d->r, d->s), d->k);
    int64_t outn = mul(mul(mul(d->n, oh), ow), d->k);
    int64_t yel = mul(m, nc);
    if (m < 0 || nc < 0 || outn < 0 || yel < 0 || mul(m, d->c) < 0 || mul(nc, d->c) < 0)
        return fail(OLLIE_EINVAL, "sizes overflow 64-bit arithmetic");
    if (m >= kMaxElems || nc >= kMaxElems || outn >= kMaxElems)
        return fail(OLLIE_EINVAL, "n*h*w, r*s*k and the output size must each be < 2^31");
    *ho = oh;
    *wo = ow;
    return OLLIE_OK;
}

ConvGeom conv_geom(const ollie_conv_desc* d, int64_t ho, int64_t wo) {
    ConvGeom g;
    g.n = d->n; g.c = d->c; g.h = d->h; g.w = d->w; g.k = d->k; g.r = d->r; g.s = d->s;
    g.ho = ho; g.wo = wo;
    g.sh = d->stride_h; g.sw = d->stride_w; g.ph = d->pad_h; g.pw = d->pad_w;
    g.dh = d->dil_h; g.dw = d->dil_w;
    return g;
}

int conv_form(int transposed, uint32_t flags) {
    return transposed ? kTransposed : (flags & OLLIE_DILATED_RESIDUES) ? kResidues : kForward;
}

bool fused_path(const ollie_conv_desc* d, int transposed, int64_t ho, int64_t wo,
                uint32_t flags) {
    return (flags & OLLIE_FUSE_EPILOGUE) && d->in_dtype == OLLIE_BF16 &&
           conv_fused_supported(conv_geom(d, ho, wo), conv_form(transposed, flags));
}

size_t conv_ws_plain(const ollie_conv_desc* d, int transposed, int64_t ho, int64_t wo,
                     uint32_t flags) {
    if (fused_path(d, transposed, ho, wo, flags)) return 0;
    return (size_t)(d->n * d->h * d->w) * (size_t)(d->r * d->s * d->k) *
           ((flags & OLLIE_Y_BF16) ? 2 : 4);
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The R x S -> 3x3 derived form (OLLIE_CONV_SPLIT_3X3): kernel blocks nbr x nbs, the
// relaxed taps er, es, and the 3x3 stage as a convolution descriptor X -> Z.
struct Split3 {
    int64_t nbr, nbs, er, es;
    ollie_conv_desc d3;
};

Split3 split3_of(const ollie_conv_desc* d) {
    Split3 q;
    q.nbr = (d->r + 2) / 3;
    q.nbs = (d->s + 2) / 3;
    q.er = 3 * q.nbr - d->r;
    q.es = 3 * q.nbs - d->s;
    q.d3 = *d;
    q.d3.k = q.nbr * q.nbs * d->k;
    q.d3.r = 3;
    q.d3.s = 3;
    q.d3.pad_h = d->pad_h + (int32_t)q.er;
    q.d3.pad_w = d->pad_w + (int32_t)q.es;
    q.d3.out_dtype = OLLIE_F32;
    return q;
}

// Checks the split form's extra conditions; fills the 3x3 stage's output size.
int check_split3(const ollie_conv_desc* d, int transposed, const Split3& q, int64_t* hz,
                 int64_t* wz) {
    if (transposed) return fail(OLLIE_EINVAL, "OLLIE_CONV_SPLIT_3X3 applies to derived_conv2d");
    if (d->stride_h != 1 || d->stride_w != 1 || d->dil_h != 1 || d->dil_w != 1)
        return fail(OLLIE_EINVAL, "OLLIE_CONV_SPLIT_3X3 needs stride 1 and dilation 1");
    if (d->pad_h > (1 << 28) || d->pad_w > (1 << 28) || d->r > (1 << 28) || d->s > (1 << 28))
        return fail(OLLIE_EINVAL, "sizes overflow 32-bit arithmetic");
    int st = check_conv_geom(&q.d3, 0, hz, wz);
    if (st) return st;
    if (mul(mul(mul(d->k, 9), q.nbr * q.nbs), d->c) >= kMaxElems)
        return fail(OLLIE_EINVAL, "split weights must have < 2^31 elements");
    return OLLIE_OK;
}

// Workspace of the split form: W3, then either Z (fp32; the 3x3 stage is the fused
// kernel) or the 3x3 stage's scope Y [n*h*w][9*nbr*nbs*K] (the GEMM stage, whose two
// eOperators run fused into one and never form Z).
size_t split3_ws(const ollie_conv_desc* d, const Split3& q, int64_t hz, int64_t wz,
                 uint32_t flags) {
    const size_t el = d->in_dtype == OLLIE_BF16 ? 2 : 4;
    const size_t w3 = (size_t)9 * (size_t)q.d3.k * (size_t)d->c * el;
    if (fused_path(&q.d3, 0, hz, wz, flags))
        return align256(w3) + (size_t)(d->n * hz * wz) * (size_t)q.d3.k * 4;
    return align256(w3) + (size_t)(d->n * d->h * d->w) * (size_t)(9 * q.d3.k) *
                              ((flags & OLLIE_Y_BF16) ? 2 : 4);
}

size_t conv_ws(const ollie_conv_desc* d, int transposed, int64_t ho, int64_t wo,
               uint32_t flags) {
    if (flags & OLLIE_CONV_SPLIT_3X3) {
        const Split3 q = split3_of(d);
        int64_t hz, wz;
        if (check_split3(d, transposed, q, &hz, &wz)) return 0;
        return split3_ws(d, q, hz, wz, flags & ~(uint32_t)OLLIE_CONV_SPLIT_3X3);
    }
    return conv_ws_plain(d, transposed, ho, wo, flags);
}

int check_gemm(int64_t m, int64_t n, int64_t k, const void* a, const void* b, const void* y,
               int32_t in_dtype, int32_t y_dtype) {
    if (m < 1 || n < 1 || k < 1) return fail(OLLIE_EINVAL, "m, n, k must be >= 1");
    if (mul(m, k) < 0 || mul(n, k) < 0 || mul(m, n) < 0)
        return fail(OLLIE_EINVAL, "sizes overflow 64-bit arithmetic");
    if (m >= kMaxElems || n >= kMaxElems) return fail(OLLIE_EINVAL, "m and n must be < 2^31");
    if (!a || !b || !y) return fail(OLLIE_EINVAL, "null tensor pointer");
    if (!dtype_ok(in_dtype) || !dtype_ok(y_dtype)) return fail(OLLIE_EDTYPE, "unknown dtype");
    if (!aligned16(a) || !aligned16(b) || !aligned16(y))
        return fail(OLLIE_EALIGN, "tensor pointers must be 16-byte aligned");
    if (in_dtype == OLLIE_BF16 && (k % 8) != 0)
        return fail(OLLIE_EALIGN, "bf16 operands need k %% 8 == 0 (16-byte rows), got k=%lld",
                    (long long)k);
    const size_t el = dsize(in_dtype), y_bytes = (size_t)(m * n) * dsize(y_dtype);
    if (overlap(y, y_bytes, a, (size_t)(m * k) * el) || overlap(y, y_bytes, b, (size_t)(n * k) * el))
        return fail(OLLIE_EINVAL, "y overlaps a or b");
    return OLLIE_OK;
}

// Validates an optional element-wise tail and converts it to the kernels' form.  The
// residual may be the output buffer itself (same pointer and dtype: each element is read
// and then written by one thread), but may not overlap it otherwise; the bias may not
// overlap it at all.
int make_epi(const ollie_conv_epilogue* e, const ollie_conv_desc* d, const void* out,
             size_t out_bytes, Epi* ep) {
    *ep = Epi{nullptr, nullptr, 0, 0, 0};
    if (!e) return OLLIE_OK;
    if (e->relu != 0 && e->relu != 1) return fail(OLLIE_EINVAL, "epilogue relu must be 0 or 1");
    if ((e->bias && !dtype_ok(e->bias_dtype)) || (e->residual && !dtype_ok(e->residual_dtype)))
        return fail(OLLIE_EDTYPE, "epilogue bias/residual dtype must be OLLIE_F32 or OLLIE_BF16");
    if (!aligned16(e->bias) || !aligned16(e->residual))
        return fail(OLLIE_EALIGN, "epilogue bias/residual pointers must be 16-byte aligned");
    const size_t n_out = out_bytes / dsize(d->out_dtype);
    if (overlap(e->bias, (size_t)d->k * dsize(e->bias_dtype), out, out_bytes))
        return fail(OLLIE_EINVAL, "epilogue bias overlaps the output");
    if (e->residual == out) {
        if (e->residual_dtype != d->out_dtype)
            return fail(OLLIE_EINVAL, "an in-place residual needs residual_dtype == out_dtype");
    } else if (overlap(e->residual, n_out * dsize(e->residual_dtype), out, out_bytes)) {
        return fail(OLLIE_EINVAL, "epilogue residual overlaps the output (other than in place)");
    }
    *ep = Epi{e->bias, e->residual, e->bias_dtype == OLLIE_BF16,
              e->residual_dtype == OLLIE_BF16, e->relu};
    return OLLIE_OK;
}

// dry = true: every check runs, and the call returns OLLIE_OK right before its first
// HIP call (nothing is launched, no pointer is dereferenced).
int conv_common(const ollie_conv_desc* d, int transposed, const void* x, const void* wt,
                void* out, void* ws, size_t ws_bytes, uint32_t flags,
                const ollie_conv_epilogue* epilogue, void* stream, bool dry = false);

// The R x S -> 3x3 derived form: the weight split, then
//   * the 3x3 stage as the fused kernel into Z (fp32), and the OffsetAdd over the kernel
//     blocks (taps spaced 3 apart in Z, shifted by er, es); or
//   * the 3x3 stage's GEMM into its scope Y, and its OffsetAdd and the block OffsetAdd
//     fused into one eOperator over Y (Z is never formed);
// the last kernel carries the element-wise tail.
int conv_split3(const ollie_conv_desc* d, int transposed, const void* x, const void* wt,
                void* out, void* ws, size_t ws_bytes, uint32_t flags, const Epi& epi,
                int64_t ho, int64_t wo, void* stream, bool dry) {
    const Split3 q = split3_of(d);
    int64_t hz, wz;
    int st = check_split3(d, transposed, q, &hz, &wz);
    if (st) return st;
    const size_t need = split3_ws(d, q, hz, wz, flags);
    if (!ws) return fail(OLLIE_EINVAL, "null workspace pointer (the split form needs W3 and Z "
                                       "or the 3x3 stage's scope)");
    if (ws_bytes < need)
        return fail(OLLIE_EWORKSPACE, "workspace too small: need %zu bytes, got %zu", need,
                    ws_bytes);
    if (!aligned16(x) || !aligned16(wt) || !aligned16(out) || !aligned16(ws))
        return fail(OLLIE_EALIGN, "tensor and workspace pointers must be 16-byte aligned");
    const size_t el = d->in_dtype == OLLIE_BF16 ? 2 : 4;
    const size_t w3_bytes = align256((size_t)9 * (size_t)q.d3.k * (size_t)d->c * el);
    char* w3 = static_cast<char*>(ws);
    char* z = w3 + w3_bytes;   // Z, or the 3x3 stage's scope Y
    const bool fused3 = fused_path(&q.d3, 0, hz, wz, flags);
    const int64_t m = d->n * d->h * d->w;
    const int y_bf16 = (flags & OLLIE_Y_BF16) ? 1 : 0;
    // everything the 3x3 stage checks, before the first launch
    if (!fused3) {
        st = check_gemm(m, 9 * q.d3.k, d->c, x, w3, z, d->in_dtype,
                        y_bf16 ? OLLIE_BF16 : OLLIE_F32);
        if (st) return st;
    }
    if (dry) return OLLIE_OK;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = launch_split_weights_3x3(conv_geom(d, ho, wo), wt, w3,
                                            d->in_dtype == OLLIE_BF16, s);
    if (e != hipSuccess) return hip_fail(e, "weight split launch");
    if (!fused3) {
        e = launch_gemm_nt(m, 9 * q.d3.k, d->c, x, w3, z, d->in_dtype == OLLIE_BF16, y_bf16,
                           gemm_tile(flags), s);
        if (e != hipSuccess) return hip_fail(e, "3x3 stage GEMM launch");
        e = launch_eop_split3_chain(conv_geom(d, ho, wo), z, y_bf16, out,
                                    d->out_dtype == OLLIE_BF16, epi, s);
        if (e != hipSuccess) return hip_fail(e, "fused eOperator chain launch");
        return OLLIE_OK;
    }
    st = conv_common(&q.d3, 0, x, w3, z, nullptr, 0, flags, nullptr, stream);
    if (st) return st;
    ConvGeom gb = conv_geom(d, ho, wo);
    gb.h = hz;
    gb.w = wz;
    gb.r = q.nbr;
    gb.s = q.nbs;
    gb.ph = -(int32_t)q.er;
    gb.pw = -(int32_t)q.es;
    gb.dh = 3;
    gb.dw = 3;
    e = launch_eop_gather(gb, 0, z, 0, out, d->out_dtype == OLLIE_BF16, epi, s);
    if (e != hipSuccess) return hip_fail(e, "block OffsetAdd launch");
    return OLLIE_OK;
}

int conv_common(const ollie_conv_desc* d, int transposed, const void* x, const void* wt,
                void* out, void* ws, size_t ws_bytes, uint32_t flags,
                const ollie_conv_epilogue* epilogue, void* stream, bool dry) {
    int64_t ho, wo;
    int st = check_conv_geom(d, transposed, &ho, &wo);
    if (st) return st;
    if (flags & ~(uint32_t)(OLLIE_Y_BF16 | OLLIE_FUSE_EPILOGUE | OLLIE_DILATED_RESIDUES |
                            OLLIE_CONV_SPLIT_3X3 | kFusedTileBits | kGemmTileBits))
        return fail(OLLIE_EINVAL, "unknown flag bits 0x%x", flags);
    if (fused_tile(flags) >= kFusedTiles || gemm_tile(flags) >= kGemmTiles)
        return fail(OLLIE_EINVAL, "tile override out of range (fused 0..%d, GEMM 0..%d)",
                    kFusedTiles - 1, kGemmTiles - 1);
    if (!x || !wt || !out) return fail(OLLIE_EINVAL, "null tensor pointer");
    if (!dtype_ok(d->in_dtype) || !dtype_ok(d->out_dtype))
        return fail(OLLIE_EDTYPE, "in_dtype/out_dtype must be OLLIE_F32 or OLLIE_BF16");
    const size_t out_bytes = (size_t)(d->n * ho * wo * d->k) * dsize(d->out_dtype);
    Epi epi;
    st = make_epi(epilogue, d, out, out_bytes, &epi);
    if (st) return st;
    {
        const size_t in_el = dsize(d->in_dtype);
        const size_t x_bytes = (size_t)(d->n * d->h * d->w) * (size_t)d->c * in_el;
        const size_t wt_bytes = (size_t)(d->r * d->s * d->k) * (size_t)d->c * in_el;
        // the part of the workspace the call would use (a short one fails later, with
        // OLLIE_EWORKSPACE)
        size_t ws_used = ws ? conv_ws(d, transposed, ho, wo, flags) : 0;
        ws_used = ws_used < ws_bytes ? ws_used : ws_bytes;
        if (overlap(out, out_bytes, x, x_bytes) || overlap(out, out_bytes, wt, wt_bytes) ||
            overlap(out, out_bytes, ws, ws_used))
            return fail(OLLIE_EINVAL, "out overlaps x, wt or the workspace");
        if (overlap(ws, ws_used, x, x_bytes) || overlap(ws, ws_used, wt, wt_bytes))
            return fail(OLLIE_EINVAL, "the workspace overlaps x or wt");
    }
    if (flags & OLLIE_CONV_SPLIT_3X3) {
        if (flags & OLLIE_DILATED_RESIDUES)
            return fail(OLLIE_EINVAL, "OLLIE_CONV_SPLIT_3X3 and OLLIE_DILATED_RESIDUES exclude "
                                      "each other");
        return conv_split3(d, transposed, x, wt, out, ws, ws_bytes,
                           flags & ~(uint32_t)OLLIE_CONV_SPLIT_3X3, epi, ho, wo, stream, dry);
    }
    if ((flags & OLLIE_DILATED_RESIDUES) && !fused_path(d, transposed, ho, wo, flags))
        return fail(OLLIE_EINVAL,
                    "OLLIE_DILATED_RESIDUES needs OLLIE_FUSE_EPILOGUE, stride 1, bf16 inputs, "
                    "c %% 64 == 0 and dil_h*dil_w <= 16");
    if (fused_path(d, transposed, ho, wo, flags)) {
        if (!aligned16(x) || !aligned16(wt) || !aligned16(out))
            return fail(OLLIE_EALIGN, "tensor pointers must be 16-byte aligned");
        if (dry) return OLLIE_OK;
        hipError_t e = launch_conv_fused(conv_geom(d, ho, wo), conv_form(transposed, flags), x,
                                         wt, out, d->out_dtype == OLLIE_BF16, epi,
                                         fused_tile(flags), (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "fused GEMM+eOperator launch");
        return OLLIE_OK;
    }
    if (!ws) return fail(OLLIE_EINVAL, "null workspace pointer (the two-stage path needs Y)");
    size_t need = conv_ws(d, transposed, ho, wo, flags);
    if (ws_bytes < need)
        return fail(OLLIE_EWORKSPACE, "workspace too small: need %zu bytes, got %zu", need,
                    ws_bytes);
    if (!aligned16(x) || !aligned16(wt) || !aligned16(out) || !aligned16(ws))
        return fail(OLLIE_EALIGN, "tensor and workspace pointers must be 16-byte aligned");
    int64_t m = d->n * d->h * d->w, nc = d->r * d->s * d->k;
    st = check_gemm(m, nc, d->c, x, wt, ws, d->in_dtype,
                    (flags & OLLIE_Y_BF16) ? OLLIE_BF16 : OLLIE_F32);
    if (st) return st;
    if (dry) return OLLIE_OK;
    hipStream_t s = (hipStream_t)stream;
    const int y_bf16 = (flags & OLLIE_Y_BF16) ? 1 : 0;
    hipError_t e = launch_gemm_nt(m, nc, d->c, x, wt, ws, d->in_dtype == OLLIE_BF16, y_bf16,
                                  gemm_tile(flags), s);
    if (e != hipSuccess) return hip_fail(e, "GEMM stage launch");
    e = launch_eop_gather(conv_geom(d, ho, wo), transposed, ws, y_bf16, out,
                          d->out_dtype == OLLIE_BF16, epi, s);
    if (e != hipSuccess) return hip_fail(e, "eOperator launch");
    return OLLIE_OK;
}

int check_band(const ollie_band_desc* d) {
    if (!d) return fail(OLLIE_EINVAL, "desc is NULL");
    if (d->b < 1 || d->l < 1 || d->w < 0 || d->dilation < 1)
        return fail(OLLIE_EINVAL, "need b >= 1, l >= 1, w >= 0, dilation >= 1");
    if (d->d != 64) return fail(OLLIE_EINVAL, "head dimension d must be 64, got %lld",
                                (long long)d->d);
    if (d->b > 65535 || d->dilation > 65535)
        return fail(OLLIE_EINVAL, "b and dilation must be <= 65535");
    if (d->in_dtype != OLLIE_BF16) return fail(OLLIE_EDTYPE, "Q, K, V must be bf16");
    if (!dtype_ok(d->out_dtype)) return fail(OLLIE_EDTYPE, "out_dtype must be F32 or BF16");
    int64_t nb = mul(2, d->w) + 1;
    if (mul(mul(d->b, d->l), nb) < 0 || mul(mul(d->b, d->l), d->d) < 0 || d->w > ((int64_t)1 << 30))
        return fail(OLLIE_EINVAL, "sizes overflow 64-bit arithmetic");
    if (mul(d->b, d->l) >= kMaxElems) return fail(OLLIE_EINVAL, "b*l must be < 2^31");
    const int64_t tiles = ((d->l + d->dilation - 1) / d->dilation + 63) / 64;
    if (mul(mul(tiles, d->dilation), d->b) >= kMaxElems)
        return fail(OLLIE_EINVAL, "too many (batch, residue, 64-row) tiles");
    return OLLIE_OK;
}

BandGeom band_geom(const ollie_band_desc* d) {
    BandGeom g;
    g.b = d->b; g.l = d->l; g.d = d->d; g.w = d->w; g.dil = d->dilation; g.scale = d->scale;
    return g;
}

size_t band_s_bytes(const ollie_band_desc* d) {
    return (size_t)(d->b * d->l) * (size_t)(2 * d->w + 1) * 4;
}
size_t band_p_offset(const ollie_band_desc* d) { return (band_s_bytes(d) + 255) & ~(size_t)255; }
size_t band_p_bytes(const ollie_band_desc* d) {
    return (size_t)(d->b * d->l) * (size_t)(2 * d->w + 1) * 2;
}
size_t band_qkv_bytes(const ollie_band_desc* d) { return (size_t)(d->b * d->l * d->d) * 2; }

constexpr int64_t kSoftmaxMaxBand = 16 * 64;   // register-resident row length of the staged softmax

// derived_conv2d with an optional element-wise tail (the exported _ex entry point and
// the allocation-free variant both end here).
int derived_conv2d_ex_impl(const ollie_conv_desc* desc, const void* x, const void* wt,
                           void* out, void* ws, size_t ws_bytes, uint32_t flags,
                           const ollie_conv_epilogue* epi, void* stream, bool dry = false) {
    if (flags & OLLIE_DILATED_RESIDUES)
        return fail(OLLIE_EINVAL, "OLLIE_DILATED_RESIDUES applies to derived_dilated_conv2d");
    if (desc && (desc->dil_h != 1 || desc->dil_w != 1))
        return fail(OLLIE_EINVAL, "derived_conv2d takes dilation 1; use derived_dilated_conv2d");
    return conv_common(desc, 0, x, wt, out, ws, ws_bytes, flags, epi, stream, dry);
}

}  // namespace

// The library's own workspace for callers that cannot allocate (ollie_derived_conv2d_
// noalloc): a file-scope device array, one copy per GPU, alive until the process ends.
// In host code `scratch` names a host-side stand-in, not device memory: kernels and
// copies get the device address that hipGetSymbolAddress returns for the current
// device, looked up on the first such call on that device and kept per device.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch array, or an OLLIE_EHIP status.
int scratch_ptr(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(OLLIE_EINVAL, "device index %d beyond the %d the scratch table holds", dev,
                    kMaxDevices);
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        // idempotent: racing first calls on one device store the same address
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(OLLIE_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return OLLIE_OK;
}

}  // namespace

#pragma GCC visibility push(default)
extern "C" {

const char* ollie_last_error(void) { return g_err; }

const char* ollie_version(void) { return "ollie-mi355x 0.2.0 (gfx950)"; }

int ollie_conv_out_hw(const ollie_conv_desc* desc, int transposed, int64_t* ho, int64_t* wo) {
    g_err[0] = 0;
    if (!ho || !wo) return fail(OLLIE_EINVAL, "ho/wo pointers are NULL");
    return check_conv_geom(desc, transposed ? 1 : 0, ho, wo);
}

size_t ollie_conv_workspace_bytes(const ollie_conv_desc* desc, int transposed, uint32_t flags) {
    int64_t ho, wo;
    if (check_conv_geom(desc, transposed ? 1 : 0, &ho, &wo)) return 0;
    return conv_ws(desc, transposed ? 1 : 0, ho, wo, flags);
}

size_t ollie_band_workspace_bytes(const ollie_band_desc* desc, uint32_t flags) {
    if (check_band(desc)) return 0;
    if (!(flags & OLLIE_BAND_STAGED)) return 0;
    if (2 * desc->w + 1 > kSoftmaxMaxBand) return 0;   // banded_bmm rejects this band
    return band_p_offset(desc) + band_p_bytes(desc);
}

int ollie_derived_conv2d_ex(const ollie_conv_desc* desc, const void* x, const void* wt, void* out,
                      void* ws, size_t ws_bytes, uint32_t flags,
                      const ollie_conv_epilogue* epi, void* stream) {
    g_err[0] = 0;
    return derived_conv2d_ex_impl(desc, x, wt, out, ws, ws_bytes, flags, epi, stream);
}

int ollie_derived_dilated_conv2d_ex(const ollie_conv_desc* desc, const void* x, const void* wt,
                              void* out, void* ws, size_t ws_bytes, uint32_t flags,
                              const ollie_conv_epilogue* epi, void* stream) {
    g_err[0] = 0;
    if (flags & OLLIE_CONV_SPLIT_3X3)
        return fail(OLLIE_EINVAL, "OLLIE_CONV_SPLIT_3X3 applies to derived_conv2d");
    return conv_common(desc, 0, x, wt, out, ws, ws_bytes, flags, epi, stream);
}

int ollie_derived_conv_transpose2d_ex(const ollie_conv_desc* desc, const void* x, const void* wt,
                                void* out, void* ws, size_t ws_bytes, uint32_t flags,
                                const ollie_conv_epilogue* epi, void* stream) {
    g_err[0] = 0;
    if (flags & OLLIE_DILATED_RESIDUES)
        return fail(OLLIE_EINVAL, "OLLIE_DILATED_RESIDUES applies to derived_dilated_conv2d");
    return conv_common(desc, 1, x, wt, out, ws, ws_bytes, flags, epi, stream);
}

int derived_conv2d(const ollie_conv_desc* desc, const void* x, const void* wt, void* out,
                   void* ws, size_t ws_bytes, uint32_t flags, void* stream) {
    return ollie_derived_conv2d_ex(desc, x, wt, out, ws, ws_bytes, flags, nullptr, stream);
}

int ollie_derived_conv2d_noalloc(const ollie_conv_desc* desc, const void* x, const void* wt,
                                 void* out, uint32_t flags, void* stream) {
    g_err[0] = 0;
    int64_t ho, wo;
    int st = check_conv_geom(desc, 0, &ho, &wo);
    if (st) return st;
    const size_t need = ollie_conv_workspace_bytes(desc, 0, flags);
    if (need > kScratchBytes)
        return fail(OLLIE_EWORKSPACE,
                    "needs %zu bytes of workspace; the static scratch holds %zu (use "
                    "derived_conv2d with a caller workspace)", need, kScratchBytes);
    // Every argument check first, without a HIP call: a dry run of the same path whose
    // workspace is a placeholder range at 2^63 (the kernel half of the address space,
    // which no caller buffer can occupy, so the overlap checks see the scratch as what
    // it is: disjoint from the caller's tensors).  Nothing is dereferenced or launched.
    void* const placeholder = reinterpret_cast<void*>(uintptr_t(1) << 63);
    st = derived_conv2d_ex_impl(desc, x, wt, out, need ? placeholder : nullptr,
                                need ? kScratchBytes : 0, flags, nullptr, stream, true);
    if (st) return st;
    void* ws = nullptr;
    if (need) {
        st = scratch_ptr(&ws);
        if (st) return st;
    }
    return derived_conv2d_ex_impl(desc, x, wt, out, ws, need ? kScratchBytes : 0, flags,
                                  nullptr, stream);
}

int derived_dilated_conv2d(const ollie_conv_desc* desc, const void* x, const void* wt,
                           void* out, void* ws, size_t ws_bytes, uint32_t flags, void* stream) {
    return ollie_derived_dilated_conv2d_ex(desc, x, wt, out, ws, ws_bytes, flags, nullptr, stream);
}

int derived_conv_transpose2d(const ollie_conv_desc* desc, const void* x, const void* wt,
                             void* out, void* ws, size_t ws_bytes, uint32_t flags,
                             void* stream) {
    return ollie_derived_conv_transpose2d_ex(desc, x, wt, out, ws, ws_bytes, flags, nullptr, stream);
}

int banded_bmm(const ollie_band_desc* desc, const void* q, const void* k, const void* v,
               void* o, float* s_out, void* ws, size_t ws_bytes, uint32_t flags, void* stream) {
    g_err[0] = 0;
    int st = check_band(desc);
    if (st) return st;
    if (flags & ~(uint32_t)(OLLIE_BAND_STAGED | OLLIE_BAND_MASK_INVALID | kBandShapeBits))
        return fail(OLLIE_EINVAL, "unknown flag bits 0x%x", flags);
    if (band_shape(flags) >= kBandShapes)
        return fail(OLLIE_EINVAL, "band shape override out of range (0..%d)", kBandShapes - 1);
    if (!q || !k || !v || !o) return fail(OLLIE_EINVAL, "null tensor pointer");
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
        return fail(OLLIE_EALIGN, "tensor pointers must be 16-byte aligned");
    const int mask = (flags & OLLIE_BAND_MASK_INVALID) ? 1 : 0;
    const int o_bf16 = desc->out_dtype == OLLIE_BF16;
    {
        const size_t in_bytes = band_qkv_bytes(desc);
        const size_t o_bytes = (size_t)(desc->b * desc->l * desc->d) * dsize(desc->out_dtype);
        size_t ws_used = (flags & OLLIE_BAND_STAGED) && ws
                             ? band_p_offset(desc) + band_p_bytes(desc) : 0;
        ws_used = ws_used < ws_bytes ? ws_used : ws_bytes;
        const size_t s_bytes = s_out ? band_s_bytes(desc) : 0;
        const void* ins[3] = {q, k, v};
        for (const void* t : ins)
            if (overlap(o, o_bytes, t, in_bytes) || overlap(s_out, s_bytes, t, in_bytes) ||
                overlap(ws, ws_used, t, in_bytes))
                return fail(OLLIE_EINVAL, "o, s_out or the workspace overlaps q, k or v");
        if (overlap(o, o_bytes, ws, ws_used) || overlap(o, o_bytes, s_out, s_bytes) ||
            overlap(s_out, s_bytes, ws, ws_used))
            return fail(OLLIE_EINVAL, "o, s_out and the workspace must not overlap");
    }
    hipStream_t s = (hipStream_t)stream;
    BandGeom g = band_geom(desc);
    if (!(flags & OLLIE_BAND_STAGED)) {
        if (s_out) return fail(OLLIE_EINVAL, "s_out needs OLLIE_BAND_STAGED");
        hipError_t e = launch_band_fused(g, q, k, v, o, o_bf16, mask, band_shape(flags), s);
        if (e != hipSuccess) return hip_fail(e, "fused band launch");
        return OLLIE_OK;
    }
    if (2 * desc->w + 1 > kSoftmaxMaxBand)
        return fail(OLLIE_EINVAL, "staged path needs 2w+1 <= %lld", (long long)kSoftmaxMaxBand);
    size_t need = band_p_offset(desc) + band_p_bytes(desc);
    if (!ws) return fail(OLLIE_EINVAL, "staged path needs a workspace");
    if (ws_bytes < need)
        return fail(OLLIE_EWORKSPACE, "workspace too small: need %zu bytes, got %zu", need,
                    ws_bytes);
    if (!aligned16(ws) || (s_out && !aligned16(s_out)))
        return fail(OLLIE_EALIGN, "workspace and s_out must be 16-byte aligned");
    float* sbuf = s_out ? s_out : (float*)ws;
    void* pbuf = (char*)ws + band_p_offset(desc);
    hipError_t e = launch_band_g2bmm(g, q, k, sbuf, s);
    if (e != hipSuccess) return hip_fail(e, "G2BMM launch");
    e = launch_band_softmax(g, sbuf, pbuf, mask, s);
    if (e != hipSuccess) return hip_fail(e, "softmax launch");
    e = launch_band_gbmm(g, pbuf, v, o, o_bf16, s);
    if (e != hipSuccess) return hip_fail(e, "GBMM launch");
    return OLLIE_OK;
}

int ollie_gemm_nt(int64_t m, int64_t n, int64_t k, const void* a, const void* b, void* y,
                  int32_t in_dtype, int32_t y_dtype, void* stream) {
    g_err[0] = 0;
    int st = check_gemm(m, n, k, a, b, y, in_dtype, y_dtype);
    if (st) return st;
    hipError_t e = launch_gemm_nt(m, n, k, a, b, y, in_dtype == OLLIE_BF16,
                                  y_dtype == OLLIE_BF16, -1, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "GEMM launch");
    return OLLIE_OK;
}

}  // extern "C"

namespace {

int eop_stage(const ollie_conv_desc* desc, int transposed, const void* y, int32_t y_dtype,
              void* out, void* stream) {
    g_err[0] = 0;
    int64_t ho, wo;
    int st = check_conv_geom(desc, transposed, &ho, &wo);
    if (st) return st;
    if (!y || !out) return fail(OLLIE_EINVAL, "null tensor pointer");
    if (!dtype_ok(y_dtype) || !dtype_ok(desc->out_dtype)) return fail(OLLIE_EDTYPE, "unknown dtype");
    if (!aligned16(y) || !aligned16(out))
        return fail(OLLIE_EALIGN, "tensor pointers must be 16-byte aligned");
    const size_t y_bytes = (size_t)(desc->n * desc->h * desc->w) *
                           (size_t)(desc->r * desc->s * desc->k) * dsize(y_dtype);
    if (overlap(out, (size_t)(desc->n * ho * wo * desc->k) * dsize(desc->out_dtype), y, y_bytes))
        return fail(OLLIE_EINVAL, "out overlaps y");
    hipError_t e = launch_eop_gather(conv_geom(desc, ho, wo), transposed, y,
                                     y_dtype == OLLIE_BF16, out, desc->out_dtype == OLLIE_BF16,
                                     Epi{nullptr, nullptr, 0, 0, 0}, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "eOperator launch");
    return OLLIE_OK;
}

}  // namespace

extern "C" {

int ollie_eop_offset_sum(const ollie_conv_desc* desc, const void* y, int32_t y_dtype,
                         void* out, void* stream) {
    return eop_stage(desc, 0, y, y_dtype, out, stream);
}

int ollie_eop_convt_gather(const ollie_conv_desc* desc, const void* y, int32_t y_dtype,
                           void* out, void* stream) {
    return eop_stage(desc, 1, y, y_dtype, out, stream);
}

int ollie_band_g2bmm(const ollie_band_desc* desc, const void* q, const void* k, float* s,
                     void* stream) {
    g_err[0] = 0;
    int st = check_band(desc);
    if (st) return st;
    if (!q || !k || !s) return fail(OLLIE_EINVAL, "null tensor pointer");
    if (!aligned16(q) || !aligned16(k) || !aligned16(s))
        return fail(OLLIE_EALIGN, "tensor pointers must be 16-byte aligned");
    if (overlap(s, band_s_bytes(desc), q, band_qkv_bytes(desc)) ||
        overlap(s, band_s_bytes(desc), k, band_qkv_bytes(desc)))
        return fail(OLLIE_EINVAL, "s overlaps q or k");
    hipError_t e = launch_band_g2bmm(band_geom(desc), q, k, s, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "G2BMM launch");
    return OLLIE_OK;
}

int ollie_band_softmax(const ollie_band_desc* desc, const float* s, void* p, uint32_t flags,
                       void* stream) {
    g_err[0] = 0;
    int st = check_band(desc);
    if (st) return st;
    if (flags & ~(uint32_t)OLLIE_BAND_MASK_INVALID)
        return fail(OLLIE_EINVAL, "unknown flag bits 0x%x", flags);
    if (!s || !p) return fail(OLLIE_EINVAL, "null tensor pointer");
    if (2 * desc->w + 1 > kSoftmaxMaxBand)
        return fail(OLLIE_EINVAL, "softmax stage needs 2w+1 <= %lld", (long long)kSoftmaxMaxBand);
    if (!aligned16(s) || !aligned16(p))
        return fail(OLLIE_EALIGN, "tensor pointers must be 16-byte aligned");
    if (overlap(p, band_p_bytes(desc), s, band_s_bytes(desc)))
        return fail(OLLIE_EINVAL, "p overlaps s");
    hipError_t e = launch_band_softmax(band_geom(desc), s, p,
                                       (flags & OLLIE_BAND_MASK_INVALID) ? 1 : 0,
                                       (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "softmax launch");
    return OLLIE_OK;
}

int ollie_band_gbmm(const ollie_band_desc* desc, const void* p, const void* v, void* o,
                    void* stream) {
    g_err[0] = 0;
    int st = check_band(desc);
    if (st) return st;
    if (!p || !v || !o) return fail(OLLIE_EINVAL, "null tensor pointer");
    if (!aligned16(p) || !aligned16(v) || !aligned16(o))
        return fail(OLLIE_EALIGN, "tensor pointers must be 16-byte aligned");
    const size_t o_bytes = (size_t)(desc->b * desc->l * desc->d) * dsize(desc->out_dtype);
    if (overlap(o, o_bytes, p, band_p_bytes(desc)) || overlap(o, o_bytes, v, band_qkv_bytes(desc)))
        return fail(OLLIE_EINVAL, "o overlaps p or v");
    hipError_t e = launch_band_gbmm(band_geom(desc), p, v, o, desc->out_dtype == OLLIE_BF16,
                                    (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "GBMM launch");
    return OLLIE_OK;
}

}  // extern "C"
#pragma GCC visibility pop
