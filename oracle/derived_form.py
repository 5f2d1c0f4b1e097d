"""Second CPU evaluation of the operators, in the derived form (test infrastructure only).

Where oracle.c evaluates each operator as its nested-summation definition, this
module evaluates the *derived* expression the method reaches, in float64 NumPy:

* convolution family: summation splitting (section 4.2) turns the sum over (c,r,s)
  into an inner scope over c -- one matrix product Y = A' @ K'  with the layouts of
  Eq. (3) and Eq. (4) -- and an outer eOperator that sums the partials of Y over
  (r,s) through the substituted indices (the OffsetAdd of section 2; the selective
  add of section 6.3 for the transposed case);
* the R x S -> 3x3 rewrite (Conv5x5 -> Conv3x3, section 6 / Table 3): the tap range
  is relaxed to whole 3x3 blocks with zero weights (boundary relaxing), the tap index
  substituted as r = 3a + r' (variable substitution), and the sum split into an inner
  3x3 convolution over (r', s', c) with one output-channel group per block (a, b) and
  an outer OffsetAdd over the blocks with offset step 3 (summation splitting); and the
  same form with its two consecutive eOperators fused into one over the 3x3 stage's
  scope (eOperator fusion, section 5.4), which never forms the intermediate Z;
* banded matmul: the dilated band is split by residue i mod dil into non-dilated
  bands over strided subsequences (the dilated-to-non-dilated G2BMM rewrite of
  section 6.4), each evaluated with dense matrix products, then re-interleaved.

The matrix product is a library step (numpy.matmul); the eOperators are written
out as explicit loops over taps.  Only used on small shapes to cross-check oracle.c.
"""
from __future__ import annotations

import numpy as np


def conv_out_size(n_in, r, stride, pad, dil, out_pad=0, transposed=False):
    if transposed:
        return (n_in - 1) * stride - 2 * pad + dil * (r - 1) + out_pad + 1
    span = n_in + 2 * pad - dil * (r - 1) - 1
    return 0 if span < 0 else span // stride + 1


def gemm_stage(x, wt):
    """Inner scope: Y[m, n] = sum_c A'[m, c] K'[c, n].

    A'[m, c] = X[n_, h, w, c] with m = (n_*H + h)*W + w      (Eq. 3, batch added)
    K'[c, n] = Wt[r, s, k, c] with n = (r*S + s)*K + k        (Eq. 4, f = k)
    """
    n_, h, w, c = x.shape
    r, s, k, c2 = wt.shape
    assert c == c2
    a_mat = x.reshape(n_ * h * w, c).astype(np.float64)
    k_mat = wt.reshape(r * s * k, c).astype(np.float64).T
    return a_mat @ k_mat                                  # [M, R*S*K]


def offset_add(y, x_shape, wt_shape, stride, pad, dil):
    """OffsetAdd eOperator: out[n,ho,wo,k] = sum_{r,s} Y[(n,hi,wi), (r,s,k)] over taps
    whose input pixel hi = ho*sh - ph + r*dh, wi = wo*sw - pw + s*dw lies inside X
    (taps outside read the zero padding and are dropped: boundary tightening)."""
    n_, h, w, _ = x_shape
    r_n, s_n, k, _ = wt_shape
    (sh, sw), (ph, pw), (dh, dw) = stride, pad, dil
    ho_n = conv_out_size(h, r_n, sh, ph, dh)
    wo_n = conv_out_size(w, s_n, sw, pw, dw)
    y6 = y.reshape(n_, h, w, r_n, s_n, k)
    out = np.zeros((n_, ho_n, wo_n, k), dtype=np.float64)
    for r in range(r_n):
        for s in range(s_n):
            for ho in range(ho_n):
                hi = ho * sh - ph + r * dh
                if hi < 0 or hi >= h:
                    continue
                for wo in range(wo_n):
                    wi = wo * sw - pw + s * dw
                    if wi < 0 or wi >= w:
                        continue
                    out[:, ho, wo, :] += y6[:, hi, wi, r, s, :]
    return out


def selective_add(y, x_shape, wt_shape, stride, pad, dil, out_pad):
    """Transposed-convolution eOperator: each output sums only the partials whose
    input pixel maps onto it, th = ho + ph - r*dh with th >= 0, th % sh == 0 and
    th // sh < H (and likewise along w)."""
    n_, h, w, _ = x_shape
    r_n, s_n, k, _ = wt_shape
    (sh, sw), (ph, pw), (dh, dw), (oph, opw) = stride, pad, dil, out_pad
    ho_n = conv_out_size(h, r_n, sh, ph, dh, oph, True)
    wo_n = conv_out_size(w, s_n, sw, pw, dw, opw, True)
    y6 = y.reshape(n_, h, w, r_n, s_n, k)
    out = np.zeros((n_, ho_n, wo_n, k), dtype=np.float64)
    for r in range(r_n):
        for s in range(s_n):
            for ho in range(ho_n):
                th = ho + ph - r * dh
                if th < 0 or th % sh != 0 or th // sh >= h:
                    continue
                for wo in range(wo_n):
                    tw = wo + pw - s * dw
                    if tw < 0 or tw % sw != 0 or tw // sw >= w:
                        continue
                    out[:, ho, wo, :] += y6[:, th // sh, tw // sw, r, s, :]
    return out


def derived_conv2d(x, wt, stride, pad, dil):
    y = gemm_stage(x, wt)
    return offset_add(y, x.shape, wt.shape, stride, pad, dil)


def derived_conv_transpose2d(x, wt, stride, pad, dil, out_pad=(0, 0)):
    y = gemm_stage(x, wt)
    return selective_add(y, x.shape, wt.shape, stride, pad, dil, out_pad)


def split_weights_3x3(wt):
    """W3[r'][s'][(a*nbs + b)*K + k][c] = Wt[3a + r'][3b + s'][k][c], zero where the
    block overhangs the R x S kernel (the relaxed taps)."""
    r_n, s_n, k, c = wt.shape
    nbr, nbs = -(-r_n // 3), -(-s_n // 3)
    w6 = np.zeros((3 * nbr, 3 * nbs, k, c), dtype=np.float64)
    w6[:r_n, :s_n] = wt
    w3 = np.zeros((3, 3, nbr * nbs * k, c), dtype=np.float64)
    for a in range(nbr):
        for b in range(nbs):
            g = a * nbs + b
            w3[:, :, g * k:(g + 1) * k, :] = w6[3 * a:3 * a + 3, 3 * b:3 * b + 3]
    return w3


def derived_conv2d_split3x3(x, wt, pad):
    """Stride-1, dilation-1 convolution in the 3x3 derived form: the inner 3x3 stage
    (itself GEMM + OffsetAdd) with padding pad + er, then the block OffsetAdd
    out[ho][wo][k] = sum_{a,b} Z[ho + er + 3a][wo + es + 3b][(a*nbs + b)*K + k]."""
    n_, h, w, _ = x.shape
    r_n, s_n, k, _ = wt.shape
    ph, pw = pad
    nbr, nbs = -(-r_n // 3), -(-s_n // 3)
    er, es = 3 * nbr - r_n, 3 * nbs - s_n
    w3 = split_weights_3x3(wt)
    z = derived_conv2d(x, w3, (1, 1), (ph + er, pw + es), (1, 1))   # [n, hz, wz, nbr*nbs*K]
    ho_n = conv_out_size(h, r_n, 1, ph, 1)
    wo_n = conv_out_size(w, s_n, 1, pw, 1)
    out = np.zeros((n_, ho_n, wo_n, k), dtype=np.float64)
    for a in range(nbr):
        for b in range(nbs):
            g = a * nbs + b
            out += z[:, er + 3 * a:er + 3 * a + ho_n, es + 3 * b:es + 3 * b + wo_n,
                     g * k:(g + 1) * k]
    return out


def derived_conv2d_split3x3_chain(x, wt, pad):
    """The 3x3 derived form with its two consecutive eOperators fused into one
    (eOperator fusion, section 5.4).  The inner 3x3 stage's scope is
        Y[m, (r'*3 + s')*nbr*nbs*K + (a*nbs + b)*K + k]   (GEMM with the split weights);
    its OffsetAdd (padding pad + er, taps r', s') substituted into the block OffsetAdd
    (offset step 3, shift er) gives one eOperator over Y,
        out[n, ho, wo, k] = sum_{a, b, r', s'} Y[(n, hi, wi), ((r'*3 + s')*nbr*nbs + a*nbs + b)*K + k]
    with hi = ho + er + 3a - (ph + er) + r' = ho - ph + 3a + r' (likewise wi), over the
    input pixels inside the image.  Every tap of the relaxed 3*nbr x 3*nbs kernel is
    summed here (the relaxed ones read partials of zero weights); Z is never formed."""
    n_, h, w, _ = x.shape
    r_n, s_n, k, _ = wt.shape
    ph, pw = pad
    nbr, nbs = -(-r_n // 3), -(-s_n // 3)
    w3 = split_weights_3x3(wt)
    y = gemm_stage(x, w3)                                    # [M, 9 * nbr*nbs*K]
    y7 = y.reshape(n_, h, w, 3, 3, nbr * nbs, k)
    ho_n = conv_out_size(h, r_n, 1, ph, 1)
    wo_n = conv_out_size(w, s_n, 1, pw, 1)
    out = np.zeros((n_, ho_n, wo_n, k), dtype=np.float64)
    for a in range(nbr):
        for b in range(nbs):
            for rp in range(3):
                for sp in range(3):
                    for ho in range(ho_n):
                        hi = ho - ph + 3 * a + rp
                        if hi < 0 or hi >= h:
                            continue
                        for wo in range(wo_n):
                            wi = wo - pw + 3 * b + sp
                            if wi < 0 or wi >= w:
                                continue
                            out[:, ho, wo, :] += y7[:, hi, wi, rp, sp, a * nbs + b, :]
    return out


def _band_nondilated(q, k, v, w, scale, mask, l_full_in_range):
    """Non-dilated band on one subsequence: rows i' attend to t' = i' + j - w.
    l_full_in_range[t'] says whether t' is a real key (always true inside [0, L'))."""
    lq = q.shape[0]
    nb = 2 * w + 1
    scores = q @ k.T * scale                                 # dense [L', L'] product
    s = np.zeros((lq, nb))
    live = np.zeros((lq, nb), dtype=bool)
    vals = np.zeros((lq, nb, v.shape[1]))
    for i in range(lq):
        for j in range(nb):
            t = i + j - w
            inside = 0 <= t < lq
            if inside:
                s[i, j] = scores[i, t]
                vals[i, j] = v[t]
            live[i, j] = inside or not mask
    m = np.where(live, s, -np.inf).max(axis=1, keepdims=True)
    e = np.where(live, np.exp(s - m), 0.0)
    p = e / e.sum(axis=1, keepdims=True)
    o = np.einsum("ij,ijd->id", p, vals)
    return s, p, o


def derived_band(q, k, v, w, dil, scale=1.0, mask=False):
    """Dilated band via per-residue non-dilated bands (strided views), re-interleaved.

    q,k,v: [B, L, d] float64.  Returns S, P [B, L, 2w+1] and O [B, L, d]."""
    b_n, l, d = q.shape
    nb = 2 * w + 1
    s_all = np.zeros((b_n, l, nb))
    p_all = np.zeros((b_n, l, nb))
    o_all = np.zeros((b_n, l, d))
    for b in range(b_n):
        for rho in range(dil):
            qs, ks, vs = q[b, rho::dil], k[b, rho::dil], v[b, rho::dil]
            if qs.shape[0] == 0:
                continue
            s, p, o = _band_nondilated(qs.astype(np.float64), ks.astype(np.float64),
                                       vs.astype(np.float64), w, scale, mask, None)
            s_all[b, rho::dil] = s
            p_all[b, rho::dil] = p
            o_all[b, rho::dil] = o
    return s_all, p_all, o_all
