"""Pins for the CPU oracle: each check ties the oracle to something other than itself.

* library routines evaluated in float64 (torch conv2d / conv_transpose2d, softmax
  attention) on shapes where they compute the same operator;
* the adjoint identity between convolution and transposed convolution;
* brute-force scatter evaluation of the transposed convolution;
* closed forms: 1x1 convolution = matrix product, dilation = zero-inserted kernel,
  dilated band = per-residue non-dilated bands;
* hand-worked examples (tests/golden/hand_worked.json);
* exact agreement with the independently written derived form (GEMM + eOperator)
  on integer-valued inputs.

Shapes are deliberately asymmetric (R != S, H != W, C != K, different stride,
pad and dilation per axis) so that a swapped index or a transposed operand fails.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import derived_form as dfm
import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def torch_conv2d(x, wt, stride, pad, dil):
    """X [N,H,W,C], Wt [R,S,K,C] -> torch NCHW/OIHW float64 -> back to NHWC."""
    xt = torch.as_tensor(np.asarray(x, dtype=np.float64)).permute(0, 3, 1, 2)
    wtt = torch.as_tensor(np.asarray(wt, dtype=np.float64)).permute(2, 3, 0, 1)
    return F.conv2d(xt, wtt, stride=stride, padding=pad, dilation=dil).permute(0, 2, 3, 1).numpy()


def torch_conv_transpose2d(x, wt, stride, pad, dil, out_pad):
    """Wt [R,S,K,C] (C in, K out) -> torch weight [C_in, C_out, R, S]."""
    xt = torch.as_tensor(np.asarray(x, dtype=np.float64)).permute(0, 3, 1, 2)
    wtt = torch.as_tensor(np.asarray(wt, dtype=np.float64)).permute(3, 2, 0, 1)
    return F.conv_transpose2d(xt, wtt, stride=stride, padding=pad, dilation=dil,
                              output_padding=out_pad).permute(0, 2, 3, 1).numpy()


# (n, c, h, w, k, r, s, stride, pad, dil)
CONV_CASES = [
    (1, 3, 5, 7, 2, 3, 2, (1, 1), (0, 0), (1, 1)),
    (2, 4, 6, 5, 3, 3, 3, (1, 1), (1, 1), (1, 1)),
    (1, 2, 9, 8, 3, 3, 2, (2, 1), (1, 0), (1, 1)),
    (1, 3, 8, 9, 2, 2, 3, (1, 2), (0, 2), (2, 1)),
    (2, 2, 7, 6, 4, 3, 3, (1, 1), (2, 2), (2, 2)),
    (1, 1, 9, 9, 1, 3, 3, (3, 3), (3, 1), (1, 3)),
    (1, 4, 4, 6, 3, 4, 1, (1, 1), (3, 0), (1, 1)),     # pad >= R - 1
    (1, 2, 5, 5, 2, 2, 2, (3, 2), (0, 0), (3, 2)),     # H < R*dil + something
    (3, 1, 3, 4, 2, 1, 1, (1, 1), (0, 0), (1, 1)),     # 1x1
    (1, 3, 2, 3, 2, 3, 3, (1, 1), (1, 1), (1, 1)),     # image smaller than kernel span
    (1, 2, 6, 6, 2, 2, 2, (4, 4), (1, 1), (1, 1)),     # stride > kernel
]

# (n, c, h, w, k, r, s, stride, pad, dil, out_pad)
CONVT_CASES = [
    (1, 3, 3, 4, 2, 2, 3, (2, 2), (0, 0), (1, 1), (0, 0)),
    (2, 2, 4, 3, 3, 4, 4, (2, 2), (1, 1), (1, 1), (0, 0)),
    (1, 2, 3, 3, 2, 3, 2, (3, 2), (1, 0), (1, 1), (2, 1)),
    (1, 3, 4, 5, 2, 3, 3, (1, 1), (1, 1), (2, 1), (1, 0)),
    (2, 1, 2, 2, 1, 4, 4, (2, 2), (1, 1), (1, 1), (1, 1)),
    (1, 4, 3, 2, 3, 2, 2, (1, 2), (0, 1), (2, 2), (1, 1)),
    (1, 2, 5, 4, 2, 5, 3, (3, 3), (2, 1), (1, 2), (0, 2)),
]


def _conv_case_inputs(case, seed, integer):
    n, c, h, w, k, r, s = case[:7]
    x = synth.random_tensor((n, h, w, c), seed, integer=integer).numpy()
    wt = synth.random_tensor((r, s, k, c), seed + 1, integer=integer).numpy()
    return x, wt


@pytest.mark.parametrize("ci", range(len(CONV_CASES)))
@pytest.mark.parametrize("integer", [False, True])
def test_conv2d_matches_torch_float64(ci, integer):
    case = CONV_CASES[ci]
    stride, pad, dil = case[7:10]
    x, wt = _conv_case_inputs(case, 100 + ci, integer)
    got = oracle.conv2d(x, wt, stride, pad, dil)
    ref = torch_conv2d(x, wt, stride, pad, dil)
    assert got.shape == ref.shape
    if integer:
        assert np.array_equal(got, ref)
    else:
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("ci", range(len(CONVT_CASES)))
@pytest.mark.parametrize("integer", [False, True])
def test_conv_transpose2d_matches_torch_float64(ci, integer):
    case = CONVT_CASES[ci]
    stride, pad, dil, op = case[7:11]
    x, wt = _conv_case_inputs(case, 200 + ci, integer)
    got = oracle.conv_transpose2d(x, wt, stride, pad, dil, op)
    ref = torch_conv_transpose2d(x, wt, stride, pad, dil, op)
    assert got.shape == ref.shape
    if integer:
        assert np.array_equal(got, ref)
    else:
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def _scatter_convt(x, wt, stride, pad, dil, out_pad):
    """Brute force: every (input pixel, tap) pair adds its product to the output
    position it lands on; positions outside the output are dropped."""
    n, h, w, c = x.shape
    r_n, s_n, k, _ = wt.shape
    ho = (h - 1) * stride[0] - 2 * pad[0] + dil[0] * (r_n - 1) + out_pad[0] + 1
    wo = (w - 1) * stride[1] - 2 * pad[1] + dil[1] * (s_n - 1) + out_pad[1] + 1
    out = np.zeros((n, ho, wo, k))
    for b, hi, wi, r, s in itertools.product(range(n), range(h), range(w), range(r_n), range(s_n)):
        oh = hi * stride[0] - pad[0] + r * dil[0]
        ow = wi * stride[1] - pad[1] + s * dil[1]
        if 0 <= oh < ho and 0 <= ow < wo:
            for kk in range(k):
                for cc in range(c):
                    out[b, oh, ow, kk] += float(x[b, hi, wi, cc]) * float(wt[r, s, kk, cc])
    return out


@pytest.mark.parametrize("ci", range(len(CONVT_CASES)))
def test_conv_transpose2d_matches_scatter_brute_force(ci):
    case = CONVT_CASES[ci]
    stride, pad, dil, op = case[7:11]
    x, wt = _conv_case_inputs(case, 300 + ci, True)
    got = oracle.conv_transpose2d(x, wt, stride, pad, dil, op)
    assert np.array_equal(got, _scatter_convt(x, wt, stride, pad, dil, op))


@pytest.mark.parametrize("ci", range(len(CONV_CASES)))
def test_adjoint_identity(ci):
    """<conv2d(x; W), y> = <x, conv_transpose2d(y; W^T)>, with W^T swapping the
    input/output channel roles and out_pad chosen so the adjoint returns H x W."""
    case = CONV_CASES[ci]
    n, c, h, w, k, r, s = case[:7]
    stride, pad, dil = case[7:10]
    x, wt = _conv_case_inputs(case, 400 + ci, False)
    fwd = oracle.conv2d(x, wt, stride, pad, dil)
    ho, wo = fwd.shape[1:3]
    if ho == 0 or wo == 0:
        pytest.skip("empty output")
    y = synth.random_tensor(fwd.shape, 500 + ci).numpy()
    op_h = h - ((ho - 1) * stride[0] - 2 * pad[0] + dil[0] * (r - 1) + 1)
    op_w = w - ((wo - 1) * stride[1] - 2 * pad[1] + dil[1] * (s - 1) + 1)
    assert op_h >= 0 and op_w >= 0
    wt_t = np.ascontiguousarray(wt.transpose(0, 1, 3, 2))      # [R,S,C,K]
    adj = oracle.conv_transpose2d(y, wt_t, stride, pad, dil, (op_h, op_w))
    assert adj.shape == x.shape
    lhs = float(np.sum(fwd * y))
    rhs = float(np.sum(x.astype(np.float64) * adj))
    assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(lhs))


def test_one_by_one_conv_is_matmul():
    x = synth.random_tensor((2, 5, 3, 7), 600).numpy()
    wt = synth.random_tensor((1, 1, 4, 7), 601).numpy()
    got = oracle.conv2d(x, wt, 1, 0, 1)
    ref = x.reshape(-1, 7).astype(np.float64) @ wt.reshape(4, 7).astype(np.float64).T
    np.testing.assert_allclose(got.reshape(-1, 4), ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("dil", [(2, 2), (3, 2), (2, 1)])
def test_dilation_equals_zero_inserted_kernel(dil):
    x = synth.random_tensor((1, 11, 10, 3), 700, integer=True).numpy()
    wt = synth.random_tensor((3, 2, 2, 3), 701, integer=True).numpy()
    dh, dw = dil
    big = np.zeros((dh * 2 + 1, dw * 1 + 1, 2, 3), dtype=np.float32)
    big[::dh, ::dw] = wt
    got = oracle.conv2d(x, wt, (1, 1), (2, 1), dil)
    ref = oracle.conv2d(x, big, (1, 1), (2, 1), (1, 1))
    assert np.array_equal(got, ref)


def test_hand_worked_examples():
    with open(os.path.join(HERE, "golden", "hand_worked.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        exp = np.array(case["expected"], dtype=np.float64)
        if case["op"] == "conv2d":
            got = oracle.conv2d(np.array(case["x"], np.float32), np.array(case["wt"], np.float32),
                                case["stride"], case["pad"], case["dil"])
        elif case["op"] == "conv_transpose2d":
            got = oracle.conv_transpose2d(np.array(case["x"], np.float32),
                                          np.array(case["wt"], np.float32), case["stride"],
                                          case["pad"], case["dil"], case["out_pad"])
        else:
            q = np.array(case["q"], np.float32)
            k = np.array(case["k"], np.float32)
            s, _, _ = oracle.band(q, k, np.zeros_like(q), case["w"], case["dil"])
            got = s
        assert got.shape == exp.shape, case["working"]
        assert np.array_equal(got, exp), case["working"]


@pytest.mark.parametrize("ci", range(len(CONV_CASES)))
def test_derived_form_conv_exact_on_integers(ci):
    case = CONV_CASES[ci]
    stride, pad, dil = case[7:10]
    x, wt = _conv_case_inputs(case, 800 + ci, True)
    got = oracle.conv2d(x, wt, stride, pad, dil)
    ref = dfm.derived_conv2d(x, wt, stride, pad, dil)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("ci", range(len(CONVT_CASES)))
def test_derived_form_convt_exact_on_integers(ci):
    case = CONVT_CASES[ci]
    stride, pad, dil, op = case[7:11]
    x, wt = _conv_case_inputs(case, 900 + ci, True)
    got = oracle.conv_transpose2d(x, wt, stride, pad, dil, op)
    ref = dfm.derived_conv_transpose2d(x, wt, stride, pad, dil, op)
    assert np.array_equal(got, ref)


# (n, c, h, w, k, r, s, pad): 5x5 with "same" and no padding, kernels that are not a
# whole number of 3x3 blocks along one or both axes, one already 3x3, one 1x1, 7x7
SPLIT3_CASES = [
    (1, 3, 9, 8, 2, 5, 5, (2, 2)),
    (2, 2, 8, 7, 3, 5, 5, (0, 0)),
    (1, 2, 7, 9, 2, 4, 2, (1, 3)),
    (1, 3, 6, 6, 2, 3, 3, (1, 1)),
    (1, 2, 5, 5, 2, 1, 1, (0, 0)),
    (1, 2, 10, 9, 2, 7, 6, (3, 2)),
]


@pytest.mark.parametrize("ci", range(len(SPLIT3_CASES)))
def test_split3x3_derived_form_exact_on_integers(ci):
    """The R x S -> 3x3 derived form equals the convolution's definition exactly on
    integer inputs (the rewrite only adds zero-weight taps and regroups the sum)."""
    n, c, h, w, k, r, s, pad = SPLIT3_CASES[ci]
    x = synth.random_tensor((n, h, w, c), 1200 + ci, integer=True).numpy()
    wt = synth.random_tensor((r, s, k, c), 1300 + ci, integer=True).numpy()
    got = dfm.derived_conv2d_split3x3(x, wt, pad)
    ref = oracle.conv2d(x, wt, 1, pad, 1)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("ci", range(len(SPLIT3_CASES)))
def test_split3x3_fused_eoperator_chain_exact_on_integers(ci):
    """The 3x3 derived form with its two consecutive eOperators fused into one over the
    3x3 stage's scope (no intermediate Z) equals the convolution's definition and the
    unfused chain (3x3 OffsetAdd into Z, then the block OffsetAdd) exactly on integer
    inputs; on real-valued inputs all three agree to float64 rounding."""
    n, c, h, w, k, r, s, pad = SPLIT3_CASES[ci]
    x = synth.random_tensor((n, h, w, c), 1200 + ci, integer=True).numpy()
    wt = synth.random_tensor((r, s, k, c), 1300 + ci, integer=True).numpy()
    got = dfm.derived_conv2d_split3x3_chain(x, wt, pad)
    ref = oracle.conv2d(x, wt, 1, pad, 1)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref)
    assert np.array_equal(got, dfm.derived_conv2d_split3x3(x, wt, pad))
    xf = synth.random_tensor((n, h, w, c), 1250 + ci).numpy()
    wf = synth.random_tensor((r, s, k, c), 1350 + ci).numpy()
    got = dfm.derived_conv2d_split3x3_chain(xf, wf, pad)
    ref = oracle.conv2d(xf, wf, 1, pad, 1)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * max(1.0, np.abs(ref).max()))


def test_split3x3_chain_reads_each_tap_of_the_kernel_once():
    """A lone 1 in the input and a kernel whose entries are distinct powers of two: the
    fused chain's output at every position is the sum of the kernel entries whose tap
    lands on the 1, so each real tap (r, s) is read exactly once and no relaxed tap
    contributes (a dropped or doubled tap changes the binary digits)."""
    r_n, s_n, h, w = 5, 4, 9, 8
    x = np.zeros((1, h, w, 1))
    x[0, 4, 3, 0] = 1.0
    wt = (2.0 ** np.arange(r_n * s_n)).reshape(r_n, s_n, 1, 1)
    got = dfm.derived_conv2d_split3x3_chain(x, wt, (2, 1))
    ho_n, wo_n = h + 4 - r_n + 1, w + 2 - s_n + 1
    assert got.shape == (1, ho_n, wo_n, 1)
    for ho in range(ho_n):
        for wo in range(wo_n):
            r, s = 4 - ho + 2, 3 - wo + 1          # the tap whose input pixel is (4, 3)
            want = wt[r, s, 0, 0] if 0 <= r < r_n and 0 <= s < s_n else 0.0
            assert got[0, ho, wo, 0] == want, (ho, wo)


def test_split3x3_weights_cover_every_tap_once():
    """Each tap of the kernel lands in exactly one (block, r', s') slot of W3 and the
    relaxed slots are zero: the block sums of W3 reproduce the kernel's total per
    (k, c), and the count of non-zero slots equals R*S on an all-ones kernel."""
    wt = np.ones((5, 4, 2, 3))
    w3 = dfm.split_weights_3x3(wt)
    assert w3.shape == (3, 3, 2 * 2 * 2, 3)
    assert int((w3 != 0).sum()) == 5 * 4 * 2 * 3
    wr = synth.random_tensor((5, 4, 2, 3), 1400).numpy().astype(np.float64)
    w3r = dfm.split_weights_3x3(wr)
    tot = w3r.sum(axis=(0, 1)).reshape(4, 2, 3).sum(axis=0)
    np.testing.assert_allclose(tot, wr.sum(axis=(0, 1)), rtol=0, atol=1e-12)


@pytest.mark.parametrize("integer", [True, False])
def test_tiny_workload_against_torch_and_derived_form(integer):
    wl = synth.WORKLOADS[1]
    x, wt = synth.conv_inputs(wl, integer=integer)
    x, wt = x.numpy(), wt.numpy()
    got = oracle.conv2d(x, wt, wl.stride, wl.pad, wl.dil)
    ref = torch_conv2d(x, wt, wl.stride, wl.pad, wl.dil)
    dref = dfm.derived_conv2d(x, wt, wl.stride, wl.pad, wl.dil)
    if integer:
        assert np.array_equal(got, ref) and np.array_equal(got, dref)
    else:
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(got, dref, rtol=0, atol=1e-12)


def test_sampled_evaluation_matches_full():
    case = CONV_CASES[4]
    stride, pad, dil = case[7:10]
    x, wt = _conv_case_inputs(case, 1000, False)
    full = oracle.conv2d(x, wt, stride, pad, dil)
    idx = np.array([0, 5, full.size - 1, full.size // 2, 17])
    assert np.array_equal(oracle.conv2d(x, wt, stride, pad, dil, idx=idx), full.reshape(-1)[idx])
    case = CONVT_CASES[1]
    stride, pad, dil, op = case[7:11]
    x, wt = _conv_case_inputs(case, 1001, False)
    full = oracle.conv_transpose2d(x, wt, stride, pad, dil, op)
    idx = np.array([0, 5, full.size - 1, full.size // 2, 17])
    assert np.array_equal(oracle.conv_transpose2d(x, wt, stride, pad, dil, op, idx=idx),
                          full.reshape(-1)[idx])


def test_workload_output_extents():
    """Output shapes of the four workloads from the definitions (section 8 sizes)."""
    assert oracle.conv_out_size(14, 3, 1, 1, 1) == 14
    assert oracle.conv_out_size(8, 4, 2, 1, 1, 0, True) == 16
    assert oracle.conv_out_size(96, 3, 1, 2, 2) == 96
    assert oracle.conv_out_size(128, 3, 1, 2, 2) == 128


# ----------------------------------------------------------------------------- band

def _band_inputs(b, l, d, seed, integer=False):
    q = synth.random_tensor((b, l, d), seed, integer=integer, dist="normal").numpy()
    k = synth.random_tensor((b, l, d), seed + 1, integer=integer, dist="normal").numpy()
    v = synth.random_tensor((b, l, d), seed + 2, dist="normal").numpy()
    return q, k, v


BAND_CASES = [  # (b, l, d, w, dil)
    (2, 17, 4, 3, 1),
    (1, 23, 5, 4, 2),
    (2, 19, 3, 2, 3),
    (1, 9, 2, 6, 2),      # band wider than the sequence
    (1, 1, 3, 2, 1),      # single row
]


@pytest.mark.parametrize("ci", range(len(BAND_CASES)))
def test_band_scores_match_dense_product(ci):
    b, l, d, w, dil = BAND_CASES[ci]
    q, k, v = _band_inputs(b, l, d, 1100 + ci, integer=True)
    s, _, _ = oracle.band(q, k, v, w, dil)
    dense = np.einsum("bid,btd->bit", q.astype(np.float64), k.astype(np.float64))
    for bi in range(b):
        for i in range(l):
            for j in range(2 * w + 1):
                t = i + (j - w) * dil
                exp = dense[bi, i, t] if 0 <= t < l else 0.0
                assert s[bi, i, j] == exp


def test_band_mask_mode_full_window_is_softmax_attention():
    b, l, d = 2, 13, 6
    q, k, v = _band_inputs(b, l, d, 1200)
    s, p, o = oracle.band(q, k, v, w=l - 1, dil=1, scale=0.5, mask=True)
    qt, kt, vt = (torch.as_tensor(a, dtype=torch.float64) for a in (q, k, v))
    att = torch.softmax(qt @ kt.transpose(1, 2) * 0.5, dim=-1)
    ref = (att @ vt).numpy()
    np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)
    # P on the band: entry j of row i is key t = i + j - (l-1)
    for i in range(l):
        np.testing.assert_allclose(p[:, i, (l - 1) - i:(l - 1) - i + l], att[:, i].numpy(),
                                   rtol=0, atol=1e-14)


def test_band_lone_entry_rows_return_v():
    """With the dilation at or above the sequence length every key t = i + (j-w)*D other
    than t = i falls outside [0, L): in mask mode each row's softmax has the single entry
    j = w, so P is one-hot and O equals V exactly; in zero mode the 2w out-of-range
    entries score 0 and O = e^s V / (e^s + 2w) with s = scale * q.k."""
    b, l, d, w, dil = 2, 3, 5, 2, 5
    q, k, v = _band_inputs(b, l, d, 1250)
    s, p, o = oracle.band(q, k, v, w, dil, scale=0.3, mask=True)
    onehot = np.zeros(2 * w + 1)
    onehot[w] = 1.0
    np.testing.assert_array_equal(p, np.broadcast_to(onehot, p.shape))
    np.testing.assert_array_equal(o, v)
    _, _, oz = oracle.band(q, k, v, w, dil, scale=0.3, mask=False)
    q64, k64, v64 = (a.astype(np.float64) for a in (q, k, v))
    es = np.exp(0.3 * np.einsum("bid,bid->bi", q64, k64))[..., None]
    np.testing.assert_allclose(oz, es * v64 / (es + 2 * w), rtol=1e-13, atol=0)


@pytest.mark.parametrize("ci", range(len(BAND_CASES)))
def test_band_zero_mode_is_attention_over_zero_padded_keys(ci):
    """Zero mode = softmax attention in which every out-of-range key and value is an
    explicit zero row (section 3: padding reads as 0)."""
    b, l, d, w, dil = BAND_CASES[ci]
    q, k, v = _band_inputs(b, l, d, 1300 + ci)
    _, p, o = oracle.band(q, k, v, w, dil, scale=0.7)
    pad = w * dil
    kp = np.zeros((b, l + 2 * pad, d))
    vp = np.zeros((b, l + 2 * pad, d))
    kp[:, pad:pad + l] = k
    vp[:, pad:pad + l] = v
    idx = np.arange(l)[:, None] + pad + (np.arange(2 * w + 1)[None, :] - w) * dil
    kb = torch.as_tensor(kp[:, idx])           # [b, l, 2w+1, d]
    vb = torch.as_tensor(vp[:, idx])
    qt = torch.as_tensor(q, dtype=torch.float64)
    att = torch.softmax(torch.einsum("bid,bijd->bij", qt, kb) * 0.7, dim=-1)
    ref_o = torch.einsum("bij,bijd->bid", att, vb).numpy()
    np.testing.assert_allclose(p, att.numpy(), rtol=0, atol=1e-14)
    np.testing.assert_allclose(o, ref_o, rtol=0, atol=1e-12)


@pytest.mark.parametrize("mask", [False, True])
def test_band_probability_invariants(mask):
    q, k, v = _band_inputs(2, 31, 4, 1400)
    _, p, _ = oracle.band(q, k, v, w=5, dil=2, mask=mask)
    assert (p >= 0).all()
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=0, atol=1e-12)
    if mask:   # out-of-range keys get exactly zero weight
        for i in range(31):
            for j in range(11):
                t = i + (j - 5) * 2
                if not 0 <= t < 31:
                    assert (p[:, i, j] == 0).all()


@pytest.mark.parametrize("mask", [False, True])
def test_dilated_band_equals_per_residue_nondilated_band(mask):
    """Section 6.4: the dilated G2BMM equals non-dilated bands on the residue
    subsequences i mod dil (only the access pattern changes)."""
    b, l, d, w, dil = 2, 29, 3, 3, 3
    q, k, v = _band_inputs(b, l, d, 1500)
    s, p, o = oracle.band(q, k, v, w, dil, mask=mask)
    for rho in range(dil):
        sub = tuple(np.ascontiguousarray(a[:, rho::dil]) for a in (q, k, v))
        s2, p2, o2 = oracle.band(*sub, w, 1, mask=mask)
        assert np.array_equal(s[:, rho::dil], s2)
        assert np.array_equal(p[:, rho::dil], p2)
        assert np.array_equal(o[:, rho::dil], o2)


@pytest.mark.parametrize("ci", range(len(BAND_CASES)))
@pytest.mark.parametrize("mask", [False, True])
def test_band_derived_form_agrees(ci, mask):
    b, l, d, w, dil = BAND_CASES[ci]
    q, k, v = _band_inputs(b, l, d, 1600 + ci, integer=True)
    s, p, o = oracle.band(q, k, v, w, dil, mask=mask)
    s2, p2, o2 = dfm.derived_band(q, k, v, w, dil, mask=mask)
    assert np.array_equal(s, s2)
    np.testing.assert_allclose(p, p2, rtol=0, atol=1e-14)
    np.testing.assert_allclose(o, o2, rtol=0, atol=1e-12)


def test_band_sampled_rows_match_full():
    q, k, v = _band_inputs(2, 21, 4, 1700)
    s, p, o = oracle.band(q, k, v, 4, 2)
    rows = np.array([0, 20, 21, 41, 7])
    s2, p2, o2 = oracle.band(q, k, v, 4, 2, rows=rows)
    assert np.array_equal(s2, s.reshape(-1, 9)[rows])
    assert np.array_equal(p2, p.reshape(-1, 9)[rows])
    assert np.array_equal(o2, o.reshape(-1, 4)[rows])


# ------------------------------------------------------ element-wise tail (§6.3)

def _torch_block_tail(conv_t, bias, residual, relu):
    """The tail as torch builds it: the conv's own bias argument, a tensor add, then
    torch.relu -- an implementation independent of the oracle's."""
    y = conv_t
    if residual is not None:
        y = y + torch.as_tensor(np.asarray(residual, dtype=np.float64)).permute(0, 3, 1, 2)
    return torch.relu(y) if relu else y


@pytest.mark.parametrize("ci", [0, 1, 4, 6])
@pytest.mark.parametrize("integer", [False, True])
@pytest.mark.parametrize("relu", [False, True])
def test_conv_epilogue_matches_torch_bias_residual_relu(ci, integer, relu):
    case = CONV_CASES[ci]
    stride, pad, dil = case[7:10]
    x, wt = _conv_case_inputs(case, 700 + ci, integer)
    k = case[4]
    bias = synth.random_tensor((k,), 720 + ci, integer=integer).numpy()
    conv = oracle.conv2d(x, wt, stride, pad, dil)
    residual = synth.random_tensor(conv.shape, 740 + ci, integer=integer).numpy()
    got = oracle.conv_epilogue(conv, bias, residual, relu)
    xt = torch.as_tensor(np.asarray(x, dtype=np.float64)).permute(0, 3, 1, 2)
    wtt = torch.as_tensor(np.asarray(wt, dtype=np.float64)).permute(2, 3, 0, 1)
    ct = F.conv2d(xt, wtt, bias=torch.as_tensor(bias, dtype=torch.float64), stride=stride,
                  padding=pad, dilation=dil)
    ref = _torch_block_tail(ct, bias, residual, relu).permute(0, 2, 3, 1).numpy()
    if integer:
        assert np.array_equal(got, ref)
    else:
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("ci", [0, 2, 4])
def test_conv_transpose_epilogue_matches_torch(ci):
    case = CONVT_CASES[ci]
    stride, pad, dil, op = case[7:11]
    x, wt = _conv_case_inputs(case, 760 + ci, True)
    bias = synth.random_tensor((case[4],), 770 + ci, integer=True).numpy()
    conv = oracle.conv_transpose2d(x, wt, stride, pad, dil, op)
    residual = synth.random_tensor(conv.shape, 780 + ci, integer=True).numpy()
    got = oracle.conv_epilogue(conv, bias, residual, True)
    xt = torch.as_tensor(np.asarray(x, dtype=np.float64)).permute(0, 3, 1, 2)
    wtt = torch.as_tensor(np.asarray(wt, dtype=np.float64)).permute(3, 2, 0, 1)
    ct = F.conv_transpose2d(xt, wtt, bias=torch.as_tensor(bias, dtype=torch.float64),
                            stride=stride, padding=pad, dilation=dil, output_padding=op)
    ref = _torch_block_tail(ct, bias, residual, True).permute(0, 2, 3, 1).numpy()
    assert np.array_equal(got, ref)


def test_conv_epilogue_terms_one_at_a_time():
    """Each term on its own: no term is the identity, the bias shifts every pixel of a
    channel by the same amount, the residual adds elementwise, ReLU zeroes exactly the
    negative entries and keeps the rest."""
    rng = np.random.default_rng(5)
    conv = rng.integers(-9, 10, size=(2, 3, 4, 5)).astype(np.float64)
    bias = rng.integers(-3, 4, size=(5,)).astype(np.float32)
    res = rng.integers(-3, 4, size=(2, 3, 4, 5)).astype(np.float32)
    assert np.array_equal(oracle.conv_epilogue(conv), conv)
    d = oracle.conv_epilogue(conv, bias=bias) - conv
    for kk in range(5):
        assert np.all(d[..., kk] == bias[kk])
    assert np.array_equal(oracle.conv_epilogue(conv, residual=res) - conv, res)
    r = oracle.conv_epilogue(conv, relu=True)
    assert np.all(r >= 0)
    assert np.array_equal(r[conv > 0], conv[conv > 0])
    assert np.all(r[conv <= 0] == 0)
    assert (conv < 0).any() and (conv > 0).any()


# ------------------------------- dilated conv = non-dilated convs of sub-images (§6.2)

@pytest.mark.parametrize("dil,pad,hw", [((2, 2), (2, 2), (9, 12)), ((3, 2), (1, 2), (10, 7)),
                                        ((2, 3), (0, 3), (8, 11)), ((4, 4), (4, 4), (13, 13))])
def test_dilated_conv_is_residue_subimage_convs(dil, pad, hw):
    """With stride 1, the outputs of residue (a, b) = (ho % dh, wo % dw) are the
    non-dilated convolution of the input sub-image of residue ((a - ph) mod dh,
    (b - pw) mod dw), shifted by floor((a - ph) / dh) rows (likewise for columns)."""
    n, c, k, r, s = 2, 3, 2, 3, 3
    h, w = hw
    x = synth.random_tensor((n, h, w, c), 801, integer=True).numpy()
    wt = synth.random_tensor((r, s, k, c), 802, integer=True).numpy()
    full = oracle.conv2d(x, wt, (1, 1), pad, dil)
    ho, wo = full.shape[1:3]
    dh, dw = dil
    for a in range(min(dh, ho)):
        for b in range(min(dw, wo)):
            qh, rh = divmod(a - pad[0], dh)
            qw, rw = divmod(b - pad[1], dw)
            sub = x[:, rh::dh, rw::dw, :]
            hc, wc = len(range(a, ho, dh)), len(range(b, wo, dw))
            # zero-extend the sub-image so that rows qh .. qh + hc + r - 2 exist
            lo_h, lo_w = max(0, -qh), max(0, -qw)
            hi_h = max(0, qh + hc + r - 1 - sub.shape[1])
            hi_w = max(0, qw + wc + s - 1 - sub.shape[2])
            padded = np.pad(sub, ((0, 0), (lo_h, hi_h), (lo_w, hi_w), (0, 0)))
            win = padded[:, qh + lo_h: qh + lo_h + hc + r - 1, qw + lo_w: qw + lo_w + wc + s - 1]
            part = oracle.conv2d(win, wt, (1, 1), (0, 0), (1, 1))
            assert np.array_equal(part, full[:, a::dh, b::dw, :])
