"""Seeded random-shape sweep of the convolution operators through the C ABI.

Each case draws one convolution problem (operator, batch, channels, image, kernel,
per-axis stride / padding / dilation / output padding) and evaluates it on integer-valued
bf16 inputs along every derived form the library offers for it: the two-stage path
(GEMM stage + eOperator, fp32 scope), the fused expression, and where they apply the
Conv5x5 -> Conv3x3 split form (fused and two-stage 3x3 stage), the residue sub-image
form of the dilated convolution and the allocation-free entry point.  With integer
inputs every partial sum is an integer below 2^24, so each form must equal the oracle's
convolution exactly.

A second sweep draws banded problems (batch, length, half-width, dilation, zero or mask
mode) and runs every wave shape of the fused kernel and the staged path against the
oracle.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2208_02025_amd as ol
import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def out_hw(kind, h, w, r, s, st, pd, dl, op):
    if kind == "conv_transpose2d":
        return ((h - 1) * st[0] - 2 * pd[0] + dl[0] * (r - 1) + op[0] + 1,
                (w - 1) * st[1] - 2 * pd[1] + dl[1] * (s - 1) + op[1] + 1)
    return ((h + 2 * pd[0] - dl[0] * (r - 1) - 1) // st[0] + 1,
            (w + 2 * pd[1] - dl[1] * (s - 1) - 1) // st[1] + 1)


def draw_cases(n_cases, seed):
    """Valid problems: positive output sizes, output padding below max(stride,
    dilation) for the transposed operator, dilation 1 for derived_conv2d, channels a
    multiple of 8 (bf16 rows of 16 bytes), most of them a multiple of 64 (the fused
    expression's k-tile)."""
    rng = np.random.default_rng(seed)
    kinds = ["conv2d", "dilated_conv2d", "conv_transpose2d"]
    cases = []
    while len(cases) < n_cases:
        kind = kinds[len(cases) % 3]
        n = int(rng.integers(1, 4))
        c = int(rng.choice([8, 24, 64, 128, 192]))
        k = int(rng.integers(1, 81))
        h, w = (int(v) for v in rng.integers(1, 21, 2))
        r, s = (int(v) for v in rng.integers(1, 6, 2))
        # stride 1 in half of the cases: the split and residue forms need it
        st = (1, 1) if rng.random() < 0.5 else tuple(int(v) for v in rng.integers(1, 4, 2))
        dl = (1, 1) if kind == "conv2d" else tuple(int(v) for v in rng.integers(1, 4, 2))
        pd = tuple(int(rng.integers(0, d * (q - 1) + 2)) for d, q in zip(dl, (r, s)))
        op = (0, 0)
        if kind == "conv_transpose2d":
            op = tuple(int(rng.integers(0, max(a, b))) for a, b in zip(st, dl))
        ho, wo = out_hw(kind, h, w, r, s, st, pd, dl, op)
        if ho < 1 or wo < 1 or ho * wo * n * k > 400_000:
            continue
        cases.append((kind, n, c, h, w, k, r, s, st, pd, dl, op))
    return cases


CASES = draw_cases(120, 20240917)


def ref_of(kind, x, wt, st, pd, dl, op):
    if kind == "conv_transpose2d":
        return oracle.conv_transpose2d(x, wt, st, pd, dl, op)
    return oracle.conv2d(x, wt, st, pd, dl)


def forms(kind, c, r, s, st, dl):
    """(name, keyword arguments) of every derived form the case can take."""
    f = [("staged", {}), ("fused", {"fuse": True})]
    if kind == "conv2d":
        f.append(("noalloc", {"noalloc": True}))
        f.append(("noalloc_fused", {"noalloc": True, "fuse": True}))
        if st == (1, 1):
            f.append(("split3x3", {"split3x3": True}))
            f.append(("split3x3_fused", {"split3x3": True, "fuse": True}))
    if kind == "dilated_conv2d" and st == (1, 1) and c % 64 == 0 and dl[0] * dl[1] <= 16:
        f.append(("residues", {"residues": True}))
    return f


def run(kind, xg, wg, st, pd, dl, op, kw):
    kw = dict(kw)
    if kw.pop("noalloc", False):
        return ol.derived_conv2d_noalloc(xg, wg, st, pd, **kw)
    if kind == "conv2d":
        return ol.derived_conv2d(xg, wg, st, pd, **kw)
    if kind == "dilated_conv2d":
        return ol.derived_dilated_conv2d(xg, wg, st, pd, dl, **kw)
    return ol.derived_conv_transpose2d(xg, wg, st, pd, op, dl, **kw)


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_random_shapes_every_form_integer_exact(ci):
    kind, n, c, h, w, k, r, s, st, pd, dl, op = CASES[ci]
    x = synth.random_tensor((n, h, w, c), 30000 + ci, "bf16", integer=True)
    wt = synth.random_tensor((r, s, k, c), 31000 + ci, "bf16", integer=True)
    ref = ref_of(kind, x, wt, st, pd, dl, op)
    xg, wg = x.to(DEV), wt.to(DEV)
    for name, kw in forms(kind, c, r, s, st, dl):
        say("sweep", ci, CASES[ci], name)
        out = run(kind, xg, wg, st, pd, dl, op, kw)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy()
        assert got.shape == ref.shape, name
        assert np.array_equal(got, ref), name


def draw_band_cases(n_cases, seed):
    """Random band problems: batch, length (several tiles and ragged tails, down to a
    single row), half-width up to 300 (2w+1 within the staged softmax's 1024) and
    dilation 1-5 (residues longer and shorter than a tile, or empty)."""
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n_cases):
        b = int(rng.integers(1, 5))
        l = int(rng.choice([1, 2, 63, 64, 65, 129, int(rng.integers(3, 900))]))
        w = int(rng.integers(0, 301))
        dil = int(rng.integers(1, 6))
        mask = bool(rng.integers(0, 2))
        cases.append((b, l, w, dil, mask))
    return cases


BAND_CASES = draw_band_cases(40, 20240918)
TOL_BF16 = 2e-2


@pytest.mark.parametrize("ci", range(len(BAND_CASES)))
def test_random_bands_every_path(ci):
    """Every fused wave shape and the staged path on a random band problem: O against
    the oracle within the bf16 bar, and the staged S (integer Q, K: exact in fp32)
    entry by entry."""
    b, l, w, dil, mask = BAND_CASES[ci]
    scale = 0.0625   # a power of two: the scaled integer scores are exact in fp32
    q = synth.random_tensor((b, l, 64), 32000 + ci, "bf16", integer=True)
    k = synth.random_tensor((b, l, 64), 32100 + ci, "bf16", integer=True)
    v = synth.random_tensor((b, l, 64), 32200 + ci, "bf16", dist="normal")
    s_ref, _, o_ref = oracle.band(q, k, v, w, dil, scale, mask, want_p=False)
    qg, kg, vg = q.to(DEV), k.to(DEV), v.to(DEV)
    den = max(float(np.abs(o_ref).max()), 1e-30)
    for shape in range(4):
        say("band sweep", ci, BAND_CASES[ci], "shape", shape)
        o = ol.banded_bmm(qg, kg, vg, w, dil, scale, mask_invalid=mask,
                          flags=ol.BAND_SHAPE(shape))
        torch.cuda.synchronize()
        on = o.float().cpu().numpy().reshape(o_ref.shape)
        assert np.isfinite(on).all(), shape
        assert np.abs(on - o_ref).max() / den <= TOL_BF16, shape
    say("band sweep", ci, BAND_CASES[ci], "staged")
    o, sg = ol.banded_bmm(qg, kg, vg, w, dil, scale, mask_invalid=mask, staged=True,
                          return_s=True)
    torch.cuda.synchronize()
    assert np.array_equal(sg.cpu().numpy().reshape(s_ref.shape), s_ref)
    on = o.float().cpu().numpy().reshape(o_ref.shape)
    assert np.abs(on - o_ref).max() / den <= TOL_BF16
