"""GPU parity: the HIP path (called through the C ABI) against the CPU oracle on the
same seeded inputs.

Bars (max-abs-normalised error  max|gpu - oracle| / max|oracle|):
  * integer-valued inputs (values in {-3..3}) with an fp32 scope Y: bit-exact;
  * fp32 inputs: <= 1e-5;
  * bf16 inputs with fp32 accumulation: <= 2e-2.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle import derived_form as dfm
import paper_2208_02025_amd as ol
import synth

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-5
TOL_BF16 = 2e-2
DEV = "cuda:0"


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), "non-finite output"
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (den if den > 0 else 1.0))


def to_np(t):
    return t.detach().float().cpu().numpy()


def run_conv(kind, x, wt, stride, pad, dil, out_pad=(0, 0), out_dtype=torch.float32,
             y_bf16=False):
    xg, wg = x.to(DEV), wt.to(DEV)
    if kind == "conv2d":
        out = ol.derived_conv2d(xg, wg, stride, pad, out_dtype=out_dtype, y_bf16=y_bf16)
    elif kind == "dilated_conv2d":
        out = ol.derived_dilated_conv2d(xg, wg, stride, pad, dil, out_dtype=out_dtype,
                                        y_bf16=y_bf16)
    else:
        out = ol.derived_conv_transpose2d(xg, wg, stride, pad, out_pad, dil,
                                          out_dtype=out_dtype, y_bf16=y_bf16)
    torch.cuda.synchronize()
    return out


def oracle_conv(kind, x, wt, stride, pad, dil, out_pad=(0, 0)):
    if kind == "conv_transpose2d":
        return oracle.conv_transpose2d(x, wt, stride, pad, dil, out_pad)
    return oracle.conv2d(x, wt, stride, pad, dil)


# ---------------------------------------------------------------- the workloads

@pytest.mark.parametrize("integer", [True, False])
def test_tiny_conv3x3_fp32(integer):
    wl = synth.WORKLOADS[1]
    say("workload 1 fp32 integer=%s" % integer)
    x, wt = synth.conv_inputs(wl, integer=integer)
    out = run_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil)
    ref = oracle_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil)
    if integer:
        assert np.array_equal(to_np(out), ref)
    else:
        assert err(to_np(out), ref) <= TOL_F32


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_workload_bf16(cfg):
    wl = synth.WORKLOADS[cfg]
    say("workload", cfg, wl.name)
    x, wt = synth.conv_inputs(wl)
    out = run_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad)
    ref = oracle_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad)
    e = err(to_np(out), ref)
    say("workload", cfg, "max-abs-normalised error %.3e" % e)
    assert e <= TOL_BF16


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_workload_integer_exact(cfg):
    """Integer-valued bf16 inputs with the fp32 scope: every partial and every sum is
    an exact integer below 2^24, so the GPU must match the definition exactly."""
    wl = synth.WORKLOADS[cfg]
    say("workload", cfg, "integer")
    x, wt = synth.conv_inputs(wl, integer=True)
    out = run_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad)
    ref = oracle_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad)
    assert np.array_equal(to_np(out), ref)


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_workload_bf16_output_and_bf16_scope(cfg):
    wl = synth.WORKLOADS[cfg]
    say("workload", cfg, "bf16 out, bf16 Y")
    x, wt = synth.conv_inputs(wl, seed_offset=10)
    ref = oracle_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad)
    out = run_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad,
                   out_dtype=torch.bfloat16)
    assert out.dtype == torch.bfloat16
    assert err(to_np(out), ref) <= TOL_BF16
    out = run_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad, y_bf16=True)
    assert err(to_np(out), ref) <= TOL_BF16


# ------------------------------------------------------- randomised small shapes
# (kind, n, c, h, w, k, r, s, stride, pad, dil, out_pad)
SMALL = [
    ("conv2d", 1, 3, 5, 7, 2, 3, 2, (1, 1), (0, 0), (1, 1), (0, 0)),
    ("conv2d", 2, 5, 9, 8, 3, 3, 3, (2, 1), (1, 2), (1, 1), (0, 0)),
    ("conv2d", 1, 4, 4, 6, 3, 4, 1, (1, 1), (3, 0), (1, 1), (0, 0)),
    ("conv2d", 3, 7, 11, 13, 5, 1, 1, (1, 1), (0, 0), (1, 1), (0, 0)),
    ("conv2d", 1, 2, 6, 6, 2, 2, 2, (4, 4), (1, 1), (1, 1), (0, 0)),
    ("conv2d", 1, 3, 2, 3, 2, 3, 3, (1, 1), (1, 1), (1, 1), (0, 0)),
    ("dilated_conv2d", 1, 3, 8, 9, 2, 2, 3, (1, 2), (0, 2), (2, 1), (0, 0)),
    ("dilated_conv2d", 2, 2, 7, 6, 4, 3, 3, (1, 1), (2, 2), (2, 2), (0, 0)),
    ("dilated_conv2d", 1, 1, 9, 9, 1, 3, 3, (3, 3), (3, 1), (1, 3), (0, 0)),
    ("conv_transpose2d", 1, 3, 3, 4, 2, 2, 3, (2, 2), (0, 0), (1, 1), (0, 0)),
    ("conv_transpose2d", 2, 2, 4, 3, 3, 4, 4, (2, 2), (1, 1), (1, 1), (0, 0)),
    ("conv_transpose2d", 1, 2, 3, 3, 2, 3, 2, (3, 2), (1, 0), (1, 1), (2, 1)),
    ("conv_transpose2d", 1, 3, 4, 5, 2, 3, 3, (1, 1), (1, 1), (2, 1), (1, 0)),
    ("conv_transpose2d", 1, 2, 5, 4, 2, 5, 3, (3, 3), (2, 1), (1, 2), (0, 2)),
]

# bf16 needs c % 8 == 0; these span several GEMM tiles with ragged tails in m, n and k
# (n*h*w not a multiple of 128, r*s*k not a multiple of 128, c not a multiple of 64).
SMALL_BF16 = [
    ("conv2d", 3, 72, 13, 11, 20, 3, 3, (1, 1), (1, 1), (1, 1), (0, 0)),
    ("conv2d", 1, 8, 17, 19, 3, 3, 2, (2, 1), (0, 1), (1, 1), (0, 0)),
    ("conv2d", 2, 136, 7, 9, 44, 1, 1, (1, 1), (0, 0), (1, 1), (0, 0)),
    ("dilated_conv2d", 1, 24, 21, 18, 12, 3, 3, (1, 1), (3, 2), (3, 2), (0, 0)),
    ("dilated_conv2d", 2, 16, 10, 10, 36, 3, 3, (2, 2), (2, 2), (2, 2), (0, 0)),
    ("conv_transpose2d", 3, 40, 5, 6, 12, 4, 4, (2, 2), (1, 1), (1, 1), (1, 0)),
    ("conv_transpose2d", 1, 64, 9, 7, 8, 3, 3, (3, 2), (1, 1), (1, 2), (2, 1)),
    ("conv_transpose2d", 2, 8, 4, 4, 5, 2, 2, (1, 1), (0, 0), (1, 1), (0, 0)),
]


@pytest.mark.parametrize("ci", range(len(SMALL)))
@pytest.mark.parametrize("integer", [True, False])
def test_small_shapes_fp32(ci, integer):
    kind, n, c, h, w, k, r, s, st, pd, dl, op = SMALL[ci]
    say("small fp32", SMALL[ci], integer)
    x = synth.random_tensor((n, h, w, c), 2000 + ci, integer=integer)
    wt = synth.random_tensor((r, s, k, c), 3000 + ci, integer=integer)
    out = run_conv(kind, x, wt, st, pd, dl, op)
    ref = oracle_conv(kind, x, wt, st, pd, dl, op)
    if integer:
        assert np.array_equal(to_np(out), ref)
    else:
        assert err(to_np(out), ref) <= TOL_F32


@pytest.mark.parametrize("ci", range(len(SMALL_BF16)))
@pytest.mark.parametrize("integer", [True, False])
def test_small_shapes_bf16(ci, integer):
    kind, n, c, h, w, k, r, s, st, pd, dl, op = SMALL_BF16[ci]
    say("small bf16", SMALL_BF16[ci], integer)
    x = synth.random_tensor((n, h, w, c), 4000 + ci, "bf16", integer=integer, dist="normal")
    wt = synth.random_tensor((r, s, k, c), 5000 + ci, "bf16", integer=integer, dist="normal")
    out = run_conv(kind, x, wt, st, pd, dl, op)
    ref = oracle_conv(kind, x, wt, st, pd, dl, op)
    if integer:
        assert np.array_equal(to_np(out), ref)
    else:
        assert err(to_np(out), ref) <= TOL_BF16


# ----------------------------------------------------------------- stage entry points

# k % 64 != 0 takes the register-staged kernel; k % 64 == 0 the DMA kernel, whose tile
# configuration follows the shape: (2100, 2100) and (4129, 4136) -> 128x128 tiles of eight
# waves, the others -> 64x128 tiles (all with ragged m and n tails).
@pytest.mark.parametrize("m,n,k", [(1, 1, 8), (129, 257, 72), (300, 130, 200), (64, 64, 64),
                                   (200, 300, 128), (300, 130, 192), (2100, 2100, 64),
                                   (4129, 4136, 128)])
def test_gemm_stage_bf16_integer_exact(m, n, k):
    say("gemm bf16", m, n, k)
    a = synth.random_tensor((m, k), 6000 + m, "bf16", integer=True)
    b = synth.random_tensor((n, k), 7000 + n, "bf16", integer=True)
    y = ol.gemm_nt(a.to(DEV), b.to(DEV))
    torch.cuda.synchronize()
    ref = a.double().numpy() @ b.double().numpy().T
    assert np.array_equal(to_np(y), ref)


def test_fused_conv_input_over_2gib_sampled():
    """An input X over 2 GiB takes the fused kernel's 64-bit address form; whole output
    rows (top, bottom, and on both sides of the row that starts at byte 2^31 of X) are
    exact against the oracle run on the input rows each output row reads."""
    n, h, w, c, k = 1, 2049, 1024, 512, 16
    say("fused conv over 2 GiB", n, h, w, c, k)
    x = synth.device_integer_tensor((n, h, w, c), 6400, DEV)
    wt = synth.device_integer_tensor((3, 3, k, c), 6401, DEV)
    out = ol.derived_conv2d(x, wt, 1, 1, fuse=True)
    torch.cuda.synchronize()
    wt_c = wt.float().cpu()
    for ho in [0, 1000, 2046, 2047, 2048]:
        lo, hi = max(0, ho - 1), min(h, ho + 2)
        ref = oracle.conv2d(x[:, lo:hi].float().cpu(), wt_c, 1, 1, 1)[:, ho - lo]
        assert np.array_equal(out[:, ho].cpu().numpy().astype(np.float64), ref), ho
    del x, out
    torch.cuda.empty_cache()


# (n, c, h, w, k, r, s, pad, dtype): the R x S -> 3x3 derived form.  c % 64 == 0 bf16
# cases take the fused 3x3 stage when fuse=True; the others its GEMM + OffsetAdd.
SPLIT3_GPU_CASES = [
    (2, 64, 13, 11, 24, 5, 5, (2, 2), "bf16"),
    (1, 72, 9, 10, 20, 5, 5, (0, 0), "bf16"),
    (1, 16, 8, 7, 12, 4, 2, (1, 3), "f32"),
    (1, 64, 12, 12, 16, 7, 7, (3, 3), "bf16"),
    (1, 64, 6, 6, 8, 3, 3, (1, 1), "bf16"),
    (3, 128, 17, 9, 40, 5, 4, (2, 1), "bf16"),
]


@pytest.mark.parametrize("ci", range(len(SPLIT3_GPU_CASES)))
@pytest.mark.parametrize("fuse", [False, True])
def test_split3x3_integer_exact(ci, fuse):
    n, c, h, w, k, r, s, pad, dt = SPLIT3_GPU_CASES[ci]
    say("split3x3", SPLIT3_GPU_CASES[ci], "fuse" if fuse else "staged")
    x = synth.random_tensor((n, h, w, c), 11000 + ci, dt, integer=True)
    wt = synth.random_tensor((r, s, k, c), 11100 + ci, dt, integer=True)
    out = ol.derived_conv2d(x.to(DEV), wt.to(DEV), 1, pad, fuse=fuse, split3x3=True)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(out), oracle.conv2d(x, wt, 1, pad, 1))


@pytest.mark.parametrize("integer", [False, True])
def test_srcnn_workload_direct_and_split_sampled(integer):
    """The SRCNN conv5x5 workload at full size, direct (fused 25 taps) and in the 3x3
    derived form (fused 3x3 stage + block OffsetAdd), on 4000 sampled outputs
    (borders included) evaluated one by one by the oracle."""
    wl = synth.WORKLOADS[6]
    say("srcnn workload", "integer" if integer else "float")
    x, wt = synth.conv_inputs(wl, integer=integer)
    ho, wo = wl.h, wl.w
    rng = np.random.default_rng(11300)
    idx = rng.integers(0, wl.n * ho * wo * wl.k, 4000)
    corners = [((i * ho + j) * wo + q) * wl.k + kk for i in range(wl.n) for j in (0, ho - 1)
               for q in (0, 1, wo - 2, wo - 1) for kk in (0, wl.k - 1)]
    idx = np.unique(np.concatenate([idx, np.array(corners)]))
    ref = oracle.conv2d(x, wt, wl.stride, wl.pad, 1, idx=idx)
    # direct (fused 25 taps); split with the fused 3x3 stage; split with the 3x3 stage's
    # GEMM and its two eOperators fused into one (no Z)
    for split, fuse in ((False, True), (True, True), (True, False)):
        out = ol.derived_conv2d(x.to(DEV), wt.to(DEV), wl.stride, wl.pad, fuse=fuse,
                                split3x3=split)
        torch.cuda.synchronize()
        got = to_np(out).reshape(-1)[idx]
        del out
        if integer:
            assert np.array_equal(got, ref), (split, fuse)
        else:
            assert err(got, ref) <= TOL_BF16, (split, fuse)
    torch.cuda.empty_cache()


@pytest.mark.parametrize("ci", [0, 1, 3, 5])
@pytest.mark.parametrize("out_bf16", [False, True])
def test_split3x3_fused_eoperator_chain(ci, out_bf16):
    """The split form's two consecutive eOperators fused into one kernel over the 3x3
    stage's scope (OLLIE_CONV_SPLIT_3X3 without OLLIE_FUSE_EPILOGUE): its workspace has
    no Z, and on integer inputs with a bias + ReLU tail it is exactly the definition and
    equal to the split form through Z (fused 3x3 stage, where covered); with a bf16
    scope, within the bf16 tolerance."""
    n, c, h, w, k, r, s, pad, dt = SPLIT3_GPU_CASES[ci]
    say("split3x3 fused chain", SPLIT3_GPU_CASES[ci], "bf16 out" if out_bf16 else "fp32 out")
    od = torch.bfloat16 if out_bf16 else torch.float32
    x = synth.random_tensor((n, h, w, c), 11400 + ci, dt, integer=True)
    wt = synth.random_tensor((r, s, k, c), 11500 + ci, dt, integer=True)
    bias = synth.random_tensor((k,), 11600 + ci, integer=True)
    desc = ol.conv_desc(tuple(x.shape), tuple(wt.shape), 1, pad, 1, 0, x.dtype, od)
    nb = ((r + 2) // 3) * ((s + 2) // 3)
    el = 2 if dt == "bf16" else 4
    w3_bytes = (9 * nb * k * c * el + 255) // 256 * 256
    assert ol.conv_workspace_bytes(desc, False, ol.CONV_SPLIT_3X3) == \
        w3_bytes + n * h * w * 9 * nb * k * 4
    ref = oracle.conv_epilogue(oracle.conv2d(x, wt, 1, pad, 1), bias, None, True)
    xg, wg, bg = x.to(DEV), wt.to(DEV), bias.to(DEV)
    out = ol.derived_conv2d(xg, wg, 1, pad, out_dtype=od, split3x3=True, bias=bg, relu=True)
    via_z = ol.derived_conv2d(xg, wg, 1, pad, out_dtype=od, split3x3=True, fuse=True,
                              bias=bg, relu=True)
    torch.cuda.synchronize()
    if out_bf16:
        assert torch.equal(out.cpu(), torch.from_numpy(ref).to(torch.bfloat16))
    else:
        assert np.array_equal(to_np(out), ref)
    assert torch.equal(out, via_z)
    out = ol.derived_conv2d(xg, wg, 1, pad, y_bf16=True, split3x3=True)
    torch.cuda.synchronize()
    assert err(to_np(out), oracle.conv2d(x, wt, 1, pad, 1)) <= TOL_BF16


def test_split3x3_float_tail_bf16_out_and_bf16_scope():
    """Random bf16 inputs: the split form with bias + ReLU and a bf16 out, and with a
    bf16 Y in its 3x3 stage, within the bf16 tolerance of the definition."""
    n, c, h, w, k, r, s, pad = 2, 64, 15, 13, 32, 5, 5, (2, 2)
    say("split3x3 float", n, c, h, w, k, r, s, pad)
    x = synth.random_tensor((n, h, w, c), 11200, "bf16", dist="normal")
    wt = synth.random_tensor((r, s, k, c), 11201, "bf16", dist="normal")
    bias = synth.random_tensor((k,), 11202)
    ref = oracle.conv2d(x, wt, 1, pad, 1)
    out = ol.derived_conv2d(x.to(DEV), wt.to(DEV), 1, pad, out_dtype=torch.bfloat16,
                            fuse=True, split3x3=True, bias=bias.to(DEV), relu=True)
    torch.cuda.synchronize()
    assert out.dtype == torch.bfloat16
    assert err(to_np(out), np.maximum(ref + bias.double().numpy(), 0.0)) <= TOL_BF16
    out = ol.derived_conv2d(x.to(DEV), wt.to(DEV), 1, pad, y_bf16=True, split3x3=True)
    torch.cuda.synchronize()
    assert err(to_np(out), ref) <= TOL_BF16


GEMM_CONFIGS = 5


@pytest.mark.parametrize("cfg", range(GEMM_CONFIGS))
@pytest.mark.parametrize("m,n,k", [(129, 257, 128), (300, 130, 192), (1000, 522, 64),
                                   (64, 64, 512), (260, 1030, 256), (300, 136, 128),
                                   (129, 260, 64)])
@pytest.mark.parametrize("y_bf16", [False, True])
def test_gemm_every_tile_config_integer_exact(cfg, m, n, k, y_bf16):
    """Every DMA tile configuration (flag bits GEMM_TILE(cfg)) of the GEMM stage, run as
    the two-stage path of a 1x1 convolution (x [1,1,m,k], wt [1,1,n,k]), whose OffsetAdd
    is the identity, so out = Y: exact for an fp32 Y, and for a bf16 Y equal to the exact
    sum rounded to nearest even.  n = 522 is not a multiple of 4 (element-wise row
    stores); n = 136 and 260 are multiples of 4 and 8 or 4 only with a ragged last tile
    (16-byte and 8-byte bf16 row stores)."""
    say("gemm cfg", cfg, m, n, k, "bf16 y" if y_bf16 else "fp32 y")
    a = synth.random_tensor((m, k), 6100 + m, "bf16", integer=True)
    b = synth.random_tensor((n, k), 7100 + n, "bf16", integer=True)
    out = ol.derived_conv2d(a.view(1, 1, m, k).to(DEV), b.view(1, 1, n, k).to(DEV), 1, 0,
                            y_bf16=y_bf16, flags=ol.GEMM_TILE(cfg))
    torch.cuda.synchronize()
    ref = a.double().numpy() @ b.double().numpy().T
    got = out.view(m, n).cpu()
    if y_bf16:
        assert torch.equal(got, torch.from_numpy(ref).to(torch.bfloat16).float())
    else:
        assert np.array_equal(got.numpy().astype(np.float64), ref)


@pytest.mark.parametrize("m,n,k", [(129, 257, 128), (300, 136, 64)])
@pytest.mark.parametrize("y_bf16", [False, True])
def test_gemm_stage_entry_point_integer_exact(m, n, k, y_bf16):
    """ollie_gemm_nt itself (automatic tile choice) on integer inputs."""
    say("gemm stage entry", m, n, k, y_bf16)
    a = synth.random_tensor((m, k), 6150 + m, "bf16", integer=True)
    b = synth.random_tensor((n, k), 7150 + n, "bf16", integer=True)
    y = ol.gemm_nt(a.to(DEV), b.to(DEV), y_dtype=torch.bfloat16 if y_bf16 else torch.float32)
    torch.cuda.synchronize()
    ref = a.double().numpy() @ b.double().numpy().T
    if y_bf16:
        assert torch.equal(y.cpu(), torch.from_numpy(ref).to(torch.bfloat16))
    else:
        assert np.array_equal(to_np(y), ref)


def test_gemm_stage_operand_over_2gib_sampled():
    """An A operand over 2 GiB takes the 64-bit address form of the DMA kernel; sampled
    rows (first, last, around the 2 GiB byte boundary and random) are exact."""
    m, n, k = (1 << 21) + 37, 72, 512
    say("gemm over 2 GiB", m, n, k)
    a = synth.device_integer_tensor((m, k), 6200, DEV)
    b = synth.device_integer_tensor((n, k), 6201, DEV)
    y = ol.gemm_nt(a, b)
    torch.cuda.synchronize()
    rng = np.random.default_rng(6202)
    rows = sorted(set([0, 1, (1 << 21) - 1, 1 << 21, m - 2, m - 1]
                      + rng.integers(0, m, 250).tolist()))
    idx = torch.tensor(rows, device=DEV)
    ref = a[idx].double().cpu().numpy() @ b.double().cpu().numpy().T
    assert np.array_equal(y[idx].cpu().numpy().astype(np.float64), ref)
    del a, y
    torch.cuda.empty_cache()


@pytest.mark.parametrize("m,n,k", [(1, 1, 1), (70, 33, 17), (200, 100, 45), (130, 136, 64)])
@pytest.mark.parametrize("y_bf16", [False, True])
def test_gemm_stage_fp32(m, n, k, y_bf16):
    """fp32 operands (the fp32 MFMA kernel) with an fp32 Y (<= 1e-5) and a bf16 Y
    (<= the bf16 tolerance; on integer inputs exactly the RNE rounding of the sum)."""
    say("gemm fp32", m, n, k, "bf16 y" if y_bf16 else "fp32 y")
    yd = torch.bfloat16 if y_bf16 else torch.float32
    a = synth.random_tensor((m, k), 8000 + m)
    b = synth.random_tensor((n, k), 9000 + n)
    y = ol.gemm_nt(a.to(DEV), b.to(DEV), y_dtype=yd)
    torch.cuda.synchronize()
    assert y.dtype == yd
    ref = a.double().numpy() @ b.double().numpy().T
    assert err(to_np(y), ref) <= (TOL_BF16 if y_bf16 else TOL_F32)
    ai = synth.random_tensor((m, k), 8100 + m, integer=True)
    bi = synth.random_tensor((n, k), 9100 + n, integer=True)
    y = ol.gemm_nt(ai.to(DEV), bi.to(DEV), y_dtype=yd)
    torch.cuda.synchronize()
    ref = torch.from_numpy(ai.double().numpy() @ bi.double().numpy().T).to(yd)
    assert torch.equal(y.cpu(), ref)


@pytest.mark.parametrize("integer", [True, False])
def test_fp32_conv_with_bf16_scope(integer):
    """fp32 inputs with OLLIE_Y_BF16 (the fp32 GEMM kernel storing a bf16 scope): the
    tiny 3x3 workload and a ragged strided shape, against the oracle within the bf16
    tolerance (bf16 Y carries the bf16 rounding of every partial)."""
    wl = synth.WORKLOADS[1]
    say("fp32 conv, bf16 Y, integer", integer)
    x, wt = synth.conv_inputs(wl, integer=integer)
    out = run_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil, y_bf16=True)
    ref = oracle_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil)
    assert err(to_np(out), ref) <= TOL_BF16
    if integer:
        # integer partials of 16 channels of {-3..3} products stay below 256: exact in bf16
        assert np.array_equal(to_np(out), ref)
    kind, n, c, h, w, k, r, s, st, pd, dl, op = SMALL[1]
    x = synth.random_tensor((n, h, w, c), 8200, integer=integer)
    wt = synth.random_tensor((r, s, k, c), 8201, integer=integer)
    out = run_conv(kind, x, wt, st, pd, dl, op, y_bf16=True)
    assert err(to_np(out), oracle_conv(kind, x, wt, st, pd, dl, op)) <= TOL_BF16


@pytest.mark.parametrize("transposed", [False, True])
def test_eop_stage_alone(transposed):
    """The eOperator kernel on a scope Y computed on the CPU, against the NumPy
    derived-form eOperator (itself pinned to the definition)."""
    say("eop stage transposed=%s" % transposed)
    if transposed:
        shape, st, pd, dl, op = (2, 5, 6, 8), (2, 2), (1, 1), (1, 1), (1, 1)
    else:
        shape, st, pd, dl, op = (2, 9, 7, 8), (1, 2), (2, 1), (2, 1), (0, 0)
    r, s, k = 3, 4, 12
    x = synth.random_tensor(shape, 10000, integer=True)
    wt = synth.random_tensor((r, s, k, shape[3]), 10001, integer=True)
    y = dfm.gemm_stage(x.numpy(), wt.numpy())
    if transposed:
        ref = dfm.selective_add(y, x.shape, wt.shape, st, pd, dl, op)
    else:
        ref = dfm.offset_add(y, x.shape, wt.shape, st, pd, dl)
    desc = ol.conv_desc(tuple(x.shape), tuple(wt.shape), st, pd, dl, op, torch.float32,
                        torch.float32)
    out = ol.eop_gather(desc, transposed, torch.as_tensor(y, dtype=torch.float32).to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(to_np(out), ref)


# (transposed, x shape, r, s, k, stride, pad, dil, out_pad): the unrolled-tap eOperator
# kernel with 2 and 3 candidates per axis (forward; transposed with tap steps 1, 2 and
# 3), the loop kernel (5x5 taps; k % 4 != 0; a grid over 2^20 threads).
EOP_CASES = [
    (False, (2, 9, 7, 8), 3, 3, 12, (1, 2), (2, 1), (2, 1), (0, 0)),
    (False, (1, 6, 5, 8), 2, 1, 8, (1, 1), (1, 0), (1, 1), (0, 0)),
    (False, (1, 8, 8, 8), 5, 5, 8, (1, 1), (2, 2), (1, 1), (0, 0)),
    (True, (2, 5, 6, 8), 4, 4, 12, (2, 2), (1, 1), (1, 1), (1, 1)),
    (True, (1, 5, 5, 8), 3, 3, 8, (1, 1), (1, 1), (1, 1), (0, 0)),
    (True, (1, 5, 6, 8), 3, 3, 8, (2, 2), (1, 2), (2, 2), (1, 1)),
    (True, (1, 4, 5, 8), 3, 3, 8, (3, 3), (1, 1), (2, 2), (2, 1)),
    (False, (1, 9, 7, 8), 3, 3, 6, (1, 1), (1, 1), (1, 1), (0, 0)),
    (False, (1, 130, 128, 8), 3, 3, 256, (1, 1), (1, 1), (1, 1), (0, 0)),
]


@pytest.mark.parametrize("ci", range(len(EOP_CASES)))
@pytest.mark.parametrize("y_bf16", [False, True])
def test_eop_kernels_integer_exact(ci, y_bf16):
    """The eOperator stage alone on an integer scope Y (exact in bf16 too), against the
    NumPy derived-form eOperator, for every kernel choice."""
    tr, shape, r, s, k, st, pd, dl, op = EOP_CASES[ci]
    say("eop kernels", EOP_CASES[ci], "bf16 y" if y_bf16 else "fp32 y")
    x = synth.random_tensor(shape, 10100 + ci, integer=True)
    wt = synth.random_tensor((r, s, k, shape[3]), 10200 + ci, integer=True)
    y = dfm.gemm_stage(x.numpy(), wt.numpy())
    if tr:
        ref = dfm.selective_add(y, x.shape, wt.shape, st, pd, dl, op)
    else:
        ref = dfm.offset_add(y, x.shape, wt.shape, st, pd, dl)
    desc = ol.conv_desc(tuple(x.shape), tuple(wt.shape), st, pd, dl, op, torch.float32,
                        torch.float32)
    yt = torch.as_tensor(y, dtype=torch.float32)
    if y_bf16:
        yt = yt.to(torch.bfloat16)
    out = ol.eop_gather(desc, tr, yt.to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(to_np(out), ref)


def test_outputs_stay_in_bounds_and_runs_are_deterministic():
    wl = synth.WORKLOADS[3]
    say("canary + determinism, workload 3")
    x, wt = synth.conv_inputs(wl)
    xg, wg = x.to(DEV), wt.to(DEV)
    desc = ol.conv_desc(tuple(x.shape), tuple(wt.shape), wl.stride, wl.pad, wl.dil, wl.out_pad,
                        x.dtype, torch.float32)
    ho, wo = ol.conv_out_hw(desc, True)
    numel = wl.n * ho * wo * wl.k
    ws_need = ol.conv_workspace_bytes(desc, True)
    big = torch.full((numel + 4096,), 12345.0, device=DEV)
    wsbig = torch.full((ws_need + 8192,), 7, dtype=torch.uint8, device=DEV)
    outs = []
    for _ in range(2):
        out = big[:numel].view(wl.n, ho, wo, wl.k)
        ol.derived_conv_transpose2d(xg, wg, wl.stride, wl.pad, wl.out_pad, wl.dil, out=out,
                                    ws=wsbig[:ws_need])
        torch.cuda.synchronize()
        outs.append(out.clone())
    assert (big[numel:] == 12345.0).all()
    assert (wsbig[ws_need:] == 7).all()
    assert torch.equal(outs[0], outs[1])


# ------------------------------------------------------------------------- band

def band_rows_sample(b, l, dil, w, n_random, seed):
    """Rows at both ends of every residue subsequence and around the band edges, plus
    a seeded random sample."""
    rng = np.random.default_rng(seed)
    rows = set()
    edge = list(range(0, min(l, 2 * dil + 2))) + list(range(max(0, l - 2 * dil - 2), l))
    edge += [i for i in (w * dil - 1, w * dil, w * dil + 1, l - w * dil - 1, l - w * dil)
             if 0 <= i < l]
    for bi in (0, b - 1):
        rows.update(bi * l + i for i in edge)
    rows.update(int(v) for v in rng.integers(0, b * l, size=n_random))
    return np.array(sorted(rows), dtype=np.int64)


def check_band(q, k, v, w, dil, scale, mask, staged, rows=None, tol=TOL_BF16,
               out_dtype=torch.float32, flags=0):
    qg, kg, vg = q.to(DEV), k.to(DEV), v.to(DEV)
    o = ol.banded_bmm(qg, kg, vg, w, dil, scale, mask_invalid=mask, staged=staged,
                      out_dtype=out_dtype, flags=flags)
    torch.cuda.synchronize()
    on = to_np(o).reshape(-1, q.shape[2])
    assert np.isfinite(on).all()
    _, _, ref = oracle.band(q, k, v, w, dil, scale, mask, rows=rows, want_s=False,
                            want_p=False)
    got = on if rows is None else on[rows]
    e = err(got, ref.reshape(got.shape))
    say("band err %.3e" % e)
    assert e <= tol
    return o


BAND_SMALL = [  # (b, l, w, dil)
    (2, 300, 17, 1),
    (1, 257, 40, 2),
    (3, 129, 5, 3),
    (1, 100, 130, 2),     # band wider than the sequence
    (2, 64, 0, 1),        # window of one
    (1, 1, 3, 1),         # single row
    (1, 515, 64, 4),
    (2, 3, 2, 5),         # dilation above the length: residues 3 and 4 are empty
]


@pytest.mark.parametrize("ci", range(len(BAND_SMALL)))
@pytest.mark.parametrize("mask", [False, True])
@pytest.mark.parametrize("staged", [False, True])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_band_small(ci, mask, staged, out_dtype):
    """Every path (fused / staged, zero / mask mode) with an fp32 and a bf16 O."""
    b, l, w, dil = BAND_SMALL[ci]
    say("band small", BAND_SMALL[ci], "mask", mask, "staged", staged, "O", out_dtype)
    q = synth.random_tensor((b, l, 64), 11000 + ci, "bf16", dist="normal")
    k = synth.random_tensor((b, l, 64), 12000 + ci, "bf16", dist="normal")
    v = synth.random_tensor((b, l, 64), 13000 + ci, "bf16", dist="normal")
    o = check_band(q, k, v, w, dil, 0.125, mask, staged, out_dtype=out_dtype)
    assert o.dtype == out_dtype


# The staged G2BMM and GBMM move S and P rows (2w+1 entries, starting at any 4- or
# 2-byte offset) as aligned 16-byte chunks, carrying the entries that straddle two key
# blocks: the widest bands the staged softmax takes (2w+1 up to 1023), several tiles per
# residue subsequence, S compared entry by entry and O through the staged path.
BAND_WIDE = [(1, 700, 511, 1), (2, 600, 300, 3), (1, 1500, 257, 2)]


@pytest.mark.parametrize("ci", range(len(BAND_WIDE)))
@pytest.mark.parametrize("mask", [False, True])
def test_band_staged_wide_bands(ci, mask):
    b, l, w, dil = BAND_WIDE[ci]
    say("band staged wide", BAND_WIDE[ci], "mask", mask)
    q = synth.random_tensor((b, l, 64), 15000 + ci, "bf16", dist="normal")
    k = synth.random_tensor((b, l, 64), 15100 + ci, "bf16", dist="normal")
    v = synth.random_tensor((b, l, 64), 15200 + ci, "bf16", dist="normal")
    o, sg = ol.banded_bmm(q.to(DEV), k.to(DEV), v.to(DEV), w, dil, 0.125, mask_invalid=mask,
                          staged=True, return_s=True)
    torch.cuda.synchronize()
    s_ref, _, o_ref = oracle.band(q, k, v, w, dil, 0.125, mask, want_p=False)
    sn = to_np(sg).reshape(s_ref.shape)
    # S is a bf16 x bf16 dot product accumulated in fp32: exact up to rounding, and
    # every entry outside [0, l) holds the zero-mode value 0 exactly
    assert err(sn, s_ref) <= 1e-5
    on = to_np(o).reshape(o_ref.shape)
    assert np.isfinite(on).all()
    assert err(on, o_ref) <= TOL_BF16


# Every wave shape of the fused band kernel (flag bits BAND_SHAPE(0..3)): 32
# or 64 queries per wave, four or two waves per workgroup, on the small cases and
# sequences long enough for several workgroups per residue subsequence (in the last,
# the second tile of every odd residue lies past its subsequence).
@pytest.mark.parametrize("ci", range(len(BAND_SMALL) + 4))
@pytest.mark.parametrize("mask", [False, True])
@pytest.mark.parametrize("cfg", [0, 1, 2, 3])
def test_band_every_wave_shape(cfg, mask, ci):
    extra = [(2, 1100, 96, 2), (48, 2000, 64, 3), (64, 2600, 40, 1), (300, 257, 16, 2)]
    b, l, w, dil = BAND_SMALL[ci] if ci < len(BAND_SMALL) else extra[ci - len(BAND_SMALL)]
    say("band wave shape", cfg, (b, l, w, dil), "mask", mask)
    q = synth.random_tensor((b, l, 64), 14000 + ci, "bf16", dist="normal")
    k = synth.random_tensor((b, l, 64), 14100 + ci, "bf16", dist="normal")
    v = synth.random_tensor((b, l, 64), 14200 + ci, "bf16", dist="normal")
    check_band(q, k, v, w, dil, 0.125, mask, False, flags=ol.BAND_SHAPE(cfg))


@pytest.mark.parametrize("mask", [False, True])
def test_band_scores_exact_on_integers(mask):
    """Staged G2BMM scores are exact for integer Q, K; softmax rows sum to one."""
    b, l, w, dil = 2, 333, 20, 3
    say("band integer scores mask", mask)
    q = synth.random_tensor((b, l, 64), 14000, "bf16", integer=True)
    k = synth.random_tensor((b, l, 64), 14001, "bf16", integer=True)
    v = synth.random_tensor((b, l, 64), 14002, "bf16", dist="normal")
    o, s = ol.banded_bmm(q.to(DEV), k.to(DEV), v.to(DEV), w, dil, 1.0, mask_invalid=mask,
                         return_s=True)
    torch.cuda.synchronize()
    sref, pref, oref = oracle.band(q, k, v, w, dil, 1.0, mask)
    assert np.array_equal(to_np(s), sref)
    assert err(to_np(o), oref) <= TOL_BF16
    p = ol.band_softmax(s, w, dil, mask_invalid=mask)
    torch.cuda.synchronize()
    pn = to_np(p)
    assert (pn >= 0).all()
    np.testing.assert_allclose(pn.sum(-1), 1.0, atol=2e-2)
    assert err(pn, pref) <= TOL_BF16


_BAND_WL_REF = {}


@pytest.mark.parametrize("staged,out_dtype", [(False, torch.float32), (True, torch.float32),
                                               (False, torch.bfloat16), (True, torch.bfloat16)])
def test_band_workload_every_row(staged, out_dtype):
    """The Longformer band workload (zero mode) against the oracle on all 393,216 rows,
    fused and staged, with an fp32 and a bf16 O (one oracle pass serves the four)."""
    wl = synth.WORKLOADS[5]
    say("band workload, every row, staged", staged, "O", out_dtype)
    q, k, v = synth.band_inputs(wl)
    if "o" not in _BAND_WL_REF:
        _BAND_WL_REF["o"] = oracle.band(q, k, v, wl.w, wl.dilation, wl.scale, wl.mask_invalid,
                                        want_s=False, want_p=False)[2]
    o = ol.banded_bmm(q.to(DEV), k.to(DEV), v.to(DEV), wl.w, wl.dilation, wl.scale,
                      mask_invalid=wl.mask_invalid, staged=staged, out_dtype=out_dtype)
    torch.cuda.synchronize()
    assert o.dtype == out_dtype
    e = err(to_np(o), _BAND_WL_REF["o"])
    say("band err %.3e" % e)
    assert e <= TOL_BF16


def test_band_workload_mask_mode_bf16_out():
    wl = synth.WORKLOADS[5]
    say("band workload mask mode, bf16 O")
    q, k, v = synth.band_inputs(wl, seed_offset=20)
    rows = band_rows_sample(wl.b, wl.l, wl.dilation, wl.w, 2000, 6)
    o = check_band(q, k, v, wl.w, wl.dilation, wl.scale, True, False, rows,
                   out_dtype=torch.bfloat16)
    assert o.dtype == torch.bfloat16


def test_band_fused_and_staged_agree_at_full_size():
    """Property at full size on every row: the fused and staged paths compute the same
    O (both within tolerance of each other) with no NaN anywhere."""
    wl = synth.WORKLOADS[5]
    say("band fused vs staged full size")
    q, k, v = (t.to(DEV) for t in synth.band_inputs(wl, seed_offset=30))
    o1 = ol.banded_bmm(q, k, v, wl.w, wl.dilation, wl.scale)
    o2 = ol.banded_bmm(q, k, v, wl.w, wl.dilation, wl.scale, staged=True)
    torch.cuda.synchronize()
    assert torch.isfinite(o1).all() and torch.isfinite(o2).all()
    d = (o1 - o2).abs().max().item() / o2.abs().max().item()
    assert d <= TOL_BF16


@pytest.mark.parametrize("staged", [False, True])
@pytest.mark.parametrize("mask", [False, True])
def test_band_subsequence_over_4gib_sampled(mask, staged):
    """A residue subsequence whose keys span more than 4 GiB takes the band kernel's
    64-bit address form (and the staged kernels' 64-bit row offsets, S and P then
    spanning 0.9 and 0.5 GB).  Sampled query rows (sequence ends, and keys on both
    sides of the 2^31- and 2^32-byte offsets of the subsequence) match the oracle run
    on the window of keys each row reaches (the same keys lie inside and outside
    [0, L), so the same rows and zero/masked entries enter its softmax)."""
    b, l, w, dil, scale = 1, (1 << 25) + 4096, 3, 2, 0.05
    say("band over 4 GiB", b, l, w, dil, "mask" if mask else "no mask",
        "staged" if staged else "fused")
    q = synth.device_integer_tensor((b, l, 64), 6300, DEV)
    k = synth.device_integer_tensor((b, l, 64), 6301, DEV)
    v = synth.device_integer_tensor((b, l, 64), 6302, DEV)
    o = ol.banded_bmm(q, k, v, w, dil, scale, mask_invalid=mask, staged=staged)
    torch.cuda.synchronize()
    rng = np.random.default_rng(6303)
    rows = sorted(set([0, 1, 5, l - 1, l - 2, l - 7, (1 << 24) - 1, 1 << 24, (1 << 24) + 1,
                       (1 << 25) - 2, (1 << 25) - 1, 1 << 25, (1 << 25) + 1]
                      + rng.integers(0, l, 40).tolist()))
    for i in rows:
        lo, hi = max(0, i - w * dil), min(l, i + w * dil + 1)
        win = [t[:, lo:hi].float().cpu() for t in (q, k, v)]
        _, _, ref = oracle.band(*win, w, dil, scale, mask, rows=[i - lo], want_s=False,
                                want_p=False)
        got = o[0, i].cpu().numpy()
        assert np.isfinite(got).all()
        assert err(got, ref.reshape(got.shape)) <= TOL_BF16, i
    del q, k, v, o
    torch.cuda.empty_cache()


@pytest.mark.parametrize("scale", [0.0, -0.3])
@pytest.mark.parametrize("mask", [False, True])
@pytest.mark.parametrize("staged", [False, True])
def test_band_scale_edge_cases(scale, mask, staged):
    """Zero scale (uniform softmax over the live entries) and a negative scale."""
    say("band scale", scale, "mask", mask, "staged", staged)
    b, l, w, dil = 2, 211, 9, 2
    q = synth.random_tensor((b, l, 64), 15000, "bf16", dist="normal")
    k = synth.random_tensor((b, l, 64), 15001, "bf16", dist="normal")
    v = synth.random_tensor((b, l, 64), 15002, "bf16", dist="normal")
    check_band(q, k, v, w, dil, scale, mask, staged)


# ------------------------------------------------------- fused GEMM + eOperator path

@pytest.mark.parametrize("cfg", [2, 3, 4])
@pytest.mark.parametrize("integer", [True, False])
def test_workload_fused(cfg, integer):
    """The fused expression (no Y) on the three convolution workloads."""
    wl = synth.WORKLOADS[cfg]
    say("workload", cfg, "fused integer=%s" % integer)
    x, wt = synth.conv_inputs(wl, integer=integer, seed_offset=40)
    xg, wg = x.to(DEV), wt.to(DEV)
    desc = ol.conv_desc(tuple(x.shape), tuple(wt.shape), wl.stride, wl.pad, wl.dil, wl.out_pad,
                        x.dtype, torch.float32)
    assert ol.conv_workspace_bytes(desc, wl.transposed, ol.FUSE_EPILOGUE) == 0
    if wl.kind == "conv2d":
        out = ol.derived_conv2d(xg, wg, wl.stride, wl.pad, fuse=True)
    elif wl.kind == "dilated_conv2d":
        out = ol.derived_dilated_conv2d(xg, wg, wl.stride, wl.pad, wl.dil, fuse=True)
    else:
        out = ol.derived_conv_transpose2d(xg, wg, wl.stride, wl.pad, wl.out_pad, wl.dil,
                                          fuse=True)
    torch.cuda.synchronize()
    ref = oracle_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad)
    if integer:
        assert np.array_equal(to_np(out), ref)
    else:
        assert err(to_np(out), ref) <= TOL_BF16


# c % 64 == 0 so the fused kernel takes them; ragged pixel counts and channel counts,
# strides, dilations, and transposed cases whose residue classes have 0, 1 or 2 taps.
SMALL_FUSED = [
    ("conv2d", 3, 64, 13, 11, 20, 3, 3, (1, 1), (1, 1), (1, 1), (0, 0)),
    ("conv2d", 1, 128, 17, 19, 36, 3, 2, (2, 1), (0, 1), (1, 1), (0, 0)),
    ("conv2d", 2, 64, 5, 6, 7, 5, 5, (1, 1), (4, 4), (1, 1), (0, 0)),
    ("dilated_conv2d", 1, 64, 21, 18, 12, 3, 3, (1, 1), (3, 2), (3, 2), (0, 0)),
    ("dilated_conv2d", 2, 128, 10, 10, 130, 3, 3, (2, 2), (2, 2), (2, 2), (0, 0)),
    ("conv_transpose2d", 3, 64, 5, 6, 12, 4, 4, (2, 2), (1, 1), (1, 1), (1, 0)),
    ("conv_transpose2d", 1, 64, 9, 7, 8, 3, 2, (3, 2), (1, 1), (1, 2), (2, 1)),
    ("conv_transpose2d", 2, 128, 4, 4, 5, 2, 2, (1, 1), (0, 0), (1, 1), (0, 0)),
    ("conv_transpose2d", 1, 64, 3, 5, 16, 1, 1, (3, 3), (0, 0), (1, 1), (2, 2)),
]


@pytest.mark.parametrize("ci", range(len(SMALL_FUSED)))
@pytest.mark.parametrize("integer", [True, False])
def test_small_shapes_fused(ci, integer):
    kind, n, c, h, w, k, r, s, st, pd, dl, op = SMALL_FUSED[ci]
    say("small fused", SMALL_FUSED[ci], integer)
    x = synth.random_tensor((n, h, w, c), 16000 + ci, "bf16", integer=integer, dist="normal")
    wt = synth.random_tensor((r, s, k, c), 17000 + ci, "bf16", integer=integer, dist="normal")
    xg, wg = x.to(DEV), wt.to(DEV)
    desc = ol.conv_desc(tuple(x.shape), tuple(wt.shape), st, pd, dl, op, x.dtype,
                        torch.float32)
    assert ol.conv_workspace_bytes(desc, kind == "conv_transpose2d", ol.FUSE_EPILOGUE) == 0
    if kind == "conv2d":
        out = ol.derived_conv2d(xg, wg, st, pd, fuse=True)
    elif kind == "dilated_conv2d":
        out = ol.derived_dilated_conv2d(xg, wg, st, pd, dl, fuse=True)
    else:
        out = ol.derived_conv_transpose2d(xg, wg, st, pd, op, dl, fuse=True)
    torch.cuda.synchronize()
    ref = oracle_conv(kind, x, wt, st, pd, dl, op)
    if integer:
        assert np.array_equal(to_np(out), ref)
    else:
        assert err(to_np(out), ref) <= TOL_BF16


# Every tile shape of the fused expression (flag bits FUSED_TILE(0..14)), on
# shapes that exercise the row-window kernel (config 9: stride-1 forms whose class width
# is a multiple of 16 dividing 192 -- ragged channel tiles, tiles straddling images,
# kernel widths 1-3) and on shapes where config 9 falls back to the automatic choice.
TILE_CASES = [
    # kind, n, c, h, w, k, r, s, stride, pad, dil, out_pad, residues
    ("conv2d", 2, 128, 9, 32, 72, 3, 3, (1, 1), (1, 1), (1, 1), (0, 0), False),
    ("dilated_conv2d", 1, 64, 13, 64, 40, 3, 3, (1, 1), (2, 2), (2, 2), (0, 0), True),
    ("dilated_conv2d", 1, 64, 10, 96, 24, 3, 2, (1, 1), (1, 1), (2, 2), (0, 0), True),
    ("conv2d", 1, 64, 6, 16, 20, 1, 1, (1, 1), (0, 0), (1, 1), (0, 0), False),
    ("conv_transpose2d", 2, 64, 5, 6, 12, 4, 4, (2, 2), (1, 1), (1, 1), (1, 0), False),
    ("dilated_conv2d", 1, 64, 8, 32, 130, 3, 3, (1, 1), (2, 2), (2, 2), (0, 0), False),
]


FUSED_CONFIGS = 15


@pytest.mark.parametrize("ci", range(len(TILE_CASES)))
@pytest.mark.parametrize("cfg", range(FUSED_CONFIGS))
def test_every_tile_shape_integer_exact(cfg, ci):
    kind, n, c, h, w, k, r, s, st, pd, dl, op, res = TILE_CASES[ci]
    say("tile shape", cfg, TILE_CASES[ci])
    fl = ol.FUSED_TILE(cfg)
    x = synth.random_tensor((n, h, w, c), 36000 + ci, "bf16", integer=True)
    wt = synth.random_tensor((r, s, k, c), 36100 + ci, "bf16", integer=True)
    xg, wg = x.to(DEV), wt.to(DEV)
    if kind == "conv2d":
        out = ol.derived_conv2d(xg, wg, st, pd, fuse=True, flags=fl)
    elif kind == "dilated_conv2d":
        out = ol.derived_dilated_conv2d(xg, wg, st, pd, dl, fuse=True, residues=res, flags=fl)
    else:
        out = ol.derived_conv_transpose2d(xg, wg, st, pd, op, dl, fuse=True, flags=fl)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(out), oracle_conv(kind, x, wt, st, pd, dl, op))


def test_fused_flag_falls_back_to_two_stages():
    """c % 64 != 0: the fused kernel does not cover the shape, the call takes the
    two-stage path (and needs its workspace)."""
    kind, n, c, h, w, k, r, s, st, pd, dl, op = SMALL_BF16[0]
    say("fused fallback", SMALL_BF16[0])
    x = synth.random_tensor((n, h, w, c), 18000, "bf16", integer=True)
    wt = synth.random_tensor((r, s, k, c), 18001, "bf16", integer=True)
    desc = ol.conv_desc(tuple(x.shape), tuple(wt.shape), st, pd, dl, op, x.dtype,
                        torch.float32)
    assert ol.conv_workspace_bytes(desc, False, ol.FUSE_EPILOGUE) == \
        ol.conv_workspace_bytes(desc, False, 0) > 0
    out = ol.derived_conv2d(x.to(DEV), wt.to(DEV), st, pd, fuse=True)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(out), oracle_conv(kind, x, wt, st, pd, dl, op))


def test_fused_bf16_output_and_determinism():
    wl = synth.WORKLOADS[4]
    say("fused bf16 out + determinism, workload 4")
    x, wt = synth.conv_inputs(wl, seed_offset=50)
    xg, wg = x.to(DEV), wt.to(DEV)
    a = ol.derived_dilated_conv2d(xg, wg, wl.stride, wl.pad, wl.dil, fuse=True)
    b = ol.derived_dilated_conv2d(xg, wg, wl.stride, wl.pad, wl.dil, fuse=True)
    o16 = ol.derived_dilated_conv2d(xg, wg, wl.stride, wl.pad, wl.dil, fuse=True,
                                    out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    ref = oracle_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil)
    assert err(to_np(o16), ref) <= TOL_BF16


def test_hip_graph_replays_match_eager():
    """The library's calls captured in a HIP graph (as the benchmark does) give the
    eager results on every replay, with eager work and synchronisations in between."""
    say("hip graph replay vs eager")
    wl2, wl4 = synth.WORKLOADS[2], synth.WORKLOADS[4]
    x2, w2 = (t.to(DEV) for t in synth.conv_inputs(wl2, seed_offset=60))
    x4, w4 = (t.to(DEV) for t in synth.conv_inputs(wl4, seed_offset=60))
    q, k, v = (synth.random_tensor((4, 777, 64), 19000 + i, "bf16", dist="normal").to(DEV)
               for i in range(3))
    desc2 = ol.conv_desc(tuple(x2.shape), tuple(w2.shape), 1, 1, 1, 0, x2.dtype, torch.float32)
    ws2 = torch.empty(ol.conv_workspace_bytes(desc2, False), dtype=torch.uint8, device=DEV)
    o2 = torch.empty((16, 14, 14, 256), device=DEV)
    o4 = torch.empty((1, 96, 128, 512), device=DEV)
    ob = torch.empty((4, 777, 64), device=DEV)
    # the 3x3 split form: weight split, 3x3 stage and block OffsetAdd in one call
    x5 = synth.random_tensor((2, 21, 19, 64), 19010, "bf16", dist="normal").to(DEV)
    w5 = synth.random_tensor((5, 5, 24, 64), 19011, "bf16", dist="normal").to(DEV)
    desc5 = ol.conv_desc(tuple(x5.shape), tuple(w5.shape), 1, 2, 1, 0, x5.dtype, torch.float32)
    ws5 = torch.empty(ol.conv_workspace_bytes(desc5, False, ol.CONV_SPLIT_3X3 | ol.FUSE_EPILOGUE),
                      dtype=torch.uint8, device=DEV)
    o5 = torch.empty((2, 21, 19, 24), device=DEV)

    def calls():
        ol.derived_conv2d(x2, w2, 1, 1, out=o2, ws=ws2)
        ol.derived_dilated_conv2d(x4, w4, 1, 2, 2, out=o4, fuse=True)
        ol.banded_bmm(q, k, v, 40, 3, 0.125, out=ob)
        ol.derived_conv2d(x5, w5, 1, 2, out=o5, ws=ws5, fuse=True, split3x3=True)

    outs = (o2, o4, ob, o5)
    calls()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    for i in range(4):
        for t in outs:
            t.fill_(float("nan"))
        ws5.fill_(0xff)                                  # stale workspace between replays
        junk = torch.randn(1 << 20, device=DEV) * i      # unrelated eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert float(junk.abs().sum()) >= 0
        for got, exp in zip(outs, ref):
            assert torch.equal(got, exp), f"replay {i} differs from the eager result"


# ------------------------------------------- element-wise tail (bias, residual, ReLU)
# (kind, n, c, h, w, k, r, s, stride, pad, dil, out_pad); c % 64 == 0 so that the
# fused path covers them too
EPI_CASES = [
    ("conv2d", 2, 64, 9, 11, 72, 3, 3, (1, 1), (1, 1), (1, 1), (0, 0)),
    ("dilated_conv2d", 1, 128, 12, 10, 48, 3, 3, (1, 1), (2, 2), (2, 2), (0, 0)),
    ("conv_transpose2d", 2, 64, 5, 6, 40, 4, 4, (2, 2), (1, 1), (1, 1), (0, 0)),
]


def _epi_run(kind, x, wt, stride, pad, dil, out_pad, fuse, **kw):
    xg, wg = x.to(DEV), wt.to(DEV)
    if kind == "conv2d":
        out = ol.derived_conv2d(xg, wg, stride, pad, fuse=fuse, **kw)
    elif kind == "dilated_conv2d":
        out = ol.derived_dilated_conv2d(xg, wg, stride, pad, dil, fuse=fuse, **kw)
    else:
        out = ol.derived_conv_transpose2d(xg, wg, stride, pad, out_pad, dil, fuse=fuse, **kw)
    torch.cuda.synchronize()
    return out


def _epi_inputs(case, seed, integer, bias_dtype=torch.float32, res_dtype=torch.float32):
    kind, n, c, h, w, k, r, s, stride, pad, dil, op = case
    x = synth.random_tensor((n, h, w, c), seed, "bf16", integer=integer)
    wt = synth.random_tensor((r, s, k, c), seed + 1, "bf16", integer=integer)
    conv = oracle_conv(kind, x, wt, stride, pad, dil, op)
    dt = lambda d: "bf16" if d == torch.bfloat16 else "f32"
    bias = synth.random_tensor((k,), seed + 2, dt(bias_dtype), integer=integer)
    res = synth.random_tensor(conv.shape, seed + 3, dt(res_dtype), integer=integer)
    return x, wt, conv, bias, res


@pytest.mark.parametrize("ci", range(len(EPI_CASES)))
@pytest.mark.parametrize("fuse", [False, True])
@pytest.mark.parametrize("relu", [False, True])
def test_epilogue_integer_exact(ci, fuse, relu):
    """Integer-valued inputs, bias and residual: conv + bias + residual is an exact
    integer, so both paths must equal the definition exactly, ReLU included."""
    case = EPI_CASES[ci]
    kind, stride, pad, dil, op = case[0], case[8], case[9], case[10], case[11]
    say("epilogue", kind, "fuse=%s relu=%s integer" % (fuse, relu))
    x, wt, conv, bias, res = _epi_inputs(case, 31000 + 10 * ci, True)
    ref = oracle.conv_epilogue(conv, bias, res, relu)
    out = _epi_run(kind, x, wt, stride, pad, dil, op, fuse, bias=bias.to(DEV),
                   residual=res.to(DEV), relu=relu)
    assert np.array_equal(to_np(out), ref)
    if relu:
        assert (ref == 0).any() and (ref > 0).any()


@pytest.mark.parametrize("ci", range(len(EPI_CASES)))
@pytest.mark.parametrize("fuse", [False, True])
def test_epilogue_terms_and_dtypes(ci, fuse):
    """Each term alone and in bf16, float inputs, fp32 and bf16 outputs."""
    case = EPI_CASES[ci]
    kind, stride, pad, dil, op = case[0], case[8], case[9], case[10], case[11]
    x, wt, conv, bias, res = _epi_inputs(case, 32000 + 10 * ci, False, torch.bfloat16,
                                         torch.bfloat16)
    for kw in ({"bias": bias}, {"residual": res}, {"relu": True},
               {"bias": bias, "residual": res, "relu": True}):
        for out_dtype in (torch.float32, torch.bfloat16):
            say("epilogue", kind, "fuse=%s" % fuse, sorted(kw), out_dtype)
            ref = oracle.conv_epilogue(conv, kw.get("bias"), kw.get("residual"),
                                       kw.get("relu", False))
            gkw = {k2: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k2, v in kw.items()}
            out = _epi_run(kind, x, wt, stride, pad, dil, op, fuse, out_dtype=out_dtype, **gkw)
            assert err(to_np(out), ref) <= TOL_BF16


@pytest.mark.parametrize("fuse", [False, True])
def test_epilogue_residual_in_place(fuse):
    """residual may be the output buffer itself (x + conv written over x)."""
    case = EPI_CASES[0]
    kind, stride, pad, dil, op = case[0], case[8], case[9], case[10], case[11]
    x, wt, conv, bias, res = _epi_inputs(case, 33000, True)
    ref = oracle.conv_epilogue(conv, bias, res, True)
    buf = res.to(DEV).clone()
    out = _epi_run(kind, x, wt, stride, pad, dil, op, fuse, bias=bias.to(DEV), residual=buf,
                   relu=True, out=buf)
    assert out.data_ptr() == buf.data_ptr()
    assert np.array_equal(to_np(buf), ref)


def test_epilogue_resnet_workload_fused():
    """The ResNet conv3x3 workload with the tail of a residual block (bias, identity
    shortcut, ReLU), fused into the single kernel of the fused expression."""
    wl = synth.WORKLOADS[2]
    say("epilogue resnet workload")
    x, wt = synth.conv_inputs(wl, seed_offset=40)
    conv = oracle_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil)
    bias = synth.random_tensor((wl.k,), 34001, "f32")
    res = synth.random_tensor(conv.shape, 34002, "bf16", dist="normal")
    ref = oracle.conv_epilogue(conv, bias, res, True)
    for fuse in (True, False):
        out = ol.derived_conv2d(x.to(DEV), wt.to(DEV), wl.stride, wl.pad, fuse=fuse,
                                bias=bias.to(DEV), residual=res.to(DEV), relu=True)
        torch.cuda.synchronize()
        assert err(to_np(out), ref) <= TOL_BF16


# ------------------------------- dilated conv as residue sub-image convolutions (§6.2)
# (n, c, h, w, k, dil, pad); stride 1, 3x3
RESIDUE_CASES = [
    (1, 64, 14, 18, 40, (2, 2), (2, 2)),
    (2, 128, 11, 9, 72, (3, 2), (1, 2)),     # ragged classes, asymmetric dilation
    (1, 64, 13, 13, 64, (4, 4), (4, 4)),     # 16 classes x 9 taps
    (1, 64, 7, 10, 24, (2, 3), (0, 0)),      # no padding
]


@pytest.mark.parametrize("ci", range(len(RESIDUE_CASES)))
def test_residue_form_integer_exact(ci):
    n, c, h, w, k, dil, pad = RESIDUE_CASES[ci]
    say("residue form", RESIDUE_CASES[ci])
    x = synth.random_tensor((n, h, w, c), 35000 + ci, "bf16", integer=True)
    wt = synth.random_tensor((3, 3, k, c), 35100 + ci, "bf16", integer=True)
    ref = oracle.conv2d(x, wt, (1, 1), pad, dil)
    out = ol.derived_dilated_conv2d(x.to(DEV), wt.to(DEV), 1, pad, dil, residues=True)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(out), ref)


def test_residue_form_workload_and_tail():
    """The CSRNet workload in the residue form: against the oracle, against the
    default fused form, and with a bias + ReLU tail."""
    wl = synth.WORKLOADS[4]
    say("residue form workload")
    x, wt = synth.conv_inputs(wl, seed_offset=50)
    ref = oracle_conv(wl.kind, x, wt, wl.stride, wl.pad, wl.dil)
    xg, wg = x.to(DEV), wt.to(DEV)
    out = ol.derived_dilated_conv2d(xg, wg, wl.stride, wl.pad, wl.dil, residues=True)
    base = ol.derived_dilated_conv2d(xg, wg, wl.stride, wl.pad, wl.dil, fuse=True)
    torch.cuda.synchronize()
    assert err(to_np(out), ref) <= TOL_BF16
    # same taps summed in the same order: the two schedules agree bit for bit
    assert torch.equal(out, base)
    bias = synth.random_tensor((wl.k,), 35201, "f32")
    out = ol.derived_dilated_conv2d(xg, wg, wl.stride, wl.pad, wl.dil, residues=True,
                                    bias=bias.to(DEV), relu=True)
    torch.cuda.synchronize()
    assert err(to_np(out), oracle.conv_epilogue(ref, bias, None, True)) <= TOL_BF16


def test_residue_form_rejections():
    x = torch.zeros((1, 9, 9, 64), dtype=torch.bfloat16, device=DEV)
    wt = torch.zeros((3, 3, 8, 64), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(ol.OllieError):
        ol.derived_dilated_conv2d(x, wt, 2, 2, 2, residues=True)          # stride 2
    with pytest.raises(ol.OllieError):
        ol.derived_dilated_conv2d(x, wt, 1, 5, 5, residues=True)          # 25 classes
    with pytest.raises(ol.OllieError):
        ol.derived_dilated_conv2d(x[..., :32].contiguous(), wt[..., :32].contiguous(), 1, 2, 2,
                                  residues=True)                          # c % 64 != 0
