"""The derivation engine drives the library: for every workload the C ABI call is built
from what the hybrid derivation emits -- the convolution descriptor's stride, padding
and dilation and the entry point from the Matmul + eOperator plan, the band's
half-width and dilation from the residue-split non-dilated band, the split form's
blocks and padding checked against the library's workspace -- not from the workload's
own definition, and the kernels' output is compared with the oracle."""
import ctypes
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2208_02025_amd as ol
from paper_2208_02025_amd import derive as D
import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL_F32, TOL_BF16 = 1e-5, 2e-2


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape and np.isfinite(got).all()
    return float(np.abs(got - ref).max() / max(np.abs(ref).max(), 1e-30))


def run_plan(plan, wl, x, wt, flags):
    """The C ABI call the plan describes, through ctypes on the current stream."""
    f = D.conv_desc_fields(plan, wl.n, wl.c, wl.h, wl.w, wl.k, wl.r, wl.s)
    in_dt = ol.BF16 if x.dtype == torch.bfloat16 else ol.F32
    op = wl.out_pad if plan.transposed else (0, 0)
    desc = ol.ConvDesc(f["n"], f["c"], f["h"], f["w"], f["k"], f["r"], f["s"],
                       f["stride_h"], f["stride_w"], f["pad_h"], f["pad_w"], f["dil_h"],
                       f["dil_w"], op[0], op[1], in_dt, ol.F32)
    ho, wo = ol.conv_out_hw(desc, plan.transposed)
    out = torch.empty((wl.n, ho, wo, wl.k), dtype=torch.float32, device=DEV)
    need = ol.conv_workspace_bytes(desc, plan.transposed, flags)
    ws = torch.empty(max(need, 16), dtype=torch.uint8, device=DEV)
    lib = ol.load_library()
    entry = D.conv_entry(plan)
    st = getattr(lib, entry)(ctypes.byref(desc), ctypes.c_void_p(x.data_ptr()),
                             ctypes.c_void_p(wt.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                             ctypes.c_void_p(ws.data_ptr()), need, flags,
                             ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == ol.OK, lib.ollie_last_error().decode()
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
@pytest.mark.parametrize("fuse", [False, True])
def test_convolution_workloads_from_derived_plans(cfg, fuse):
    wl = synth.WORKLOADS[cfg]
    say("engine plan, workload", cfg, wl.name, "fused" if fuse else "two-stage")
    if wl.transposed:
        prog = D.conv_transpose2d_expr(wl.n, wl.c, wl.h, wl.w, wl.k, wl.r, wl.s, wl.stride,
                                       wl.pad, wl.dil, wl.out_pad)
    else:
        prog = D.conv2d_expr(wl.n, wl.c, wl.h, wl.w, wl.k, wl.r, wl.s, wl.stride, wl.pad,
                             wl.dil)
    plan, dv = D.derive_conv(prog, transposed=wl.transposed)
    assert dv.guided > 0 and dv.matches[0].op == "Matmul"
    # the plan's entry point is the one the workload's operator calls for
    assert D.conv_entry(plan) == {"conv2d": "derived_conv2d",
                                  "dilated_conv2d": "derived_dilated_conv2d",
                                  "conv_transpose2d": "derived_conv_transpose2d"}[wl.kind]
    integer = cfg != 1
    x, wt = synth.conv_inputs(wl, integer=integer)
    out = run_plan(plan, wl, x.to(DEV), wt.to(DEV), ol.FUSE_EPILOGUE if fuse else 0)
    if wl.transposed:
        ref = oracle.conv_transpose2d(x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad)
    else:
        ref = oracle.conv2d(x, wt, wl.stride, wl.pad, wl.dil)
    if integer:
        assert np.array_equal(out.cpu().numpy(), ref)
    else:
        assert err(out.cpu().numpy(), ref) <= TOL_F32


def test_band_workload_from_the_derived_band():
    wl = synth.WORKLOADS[5]
    say("engine plan, band workload")
    plan, m0, m1 = D.derive_band(wl.b, wl.l, wl.d, wl.w, wl.dilation)
    assert m0.detail["dilation"] == wl.dilation and m1.detail["dilation"] == 1
    assert sum(n for _, _, n in plan.residues) == wl.l
    q, k, v = synth.band_inputs(wl)
    desc = ol.BandDesc(wl.b, wl.l, wl.d, plan.w, plan.dilation, wl.scale, ol.BF16, ol.F32)
    qg, kg, vg = q.to(DEV), k.to(DEV), v.to(DEV)
    o = torch.empty(tuple(q.shape), dtype=torch.float32, device=DEV)
    lib = ol.load_library()
    st = lib.banded_bmm(ctypes.byref(desc), ctypes.c_void_p(qg.data_ptr()),
                        ctypes.c_void_p(kg.data_ptr()), ctypes.c_void_p(vg.data_ptr()),
                        ctypes.c_void_p(o.data_ptr()), None, None, 0, 0,
                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == ol.OK, lib.ollie_last_error().decode()
    torch.cuda.synchronize()
    _, _, ref = oracle.band(q, k, v, wl.w, wl.dilation, wl.scale, wl.mask_invalid,
                            want_s=False, want_p=False)
    assert err(o.cpu().numpy(), ref) <= TOL_BF16


@pytest.mark.parametrize("fuse", [False, True])
def test_srcnn_workload_from_the_derived_split_form(fuse):
    wl = synth.WORKLOADS[6]
    say("engine plan, SRCNN split form", "fused 3x3 stage" if fuse else "fused eOperators")
    plan, _ = D.derive_split3x3(wl.n, wl.c, wl.h, wl.w, wl.k, wl.r, wl.s, wl.pad)
    flags = ol.CONV_SPLIT_3X3 | (ol.FUSE_EPILOGUE if fuse else 0)
    desc = ol.conv_desc((wl.n, wl.h, wl.w, wl.c), (wl.r, wl.s, wl.k, wl.c), 1, wl.pad, 1, 0,
                        torch.bfloat16, torch.float32)
    # the library lays the workspace out exactly as the plan derives it
    assert ol.conv_workspace_bytes(desc, False, flags) == D.split3_workspace_bytes(
        plan, wl.n, wl.c, wl.h, wl.w, wl.k, 2, fuse)
    x, wt = synth.conv_inputs(wl, integer=True)
    out = ol.derived_conv2d(x.to(DEV), wt.to(DEV), 1, plan.pad3[0] - (3 * plan.nbr - wl.r),
                            fuse=fuse, split3x3=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(53000)
    idx = np.unique(rng.integers(0, out.numel(), 3000))
    ref = oracle.conv2d(x, wt, 1, wl.pad, 1, idx=idx)
    assert np.array_equal(out.cpu().numpy().reshape(-1)[idx], ref)
    del out
    torch.cuda.empty_cache()
