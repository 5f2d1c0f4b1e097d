"""CPU-only checks of the C ABI: the library loads, exports every function that
include/ollie.h declares, and rejects invalid arguments with the documented status
before touching the GPU (no compute call is made here)."""
import ctypes
import os
import re

import pytest

import paper_2208_02025_amd as ol

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ollie.h")

# Fake, never-dereferenced device addresses: validation fails before any HIP call.
A16 = ctypes.c_void_p(0x10000)
B16 = ctypes.c_void_p(0x20000)
C16 = ctypes.c_void_p(0x30000)
W16 = ctypes.c_void_p(0x40000)
MIS = ctypes.c_void_p(0x2000008)   # misaligned, clear of the other fake tensors
WSB = ctypes.c_void_p(0x1000000)   # a band workspace clear of the fake tensors above


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    return ol.load_library()


def test_header_declares_the_four_entry_points():
    names = header_functions()
    for n in ("derived_conv2d", "derived_conv_transpose2d", "derived_dilated_conv2d",
              "banded_bmm"):
        assert n in names


def test_library_exports_every_declared_function(lib):
    names = header_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), f"{n} declared in ollie.h but not exported"
    assert set(names) == set(ol.EXPORTS)


def test_version(lib):
    assert "gfx950" in ol.version()


def conv(n=1, c=16, h=14, w=14, k=16, r=3, s=3, stride=1, pad=1, dil=1, op=0,
         in_dtype=ol.BF16, out_dtype=ol.F32):
    return ol.ConvDesc(n, c, h, w, k, r, s, stride, stride, pad, pad, dil, dil, op, op,
                       in_dtype, out_dtype)


def call_conv(lib, entry, d, x=A16, wt=B16, out=C16, ws=W16, ws_bytes=None, flags=0):
    if ws_bytes is None:
        ws_bytes = 1 << 40
    st = getattr(lib, entry)(ctypes.byref(d) if d is not None else None, x, wt, out, ws,
                             ws_bytes, flags, None)
    return st, lib.ollie_last_error().decode()


@pytest.mark.parametrize("entry", ["derived_conv2d", "derived_dilated_conv2d",
                                   "derived_conv_transpose2d"])
def test_conv_error_paths(lib, entry):
    tr = entry == "derived_conv_transpose2d"
    good_stride = 2 if tr else 1
    cases = [
        (None, {}, ol.EINVAL),
        (conv(n=0), {}, ol.EINVAL),
        (conv(c=0), {}, ol.EINVAL),
        (conv(stride=0), {}, ol.EINVAL),
        (conv(dil=0), {}, ol.EINVAL),
        (conv(pad=-1), {}, ol.EINVAL),
        (conv(in_dtype=7), {}, ol.EDTYPE),
        (conv(out_dtype=3, stride=good_stride), {}, ol.EDTYPE),
        (conv(stride=good_stride), {"x": None}, ol.EINVAL),
        (conv(stride=good_stride), {"ws": None}, ol.EINVAL),
        (conv(stride=good_stride), {"ws_bytes": 10}, ol.EWORKSPACE),
        (conv(stride=good_stride), {"out": MIS}, ol.EALIGN),
        (conv(c=12, stride=good_stride), {}, ol.EALIGN),          # bf16 rows not 16-byte multiples
        (conv(stride=good_stride), {"flags": 1 << 9}, ol.EINVAL),
        (conv(n=1 << 40, stride=good_stride), {}, ol.EINVAL),     # overflow
    ]
    if tr:
        cases += [(conv(stride=2, op=2), {}, ol.EINVAL),          # out_pad >= max(stride, dil)
                  (conv(stride=1, op=1), {}, ol.EINVAL),
                  (conv(h=1, w=1, r=1, s=1, stride=1, pad=1), {}, ol.EINVAL)]   # empty output
    else:
        cases += [(conv(op=1), {}, ol.EINVAL),                    # out_pad on a forward conv
                  (conv(h=2, w=2, r=5, s=5, pad=0), {}, ol.EINVAL)]           # empty output
    if entry == "derived_conv2d":
        cases.append((conv(dil=2, pad=2), {}, ol.EINVAL))
    for d, kw, want in cases:
        st, msg = call_conv(lib, entry, d, **kw)
        assert st == want, (entry, kw, msg)
        assert msg, "every failure sets a message"


def test_conv_out_hw_and_workspace(lib):
    d = conv(n=16, c=256, k=256)                                  # 3x3 conv, 14x14, pad 1
    assert ol.conv_out_hw(d, False) == (14, 14)
    assert ol.conv_workspace_bytes(d, False) == 16 * 14 * 14 * 9 * 256 * 4
    assert ol.conv_workspace_bytes(d, False, ol.Y_BF16) == 16 * 14 * 14 * 9 * 256 * 2
    d = conv(n=16, c=512, h=8, w=8, k=256, r=4, s=4, stride=2, pad=1)
    assert ol.conv_out_hw(d, True) == (16, 16)
    d = conv(n=1, c=512, h=96, w=128, k=512, pad=2, dil=2)
    assert ol.conv_out_hw(d, False) == (96, 128)
    with pytest.raises(ol.OllieError):
        ol.conv_out_hw(conv(h=2, w=2, r=5, s=5, pad=0), False)
    assert ol.conv_workspace_bytes(conv(n=0), False) == 0


def band(b=2, l=64, d=64, w=4, dil=2, in_dtype=ol.BF16, out_dtype=ol.F32):
    return ol.BandDesc(b, l, d, w, dil, 1.0, in_dtype, out_dtype)


def test_band_error_paths(lib):
    def call(d, q=A16, s_out=None, ws=None, ws_bytes=0, flags=0, o=C16):
        st = lib.banded_bmm(ctypes.byref(d), q, B16, W16, o, s_out, ws, ws_bytes, flags, None)
        return st, lib.ollie_last_error().decode()

    cases = [
        (band(d=32), {}, ol.EINVAL),
        (band(b=0), {}, ol.EINVAL),
        (band(l=0), {}, ol.EINVAL),
        (band(w=-1), {}, ol.EINVAL),
        (band(dil=0), {}, ol.EINVAL),
        (band(in_dtype=ol.F32), {}, ol.EDTYPE),
        (band(out_dtype=9), {}, ol.EDTYPE),
        (band(), {"q": None}, ol.EINVAL),
        (band(), {"o": MIS}, ol.EALIGN),
        (band(), {"s_out": C16}, ol.EINVAL),                        # s_out needs the staged path
        (band(), {"flags": 1 << 7}, ol.EINVAL),
        (band(), {"flags": ol.BAND_STAGED}, ol.EINVAL),             # staged without workspace
        (band(), {"flags": ol.BAND_STAGED, "ws": WSB, "ws_bytes": 100}, ol.EWORKSPACE),
        (band(w=600), {"flags": ol.BAND_STAGED, "ws": WSB, "ws_bytes": 1 << 40}, ol.EINVAL),
    ]
    for d, kw, want in cases:
        st, msg = call(d, **kw)
        assert st == want, (kw, msg)
        assert msg


def test_band_workspace_bytes(lib):
    d = band(b=96, l=4096, w=256, dil=2)
    assert ol.band_workspace_bytes(d, 0) == 0
    s_bytes = 96 * 4096 * 513 * 4
    p_off = (s_bytes + 255) // 256 * 256
    assert ol.band_workspace_bytes(d, ol.BAND_STAGED) == p_off + 96 * 4096 * 513 * 2
    # the staged softmax holds at most 1024 band entries per row: wider bands, which
    # banded_bmm rejects, and invalid descriptors need no workspace size
    assert ol.band_workspace_bytes(band(w=511), ol.BAND_STAGED) > 0
    assert ol.band_workspace_bytes(band(w=512), ol.BAND_STAGED) == 0
    assert ol.band_workspace_bytes(band(w=1 << 29), ol.BAND_STAGED) == 0
    assert ol.band_workspace_bytes(band(b=0), ol.BAND_STAGED) == 0


def test_gemm_error_paths(lib):
    def call(m=64, n=64, k=64, a=A16, b=B16, y=C16, it=ol.BF16, yt=ol.F32):
        return lib.ollie_gemm_nt(m, n, k, a, b, y, it, yt, None)

    assert call(m=0) == ol.EINVAL
    assert call(k=-1) == ol.EINVAL
    assert call(a=None) == ol.EINVAL
    assert call(it=4) == ol.EDTYPE
    assert call(y=MIS) == ol.EALIGN
    assert call(k=20) == ol.EALIGN                                  # bf16 needs k % 8 == 0
    assert call(m=1 << 40, k=1 << 30) == ol.EINVAL


def test_stage_error_paths(lib):
    d = conv()
    for entry in ("ollie_eop_offset_sum", "ollie_eop_convt_gather"):
        fn = getattr(lib, entry)
        assert fn(ctypes.byref(d), None, ol.F32, C16, None) == ol.EINVAL
        assert fn(ctypes.byref(d), A16, 5, C16, None) == ol.EDTYPE
        assert fn(ctypes.byref(d), A16, ol.F32, MIS, None) == ol.EALIGN
    bd = band()
    assert lib.ollie_band_g2bmm(ctypes.byref(bd), A16, None, C16, None) == ol.EINVAL
    assert lib.ollie_band_softmax(ctypes.byref(bd), A16, MIS, 0, None) == ol.EALIGN
    assert lib.ollie_band_softmax(ctypes.byref(bd), A16, C16, 1 << 5, None) == ol.EINVAL
    assert lib.ollie_band_gbmm(ctypes.byref(band(d=16)), A16, B16, C16, None) == ol.EINVAL


def test_python_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(1, 4, 4, 8, dtype=torch.bfloat16)
    wt = torch.zeros(3, 3, 8, 8, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        ol.derived_conv2d(x, wt, 1, 1)
    q = torch.zeros(1, 8, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        ol.banded_bmm(q, q, q, 2, 1)


def test_fused_workspace_sizes(lib):
    d = conv(n=16, c=256, k=256)
    assert ol.conv_workspace_bytes(d, False, ol.FUSE_EPILOGUE) == 0
    assert ol.conv_workspace_bytes(d, False, 0) == 16 * 14 * 14 * 9 * 256 * 4
    d = conv(n=2, c=72, k=16)                      # c % 64 != 0: two-stage path
    assert ol.conv_workspace_bytes(d, False, ol.FUSE_EPILOGUE) == 2 * 14 * 14 * 9 * 16 * 4
    d = conv(n=1, c=64, k=16, in_dtype=ol.F32)     # fp32 inputs: two-stage path
    assert ol.conv_workspace_bytes(d, False, ol.FUSE_EPILOGUE) > 0
    d = conv(n=16, c=512, h=8, w=8, k=256, r=4, s=4, stride=2, pad=1)
    assert ol.conv_workspace_bytes(d, True, ol.FUSE_EPILOGUE) == 0


def test_epilogue_error_paths(lib):
    d = conv()
    def call(entry, **kw):
        e = ol.ConvEpilogue(kw.get("bias", W16.value), kw.get("residual", None),
                            kw.get("bias_dtype", ol.F32), kw.get("residual_dtype", ol.F32),
                            kw.get("relu", 1))
        st = getattr(lib, entry)(ctypes.byref(d), A16, B16, C16, W16, 1 << 40, 0,
                                 ctypes.byref(e), None)
        return st, lib.ollie_last_error().decode()
    for entry in ("ollie_derived_conv2d_ex", "ollie_derived_dilated_conv2d_ex"):
        assert call(entry, relu=2)[0] == ol.EINVAL
        assert call(entry, bias_dtype=7)[0] == ol.EDTYPE
        assert call(entry, residual=C16.value, residual_dtype=5)[0] == ol.EDTYPE
        assert call(entry, bias=0x40008)[0] == ol.EALIGN
        assert call(entry, residual=0x40004)[0] == ol.EALIGN
        st, msg = call(entry, relu=3)
        assert msg
    # a NULL tensor's dtype is not looked at
    dt = conv(stride=2)
    e = ol.ConvEpilogue(None, None, 9, 9, 0)
    st = lib.ollie_derived_conv_transpose2d_ex(ctypes.byref(dt), A16, B16, C16, W16, 10, 0,
                                               ctypes.byref(e), None)
    assert st == ol.EWORKSPACE          # the epilogue passed; the workspace check fired
    # the plain entry points are the _ex ones with no tail
    st = lib.ollie_derived_conv2d_ex(ctypes.byref(conv(dil=2, pad=2)), A16, B16, C16, W16,
                                     1 << 40, 0, None, None)
    assert st == ol.EINVAL


def test_library_exports_nothing_else(lib):
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    res = subprocess.run([nm, "-D", "--defined-only", ol.LIB_PATH], capture_output=True,
                         text=True, check=True)
    funcs = {ln.split()[-1] for ln in res.stdout.splitlines() if " T " in ln}
    assert funcs == set(header_functions())


def test_residue_flag_rejections(lib):
    def call(entry, d, flags):
        return getattr(lib, entry)(ctypes.byref(d), A16, B16, C16, W16, 1 << 40, flags, None)
    R = ol.DILATED_RESIDUES | ol.FUSE_EPILOGUE
    d_ok = conv(c=64, dil=2, pad=2)
    assert call("derived_conv2d", conv(c=64), R) == ol.EINVAL                 # wrong entry
    assert call("derived_conv_transpose2d", conv(c=64, stride=2), R) == ol.EINVAL
    assert call("derived_dilated_conv2d", d_ok, ol.DILATED_RESIDUES) == ol.EINVAL  # no fuse
    assert call("derived_dilated_conv2d", conv(c=64, dil=2, pad=2, stride=2), R) == ol.EINVAL
    assert call("derived_dilated_conv2d", conv(c=32, dil=2, pad=2), R) == ol.EINVAL
    assert call("derived_dilated_conv2d", conv(c=64, dil=5, pad=5), R) == ol.EINVAL
    assert call("derived_dilated_conv2d", conv(c=64, dil=2, pad=2, in_dtype=ol.F32), R) == ol.EINVAL
    assert ol.conv_workspace_bytes(d_ok, False, R) == 0


def test_split3x3_flag_rejections_and_workspace(lib):
    S = ol.CONV_SPLIT_3X3
    d5 = conv(c=64, r=5, s=5, pad=2)
    assert call_conv(lib, "derived_conv_transpose2d", conv(c=64, r=5, s=5, stride=2, pad=2),
                     flags=S)[0] == ol.EINVAL
    assert call_conv(lib, "derived_dilated_conv2d", d5, flags=S)[0] == ol.EINVAL
    assert call_conv(lib, "derived_conv2d", conv(c=64, r=5, s=5, stride=2, pad=2),
                     flags=S)[0] == ol.EINVAL
    assert call_conv(lib, "derived_conv2d", d5, ws=None, flags=S)[0] == ol.EINVAL
    assert call_conv(lib, "derived_conv2d", d5, ws_bytes=1000, flags=S)[0] == ol.EWORKSPACE
    assert call_conv(lib, "derived_conv2d", conv(c=12, r=5, s=5, pad=2),
                     flags=S)[0] == ol.EALIGN            # bf16 rows of 24 bytes
    assert call_conv(lib, "derived_conv2d", d5, out=MIS, flags=S)[0] == ol.EALIGN
    # W3 [3][3][4*16][64] bf16, then Z [1][18][18][64] fp32 (fused 3x3 stage) or the 3x3
    # stage's scope Y [14*14][9*64] (GEMM stage; its two eOperators run fused, no Z)
    w3, z, y = 9 * 64 * 64 * 2, 18 * 18 * 64 * 4, 14 * 14 * 9 * 64 * 4
    assert ol.conv_workspace_bytes(d5, False, S) == w3 + y
    assert ol.conv_workspace_bytes(d5, False, S | ol.FUSE_EPILOGUE) == w3 + z
    assert ol.conv_workspace_bytes(d5, False, S | ol.Y_BF16) == w3 + y // 2
    assert ol.conv_workspace_bytes(d5, True, S) == 0
    # a 4x2 kernel: blocks 2x1, relaxed taps er = 2, es = 1: Z is (14+2*3-2) x (14+2*2-2)
    d42 = conv(c=64, r=4, s=2, pad=1)
    assert ol.conv_workspace_bytes(d42, False, S | ol.FUSE_EPILOGUE) == \
        9 * 32 * 64 * 2 + 18 * 16 * 32 * 4


def test_validation_never_lets_a_bad_descriptor_through(lib):
    """Randomised descriptors with invalid fields: every call returns a non-zero status
    with a message before any HIP call (fake device pointers are never touched)."""
    import random
    rng = random.Random(7)
    bad = 0
    for _ in range(400):
        d = conv(n=rng.choice([0, 1, 2, -1]), c=rng.choice([0, 16, 64, -5]),
                 h=rng.choice([0, 1, 7]), w=rng.choice([1, 9, 0]), k=rng.choice([0, 8, -1]),
                 r=rng.choice([0, 1, 3, 9]), s=rng.choice([1, 3, -2]),
                 stride=rng.choice([0, 1, 2]), pad=rng.choice([-1, 0, 1, 4]),
                 dil=rng.choice([0, 1, 2]), op=rng.choice([0, 1, 3]),
                 in_dtype=rng.choice([ol.BF16, ol.F32, 5]), out_dtype=rng.choice([ol.F32, 9]))
        invalid = (min(d.n, d.c, d.h, d.w, d.k, d.r, d.s) < 1 or d.stride_h < 1 or d.dil_h < 1
                   or d.pad_h < 0 or d.in_dtype not in (0, 1) or d.out_dtype not in (0, 1))
        if not invalid:
            continue
        bad += 1
        for entry in ("derived_conv2d", "derived_dilated_conv2d", "derived_conv_transpose2d"):
            st, msg = call_conv(lib, entry, d)
            assert st != ol.OK and msg, (entry, st)
    assert bad > 100


def test_tile_override_bits(lib):
    """Tile-configuration flag bits: in range they pass validation (the call then fails
    later on the deliberately short workspace), out of range they give OLLIE_EINVAL."""
    d = conv(c=64)
    for fl in (ol.FUSED_TILE(0), ol.FUSED_TILE(14), ol.GEMM_TILE(0), ol.GEMM_TILE(4)):
        assert call_conv(lib, "derived_conv2d", d, ws_bytes=8, flags=fl)[0] == ol.EWORKSPACE
    for fl in (ol.FUSED_TILE(15), ol.FUSED_TILE(200), ol.GEMM_TILE(5), ol.GEMM_TILE(14)):
        st, msg = call_conv(lib, "derived_conv2d", d, flags=fl)
        assert st == ol.EINVAL and "tile" in msg
    assert call_conv(lib, "derived_conv2d", d, flags=1 << 30)[0] == ol.EINVAL  # unknown bit
    bd = band()
    def bcall(flags, ws_bytes=0):
        return lib.banded_bmm(ctypes.byref(bd), A16, B16, C16, W16, None, WSB, ws_bytes,
                              flags, None)
    assert bcall(ol.BAND_SHAPE(4)) == ol.EINVAL
    assert bcall(ol.BAND_STAGED | ol.BAND_SHAPE(2), ws_bytes=8) == ol.EWORKSPACE
    assert bcall(ol.GEMM_TILE(0)) == ol.EINVAL                # not a band flag


def test_overlapping_buffers_are_rejected(lib):
    """Outputs may not overlap inputs or the workspace (OLLIE_EINVAL); a residual may be
    the output buffer itself (same dtype) but may not overlap it otherwise."""
    d = conv(c=64, k=32)                      # x 25088 B, wt 36864 B, out 25088 B (fp32)
    x, wt, out, ws = 0x100000, 0x200000, 0x300000, 0x400000
    P = ctypes.c_void_p
    def c(**kw):
        a = dict(x=x, wt=wt, out=out, ws=ws)
        a.update(kw)
        return call_conv(lib, "derived_conv2d", d, P(a["x"]), P(a["wt"]), P(a["out"]),
                         P(a["ws"]), 1 << 30)
    assert c(out=x + 1024)[0] == ol.EINVAL              # out inside x
    assert c(out=wt - 1024)[0] == ol.EINVAL             # out runs into wt
    assert c(out=ws + 4096)[0] == ol.EINVAL             # out inside the workspace
    assert c(ws=x + 4096)[0] == ol.EINVAL               # workspace over x
    st, msg = c(x=out)
    assert st == ol.EINVAL and "overlap" in msg
    # epilogue aliasing
    def e(bias, res, res_dtype=ol.F32):
        ep = ol.ConvEpilogue(bias, res, ol.F32, res_dtype, 0)
        st = lib.ollie_derived_conv2d_ex(ctypes.byref(d), P(x), P(wt), P(out), P(ws), 8, 0,
                                         ctypes.byref(ep), None)
        return st, lib.ollie_last_error().decode()
    assert e(None, out)[0] == ol.EWORKSPACE              # in place: allowed
    assert e(None, out, ol.BF16)[0] == ol.EINVAL         # in place with another dtype
    assert e(None, out + 16)[0] == ol.EINVAL             # shifted residual
    assert e(out + 64, None)[0] == ol.EINVAL             # bias inside out
    assert e(out - 64, None)[0] == ol.EINVAL             # 32 fp32 bias values run into out
    assert e(out - 128, out - (1 << 20))[0] == ol.EWORKSPACE
    # GEMM stage, eOperator stage, band
    assert lib.ollie_gemm_nt(64, 64, 64, P(x), P(wt), P(x + 4096), ol.BF16, ol.F32,
                             None) == ol.EINVAL
    assert lib.ollie_eop_offset_sum(ctypes.byref(conv()), P(x), ol.F32, P(x + 16), None) == \
        ol.EINVAL
    bd = band(b=1, l=64)                                  # q/k/v 8 KB each, O fp32 16 KB
    def b(q, k, v, o, flags=0, ws_=None, ws_bytes=0, s_out=None):
        return lib.banded_bmm(ctypes.byref(bd), P(q), P(k), P(v), P(o), P(s_out), P(ws_),
                              ws_bytes, flags, None)
    assert b(x, wt, out, x + 4096) == ol.EINVAL          # o over q
    assert b(x, wt, out, ws, ol.BAND_STAGED, ws, 1 << 30) == ol.EINVAL   # o over ws
    assert b(x, wt, out, ws, ol.BAND_STAGED, ws + (1 << 20), 1 << 30, s_out=out + 32) == \
        ol.EINVAL                                        # s_out over v
    assert lib.ollie_band_gbmm(ctypes.byref(bd), P(x), P(wt), P(x + 64), None) == ol.EINVAL
    assert lib.ollie_band_softmax(ctypes.byref(bd), P(x), P(x + 64), 0, None) == ol.EINVAL
    assert lib.ollie_band_g2bmm(ctypes.byref(bd), P(x), P(wt), P(wt + 64), None) == ol.EINVAL


def test_build_digest_tracks_the_sources(tmp_path):
    """The digest stored beside libollie.so covers every source, the header and the
    flags: editing any of them changes it."""
    import shutil
    from paper_2208_02025_amd import _build
    csrc = tmp_path / "csrc"
    shutil.copytree(_build.CSRC, csrc)
    hdr = tmp_path / "ollie.h"
    shutil.copy(_build.HEADER, hdr)
    base = _build.source_digest(str(csrc), str(hdr))
    assert base == _build.source_digest(str(csrc), str(hdr))
    assert base == _build.source_digest()                 # same content, other place
    src = csrc / "eop.hip"
    src.write_text(src.read_text() + "\n// edit\n")
    assert _build.source_digest(str(csrc), str(hdr)) != base
    src.write_text(src.read_text()[: -len("\n// edit\n")])
    assert _build.source_digest(str(csrc), str(hdr)) == base
    hdr.write_text(hdr.read_text().replace("OLLIE_OK = 0", "OLLIE_OK = 0 "))
    assert _build.source_digest(str(csrc), str(hdr)) != base


def test_stale_library_is_rebuilt(tmp_path, monkeypatch):
    """A library whose recorded digest differs from the sources is not current, and
    load_library() then rebuilds before loading."""
    from paper_2208_02025_amd import _build
    lib, stamp = tmp_path / "libx.so", tmp_path / "libx.so.sha256"
    lib.write_bytes(b"")
    assert not _build.is_current(str(lib), str(stamp))      # no stamp
    stamp.write_text("0" * 64 + "\n")
    assert not _build.is_current(str(lib), str(stamp))      # stale stamp
    stamp.write_text(_build.source_digest() + "\n")
    assert _build.is_current(str(lib), str(stamp))
    calls = []
    monkeypatch.setattr(ol, "_lib", None)
    monkeypatch.setattr(_build, "is_current", lambda *a: False)
    monkeypatch.setattr(_build, "build", lambda *a, **k: calls.append(1) or _build.LIB)
    ol.load_library()
    assert calls == [1]


def test_noalloc_entry_rejects_oversized_and_invalid_calls(lib):
    """ollie_derived_conv2d_noalloc: a workspace beyond its 64 MiB static scratch gives
    OLLIE_EWORKSPACE, invalid descriptors the usual status, all before any HIP call."""
    def call(d, flags=0):
        st = lib.ollie_derived_conv2d_noalloc(ctypes.byref(d) if d is not None else None,
                                              A16, B16, C16, flags, None)
        return st, lib.ollie_last_error().decode()
    big = conv(n=1, c=512, h=96, w=128, k=512, pad=2)          # 226 MB fp32 scope
    st, msg = call(big)
    assert st == ol.EWORKSPACE and "scratch" in msg
    assert call(None)[0] == ol.EINVAL
    assert call(conv(stride=0))[0] == ol.EINVAL
    assert call(conv(dil=2, pad=2))[0] == ol.EINVAL             # dilation belongs elsewhere
    assert call(conv(in_dtype=7))[0] == ol.EDTYPE
