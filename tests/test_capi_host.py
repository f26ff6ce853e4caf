"""C-ABI contract checks that need no GPU: the library loads, exports every entry point the
header declares, and rejects bad arguments synchronously with the documented status codes
(validation returns before any HIP call, so these run on a machine without a GPU).

The validation tests pass made-up device addresses, which only validation ever sees.  Should a
check regress, the call would go on to launch a kernel on an unmapped address; on a machine with
a visible GPU that could fault the device, so there those tests are skipped (the GPU suite
covers the same entry points with real buffers)."""
import ctypes
import re
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
HEADER = ROOT / "include" / "nvfp4ss.h"


@pytest.fixture(scope="module")
def nv():
    import paper_2606_07618_amd as nv
    return nv


def declared_functions():
    text = re.sub(r"/\*.*?\*/", "", HEADER.read_text(), flags=re.S)
    return sorted(set(re.findall(r"\b(nvfp4_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol(nv):
    names = declared_functions()
    assert {"nvfp4_quant_absmax", "nvfp4_quant_four_over_six", "nvfp4_quant_scalesweep_mse",
            "nvfp4_quant_scalesweep_wmse", "nvfp4_dequant", "nvfp4_workspace_bytes",
            "nvfp4_status_string"} <= set(names)
    raw = ctypes.CDLL(str(nv.LIB_PATH))
    for n in names:
        assert hasattr(raw, n), n


def test_status_strings_and_workspace_size(nv):
    assert nv.nvfp4_workspace_bytes() >= 16
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -8, 12345):
        assert isinstance(nv.nvfp4_status_string(code), bytes)


P = ctypes.c_void_p
FAKE = P(0x100000)        # never dereferenced: validation fails before any use
FAKE8 = P(0x100008)


def _device_visible() -> bool:
    import torch
    return torch.cuda.device_count() > 0     # counts devices without initializing one


fake_pointers = pytest.mark.skipif(_device_visible(),
                                   reason="made-up device addresses only where no GPU is visible")


def call(nv, name, **kw):
    a = dict(x=FAKE, dtype=1, rows=4, cols=64, block=16, w=FAKE, D=256.0, static=0.0,
             S=FAKE, q=FAKE, sc=FAKE, ws=None, wsb=0, stream=None)
    a.update(kw)
    f = getattr(nv, name)
    head = (a["x"], a["dtype"], a["rows"], a["cols"], a["block"])
    tail = (ctypes.c_float(a["D"]), ctypes.c_float(a["static"]), a["S"], a["q"], a["sc"], a["ws"],
            a["wsb"], a["stream"])
    if name in ("nvfp4_quant_four_over_six", "nvfp4_quant_scalesweep_wmse"):
        return f(*head, a["w"], *tail)
    return f(*head, *tail)


QUANTS = ["nvfp4_quant_absmax", "nvfp4_quant_four_over_six", "nvfp4_quant_scalesweep_mse",
          "nvfp4_quant_scalesweep_wmse"]


@pytest.mark.parametrize("name", QUANTS)
@fake_pointers
def test_validation_errors(nv, name):
    st = dict(static=1.0)                 # static scale: no workspace needed
    assert call(nv, name, S=None, **st) == -1
    assert call(nv, name, x=None, **st) == -1
    assert call(nv, name, q=None, **st) == -1
    assert call(nv, name, sc=None, **st) == -1
    assert call(nv, name, dtype=2, **st) == -4
    assert call(nv, name, block=24, **st) == -3
    assert call(nv, name, block=8, **st) == -3
    assert call(nv, name, cols=40, **st) == -2
    assert call(nv, name, rows=-1, **st) == -2
    assert call(nv, name, D=0.0, **st) == -5
    assert call(nv, name, D=449.0, **st) == -5
    assert call(nv, name, D=float("nan"), **st) == -5
    assert call(nv, name, static=-1.0) == -5
    assert call(nv, name, static=float("inf")) == -5
    assert call(nv, name, static=float("nan")) == -5
    assert call(nv, name) == -6                            # dynamic scale without workspace
    assert call(nv, name, ws=FAKE, wsb=8) == -6            # workspace too small
    assert call(nv, name, ws=P(0x100004), wsb=nv.nvfp4_workspace_bytes()) == -7  # misaligned
    assert call(nv, name, x=P(0x100004), **st) == -7       # misaligned x
    assert call(nv, name, q=P(0x100004), **st) == -7       # misaligned q
    if name == "nvfp4_quant_scalesweep_wmse":
        assert call(nv, name, w=None, **st) == -1
    if name in ("nvfp4_quant_four_over_six", "nvfp4_quant_scalesweep_wmse"):
        assert call(nv, name, w=P(0x100004), **st) == -7


@fake_pointers
def test_dequant_validation(nv):
    f = nv.nvfp4_dequant
    assert f(FAKE8, FAKE, None, 4, 64, 16, 0, FAKE, None) == -1
    assert f(FAKE8, FAKE, FAKE, 4, 64, 16, 1, FAKE, None) == -4
    assert f(FAKE8, FAKE, FAKE, 4, 64, 12, 0, FAKE, None) == -3
    assert f(FAKE8, FAKE, FAKE, 4, 60, 16, 0, FAKE, None) == -2
    assert f(None, FAKE, FAKE, 4, 64, 16, 0, FAKE, None) == -1
    assert f(P(0x100004), FAKE, FAKE, 4, 64, 16, 0, FAKE, None) == -7
    assert f(FAKE8, FAKE, FAKE, 0, 64, 16, 0, FAKE, None) == 0   # empty: nothing to do


def test_binding_rejects_host_tensors(nv):
    import torch
    with pytest.raises(ValueError):
        nv.quantize(torch.zeros(4, 64, dtype=torch.bfloat16), "scalesweep_mse")


def test_no_oracle_in_the_product_path():
    """The product package neither imports nor links the oracle."""
    pkg = ROOT / "paper_2606_07618_amd"
    for f in list(pkg.rglob("*.py")) + list(pkg.rglob("*.hip")) + list(pkg.rglob("*.cpp")):
        text = f.read_text()
        assert "oracle" not in text.lower().replace("# the checker", ""), f


@fake_pointers
def test_batched_validation(nv):
    T = nv.nvfp4.NVFP4Tensor
    arr = (T * 2)(T(0x100000, 4, 64, 0x100000, 0x100000, 0x100000, 0x100000),
                  T(0x100000, 4, 64, 0x100000, 0x100000, 0x100000, 0x100000))
    f = nv.nvfp4_quant_batched
    ws, wsb = FAKE, nv.nvfp4_batched_workspace_bytes(2)
    a = ctypes.cast(arr, ctypes.c_void_p)
    assert f(3, a, -1, 1, 16, ctypes.c_float(256.0), ws, wsb, None) == -5
    assert f(9, a, 2, 1, 16, ctypes.c_float(256.0), ws, wsb, None) == -5
    assert f(3, None, 2, 1, 16, ctypes.c_float(256.0), ws, wsb, None) == -1
    assert f(3, a, 2, 1, 16, ctypes.c_float(256.0), ws, wsb - 16, None) == -6
    assert f(3, a, 2, 1, 24, ctypes.c_float(256.0), ws, wsb, None) == -3
    assert f(3, a, 2, 7, 16, ctypes.c_float(256.0), ws, wsb, None) == -4
    arr[1].cols = 60
    assert f(3, a, 2, 1, 16, ctypes.c_float(256.0), ws, wsb, None) == -2
    arr[1].cols = 64
    arr[1].col_weight = None
    assert f(3, a, 2, 1, 16, ctypes.c_float(256.0), ws, wsb, None) == -1
    assert f(3, a, 0, 1, 16, ctypes.c_float(256.0), None, 0, None) == 0


@fake_pointers
def test_window_validation(nv):
    f = nv.nvfp4_quant_scalesweep_window

    def call(mode=0, lo=-3, hi=7, w=None, S=FAKE, block=16, static=1.0, cols=64):
        return f(FAKE, 1, 4, cols, block, w, mode, lo, hi, ctypes.c_float(256.0),
                 ctypes.c_float(static), S, FAKE, FAKE, None, 0, None)

    assert call(mode=2) == -5
    assert call(mode=-1) == -5
    assert call(lo=2, hi=1) == -5
    assert call(lo=-127) == -5
    assert call(hi=127) == -5
    assert call(S=None) == -1
    assert call(block=24) == -3
    assert call(cols=40) == -2
    assert call(static=0.0) == -6              # dynamic scale without a workspace
    assert call(w=P(0x100004)) == -7           # misaligned weights
    assert call(mode=1, lo=99, hi=-99, static=-1.0) == -5


@fake_pointers
def test_analysis_call_validation(nv):
    opt = nv.nvfp4_block_optimum
    # (x, dtype, rows, cols, block, w, S, opt_loss, opt_scale, code, fp8_loss, stream)
    assert opt(FAKE, 1, 4, 64, 16, None, None, FAKE8, None, None, None, None) == -1
    assert opt(FAKE, 2, 4, 64, 16, None, FAKE, FAKE8, None, None, None, None) == -4
    assert opt(FAKE, 1, 4, 64, 24, None, FAKE, FAKE8, None, None, None, None) == -3
    assert opt(FAKE, 1, 4, 60, 16, None, FAKE, FAKE8, None, None, None, None) == -2
    assert opt(FAKE, 1, 4, 64, 16, None, FAKE, None, None, None, None, None) == -1
    assert opt(FAKE, 1, 4, 64, 16, None, FAKE, P(0x100004), None, None, None, None) == -7
    assert opt(FAKE, 1, 0, 64, 16, None, FAKE, None, None, None, None, None) == 0   # empty
    loss = nv.nvfp4_block_loss
    assert loss(FAKE, 1, 4, 64, 16, None, FAKE, None, FAKE8, None) == -1
    assert loss(FAKE, 1, 4, 64, 16, None, FAKE, FAKE, P(0x100004), None) == -7
    assert loss(FAKE, 1, 4, 64, 16, P(0x100002), FAKE, FAKE, FAKE8, None) == -7
    s = nv.nvfp4_sum_f64
    wsb = nv.nvfp4_sum_workspace_bytes()
    assert s(FAKE8, 10, None, FAKE8, wsb, None) == -1
    assert s(FAKE8, -1, FAKE8, FAKE8, wsb, None) == -2
    assert s(FAKE8, 10, FAKE8, FAKE8, wsb - 8, None) == -6
    assert s(P(0x100004), 10, FAKE8, FAKE8, wsb, None) == -7


@fake_pointers
def test_online_validation(nv):
    f = nv.nvfp4_quant_online

    def call(method=2, dtype=1, rows=4, cols=64, block=16, imp=None, groups=1, grows=1,
             S=1.0, layout=0, q=FAKE, sc=FAKE, x=FAKE):
        return f(method, x, dtype, rows, cols, block, imp, groups, grows, ctypes.c_float(S),
                 layout, None, q, sc, None)

    assert call(method=4) == -5
    assert call(S=0.0) == -5                     # the online path needs a static scale
    assert call(S=float("inf")) == -5
    assert call(layout=2) == -5
    assert call(layout=1, block=32) == -5        # swizzled scales are for block 16
    assert call(method=3) == -1                  # WMSE needs importance
    assert call(method=3, imp=FAKE, groups=0) == -5
    assert call(method=3, imp=FAKE, grows=0) == -5
    assert call(method=3, imp=P(0x100004)) == -7
    assert call(dtype=5) == -4
    assert call(cols=40) == -2
    assert call(q=None) == -1
    assert call(x=P(0x100004)) == -7
    assert nv.nvfp4_scales_bytes(130, 64, 16, 1) == 256 * 4
    assert nv.nvfp4_scales_bytes(130, 64, 16, 0) == 130 * 4
    assert nv.nvfp4_scales_bytes(4, 64, 32, 1) == -5
    assert nv.nvfp4_scales_bytes(4, 60, 16, 0) == -2


@fake_pointers
def test_channel_norms_validation(nv):
    f = nv.nvfp4_channel_sq_norms
    wsb = nv.nvfp4_channel_sq_norms_workspace_bytes(512, 64, 8, 2)
    assert wsb == 2 * 4 * 64 * 8
    assert nv.nvfp4_channel_sq_norms_workspace_bytes(512, 64, 3, 2) == -5
    assert nv.nvfp4_channel_sq_norms_workspace_bytes(512, 64, 130, 2) == -5   # > 64 groups
    assert f(FAKE, 3, 512, 64, 1, 8, 2, 1, FAKE, FAKE8, wsb, None) == -4
    assert f(FAKE, 1, 512, 64, 0, 8, 2, 1, FAKE, FAKE8, wsb, None) == -5
    assert f(FAKE, 1, 512, 64, 1, 8, 2, 0, FAKE, FAKE8, wsb, None) == -5
    assert f(FAKE, 1, 512, 64, 1, 8, 2, 1, None, FAKE8, wsb, None) == -1
    assert f(FAKE, 1, 512, 64, 1, 8, 2, 1, FAKE, FAKE8, wsb - 8, None) == -6
    assert f(FAKE, 1, 512, 64, 1, 8, 2, 1, FAKE, P(0x100004), wsb, None) == -7


@fake_pointers
def test_ldlq_validation(nv):
    f = nv.nvfp4_ldlq
    wsb = nv.nvfp4_ldlq_workspace_bytes(8, 64)
    assert wsb >= 8 * (64 * 64 + 2 * 8 * 64)

    def call(dtype=1, rows=8, cols=64, block=16, H=FAKE8, sc=FAKE, S=FAKE, damp=0.01, q=FAKE,
             st=FAKE, ws=P(0x200000), wsb=wsb):
        return f(FAKE, dtype, rows, cols, block, H, sc, S, ctypes.c_double(damp), q, st, ws, wsb,
                 None)

    assert call(dtype=3) == -4
    assert call(block=24) == -3
    assert call(cols=48) == -2                   # columns in tiles of 64
    assert call(damp=-1.0) == -5
    assert call(damp=float("nan")) == -5
    assert call(st=None) == -1
    assert call(S=None) == -1
    assert call(H=None) == -1
    assert call(H=P(0x100004)) == -7
    assert call(wsb=wsb - 1) == -6
    assert call(ws=P(0x200010)) == -7


@fake_pointers
def test_swiglu_validation(nv):
    f = nv.nvfp4_quant_online_swiglu

    def call(method=2, rows=4, cols=64, up=FAKE, S=1.0, layout=0, gate=FAKE, imp=None):
        return f(method, gate, up, rows, cols, imp, 1, 1, ctypes.c_float(S), layout, None, FAKE,
                 FAKE, None)

    assert call(up=None) == -1
    assert call(up=P(0x100004)) == -7
    assert call(gate=P(0x100004)) == -7
    assert call(method=3) == -1                  # WMSE needs importance
    assert call(S=0.0) == -5
    assert call(cols=40) == -2
    assert call(layout=3) == -5
    assert call(rows=0, up=None) == 0             # empty: nothing to read
    p = nv.nvfp4_swiglu
    assert p(FAKE, FAKE, 4, 40, FAKE, None) == -2
    assert p(FAKE, None, 4, 64, FAKE, None) == -1
    assert p(FAKE, FAKE, 4, 64, P(0x100004), None) == -7
    assert p(FAKE, FAKE, 0, 64, FAKE, None) == 0
