"""NVFP4 ScaleSweep oracle -- TEST INFRASTRUCTURE ONLY.

ctypes binding of ``nvfp4_oracle.c``: the plain single-threaded CPU reference for the
ScaleSweep hot path (arXiv 2606.07618), written from the paper.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import this
package; the product library never loads it.

Inputs are numpy arrays on the host: ``float32`` for binary32 tensors and ``uint16`` (raw
bit patterns) for bfloat16 tensors.  Every function returns numpy arrays / Python scalars.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

HERE = Path(__file__).resolve().parent
SRC = HERE / "nvfp4_oracle.c"
LIB = HERE / "liboracle.so"

ABSMAX, FOUR_OVER_SIX, SCALESWEEP_MSE, SCALESWEEP_WMSE = 0, 1, 2, 3
METHODS = {
    "absmax": ABSMAX,
    "four_over_six": FOUR_OVER_SIX,
    "scalesweep_mse": SCALESWEEP_MSE,
    "scalesweep_wmse": SCALESWEEP_WMSE,
}
STATUS = {0: "ok", -1: "null", -2: "shape", -3: "block", -4: "dtype", -5: "arg", -9: "nonfinite"}


class OracleError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"oracle {where}: status {code} ({STATUS.get(code, '?')})")
        self.code = code


def build(out: Path = LIB, extra_flags: tuple[str, ...] = ()) -> Path:
    """Compile the oracle with gcc: no fused multiply-add, no fast-math."""
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
           *extra_flags, "-o", str(out), str(SRC), "-lm"]
    subprocess.run(cmd, check=True)
    return out


_lib = None


def _load(path: Path | None = None):
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(str(path)))
    if _lib is None:
        alt = os.environ.get("NVFP4_ORACLE_LIB")   # a deliberately broken build (tests only)
        if alt:
            _lib = _bind(ctypes.CDLL(alt))
            return _lib
        if not LIB.exists() or LIB.stat().st_mtime < SRC.stat().st_mtime:
            build()
        _lib = _bind(ctypes.CDLL(str(LIB)))
    return _lib


def _bind(lib):
    P, I64, I, F, D = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_double
    sig = {
        "nvfp4_ref_eemm_value": (D, [I, I, I]),
        "nvfp4_ref_e2m1": (D, [I]),
        "nvfp4_ref_e4m3": (D, [I]),
        "nvfp4_ref_round_fp4": (I, [D, D]),
        "nvfp4_ref_floor_fp8": (I, [D, D]),
        "nvfp4_ref_nearest_fp8": (I, [D, D]),
        "nvfp4_ref_block_loss": (D, [P, P, I, D]),
        "nvfp4_ref_window_lower": (I, [I, I]),
        "nvfp4_ref_window_upper": (I, []),
        "nvfp4_ref_block_sweep": (I, [P, P, I, I, I, P, P, P, P, P, P]),
        "nvfp4_ref_block_choose": (I, [I, P, P, I]),
        "nvfp4_ref_window_tight": (I, [I, I, I, P, P]),
        "nvfp4_ref_window_codes": (I, [I, I, I, I, I, I, P, P]),
        "nvfp4_ref_quant_scalesweep_window": (I, [P, I, I64, I64, I, P, I, I, I, F, F, P, P, P]),
        "nvfp4_ref_swizzled_offset": (I64, [I64, I64, I64]),
        "nvfp4_ref_scales_bytes": (I64, [I64, I64, I, I]),
        "nvfp4_ref_quant_online": (I, [I, P, I, I64, I64, I, P, I64, I64, F, I, P, P, P]),
        "nvfp4_ref_channel_sq_norms": (I, [P, I, I64, I64, I64, I64, I64, I64, P]),
        "nvfp4_ref_swiglu_exp": (ctypes.c_float, [ctypes.c_float]),
        "nvfp4_ref_swiglu": (I, [P, P, I64, P]),
        "nvfp4_ref_ldlq_order": (I, [P, I64, P]),
        "nvfp4_ref_ldlq_factor": (I, [P, I64, D, P, P, P]),
        "nvfp4_ref_ldlq": (I, [P, I, I64, I64, I, P, P, F, D, P]),
        "nvfp4_ref_tensor_scale": (I, [P, I, I64, F, P]),
        "nvfp4_ref_quantize": (I, [I, P, I, I64, I64, I, F, F, P, P, P, P]),
        "nvfp4_ref_dequant": (I, [P, P, F, I64, I64, I, P]),
        "nvfp4_ref_continuous_opt": (D, [P, P, I, P]),
        "nvfp4_ref_fp8_quantized_opt": (I, [P, P, I, P]),
        "nvfp4_ref_metrics": (I, [P, I, P, I64, I64, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def _tensor(x):
    x = np.ascontiguousarray(x)
    if x.dtype == np.float32:
        return x, 0
    if x.dtype == np.uint16:
        return x, 1
    raise TypeError("oracle takes float32 or uint16 (bfloat16 bit patterns)")


# --- formats and rounding -------------------------------------------------------------

def eemm_value(e: int, m: int, code: int) -> float:
    return _load().nvfp4_ref_eemm_value(e, m, code)


def e2m1(k: int) -> float:
    return _load().nvfp4_ref_e2m1(k)


def e4m3(c: int) -> float:
    return _load().nvfp4_ref_e4m3(c)


def e2m1_table() -> np.ndarray:
    return np.array([e2m1(k) for k in range(8)])


def e4m3_table() -> np.ndarray:
    return np.array([e4m3(c) for c in range(127)])


def round_fp4(a: float, s: float) -> int:
    return _load().nvfp4_ref_round_fp4(float(a), float(s))


def floor_fp8(num: float, den: float) -> int:
    return _load().nvfp4_ref_floor_fp8(float(num), float(den))


def nearest_fp8(num: float, den: float) -> int:
    return _load().nvfp4_ref_nearest_fp8(float(num), float(den))


# --- block level ----------------------------------------------------------------------

def block_loss(y, w, s: float) -> float:
    y = _f32(y)
    w = _f32(w)
    return _load().nvfp4_ref_block_loss(_ptr(y), _ptr(w), y.size, float(s))


def window_lower(method: str | int, n: int) -> int:
    m = METHODS[method] if isinstance(method, str) else method
    return _load().nvfp4_ref_window_lower(m, n)


def window_upper() -> int:
    return _load().nvfp4_ref_window_upper()


def block_sweep(y, w=None, L: int = 3, U: int = 7) -> dict:
    """Full and windowed sweep of one block of normalized values."""
    y = _f32(y)
    w = _f32(w)
    outs = [ctypes.c_int() for _ in range(5)]
    J = np.zeros(127, dtype=np.float64)
    rc = _load().nvfp4_ref_block_sweep(_ptr(y), _ptr(w), y.size, L, U,
                                       *[ctypes.byref(o) for o in outs], _ptr(J))
    if rc:
        raise OracleError(rc, "block_sweep")
    c0, lo, hi, cw, cf = (o.value for o in outs)
    return {"c0": c0, "lo": lo, "hi": hi, "c_win": cw, "c_full": cf, "J": J}


def block_choose(method: str | int, y, w=None) -> int:
    m = METHODS[method] if isinstance(method, str) else method
    y = _f32(y)
    w = _f32(w)
    return _load().nvfp4_ref_block_choose(m, _ptr(y), _ptr(w), y.size)


WINDOW_MODES = {"offsets": 0, "tight": 1}


def window_tight(method: str | int, n: int, b: int) -> tuple[int, int]:
    """(lower, upper) offsets of the per-mantissa window for mantissa field b."""
    m = METHODS[method] if isinstance(method, str) else method
    lo, hi = ctypes.c_int(), ctypes.c_int()
    rc = _load().nvfp4_ref_window_tight(m, n, b, ctypes.byref(lo), ctypes.byref(hi))
    if rc:
        raise OracleError(rc, "window_tight")
    return lo.value, hi.value


def window_codes(method: str | int, n: int, mode: str, lo_off: int, hi_off: int,
                 c0: int) -> tuple[int, int]:
    """The code range [lo, hi] a block with base code c0 sweeps under a window variant."""
    m = METHODS[method] if isinstance(method, str) else method
    lo, hi = ctypes.c_int(), ctypes.c_int()
    rc = _load().nvfp4_ref_window_codes(m, n, WINDOW_MODES[mode], lo_off, hi_off, c0,
                                        ctypes.byref(lo), ctypes.byref(hi))
    if rc:
        raise OracleError(rc, "window_codes")
    return lo.value, hi.value


def quantize_window(x, block: int = 16, weight=None, mode: str = "offsets", lo: int = -3,
                    hi: int = 7, fp8_range: float = 256.0, static_scale: float = 0.0):
    """ScaleSweep with a window variant (MSE objective if weight is None, else WMSE).
    Returns (S, q, scales) like quantize()."""
    x, dt = _tensor(x)
    if x.ndim != 2:
        raise ValueError("x must be 2-D [rows, cols]")
    rows, cols = x.shape
    w = _f32(weight)
    q = np.zeros((rows, cols // 2), dtype=np.uint8)
    sc = np.zeros((rows, max(cols // block, 0)), dtype=np.uint8)
    S = ctypes.c_float()
    rc = _load().nvfp4_ref_quant_scalesweep_window(
        _ptr(x), dt, rows, cols, block, _ptr(w), WINDOW_MODES.get(mode, mode) if isinstance(mode, str) else mode,
        lo, hi, float(fp8_range), float(static_scale), ctypes.byref(S), _ptr(q), _ptr(sc))
    if rc:
        raise OracleError(rc, "quantize_window")
    return S.value, q, sc


def continuous_opt(y, w=None) -> tuple[float, float]:
    y = _f32(y)
    w = _f32(w)
    s = ctypes.c_double()
    val = _load().nvfp4_ref_continuous_opt(_ptr(y), _ptr(w), y.size, ctypes.byref(s))
    return val, s.value


def fp8_quantized_opt(y, w=None) -> tuple[int, float]:
    y = _f32(y)
    w = _f32(w)
    loss = ctypes.c_double()
    c = _load().nvfp4_ref_fp8_quantized_opt(_ptr(y), _ptr(w), y.size, ctypes.byref(loss))
    return c, loss.value


# --- tensor level ---------------------------------------------------------------------

def tensor_scale(x, fp8_range: float) -> float:
    x, dt = _tensor(x)
    S = ctypes.c_float()
    rc = _load().nvfp4_ref_tensor_scale(_ptr(x), dt, x.size, float(fp8_range), ctypes.byref(S))
    if rc:
        raise OracleError(rc, "tensor_scale")
    return S.value


def quantize(method: str | int, x, block: int = 16, fp8_range: float = 256.0,
             static_scale: float = 0.0, weight=None):
    """Returns (S, q[rows, cols/2] uint8, scales[rows, cols/block] uint8)."""
    m = METHODS[method] if isinstance(method, str) else method
    x, dt = _tensor(x)
    if x.ndim != 2:
        raise ValueError("x must be 2-D [rows, cols]")
    rows, cols = x.shape
    w = _f32(weight)
    q = np.zeros((rows, cols // 2), dtype=np.uint8)
    sc = np.zeros((rows, max(cols // block, 0)), dtype=np.uint8)
    S = ctypes.c_float()
    rc = _load().nvfp4_ref_quantize(m, _ptr(x), dt, rows, cols, block, float(fp8_range),
                                    float(static_scale), _ptr(w), ctypes.byref(S), _ptr(q),
                                    _ptr(sc))
    if rc:
        raise OracleError(rc, "quantize")
    return S.value, q, sc


def quantize_status(method, x, block=16, fp8_range=256.0, static_scale=0.0, weight=None,
                    rows=None, cols=None) -> int:
    """Raw status of a quantize call (argument-validation tests)."""
    m = METHODS[method] if isinstance(method, str) else method
    x, dt = _tensor(x)
    r = x.shape[0] if rows is None else rows
    c = x.shape[1] if cols is None else cols
    w = _f32(weight)
    q = np.zeros(max(x.size // 2, 1), dtype=np.uint8)
    sc = np.zeros(max(x.size, 1), dtype=np.uint8)
    S = ctypes.c_float()
    return _load().nvfp4_ref_quantize(m, _ptr(x), dt, r, c, block, float(fp8_range),
                                      float(static_scale), _ptr(w), ctypes.byref(S), _ptr(q),
                                      _ptr(sc))


def dequant(q, scales, S: float, block: int = 16) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.uint8)
    scales = np.ascontiguousarray(scales, dtype=np.uint8)
    rows, cols = q.shape[0], q.shape[1] * 2
    out = np.zeros((rows, cols), dtype=np.float32)
    rc = _load().nvfp4_ref_dequant(_ptr(q), _ptr(scales), float(S), rows, cols, block, _ptr(out))
    if rc:
        raise OracleError(rc, "dequant")
    return out


def metrics(x, xhat, weight=None) -> dict:
    x, dt = _tensor(x)
    xhat = _f32(xhat)
    w = _f32(weight)
    out = np.zeros(4, dtype=np.float64)
    rc = _load().nvfp4_ref_metrics(_ptr(x), dt, _ptr(xhat), x.shape[0], x.shape[1], _ptr(w),
                                   _ptr(out))
    if rc:
        raise OracleError(rc, "metrics")
    return dict(zip(("mse", "nmse", "wmse", "nwmse"), out.tolist()))


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact bfloat16 -> binary32 of raw bit patterns (a widening, no arithmetic)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normalize(x, S: float) -> np.ndarray:
    """y = RN32(x / S), as the oracle forms it (numpy float32 division is IEEE)."""
    xf = bf16_to_f32(x) if np.asarray(x).dtype == np.uint16 else np.asarray(x, np.float32)
    return (xf / np.float32(S)).astype(np.float32)


# --- online quantization ------------------------------------------------------------------

SCALE_LAYOUTS = {"row_major": 0, "swizzled": 1}


def swizzled_offset(m: int, k: int, k16: int) -> int:
    return _load().nvfp4_ref_swizzled_offset(m, k, k16)


def scales_bytes(rows: int, cols: int, block: int, layout: str) -> int:
    return _load().nvfp4_ref_scales_bytes(rows, cols, block, SCALE_LAYOUTS[layout])


def quantize_online(method: str | int, x, static_scale: float, block: int = 16,
                    importance=None, imp_groups: int = 1, imp_group_rows: int = 1,
                    layout: str = "row_major"):
    """Static-scale quantization with per-group importance vectors [imp_groups, cols].
    Returns (q [rows, cols/2], scales (1-D for the swizzled layout))."""
    m = METHODS[method] if isinstance(method, str) else method
    x, dt = _tensor(x)
    rows, cols = x.shape
    imp = _f32(importance)
    nbytes = scales_bytes(rows, cols, block, layout)
    if nbytes < 0:
        raise OracleError(-5, "quantize_online")
    q = np.zeros((rows, cols // 2), dtype=np.uint8)
    sc = np.zeros(max(nbytes, 1), dtype=np.uint8)[:nbytes]
    rc = _load().nvfp4_ref_quant_online(m, _ptr(x), dt, rows, cols, block, _ptr(imp),
                                        imp_groups, imp_group_rows, float(static_scale),
                                        SCALE_LAYOUTS[layout], None, _ptr(q), _ptr(sc))
    if rc:
        raise OracleError(rc, "quantize_online")
    if layout == "row_major":
        sc = sc.reshape(rows, cols // block)
    return q, sc


def swiglu_exp(x: float) -> float:
    return _load().nvfp4_ref_swiglu_exp(float(x))


def swiglu(gate: np.ndarray, up: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns h = bf16(silu(gate) * up) of two bfloat16 (uint16 bit pattern)
    arrays of one shape."""
    g = np.ascontiguousarray(gate, dtype=np.uint16)
    u = np.ascontiguousarray(up, dtype=np.uint16)
    if g.shape != u.shape:
        raise ValueError("gate and up must have one shape")
    h = np.zeros(g.shape, dtype=np.uint16)
    rc = _load().nvfp4_ref_swiglu(_ptr(g), _ptr(u), g.size, _ptr(h))
    if rc:
        raise OracleError(rc, "swiglu")
    return h


def channel_sq_norms(x, group_rows: int = 1, groups: int = 1, group_div: int = 1,
                     rep_out: int = 1) -> np.ndarray:
    """[groups / group_div * rep_out, cols] binary32 squared channel norms (see the C doc)."""
    x, dt = _tensor(x)
    rows, cols = x.shape
    out = np.zeros((groups // group_div * rep_out, cols), dtype=np.float32)
    rc = _load().nvfp4_ref_channel_sq_norms(_ptr(x), dt, rows, cols, group_rows, groups,
                                            group_div, rep_out, _ptr(out))
    if rc:
        raise OracleError(rc, "channel_sq_norms")
    return out


# --- GPTQ / LDLQ with fixed block scales -----------------------------------------------------

def ldlq_order(H) -> np.ndarray:
    H = np.ascontiguousarray(H, dtype=np.float64)
    perm = np.zeros(H.shape[0], dtype=np.int64)
    rc = _load().nvfp4_ref_ldlq_order(_ptr(H), H.shape[0], _ptr(perm))
    if rc:
        raise OracleError(rc, "ldlq_order")
    return perm


def ldlq_factor(H, damp: float = 0.01, perm=None):
    """(U strictly upper [n, n], D [n]) of the damped, reordered Hessian."""
    H = np.ascontiguousarray(H, dtype=np.float64)
    n = H.shape[0]
    perm = ldlq_order(H) if perm is None else np.ascontiguousarray(perm, dtype=np.int64)
    U = np.zeros((n, n))
    D = np.zeros(n)
    rc = _load().nvfp4_ref_ldlq_factor(_ptr(H), n, float(damp), _ptr(perm), _ptr(U), _ptr(D))
    if rc:
        raise OracleError(rc, "ldlq_factor")
    return U, D


def ldlq(w, H, scales, S: float, block: int = 16, damp: float = 0.01) -> np.ndarray:
    """GPTQ (LDLQ form) nibbles [rows, n/2] with the given fixed block scales."""
    w, dt = _tensor(w)
    rows, n = w.shape
    H = np.ascontiguousarray(H, dtype=np.float64)
    sc = np.ascontiguousarray(scales, dtype=np.uint8)
    q = np.zeros((rows, n // 2), dtype=np.uint8)
    rc = _load().nvfp4_ref_ldlq(_ptr(w), dt, rows, n, block, _ptr(H), _ptr(sc), float(S),
                                float(damp), _ptr(q))
    if rc:
        raise OracleError(rc, "ldlq")
    return q
