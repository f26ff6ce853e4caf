"""ctypes binding of libnvfp4ss.so: the C entry points under their own names, plus
``quantize`` / ``dequant`` helpers that allocate outputs with torch on the input's device and
pass raw device pointers and the current HIP stream."""
from __future__ import annotations

import ctypes
from pathlib import Path

import torch

LIB_PATH = Path(__file__).resolve().parent / "libnvfp4ss.so"

F32, BF16 = 0, 1
STATUS = {
    0: "ok", -1: "null pointer", -2: "bad shape", -3: "bad block", -4: "bad dtype",
    -5: "bad argument", -6: "workspace", -7: "alignment", -8: "HIP launch failed",
    -10: "beyond the no-allocation call's fixed scratch",
}
DEFAULT_RANGE = {"absmax": 448.0, "four_over_six": 256.0, "scalesweep_mse": 256.0,
                 "scalesweep_wmse": 256.0}


class NVFP4Error(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: status {status} ({STATUS.get(status, '?')})")
        self.status = status


def _load():
    if not LIB_PATH.exists():
        raise ImportError(f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; "
                          "g.build()'` (hipcc for gfx950)")
    L = ctypes.CDLL(str(LIB_PATH))
    P, I64, I, F, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    quant = [P, I, I64, I64, I, F, F, P, P, P, P, SZ, P]
    quant_w = [P, I, I64, I64, I, P, F, F, P, P, P, P, SZ, P]
    sigs = {
        "nvfp4_workspace_bytes": (SZ, []),
        "nvfp4_batched_workspace_bytes": (SZ, [I]),
        "nvfp4_quant_batched": (I, [I, P, I, I, I, F, P, SZ, P]),
        "nvfp4_quant_batched_noalloc": (I, [I, P, I, I, I, F, P]),
        "nvfp4_status_string": (ctypes.c_char_p, [I]),
        "nvfp4_quant_absmax": (I, quant),
        "nvfp4_quant_four_over_six": (I, quant_w),
        "nvfp4_quant_scalesweep_mse": (I, quant),
        "nvfp4_quant_scalesweep_wmse": (I, quant_w),
        "nvfp4_quant_scalesweep_window": (I, [P, I, I64, I64, I, P, I, I, I, F, F, P, P, P, P, SZ, P]),
        "nvfp4_dequant": (I, [P, P, P, I64, I64, I, I, P, P]),
        "nvfp4_block_optimum": (I, [P, I, I64, I64, I, P, P, P, P, P, P, P]),
        "nvfp4_block_loss": (I, [P, I, I64, I64, I, P, P, P, P, P]),
        "nvfp4_sum_workspace_bytes": (SZ, []),
        "nvfp4_sum_f64": (I, [P, I64, P, P, SZ, P]),
        "nvfp4_scales_bytes": (I64, [I64, I64, I, I]),
        "nvfp4_quant_online": (I, [I, P, I, I64, I64, I, P, I64, I64, F, I, P, P, P, P]),
        "nvfp4_quant_online_swiglu": (I, [I, P, P, I64, I64, P, I64, I64, F, I, P, P, P, P]),
        "nvfp4_swiglu": (I, [P, P, I64, I64, P, P]),
        "nvfp4_channel_sq_norms_workspace_bytes": (I64, [I64, I64, I64, I64]),
        "nvfp4_channel_sq_norms": (I, [P, I, I64, I64, I64, I64, I64, I64, P, P, SZ, P]),
        "nvfp4_ldlq_workspace_bytes": (SZ, [I64, I64]),
        "nvfp4_ldlq": (I, [P, I, I64, I64, I, P, P, P, ctypes.c_double, P, P, P, SZ, P]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    return L


class NVFP4Tensor(ctypes.Structure):
    """The C struct nvfp4_tensor."""
    _fields_ = [("x", ctypes.c_void_p), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("col_weight", ctypes.c_void_p), ("tensor_scale", ctypes.c_void_p),
                ("q", ctypes.c_void_p), ("scales", ctypes.c_void_p)]


lib = _load()

# The C entry points, under the header's names.
nvfp4_workspace_bytes = lib.nvfp4_workspace_bytes
nvfp4_status_string = lib.nvfp4_status_string
nvfp4_quant_absmax = lib.nvfp4_quant_absmax
nvfp4_quant_four_over_six = lib.nvfp4_quant_four_over_six
nvfp4_quant_scalesweep_mse = lib.nvfp4_quant_scalesweep_mse
nvfp4_quant_scalesweep_wmse = lib.nvfp4_quant_scalesweep_wmse
nvfp4_quant_scalesweep_window = lib.nvfp4_quant_scalesweep_window
nvfp4_dequant = lib.nvfp4_dequant
nvfp4_block_optimum = lib.nvfp4_block_optimum
nvfp4_block_loss = lib.nvfp4_block_loss
nvfp4_sum_workspace_bytes = lib.nvfp4_sum_workspace_bytes
nvfp4_sum_f64 = lib.nvfp4_sum_f64
nvfp4_scales_bytes = lib.nvfp4_scales_bytes
nvfp4_quant_online = lib.nvfp4_quant_online
nvfp4_quant_online_swiglu = lib.nvfp4_quant_online_swiglu
nvfp4_swiglu = lib.nvfp4_swiglu
nvfp4_channel_sq_norms_workspace_bytes = lib.nvfp4_channel_sq_norms_workspace_bytes
nvfp4_channel_sq_norms = lib.nvfp4_channel_sq_norms
nvfp4_ldlq_workspace_bytes = lib.nvfp4_ldlq_workspace_bytes
nvfp4_ldlq = lib.nvfp4_ldlq
nvfp4_batched_workspace_bytes = lib.nvfp4_batched_workspace_bytes
nvfp4_quant_batched = lib.nvfp4_quant_batched
nvfp4_quant_batched_noalloc = lib.nvfp4_quant_batched_noalloc
NOALLOC_MAX_TENSORS = 32
METHOD_IDS = {"absmax": 0, "four_over_six": 1, "scalesweep_mse": 2, "scalesweep_wmse": 3}


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def workspace(device) -> torch.Tensor:
    """A workspace for the dynamic-scale path (no initialization needed; reusable by calls
    that are ordered on one stream)."""
    return torch.empty(nvfp4_workspace_bytes() // 4, dtype=torch.int32, device=device)


def quantize(x: torch.Tensor, method: str = "scalesweep_wmse", block: int = 16,
             weight: torch.Tensor | None = None, fp8_range: float | None = None,
             static_scale: float = 0.0, ws: torch.Tensor | None = None, out=None):
    """Quantize a 2-D device tensor [rows, cols] (bfloat16 or float32) to NVFP4.

    Returns (q [rows, cols/2] uint8, scales [rows, cols/block] uint8, S [1] float32), all on
    x's device; the work is enqueued on the current stream.  ``out`` may pass preallocated
    (q, scales, S) tensors."""
    if x.dim() != 2:
        raise ValueError("x must be 2-D [rows, cols]")
    if not x.is_cuda:
        raise ValueError("x must be a device tensor (the library runs on the GPU only)")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    if x.dtype == torch.bfloat16:
        dt = BF16
    elif x.dtype == torch.float32:
        dt = F32
    else:
        raise TypeError("x must be bfloat16 or float32")
    rows, cols = x.shape
    D = DEFAULT_RANGE[method] if fp8_range is None else float(fp8_range)
    if out is None:
        q = torch.empty((rows, cols // 2), dtype=torch.uint8, device=x.device)
        sc = torch.empty((rows, cols // block if block else 0), dtype=torch.uint8, device=x.device)
        S = torch.empty(1, dtype=torch.float32, device=x.device)
    else:
        q, sc, S = out
    if static_scale == 0.0 and ws is None:
        ws = workspace(x.device)
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    common = (_ptr(x), dt, rows, cols, block)
    tail = (ctypes.c_float(D), ctypes.c_float(static_scale), _ptr(S), _ptr(q), _ptr(sc),
            _ptr(ws), wsb, _stream(x.device))
    if weight is not None:
        if not (weight.is_cuda and weight.dtype == torch.float32 and weight.is_contiguous()
                and weight.numel() == cols):
            raise ValueError("weight must be a contiguous float32 device tensor of length cols")
    if method == "absmax":
        rc = nvfp4_quant_absmax(*common, *tail)
    elif method == "four_over_six":
        rc = nvfp4_quant_four_over_six(*common, _ptr(weight), *tail)
    elif method == "scalesweep_mse":
        rc = nvfp4_quant_scalesweep_mse(*common, *tail)
    elif method == "scalesweep_wmse":
        rc = nvfp4_quant_scalesweep_wmse(*common, _ptr(weight), *tail)
    else:
        raise ValueError(f"unknown method {method!r}")
    if rc != 0:
        raise NVFP4Error(rc, f"nvfp4_quant_{method}")
    return q, sc, S


WINDOW_MODES = {"offsets": 0, "tight": 1}


def _check_input(x):
    if x.dim() != 2:
        raise ValueError("x must be 2-D [rows, cols]")
    if not x.is_cuda:
        raise ValueError("x must be a device tensor (the library runs on the GPU only)")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    if x.dtype == torch.bfloat16:
        return BF16
    if x.dtype == torch.float32:
        return F32
    raise TypeError("x must be bfloat16 or float32")


def quantize_window(x: torch.Tensor, block: int = 16, weight: torch.Tensor | None = None,
                    mode: str = "offsets", lo: int = -3, hi: int = 7,
                    fp8_range: float = 256.0, static_scale: float = 0.0,
                    ws: torch.Tensor | None = None, out=None):
    """ScaleSweep over a window variant: ``mode`` "offsets" sweeps codes c0+lo .. c0+hi,
    "tight" the per-mantissa windows; MSE objective if ``weight`` is None, else WMSE.
    Returns (q, scales, S) like quantize()."""
    dt = _check_input(x)
    rows, cols = x.shape
    if out is None:
        q = torch.empty((rows, cols // 2), dtype=torch.uint8, device=x.device)
        sc = torch.empty((rows, cols // block if block else 0), dtype=torch.uint8, device=x.device)
        S = torch.empty(1, dtype=torch.float32, device=x.device)
    else:
        q, sc, S = out
    if static_scale == 0.0 and ws is None:
        ws = workspace(x.device)
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    if weight is not None and not (weight.is_cuda and weight.dtype == torch.float32
                                   and weight.is_contiguous() and weight.numel() == cols):
        raise ValueError("weight must be a contiguous float32 device tensor of length cols")
    rc = nvfp4_quant_scalesweep_window(
        _ptr(x), dt, rows, cols, block, _ptr(weight), WINDOW_MODES[mode], int(lo), int(hi),
        ctypes.c_float(fp8_range), ctypes.c_float(static_scale), _ptr(S), _ptr(q), _ptr(sc),
        _ptr(ws), wsb, _stream(x.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_quant_scalesweep_window")
    return q, sc, S


def quantize_batched(xs, method: str = "scalesweep_wmse", block: int = 16, weights=None,
                     fp8_range: float | None = None, ws: torch.Tensor | None = None,
                     outs=None, noalloc: bool = False):
    """Quantize a list of 2-D device tensors (one dtype) with one method and a dynamic global
    scale each, in one batched call.  Returns a list of (q, scales, S).  ``noalloc`` calls
    nvfp4_quant_batched_noalloc (the library's fixed scratch, at most NOALLOC_MAX_TENSORS
    tensors) instead of passing a workspace."""
    if not xs:
        return []
    dev = xs[0].device
    dt = BF16 if xs[0].dtype == torch.bfloat16 else F32
    D = DEFAULT_RANGE[method] if fp8_range is None else float(fp8_range)
    weights = weights or [None] * len(xs)
    if outs is None:
        outs = [(torch.empty((x.shape[0], x.shape[1] // 2), dtype=torch.uint8, device=dev),
                 torch.empty((x.shape[0], x.shape[1] // block), dtype=torch.uint8, device=dev),
                 torch.empty(1, dtype=torch.float32, device=dev)) for x in xs]
    arr = (NVFP4Tensor * len(xs))()
    for k, (x, w, (q, sc, S)) in enumerate(zip(xs, weights, outs)):
        if x.dim() != 2 or not x.is_cuda or not x.is_contiguous() or x.dtype != xs[0].dtype:
            raise ValueError("every tensor must be a contiguous 2-D device tensor of one dtype")
        arr[k] = NVFP4Tensor(x.data_ptr(), x.shape[0], x.shape[1],
                             None if w is None else w.data_ptr(), S.data_ptr(), q.data_ptr(),
                             sc.data_ptr())
    if noalloc:
        rc = nvfp4_quant_batched_noalloc(METHOD_IDS[method], ctypes.cast(arr, ctypes.c_void_p),
                                         len(xs), dt, block, ctypes.c_float(D), _stream(dev))
        if rc != 0:
            raise NVFP4Error(rc, "nvfp4_quant_batched_noalloc")
        return outs
    nbytes = nvfp4_batched_workspace_bytes(len(xs))
    if ws is None or ws.numel() * ws.element_size() < nbytes:
        ws = torch.empty(nbytes // 4, dtype=torch.int32, device=dev)
    rc = nvfp4_quant_batched(METHOD_IDS[method], ctypes.cast(arr, ctypes.c_void_p), len(xs), dt,
                             block, ctypes.c_float(D), _ptr(ws), nbytes, _stream(dev))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_quant_batched")
    return outs


def dequant(q: torch.Tensor, scales: torch.Tensor, S: torch.Tensor, block: int = 16,
            out: torch.Tensor | None = None) -> torch.Tensor:
    """x_hat [rows, cols] float32 from (q, scales, S)."""
    rows, cols = q.shape[0], q.shape[1] * 2
    if out is None:
        out = torch.empty((rows, cols), dtype=torch.float32, device=q.device)
    rc = nvfp4_dequant(_ptr(q), _ptr(scales), _ptr(S), rows, cols, block, F32, _ptr(out),
                       _stream(q.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_dequant")
    return out


# ---- reference scales and gap reports ------------------------------------------------------

def _check_scale(S, device):
    if not (S.is_cuda and S.dtype == torch.float32 and S.numel() >= 1 and S.device == device):
        raise ValueError("S must be a float32 device tensor on x's device")


def block_optimum(x: torch.Tensor, S: torch.Tensor, block: int = 16,
                  weight: torch.Tensor | None = None):
    """Per-block optimal real scale and FP8-quantized optimum on y = RN32(x / S).
    Returns (opt_loss f64, opt_scale f64, fp8_code u8, fp8_loss f64), each [rows, cols/block]."""
    dt = _check_input(x)
    _check_scale(S, x.device)
    rows, cols = x.shape
    shape = (rows, cols // block)
    out = (torch.empty(shape, dtype=torch.float64, device=x.device),
           torch.empty(shape, dtype=torch.float64, device=x.device),
           torch.empty(shape, dtype=torch.uint8, device=x.device),
           torch.empty(shape, dtype=torch.float64, device=x.device))
    rc = nvfp4_block_optimum(_ptr(x), dt, rows, cols, block, _ptr(weight), _ptr(S),
                             *map(_ptr, out), _stream(x.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_block_optimum")
    return out


def block_loss(x: torch.Tensor, S: torch.Tensor, scales: torch.Tensor, block: int = 16,
               weight: torch.Tensor | None = None) -> torch.Tensor:
    """Exact binary64 loss of every block of y = RN32(x / S) at its E4M3 code in ``scales``."""
    dt = _check_input(x)
    _check_scale(S, x.device)
    rows, cols = x.shape
    if not (scales.is_cuda and scales.dtype == torch.uint8 and scales.is_contiguous()
            and scales.numel() == rows * (cols // block)):
        raise ValueError("scales must be a contiguous uint8 device tensor [rows, cols/block]")
    loss = torch.empty((rows, cols // block), dtype=torch.float64, device=x.device)
    rc = nvfp4_block_loss(_ptr(x), dt, rows, cols, block, _ptr(weight), _ptr(S), _ptr(scales),
                          _ptr(loss), _stream(x.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_block_loss")
    return loss


def sum_f64(v: torch.Tensor) -> torch.Tensor:
    """Deterministic binary64 sum of a contiguous float64 device tensor, as a [1] tensor."""
    if not (v.is_cuda and v.dtype == torch.float64 and v.is_contiguous()):
        raise ValueError("v must be a contiguous float64 device tensor")
    out = torch.empty(1, dtype=torch.float64, device=v.device)
    ws = torch.empty(nvfp4_sum_workspace_bytes() // 8, dtype=torch.float64, device=v.device)
    rc = nvfp4_sum_f64(_ptr(v), v.numel(), _ptr(out), _ptr(ws), nvfp4_sum_workspace_bytes(),
                       _stream(v.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_sum_f64")
    return out


def gap_report(x: torch.Tensor, block: int = 16, weight: torch.Tensor | None = None,
               methods=("absmax", "four_over_six", "scalesweep_mse", "scalesweep_wmse")) -> dict:
    """Relative gap of each block-scale rule to the optimal real block scale, as in the
    paper's Figures 1 and 4: sum of S^2 L over the blocks of the rule, over the same sum for
    the optimum, minus one.  The objective is WMSE if ``weight`` is given, else MSE; each
    method runs with its own global scale (D = 448 for AbsMax, 256 otherwise), the optimum and
    its FP8-quantized version with D = 256.  Also reports the exhaustive FP8 sweep."""
    def total(loss, S):
        return float(sum_f64(loss.reshape(-1)).item()) * float(S.item()) ** 2

    q, sc, S = quantize_window(x, block, weight, "offsets", -126, 126)
    opt_loss, _, fp8_code, fp8_loss = block_optimum(x, S, block, weight)
    j_opt = total(opt_loss, S)
    report = {"optimum": 0.0}
    if j_opt > 0:
        report["fp8_quantized_optimum"] = total(fp8_loss, S) / j_opt - 1.0
        report["exhaustive_fp8_sweep"] = total(block_loss(x, S, sc, block, weight), S) / j_opt - 1.0
        for m in methods:
            w_m = weight if m in ("four_over_six", "scalesweep_wmse") else None
            if m == "scalesweep_wmse" and weight is None:
                continue
            _, sc_m, S_m = quantize(x, m, block, weight=w_m)
            report[m] = total(block_loss(x, S_m, sc_m, block, weight), S_m) / j_opt - 1.0
    return report


# ---- online quantization (static global scale) ----------------------------------------------

SCALE_LAYOUTS = {"row_major": 0, "swizzled": 1}


def quantize_online(x: torch.Tensor, method: str, static_scale: float, block: int = 16,
                    importance: torch.Tensor | None = None, imp_groups: int = 1,
                    imp_group_rows: int = 1, layout: str = "row_major", out=None):
    """Quantize with a calibrated static global scale; importance [imp_groups, cols] selects a
    vector per row group (see nvfp4_quant_online).  Returns (q, scales): scales is
    [rows, cols/block] row-major or the flat swizzled buffer."""
    dt = _check_input(x)
    rows, cols = x.shape
    nbytes = nvfp4_scales_bytes(rows, cols, block, SCALE_LAYOUTS[layout])
    if nbytes < 0:
        raise NVFP4Error(int(nbytes), "nvfp4_scales_bytes")
    if importance is not None and not (importance.is_cuda and importance.dtype == torch.float32
                                       and importance.is_contiguous()
                                       and importance.numel() == imp_groups * cols):
        raise ValueError("importance must be a contiguous float32 device tensor [imp_groups, cols]")
    if out is None:
        q = torch.empty((rows, cols // 2), dtype=torch.uint8, device=x.device)
        sc = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
    else:
        q, sc = out
    rc = nvfp4_quant_online(METHOD_IDS[method], _ptr(x), dt, rows, cols, block, _ptr(importance),
                            imp_groups, imp_group_rows, ctypes.c_float(static_scale),
                            SCALE_LAYOUTS[layout], None, _ptr(q), _ptr(sc), _stream(x.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_quant_online")
    if layout == "row_major" and out is None:
        sc = sc.view(rows, cols // block)
    return q, sc


def swiglu(gate: torch.Tensor, up: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """h = bf16(silu(gate) * up) of two bfloat16 device tensors [rows, cols] (the SwiGLU
    producer of nvfp4_quant_online_swiglu, unfused)."""
    if not (gate.is_cuda and gate.dtype == torch.bfloat16 and up.dtype == torch.bfloat16
            and gate.shape == up.shape and gate.dim() == 2 and gate.is_contiguous()
            and up.is_contiguous()):
        raise ValueError("gate and up must be contiguous bfloat16 device tensors of one 2-D shape")
    rows, cols = gate.shape
    h = torch.empty_like(gate) if out is None else out
    rc = nvfp4_swiglu(_ptr(gate), _ptr(up), rows, cols, _ptr(h), _stream(gate.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_swiglu")
    return h


def quantize_online_swiglu(gate: torch.Tensor, up: torch.Tensor, method: str, static_scale: float,
                           importance: torch.Tensor | None = None, imp_groups: int = 1,
                           imp_group_rows: int = 1, layout: str = "row_major", out=None):
    """NVFP4 of h = bf16(silu(gate) * up) with a static global scale, h never written
    (nvfp4_quant_online_swiglu; block 16).  Returns (q, scales) like quantize_online()."""
    if not (gate.is_cuda and gate.dtype == torch.bfloat16 and up.dtype == torch.bfloat16
            and gate.shape == up.shape and gate.dim() == 2 and gate.is_contiguous()
            and up.is_contiguous()):
        raise ValueError("gate and up must be contiguous bfloat16 device tensors of one 2-D shape")
    rows, cols = gate.shape
    nbytes = nvfp4_scales_bytes(rows, cols, 16, SCALE_LAYOUTS[layout])
    if nbytes < 0:
        raise NVFP4Error(int(nbytes), "nvfp4_scales_bytes")
    if importance is not None and not (importance.is_cuda and importance.dtype == torch.float32
                                       and importance.is_contiguous()
                                       and importance.numel() == imp_groups * cols):
        raise ValueError("importance must be a contiguous float32 device tensor [imp_groups, cols]")
    if out is None:
        q = torch.empty((rows, cols // 2), dtype=torch.uint8, device=gate.device)
        sc = torch.empty(nbytes, dtype=torch.uint8, device=gate.device)
    else:
        q, sc = out
    rc = nvfp4_quant_online_swiglu(METHOD_IDS[method], _ptr(gate), _ptr(up), rows, cols,
                                   _ptr(importance), imp_groups, imp_group_rows,
                                   ctypes.c_float(static_scale), SCALE_LAYOUTS[layout], None,
                                   _ptr(q), _ptr(sc), _stream(gate.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_quant_online_swiglu")
    if layout == "row_major" and out is None:
        sc = sc.view(rows, cols // 16)
    return q, sc


def channel_sq_norms(x: torch.Tensor, group_rows: int = 1, groups: int = 1, group_div: int = 1,
                     rep_out: int = 1) -> torch.Tensor:
    """Squared input-channel norms of x [rows, cols] per row group (importance vectors):
    [groups / group_div * rep_out, cols] float32 (see nvfp4_channel_sq_norms)."""
    dt = _check_input(x)
    rows, cols = x.shape
    need = nvfp4_channel_sq_norms_workspace_bytes(rows, cols, groups, group_div)
    if need < 0:
        raise NVFP4Error(int(need), "nvfp4_channel_sq_norms_workspace_bytes")
    ws = torch.empty(max(need // 8, 1), dtype=torch.float64, device=x.device)
    out = torch.empty((groups // group_div * rep_out, cols), dtype=torch.float32, device=x.device)
    rc = nvfp4_channel_sq_norms(_ptr(x), dt, rows, cols, group_rows, groups, group_div, rep_out,
                                _ptr(out), _ptr(ws), ws.numel() * 8, _stream(x.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_channel_sq_norms")
    return out


# ---- GPTQ (LDLQ form) with fixed block scales ----------------------------------------------

def ldlq(w: torch.Tensor, hessian: torch.Tensor, scales: torch.Tensor, S: torch.Tensor,
         block: int = 16, damp: float = 0.01, check: bool = True) -> torch.Tensor:
    """GPTQ nibbles [rows, cols/2] of w with the given fixed scales (see nvfp4_ldlq).
    hessian: [cols, cols] float64 device tensor.  With ``check`` the call synchronizes and
    raises if the damped Hessian is not positive definite."""
    dt = _check_input(w)
    _check_scale(S, w.device)
    rows, cols = w.shape
    if not (hessian.is_cuda and hessian.dtype == torch.float64 and hessian.is_contiguous()
            and tuple(hessian.shape) == (cols, cols)):
        raise ValueError("hessian must be a contiguous float64 device tensor [cols, cols]")
    if not (scales.is_cuda and scales.dtype == torch.uint8 and scales.is_contiguous()
            and scales.numel() == rows * (cols // block)):
        raise ValueError("scales must be a contiguous uint8 device tensor [rows, cols/block]")
    nbytes = nvfp4_ldlq_workspace_bytes(rows, cols)
    ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=w.device)
    q = torch.empty((rows, cols // 2), dtype=torch.uint8, device=w.device)
    status = torch.empty(1, dtype=torch.int32, device=w.device)
    rc = nvfp4_ldlq(_ptr(w), dt, rows, cols, block, _ptr(hessian), _ptr(scales), _ptr(S),
                    ctypes.c_double(damp), _ptr(q), _ptr(status), _ptr(ws), nbytes,
                    _stream(w.device))
    if rc != 0:
        raise NVFP4Error(rc, "nvfp4_ldlq")
    if check and int(status.item()) != 0:
        raise NVFP4Error(-5, "nvfp4_ldlq: the damped Hessian is not positive definite")
    return q


def gptq_quantize(w: torch.Tensor, hessian: torch.Tensor, method: str = "scalesweep_wmse",
                  block: int = 16, damp: float = 0.01):
    """The paper's GPTQ pipeline for one weight: block scales by ``method`` first (WMSE
    importance = the Hessian diagonal), then the LDLQ pass with those scales fixed.
    Returns (q, scales, S)."""
    imp = torch.diagonal(hessian).to(torch.float32).contiguous()
    wm = imp if method in ("four_over_six", "scalesweep_wmse") else None
    _, sc, S = quantize(w, method, block, weight=wm)
    return ldlq(w, hessian, sc, S, block, damp), sc, S
