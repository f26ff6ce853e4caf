"""Seeded synthetic inputs for the NVFP4 ScaleSweep hot path.

This module only draws random tensors; it holds none of the quantizer's arithmetic.  The
paper measures on real Llama / Qwen tensors and RedPajama calibration activations, which
are not available here; these generators stand in for them with the same shapes and with
value distributions chosen to resemble LLM weights (heavy tails, a few outlier input
channels) and activations (outlier channels, per-channel scales).

Both the GPU path and the oracle receive the *same* arrays: tensors drawn on a device are
copied to the host before the oracle sees them.

Workloads (blocks always run along the last, input dimension):
  * ``c0``  binary32 [1024, 1024], i.i.d. N(0, 1) from numpy ``default_rng(0)``.
  * ``llama8b_layer``  bfloat16 q/o [4096, 4096], k/v [1024, 4096], gate/up [14336, 4096],
    down [4096, 14336]: entries 0.02 * Student-t(4); round(0.001 * d_in) random input
    columns scaled by 10.  Column-importance weights w_j = mean_t X_tj^2 over 2048
    calibration tokens X_tj ~ N(0, s_j^2), s_j = exp(N(0, 0.5^2)).
  * ``square8192``  one bfloat16 [8192, 8192] weight drawn like the layer above.
  * ``online``  activations [8192, 4096] N(0, 1) with 8 random channels x50; K and V
    [16, 8, 4096, 128] and Q [16, 32, 4096, 128] N(0, 1) times a per-(head, head_dim)
    log-normal(0, 1) channel scale.
  * ``llama70b``  80 layers of q/o [8192, 8192], k/v [1024, 8192], gate/up [28672, 8192],
    down [8192, 28672], drawn per layer on the device like the 8B layer.
"""
from __future__ import annotations

import numpy as np
import torch

LLAMA8B_SHAPES = {
    "q_proj": (4096, 4096), "k_proj": (1024, 4096), "v_proj": (1024, 4096),
    "o_proj": (4096, 4096), "gate_proj": (14336, 4096), "up_proj": (14336, 4096),
    "down_proj": (4096, 14336),
}
LLAMA70B_SHAPES = {
    "q_proj": (8192, 8192), "k_proj": (1024, 8192), "v_proj": (1024, 8192),
    "o_proj": (8192, 8192), "gate_proj": (28672, 8192), "up_proj": (28672, 8192),
    "down_proj": (8192, 28672),
}
CONFIG_IDS = {"c0": 0, "llama8b_layer": 1, "square8192": 2, "online": 3, "llama70b": 4}


def seed_of(*key: int) -> int:
    """A 63-bit torch seed from an integer key via numpy's SeedSequence."""
    return int(np.random.SeedSequence(list(key)).generate_state(1, dtype=np.uint64)[0] >> 1)


def generator(device, *key: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed_of(*key))
    return g


def c0_matrix() -> np.ndarray:
    """binary32 [1024, 1024], i.i.d. N(0, 1), numpy default_rng(0)."""
    return np.random.default_rng(0).standard_normal((1024, 1024), dtype=np.float32)


def student_t4(shape, g: torch.Generator, device) -> torch.Tensor:
    """Student-t with 4 degrees of freedom: Z / sqrt(V / 4), V ~ chi^2(4) = -2 ln(U1 U2)."""
    z = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    u1 = 1.0 - torch.rand(shape, generator=g, device=device, dtype=torch.float32)
    v = torch.log(u1)
    u2 = 1.0 - torch.rand(shape, generator=g, device=device, dtype=torch.float32)
    v.add_(torch.log(u2)).mul_(-2.0)
    return z.div_(torch.sqrt(v.div_(4.0)))


def llm_weight(rows: int, cols: int, g: torch.Generator, device, scale: float = 0.02,
               outlier_frac: float = 0.001, outlier_mult: float = 10.0) -> torch.Tensor:
    """bfloat16 [rows, cols] weight: scale * Student-t(4), round(outlier_frac * cols) random
    input columns multiplied by outlier_mult."""
    w = student_t4((rows, cols), g, device).mul_(scale)
    k = int(round(outlier_frac * cols))
    if k > 0:
        cols_idx = torch.randperm(cols, generator=g, device=device)[:k]
        w[:, cols_idx] *= outlier_mult
    return w.to(torch.bfloat16)


def column_importance(cols: int, g: torch.Generator, device, tokens: int = 2048,
                      chunk: int = 512) -> torch.Tensor:
    """w_j = mean_t X_tj^2 over `tokens` calibration rows, X_tj ~ N(0, s_j^2),
    s_j = exp(N(0, 0.5^2)).  binary32 [cols]."""
    s = torch.exp(torch.randn(cols, generator=g, device=device) * 0.5)
    acc = torch.zeros(cols, device=device, dtype=torch.float64)
    done = 0
    while done < tokens:
        t = min(chunk, tokens - done)
        X = torch.randn((t, cols), generator=g, device=device) * s
        acc += (X.double() ** 2).sum(0)
        done += t
    return (acc / tokens).float()


def llama8b_layer(device="cpu", seed: int = 0, with_weights: bool = True):
    """dict name -> (bf16 weight [out, in], binary32 importance [in] or None)."""
    out = {}
    for ti, (name, (r, c)) in enumerate(LLAMA8B_SHAPES.items()):
        g = generator(device, seed, CONFIG_IDS["llama8b_layer"], ti)
        w = llm_weight(r, c, g, device)
        imp = column_importance(c, g, device) if with_weights else None
        out[name] = (w, imp)
    return out


def square8192(device="cpu", seed: int = 0, n: int = 8192):
    g = generator(device, seed, CONFIG_IDS["square8192"], 0)
    w = llm_weight(n, n, g, device)
    imp = column_importance(n, g, device)
    return w, imp


def online_tensors(device="cpu", seed: int = 0, scale_down: int = 1):
    """Activations, K, V, Q for online quantization.  `scale_down` divides the token /
    sequence extent (tests use small versions of the same recipe)."""
    g = generator(device, seed, CONFIG_IDS["online"], 0)
    tokens = 8192 // scale_down
    act = torch.randn((tokens, 4096), generator=g, device=device)
    ch = torch.randperm(4096, generator=g, device=device)[:8]
    act[:, ch] *= 50.0
    seq = 4096 // scale_down
    out = {"act": act.to(torch.bfloat16)}
    for name, heads in (("k", 8), ("v", 8), ("q", 32)):
        c = torch.exp(torch.randn((heads, 128), generator=g, device=device))
        t = torch.randn((16, heads, seq, 128), generator=g, device=device)
        t.mul_(c[None, :, None, :])
        out[name] = t.to(torch.bfloat16)
    return out


def llama70b_layer(layer: int, device="cuda", seed: int = 0):
    out = {}
    for ti, (name, (r, c)) in enumerate(LLAMA70B_SHAPES.items()):
        g = generator(device, seed, CONFIG_IDS["llama70b"], ti, layer)
        w = llm_weight(r, c, g, device)
        imp = column_importance(c, g, device)
        out[name] = (w, imp)
    return out


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bfloat16 bit patterns of a tensor as a host uint16 array (no arithmetic)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def host_array(t: torch.Tensor) -> np.ndarray:
    """Host copy in the oracle's input convention: float32, or uint16 for bfloat16."""
    if t.dtype == torch.bfloat16:
        return bf16_bits(t)
    return t.detach().contiguous().float().cpu().numpy()


def random_blocks(n_blocks: int, n: int, rng: np.random.Generator, kind: str = "normal"):
    """Normalized blocks for block-level tests: rows of n binary32 values."""
    if kind == "normal":
        y = rng.standard_normal((n_blocks, n)).astype(np.float32)
        y *= np.float32(100.0) / np.abs(y).max(axis=1, keepdims=True)
        return y.astype(np.float32)
    if kind == "t4":
        z = rng.standard_normal((n_blocks, n))
        v = rng.chisquare(4, (n_blocks, n))
        y = z / np.sqrt(v / 4)
        return (y * rng.uniform(0.05, 300.0, (n_blocks, 1))).astype(np.float32)
    if kind == "uniform":
        return rng.uniform(-1, 1, (n_blocks, n)).astype(np.float32) * np.float32(50.0)
    raise ValueError(kind)
