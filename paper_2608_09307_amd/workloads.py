"""Seeded synthetic workloads for LinSimp (shared by tests, smoke and bench).

This module only draws random numbers and shapes them; it holds none of the
layer's arithmetic.  The oracle and the GPU path both consume the tensors it
returns (the oracle after an exact upcast of the same values to float64).

Recipe (every workload):
  * one ``torch.Generator`` on the target device, seeded with ``seed``;
  * draw order q, k, v, r, u (each N(0,1) float32, times d^{-1/4}, then cast
    to the workload dtype with round-to-nearest-even), then Omega [H, m, D]
    (N(0,1) float32, one bank per head), then dO (N(0,1), workload dtype)
    for backward workloads, then the key-boost mask;
  * key boost (stress workload): each (batch, position) is picked with
    probability ``boost_frac`` and its key is multiplied by ``boost`` in every
    head (the multiply is a power of two, exact in bfloat16).
Decode workloads draw a prefix of ``n_prefix`` tokens per sequence (streams
[S, H, n_prefix, D]) and then one new token per sequence ([S, H, D]).

The five named workloads are the paper's layer shapes: a single fp32 head, the
2k-context layer (d=64, m=64), the 16k-context layer (d=128, m=128; the
throughput workload), the decode step over 256 sequences, and the 64k stress
shape with boosted keys.
"""

from __future__ import annotations

import dataclasses
from typing import Optional

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    n: int
    D: int
    Dv: int
    m: int
    w: int
    dtype: str            # "f32" | "bf16"
    mode: str             # "fwd" | "fwdbwd" | "decode"
    boost_frac: float = 0.0
    boost: float = 1.0
    n_prefix: int = 0     # decode: tokens already in the state
    seed: int = 0

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    "head_f32_n256": Workload("head_f32_n256", 1, 1, 256, 32, 32, 32, 64, "f32", "fwd"),
    "layer2k_bf16": Workload("layer2k_bf16", 4, 8, 2048, 64, 64, 64, 64, "bf16", "fwd"),
    "layer16k_bf16": Workload("layer16k_bf16", 2, 16, 16384, 128, 128, 128, 64, "bf16", "fwdbwd"),
    "decode_s256_h16": Workload("decode_s256_h16", 256, 16, 1, 128, 128, 128, 64, "bf16",
                                "decode", n_prefix=8192),
    "stress64k_m256": Workload("stress64k_m256", 1, 32, 65536, 128, 128, 256, 64, "bf16",
                               "fwdbwd", boost_frac=0.05, boost=4.0),
    # the layer the paper times (8 sequences x 6 heads of 2048 tokens, d = 64, m = 128)
    "layer2k_h6_d64_m128": Workload("layer2k_h6_d64_m128", 8, 6, 2048, 64, 64, 128, 64, "bf16", "fwdbwd"),
}


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _normal(shape, g, device):
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32)


def make_inputs(wl: Workload, device="cpu", with_grad: Optional[bool] = None):
    """Draw the streams of a forward / backward workload.

    Returns a dict of tensors on ``device``: q, k, r [B, H, n, D];
    v, u [B, H, n, Dv] (workload dtype); omega [H, m, D] float32; and dO
    [B, H, n, Dv] when the workload has a backward (or ``with_grad``).
    """
    g = _gen(device, wl.seed)
    dt = wl.torch_dtype
    s = wl.D ** -0.25
    out = {}
    for name, width in (("q", wl.D), ("k", wl.D), ("v", wl.Dv), ("r", wl.D), ("u", wl.Dv)):
        out[name] = (_normal((wl.B, wl.H, wl.n, width), g, device) * s).to(dt)
    out["omega"] = _normal((wl.H, wl.m, wl.D), g, device)
    need_grad = (wl.mode == "fwdbwd") if with_grad is None else with_grad
    if need_grad:
        out["dO"] = _normal((wl.B, wl.H, wl.n, wl.Dv), g, device).to(dt)
    if wl.boost_frac > 0:
        pick = torch.rand((wl.B, 1, wl.n, 1), generator=g, device=device) < wl.boost_frac
        k = out["k"].float()
        k = torch.where(pick, k * wl.boost, k)
        out["k"] = k.to(dt)
        out["boost_mask"] = pick[:, 0, :, 0]
    return out


def make_head_params(wl: Workload, device="cpu", channel_gate: bool = False):
    """Per-head parameters of the full head, from their own generator (seed
    + 7919, so the streams of ``make_inputs`` are unchanged): tau [H] float32
    around the paper's initial sqrt(D) (times exp(0.1 N(0,1))), and either
    gamma [H] float32 around the initial -2 (plus 0.5 N(0,1)) or channel-gate
    logits [B, H, n, Dv] (N(0,1), workload dtype)."""
    g = _gen(device, wl.seed + 7919)
    tau = torch.exp(0.1 * _normal((wl.H,), g, device)) * wl.D ** 0.5
    if channel_gate:
        gate = _normal((wl.B, wl.H, wl.n, wl.Dv), g, device).to(wl.torch_dtype)
    else:
        gate = -2.0 + 0.5 * _normal((wl.H,), g, device)
    return {"tau": tau, "gate": gate}


def make_bank_draws(H: int, m: int, D: int, seed: int = 0, device="cpu"):
    """Random draws of the orthogonal feature-bank sampler: gauss [H, nb, D, D]
    iid N(0,1) float32 (nb = ceil(m / D)) and radii [H, nb, D], each the norm
    of a fresh D-dimensional N(0, I) vector (a chi_D draw)."""
    g = _gen(device, seed)
    nb = (m + D - 1) // D
    gauss = _normal((H, nb, D, D), g, device)
    radii = torch.linalg.vector_norm(_normal((H, nb, D, D), g, device), dim=-1)
    return gauss, radii


def make_decode_inputs(wl: Workload, device="cpu"):
    """Draw a decode workload: a prefix of ``n_prefix`` tokens per sequence
    (k, v, r, u [S, H, n_prefix, *]) and one new token per sequence
    (q, k, v, r, u [S, H, *]); omega [H, m, D] float32.  S = wl.B."""
    g = _gen(device, wl.seed)
    dt = wl.torch_dtype
    s = wl.D ** -0.25
    S, H, P = wl.B, wl.H, wl.n_prefix
    pre = {}
    for name, width in (("k", wl.D), ("v", wl.Dv), ("r", wl.D), ("u", wl.Dv)):
        pre[name] = (_normal((S, H, P, width), g, device) * s).to(dt)
    omega = _normal((H, wl.m, wl.D), g, device)
    tok = {}
    for name, width in (("q", wl.D), ("k", wl.D), ("v", wl.Dv), ("r", wl.D), ("u", wl.Dv)):
        tok[name] = (_normal((S, H, width), g, device) * s).to(dt)
    return {"prefix": pre, "token": tok, "omega": omega}
