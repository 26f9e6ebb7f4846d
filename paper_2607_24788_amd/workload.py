"""Synthetic workloads: shapes, window schedules and seeded inputs.

Holds none of the layer's arithmetic -- only sizes and random numbers -- so
both the GPU path and the CPU oracle consume exactly the same input bytes.
The shapes are those of the Llama-3-8B / 70B-class layers the GLIDE paper
evaluates (Sec. IV-A: d_model 4096, 32 layers; GQA 32/8 and 64/8 heads,
head_dim 128); no dataset or trained weight is used or needed.

Input recipe (every tensor, every workload):
  q, k, v ~ N(0, 1) / sqrt(d), rounded to the element type (round to nearest even)
  Wf[l]   ~ N(0, 1/d)  (variance 1/d), one d x Df matrix per layer
  tau     = 1/sqrt(d)
  log-gates of the gated state (when used) ~ U[-0.4, 0], fp32, per token and KV head
Random streams are torch Philox generators seeded from (workload seed,
layer, tensor, part) so any slice can be regenerated on its own.
"""
import math
from dataclasses import dataclass, field

import numpy as np
import torch


def geo_windows(lo, hi, n_layers):
    """Window rising geometrically with depth: round(lo * (hi/lo)^(l/(L-1)))."""
    if n_layers == 1:
        return [int(lo)]
    return [int(round(lo * (hi / lo) ** (l / (n_layers - 1)))) for l in range(n_layers)]


def blockwise_windows(w, n_layers, middle_delta):
    """The paper's three-block allocation (Sec. III-C, Algorithm 1): early
    layers keep the whole window (delta = 0), late layers are fully linear
    (delta = w), the middle block uses ``middle_delta``; 11/10/11 split for 32
    layers.  Returns the softmax windows W_l = w - delta_l."""
    from . import allocation
    return allocation.windows(n_layers, w, middle_delta)


@dataclass
class Workload:
    name: str
    n_layers: int
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    feat_dim: int
    windows: list
    context: list            # tokens prefilled per sequence
    decode_steps: int
    dtype: torch.dtype
    seed: int
    chunk: int = 64
    notes: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def G(self):
        return self.n_q_heads // self.n_kv_heads

    @property
    def tau(self):
        return 1.0 / math.sqrt(self.head_dim)

    def describe(self):
        return {"workload": self.name, "n_layers": self.n_layers, "batch": self.batch,
                "n_q_heads": self.n_q_heads, "n_kv_heads": self.n_kv_heads, "head_dim": self.head_dim,
                "feat_dim": self.feat_dim, "windows": f"{min(self.windows)}..{max(self.windows)}",
                "sum_windows": int(sum(self.windows)),
                "context": (self.context[0] if len(set(self.context)) == 1
                            else f"{min(self.context)}..{max(self.context)}"),
                "decode_steps": self.decode_steps,
                "dtype": {torch.float32: "fp32", torch.bfloat16: "bf16"}[self.dtype]}


def _ragged(seed, batch, lo, hi):
    g = np.random.Generator(np.random.Philox(seed))
    return [int(x) for x in g.integers(lo, hi + 1, size=batch)]


def workload(name):
    """The five workloads: single fp32 layer, 8B-shaped stack (B=1 and B=32),
    chunked prefill, and a 70B-shaped slice."""
    n = name.lower()
    if n in ("c1", "layer1_fp32"):
        return Workload("layer1_fp32_d64_w64_ctx512", 1, 1, 4, 4, 64, 64, [64], [512], 16, torch.float32, 0)
    if n in ("c2", "llama8b_b1_ctx8k"):
        return Workload("llama8b_32L_b1_ctx8k_geo16-2048", 32, 1, 32, 8, 128, 128, geo_windows(16, 2048, 32),
                        [8192], 256, torch.bfloat16, 1)
    if n in ("c3", "llama8b_b32_ctx32k"):
        return Workload("llama8b_32L_b32_ctx16k-32k_geo64-4096", 32, 32, 32, 8, 128, 128,
                        geo_windows(64, 4096, 32), _ragged(2, 32, 16384, 32768), 128, torch.bfloat16, 2)
    if n in ("c4u", "prefill32k_w512"):
        return Workload("prefill_32L_b4_seq32k_w512", 32, 4, 32, 8, 128, 128, [512] * 32, [32768] * 4, 0,
                        torch.bfloat16, 3)
    if n in ("c4", "c4n", "prefill32k_geo"):
        return Workload("prefill_32L_b4_seq32k_geo16-2048", 32, 4, 32, 8, 128, 128, geo_windows(16, 2048, 32),
                        [32768] * 4, 0, torch.bfloat16, 3)
    if n in ("c2r", "llama8b_b1_ctx8k_reversed"):
        # the same windows falling with depth, the orientation the paper allocates in
        return Workload("llama8b_32L_b1_ctx8k_geo2048-16", 32, 1, 32, 8, 128, 128,
                        geo_windows(16, 2048, 32)[::-1], [8192], 256, torch.bfloat16, 1)
    if n in ("c2b", "llama8b_b1_ctx8k_blockwise"):
        # the paper's (0, w/2, w) allocation at its base window w = 1024
        return Workload("llama8b_32L_b1_ctx8k_blockwise_w1024_0-w/2-w", 32, 1, 32, 8, 128, 128,
                        blockwise_windows(1024, 32, 512), [8192], 256, torch.bfloat16, 5)
    if n in ("c3b", "llama8b_b32_ctx32k_blockwise"):
        return Workload("llama8b_32L_b32_ctx16k-32k_blockwise_w1024_0-w/2-w", 32, 32, 32, 8, 128, 128,
                        blockwise_windows(1024, 32, 512), _ragged(2, 32, 16384, 32768), 128, torch.bfloat16, 6)
    if n in ("c5", "llama70b_b8_ctx64k"):
        return Workload("llama70b_80L_b8_ctx64k_geo32-8192", 80, 8, 64, 8, 128, 128, geo_windows(32, 8192, 80),
                        [65536] * 8, 64, torch.bfloat16, 4)
    raise KeyError(name)


ALL = ["c1", "c2", "c3", "c4u", "c4", "c5"]


# ---------------------------------------------------------------------------
# Seeded tensors.

_TENSOR_ID = {"q": 1, "k": 2, "v": 3, "phi_w": 4, "dq": 5, "dk": 6, "dv": 7, "gate": 8, "dgate": 9}


def _gen(seed, layer, tensor, part, device):
    s = (int(seed) * 1_000_003 + int(layer) * 10_007 + _TENSOR_ID[tensor] * 101 + int(part)) % (2 ** 63)
    g = torch.Generator(device=device)
    g.manual_seed(s)
    return g


def randn(shape, seed, layer, tensor, part=0, scale=1.0, dtype=torch.bfloat16, device="cpu"):
    """N(0,1) * scale from its own Philox stream, rounded to ``dtype``."""
    g = _gen(seed, layer, tensor, part, device)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if scale != 1.0:
        x.mul_(scale)
    return x.to(dtype)


def phi_weights(wl, layers=None, device="cpu"):
    """Wf for the given layers: [len][d][Df], N(0, 1/d)."""
    layers = range(wl.n_layers) if layers is None else layers
    return torch.stack([randn((wl.head_dim, wl.feat_dim), wl.seed, l, "phi_w", scale=wl.head_dim ** -0.5,
                              dtype=wl.dtype, device=device) for l in layers])


def prefill_inputs(wl, layer, seqlens, part=0, device="cpu", qkv_scale=None):
    """Packed prefill inputs of one layer: q [T][Hq][d], k/v [T][Hkv][d]."""
    T = int(sum(seqlens))
    s = wl.head_dim ** -0.5 if qkv_scale is None else qkv_scale
    q = randn((T, wl.n_q_heads, wl.head_dim), wl.seed, layer, "q", part, s, wl.dtype, device)
    k = randn((T, wl.n_kv_heads, wl.head_dim), wl.seed, layer, "k", part, s, wl.dtype, device)
    v = randn((T, wl.n_kv_heads, wl.head_dim), wl.seed, layer, "v", part, s, wl.dtype, device)
    return q, k, v


def decode_inputs(wl, step, layers=None, device="cpu", qkv_scale=None):
    """Decode inputs of one step: q [L][B][Hq][d], k/v [L][B][Hkv][d]."""
    layers = range(wl.n_layers) if layers is None else layers
    s = wl.head_dim ** -0.5 if qkv_scale is None else qkv_scale
    n = len(layers)
    q = torch.empty((n, wl.batch, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=device)
    k = torch.empty((n, wl.batch, wl.n_kv_heads, wl.head_dim), dtype=wl.dtype, device=device)
    v = torch.empty_like(k)
    for i, l in enumerate(layers):
        q[i] = randn(q.shape[1:], wl.seed, l, "dq", step, s, wl.dtype, device)
        k[i] = randn(k.shape[1:], wl.seed, l, "dk", step, s, wl.dtype, device)
        v[i] = randn(v.shape[1:], wl.seed, l, "dv", step, s, wl.dtype, device)
    return q, k, v


GATE_LO = -0.4  # log-gates of the gated state: uniform in [GATE_LO, 0]


def prefill_log_gates(wl, layer, seqlens, part=0, device="cpu"):
    """Packed log-gates of one layer's prefill, [T][Hkv] fp32, uniform in
    [GATE_LO, 0] (the paper fixes no gate; a per-token decay of e^-0.4 .. 1)."""
    T = int(sum(seqlens))
    g = _gen(wl.seed, layer, "gate", part, device)
    return torch.rand((T, wl.n_kv_heads), generator=g, device=device) * GATE_LO


def decode_log_gates(wl, step, device="cpu"):
    """Log-gates of one decode step, [L][B][Hkv] fp32, uniform in [GATE_LO, 0]."""
    g = _gen(wl.seed, 0, "dgate", step, device)
    return torch.rand((wl.n_layers, wl.batch, wl.n_kv_heads), generator=g, device=device) * GATE_LO
