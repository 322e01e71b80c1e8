"""Seeded synthetic inputs for the TreeFlash drafting path.

This module only draws random tensors; it holds none of the method's
arithmetic.  The same tensors are handed to the HIP library and to the CPU
oracle, so both sides see bit-identical inputs.

Recipe (stand-in for the paper's real drafter states, which need trained
checkpoints and evaluation prompts that are not available here):

* every weight -- LM head ``[V, d]``, input embedding ``[V, d]``, SwiGLU gate
  ``[I, 2d]``, up ``[I, 2d]``, down ``[d, I]`` -- is drawn from N(0, 0.02) in
  fp32 and rounded to bf16 (round-to-nearest-even) for the bf16 workloads;
  the tiny workload stays fp32;
* drafter hidden states ``h[b, gamma, d]`` ~ N(0, 1);
* the w/ Linear workloads draw ``W_lin [d, 2d]`` from N(0, 0.02) in place of
  the three SwiGLU matrices; the w/ 2-prev workloads draw gate and up as
  ``[I, 3d]``;
* both RMSNorm gains are ones (no biases anywhere);
* the root token of each sequence, and the context token before it, are
  uniform over the vocabulary.

Weights use one seed per model shape (tiny 1, 4B-shaped 2, 8B-shaped 3), so the
three 8B-shaped workloads share weights.  Hidden states use one seed per
workload; in the batched workload sequence ``s`` uses seed ``1500 + s``.

Values come from torch's generator on the device the tensors are made on
(mt19937 on the CPU, Philox on the GPU), so a workload is reproducible per
device type.  Small workloads are made on the CPU and copied to the GPU; the
Qwen3-shaped ones are made directly on the GPU and copied back when the oracle
needs them.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import torch

__all__ = ["Workload", "WORKLOADS", "get_workload", "make_inputs", "make_weights",
           "make_states", "WEIGHT_STD"]

WEIGHT_STD = 0.02


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape of one drafting workload.

    ``k`` is the stage-1 candidate count M, ``B`` the draft budget,
    ``I`` the SwiGLU width.  ``inv_temperature`` scales logits in both stages.
    """
    name: str
    b: int
    d: int
    V: int
    gamma: int
    k: int
    B: int
    I: int
    dtype: str            # "f32" or "bf16"
    inv_temperature: float
    weight_seed: int
    state_seed: int       # per-sequence seed = state_seed + s when b > 1
    description: str = ""
    # "swiglu" (Eq. 1), "silu" (the plain two-layer SiLU MLP: no up
    # projection), "linear" (the w/ Linear ablation) or "2prev" (the w/
    # 2-prev ablation: SwiGLU on [h~; e~(prev1); e~(prev2)])
    approximator: str = "swiglu"

    @property
    def rows(self) -> int:
        """Conditional rows per sequence: one for depth 1, k per deeper depth
        (2prev: one, then k at depth 2 and k*k per deeper depth)."""
        if self.approximator == "2prev":
            return 1 if self.gamma == 1 else 1 + self.k + (self.gamma - 2) * self.k * self.k
        return 1 + (self.gamma - 1) * self.k

    @property
    def topk2(self) -> int:
        """Stage-2 candidates kept per row: min(B, V)."""
        return min(self.B, self.V)

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    w.name: w for w in [
        Workload("tiny-f32", 1, 256, 4096, 8, 4, 16, 256, "f32", 1.0, 1, 11,
                 "tiny fp32 case the oracle finishes in well under a second"),
        Workload("qwen3-4b-shape", 1, 2560, 151936, 16, 8, 32, 2560, "bf16", 1.0 / 0.7, 2, 12,
                 "Qwen3-4B-shaped bf16, batch 1, drafter temperature 0.7"),
        Workload("qwen3-8b-shape", 1, 4096, 151936, 16, 8, 32, 4096, "bf16", 1.0, 3, 13,
                 "Qwen3-8B-shaped bf16, batch 1: weight-streaming, HBM-bound"),
        Workload("qwen3-8b-shape-k16-b64", 1, 4096, 151936, 16, 16, 64, 4096, "bf16", 1.0, 3, 14,
                 "Qwen3-8B-shaped bf16, batch 1, M=16 candidates, budget 64"),
        Workload("qwen3-8b-shape-batch16", 16, 4096, 151936, 16, 8, 32, 4096, "bf16", 1.0, 3, 1500,
                 "Qwen3-8B-shaped bf16, 16 independent sequences: MFMA-bound"),
        # ends of the budget and branching sweeps (drafting cost only)
        Workload("qwen3-8b-shape-b512", 1, 4096, 151936, 16, 8, 512, 4096, "bf16", 1.0, 3, 13,
                 "Qwen3-8B-shaped bf16, batch 1, budget 512 (512-entry stage-2 lists)"),
        Workload("qwen3-8b-shape-m64", 1, 4096, 151936, 16, 64, 32, 4096, "bf16", 1.0, 3, 13,
                 "Qwen3-8B-shaped bf16, batch 1, M=64 candidates (961 conditional rows)"),
        # the AR approximator at the width the paper's parameter counts imply
        # (5*d*I = +125M / +251M: the target models' MLP widths)
        Workload("qwen3-4b-shape-i9728", 1, 2560, 151936, 16, 8, 32, 9728, "bf16", 1.0 / 0.7, 2, 12,
                 "Qwen3-4B-shaped bf16, SwiGLU width 9728 (the paper's AR-approximator size)"),
        Workload("qwen3-8b-shape-i12288", 1, 4096, 151936, 16, 8, 32, 12288, "bf16", 1.0, 3, 13,
                 "Qwen3-8B-shaped bf16, SwiGLU width 12288 (the paper's AR-approximator size)"),
        # the w/ Linear ablation: one [d, 2d] layer in place of the SwiGLU
        # (I is unused); same LM head, embedding and states as qwen3-8b-shape
        # the w/ 2-prev ablation: bigram rows (1 + 8 + 14*64 = 905 per sequence)
        Workload("qwen3-8b-shape-2prev", 1, 4096, 151936, 16, 8, 32, 4096, "bf16", 1.0, 3, 13,
                 "Qwen3-8B-shaped bf16, w/ 2-prev approximator (905 bigram rows)", "2prev"),
        Workload("qwen3-8b-shape-linear", 1, 4096, 151936, 16, 8, 32, 0, "bf16", 1.0, 3, 13,
                 "Qwen3-8B-shaped bf16, w/ Linear approximator", "linear"),
        # the plain two-layer SiLU MLP (no up projection) in place of the SwiGLU
        Workload("qwen3-8b-shape-silu", 1, 4096, 151936, 16, 8, 32, 4096, "bf16", 1.0, 3, 13,
                 "Qwen3-8B-shaped bf16, plain SiLU MLP approximator", "silu"),
    ]
}


def get_workload(name: str) -> Workload:
    try:
        return WORKLOADS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}") from None


def _generator(device: torch.device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _normal(shape, std, g, device, dtype):
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    # float32 -> bfloat16 conversion in torch is round-to-nearest-even
    return x.to(dtype)


def make_weights(w: Workload, device="cpu", weight_std: float = WEIGHT_STD) -> Dict[str, torch.Tensor]:
    """Weights in draw order: LM head, embedding, gate, up, down (no up for
    the plain SiLU MLP; for the linear approximator, W_lin [d, 2d] in their
    place), then gains.

    ``weight_std`` other than 0.02 is only used by tests that want sharper
    distributions on small shapes.
    """
    device = torch.device(device)
    dt = w.torch_dtype
    g = _generator(device, w.weight_seed)
    out = {}
    out["lm_head"] = _normal((w.V, w.d), weight_std, g, device, dt)
    out["emb"] = _normal((w.V, w.d), weight_std, g, device, dt)
    if w.approximator == "linear":
        out["w_lin"] = _normal((w.d, 2 * w.d), weight_std, g, device, dt)
    else:
        kin = 3 * w.d if w.approximator == "2prev" else 2 * w.d
        out["w_gate"] = _normal((w.I, kin), weight_std, g, device, dt)
        if w.approximator != "silu":
            out["w_up"] = _normal((w.I, kin), weight_std, g, device, dt)
        out["w_down"] = _normal((w.d, w.I), weight_std, g, device, dt)
    out["norm_h_gain"] = torch.ones(w.d, device=device, dtype=dt)
    out["norm_e_gain"] = torch.ones(w.d, device=device, dtype=dt)
    return out


def make_states(w: Workload, device="cpu") -> Dict[str, torch.Tensor]:
    """Drafter hidden states h[b, gamma, d] ~ N(0,1), root tokens [b] and the
    context token before each root [b] (read by the 2-prev rows only)."""
    device = torch.device(device)
    hs, roots, ctx = [], [], []
    for s in range(w.b):
        seed = w.state_seed + s if w.b > 1 else w.state_seed
        g = _generator(device, seed)
        hs.append(_normal((w.gamma, w.d), 1.0, g, device, w.torch_dtype))
        roots.append(torch.randint(0, w.V, (1,), generator=g, device=device, dtype=torch.int64))
        ctx.append(torch.randint(0, w.V, (1,), generator=g, device=device, dtype=torch.int64))
    h = torch.stack(hs, 0).contiguous()
    root = torch.cat(roots).to(torch.int32)
    context = torch.cat(ctx).to(torch.int32)
    return {"h": h, "root": root, "context": context}


def default_device_for(w: Workload) -> str:
    """Small workloads are drawn on the CPU, Qwen3-shaped ones on the GPU."""
    return "cpu" if w.V * w.d <= (1 << 22) else "cuda"


def make_inputs(w: Workload, device: Optional[str] = None,
                weight_std: float = WEIGHT_STD) -> Dict[str, torch.Tensor]:
    """All inputs of one workload, drawn on ``device`` (default per workload)."""
    device = device or default_device_for(w)
    out = make_weights(w, device, weight_std)
    out.update(make_states(w, device))
    return out


def to_numpy64(t: torch.Tensor):
    """Exact float64 (or int64) numpy copy of a tensor, for the oracle."""
    t = t.detach().to("cpu")
    if t.is_floating_point():
        return t.to(torch.float64).numpy()
    return t.to(torch.int64).numpy()
