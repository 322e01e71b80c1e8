"""GPU parity of the AR approximator's products (Eq. 1, and the plain SiLU
MLP without an up projection) on every launch path:

* one row block (at most 128 conditional rows, 32 drafter states, widths a
  multiple of 64): the LDS-DMA kernels, with the h~ half of W_gate/W_up
  computed once per drafter state -- one, two and four activation tiles,
  items cut between workgroups and several whole items per workgroup; the
  inputs normalised by whole 16-byte pieces, or element by element when the
  embedding or a gain is not 16-byte aligned;
* 129-256 rows: the input projections on the LDS-DMA kernel with eight
  activation tiles, the down projection register-staged;
* more rows, or widths that are not a multiple of 64: the register-staged
  products;
* fp32.

h' is compared element by element with ``oracle.ar_approximator``: fp32
within 1e-4 relative; bf16 within one bf16 unit in the last place plus 1e-3
(both sides round the same sum to bf16, so a sum next to a rounding boundary
may round either way).  Whole drafting steps of the SiLU MLP go through the
shared comparator.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
from paper_2606_03819_amd import binding, synth
from parity import check_draft, oracle_inputs

pytestmark = pytest.mark.gpu

W = synth.Workload
# (workload, weight std); approximator "swiglu" or "silu"
CASES = [
    # one row block, four activation tiles (106 rows), cut gate/up items
    (W("mlp-dma-nte4", 1, 256, 3000, 16, 7, 24, 256, "bf16", 1.0, 61, 71), 0.08),
    (W("mlp-dma-nte4-silu", 1, 256, 3000, 16, 7, 24, 256, "bf16", 1.0, 61, 71, "", "silu"), 0.08),
    # two tiles, two sequences sharing the row block
    (W("mlp-dma-nte2-b2", 2, 128, 2000, 5, 6, 20, 320, "bf16", 1.0, 62, 72), 0.12),
    # one tile, three sequences (21 rows, 12 drafter states)
    (W("mlp-dma-nte1-b3", 3, 64, 900, 4, 2, 10, 64, "bf16", 1.0, 63, 73), 0.2),
    (W("mlp-dma-nte1-b3-silu", 3, 64, 900, 4, 2, 10, 64, "bf16", 1.0, 63, 73, "", "silu"), 0.2),
    # many cut items (gate/up 32 items over 42 workgroups)
    (W("mlp-dma-cut", 1, 512, 2500, 8, 8, 20, 1024, "bf16", 1.0, 64, 74), 0.05),
    # several whole items per workgroup (256 gate/up items of two chunks each)
    (W("mlp-dma-wide", 1, 64, 1500, 6, 5, 16, 8192, "bf16", 1.0, 65, 75), 0.05),
    (W("mlp-dma-wide-silu", 1, 64, 1500, 6, 5, 16, 8192, "bf16", 1.0, 65, 75, "", "silu"), 0.05),
    # 32 drafter states, the most one activation tile holds
    (W("mlp-dma-32-states", 4, 128, 1200, 8, 3, 12, 128, "bf16", 1.0, 66, 76), 0.1),
    # eight activation tiles for the input projections (241 rows; 171 rows of three sequences)
    (W("mlp-dma-nte8", 1, 256, 3000, 16, 16, 24, 256, "bf16", 1.0, 60, 70), 0.08),
    (W("mlp-dma-nte8-silu", 1, 256, 3000, 16, 16, 24, 256, "bf16", 1.0, 60, 70, "", "silu"), 0.08),
    (W("mlp-dma-nte8-b3", 3, 128, 2048, 8, 8, 20, 128, "bf16", 1.0, 68, 78), 0.1),
    # register-staged products: a width that is not a multiple of 64; more rows than one block
    (W("mlp-reg-d96", 2, 96, 1000, 5, 3, 12, 96, "bf16", 1.0, 67, 77), 0.15),
    (W("mlp-reg-d96-silu", 2, 96, 1000, 5, 3, 12, 96, "bf16", 1.0, 67, 77, "", "silu"), 0.15),
    (W("mlp-reg-rows", 5, 128, 2048, 8, 8, 20, 128, "bf16", 1.0, 68, 78), 0.1),
    (W("mlp-reg-rows-silu", 5, 128, 2048, 8, 8, 20, 128, "bf16", 1.0, 68, 78, "", "silu"), 0.1),
    (W("mlp-f32-silu", 2, 96, 1000, 5, 3, 12, 64, "f32", 1.0, 69, 79, "", "silu"), 0.15),
]


def tol_for(w):
    return 2e-2 if w.dtype == "bf16" else 1e-4


def bf16_ulp(x):
    """Unit in the last place of bf16 values of magnitude |x| (8 significant bits)."""
    a = np.maximum(np.abs(x), np.finfo(np.float32).tiny)
    return np.exp2(np.floor(np.log2(a)) - 7)


def seeded_candidates(w, seed):
    """Distinct seeded stage-1 candidate ids [b, gamma, k] (inputs of the row table)."""
    gen = torch.Generator().manual_seed(seed)
    return np.stack([np.stack([torch.randperm(w.V, generator=gen)[:w.k].numpy() for _ in range(w.gamma)])
                     for _ in range(w.b)]).astype(np.int64)


def hprime_bound(w, ref, got):
    if w.dtype == "bf16":
        return bf16_ulp(np.maximum(np.abs(ref), np.abs(got))) + 1e-3
    return 1e-4 * (1.0 + np.abs(ref))


def check_hprime(w, g, o_in, topk):
    """GPU h' against the oracle for every sequence and row; returns the worst error / bound."""
    tk = torch.from_numpy(topk).to(torch.int32).cuda()
    hp = binding.treeflash_arapprox_hidden(g["h"], g["root"], tk, g["emb"], g["norm_h_gain"], g["norm_e_gain"],
                                           g["w_gate"], g.get("w_up"), g["w_down"])
    got = synth.to_numpy64(hp)
    depth, _ = oracle.row_table(w.gamma, w.k)
    worst = 0.0
    for s in range(w.b):
        prev = oracle.previous_tokens(int(o_in["root"][s]), topk[s], w.gamma, w.k)
        ref = oracle.ar_approximator(o_in["h"][s], prev, depth, o_in["emb"], o_in["norm_h_gain"],
                                     o_in["norm_e_gain"], o_in["w_gate"], o_in.get("w_up"), o_in["w_down"],
                                     mirror_bf16=(w.dtype == "bf16"))
        err = np.abs(got[s] - ref)
        bound = hprime_bound(w, ref, got[s])
        bad = np.argwhere(err > bound)
        assert bad.size == 0, (f"{w.name} seq {s}: h' differs at {bad[:5].tolist()}: "
                               f"{got[s][tuple(bad[0])]} vs {ref[tuple(bad[0])]}")
        worst = max(worst, float(np.max(err / bound)))
    return worst


@pytest.mark.parametrize("w,std", CASES, ids=[c[0].name for c in CASES])
def test_hprime_matches_oracle(w, std):
    print(f"[mlp] h' case={w.name} {w.approximator} b{w.b} d{w.d} I{w.I} g{w.gamma} k{w.k}", flush=True)
    cpu = synth.make_inputs(w, "cpu", weight_std=std)
    g = {k: v.cuda() for k, v in cpu.items()}
    o_in = oracle_inputs(cpu)
    ratio = check_hprime(w, g, o_in, seeded_candidates(w, w.state_seed))
    # a second call on the same workspace (arrival counters reset by the call)
    ratio2 = check_hprime(w, g, o_in, seeded_candidates(w, w.state_seed + 1))
    print(f"[mlp] {w.name}: worst error / bound {max(ratio, ratio2):.3f}", flush=True)


def misaligned(t):
    """A copy of `t` at an address 2 bytes past a 16-byte boundary (element aligned only)."""
    flat = torch.empty(t.numel() + 8, dtype=t.dtype, device=t.device)
    view = flat[1:1 + t.numel()].view(t.shape)
    view.copy_(t)
    assert view.data_ptr() % 16 == 2
    return view


@pytest.mark.parametrize("which", ["emb", "norm_e_gain"])
def test_hprime_misaligned_inputs(which):
    """An embedding table or gain that is element aligned only: the normalisation reads them element by
    element."""
    w, std = CASES[0]
    print(f"[mlp] h' case={w.name} with {which} misaligned", flush=True)
    cpu = synth.make_inputs(w, "cpu", weight_std=std)
    g = {k: v.cuda() for k, v in cpu.items()}
    g[which] = misaligned(g[which])
    o_in = oracle_inputs(cpu)
    ratio = check_hprime(w, g, o_in, seeded_candidates(w, w.state_seed + 2))
    print(f"[mlp] {w.name} ({which} misaligned): worst error / bound {ratio:.3f}", flush=True)


SILU_DRAFTS = [c for c in CASES if c[0].approximator == "silu"]


@pytest.mark.parametrize("w,std", SILU_DRAFTS, ids=[c[0].name for c in SILU_DRAFTS])
def test_silu_mlp_draft_matches_oracle(w, std):
    print(f"[mlp] draft case={w.name} b{w.b} d{w.d} V{w.V} g{w.gamma} k{w.k} B{w.B}", flush=True)
    cpu = synth.make_inputs(w, "cpu", weight_std=std)
    check_draft(w, {k: v.cuda() for k, v in cpu.items()}, oracle_inputs(cpu), range(w.b), tol_for(w))


@pytest.mark.parametrize("name", ["qwen3-8b-shape", "qwen3-4b-shape", "qwen3-8b-shape-silu",
                                  "qwen3-8b-shape-i12288"])
def test_full_size_hprime(name):
    """h' at the Qwen3 shapes, in the benchmark's launch configuration."""
    w = synth.get_workload(name)
    print(f"[mlp] full-size h' {w.name}", flush=True)
    g = synth.make_inputs(w, "cuda")
    small = {k: g[k] for k in ("h", "root", "norm_h_gain", "norm_e_gain", "w_gate", "w_down") + (
        ("w_up",) if "w_up" in g else ())}
    o_in = oracle_inputs(small)
    # the embedding rows the row table reads, gathered on the GPU and copied
    # exactly; ids are remapped to the gathered rows on the oracle side only
    topk = seeded_candidates(w, 91)
    ids = np.unique(np.concatenate([topk.reshape(-1), synth.to_numpy64(g["root"]).reshape(-1)]))
    o_in["emb"] = synth.to_numpy64(g["emb"][torch.from_numpy(ids).cuda()])
    remap = {int(t): i for i, t in enumerate(ids)}
    tk = torch.from_numpy(topk).to(torch.int32).cuda()
    hp = binding.treeflash_arapprox_hidden(g["h"], g["root"], tk, g["emb"], g["norm_h_gain"], g["norm_e_gain"],
                                           g["w_gate"], g.get("w_up"), g["w_down"])
    got = synth.to_numpy64(hp)[0]
    depth, _ = oracle.row_table(w.gamma, w.k)
    prev = oracle.previous_tokens(int(o_in["root"][0]), topk[0], w.gamma, w.k)
    prev = np.array([remap[int(t)] for t in prev])
    ref = oracle.ar_approximator(o_in["h"][0], prev, depth, o_in["emb"], o_in["norm_h_gain"], o_in["norm_e_gain"],
                                 o_in["w_gate"], o_in.get("w_up"), o_in["w_down"], mirror_bf16=True)
    err = np.abs(got - ref)
    bound = hprime_bound(w, ref, got)
    print(f"[mlp] {w.name}: worst error / bound {float(np.max(err / bound)):.3f}, max |err| {float(err.max()):.3g}",
          flush=True)
    assert np.all(err <= bound)
    del g
    gc.collect()
    torch.cuda.empty_cache()
