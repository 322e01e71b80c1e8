"""GPU parity of the marginal OPT-Tree mode (the DDTree baseline) against the
oracle: stage 1 with K = min(B, V) entries per depth, then the marginal tree.

The tree kernel must reproduce the oracle's tree exactly from the same rows
(teacher forcing with the oracle's rows, and the oracle replaying the GPU's
own rows); the GPU's stage-1 lists must match the oracle within the bf16 /
fp32 tolerances of the other parity tests.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03819_amd import binding, synth
from parity import check_topk, check_tree_exact, oracle_inputs, to_cpu_tree

pytestmark = pytest.mark.gpu

W = synth.Workload
CASES = [
    (synth.get_workload("tiny-f32"), 0.05),
    (W("m-bf16-ragged", 2, 96, 1000, 5, 3, 12, 64, "bf16", 1.0, 7, 70), 0.15),
    (W("m-bf16-gamma1", 3, 64, 300, 1, 2, 7, 32, "bf16", 1.0, 9, 90), 0.2),
    (W("m-bf16-vocab-below-budget", 2, 48, 20, 3, 2, 30, 32, "bf16", 1.0, 11, 110), 0.3),
    (W("m-bf16-budget-300", 1, 128, 2048, 4, 2, 300, 64, "bf16", 1.0 / 0.7, 12, 120), 0.1),
    (W("m-bf16-budget-1100-lds-frontier", 1, 64, 1000, 3, 2, 1100, 32, "bf16", 1.0, 13, 130), 0.2),
]


def tol_for(w):
    return 2e-2 if w.dtype == "bf16" else 1e-4


def _subtree_paths(tree, node):
    kids = {}
    for i, p in enumerate(tree["parent"]):
        kids.setdefault(int(p), []).append(i)
    out = set()

    def walk(n, path):
        for c in kids.get(n, []):
            q = path + (int(tree["token"][c]),)
            out.add(q)
            walk(c, q)
    walk(node, ())
    return out


def run_marginal(w, cpu, seqs):
    g = {k: cpu[k].cuda() for k in ("h", "lm_head")}
    o_in = oracle_inputs({k: cpu[k] for k in ("h", "lm_head")})   # the marginal path reads nothing else
    md = binding.MarginalDrafter(g["lm_head"], w.b, w.gamma, w.B, w.inv_temperature)
    tree = md.step(g["h"])
    torch.cuda.synchronize()
    gidx, glp = md.idx.cpu().numpy(), md.lp.cpu().numpy()
    for s in seqs:
        st1 = oracle.marginal_stage(o_in["h"][s:s + 1], o_in["lm_head"], md.K, w.inv_temperature)
        check_topk(gidx[s], glp[s], st1["logprob"][0], tol_for(w), f"{w.name} stage 1 seq {s}")
        ref = oracle.build_marginal_tree(gidx[s], glp[s], w.gamma, w.B)
        check_tree_exact(to_cpu_tree(tree, s), ref, f"{w.name} tree from GPU rows, seq {s}")
    return md, tree, o_in


@pytest.mark.parametrize("w,std", CASES, ids=[c[0].name for c in CASES])
def test_marginal_draft_matches_oracle(w, std):
    print(f"[marginal] case={w.name} b{w.b} d{w.d} V{w.V} g{w.gamma} B{w.B}", flush=True)
    cpu = synth.make_inputs(w, "cpu", weight_std=std)
    md, _, o_in = run_marginal(w, cpu, range(w.b))
    # teacher forcing: the oracle's own rows through the GPU tree kernel
    o = oracle.draft_marginal(o_in, w.gamma, w.B, w.inv_temperature)
    idx = torch.tensor(np.stack([t["topk_idx"] for t in o["stage1"]]), dtype=torch.int32).cuda()
    lp = torch.tensor(np.stack([t["topk_logprob"] for t in o["stage1"]]).astype(np.float32)).cuda()
    gt = binding.treeflash_build_tree_marginal(idx, lp, w.B)
    torch.cuda.synchronize()
    for s in range(w.b):
        check_tree_exact(to_cpu_tree(gt, s), o["tree"][s], f"{w.name} tree from oracle rows, seq {s}")


def test_marginal_tree_with_exact_ties():
    w = W("m-bf16-ties", 1, 64, 2000, 3, 4, 40, 32, "bf16", 1.0, 14, 140)
    cpu = synth.make_inputs(w, "cpu", weight_std=0.1)
    cpu["lm_head"] = cpu["lm_head"][torch.arange(w.V) % 5].contiguous()
    run_marginal(w, cpu, [0])


@pytest.mark.parametrize("name", ["qwen3-8b-shape", "qwen3-4b-shape"])
def test_marginal_full_size(name):
    """Qwen-shaped stage 1 (K = B = 32) and the marginal tree, checked against
    the oracle, plus the nested structure of Appendix C on the GPU tree."""
    w = synth.get_workload(name)
    print(f"[marginal] full size {name}", flush=True)
    g = synth.make_inputs(w, "cuda")
    cpu = {k: g[k].cpu() for k in ("h", "lm_head")}
    del g
    md, tree, _ = run_marginal(w, cpu, [0])
    t = to_cpu_tree(tree, 0)
    checked = 0
    for p in set(int(x) for x in t["parent"]):
        sibs = [i for i in range(w.B) if t["parent"][i] == p]
        for a, b in zip(sibs, sibs[1:]):
            assert _subtree_paths(t, b) <= _subtree_paths(t, a)
            checked += 1
    assert checked > 0
