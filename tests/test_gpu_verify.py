"""GPU parity of the verification hand-off against the oracle: tree-attention
inputs (tokens, positions, ancestor mask) and the greedy acceptance walk, on
real OPT-Trees from random rows (small and at the maximum budget) and on the
trees of the Qwen-shaped drafting step; synthetic verifiers agree with the
drafter on a random share of positions.  Integer outputs: exact."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03819_amd import binding, synth

pytestmark = pytest.mark.gpu


def random_trees(rng, b, V, gamma, M, B):
    R = 1 + (gamma - 1) * M
    trees = []
    for s in range(b):
        z = rng.standard_normal((R, V)) * 2.0
        lp, _ = oracle.log_softmax(z)
        idx = oracle.topk_sorted(lp, V)
        topk = np.stack([rng.permutation(V)[:M] for _ in range(gamma)]).astype(np.int32)
        trees.append(oracle.build_tree(idx.astype(np.int32), np.take_along_axis(lp, idx, -1).astype(np.float32),
                                       topk, gamma, M, B))
    return trees


def to_dev(trees):
    return {f: torch.tensor(np.stack([t[f] for t in trees]), dtype=torch.int32).cuda()
            for f in ("token", "parent", "depth")}


def synthetic_targets(rng, trees, V, agree):
    """Verifier next tokens: with probability `agree` the position's best child, else a random token."""
    out = []
    for t in trees:
        B = len(t["token"])
        tg = rng.integers(0, V, B + 1)
        first = {}
        for j in range(B):
            first.setdefault(int(t["parent"][j]), j)
        for i in range(B + 1):
            if (i - 1) in first and rng.random() < agree:
                tg[i] = t["token"][first[i - 1]]
        out.append(tg)
    return np.stack(out).astype(np.int32)


def check(trees, roots, targets, gamma):
    dev_tree = to_dev(trees)
    root = torch.tensor(roots, dtype=torch.int32).cuda()
    vi = binding.treeflash_tree_attention_inputs(root, dev_tree)
    acc = binding.treeflash_accept(dev_tree, torch.tensor(targets).cuda(), gamma)
    torch.cuda.synchronize()
    for s, t in enumerate(trees):
        ref = oracle.verification_inputs(int(roots[s]), t["token"], t["parent"], t["depth"])
        assert np.array_equal(vi["tokens"][s].cpu().numpy(), ref["tokens"])
        assert np.array_equal(vi["positions"][s].cpu().numpy(), ref["positions"])
        assert np.array_equal(vi["mask"][s].cpu().numpy().astype(bool), ref["mask"]), f"mask of sequence {s}"
        w = oracle.acceptance_walk(t["token"], t["parent"], targets[s])
        n = int(acc["accept_len"][s])
        assert n + 1 == w["tau"]
        assert acc["accepted"][s, :n].cpu().numpy().tolist() == w["accepted"]
        assert np.all(acc["accepted"][s, n:].cpu().numpy() == -1)
        assert int(acc["bonus"][s]) == w["bonus"]


@pytest.mark.parametrize("b,V,gamma,M,B,agree", [(3, 12, 4, 3, 40, 0.7), (2, 30, 5, 4, 1, 0.9),
                                                   (4, 50, 6, 5, 200, 0.9), (1, 9, 3, 2, 50, 0.0),
                                                   (2, 64, 8, 8, 777, 0.95)])
def test_handoff_matches_oracle(b, V, gamma, M, B, agree):
    rng = np.random.default_rng(B + V)
    trees = random_trees(rng, b, V, gamma, M, B)
    check(trees, rng.integers(0, V, b), synthetic_targets(rng, trees, V, agree), gamma)


def test_handoff_at_the_largest_budget():
    rng = np.random.default_rng(4095)
    V, gamma, M, B = 200, 6, 8, 4095
    trees = random_trees(rng, 1, V, gamma, M, B)
    check(trees, np.array([3]), synthetic_targets(rng, trees, V, 0.95), gamma)


def test_handoff_on_the_qwen_shaped_step():
    w = synth.get_workload("qwen3-8b-shape-batch16")
    g = synth.make_inputs(w, "cuda")
    dr = binding.Drafter(g, w.b, w.gamma, w.k, w.B, w.inv_temperature)
    tree = dr.step(g["h"], g["root"])
    torch.cuda.synchronize()
    trees = [{f: tree[f][s].cpu().numpy() for f in ("token", "parent", "depth")} for s in range(w.b)]
    rng = np.random.default_rng(16)
    check(trees, g["root"].cpu().numpy(), synthetic_targets(rng, trees, w.V, 0.8), w.gamma)
