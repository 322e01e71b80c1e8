"""Pins for the oracle's marginal OPT-Tree (the paper's DDTree baseline:
OPT-Tree selection on the drafter's marginal distributions, Related Work and
Appendix C).

Pinned against brute-force enumeration of every token path, against the
TreeFlash oracle in the case where the two must coincide (every token a
stage-1 candidate and a zero down projection, so every conditional row is
its depth's marginal row), against row truncation, and against the nested
structure Appendix C describes.
"""
import numpy as np
import pytest

import oracle
from brute_force import brute_force_marginal_tree


def marginal_rows(rng, V, gamma, peak=2.0, quantize=None):
    z = rng.standard_normal((gamma, V)) * peak
    if quantize:
        z = np.round(z * quantize) / quantize       # force exact ties
    lp, _ = oracle.log_softmax(z)
    idx = oracle.topk_sorted(lp, V)
    return idx.astype(np.int32), np.take_along_axis(lp, idx, -1).astype(np.float32)


def same_tree(a, b, fields=("token", "parent", "depth", "score", "rank")):
    return all(np.array_equal(np.asarray(a[f]), np.asarray(b[f])) for f in fields)


def n_paths(V, gamma):
    return sum(V ** i for i in range(1, gamma + 1))


@pytest.mark.parametrize("V,gamma", [(3, 1), (3, 3), (4, 2), (5, 3), (6, 3), (8, 2), (4, 4)])
def test_marginal_tree_equals_brute_force(V, gamma):
    rng = np.random.default_rng(10 * V + gamma)
    for trial in range(4):
        idx, lp = marginal_rows(rng, V, gamma, peak=rng.uniform(0.3, 3.0))
        for B in sorted({1, 3, min(20, n_paths(V, gamma)), n_paths(V, gamma)}):
            got = oracle.build_marginal_tree(idx, lp, gamma, B)
            assert same_tree(got, brute_force_marginal_tree(idx, lp, gamma, B)), (V, gamma, B, trial)
            assert np.array_equal(got["child_row"], np.where(got["depth"] < gamma, got["depth"], -1))


@pytest.mark.parametrize("V,gamma", [(4, 3), (6, 2)])
def test_marginal_tree_with_exact_ties_equals_brute_force(V, gamma):
    rng = np.random.default_rng(7 + V)
    for trial in range(5):
        idx, lp = marginal_rows(rng, V, gamma, peak=1.0, quantize=2)
        for B in (2, 7, min(25, n_paths(V, gamma))):
            assert same_tree(oracle.build_marginal_tree(idx, lp, gamma, B),
                             brute_force_marginal_tree(idx, lp, gamma, B))


@pytest.mark.parametrize("V,gamma,B", [(16, 3, 10), (40, 4, 25), (9, 4, 30)])
def test_marginal_rows_truncated_to_budget_give_same_tree(V, gamma, B):
    rng = np.random.default_rng(V + B)
    idx, lp = marginal_rows(rng, V, gamma, peak=2.0)
    k = min(B, V)
    assert same_tree(oracle.build_marginal_tree(idx, lp, gamma, B),
                     oracle.build_marginal_tree(idx[:, :k], lp[:, :k], gamma, B))


def _inputs(rng, V, d, gamma, zero_down=True):
    return {
        "h": oracle.bf16_round(rng.standard_normal((1, gamma, d)) * 1.5),
        "root": np.array([1]),
        "lm_head": oracle.bf16_round(rng.standard_normal((V, d)) * 0.4),
        "emb": oracle.bf16_round(rng.standard_normal((V, d)) * 0.02),
        "norm_h_gain": np.ones(d), "norm_e_gain": np.ones(d),
        "w_gate": rng.standard_normal((d, 2 * d)), "w_up": rng.standard_normal((d, 2 * d)),
        "w_down": np.zeros((d, d)) if zero_down else rng.standard_normal((d, d)) * 0.1,
    }


@pytest.mark.parametrize("V,gamma,B", [(6, 3, 20), (10, 3, 40), (5, 4, 60)])
def test_treeflash_with_all_candidates_and_zero_down_is_the_marginal_tree(V, gamma, B):
    """M = V makes every token a stage-1 candidate (every node expandable), and
    W_down = 0 makes every conditional row of depth i the marginal row of
    depth i (h' = h for bf16-exact h): the TreeFlash tree is then the
    marginal tree."""
    rng = np.random.default_rng(V * gamma + B)
    inputs = _inputs(rng, V, 16, gamma)
    tf = oracle.draft(inputs, gamma, V, B, mirror_bf16=True)["tree"][0]
    mg = oracle.draft_marginal(inputs, gamma, B)["tree"][0]
    assert same_tree(tf, mg)


def test_treeflash_with_a_real_approximator_differs_from_the_marginal_tree():
    rng = np.random.default_rng(3)
    V, gamma, B = 12, 3, 40
    inputs = _inputs(rng, V, 16, gamma, zero_down=False)
    tf = oracle.draft(inputs, gamma, V, B, mirror_bf16=True)["tree"][0]
    mg = oracle.draft_marginal(inputs, gamma, B)["tree"][0]
    assert not same_tree(tf, mg)


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


def test_marginal_tree_is_nested():
    """Appendix C: for siblings i before j, the descendants of j form a subtree
    of the descendants of i."""
    rng = np.random.default_rng(12)
    checked = 0
    for trial in range(6):
        idx, lp = marginal_rows(rng, 7, 3, peak=1.5)
        t = oracle.build_marginal_tree(idx, lp, 3, 60)
        for p in set(int(x) for x in t["parent"]):
            sibs = [i for i in range(60) if t["parent"][i] == p]
            for a, b in zip(sibs, sibs[1:]):
                assert _subtree_paths(t, b) <= _subtree_paths(t, a)
                checked += 1
    assert checked > 0


def test_planted_marginal_mistake_is_caught():
    """Expanding a depth-d node from its own depth's row (one row too early)
    disagrees with brute force."""
    rng = np.random.default_rng(8)
    caught = False
    for trial in range(20):
        idx, lp = marginal_rows(rng, 5, 3, peak=2.0)
        shifted = np.concatenate([idx[:1], idx[:-1]]), np.concatenate([lp[:1], lp[:-1]])
        got = oracle.build_marginal_tree(shifted[0], shifted[1], 3, 30)
        if not same_tree(got, brute_force_marginal_tree(idx, lp, 3, 30)):
            caught = True
            break
    assert caught
