"""Pins for the oracle's OPT-Tree selection (Appendix B, Part 2).

The tree is pinned against brute-force enumeration of every admissible
depth-limited path, against the structural invariants of a draft tree, and
against special cases: gamma = 1 (the tree is the best B entries of one row),
truncated rows (top-min(B, V) per row gives the same tree as full rows), the
marginal-only case (a nested tree), exact ties, and a vocabulary relabelling.
"""
import itertools

import numpy as np
import pytest

import oracle
from brute_force import brute_force_tree, check_tree_invariants, count_admissible


def random_rows(rng, V, gamma, M, peak=2.0, quantize=None):
    """Random sorted conditional rows and stage-1 candidates for one sequence."""
    R = 1 + (gamma - 1) * M
    z = rng.standard_normal((R, V)) * peak
    if quantize:
        z = np.round(z * quantize) / quantize       # force exact ties
    lp, _ = oracle.log_softmax(z)
    idx = oracle.topk_sorted(lp, V)
    rows_idx = idx.astype(np.int32)
    rows_lp = np.take_along_axis(lp, idx, -1).astype(np.float32)
    topk = np.stack([rng.permutation(V)[:M] for _ in range(gamma)]).astype(np.int32)
    return rows_idx, rows_lp, topk


def same_tree(a, b, fields=("token", "parent", "depth", "score", "rank")):
    return all(np.array_equal(np.asarray(a[f]), np.asarray(b[f])) for f in fields)


CASES = list(itertools.product([8, 16, 32, 64], [1, 2, 3, 4], [1, 2, 3]))


@pytest.mark.parametrize("V,gamma,M", CASES)
def test_tree_equals_brute_force(V, gamma, M):
    rng = np.random.default_rng(V * 100 + gamma * 10 + M)
    for trial in range(3):
        ridx, rlp, topk = random_rows(rng, V, gamma, M, peak=rng.uniform(0.5, 4.0))
        n_adm = count_admissible(ridx, topk, gamma, M)
        for B in sorted({1, 2, 5, min(40, n_adm), min(17, n_adm)}):
            got = oracle.build_tree(ridx, rlp, topk, gamma, M, B)
            ref = brute_force_tree(ridx, rlp, topk, gamma, M, B)
            assert same_tree(got, ref), (V, gamma, M, B, trial)
            check_tree_invariants(got, ridx, rlp, topk, gamma, M, B)


@pytest.mark.parametrize("V,gamma,M", [(8, 3, 2), (16, 4, 3), (12, 2, 3)])
def test_tree_with_exact_ties_equals_brute_force(V, gamma, M):
    rng = np.random.default_rng(99 + V)
    for trial in range(5):
        ridx, rlp, topk = random_rows(rng, V, gamma, M, peak=1.0, quantize=2)
        n_adm = count_admissible(ridx, topk, gamma, M)
        for B in (3, 9, min(30, n_adm)):
            got = oracle.build_tree(ridx, rlp, topk, gamma, M, B)
            ref = brute_force_tree(ridx, rlp, topk, gamma, M, B)
            assert same_tree(got, ref)


def test_gamma1_tree_is_best_entries_of_root_row():
    rng = np.random.default_rng(4)
    V = 50
    ridx, rlp, topk = random_rows(rng, V, 1, 4)
    for B in (1, 7, 50):
        t = oracle.build_tree(ridx, rlp, topk, 1, 4, B)
        assert list(t["token"]) == list(ridx[0, :B])
        assert np.all(t["parent"] == -1) and np.all(t["depth"] == 1)
        assert np.array_equal(t["score"], rlp[0, :B])


@pytest.mark.parametrize("V,gamma,M,B", [(16, 3, 2, 10), (32, 4, 3, 25), (64, 4, 2, 40), (9, 4, 3, 30)])
def test_truncated_rows_give_same_tree(V, gamma, M, B):
    """Keeping min(B, V) entries per row gives the tree of the full rows."""
    rng = np.random.default_rng(V + B)
    for trial in range(4):
        ridx, rlp, topk = random_rows(rng, V, gamma, M, peak=rng.uniform(0.3, 3.0))
        n_adm = count_admissible(ridx, topk, gamma, M)
        b = min(B, n_adm)
        k2 = min(b, V)
        full = oracle.build_tree(ridx, rlp, topk, gamma, M, b)
        cut = oracle.build_tree(ridx[:, :k2], rlp[:, :k2], topk, gamma, M, b)
        assert same_tree(full, cut)


def _descendant_paths(tree, node):
    """Relative token paths below ``node`` (None = root)."""
    kids = {}
    for i, p in enumerate(tree["parent"]):
        kids.setdefault(int(p), []).append(i)
    out = set()

    def walk(n, path):
        for c in kids.get(n, []):
            q = path + (int(tree["token"][c]),)
            out.add(q)
            walk(c, q)
    walk(-1 if node is None else node, ())
    return out


def test_marginal_tree_is_nested():
    """With W_down = 0 every row of a depth is that depth's marginal row, and
    the tree is nested: a later sibling's subtree is contained in an earlier
    sibling's subtree (Appendix C)."""
    rng = np.random.default_rng(11)
    V, d, gamma, M, B = 24, 16, 4, 3, 30
    inputs = {
        "h": oracle.bf16_round(rng.standard_normal((1, gamma, d)) * 1.5),
        "root": np.array([1]),
        "lm_head": oracle.bf16_round(rng.standard_normal((V, d)) * 0.4),
        "emb": rng.standard_normal((V, d)) * 0.02,
        "norm_h_gain": np.ones(d), "norm_e_gain": np.ones(d),
        "w_gate": rng.standard_normal((d, 2 * d)), "w_up": rng.standard_normal((d, 2 * d)),
        "w_down": np.zeros((d, d)),
    }
    out = oracle.draft(inputs, gamma, M, B, mirror_bf16=True, topk2=V)
    t = out["tree"][0]
    checked = 0
    for p in set(int(x) for x in t["parent"]):
        sibs = [i for i in range(B) if t["parent"][i] == p and t["child_row"][i] >= 0]
        for a, b in zip(sibs, sibs[1:]):
            assert _descendant_paths(t, b) <= _descendant_paths(t, a)
            checked += 1
    assert checked > 0


def test_vocabulary_relabelling_permutes_the_draft():
    """Relabelling tokens in every weight permutes all outputs the same way."""
    rng = np.random.default_rng(21)
    V, d, gamma, M, B = 40, 16, 3, 2, 12
    inputs = {
        "h": oracle.bf16_round(rng.standard_normal((1, gamma, d)) * 1.5),
        "root": np.array([7]),
        "lm_head": oracle.bf16_round(rng.standard_normal((V, d)) * 0.4),
        "emb": oracle.bf16_round(rng.standard_normal((V, d)) * 0.02),
        "norm_h_gain": np.ones(d), "norm_e_gain": np.ones(d),
        "w_gate": rng.standard_normal((d, 2 * d)) * 0.3, "w_up": rng.standard_normal((d, 2 * d)) * 0.3,
        "w_down": rng.standard_normal((d, d)) * 0.3,
    }
    perm = rng.permutation(V)           # new id of old token v is perm[v]
    inv = np.argsort(perm)
    p_in = dict(inputs)
    p_in["lm_head"] = inputs["lm_head"][inv]
    p_in["emb"] = inputs["emb"][inv]
    p_in["root"] = perm[inputs["root"]]
    a = oracle.draft(inputs, gamma, M, B, mirror_bf16=True)
    b = oracle.draft(p_in, gamma, M, B, mirror_bf16=True)
    assert np.array_equal(perm[a["stage1"][0]["topk_idx"]], b["stage1"][0]["topk_idx"])
    ta, tb = a["tree"][0], b["tree"][0]
    assert np.array_equal(perm[ta["token"]], tb["token"])
    assert np.array_equal(ta["parent"], tb["parent"])
    assert np.array_equal(ta["score"], tb["score"])


def test_full_pipeline_tree_equals_brute_force():
    """The whole oracle step on tiny weights: its tree matches brute force."""
    rng = np.random.default_rng(8)
    for trial in range(6):
        V, d, gamma, M = int(rng.choice([8, 16, 32])), 16, int(rng.integers(1, 5)), int(rng.integers(1, 4))
        inputs = {
            "h": oracle.bf16_round(rng.standard_normal((1, gamma, d)) * 1.5),
            "root": np.array([int(rng.integers(V))]),
            "lm_head": oracle.bf16_round(rng.standard_normal((V, d)) * 0.5),
            "emb": oracle.bf16_round(rng.standard_normal((V, d)) * 0.02),
            "norm_h_gain": np.ones(d), "norm_e_gain": np.ones(d),
            "w_gate": oracle.bf16_round(rng.standard_normal((d, 2 * d)) * 0.3),
            "w_up": oracle.bf16_round(rng.standard_normal((d, 2 * d)) * 0.3),
            "w_down": oracle.bf16_round(rng.standard_normal((d, d)) * 0.3),
        }
        B = min(20, V)
        out = oracle.draft(inputs, gamma, M, B, mirror_bf16=True, topk2=V)
        rows = out["rows"][0]
        topk = out["stage1"][0]["topk_idx"]
        ref = brute_force_tree(rows["cond_idx"], rows["cond_logprob"], topk, gamma, M, B)
        assert same_tree(out["tree"][0], ref)
        check_tree_invariants(out["tree"][0], rows["cond_idx"], rows["cond_logprob"], topk, gamma, M, B)


def test_planted_tree_mistakes_are_caught(monkeypatch):
    """A tree that expands past the last draft depth disagrees with brute force."""
    import oracle.treeflash_oracle as ot
    real = ot.build_tree

    def no_depth_limit(cond_idx, cond_logprob, topk_idx_seq, gamma, M, B):
        return real(cond_idx, cond_logprob, np.concatenate([topk_idx_seq, topk_idx_seq[-1:]]),
                    gamma + 1, M, B)

    rng = np.random.default_rng(5)
    caught = False
    for trial in range(20):
        V, gamma, M = 8, 2, 2
        ridx, rlp, topk = random_rows(rng, V, gamma, M, peak=3.0)
        ridx2 = np.concatenate([ridx, ridx[1:]])   # rows a depth-3 expansion would index
        rlp2 = np.concatenate([rlp, rlp[1:]])
        B = min(30, count_admissible(ridx, topk, gamma, M))
        got = no_depth_limit(ridx2, rlp2, topk, gamma, M, B)
        ref = brute_force_tree(ridx, rlp, topk, gamma, M, B)
        if not same_tree(got, ref):
            caught = True
            break
    assert caught


def test_hand_worked_tree():
    """A tree small enough to derive by hand from the selection rule.

    V = 3, gamma = 2, M = 1, B = 4.  Depth-1 row (conditioned on the root):
    P(2) = .5, P(0) = .3, P(1) = .2; the only depth-1 candidate is token 2, and
    its depth-2 row is P(1) = .7, P(0) = .2, P(2) = .1.  Path probabilities:
    (2) .5, (2,1) .35, (0) .3, (1) .2, (2,0) .1, (2,2) .05, so the best four in
    order are (2), (2,1), (0), (1).
    """
    ridx = np.array([[2, 0, 1], [1, 0, 2]], dtype=np.int32)
    rlp = np.log(np.array([[0.5, 0.3, 0.2], [0.7, 0.2, 0.1]])).astype(np.float32)
    topk = np.array([[2], [1]], dtype=np.int32)
    t = oracle.build_tree(ridx, rlp, topk, 2, 1, 4)
    assert list(t["token"]) == [2, 1, 0, 1]
    assert list(t["parent"]) == [-1, 0, -1, -1]
    assert list(t["depth"]) == [1, 2, 1, 1]
    assert list(t["child_row"]) == [1, -1, -1, -1]
    assert np.allclose(np.exp(t["score"].astype(np.float64)), [0.5, 0.35, 0.3, 0.2], rtol=1e-6)
