"""Pins of the oracle's w/ 2-prev ablation (Ablations, Model Design: the AR
approximator reads the previous bigram).

* the row table has 1 + M + (gamma-2) M^2 rows and reads every (candidate of
  depth i-2, candidate of depth i-1) pair once per depth;
* with the prev2 block of W_gate / W_up zero the approximator is the
  single-token one of Eq. 1 (pinned elsewhere) on the same previous token;
* the tree equals a brute force over every admissible bigram path whose rows
  are looked up by token keys, with and without exact ties;
* when every row of a (depth, prev1) group is the same, the tree is the
  single-token OPT-Tree of those rows.
"""
import numpy as np
import pytest

import oracle
from brute_force import brute_force_tree_2prev


def rand_rows(rng, R, V, K, ties=False):
    z = rng.normal(size=(R, V)) * 2.0
    if ties:
        z = np.round(z * 2.0) / 2.0
    lp, _ = oracle.log_softmax(z)
    idx = oracle.topk_sorted(lp, K)
    return idx.astype(np.int32), np.take_along_axis(lp, idx, axis=1).astype(np.float32)


def candidates(rng, gamma, M, V, avoid=()):
    pool = np.array([t for t in range(V) if t not in avoid])
    return np.stack([rng.choice(pool, size=M, replace=False) for _ in range(gamma)]).astype(np.int64)


@pytest.mark.parametrize("gamma,M", [(1, 3), (2, 3), (3, 2), (5, 4), (6, 1)])
def test_row_table_counts_and_pairs(gamma, M):
    depth, s1, s2 = oracle.row_table_2prev(gamma, M)
    R = 1 if gamma == 1 else 1 + M + (gamma - 2) * M * M
    assert depth.shape == (R,)
    assert (depth[0], s1[0], s2[0]) == (1, -1, -2)
    for i in range(2, gamma + 1):
        rows = np.nonzero(depth == i)[0]
        pairs = {(int(s2[r]), int(s1[r])) for r in rows}
        want = {(-1, m) for m in range(M)} if i == 2 else {(a, c) for a in range(M) for c in range(M)}
        assert pairs == want and len(rows) == len(want)
    assert np.all(np.diff(depth) >= 0)


def test_previous_pairs_follow_the_candidates():
    rng = np.random.default_rng(3)
    gamma, M = 4, 3
    topk = candidates(rng, gamma, M, 50)
    p1, p2 = oracle.previous_pairs(101, 100, topk, gamma, M)
    depth, s1, s2 = oracle.row_table_2prev(gamma, M)
    assert (p1[0], p2[0]) == (100, 101)
    for r in range(1, depth.shape[0]):
        assert p1[r] == topk[depth[r] - 2, s1[r]]
        assert p2[r] == (100 if depth[r] == 2 else topk[depth[r] - 3, s2[r]])


@pytest.mark.parametrize("mirror", [False, True])
def test_zero_prev2_block_is_the_single_token_approximator(mirror):
    rng = np.random.default_rng(5)
    gamma, M, d, I, V = 4, 3, 32, 48, 60
    h = rng.normal(size=(gamma, d))
    emb = rng.normal(size=(V, d)) * 0.5
    gh, ge = 1.0 + 0.1 * rng.normal(size=d), 1.0 + 0.1 * rng.normal(size=d)
    wg, wu = rng.normal(size=(I, 3 * d)) * 0.1, rng.normal(size=(I, 3 * d)) * 0.1
    wd = rng.normal(size=(d, I)) * 0.1
    wg[:, 2 * d:] = 0.0
    wu[:, 2 * d:] = 0.0
    if mirror:   # bf16-representable weights, so the rounding points are the only difference
        wg, wu, wd = oracle.bf16_round(wg), oracle.bf16_round(wu), oracle.bf16_round(wd)
    topk = candidates(rng, gamma, M, V, avoid=(7, 8))
    depth, _, _ = oracle.row_table_2prev(gamma, M)
    p1, p2 = oracle.previous_pairs(8, 7, topk, gamma, M)
    got = oracle.ar_approximator_2prev(h, p1, p2, depth, emb, gh, ge, wg, wu, wd, mirror_bf16=mirror)
    ref = oracle.ar_approximator(h, p1, depth, emb, gh, ge, wg[:, :2 * d], wu[:, :2 * d], wd, mirror_bf16=mirror)
    if mirror:
        # same bf16 x and activation operands; sums may differ in the last float64 bit
        assert np.max(np.abs(got - ref) / (np.abs(ref) + 1e-30)) <= 2.0 ** -7
        assert np.mean(got == ref) > 0.98
    else:
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    # and the prev2 block is not ignored when it is not zero
    wg2 = wg.copy()
    wg2[:, 2 * d:] = rng.normal(size=(I, d)) * 0.1
    moved = oracle.ar_approximator_2prev(h, p1, p2, depth, emb, gh, ge, wg2, wu, wd)
    assert np.max(np.abs(moved[1 + M:] - ref[1 + M:])) > 1e-3


def test_prev1_block_zero_makes_rows_depend_on_prev2_only():
    rng = np.random.default_rng(6)
    gamma, M, d, I, V = 4, 3, 16, 32, 40
    h = rng.normal(size=(gamma, d))
    emb = rng.normal(size=(V, d))
    wg, wu = rng.normal(size=(I, 3 * d)) * 0.2, rng.normal(size=(I, 3 * d)) * 0.2
    wd = rng.normal(size=(d, I)) * 0.2
    wg[:, d:2 * d] = 0.0
    wu[:, d:2 * d] = 0.0
    topk = candidates(rng, gamma, M, V, avoid=(1, 2))
    depth, s1, s2 = oracle.row_table_2prev(gamma, M)
    p1, p2 = oracle.previous_pairs(2, 1, topk, gamma, M)
    hp = oracle.ar_approximator_2prev(h, p1, p2, depth, emb, np.ones(d), np.ones(d), wg, wu, wd)
    for i in range(3, gamma + 1):
        for m2 in range(M):
            rows = np.nonzero((depth == i) & (s2 == m2))[0]
            for r in rows[1:]:
                np.testing.assert_allclose(hp[r], hp[rows[0]], rtol=1e-12, atol=1e-12)
        # different m2 give different rows
        a = np.nonzero((depth == i) & (s2 == 0))[0][0]
        b = np.nonzero((depth == i) & (s2 == 1))[0][0]
        assert np.max(np.abs(hp[a] - hp[b])) > 1e-3


@pytest.mark.parametrize("gamma,M,V,K,B,ties,seed", [
    (1, 2, 12, 12, 5, False, 0),
    (2, 3, 15, 15, 20, False, 1),
    (3, 2, 10, 10, 40, False, 2),
    (4, 3, 9, 9, 60, True, 3),
    (4, 3, 12, 6, 25, False, 4),
    (5, 2, 8, 8, 80, True, 5),
])
def test_tree_equals_brute_force(gamma, M, V, K, B, ties, seed):
    rng = np.random.default_rng(seed)
    R = 1 if gamma == 1 else 1 + M + (gamma - 2) * M * M
    topk = candidates(rng, gamma, M, V)
    idx, lp = rand_rows(rng, R, V, K, ties)
    B = min(B, brute_force_tree_2prev(idx, lp, topk, gamma, M, 1)["admissible"])
    tree = oracle.build_tree_2prev(idx, lp, topk, gamma, M, B)
    ref = brute_force_tree_2prev(idx, lp, topk, gamma, M, B)
    for f in ("token", "parent", "depth", "score", "rank"):
        assert np.array_equal(tree[f], ref[f]), f


def test_identical_rows_per_prev1_give_the_single_token_tree():
    rng = np.random.default_rng(11)
    gamma, M, V, B = 5, 3, 12, 60
    topk = candidates(rng, gamma, M, V)
    R1 = 1 + (gamma - 1) * M
    idx1, lp1 = rand_rows(rng, R1, V, V)
    depth, s1, _ = oracle.row_table_2prev(gamma, M)
    # row of the single-token table for the same (depth, prev1)
    src = np.array([0 if depth[r] == 1 else 1 + (depth[r] - 2) * M + s1[r] for r in range(depth.shape[0])])
    t2 = oracle.build_tree_2prev(idx1[src], lp1[src], topk, gamma, M, B)
    t1 = oracle.build_tree(idx1, lp1, topk, gamma, M, B)
    for f in ("token", "parent", "depth", "score", "rank"):
        assert np.array_equal(t2[f], t1[f]), f
    expanded = t2["child_row"] >= 0
    assert np.array_equal(expanded, t1["child_row"] >= 0)
    assert np.array_equal(src[t2["child_row"][expanded]], t1["child_row"][expanded])


def test_draft_2prev_with_zero_prev2_block_matches_draft():
    rng = np.random.default_rng(13)
    b, gamma, M, d, I, V, B = 2, 4, 3, 16, 24, 50, 12
    inp = {"h": rng.normal(size=(b, gamma, d)), "root": np.array([3, 4]), "context": np.array([9, 10]),
           "lm_head": rng.normal(size=(V, d)) * 0.5, "emb": rng.normal(size=(V, d)),
           "norm_h_gain": np.ones(d), "norm_e_gain": np.ones(d),
           "w_gate": rng.normal(size=(I, 3 * d)) * 0.3, "w_up": rng.normal(size=(I, 3 * d)) * 0.3,
           "w_down": rng.normal(size=(d, I)) * 0.3}
    inp["w_gate"][:, 2 * d:] = 0.0
    inp["w_up"][:, 2 * d:] = 0.0
    two = oracle.draft_2prev(inp, gamma, M, B)
    one_inp = dict(inp, w_gate=inp["w_gate"][:, :2 * d], w_up=inp["w_up"][:, :2 * d])
    one = oracle.draft(one_inp, gamma, M, B)
    for s in range(b):
        for f in ("token", "parent", "depth"):
            assert np.array_equal(two["tree"][s][f], one["tree"][s][f]), f
        np.testing.assert_allclose(two["tree"][s]["score"], one["tree"][s]["score"], rtol=0, atol=1e-5)
