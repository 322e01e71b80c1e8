"""Pins for the oracle's verification hand-off (Method, "Inference":
equality-check verification; Experiments, "Metrics": block efficiency tau =
accepted tokens + the verifier's residual token).

The ancestor mask is pinned by structural facts (reflexive, root in every
row, rows nested along parent edges, row sums = depth + 1, a chain gives the
lower triangle); the acceptance walk by an independent closed form: the
accepted node is the deepest node whose every ancestor-or-self token equals
the target of its parent, and by synthetic verifiers that agree with a chosen
path.
"""
import numpy as np
import pytest

import oracle


def random_tree(rng, V=12, gamma=4, M=3, B=40):
    """A real OPT-Tree from random rows (the oracle's tree builder)."""
    R = 1 + (gamma - 1) * M
    z = rng.standard_normal((R, V)) * 2.0
    lp, _ = oracle.log_softmax(z)
    idx = oracle.topk_sorted(lp, V)
    topk = np.stack([rng.permutation(V)[:M] for _ in range(gamma)]).astype(np.int32)
    t = oracle.build_tree(idx.astype(np.int32), np.take_along_axis(lp, idx, -1).astype(np.float32),
                          topk, gamma, M, B)
    return t, V


def test_mask_structure():
    rng = np.random.default_rng(1)
    for trial in range(10):
        t, V = random_tree(rng, B=int(rng.integers(1, 45)))
        vi = oracle.verification_inputs(5, t["token"], t["parent"], t["depth"])
        m = vi["mask"]
        B = len(t["token"])
        assert m.shape == (B + 1, B + 1)
        assert vi["tokens"][0] == 5 and np.array_equal(vi["tokens"][1:], t["token"])
        assert vi["positions"][0] == 0 and np.array_equal(vi["positions"][1:], t["depth"])
        assert np.all(np.diag(m)) and np.all(m[:, 0])
        assert np.array_equal(m.sum(1), np.concatenate([[1], t["depth"] + 1]))
        for j in range(B):
            p = int(t["parent"][j])
            par_row = m[1 + p] if p >= 0 else m[0]
            # the child's row is the parent's row plus itself
            expect = par_row.copy()
            expect[1 + j] = True
            assert np.array_equal(m[1 + j], expect)
        assert not np.any(np.triu(m, 1)), "parents precede children, so the mask is lower triangular"


def test_chain_tree_mask_is_the_lower_triangle():
    B = 6
    tok = np.arange(B, dtype=np.int32)
    par = np.arange(-1, B - 1, dtype=np.int32)
    dep = np.arange(1, B + 1, dtype=np.int32)
    m = oracle.verification_inputs(0, tok, par, dep)["mask"]
    assert np.array_equal(m, np.tril(np.ones((B + 1, B + 1), dtype=bool)))


def deepest_matching_node(token, parent, depth, target):
    """Closed form: nodes whose every ancestor-or-self token equals the target
    of its parent position; the deepest of them (or the root)."""
    B = len(token)
    ok = np.zeros(B, dtype=bool)
    for j in np.argsort(depth, kind="stable"):      # parents before children
        p = int(parent[j])
        ok[j] = (token[j] == target[1 + p]) and (p < 0 or ok[p])
    if not ok.any():
        return -1, 0
    j = int(np.argmax(np.where(ok, depth, -1)))
    return j, int(depth[j])


def test_acceptance_walk_equals_closed_form():
    rng = np.random.default_rng(2)
    for trial in range(200):
        t, V = random_tree(rng, B=int(rng.integers(1, 45)))
        B = len(t["token"])
        # a verifier that mostly agrees with the drafter's best child, else random
        target = rng.integers(0, V, B + 1)
        for i in range(B + 1):
            kids = [j for j in range(B) if t["parent"][j] == i - 1]
            if kids and rng.random() < 0.7:
                target[i] = t["token"][kids[0]]
        w = oracle.acceptance_walk(t["token"], t["parent"], target)
        j, d = deepest_matching_node(t["token"], t["parent"], t["depth"], target)
        assert w["tau"] == d + 1
        assert (w["accepted"][-1] if w["accepted"] else -1) == j
        assert w["bonus"] == target[1 + j]
        # the accepted nodes form a root path
        prev = -1
        for a in w["accepted"]:
            assert t["parent"][a] == prev
            prev = a


def test_verifier_agreeing_with_a_path_accepts_exactly_that_path():
    rng = np.random.default_rng(3)
    t, V = random_tree(rng, B=40)
    B = len(t["token"])
    leaf = int(np.argmax(t["depth"]))
    path = []
    n = leaf
    while n >= 0:
        path.append(n)
        n = int(t["parent"][n])
    path = path[::-1]
    target = np.full(B + 1, -7)          # a token no node carries
    cur = -1
    for n in path:
        target[1 + cur] = t["token"][n]
        cur = n
    w = oracle.acceptance_walk(t["token"], t["parent"], target)
    assert w["accepted"] == path and w["tau"] == len(path) + 1 and w["bonus"] == -7


def test_rejected_first_token_gives_tau_one():
    rng = np.random.default_rng(4)
    t, V = random_tree(rng, B=20)
    target = np.full(len(t["token"]) + 1, -1)
    w = oracle.acceptance_walk(t["token"], t["parent"], target)
    assert w["accepted"] == [] and w["tau"] == 1 and w["bonus"] == -1


def test_planted_walk_mistake_is_caught():
    """A walk that keeps going after a mismatch (skips a level) disagrees with
    the closed form."""
    def bad_walk(token, parent, target):
        cur, acc = -1, []
        for _ in range(8):
            want = target[1 + cur]
            hit = [j for j in range(len(token)) if parent[j] == cur and token[j] == want]
            if not hit:
                kids = [j for j in range(len(token)) if parent[j] == cur]
                if not kids:
                    break
                hit = kids[:1]
            cur = hit[0]
            acc.append(cur)
        return len(acc) + 1

    rng = np.random.default_rng(5)
    caught = False
    for trial in range(50):
        t, V = random_tree(rng, B=30)
        target = rng.integers(0, V, len(t["token"]) + 1)
        _, d = deepest_matching_node(t["token"], t["parent"], t["depth"], target)
        if bad_walk(t["token"], t["parent"], target) != d + 1:
            caught = True
            break
    assert caught
