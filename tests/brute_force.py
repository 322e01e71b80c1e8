"""Independent checkers for the tree part of the oracle.

``brute_force_tree`` enumerates every admissible node (every depth-limited path
whose inner nodes are stage-1 candidates of their depth) with float32
left-to-right path sums, sorts all of them by the candidate order and keeps the
best B.  It shares no code with the oracle's heap-based selection.
``check_tree_invariants`` checks the structural facts any valid draft tree has.
"""
from __future__ import annotations

import numpy as np


def _key(score32, depth, path):
    return (-float(score32), depth, path)


def brute_force_tree(cond_idx, cond_logprob, topk_idx_seq, gamma, M, B):
    cond_idx = np.asarray(cond_idx)
    lp = np.asarray(cond_logprob, dtype=np.float32)
    K = cond_idx.shape[1]
    cand = {}
    for dep in range(1, gamma + 1):
        row_of = {int(t): m for m, t in enumerate(np.asarray(topk_idx_seq[dep - 1]))}
        cand[dep] = row_of
    found = []

    stack = [(0, 1, np.float32(0.0), ())]
    while stack:
        row, dep, s_par, path = stack.pop()
        for c in range(K):
            s = np.float32(s_par + lp[row, c])
            p = path + (c,)
            tok = int(cond_idx[row, c])
            found.append((_key(s, dep, p), s, tok, row))
            if dep < gamma and tok in cand[dep]:
                m = cand[dep][tok]
                stack.append((1 + (dep - 1) * M + m, dep + 1, s, p))
    if len(found) < B:
        raise ValueError("budget exceeds admissible nodes")
    found.sort(key=lambda t: t[0])
    top = found[:B]
    pos = {t[0][2]: i for i, t in enumerate(top)}
    out = {k: [] for k in ("token", "parent", "depth", "score", "rank")}
    for key, s, tok, row in top:
        path = key[2]
        out["token"].append(tok)
        out["parent"].append(pos[path[:-1]] if len(path) > 1 else -1)
        out["depth"].append(key[1])
        out["score"].append(s)
        out["rank"].append(path[-1])
    return {
        "token": np.asarray(out["token"], dtype=np.int32),
        "parent": np.asarray(out["parent"], dtype=np.int32),
        "depth": np.asarray(out["depth"], dtype=np.int32),
        "score": np.asarray(out["score"], dtype=np.float32),
        "rank": np.asarray(out["rank"], dtype=np.int32),
        "admissible": len(found),
    }


def count_admissible(cond_idx, topk_idx_seq, gamma, M):
    """Number of admissible nodes given the rows (same enumeration, no scores)."""
    cond_idx = np.asarray(cond_idx)
    total = 0
    stack = [(0, 1)]
    while stack:
        row, dep = stack.pop()
        toks = cond_idx[row]
        total += toks.shape[0]
        if dep < gamma:
            for m, t in enumerate(np.asarray(topk_idx_seq[dep - 1])):
                if np.any(toks == t):
                    stack.append((1 + (dep - 1) * M + m, dep + 1))
    return total


def check_tree_invariants(tree, cond_idx, cond_logprob, topk_idx_seq, gamma, M, B):
    """Assert the structural properties every draft tree must have."""
    tok = np.asarray(tree["token"])
    par = np.asarray(tree["parent"])
    dep = np.asarray(tree["depth"])
    sc = np.asarray(tree["score"], dtype=np.float32)
    rank = np.asarray(tree["rank"]) if "rank" in tree else None
    lp = np.asarray(cond_logprob, dtype=np.float32)
    assert tok.shape == (B,), "tree must hold exactly B nodes besides the root"
    seen = set()
    keys = []
    for i in range(B):
        p = int(par[i])
        assert -1 <= p < i, "parent must precede its child"
        if p < 0:
            assert dep[i] == 1
            row = 0
            ps = np.float32(0.0)
        else:
            assert dep[i] == dep[p] + 1
            hits = np.nonzero(np.asarray(topk_idx_seq[dep[p] - 1]) == tok[p])[0]
            assert hits.size == 1, "inner nodes must be stage-1 candidates of their depth"
            row = 1 + (dep[p] - 1) * M + int(hits[0])
            ps = sc[p]
        assert 1 <= dep[i] <= gamma
        assert (p, int(tok[i])) not in seen, "duplicate child"
        seen.add((p, int(tok[i])))
        c = np.nonzero(np.asarray(cond_idx[row]) == tok[i])[0]
        assert c.size == 1
        c = int(c[0])
        if rank is not None:
            assert rank[i] == c
        assert np.float32(ps + lp[row, c]) == sc[i], "score must be the float32 path sum"
        keys.append((-float(sc[i]), int(dep[i])))
    for a, b in zip(keys, keys[1:]):
        assert a <= b, "pops must come in non-increasing candidate order"


def brute_force_marginal_tree(marg_idx, marg_logprob, gamma, B):
    """Every token path of length 1..gamma over the marginal rows (depth d uses
    row d-1), float32 left-to-right sums, sorted by the candidate order; the
    best B.  Independent of the oracle's heap."""
    marg_idx = np.asarray(marg_idx)
    lp = np.asarray(marg_logprob, dtype=np.float32)
    K = marg_idx.shape[1]
    found = []
    stack = [(1, np.float32(0.0), ())]
    while stack:
        dep, s_par, path = stack.pop()
        for c in range(K):
            s = np.float32(s_par + lp[dep - 1, c])
            p = path + (c,)
            found.append((_key(s, dep, p), s, int(marg_idx[dep - 1, c])))
            if dep < gamma:
                stack.append((dep + 1, s, p))
    if len(found) < B:
        raise ValueError("budget exceeds admissible nodes")
    found.sort(key=lambda t: t[0])
    top = found[:B]
    pos = {t[0][2]: i for i, t in enumerate(top)}
    out = {k: [] for k in ("token", "parent", "depth", "score", "rank")}
    for key, s, tok in top:
        path = key[2]
        out["token"].append(tok)
        out["parent"].append(pos[path[:-1]] if len(path) > 1 else -1)
        out["depth"].append(key[1])
        out["score"].append(s)
        out["rank"].append(path[-1])
    return {
        "token": np.asarray(out["token"], dtype=np.int32),
        "parent": np.asarray(out["parent"], dtype=np.int32),
        "depth": np.asarray(out["depth"], dtype=np.int32),
        "score": np.asarray(out["score"], dtype=np.float32),
        "rank": np.asarray(out["rank"], dtype=np.int32),
    }


def brute_force_tree_2prev(cond_idx, cond_logprob, topk_idx_seq, gamma, M, B, context=-2, root=-1):
    """Every admissible node of the bigram-conditioned tree, best B by the
    candidate order.  Rows are found by their (depth, token two back, previous
    token) key, enumerated here in the table's stated order: depth 1 is
    (context, root), depth 2 (root, candidate m of depth 1), depth i >= 3
    (candidate m2 of depth i-2, candidate m1 of depth i-1) with m1 fastest.
    ``context`` and ``root`` only need to differ from every candidate token."""
    cond_idx = np.asarray(cond_idx)
    lp = np.asarray(cond_logprob, dtype=np.float32)
    K = cond_idx.shape[1]
    cands = [list(np.asarray(topk_idx_seq[i]).tolist()) for i in range(gamma)]
    key_row = {}
    r = 0
    key_row[(1, context, root)] = r
    r += 1
    if gamma >= 2:
        for t1 in cands[0]:
            key_row[(2, root, t1)] = r
            r += 1
    for dep in range(3, gamma + 1):
        for t2 in cands[dep - 3]:
            for t1 in cands[dep - 2]:
                key_row[(dep, t2, t1)] = r
                r += 1
    found = []
    # (row, depth of the row's tokens, parent score, rank path, token two back, previous token)
    stack = [(0, 1, np.float32(0.0), (), context, root)]
    while stack:
        row, dep, s_par, path, t2, t1 = stack.pop()
        for c in range(K):
            s = np.float32(s_par + lp[row, c])
            p = path + (c,)
            tok = int(cond_idx[row, c])
            found.append((_key(s, dep, p), s, tok))
            nxt = key_row.get((dep + 1, t1, tok))
            if dep < gamma and nxt is not None and tok in cands[dep - 1]:
                stack.append((nxt, dep + 1, s, p, t1, tok))
    if len(found) < B:
        raise ValueError("budget exceeds admissible nodes")
    found.sort(key=lambda t: t[0])
    top = found[:B]
    pos = {t[0][2]: i for i, t in enumerate(top)}
    out = {k: [] for k in ("token", "parent", "depth", "score", "rank")}
    for key, s, tok in top:
        path = key[2]
        out["token"].append(tok)
        out["parent"].append(pos[path[:-1]] if len(path) > 1 else -1)
        out["depth"].append(key[1])
        out["score"].append(s)
        out["rank"].append(path[-1])
    res = {k: np.asarray(v, dtype=np.float32 if k == "score" else np.int32) for k, v in out.items()}
    res["admissible"] = len(found)
    return res
