"""GPU parity of OPT-Tree selection (Appendix B, Part 2) on rows built for it.

The tree kernels are fed seeded sorted rows whose log-probs are multiples of
1/8 with a leading entry near 0 and a decaying tail (so path sums are exact
in fp32 and exact score ties between siblings, cousins and different depths
are frequent; some rows carry -0.0), over a small vocabulary, with the
stage-1 candidates of every other sequence drawn from the leading tokens of
their depth's rows so that the trees run deep.  Each tree must equal the
oracle's field by field.

The budgets cover every launch shape: the lane-table kernel with one, two,
four and eight frontier slots per lane (each at both ends of its range;
peaked rows, whose trees run deep, and flat rows, whose star-shaped trees
are popped in sibling runs), with every row in LDS and with rows longer than
the LDS copy, the register frontier with sixteen slots, the LDS frontier,
the bigram rows of the w/ 2-prev approximator and the marginal rows.  Rows shorter than the budget whose expansions run out
leave the tail of the tree empty (token and parent -1, depth 0, score -inf).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03819_amd import binding
from parity import check_tree_exact, to_cpu_tree

pytestmark = pytest.mark.gpu


def sorted_rows(rng, R, K, vocab, base=0.0):
    """[R, K] rows: distinct tokens, log-probs -(base + q/8) sorted descending
    (ties by token).

    q starts at 0, 1 or 2 and grows by steps drawn from [0, s) with s in
    {2, 3, 5} per row: a leading entry near -base and a decaying tail, with
    runs of equal values.  base 0 gives peaked rows (deep trees); a base of a
    few units gives flat rows, whose children score below most of the root's
    row (star-shaped trees, popped in long sibling runs).
    """
    idx = np.stack([rng.choice(vocab, K, replace=False) for _ in range(R)]).astype(np.int32)
    steps = rng.integers(0, rng.choice([2, 3, 5], size=(R, 1)), size=(R, K))
    steps[:, 0] = rng.integers(0, 3, size=R)
    q = np.cumsum(steps, axis=1)
    lp = (-(base + q / 8.0)).astype(np.float32)
    if base == 0.0:
        lp[::2][q[::2] == 0] = np.float32(-0.0)
    for r in range(R):
        o = np.lexsort((idx[r], -lp[r].astype(np.float64)))
        idx[r], lp[r] = idx[r][o], lp[r][o]
    return idx, lp


def row_depth(mode, M, r):
    if r == 0:
        return 1
    if mode == "single":
        return 2 + (r - 1) // M
    return 2 if r <= M else 3 + (r - 1 - M) // (M * M)


def candidates(rng, mode, gamma, M, vocab, idx, lead):
    """[gamma, M] distinct candidates per depth.  With ``lead`` they are drawn
    from the three leading tokens of the rows at that depth (as stage-1
    candidates tend to head the conditional rows), which makes deep trees;
    otherwise from the whole vocabulary."""
    out = []
    for d in range(1, gamma + 1):
        pool = []
        if lead:
            for r in range(idx.shape[0]):
                if row_depth(mode, M, r) == d:
                    pool.extend(int(t) for t in idx[r, :3] if int(t) not in pool)
        pool = list(rng.permutation(pool))[:M]
        rest = [t for t in rng.permutation(vocab) if t not in pool]
        out.append(pool + rest[:M - len(pool)])
    return np.array(out, dtype=np.int32)


def rows_of(mode, gamma, M):
    if mode == "single":
        return 1 + (gamma - 1) * M
    return 1 if gamma == 1 else 1 + M + (gamma - 2) * M * M


def admissible(mode, idx, topk, gamma, M, limit):
    """Nodes the full best-first expansion can reach (counted up to ``limit``)."""
    count = 0
    stack = [(0, 1, -1)]   # (row, depth of its entries, parent's candidate index)
    while stack and count < limit:
        row, depth, mp = stack.pop()
        count += idx.shape[1]
        if depth >= gamma:
            continue
        for tok in idx[row]:
            hit = np.nonzero(topk[depth - 1] == tok)[0]
            if hit.size:
                m = int(hit[0])
                if mode == "single":
                    stack.append((1 + (depth - 1) * M + m, depth + 1, m))
                elif depth == 1:
                    stack.append((1 + m, 2, m))
                else:
                    stack.append((1 + M + (depth - 2) * M * M + mp * M + m, depth + 1, m))
    return min(count, limit)


def expect_tree(mode, idx, lp, topk, gamma, M, B):
    fn = oracle.build_tree if mode == "single" else oracle.build_tree_2prev
    n = admissible(mode, idx, topk, gamma, M, B)
    ref = fn(idx, lp, topk, gamma, M, n)
    pad = {"token": -1, "parent": -1, "depth": 0, "score": -np.inf, "child_row": -1}
    return {f: np.concatenate([np.asarray(ref[f]), np.full(B - n, v, dtype=np.asarray(ref[f]).dtype)])
            for f, v in pad.items()}


# (mode, gamma, M, K2, B, vocabulary, sequences, seed[, base])
ROW_CASES = [
    ("single", 4, 3, 8, 1, 12, 2, 1),
    ("single", 5, 4, 40, 37, 44, 3, 2),
    ("single", 6, 4, 63, 63, 66, 2, 3),
    ("single", 6, 4, 64, 64, 68, 2, 4),
    ("single", 5, 4, 127, 127, 130, 2, 5),
    ("single", 4, 3, 128, 128, 132, 2, 6),
    ("single", 4, 2, 255, 255, 260, 1, 7),
    ("single", 3, 2, 300, 300, 305, 1, 8),
    ("single", 3, 2, 511, 511, 515, 1, 9),
    ("single", 3, 2, 600, 600, 605, 1, 10),     # register frontier, 16 slots per lane
    ("single", 16, 16, 128, 100, 140, 1, 11),   # records do not fit: rows cached in LDS
    ("single", 3, 2, 1100, 1100, 1105, 1, 12),  # LDS frontier
    ("single", 2, 2, 4, 10, 9, 3, 13),          # rows shorter than the budget: expansions run out
    ("single", 16, 8, 32, 32, 36, 4, 14),       # the Qwen3 drafting shape's tree
    ("bigram", 4, 3, 40, 40, 44, 2, 15),
    ("bigram", 3, 4, 130, 130, 134, 1, 16),
    ("bigram", 2, 2, 4, 9, 8, 2, 17),
    # flat rows: star-shaped trees (sibling runs, stopped by children and ties)
    ("single", 16, 8, 32, 32, 36, 3, 18, 3.0),
    ("single", 16, 8, 32, 32, 36, 3, 19, 1.0),
    ("single", 5, 4, 100, 100, 104, 2, 20, 3.0),
    ("single", 4, 4, 127, 127, 131, 2, 21, 0.5),
    ("bigram", 4, 3, 60, 60, 64, 2, 22, 2.0),
    ("single", 3, 2, 200, 200, 204, 1, 23, 3.0),
    # rows longer than the LDS copy (ranks past it read from memory), deep and star-shaped
    ("single", 16, 8, 200, 200, 210, 1, 24),
    ("single", 16, 8, 300, 300, 304, 1, 25, 3.0),
    ("single", 16, 8, 511, 511, 520, 1, 26, 3.0),
    ("single", 16, 8, 512, 512, 520, 1, 27, 3.0),   # B = 64 * 8: the last pop's child slot is dropped
    ("single", 4, 3, 64, 64, 70, 2, 28, 0.5),       # B = 64 on one slot per lane
    ("single", 4, 3, 128, 128, 135, 2, 29, 1.0),
]


@pytest.mark.parametrize("case", ROW_CASES,
                         ids=[f"{c[0]}-g{c[1]}-M{c[2]}-K{c[3]}-B{c[4]}" + (f"-flat{c[8]}" if len(c) > 8 else "")
                              for c in ROW_CASES])
def test_tree_matches_oracle(case):
    mode, gamma, M, K2, B, vocab, b, seed = case[:8]
    base = case[8] if len(case) > 8 else 0.0
    print(f"[tree] {mode} gamma={gamma} M={M} K2={K2} B={B} b={b} seed={seed} base={base}", flush=True)
    rng = np.random.default_rng(seed)
    R = rows_of(mode, gamma, M)
    rows = [sorted_rows(rng, R, K2, vocab, base) for _ in range(b)]
    topk = np.stack([candidates(rng, mode, gamma, M, vocab, rows[s][0], s % 2 == 0) for s in range(b)])
    ci = torch.from_numpy(np.stack([r[0] for r in rows])).cuda()
    cl = torch.from_numpy(np.stack([r[1] for r in rows])).cuda()
    tk = torch.from_numpy(topk).cuda()
    fn = binding.treeflash_build_tree if mode == "single" else binding.treeflash_build_tree_2prev
    got = fn(ci, cl, tk, B)
    for s in range(b):
        ref = expect_tree(mode, rows[s][0], rows[s][1], topk[s], gamma, M, B)
        check_tree_exact(to_cpu_tree(got, s), ref, f"{mode} B={B} seq {s}")
    # the same buffers again: every output slot is rewritten
    got2 = fn(ci, cl, tk, B, out=got)
    for s in range(b):
        ref = expect_tree(mode, rows[s][0], rows[s][1], topk[s], gamma, M, B)
        check_tree_exact(to_cpu_tree(got2, s), ref, f"{mode} B={B} seq {s}, second call")


# (gamma, K, B, seed)
MARGINAL_CASES = [(5, 33, 33, 21), (1, 12, 12, 22), (3, 200, 200, 23), (4, 70, 70, 24), (2, 600, 600, 25)]


@pytest.mark.parametrize("gamma,K,B,seed", MARGINAL_CASES, ids=[f"g{c[0]}-K{c[1]}-B{c[2]}" for c in MARGINAL_CASES])
def test_marginal_tree_matches_oracle(gamma, K, B, seed):
    print(f"[tree] marginal gamma={gamma} K={K} B={B} seed={seed}", flush=True)
    rng = np.random.default_rng(seed)
    idx, lp = sorted_rows(rng, gamma, K, K + 5)
    got = binding.treeflash_build_tree_marginal(torch.from_numpy(idx[None]).cuda(),
                                                torch.from_numpy(lp[None]).cuda(), B)
    ref = oracle.build_marginal_tree(idx, lp, gamma, B)
    check_tree_exact(to_cpu_tree(got, 0), ref, f"marginal B={B}")
