"""Comparators between the HIP path and the CPU oracle.

* ``check_topk``: a GPU top-k list passes when its ids are distinct, the
  oracle value of the GPU id at position j is within tol of the oracle's own
  j-th best value, and the GPU value is within tol of the oracle value of the
  same id.  This forces equal ids wherever the oracle's neighbouring values
  are more than tol apart, and admits any order inside a cluster of near-ties.
* ``check_tree_exact``: the tree kernel fed the oracle's rows must reproduce
  the oracle tree bit for bit.
* ``replay_tree``: end to end, every GPU pop must be an admissible candidate
  whose oracle path score is within tol of the best admissible oracle score,
  and whose GPU score is within tol of its oracle score.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2606_03819_amd import synth

# One line per checked workload (worst errors, end-to-end count), printed by
# the test session's terminal summary so that a quiet run still shows them.
SUMMARY = []


def np64(t):
    return synth.to_numpy64(t)


def oracle_inputs(inputs):
    """float64/int64 numpy copies of every input tensor."""
    return {k: np64(v) for k, v in inputs.items()}


def topk_values_sorted(full: np.ndarray, k: int) -> np.ndarray:
    """The k largest values of each row, descending."""
    V = full.shape[-1]
    part = np.partition(full, V - k, axis=-1)[..., V - k:]
    return -np.sort(-part, axis=-1)


def check_topk(gpu_idx, gpu_val, oracle_full, tol, what=""):
    """P1 comparator; gpu_idx/gpu_val [n, k], oracle_full [n, V] in the same units."""
    gpu_idx = np.asarray(gpu_idx).reshape(-1, np.asarray(gpu_idx).shape[-1]).astype(np.int64)
    gpu_val = np.asarray(gpu_val, dtype=np.float64).reshape(gpu_idx.shape)
    full = np.asarray(oracle_full, dtype=np.float64).reshape(gpu_idx.shape[0], -1)
    n, k = gpu_idx.shape
    V = full.shape[1]
    assert np.all((gpu_idx >= 0) & (gpu_idx < V)), f"{what}: ids out of range"
    for r in range(n):
        assert len(set(gpu_idx[r].tolist())) == k, f"{what}: duplicate ids in row {r}"
    ref = topk_values_sorted(full, k)
    o_of_gpu = np.take_along_axis(full, gpu_idx, axis=1)
    err_rank = np.abs(o_of_gpu - ref)
    err_val = np.abs(gpu_val - o_of_gpu)
    worst_rank = float(err_rank.max())
    worst_val = float(err_val.max())
    assert worst_rank <= tol, f"{what}: GPU list departs from the oracle order by {worst_rank:.3g} > {tol}"
    assert worst_val <= tol, f"{what}: GPU values differ from the oracle by {worst_val:.3g} > {tol}"
    return {"max_rank_err": worst_rank, "max_val_err": worst_val,
            "exact_ids": float(np.mean(gpu_idx == np.argsort(-full, axis=1, kind="stable")[:, :k]))}


def check_tree_exact(gpu_tree, ref_tree, what=""):
    for f in ("token", "parent", "depth", "score", "child_row"):
        g = np.asarray(gpu_tree[f])
        o = np.asarray(ref_tree[f])
        assert np.array_equal(g, o), f"{what}: tree field {f} differs\nGPU {g}\noracle {o}"


def replay_tree(gpu_tree, row_lp, topk_seq, gamma, M, B, tol, what="", bigram=False):
    """End-to-end tree check against oracle rows.

    gpu_tree: dict of numpy arrays for one sequence; row_lp: dict row -> full
    oracle log-prob row (float64, length V) for every row the replay needs;
    topk_seq: [gamma, M] stage-1 candidates the rows were conditioned on.
    bigram: the rows are the w/ 2-prev table (a node's row depends on its own
    and its parent's candidate index).
    """
    tok = np.asarray(gpu_tree["token"])
    par = np.asarray(gpu_tree["parent"])
    dep = np.asarray(gpu_tree["depth"])
    gsc = np.asarray(gpu_tree["score"], dtype=np.float64)
    osc = np.zeros(B)
    children = {-1: set()}
    rowof = {-1: 0}
    slot = {-1: -1}
    order = {}
    worst = 0.0

    def best_child(p):
        lp = row_lp[rowof[p]]
        if p not in order:
            order[p] = np.argsort(-lp, kind="stable")
        for t in order[p]:
            if int(t) not in children[p]:
                return (osc[p] if p >= 0 else 0.0) + lp[t]
        return -np.inf

    for j in range(B):
        p = int(par[j])
        assert -1 <= p < j, f"{what}: node {j} has parent {p}"
        assert p in rowof, f"{what}: node {j} hangs below a node that is not expandable"
        assert dep[j] == (1 if p < 0 else dep[p] + 1), f"{what}: node {j} depth"
        assert int(tok[j]) not in children[p], f"{what}: node {j} duplicates a sibling"
        best = max(best_child(q) for q in rowof)
        lp = row_lp[rowof[p]]
        osc[j] = (osc[p] if p >= 0 else 0.0) + lp[int(tok[j])]
        gap = best - osc[j]
        worst = max(worst, gap, abs(gsc[j] - osc[j]))
        assert gap <= tol, f"{what}: pop {j} is {gap:.3g} below the best admissible candidate"
        assert abs(gsc[j] - osc[j]) <= tol, f"{what}: pop {j} score {gsc[j]} vs oracle {osc[j]}"
        children[p].add(int(tok[j]))
        children[j] = set()
        hits = np.nonzero(np.asarray(topk_seq[dep[j] - 1]) == tok[j])[0]
        slot[j] = int(hits[0]) if hits.size else -1
        if dep[j] < gamma:
            if hits.size:
                if not bigram:
                    rowof[j] = 1 + (dep[j] - 1) * M + slot[j]
                elif dep[j] == 1:
                    rowof[j] = 1 + slot[j]
                else:
                    rowof[j] = 1 + M + (dep[j] - 2) * M * M + slot[p] * M + slot[j]
                assert int(gpu_tree["child_row"][j]) == rowof[j], f"{what}: node {j} child_row"
            else:
                assert int(gpu_tree["child_row"][j]) == -1
        else:
            assert int(gpu_tree["child_row"][j]) == -1
    return worst


def rows_needed(gpu_tree, B):
    """Rows whose entries appear in the tree (the root row and expanded nodes' rows)."""
    need = {0}
    for j in range(B):
        c = int(gpu_tree["child_row"][j])
        if c >= 0:
            need.add(c)
    return sorted(need)


def to_cpu_tree(tree, s):
    return {k: v[s].cpu().numpy() for k, v in tree.items()}


def _oracle_rows(o_in, w, topk_seq, s):
    if w.approximator == "2prev":
        depth, _, _ = oracle.row_table_2prev(w.gamma, w.k)
        p1, p2 = oracle.previous_pairs(int(o_in["context"][s]), int(o_in["root"][s]), topk_seq, w.gamma, w.k)
        hp = oracle.ar_approximator_2prev(o_in["h"][s], p1, p2, depth, o_in["emb"], o_in["norm_h_gain"],
                                          o_in["norm_e_gain"], o_in["w_gate"], o_in["w_up"], o_in["w_down"],
                                          mirror_bf16=(w.dtype == "bf16"))
        return oracle.conditional_stage(hp, o_in["lm_head"], w.topk2, w.inv_temperature, keep_full=True)
    depth, _ = oracle.row_table(w.gamma, w.k)
    prev = oracle.previous_tokens(int(o_in["root"][s]), topk_seq, w.gamma, w.k)
    if "w_lin" in o_in:
        hp = oracle.ar_approximator_linear(o_in["h"][s], prev, depth, o_in["emb"], o_in["norm_h_gain"],
                                           o_in["norm_e_gain"], o_in["w_lin"], mirror_bf16=(w.dtype == "bf16"))
    else:
        hp = oracle.ar_approximator(o_in["h"][s], prev, depth, o_in["emb"], o_in["norm_h_gain"],
                                    o_in["norm_e_gain"], o_in["w_gate"], o_in.get("w_up"), o_in["w_down"],
                                    mirror_bf16=(w.dtype == "bf16"))
    return oracle.conditional_stage(hp, o_in["lm_head"], w.topk2, w.inv_temperature, keep_full=True)


def _row_permutation(gpu_topk, o_topk, gamma, M, bigram):
    """rmap with GPU-chain row r == teacher-forced row rmap[r], or None.

    Rows of depth i >= 2 are conditioned on candidate m of depth i-1; when the
    GPU's candidates of depths 1..gamma-1 are the oracle's up to order, row
    1 + (i-2)M + m_gpu is the forced row 1 + (i-2)M + m_oracle of the same
    token.  The bigram rows need the identical lists.
    """
    if bigram:
        return np.arange(int(cond_rows(gamma, M, True))) if np.array_equal(gpu_topk, o_topk) else None
    R = 1 + (gamma - 1) * M
    rmap = np.arange(R)
    for i in range(gamma - 1):
        g_ids, o_ids = list(gpu_topk[i]), list(o_topk[i])
        if sorted(g_ids) != sorted(o_ids):
            return None
        for m, t in enumerate(g_ids):
            rmap[1 + i * M + m] = 1 + i * M + o_ids.index(t)
    return rmap


def cond_rows(gamma, M, bigram):
    if not bigram:
        return 1 + (gamma - 1) * M
    return 1 if gamma == 1 else 1 + M + (gamma - 2) * M * M


def check_draft(w, g, o_in, seqs, tol, log=print, require_e2e=False):
    """Whole-path parity for the sequences ``seqs`` of workload ``w``.

    g: GPU input tensors; o_in: float64 numpy copies of the same inputs.
    1. stage 1 (GPU) against the oracle's marginal rows;
    2. stage 2 and the tree on the GPU, fed the oracle's stage-1 candidates,
       against the oracle's conditional rows (top-k lists, log-sum-exp, tree
       replay);
    3. the tree kernel fed the oracle's own rows reproduces the oracle tree
       bit for bit;
    4. the GPU's own end-to-end step equals the teacher-forced GPU outputs
       (rows permuted when its stage-1 lists order a near-tie differently)
       whenever its stage-1 candidates are the oracle's (else a candidate sits
       on a stage-1 near-tie at the list boundary and only steps 1-3 apply).  With
       ``require_e2e`` at least one sequence must take this leg.
    The oracle never consumes a HIP-path output.
    """
    from paper_2606_03819_amd import binding
    bigram = w.approximator == "2prev"
    if bigram:
        dr = binding.Drafter2Prev(g, w.b, w.gamma, w.k, w.B, w.inv_temperature)
        dr.context = g["context"]
        gpu_tree_fn, oracle_tree_fn = binding.treeflash_build_tree_2prev, oracle.build_tree_2prev
    else:
        dr = binding.Drafter(g, w.b, w.gamma, w.k, w.B, w.inv_temperature)
        gpu_tree_fn, oracle_tree_fn = binding.treeflash_build_tree, oracle.build_tree
    idx1, lp1 = dr.stage1(g["h"])
    gpu_topk = idx1.cpu().numpy()
    gpu_lp1 = lp1.cpu().numpy()
    o_topk = np.zeros_like(gpu_topk)
    stats = {}
    for s in seqs:
        st1 = oracle.marginal_stage(o_in["h"][s:s + 1], o_in["lm_head"], w.k, w.inv_temperature)
        r = check_topk(gpu_topk[s], gpu_lp1[s], st1["logprob"][0], tol, f"{w.name} stage 1 seq {s}")
        stats[f"stage1_seq{s}"] = r
        o_topk[s] = st1["topk_idx"][0]
    # teacher forcing: the oracle's candidates for the sampled sequences (the
    # others keep the GPU's, they are not checked)
    forced = gpu_topk.copy()
    forced[list(seqs)] = o_topk[list(seqs)]
    forced_t = torch.from_numpy(forced).to(torch.int32).cuda()
    ci, cl, lse = dr.stage2(g["h"], g["root"], topk_idx=forced_t)
    tree_tf = dr.tree_build(topk_idx=forced_t)
    ci, cl, lse = ci.cpu().numpy(), cl.cpu().numpy(), lse.cpu().numpy()
    tree_tf = {k: v.cpu().numpy() for k, v in tree_tf.items()}
    for s in seqs:
        rows = _oracle_rows(o_in, w, o_topk[s], s)
        stats[f"stage2_seq{s}"] = check_topk(ci[s], cl[s], rows["logprob"], tol, f"{w.name} stage 2 seq {s}")
        lse_err = float(np.max(np.abs(lse[s] - rows["cond_lse"])))
        assert lse_err <= tol, f"{w.name}: log-sum-exp off by {lse_err}"
        t = {k: v[s] for k, v in tree_tf.items()}
        rl = {r: rows["logprob"][r] for r in rows_needed(t, w.B)}
        stats[f"tree_replay_seq{s}"] = replay_tree(t, rl, o_topk[s], w.gamma, w.k, w.B, tol, f"{w.name} tree seq {s}",
                                                   bigram=bigram)
        gt = gpu_tree_fn(torch.from_numpy(rows["cond_idx"][None]).cuda(),
                         torch.from_numpy(rows["cond_logprob"][None]).cuda(),
                         torch.from_numpy(o_topk[s][None]).to(torch.int32).cuda(), w.B)
        ref = oracle_tree_fn(rows["cond_idx"], rows["cond_logprob"], o_topk[s], w.gamma, w.k, w.B)
        check_tree_exact(to_cpu_tree(gt, 0), ref, f"{w.name} tree kernel seq {s}")
    # end to end: a conditional row depends only on its (depth, previous
    # token) pair, so when the GPU's own stage-1 lists hold the oracle's
    # candidates at every depth that conditions a row (in any order inside a
    # near-tie), its own chain must reproduce the teacher-forced outputs with
    # the rows permuted accordingly
    full = {k: v.clone() for k, v in dr.step(g["h"], g["root"]).items()}
    full = {k: v.cpu().numpy() for k, v in full.items()}
    e2e_ci, e2e_cl = dr.cond_idx.cpu().numpy(), dr.cond_lp.cpu().numpy()
    same = 0
    for s in seqs:
        rmap = _row_permutation(gpu_topk[s], o_topk[s], w.gamma, w.k, bigram)
        if rmap is None:
            continue
        same += 1
        assert np.array_equal(e2e_ci[s], ci[s][rmap]) and np.array_equal(e2e_cl[s], cl[s][rmap]), \
            f"{w.name}: e2e stage-2 rows of seq {s}"
        for k in ("token", "parent", "depth", "score"):
            assert np.array_equal(full[k][s], tree_tf[k][s]), f"{w.name}: e2e tree {k} of seq {s}"
        inv = np.empty_like(rmap)
        inv[rmap] = np.arange(rmap.size)
        cr_f = tree_tf["child_row"][s]
        want = np.where(cr_f >= 0, inv[np.maximum(cr_f, 0)], -1)
        assert np.array_equal(full["child_row"][s], want), f"{w.name}: e2e child rows of seq {s}"
    stats["e2e_sequences_equal_to_forced"] = same
    log(f"[parity] {w.name}: {stats}")
    worst = {
        "stage1": max(v["max_rank_err"] for k, v in stats.items() if k.startswith("stage1")),
        "stage1_val": max(v["max_val_err"] for k, v in stats.items() if k.startswith("stage1")),
        "stage2": max(v["max_rank_err"] for k, v in stats.items() if k.startswith("stage2")),
        "stage2_val": max(v["max_val_err"] for k, v in stats.items() if k.startswith("stage2")),
        "tree": max(v for k, v in stats.items() if k.startswith("tree_replay")),
    }
    SUMMARY.append(f"{w.name}: {len(list(seqs))} seq(s) checked, worst |err| stage-1 rank {worst['stage1']:.2e} "
                   f"value {worst['stage1_val']:.2e}, stage-2 rank {worst['stage2']:.2e} value "
                   f"{worst['stage2_val']:.2e}, tree score {worst['tree']:.2e}; end-to-end equal on {same} "
                   f"of {len(list(seqs))}")
    if require_e2e:
        assert same >= 1, (f"{w.name}: no checked sequence took the end-to-end leg (every one sits on a "
                           f"stage-1 near-tie)")
    return stats
