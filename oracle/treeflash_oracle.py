"""Plain CPU oracle of TreeFlash drafting (arXiv 2606.03819).

TEST INFRASTRUCTURE ONLY.  This module is imported by the tests, by the smoke
check of the entry module and by the CPU-baseline leg of the benchmark.  The
HIP library never imports, links or calls it, and it shares no code with the
library: it uses nothing but NumPy and the Python standard library.

What it computes (paper: Method section, "AR-Approximation", Eq. 1, and
Appendix B, the "AR-approximated OPT-Tree Construction" algorithm):

Part 1 -- AR-approximated distributions
  * stage 1: ``q_{t+i} = LMHead(h_{t+i})`` for every draft depth i, and the
    top-M candidate tokens of each depth;
  * one conditional row per (depth, previous token) pair of the M-ary tree:
    depth 1 is conditioned on the root token x_t, depth i >= 2 on each of the
    M candidates of depth i-1 (so 1 + (gamma-1)*M rows per sequence);
  * Eq. 1: ``h' = h + SwiGLU(norm(h) :: norm(Embd(prev)))`` followed by the
    LM head and a log-softmax over the whole vocabulary.
Part 2 -- OPT-Tree selection
  * best-first pops of the candidate with the highest path probability until
    the tree holds B nodes besides the root; a popped node contributes its
    children only when its token is one of the M candidates of its depth.
Verification hand-off (Method, "Inference": equality-check verification;
Experiments, "Metrics": block efficiency)
  * the tree laid out for a verifier pass with tree attention (root first,
    positions = depths, ancestor mask) and the greedy acceptance walk that
    turns the verifier's per-node next tokens into accepted nodes and tau.
The w/ Linear and w/ 2-prev ablations (Ablations, Model Design)
  * one linear layer in place of the SwiGLU of Eq. 1;
  * the previous bigram instead of one previous token: 1 + M + (gamma-2)*M^2
    conditional rows, and a tree whose nodes expand into the row of their
    (parent token, own token) pair.
Marginal baseline (the paper's DDTree comparison, Related Work and Appendix C)
  * the same selection on the marginal distributions alone: every node above
    the last depth expands into the marginal row of the next depth, so all
    paths share one child ranking (a nested tree).

Arithmetic is float64 throughout, with the following readings where the paper
is silent (each is listed in the design doc):
  * "normalized" is RMSNorm with its own gain, eps = 1e-6;
  * SwiGLU(x) = W_down (silu(W_gate x) * (W_up x)), no biases, x = [h~ ; e~];
    without W_up, the plain two-layer SiLU MLP W_down silu(W_gate x) on the
    same input and residual (a side mode);
  * the LM head is a plain product with the [V, d] output embedding; logits are
    multiplied by the inverse drafter temperature before the softmax;
  * for bf16 workloads the oracle rounds to bf16 exactly where a bf16 operand
    is formed for a matrix product: x and h' ("mirror" rounding points); the
    SwiGLU activation a enters the down projection as a bf16 hi/lo pair, about
    16 significant bits, which float64 stands in for; all else stays float64;
  * path scores are float32 running sums of float32 row log-probabilities, so
    a tree is reproducible bit for bit from the same rows;
  * ties: top-k lists order by (value desc, token asc); tree candidates order by
    (score desc, depth asc, rank path lexicographic asc), where the rank path
    lists each node's position in its parent's sorted row, root to node.
"""
from __future__ import annotations

import heapq
from typing import Dict, List, Optional, Tuple

import numpy as np

__all__ = [
    "bf16_round", "rms_norm", "silu", "log_softmax", "topk_sorted",
    "marginal_stage", "row_table", "previous_tokens", "ar_approximator",
    "conditional_stage", "build_tree", "draft", "build_marginal_tree", "draft_marginal",
    "verification_inputs", "acceptance_walk", "ar_approximator_linear", "RMS_EPS",
    "row_table_2prev", "previous_pairs", "ar_approximator_2prev", "build_tree_2prev", "draft_2prev",
]

RMS_EPS = 1e-6


# ---------------------------------------------------------------- elementwise

def bf16_round(x) -> np.ndarray:
    """Round to the nearest bfloat16 value, ties to even.

    bfloat16 keeps 8 significant bits.  Writing x = f * 2**e with
    0.5 <= |f| < 1, the rounded value is round_half_even(f * 2**8) * 2**(e-8).
    Valid for the normal bfloat16 range (|x| >= 2**-126) and for zero.
    """
    x = np.asarray(x, dtype=np.float64)
    f, e = np.frexp(x)
    return np.ldexp(np.round(np.ldexp(f, 8)), e - 8)


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    """x / sqrt(mean(x**2) + eps) * gain over the last axis (Method, Eq. 1)."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype=np.float64)


def silu(g: np.ndarray) -> np.ndarray:
    """SiLU(g) = g * sigmoid(g) = g / (1 + exp(-g))."""
    g = np.asarray(g, dtype=np.float64)
    return g / (1.0 + np.exp(-g))


def log_softmax(z: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Log-softmax over the last axis; returns (log-probs, log-sum-exp)."""
    z = np.asarray(z, dtype=np.float64)
    m = np.max(z, axis=-1, keepdims=True)
    lse = m + np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True))
    return z - lse, lse[..., 0]


def topk_sorted(values: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest entries per row, ordered (value desc, index asc).

    A stable sort of the negated values keeps equal values in ascending index
    order, which is the tie rule.
    """
    order = np.argsort(-np.asarray(values, dtype=np.float64), axis=-1, kind="stable")
    return order[..., :k]


# ------------------------------------------------------------------- Part 1

def marginal_stage(h: np.ndarray, lm_head: np.ndarray, k: int,
                   inv_temperature: float = 1.0) -> Dict[str, np.ndarray]:
    """Stage 1 (Appendix B, Part 1, first loop): LM head on every depth, top-M.

    h: [b, gamma, d]; lm_head: [V, d] (row v is the output embedding of v).
    Returns logits z [b, gamma, V] (temperature applied), log-probs, the top-k
    ids [b, gamma, k] and their log-probs.
    """
    h = np.asarray(h, dtype=np.float64)
    w = np.asarray(lm_head, dtype=np.float64)
    z = inv_temperature * np.matmul(h, w.T)
    lp, lse = log_softmax(z)
    idx = topk_sorted(z, k)
    return {
        "logits": z,
        "logprob": lp,
        "lse": lse,
        "topk_idx": idx.astype(np.int32),
        "topk_logprob": np.take_along_axis(lp, idx, axis=-1),
    }


def row_table(gamma: int, M: int) -> Tuple[np.ndarray, np.ndarray]:
    """Rows of the conditional table (Appendix B, Part 1, second block).

    Row 0 is depth 1 conditioned on the root token.  For depth i = 2..gamma and
    candidate m = 0..M-1 the row is 1 + (i-2)*M + m, conditioned on the m-th
    candidate of depth i-1.  Returns (depth [R], candidate slot [R]; -1 = root).
    """
    depth = [1]
    slot = [-1]
    for i in range(2, gamma + 1):
        for m in range(M):
            depth.append(i)
            slot.append(m)
    return np.asarray(depth, dtype=np.int64), np.asarray(slot, dtype=np.int64)


def previous_tokens(root: int, topk_idx_seq: np.ndarray, gamma: int, M: int) -> np.ndarray:
    """Token each conditional row is conditioned on (the previous token)."""
    depth, slot = row_table(gamma, M)
    prev = np.empty(depth.shape[0], dtype=np.int64)
    for r in range(depth.shape[0]):
        if slot[r] < 0:
            prev[r] = int(root)
        else:
            # candidate slot[r] of depth depth[r]-1 (1-based) = index depth[r]-2
            prev[r] = int(topk_idx_seq[depth[r] - 2, slot[r]])
    return prev


def ar_approximator(h_seq: np.ndarray, prev: np.ndarray, depth: np.ndarray,
                    emb: np.ndarray, norm_h_gain: np.ndarray, norm_e_gain: np.ndarray,
                    w_gate: np.ndarray, w_up: Optional[np.ndarray], w_down: np.ndarray,
                    eps: float = RMS_EPS, mirror_bf16: bool = False) -> np.ndarray:
    """Eq. 1 for every conditional row of one sequence.

    h_seq: [gamma, d] drafter states; prev/depth: [R] from row_table.
    h'_r = h_{depth_r} + W_down( silu(W_gate x_r) * (W_up x_r) ),
    x_r = [ rms(h_{depth_r}) ; rms(Embd(prev_r)) ].
    With w_up None the gate is dropped: the plain two-layer SiLU MLP
    h'_r = h_{depth_r} + W_down silu(W_gate x_r) on the same input and
    residual (a side mode; Eq. 1 names the gated form).
    With mirror_bf16, x and h' are rounded to bf16 (the activation is not).
    """
    hd = np.asarray(h_seq, dtype=np.float64)[np.asarray(depth) - 1]
    e = np.asarray(emb, dtype=np.float64)[np.asarray(prev)]
    x = np.concatenate([rms_norm(hd, norm_h_gain, eps), rms_norm(e, norm_e_gain, eps)], axis=-1)
    if mirror_bf16:
        x = bf16_round(x)
    g = x @ np.asarray(w_gate, dtype=np.float64).T
    a = silu(g)
    if w_up is not None:
        a = a * (x @ np.asarray(w_up, dtype=np.float64).T)
    hp = hd + a @ np.asarray(w_down, dtype=np.float64).T
    if mirror_bf16:
        hp = bf16_round(hp)
    return hp


def ar_approximator_linear(h_seq: np.ndarray, prev: np.ndarray, depth: np.ndarray,
                           emb: np.ndarray, norm_h_gain: np.ndarray, norm_e_gain: np.ndarray,
                           w_lin: np.ndarray, eps: float = RMS_EPS, mirror_bf16: bool = False) -> np.ndarray:
    """The paper's "w/ Linear" ablation (Ablations, Model Design): the SwiGLU of
    Eq. 1 replaced by one linear layer on the same normalised input,
    h'_r = h_{depth_r} + W_lin x_r, x_r = [ rms(h_{depth_r}) ; rms(Embd(prev_r)) ],
    W_lin [d, 2d] with no bias; its e-half is the previous-token-conditioned
    shift the paper describes.  With mirror_bf16, x and h' are rounded to bf16.
    """
    hd = np.asarray(h_seq, dtype=np.float64)[np.asarray(depth) - 1]
    e = np.asarray(emb, dtype=np.float64)[np.asarray(prev)]
    x = np.concatenate([rms_norm(hd, norm_h_gain, eps), rms_norm(e, norm_e_gain, eps)], axis=-1)
    if mirror_bf16:
        x = bf16_round(x)
    hp = hd + x @ np.asarray(w_lin, dtype=np.float64).T
    if mirror_bf16:
        hp = bf16_round(hp)
    return hp


def conditional_stage(hp: np.ndarray, lm_head: np.ndarray, topk2: int,
                      inv_temperature: float = 1.0, keep_full: bool = False
                      ) -> Dict[str, np.ndarray]:
    """LM head + log-softmax on every conditional row (Appendix B, Part 1).

    hp: [..., R, d].  Keeps the top-topk2 entries of each row in (log-prob
    desc, token asc) order; log-probs are handed on as float32, the precision
    of the tree's path sums.  Each full row must sum to one.
    """
    z = inv_temperature * np.matmul(np.asarray(hp, dtype=np.float64),
                                    np.asarray(lm_head, dtype=np.float64).T)
    lp, lse = log_softmax(z)
    total = np.sum(np.exp(lp), axis=-1)
    if not np.all(np.abs(total - 1.0) < 1e-12):
        raise AssertionError("conditional row does not sum to one")
    idx = topk_sorted(lp, topk2)
    out = {
        "cond_idx": idx.astype(np.int32),
        "cond_logprob": np.take_along_axis(lp, idx, axis=-1).astype(np.float32),
        "cond_lse": lse,
    }
    if keep_full:
        out["logprob"] = lp
    return out


# ------------------------------------------------------------------- Part 2

def build_tree(cond_idx: np.ndarray, cond_logprob: np.ndarray, topk_idx_seq: np.ndarray,
               gamma: int, M: int, B: int) -> Dict[str, np.ndarray]:
    """OPT-Tree selection for one sequence (Appendix B, Part 2).

    cond_idx / cond_logprob: [R, K] rows sorted (log-prob desc, token asc);
    K is the full vocabulary or any K >= B (the truncated rows give the same
    tree).  topk_idx_seq: [gamma, M] stage-1 candidates.

    The queue starts with every child of the root (row 0).  Each pop appends
    the best candidate to the tree; when the popped token is candidate m of its
    depth and the depth is below gamma, every entry of row 1+(depth-1)*M+m is
    queued as its child.  Pops stop when the tree holds B nodes besides the
    root.  Returns per node, in pop order: token, parent (-1 = root), depth,
    score (float32 path log-probability), child_row (-1 if not expandable)
    and rank (position in the parent's row).
    """
    cond_idx = np.asarray(cond_idx)
    lp32 = np.asarray(cond_logprob, dtype=np.float32)
    K = cond_idx.shape[1]
    heap: List[tuple] = []

    def push_row(row: int, parent: int, parent_score: np.float32, depth: int, path: tuple):
        for c in range(K):
            s = np.float32(parent_score + lp32[row, c])        # float32 add
            heapq.heappush(heap, (-float(s), depth, path + (c,), parent, row, c))

    push_row(0, -1, np.float32(0.0), 1, ())
    token, parent, depth_o, score, child_row, rank = [], [], [], [], [], []
    while len(token) < B:
        if not heap:
            raise ValueError("draft budget exceeds the number of admissible nodes")
        negs, dep, path, par, row, c = heapq.heappop(heap)
        tok = int(cond_idx[row, c])
        crow = -1
        if dep < gamma:
            hits = np.nonzero(np.asarray(topk_idx_seq[dep - 1]) == tok)[0]
            if hits.size:
                crow = 1 + (dep - 1) * M + int(hits[0])
        token.append(tok)
        parent.append(par)
        depth_o.append(dep)
        score.append(np.float32(-negs))
        child_row.append(crow)
        rank.append(c)
        if crow >= 0:
            push_row(crow, len(token) - 1, np.float32(-negs), dep + 1, path)
    return {
        "token": np.asarray(token, dtype=np.int32),
        "parent": np.asarray(parent, dtype=np.int32),
        "depth": np.asarray(depth_o, dtype=np.int32),
        "score": np.asarray(score, dtype=np.float32),
        "child_row": np.asarray(child_row, dtype=np.int32),
        "rank": np.asarray(rank, dtype=np.int32),
    }


def build_marginal_tree(marg_idx: np.ndarray, marg_logprob: np.ndarray, gamma: int,
                        B: int) -> Dict[str, np.ndarray]:
    """OPT-Tree selection on the marginal distributions (the DDTree baseline).

    marg_idx / marg_logprob: [gamma, K] stage-1 rows sorted (log-prob desc,
    token asc), row i-1 being depth i; K >= min(B, V) gives the tree of full
    rows.  Every node of depth d < gamma takes its children from row d (the
    marginal of depth d+1), whatever its token; the root's children come from
    row 0.  Pops, scores (float32 running sums) and ties follow build_tree.
    Returns the same fields as build_tree; child_row is the row a node expands
    into (-1 at depth gamma).
    """
    marg_idx = np.asarray(marg_idx)
    lp32 = np.asarray(marg_logprob, dtype=np.float32)
    K = marg_idx.shape[1]
    heap: List[tuple] = []

    def push_row(row: int, parent: int, parent_score: np.float32, depth: int, path: tuple):
        for c in range(K):
            s = np.float32(parent_score + lp32[row, c])        # float32 add
            heapq.heappush(heap, (-float(s), depth, path + (c,), parent, row, c))

    push_row(0, -1, np.float32(0.0), 1, ())
    token, parent, depth_o, score, child_row, rank = [], [], [], [], [], []
    while len(token) < B:
        if not heap:
            raise ValueError("draft budget exceeds the number of admissible nodes")
        negs, dep, path, par, row, c = heapq.heappop(heap)
        crow = dep if dep < gamma else -1
        token.append(int(marg_idx[row, c]))
        parent.append(par)
        depth_o.append(dep)
        score.append(np.float32(-negs))
        child_row.append(crow)
        rank.append(c)
        if crow >= 0:
            push_row(crow, len(token) - 1, np.float32(-negs), dep + 1, path)
    return {
        "token": np.asarray(token, dtype=np.int32),
        "parent": np.asarray(parent, dtype=np.int32),
        "depth": np.asarray(depth_o, dtype=np.int32),
        "score": np.asarray(score, dtype=np.float32),
        "child_row": np.asarray(child_row, dtype=np.int32),
        "rank": np.asarray(rank, dtype=np.int32),
    }


# ------------------------------------------------------------- whole step

def draft(inputs: Dict[str, np.ndarray], gamma: int, k: int, B: int,
          inv_temperature: float = 1.0, mirror_bf16: bool = False,
          topk2: Optional[int] = None, eps: float = RMS_EPS,
          keep_full: bool = False, sequences: Optional[List[int]] = None
          ) -> Dict[str, object]:
    """One drafting step for every sequence: Part 1 then Part 2.

    ``inputs`` holds float64/int64 numpy arrays: h [b, gamma, d], root [b],
    lm_head, emb, norm_h_gain, norm_e_gain, w_gate, w_up, w_down (or w_lin
    for the w/ Linear ablation, which then replaces Eq. 1's SwiGLU; without
    w_up the plain SiLU MLP).
    ``sequences`` restricts the work to a subset of the batch (the sequences
    are independent).
    """
    h = inputs["h"]
    b = h.shape[0]
    V = inputs["lm_head"].shape[0]
    K2 = min(B, V) if topk2 is None else topk2
    seqs = list(range(b)) if sequences is None else list(sequences)
    depth, _ = row_table(gamma, k)
    out = {"stage1": [], "rows": [], "hprime": [], "tree": [], "prev": []}
    for s in seqs:
        st1 = marginal_stage(h[s:s + 1], inputs["lm_head"], k, inv_temperature)
        st1 = {key: val[0] for key, val in st1.items()}
        prev = previous_tokens(int(inputs["root"][s]), st1["topk_idx"], gamma, k)
        if "w_lin" in inputs:
            hp = ar_approximator_linear(h[s], prev, depth, inputs["emb"], inputs["norm_h_gain"],
                                        inputs["norm_e_gain"], inputs["w_lin"], eps=eps,
                                        mirror_bf16=mirror_bf16)
        else:
            hp = ar_approximator(h[s], prev, depth, inputs["emb"], inputs["norm_h_gain"],
                                 inputs["norm_e_gain"], inputs["w_gate"], inputs.get("w_up"),
                                 inputs["w_down"], eps=eps, mirror_bf16=mirror_bf16)
        rows = conditional_stage(hp, inputs["lm_head"], K2, inv_temperature, keep_full=keep_full)
        tree = build_tree(rows["cond_idx"], rows["cond_logprob"], st1["topk_idx"], gamma, k, B)
        if not keep_full:
            st1.pop("logits")
            st1.pop("logprob")
        out["stage1"].append(st1)
        out["rows"].append(rows)
        out["hprime"].append(hp)
        out["tree"].append(tree)
        out["prev"].append(prev)
    return out


def draft_marginal(inputs: Dict[str, np.ndarray], gamma: int, B: int, inv_temperature: float = 1.0,
                   K: Optional[int] = None, sequences: Optional[List[int]] = None) -> Dict[str, object]:
    """The marginal baseline for every sequence: stage 1 with K = min(B, V)
    entries per depth, then build_marginal_tree."""
    h = inputs["h"]
    V = inputs["lm_head"].shape[0]
    K = min(B, V) if K is None else K
    seqs = list(range(h.shape[0])) if sequences is None else list(sequences)
    out = {"stage1": [], "tree": []}
    for s in seqs:
        st1 = marginal_stage(h[s:s + 1], inputs["lm_head"], K, inv_temperature)
        st1 = {key: val[0] for key, val in st1.items()}
        tree = build_marginal_tree(st1["topk_idx"], st1["topk_logprob"], gamma, B)
        st1.pop("logits")
        st1.pop("logprob")
        out["stage1"].append(st1)
        out["tree"].append(tree)
    return out


# ------------------------------------------------- the w/ 2-prev ablation
#
# Ablations, Model Design: the AR approximator reads the two previous tokens
# (the previous bigram) instead of one.  Readings (the paper gives no more):
#   * x_r = [ rms(h_{depth_r}) ; rms(Embd(prev1_r)) ; rms(Embd(prev2_r)) ], the
#     embedding RMSNorm (one gain) applied to each token, prev1 the token
#     right before the drafted position, prev2 the one before it; W_gate and
#     W_up are [I, 3d], W_down [d, I];
#   * depth 1 reads (x_{t-1}, x_t): the context token before the root and the
#     root; depth 2 reads (x_t, candidate m of depth 1); depth i >= 3 reads
#     (candidate m2 of depth i-2, candidate m1 of depth i-1): M^2 rows;
#   * a node expands when its token is a candidate of its depth and, below
#     depth 1, its parent's token is one of the parent depth (which holds for
#     every node whose parent was expanded).

def row_table_2prev(gamma: int, M: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Rows of the bigram-conditioned table: row 0 is depth 1, rows 1..M depth
    2 (candidate m1 = row-1 of depth 1), then for depth i >= 3 the M^2 rows
    1 + M + (i-3)*M^2 + m2*M + m1.  Returns (depth, slot1, slot2) [R]: the
    candidate indices of prev1 (depth-1 list) and prev2 (depth-2 list); -1
    marks the root token, -2 the context token before the root."""
    depth, slot1, slot2 = [1], [-1], [-2]
    if gamma >= 2:
        for m1 in range(M):
            depth.append(2)
            slot1.append(m1)
            slot2.append(-1)
    for i in range(3, gamma + 1):
        for m2 in range(M):
            for m1 in range(M):
                depth.append(i)
                slot1.append(m1)
                slot2.append(m2)
    return (np.asarray(depth, dtype=np.int64), np.asarray(slot1, dtype=np.int64),
            np.asarray(slot2, dtype=np.int64))


def previous_pairs(context: int, root: int, topk_idx_seq: np.ndarray, gamma: int,
                   M: int) -> Tuple[np.ndarray, np.ndarray]:
    """(prev1, prev2) tokens of every row of row_table_2prev."""
    depth, slot1, slot2 = row_table_2prev(gamma, M)

    def token(d_list: int, slot: int) -> int:
        if slot == -1:
            return int(root)
        if slot == -2:
            return int(context)
        return int(topk_idx_seq[d_list - 1, slot])

    prev1 = np.array([token(depth[r] - 1, slot1[r]) for r in range(depth.shape[0])], dtype=np.int64)
    prev2 = np.array([token(depth[r] - 2, slot2[r]) for r in range(depth.shape[0])], dtype=np.int64)
    return prev1, prev2


def ar_approximator_2prev(h_seq: np.ndarray, prev1: np.ndarray, prev2: np.ndarray, depth: np.ndarray,
                          emb: np.ndarray, norm_h_gain: np.ndarray, norm_e_gain: np.ndarray,
                          w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray,
                          eps: float = RMS_EPS, mirror_bf16: bool = False) -> np.ndarray:
    """Eq. 1 with the bigram input x_r = [h~ ; e~(prev1) ; e~(prev2)] (3d wide).
    With mirror_bf16, x and h' are rounded to bf16 (the activation is not)."""
    hd = np.asarray(h_seq, dtype=np.float64)[np.asarray(depth) - 1]
    E = np.asarray(emb, dtype=np.float64)
    x = np.concatenate([rms_norm(hd, norm_h_gain, eps), rms_norm(E[np.asarray(prev1)], norm_e_gain, eps),
                        rms_norm(E[np.asarray(prev2)], norm_e_gain, eps)], axis=-1)
    if mirror_bf16:
        x = bf16_round(x)
    g = x @ np.asarray(w_gate, dtype=np.float64).T
    u = x @ np.asarray(w_up, dtype=np.float64).T
    a = silu(g) * u
    hp = hd + a @ np.asarray(w_down, dtype=np.float64).T
    if mirror_bf16:
        hp = bf16_round(hp)
    return hp


def build_tree_2prev(cond_idx: np.ndarray, cond_logprob: np.ndarray, topk_idx_seq: np.ndarray,
                     gamma: int, M: int, B: int) -> Dict[str, np.ndarray]:
    """OPT-Tree selection over the bigram-conditioned rows.

    Pops, scores and ties as in build_tree.  A popped node of depth i < gamma
    whose token is candidate m1 of depth i expands into row 1 + m1 when i = 1,
    else into row 1 + M + (i-2)*M^2 + m2*M + m1, m2 being its parent's
    candidate index at depth i-1.  Returns build_tree's fields.
    """
    cond_idx = np.asarray(cond_idx)
    lp32 = np.asarray(cond_logprob, dtype=np.float32)
    K = cond_idx.shape[1]
    heap: List[tuple] = []

    def push_row(row: int, parent: int, parent_score: np.float32, depth: int, path: tuple):
        for c in range(K):
            s = np.float32(parent_score + lp32[row, c])        # float32 add
            heapq.heappush(heap, (-float(s), depth, path + (c,), parent, row, c))

    push_row(0, -1, np.float32(0.0), 1, ())
    token, parent, depth_o, score, child_row, rank, slot = [], [], [], [], [], [], []
    while len(token) < B:
        if not heap:
            raise ValueError("draft budget exceeds the number of admissible nodes")
        negs, dep, path, par, row, c = heapq.heappop(heap)
        tok = int(cond_idx[row, c])
        hits = np.nonzero(np.asarray(topk_idx_seq[dep - 1]) == tok)[0]
        m1 = int(hits[0]) if hits.size else -1
        crow = -1
        if dep < gamma and m1 >= 0:
            if dep == 1:
                crow = 1 + m1
            else:
                crow = 1 + M + (dep - 2) * M * M + slot[par] * M + m1
        token.append(tok)
        parent.append(par)
        depth_o.append(dep)
        score.append(np.float32(-negs))
        child_row.append(crow)
        rank.append(c)
        slot.append(m1)
        if crow >= 0:
            push_row(crow, len(token) - 1, np.float32(-negs), dep + 1, path)
    return {
        "token": np.asarray(token, dtype=np.int32),
        "parent": np.asarray(parent, dtype=np.int32),
        "depth": np.asarray(depth_o, dtype=np.int32),
        "score": np.asarray(score, dtype=np.float32),
        "child_row": np.asarray(child_row, dtype=np.int32),
        "rank": np.asarray(rank, dtype=np.int32),
    }


def draft_2prev(inputs: Dict[str, np.ndarray], gamma: int, k: int, B: int,
                inv_temperature: float = 1.0, mirror_bf16: bool = False,
                topk2: Optional[int] = None, eps: float = RMS_EPS,
                keep_full: bool = False, sequences: Optional[List[int]] = None) -> Dict[str, object]:
    """One w/ 2-prev drafting step: ``inputs`` as for draft plus ``context``
    [b] (the token before each root); w_gate and w_up are [I, 3d]."""
    h = inputs["h"]
    V = inputs["lm_head"].shape[0]
    K2 = min(B, V) if topk2 is None else topk2
    seqs = list(range(h.shape[0])) if sequences is None else list(sequences)
    depth, _, _ = row_table_2prev(gamma, k)
    out = {"stage1": [], "rows": [], "hprime": [], "tree": []}
    for s in seqs:
        st1 = marginal_stage(h[s:s + 1], inputs["lm_head"], k, inv_temperature)
        st1 = {key: val[0] for key, val in st1.items()}
        p1, p2 = previous_pairs(int(inputs["context"][s]), int(inputs["root"][s]), st1["topk_idx"], gamma, k)
        hp = ar_approximator_2prev(h[s], p1, p2, depth, inputs["emb"], inputs["norm_h_gain"],
                                   inputs["norm_e_gain"], inputs["w_gate"], inputs["w_up"], inputs["w_down"],
                                   eps=eps, mirror_bf16=mirror_bf16)
        rows = conditional_stage(hp, inputs["lm_head"], K2, inv_temperature, keep_full=keep_full)
        tree = build_tree_2prev(rows["cond_idx"], rows["cond_logprob"], st1["topk_idx"], gamma, k, B)
        if not keep_full:
            st1.pop("logits")
            st1.pop("logprob")
        out["stage1"].append(st1)
        out["rows"].append(rows)
        out["hprime"].append(hp)
        out["tree"].append(tree)
    return out


# ------------------------------------------------------- verification hand-off

def verification_inputs(root_token: int, token: np.ndarray, parent: np.ndarray,
                        depth: np.ndarray) -> Dict[str, np.ndarray]:
    """The draft tree as one verifier input with tree attention.

    Position 0 is the root token x_t; position 1 + j is node j of the tree (pop
    order).  Returns tokens [B+1], positions [B+1] (the depth: 0 for the root)
    and mask [B+1, B+1] (bool): mask[i, j] is true when position j is position
    i or one of its ancestors, i.e. the tokens position i may attend to.
    """
    B = len(token)
    tokens = np.concatenate([[root_token], np.asarray(token)]).astype(np.int32)
    positions = np.concatenate([[0], np.asarray(depth)]).astype(np.int32)
    mask = np.zeros((B + 1, B + 1), dtype=bool)
    mask[0, 0] = True
    for j in range(B):
        i = 1 + j
        mask[i, i] = True
        mask[i, 0] = True
        p = int(parent[j])
        while p >= 0:
            mask[i, 1 + p] = True
            p = int(parent[p])
    return {"tokens": tokens, "positions": positions, "mask": mask}


def acceptance_walk(token: np.ndarray, parent: np.ndarray, target: np.ndarray) -> Dict[str, object]:
    """Greedy equality verification of one draft tree.

    target[0] is the verifier's next token after the root, target[1 + j] its
    next token after the path ending at node j.  From the root, move to the
    child whose token equals the current position's target, as long as there
    is one (siblings carry distinct tokens).  Returns the accepted node ids in
    order, tau = accepted + 1 (the verifier's own next token after the last
    accepted node is always gained) and that bonus token.
    """
    token = np.asarray(token)
    parent = np.asarray(parent)
    accepted: List[int] = []
    cur = -1
    while True:
        want = int(target[1 + cur])
        hit = [j for j in range(len(token)) if parent[j] == cur and token[j] == want]
        if not hit:
            break
        cur = hit[0]
        accepted.append(cur)
    return {"accepted": accepted, "tau": len(accepted) + 1, "bonus": int(target[1 + cur])}

