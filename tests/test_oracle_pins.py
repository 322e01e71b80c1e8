"""Pins for the CPU oracle: library routines, closed forms, special cases.

Every check here computes its expectation by a route that does not go through
the oracle's own code (torch / scipy library routines, hand-built weights whose
effect is known in closed form, structural facts of the algorithm).  The
mutation tests at the end plant plausible mistakes in the oracle and assert
that at least one pin catches each of them.
"""
import math

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

import oracle
import oracle.treeflash_oracle as ot


# ------------------------------------------------------------------ helpers

def _perm_matrix(perm):
    n = len(perm)
    p = np.zeros((n, n))
    p[np.arange(n), perm] = 1.0
    return p


def pin_bf16_round(rng):
    """bf16 rounding agrees with torch's float32 -> bfloat16 conversion (RNE)."""
    x = rng.standard_normal(20000).astype(np.float32) * np.float32(3.0)
    # add exact halfway points: mantissa with bit pattern ...1000 0000 0000 0000 below bf16
    base = rng.integers(0, 2**16, size=4000, dtype=np.uint32) << 16
    half = (base | np.uint32(0x8000)).view(np.float32)
    half = half[np.isfinite(half) & (np.abs(half) > 1e-30) & (np.abs(half) < 1e30)]
    x = np.concatenate([x, half])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = oracle.bf16_round(x.astype(np.float64))
    return np.array_equal(ref, got)


def pin_rms_norm(rng):
    x = rng.standard_normal((7, 33)) * 3.0
    g = rng.standard_normal(33)
    ref = F.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), eps=1e-6).numpy()
    return np.allclose(oracle.rms_norm(x, g, 1e-6), ref, rtol=1e-13, atol=1e-13)


def pin_silu(rng):
    g = rng.standard_normal(1000) * 6.0
    ref = F.silu(torch.from_numpy(g)).numpy()
    return (np.allclose(oracle.silu(g), ref, rtol=1e-13, atol=1e-15)
            and abs(oracle.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-15)


def pin_marginal_permuted_identity(rng, d=24, k=5, inv_t=1.7):
    """W_lm = c * P: logit v = inv_T * c * h[perm[v]]; compare with scipy."""
    perm = rng.permutation(d)
    c = 0.75
    w = c * _perm_matrix(perm)
    h = rng.standard_normal((2, 3, d))
    st = oracle.marginal_stage(h, w, k, inv_t)
    z = inv_t * c * h[..., perm]
    ok = np.allclose(st["logits"], z, rtol=1e-14, atol=1e-14)
    ok &= np.allclose(st["logprob"], scipy.special.log_softmax(z, axis=-1), atol=1e-12)
    # top-k by hand: vocabulary ids sorted by their logit
    for bi in range(2):
        for i in range(3):
            want = sorted(range(d), key=lambda v: (-z[bi, i, v], v))[:k]
            ok &= list(st["topk_idx"][bi, i]) == want
    return bool(ok)


def pin_ar_closed_form(rng, d=12, mirror=False):
    """Identity-block SwiGLU: W_gate=[P,0], W_up=[0,I], W_down=I.

    Then h' = h + silu(P rms(h) g_h) * rms(E[prev]) g_e elementwise, computed
    here with torch's rms_norm / silu.
    """
    V, gamma, M = 9, 3, 2
    perm = rng.permutation(d)
    p = _perm_matrix(perm)
    w_gate = np.concatenate([p, np.zeros((d, d))], axis=1)
    w_up = np.concatenate([np.zeros((d, d)), np.eye(d)], axis=1)
    w_down = np.eye(d)
    h = rng.standard_normal((gamma, d)) * 2.0
    emb = rng.standard_normal((V, d)) * 0.05
    gh = rng.uniform(0.5, 1.5, d)
    ge = rng.uniform(0.5, 1.5, d)
    if mirror:
        h = oracle.bf16_round(h)
    topk = np.array([[1, 4], [7, 2], [0, 8]])
    root = 5
    depth, _ = oracle.row_table(gamma, M)
    prev = oracle.previous_tokens(root, topk, gamma, M)
    got = oracle.ar_approximator(h, prev, depth, emb, gh, ge, w_gate, w_up, w_down,
                                 eps=1e-6, mirror_bf16=mirror)
    th = torch.from_numpy(h[depth - 1])
    hn = F.rms_norm(th, (d,), torch.from_numpy(gh), eps=1e-6)
    en = F.rms_norm(torch.from_numpy(emb[prev]), (d,), torch.from_numpy(ge), eps=1e-6)
    if mirror:
        hn = hn.to(torch.float32).to(torch.bfloat16).to(torch.float64)
        en = en.to(torch.float32).to(torch.bfloat16).to(torch.float64)
    a = F.silu(hn[:, perm]) * en          # the activation is not a rounding point
    want = th + a
    if mirror:
        want = want.to(torch.float32).to(torch.bfloat16).to(torch.float64)
    # rows: depth-1 row conditioned on root, then (depth 2, cand m of depth 1), ...
    ok = list(prev) == [5, 1, 4, 7, 2]
    tol = 0.0 if not mirror else 0.0
    if mirror:
        # torch rounds the float64 value through float32 first; where that double
        # rounding differs from a direct bf16 rounding (exact halfway cases) the
        # two may disagree by one bf16 ulp, so compare to that bound.
        ulp = np.abs(want.numpy()) * 2.0 ** -7 + 1e-30
        return ok and bool(np.all(np.abs(got - want.numpy()) <= ulp))
    return ok and bool(np.allclose(got, want.numpy(), rtol=1e-13, atol=1e-13 + tol))


def pin_silu_mlp_closed_form(rng, d=20, mirror=False):
    """Without W_up (the plain SiLU MLP side mode): with W_gate = [P | c I]
    (P a permutation) and a diagonal W_down = diag(s), every row is
    h' = h + s * silu(P h~ + c e~); checked against torch's rms_norm and
    silu, also with the bf16 rounding points."""
    V, gamma, M = 11, 4, 2
    perm = rng.permutation(d)
    c = 0.75
    w_gate = np.concatenate([_perm_matrix(perm), c * np.eye(d)], axis=1)
    sc = rng.uniform(-1.5, 1.5, d)
    w_down = np.diag(sc)
    h = rng.standard_normal((gamma, d)) * 1.5
    emb = rng.standard_normal((V, d)) * 0.05
    gh = rng.uniform(0.5, 1.5, d)
    ge = rng.uniform(0.5, 1.5, d)
    if mirror:
        h = oracle.bf16_round(h)
    topk = np.array([[3, 9], [10, 0], [6, 2], [1, 4]])
    depth, _ = oracle.row_table(gamma, M)
    prev = oracle.previous_tokens(8, topk, gamma, M)
    got = oracle.ar_approximator(h, prev, depth, emb, gh, ge, w_gate, None, w_down, eps=1e-6, mirror_bf16=mirror)
    th = torch.from_numpy(h[depth - 1])
    hn = F.rms_norm(th, (d,), torch.from_numpy(gh), eps=1e-6)
    en = F.rms_norm(torch.from_numpy(emb[prev]), (d,), torch.from_numpy(ge), eps=1e-6)
    if mirror:
        hn = hn.to(torch.float32).to(torch.bfloat16).to(torch.float64)
        en = en.to(torch.float32).to(torch.bfloat16).to(torch.float64)
    want = th + F.silu(hn[:, perm] + c * en) * torch.from_numpy(sc)
    if mirror:
        want = want.to(torch.float32).to(torch.bfloat16).to(torch.float64)
        ulp = np.abs(want.numpy()) * 2.0 ** -7 + 1e-30
        return bool(np.all(np.abs(got - want.numpy()) <= ulp))
    return bool(np.allclose(got, want.numpy(), rtol=1e-13, atol=1e-13))


def pin_zero_down(rng, mirror=True):
    """Zero-initialised AR approximator reproduces the drafter (Training paragraph)."""
    V, d, gamma, M = 30, 16, 4, 3
    h = oracle.bf16_round(rng.standard_normal((gamma, d)))
    emb = rng.standard_normal((V, d)) * 0.02
    wg = rng.standard_normal((d, 2 * d)) * 0.3
    wu = rng.standard_normal((d, 2 * d)) * 0.3
    wd = np.zeros((d, d))
    topk = np.stack([rng.permutation(V)[:M] for _ in range(gamma)])
    depth, _ = oracle.row_table(gamma, M)
    prev = oracle.previous_tokens(3, topk, gamma, M)
    hp = oracle.ar_approximator(h, prev, depth, emb, np.ones(d), np.ones(d), wg, wu, wd,
                                mirror_bf16=mirror)
    return bool(np.array_equal(hp, h[depth - 1]))


def pin_row_table(rng):
    gamma, M = 5, 3
    depth, slot = oracle.row_table(gamma, M)
    ok = depth.shape[0] == 1 + (gamma - 1) * M
    topk = np.arange(gamma * M).reshape(gamma, M) * 10 + 1000
    prev = oracle.previous_tokens(77, topk, gamma, M)
    want = [77]
    for i in range(2, gamma + 1):          # depth i is conditioned on depth i-1's candidates
        want += [1000 + 10 * ((i - 2) * M + m) for m in range(M)]
    return bool(ok and list(prev) == want and list(depth) == [1] + sum(([i] * M for i in range(2, gamma + 1)), []))


def pin_rows_sum_to_one(rng):
    hp = rng.standard_normal((6, 10))
    w = rng.standard_normal((40, 10))
    out = oracle.conditional_stage(hp, w, 40, 1.3, keep_full=True)
    full = np.exp(out["logprob"])
    ref = scipy.special.softmax(1.3 * hp @ w.T, axis=-1)
    return bool(np.allclose(full, ref, atol=1e-14) and np.allclose(full.sum(-1), 1.0, atol=1e-13))


def pin_uniform_head(rng):
    """A zero LM head gives the uniform row: log-prob -log V, ties in id order."""
    V, d, k = 50, 8, 6
    h = rng.standard_normal((1, 4, d))
    st = oracle.marginal_stage(h, np.zeros((V, d)), k, 1.0)
    return bool(np.allclose(st["logprob"], -math.log(V), atol=1e-15)
                and np.array_equal(st["topk_idx"], np.broadcast_to(np.arange(k), (1, 4, k))))


ALL_PINS = [pin_uniform_head, pin_bf16_round, pin_rms_norm, pin_silu, pin_marginal_permuted_identity,
            pin_ar_closed_form, pin_silu_mlp_closed_form, pin_zero_down, pin_row_table, pin_rows_sum_to_one]


# ------------------------------------------------------------------- tests

@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    assert pin(np.random.default_rng(1234))


def test_bf16_round_known_values():
    x = np.array([1 + 2**-8, 1 + 3 * 2**-8, 1 + 2**-7, -(1 + 2**-8), 0.0, 2**-126, 65535.0])
    want = np.array([1.0, 1 + 2**-6, 1 + 2**-7, -1.0, 0.0, 2**-126, 65536.0])
    assert np.array_equal(oracle.bf16_round(x), want)


def test_ar_closed_form_mirror():
    assert pin_ar_closed_form(np.random.default_rng(7), mirror=True)


def test_silu_mlp_closed_form_mirror():
    assert pin_silu_mlp_closed_form(np.random.default_rng(8), mirror=True)


def test_silu_mlp_zero_down_keeps_the_state():
    rng = np.random.default_rng(9)
    V, d, gamma, M = 25, 16, 3, 2
    h = oracle.bf16_round(rng.standard_normal((gamma, d)))
    topk = np.stack([rng.permutation(V)[:M] for _ in range(gamma)])
    depth, _ = oracle.row_table(gamma, M)
    prev = oracle.previous_tokens(4, topk, gamma, M)
    hp = oracle.ar_approximator(h, prev, depth, rng.standard_normal((V, d)), np.ones(d), np.ones(d),
                                rng.standard_normal((d, 2 * d)), None, np.zeros((d, d)), mirror_bf16=True)
    assert np.array_equal(hp, h[depth - 1])


def test_topk_tie_rule():
    v = np.array([[1.0, 3.0, 3.0, 2.0, 3.0, -1.0]])
    assert list(oracle.topk_sorted(v, 4)[0]) == [1, 2, 4, 3]


def test_temperature_keeps_order():
    rng = np.random.default_rng(3)
    h = rng.standard_normal((1, 3, 16))
    w = rng.standard_normal((100, 16))
    a = oracle.marginal_stage(h, w, 10, 1.0)["topk_idx"]
    b = oracle.marginal_stage(h, w, 10, 1 / 0.7)["topk_idx"]
    assert np.array_equal(a, b)


def test_zero_down_rows_match_stage1():
    """With W_down = 0 every depth-i conditional row equals the stage-1 row i."""
    rng = np.random.default_rng(5)
    V, d, gamma, M, B = 40, 16, 4, 3, 12
    inputs = {
        "h": oracle.bf16_round(rng.standard_normal((1, gamma, d))),
        "root": np.array([3]),
        "lm_head": oracle.bf16_round(rng.standard_normal((V, d)) * 0.3),
        "emb": rng.standard_normal((V, d)) * 0.02,
        "norm_h_gain": np.ones(d), "norm_e_gain": np.ones(d),
        "w_gate": rng.standard_normal((d, 2 * d)), "w_up": rng.standard_normal((d, 2 * d)),
        "w_down": np.zeros((d, d)),
    }
    out = oracle.draft(inputs, gamma, M, B, mirror_bf16=True, topk2=V, keep_full=True)
    lp1 = out["stage1"][0]["logprob"]
    lp2 = out["rows"][0]["logprob"]
    depth, _ = oracle.row_table(gamma, M)
    assert np.allclose(lp2, lp1[depth - 1], atol=1e-12)


# ------------------------------------------------------- planted mistakes

MUTATIONS = {
    "silu_sign": ("silu", lambda g: np.asarray(g) / (1.0 + np.exp(np.asarray(g)))),
    "rms_no_sqrt": ("rms_norm", lambda x, g, eps=1e-6: np.asarray(x) / (np.mean(np.asarray(x) ** 2, -1, keepdims=True) + eps) * g),
    "bf16_truncate": ("bf16_round", lambda x: np.ldexp(np.trunc(np.ldexp(np.frexp(np.asarray(x, dtype=np.float64))[0], 8)),
                                                       np.frexp(np.asarray(x, dtype=np.float64))[1] - 8)),
    "softmax_no_max_shift_wrong": ("log_softmax", lambda z: (np.asarray(z) - np.log(np.sum(np.exp(np.asarray(z)), -1, keepdims=True)) + 1e-3,
                                                             np.log(np.sum(np.exp(np.asarray(z)), -1)))),
    "topk_ties_descending": ("topk_sorted", lambda v, k: (np.asarray(v).shape[-1] - 1 - np.argsort(
        -np.asarray(v)[..., ::-1], axis=-1, kind="stable"))[..., :k]),
}


def _prev_wrong_depth(root, topk_idx_seq, gamma, M):
    depth, slot = ot.row_table(gamma, M)
    prev = np.empty(depth.shape[0], dtype=np.int64)
    for r in range(depth.shape[0]):
        prev[r] = root if slot[r] < 0 else int(topk_idx_seq[depth[r] - 1, slot[r]])
    return prev


def _ar_swapped_halves(h_seq, prev, depth, emb, gh, ge, wg, wu, wd, eps=1e-6, mirror_bf16=False):
    hd = np.asarray(h_seq, dtype=np.float64)[np.asarray(depth) - 1]
    e = np.asarray(emb, dtype=np.float64)[np.asarray(prev)]
    x = np.concatenate([ot.rms_norm(e, ge, eps), ot.rms_norm(hd, gh, eps)], axis=-1)
    a = ot.silu(x @ np.asarray(wg).T) * (x @ np.asarray(wu).T)
    return hd + a @ np.asarray(wd).T


def _ar_no_residual(h_seq, prev, depth, emb, gh, ge, wg, wu, wd, eps=1e-6, mirror_bf16=False):
    hd = np.asarray(h_seq, dtype=np.float64)[np.asarray(depth) - 1]
    e = np.asarray(emb, dtype=np.float64)[np.asarray(prev)]
    x = np.concatenate([ot.rms_norm(hd, gh, eps), ot.rms_norm(e, ge, eps)], axis=-1)
    if mirror_bf16:
        x = ot.bf16_round(x)
    a = ot.silu(x @ np.asarray(wg).T) * (x @ np.asarray(wu).T)
    if mirror_bf16:
        a = ot.bf16_round(a)
    out = a @ np.asarray(wd).T
    return ot.bf16_round(out) if mirror_bf16 else out


def _marginal_transposed(h, lm_head, k, inv_temperature=1.0):
    h = np.asarray(h, dtype=np.float64)
    w = np.asarray(lm_head, dtype=np.float64)
    z = inv_temperature * np.matmul(h, w)          # wrong operand orientation
    lp, lse = ot.log_softmax(z)
    idx = ot.topk_sorted(z, k)
    return {"logits": z, "logprob": lp, "lse": lse, "topk_idx": idx.astype(np.int32),
            "topk_logprob": np.take_along_axis(lp, idx, axis=-1)}


def _ar_silu_gate_squared(h_seq, prev, depth, emb, gh, ge, wg, wu, wd, eps=1e-6, mirror_bf16=False):
    # without an up projection, multiplies the activation by the gate again
    hd = np.asarray(h_seq, dtype=np.float64)[np.asarray(depth) - 1]
    e = np.asarray(emb, dtype=np.float64)[np.asarray(prev)]
    x = np.concatenate([ot.rms_norm(hd, gh, eps), ot.rms_norm(e, ge, eps)], axis=-1)
    if mirror_bf16:
        x = ot.bf16_round(x)
    g = x @ np.asarray(wg).T
    a = ot.silu(g) * (x @ np.asarray(wu).T if wu is not None else g)
    out = hd + a @ np.asarray(wd).T
    return ot.bf16_round(out) if mirror_bf16 else out


MUTATIONS.update({
    "silu_mode_gate_squared": ("ar_approximator", _ar_silu_gate_squared),
    "prev_from_same_depth": ("previous_tokens", _prev_wrong_depth),
    "concat_halves_swapped": ("ar_approximator", _ar_swapped_halves),
    "residual_dropped": ("ar_approximator", _ar_no_residual),
    "lm_head_transposed": ("marginal_stage", _marginal_transposed),
})


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(ot, attr, fn)
    monkeypatch.setattr(oracle, attr, fn)
    caught = []
    for pin in ALL_PINS:
        try:
            ok = pin(np.random.default_rng(1234))
        except Exception:
            ok = False
        if not ok:
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake {name}"
