"""Pins for the oracle's "w/ Linear" AR approximator (Ablations, Model Design:
the SwiGLU head replaced by a linear layer on the same input).

Pinned by special cases whose results follow from the definition without
restating it: a zero map is the identity on h, a map that copies the
embedding half adds the normalised embedding (torch's rms_norm), the map is
additive in W_lin, and it differs from the SwiGLU head (a planted swap of
the two halves of the input is caught)."""
import numpy as np
import torch

import oracle


def setup(rng, d=16, V=10, gamma=3, M=2):
    depth, _ = oracle.row_table(gamma, M)
    topk = np.stack([rng.permutation(V)[:M] for _ in range(gamma)])
    prev = oracle.previous_tokens(int(rng.integers(V)), topk, gamma, M)
    h = rng.standard_normal((gamma, d))
    emb = rng.standard_normal((V, d))
    return h, prev, depth, emb, np.ones(d), np.ones(d)


def test_zero_map_is_identity():
    rng = np.random.default_rng(1)
    h, prev, depth, emb, gh, ge = setup(rng)
    hp = oracle.ar_approximator_linear(h, prev, depth, emb, gh, ge, np.zeros((16, 32)))
    assert np.array_equal(hp, h[depth - 1])


def test_copying_the_embedding_half_adds_the_normalised_embedding():
    rng = np.random.default_rng(2)
    h, prev, depth, emb, gh, ge = setup(rng)
    ge = rng.uniform(0.5, 1.5, 16)
    w = np.concatenate([np.zeros((16, 16)), np.eye(16)], axis=1)
    hp = oracle.ar_approximator_linear(h, prev, depth, emb, gh, ge, w)
    ref = torch.nn.functional.rms_norm(torch.tensor(emb[prev]), (16,), torch.tensor(ge), eps=1e-6).numpy()
    assert np.allclose(hp - h[depth - 1], ref, atol=1e-12)


def test_additive_in_the_map():
    rng = np.random.default_rng(3)
    h, prev, depth, emb, gh, ge = setup(rng)
    w1, w2 = rng.standard_normal((16, 32)), rng.standard_normal((16, 32))
    f = lambda w: oracle.ar_approximator_linear(h, prev, depth, emb, gh, ge, w) - h[depth - 1]
    assert np.allclose(f(w1 + w2), f(w1) + f(w2), atol=1e-10)


def test_swapped_input_halves_are_caught():
    rng = np.random.default_rng(4)
    h, prev, depth, emb, gh, ge = setup(rng)
    w = np.concatenate([np.eye(16), np.zeros((16, 16))], axis=1)   # copies the h half
    hp = oracle.ar_approximator_linear(h, prev, depth, emb, gh, ge, w)
    ref = torch.nn.functional.rms_norm(torch.tensor(h[depth - 1]), (16,), eps=1e-6).numpy()
    assert np.allclose(hp - h[depth - 1], ref, atol=1e-12)
    e_ref = torch.nn.functional.rms_norm(torch.tensor(emb[prev]), (16,), eps=1e-6).numpy()
    assert not np.allclose(hp - h[depth - 1], e_ref, atol=1e-3)


def test_mirror_rounding_points():
    rng = np.random.default_rng(5)
    h, prev, depth, emb, gh, ge = setup(rng)
    h = oracle.bf16_round(h)
    w = rng.standard_normal((16, 32)) * 0.1
    hp = oracle.ar_approximator_linear(h, prev, depth, emb, gh, ge, w, mirror_bf16=True)
    assert np.array_equal(hp, oracle.bf16_round(hp))
    x = np.concatenate([oracle.rms_norm(h[depth - 1], gh), oracle.rms_norm(emb[prev], ge)], -1)
    assert np.array_equal(hp, oracle.bf16_round(h[depth - 1] + oracle.bf16_round(x) @ w.T))
