"""GPU parity of the w/ 2-prev approximator (Ablations, Model Design: the
previous bigram as the approximator's input) and of its bigram-row tree.

* h' element by element against ``oracle.ar_approximator_2prev``: fp32 within
  1e-4 relative; bf16 within one bf16 unit in the last place plus 1e-3 (both
  sides round the same sum to bf16);
* the whole step through ``check_draft``: stage-1 and stage-2 lists and the
  log-sum-exp within 2e-2 (bf16) / 1e-4 (fp32), the tree replayed against the
  oracle's rows, and the tree kernel fed the oracle's rows bit for bit;
* with the prev2 block of W_gate / W_up zero, every bigram row equals the
  single-token row of the same (depth, previous token) computed by the
  single-token kernels: bit for bit in fp32 (the same products in the same
  order, then zero terms), within one bf16 unit in bf16 (the k-cut of a
  3d-wide product sums its pieces in another order);
* the Qwen3-8B-shaped step (905 rows per sequence) on one sampled sequence.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
from paper_2606_03819_amd import binding, synth
from parity import check_draft, oracle_inputs

pytestmark = pytest.mark.gpu

W = synth.Workload
CASES = [
    # (workload, weight std, factor on W_down): a small W_down keeps h' near h,
    # so the candidates of each depth lead the conditional rows and the trees
    # grow deep through the bigram rows
    (W("2prev-f32", 1, 128, 2048, 5, 3, 16, 128, "f32", 1.0, 41, 51, "", "2prev"), 0.05, 1.0),
    (W("2prev-bf16-ragged", 2, 96, 1000, 4, 3, 12, 64, "bf16", 1.0, 42, 52, "", "2prev"), 0.15, 1.0),
    (W("2prev-bf16-d48", 2, 48, 700, 5, 2, 10, 48, "bf16", 1.0, 43, 53, "", "2prev"), 0.2, 1.0),
    (W("2prev-bf16-temp", 1, 256, 5003, 6, 4, 20, 128, "bf16", 1.0 / 0.7, 44, 54, "", "2prev"), 0.08, 1.0),
    (W("2prev-bf16-gamma1", 3, 64, 300, 1, 2, 7, 32, "bf16", 1.0, 45, 55, "", "2prev"), 0.2, 1.0),
    (W("2prev-bf16-gamma2", 2, 64, 300, 2, 3, 9, 32, "bf16", 1.0, 46, 56, "", "2prev"), 0.2, 1.0),
    (W("2prev-bf16-many-rows", 3, 128, 2048, 6, 6, 40, 64, "bf16", 1.0, 47, 57, "", "2prev"), 0.1, 1.0),
    (W("2prev-bf16-deep", 2, 128, 1500, 6, 4, 60, 64, "bf16", 1.0, 49, 59, "", "2prev"), 0.3, 0.002),
    (W("2prev-f32-deep", 1, 64, 800, 5, 3, 40, 64, "f32", 1.0, 50, 60, "", "2prev"), 0.4, 0.002),
]


def inputs_of(w, std, down):
    cpu = synth.make_inputs(w, "cpu", weight_std=std)
    if down != 1.0:
        cpu["w_down"] = (cpu["w_down"].float() * down).to(cpu["w_down"].dtype)
    return cpu


def tol_for(w):
    return 2e-2 if w.dtype == "bf16" else 1e-4


def bf16_ulp(x):
    a = np.maximum(np.abs(x), np.finfo(np.float32).tiny)
    return np.exp2(np.floor(np.log2(a)) - 7)


def seeded_candidates(w, seed):
    gen = torch.Generator().manual_seed(seed)
    return np.stack([np.stack([torch.randperm(w.V, generator=gen)[:w.k].numpy() for _ in range(w.gamma)])
                     for _ in range(w.b)]).astype(np.int64)


def gpu_hprime(g, topk):
    tk = torch.from_numpy(topk).to(torch.int32).cuda()
    return binding.treeflash_arapprox_2prev_hidden(g["h"], g["context"], g["root"], tk, g["emb"], g["norm_h_gain"],
                                                   g["norm_e_gain"], g["w_gate"], g["w_up"], g["w_down"])


@pytest.mark.parametrize("w,std,down", CASES, ids=[c[0].name for c in CASES])
def test_2prev_hidden_matches_oracle(w, std, down):
    print(f"[2prev] h' case={w.name} b{w.b} d{w.d} V{w.V} g{w.gamma} k{w.k} I{w.I} rows{w.rows}", flush=True)
    cpu = inputs_of(w, std, down)
    g = {k: v.cuda() for k, v in cpu.items()}
    o_in = oracle_inputs(cpu)
    topk = seeded_candidates(w, w.state_seed)
    got = synth.to_numpy64(gpu_hprime(g, topk))
    depth, _, _ = oracle.row_table_2prev(w.gamma, w.k)
    assert got.shape == (w.b, w.rows, w.d)
    for s in range(w.b):
        p1, p2 = oracle.previous_pairs(int(o_in["context"][s]), int(o_in["root"][s]), topk[s], w.gamma, w.k)
        ref = oracle.ar_approximator_2prev(o_in["h"][s], p1, p2, depth, o_in["emb"], o_in["norm_h_gain"],
                                           o_in["norm_e_gain"], o_in["w_gate"], o_in["w_up"], o_in["w_down"],
                                           mirror_bf16=(w.dtype == "bf16"))
        err = np.abs(got[s] - ref)
        if w.dtype == "bf16":
            # the activation is a bf16 operand too: one unit there moves h' by
            # at most |w_down| * ulp, far below one unit of h' at these scales
            bound = bf16_ulp(np.maximum(np.abs(ref), np.abs(got[s]))) + 1e-3
        else:
            bound = 1e-4 * (1.0 + np.abs(ref))
        bad = np.argwhere(err > bound)
        assert bad.size == 0, f"{w.name} seq {s}: h' differs at {bad[:5].tolist()}"


@pytest.mark.parametrize("w,std,down", CASES, ids=[c[0].name for c in CASES])
def test_2prev_draft_matches_oracle(w, std, down):
    print(f"[2prev] draft case={w.name} b{w.b} d{w.d} V{w.V} g{w.gamma} k{w.k} B{w.B}", flush=True)
    cpu = inputs_of(w, std, down)
    stats = check_draft(w, {k: v.cuda() for k, v in cpu.items()}, oracle_inputs(cpu), range(w.b), tol_for(w))
    print(f"[2prev] {w.name}: {stats}", flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_zero_prev2_block_matches_the_single_token_kernels(dtype):
    w2 = W("2prev-zero", 2, 128, 900, 5, 3, 12, 96, dtype, 1.0, 48, 58, "", "2prev")
    g = {k: v.cuda() for k, v in synth.make_inputs(w2, "cpu", weight_std=0.1).items()}
    d = w2.d
    g["w_gate"][:, 2 * d:] = 0
    g["w_up"][:, 2 * d:] = 0
    topk = seeded_candidates(w2, 9)
    hp2 = gpu_hprime(g, topk)
    tk = torch.from_numpy(topk).to(torch.int32).cuda()
    hp1 = binding.treeflash_arapprox_hidden(g["h"], g["root"], tk, g["emb"], g["norm_h_gain"], g["norm_e_gain"],
                                            g["w_gate"][:, :2 * d].contiguous(), g["w_up"][:, :2 * d].contiguous(),
                                            g["w_down"])
    depth, s1, _ = oracle.row_table_2prev(w2.gamma, w2.k)
    src = torch.from_numpy(np.array([0 if depth[r] == 1 else 1 + (depth[r] - 2) * w2.k + s1[r]
                                     for r in range(depth.shape[0])])).cuda()
    want = hp1[:, src]
    if dtype == "f32":
        assert torch.equal(hp2, want)
    else:
        diff = (hp2.float() - want.float()).abs()
        ulp = torch.from_numpy(bf16_ulp(np.maximum(np.abs(synth.to_numpy64(want)), 1e-3))).cuda().float()
        assert bool((diff <= ulp + 1e-3).all())


def test_full_size_2prev_step():
    w = synth.get_workload("qwen3-8b-shape-2prev")
    print(f"[2prev] full-size {w.name}: drawing inputs on the GPU", flush=True)
    g = synth.make_inputs(w, "cuda")
    o_in = oracle_inputs(g)
    print(f"[2prev] full-size {w.name}: checking sequence 0 ({w.rows} rows)", flush=True)
    check_draft(w, g, o_in, [0], 2e-2, log=lambda m: print(m, flush=True))
    del g, o_in
    gc.collect()
    torch.cuda.empty_cache()
