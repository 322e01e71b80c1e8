"""Parity at the full Qwen3-shaped sizes, in the launch configuration the
benchmark times (same plans, same kernels): stage 1 on every depth, stage 2
on every conditional row, the tree replay and the bit-exact tree kernel
check, for every sequence of every workload (all 16 of the batched one).
At least one checked sequence per workload must also take the end-to-end
leg (its GPU stage-1 candidates equal the oracle's, so the GPU's own chain is
compared with the teacher-forced one).  Weights are drawn on the GPU and
copied to the host as float64 for the oracle."""
import gc

import pytest
import torch

from paper_2606_03819_amd import synth
from parity import check_draft, oracle_inputs

pytestmark = pytest.mark.gpu

FULL = [("qwen3-4b-shape", [0]), ("qwen3-8b-shape", [0]), ("qwen3-8b-shape-k16-b64", [0]),
        ("qwen3-8b-shape-batch16", list(range(16))), ("qwen3-8b-shape-b512", [0]), ("qwen3-8b-shape-m64", [0]),
        ("qwen3-4b-shape-i9728", [0]), ("qwen3-8b-shape-i12288", [0]), ("qwen3-8b-shape-linear", [0])]


@pytest.mark.parametrize("name,seqs", FULL, ids=[f[0] for f in FULL])
def test_full_size_parity(name, seqs):
    w = synth.get_workload(name)
    print(f"[fullsize] {name}: drawing inputs on the GPU", flush=True)
    g = synth.make_inputs(w, "cuda")
    o_in = oracle_inputs(g)
    print(f"[fullsize] {name}: oracle inputs ready; checking sequences {seqs}", flush=True)
    check_draft(w, g, o_in, seqs, 2e-2, log=lambda m: print(m, flush=True), require_e2e=True)
    del g, o_in
    gc.collect()
    torch.cuda.empty_cache()
