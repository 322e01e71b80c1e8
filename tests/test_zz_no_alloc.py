"""The allocation-free LM-head call (treeflash_marginal_topk_static, scratch in
the library's own device array) against the workspace call on the same
inputs: top-k ids, log-probs and log-sum-exp bit for bit (same kernels, same
data), on two calls in a row, the second smaller than the first, so stale
contents of the shared array would show."""
import pytest
import torch

from paper_2606_03819_amd import binding, synth

pytestmark = pytest.mark.gpu


def _case(b, rows, d, V, k, seed, inv_t=1.0):
    gen = torch.Generator(device="cuda").manual_seed(seed)
    h = torch.randn((b, rows, d), generator=gen, device="cuda").to(torch.bfloat16)
    w = (0.02 * torch.randn((V, d), generator=gen, device="cuda")).to(torch.bfloat16)
    return h, w, k, inv_t


def _both(h, w, k, inv_t):
    b, rows, _ = h.shape
    lse_a = torch.empty((b, rows), dtype=torch.float32, device="cuda")
    lse_b = torch.empty_like(lse_a)
    ia, la = binding.treeflash_marginal_topk(h, w, k, inv_t, lse=lse_a)
    ib, lb = binding.treeflash_marginal_topk_static(h, w, k, inv_t, lse=lse_b)
    torch.cuda.synchronize()
    return (ia, la, lse_a), (ib, lb, lse_b)


def test_static_scratch_matches_the_workspace_call():
    cases = [
        # the 8B shape's 121 conditional rows, 32-entry lists (the larger call) ...
        (1, 121, 4096, 151936, 32, 1),
        # ... then a smaller one: 16 drafter states, 8 entries, a ragged vocabulary
        (1, 16, 1024, 30011, 8, 2),
        # and a second large one after the small one (long lists, temperature)
        (2, 40, 2048, 60000, 64, 3, 1 / 0.7),
    ]
    for c in cases:
        print(f"[no-alloc] b{c[0]} rows{c[1]} d{c[2]} V{c[3]} k{c[4]}", flush=True)
        h, w, k, inv_t = _case(*c)
        (ia, la, sa), (ib, lb, sb) = _both(h, w, k, inv_t)
        assert torch.equal(ia, ib), "top-k ids differ"
        assert torch.equal(la, lb), "log-probs differ"
        assert torch.equal(sa, sb), "log-sum-exp differs"
        del h, w
        torch.cuda.empty_cache()


def test_static_scratch_rejects_oversized_calls():
    # 16 sequences' 121 conditional rows need far more than the array holds
    h = torch.zeros((16, 121, 4096), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((151936, 4096), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(binding.TreeflashError) as e:
        binding.treeflash_marginal_topk_static(h, w, 32)
    assert e.value.status == 3   # TF_ERR_WORKSPACE
