"""C ABI checks that need no GPU: the library loads, exports every function the
header declares, and rejects invalid arguments before touching HIP."""
import ctypes
import os
import re

import pytest

from paper_2606_03819_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "treeflash.h")

pytestmark = pytest.mark.skipif(not os.path.exists(binding.LIB_PATH), reason="libtreeflash.so not built")

FAKE = 0x10000          # 16-byte aligned non-null dummy pointers: never dereferenced
FAKE2 = 0x20000
BF16, F32 = binding.TF_BF16, binding.TF_F32
INVALID, UNSUPPORTED, WORKSPACE = 1, 2, 3


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(treeflash_[a-z0-9_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(binding.EXPORTED)


def test_every_declared_symbol_is_exported():
    lib = binding.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings():
    for s in range(5):
        assert binding.status_string(s) and binding.status_string(s) != "unknown status"
    assert binding.status_string(99) == "unknown status"


def test_workspace_size_covers_the_buffers_and_rejects_bad_shapes():
    f = binding.lib().treeflash_workspace_bytes
    for b in (1, 2, 16):
        rows = b * (1 + 15 * 8)
        # at least h' and the normalised embeddings [b*R, d] and the SwiGLU activation [b*R, I] in bf16
        assert f(b, 16, 4096, 4096, 151936, 8, 32, BF16) >= 3 * rows * 4096 * 2
    assert f(1, 8, 256, 256, 4096, 4, 16, F32) > 0
    assert f(0, 16, 4096, 4096, 151936, 8, 32, BF16) == 0         # b < 1
    assert f(1, 16, 4100, 4096, 151936, 8, 32, BF16) == 0         # d % 16
    assert f(1, 16, 4096, 4096, 151936, 8, 151937, BF16) == 0     # topk2 > V
    assert f(1, 16, 4096, 4096, 8, 9, 8, BF16) == 0               # k > V
    assert f(1, 16, 4096, 4096, 151936, 8, 32, 7) == 0            # dtype


def _marginal(timed=False, **over):
    a = dict(h=FAKE, w=FAKE, b=1, gamma=16, d=4096, V=151936, k=8, it=1.0, dt=BF16, idx=FAKE2, lp=None,
             lse=None, ws=FAKE, wsb=1 << 40, st=None)
    a.update(over)
    args = (a["h"], a["w"], a["b"], a["gamma"], a["d"], a["V"], a["k"], a["it"], a["dt"], a["idx"], a["lp"],
            a["lse"], a["ws"], a["wsb"], a["st"])
    if timed:   # events are never touched when validation fails
        return binding.lib().treeflash_marginal_topk_timed(*args, FAKE, FAKE)
    return binding.lib().treeflash_marginal_topk(*args)


@pytest.mark.parametrize("over,code", [
    (dict(h=None), INVALID), (dict(w=None), INVALID), (dict(idx=None), INVALID),
    (dict(b=0), INVALID), (dict(gamma=0), INVALID), (dict(d=4090), UNSUPPORTED), (dict(d=0), INVALID),
    (dict(k=0), INVALID), (dict(k=151937), INVALID), (dict(k=2000), INVALID), (dict(V=0), INVALID),
    (dict(it=0.0), INVALID), (dict(it=-1.0), INVALID), (dict(it=float("inf")), INVALID),
    (dict(it=float("nan")), INVALID), (dict(dt=5), INVALID), (dict(h=FAKE + 4), UNSUPPORTED), (dict(h=FAKE + 1), INVALID),
    (dict(lp=FAKE + 2), INVALID), (dict(lse=FAKE + 1), INVALID), (dict(w=FAKE + 4), UNSUPPORTED),
    (dict(ws=None), WORKSPACE), (dict(ws=FAKE + 8), WORKSPACE),
    (dict(wsb=1024), WORKSPACE),
])
@pytest.mark.parametrize("timed", [False, True])
def test_marginal_topk_rejects(over, code, timed):
    assert _marginal(timed, **over) == code


def _expand(**over):
    a = dict(h=FAKE, root=FAKE, topk=FAKE, emb=FAKE, gh=None, ge=None, wg=FAKE, wu=FAKE, wd=FAKE, lm=FAKE,
             b=1, gamma=16, d=4096, I=4096, V=151936, k=8, topk2=32, it=1.0, eps=1e-6, dt=BF16,
             ci=FAKE2, cl=FAKE2, lse=None, ws=FAKE, wsb=1 << 40, st=None)
    a.update(over)
    return binding.lib().treeflash_arapprox_expand(
        a["h"], a["root"], a["topk"], a["emb"], a["gh"], a["ge"], a["wg"], a["wu"], a["wd"], a["lm"], a["b"],
        a["gamma"], a["d"], a["I"], a["V"], a["k"], a["topk2"], a["it"], a["eps"], a["dt"], a["ci"], a["cl"],
        a["lse"], a["ws"], a["wsb"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(h=None), INVALID), (dict(root=None), INVALID), (dict(topk=None), INVALID), (dict(emb=None), INVALID),
    (dict(wg=None), INVALID), (dict(wd=None), INVALID), (dict(lm=None), INVALID),
    (dict(ci=None), INVALID), (dict(cl=None), INVALID), (dict(I=0), INVALID), (dict(I=100), UNSUPPORTED),
    (dict(topk2=0), INVALID), (dict(topk2=151937), INVALID), (dict(topk2=2048), INVALID),
    (dict(eps=-1.0), INVALID), (dict(eps=float("nan")), INVALID), (dict(it=0.0), INVALID),
    (dict(gh=FAKE + 1), INVALID), (dict(lse=FAKE + 2), INVALID), (dict(gamma=300), INVALID),
    (dict(wd=FAKE + 4), UNSUPPORTED), (dict(lm=FAKE + 8), UNSUPPORTED), (dict(ci=FAKE + 1), INVALID),
    (dict(wd=FAKE + 1), INVALID), (dict(d=4090), UNSUPPORTED),
    (dict(ws=None), WORKSPACE), (dict(wsb=4096), WORKSPACE),
    # no up projection (the plain SiLU MLP) is a valid request: the workspace check comes next
    (dict(wu=None, wsb=4096), WORKSPACE), (dict(wu=None, wg=None), INVALID),
])
def test_arapprox_expand_rejects(over, code):
    assert _expand(**over) == code


def _hidden(**over):
    a = dict(h=FAKE, root=FAKE, topk=FAKE, emb=FAKE, gh=None, ge=None, wg=FAKE, wu=FAKE, wd=FAKE,
             b=1, gamma=16, d=4096, I=4096, V=151936, k=8, eps=1e-6, dt=BF16, hp=FAKE2, ws=FAKE, wsb=1 << 40,
             st=None)
    a.update(over)
    return binding.lib().treeflash_arapprox_hidden(
        a["h"], a["root"], a["topk"], a["emb"], a["gh"], a["ge"], a["wg"], a["wu"], a["wd"], a["b"], a["gamma"],
        a["d"], a["I"], a["V"], a["k"], a["eps"], a["dt"], a["hp"], a["ws"], a["wsb"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(h=None), INVALID), (dict(root=None), INVALID), (dict(topk=None), INVALID), (dict(emb=None), INVALID),
    (dict(wg=None), INVALID), (dict(wd=None), INVALID), (dict(hp=None), INVALID),
    (dict(hp=FAKE2 + 2), UNSUPPORTED), (dict(hp=FAKE2 + 1), INVALID), (dict(I=24), UNSUPPORTED),
    (dict(eps=float("inf")), INVALID), (dict(k=0), INVALID), (dict(ws=None), WORKSPACE), (dict(wsb=100), WORKSPACE),
    (dict(wu=None, wsb=100), WORKSPACE), (dict(wu=FAKE + 4), UNSUPPORTED), (dict(dt=F32, wu=FAKE + 2), INVALID),
])
def test_arapprox_hidden_rejects(over, code):
    assert _hidden(**over) == code


def _linear(**over):
    a = dict(h=FAKE, root=FAKE, topk=FAKE, emb=FAKE, gh=None, ge=None, wl=FAKE,
             b=1, gamma=16, d=4096, V=151936, k=8, eps=1e-6, dt=BF16, hp=FAKE2, ws=FAKE, wsb=1 << 40, st=None)
    a.update(over)
    return binding.lib().treeflash_arapprox_linear_hidden(
        a["h"], a["root"], a["topk"], a["emb"], a["gh"], a["ge"], a["wl"], a["b"], a["gamma"], a["d"], a["V"],
        a["k"], a["eps"], a["dt"], a["hp"], a["ws"], a["wsb"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(h=None), INVALID), (dict(root=None), INVALID), (dict(topk=None), INVALID), (dict(emb=None), INVALID),
    (dict(wl=None), INVALID), (dict(wl=FAKE + 8), UNSUPPORTED), (dict(hp=None), INVALID),
    (dict(hp=FAKE2 + 2), UNSUPPORTED), (dict(d=24), UNSUPPORTED), (dict(d=-16), INVALID),
    (dict(eps=float("inf")), INVALID), (dict(k=0), INVALID), (dict(k=2000), INVALID),
    (dict(gamma=300), INVALID), (dict(dt=7), INVALID), (dict(gh=FAKE + 1), INVALID),
    (dict(ws=None), WORKSPACE), (dict(ws=FAKE + 8), WORKSPACE), (dict(wsb=100), WORKSPACE),
])
def test_arapprox_linear_hidden_rejects(over, code):
    assert _linear(**over) == code


def test_linear_workspace_fits_in_the_swiglu_one():
    # the linear variant's workspace (any SwiGLU width stands in) never exceeds
    # what treeflash_workspace_bytes gives for the smallest width
    for (b, gamma, d, V, k) in [(1, 16, 4096, 151936, 8), (16, 16, 4096, 151936, 8), (1, 4, 64, 1000, 3),
                                (4, 7, 2560, 151936, 32)]:
        n16 = binding.lib().treeflash_workspace_bytes(b, gamma, d, 16, V, k, 8, BF16)
        assert n16 > 0
        # one byte short of it is refused before any launch
        assert _linear(b=b, gamma=gamma, d=d, V=V, k=k, wsb=n16 - 1) == WORKSPACE


def _hidden2(**over):
    a = dict(h=FAKE, ctx=FAKE, root=FAKE, topk=FAKE, emb=FAKE, gh=None, ge=None, wg=FAKE, wu=FAKE, wd=FAKE,
             b=1, gamma=16, d=4096, I=4096, V=151936, k=8, eps=1e-6, dt=BF16, hp=FAKE2, ws=FAKE, wsb=1 << 40,
             st=None)
    a.update(over)
    return binding.lib().treeflash_arapprox_2prev_hidden(
        a["h"], a["ctx"], a["root"], a["topk"], a["emb"], a["gh"], a["ge"], a["wg"], a["wu"], a["wd"], a["b"],
        a["gamma"], a["d"], a["I"], a["V"], a["k"], a["eps"], a["dt"], a["hp"], a["ws"], a["wsb"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(h=None), INVALID), (dict(ctx=None), INVALID), (dict(ctx=FAKE + 2), INVALID), (dict(root=None), INVALID),
    (dict(topk=None), INVALID), (dict(emb=None), INVALID), (dict(wg=None), INVALID), (dict(wu=FAKE + 8), UNSUPPORTED),
    (dict(wu=None), INVALID), (dict(hp=None), INVALID), (dict(I=24), UNSUPPORTED), (dict(k=0), INVALID),
    (dict(gamma=256), INVALID),
    # 32 * (1 + 64 + 14 * 64 * 64) bigram rows exceed the 2^20 row limit
    (dict(b=32, k=64), INVALID),
    (dict(ws=None), WORKSPACE), (dict(wsb=4096), WORKSPACE),
])
def test_arapprox_2prev_hidden_rejects(over, code):
    assert _hidden2(**over) == code


def test_workspace_2prev_covers_the_bigram_rows():
    lib = binding.lib()
    for (b, gamma, d, I, V, k) in [(1, 16, 4096, 4096, 151936, 8), (2, 5, 96, 64, 1000, 3), (3, 1, 64, 32, 300, 2)]:
        two = lib.treeflash_workspace_bytes_2prev(b, gamma, d, I, V, k, 8, BF16)
        assert two > 0
        assert _hidden2(b=b, gamma=gamma, d=d, I=I, V=V, k=k, wsb=two - 1) == WORKSPACE
    assert lib.treeflash_workspace_bytes_2prev(32, 16, 4096, 4096, 151936, 64, 8, BF16) == 0


def _tree2(**over):
    a = dict(ci=FAKE, cl=FAKE, tk=FAKE, b=1, gamma=16, k=8, topk2=32, B=32, tok=FAKE2, par=FAKE2, dep=FAKE2,
             sc=FAKE2, cr=None, st=None)
    a.update(over)
    return binding.lib().treeflash_build_tree_2prev(a["ci"], a["cl"], a["tk"], a["b"], a["gamma"], a["k"],
                                                    a["topk2"], a["B"], a["tok"], a["par"], a["dep"], a["sc"],
                                                    a["cr"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(ci=None), INVALID), (dict(tk=None), INVALID), (dict(sc=None), INVALID), (dict(B=0), INVALID),
    (dict(B=5000), INVALID), (dict(k=0), INVALID), (dict(cr=FAKE + 2), INVALID),
    (dict(b=32, k=64), INVALID),
    (dict(gamma=2, k=2, topk2=4, B=13), INVALID),
])
def test_build_tree_2prev_rejects(over, code):
    assert _tree2(**over) == code


def test_binding_checks_row_counts_before_calling():
    # [1, R, topk2] rows that do not match the candidates are refused in Python
    import torch
    ci = torch.zeros((1, 7, 4), dtype=torch.int32)
    tk = torch.zeros((1, 3, 2), dtype=torch.int32)
    with pytest.raises(ValueError):
        binding.treeflash_build_tree(ci, ci.float(), tk, 4)
    with pytest.raises(ValueError):
        binding.treeflash_build_tree_2prev(ci, ci.float(), tk, 4)


def _tree(**over):
    a = dict(ci=FAKE, cl=FAKE, tk=FAKE, b=1, gamma=16, k=8, topk2=32, B=32, tok=FAKE2, par=FAKE2, dep=FAKE2,
             sc=FAKE2, cr=None, st=None)
    a.update(over)
    return binding.lib().treeflash_build_tree(a["ci"], a["cl"], a["tk"], a["b"], a["gamma"], a["k"], a["topk2"],
                                              a["B"], a["tok"], a["par"], a["dep"], a["sc"], a["cr"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(ci=None), INVALID), (dict(cl=None), INVALID), (dict(tk=None), INVALID), (dict(tok=None), INVALID),
    (dict(par=None), INVALID), (dict(dep=None), INVALID), (dict(sc=None), INVALID), (dict(B=0), INVALID),
    (dict(B=5000), INVALID), (dict(b=0), INVALID), (dict(k=0), INVALID), (dict(topk2=0), INVALID),
    (dict(cr=FAKE + 2), INVALID), (dict(tk=FAKE + 1), INVALID),
    # rows shorter than B must be full rows able to hold B nodes: 4 * (1 + 2) = 12 < 13
    (dict(gamma=2, k=2, topk2=4, B=13), INVALID),
    # the frontier and node arrays of a very large budget do not fit in LDS
    (dict(gamma=200, k=200, topk2=4000, B=4000), UNSUPPORTED),
])
def test_build_tree_rejects(over, code):
    assert _tree(**over) == code


def test_binding_refuses_cpu_tensors():
    import torch
    h = torch.zeros(1, 2, 16, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        binding.treeflash_marginal_topk(h, torch.zeros(8, 16, dtype=torch.bfloat16), 2,
                                        workspace=torch.zeros(1 << 16, dtype=torch.uint8),
                                        topk_idx=torch.zeros(1, 2, 2, dtype=torch.int32),
                                        topk_logprob=torch.zeros(1, 2, 2))


def _margtree(**over):
    a = dict(idx=FAKE, lp=FAKE2, b=1, gamma=16, K=32, B=32, tok=FAKE, par=FAKE, dep=FAKE, sc=FAKE2, crow=None,
             st=None)
    a.update(over)
    return binding.lib().treeflash_build_tree_marginal(a["idx"], a["lp"], a["b"], a["gamma"], a["K"], a["B"],
                                                       a["tok"], a["par"], a["dep"], a["sc"], a["crow"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(idx=None), INVALID), (dict(lp=None), INVALID), (dict(tok=None), INVALID), (dict(sc=None), INVALID),
    (dict(b=0), INVALID), (dict(gamma=0), INVALID), (dict(gamma=256), INVALID), (dict(K=0), INVALID),
    (dict(K=5000), INVALID), (dict(B=0), INVALID), (dict(B=4096), INVALID),
    (dict(gamma=2, K=2, B=7), INVALID),          # only 2 + 4 paths exist
    (dict(idx=FAKE + 2), INVALID), (dict(crow=FAKE + 1), INVALID),
    (dict(gamma=200, K=4000, B=4000), UNSUPPORTED),
])
def test_build_tree_marginal_rejects(over, code):
    assert _margtree(**over) == code


def _attn(**over):
    a = dict(root=FAKE, tok=FAKE, par=FAKE, dep=FAKE, b=1, B=32, otok=FAKE2, opos=FAKE2, mask=FAKE2, st=None)
    a.update(over)
    return binding.lib().treeflash_tree_attention_inputs(a["root"], a["tok"], a["par"], a["dep"], a["b"], a["B"],
                                                         a["otok"], a["opos"], a["mask"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(root=None), INVALID), (dict(tok=None), INVALID), (dict(par=None), INVALID), (dict(dep=None), INVALID),
    (dict(otok=None), INVALID), (dict(mask=None), INVALID), (dict(b=0), INVALID), (dict(B=0), INVALID),
    (dict(B=4096), INVALID), (dict(par=FAKE + 2), INVALID), (dict(opos=FAKE2 + 1), INVALID),
])
def test_tree_attention_inputs_rejects(over, code):
    assert _attn(**over) == code


def _accept(**over):
    a = dict(tok=FAKE, par=FAKE, tgt=FAKE, b=1, B=32, gamma=16, acc=FAKE2, alen=FAKE2, bonus=FAKE2, st=None)
    a.update(over)
    return binding.lib().treeflash_accept(a["tok"], a["par"], a["tgt"], a["b"], a["B"], a["gamma"], a["acc"],
                                          a["alen"], a["bonus"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(tok=None), INVALID), (dict(tgt=None), INVALID), (dict(acc=None), INVALID), (dict(bonus=None), INVALID),
    (dict(b=0), INVALID), (dict(B=0), INVALID), (dict(B=5000), INVALID), (dict(gamma=0), INVALID),
    (dict(gamma=256), INVALID), (dict(tgt=FAKE + 2), INVALID),
])
def test_accept_rejects(over, code):
    assert _accept(**over) == code


def _static(**over):
    a = dict(h=FAKE, w=FAKE, b=1, gamma=16, d=4096, V=151936, k=8, it=1.0, dt=BF16, idx=FAKE2, lp=None,
             lse=None, st=None)
    a.update(over)
    return binding.lib().treeflash_marginal_topk_static(a["h"], a["w"], a["b"], a["gamma"], a["d"], a["V"], a["k"],
                                                        a["it"], a["dt"], a["idx"], a["lp"], a["lse"], a["st"])


@pytest.mark.parametrize("over,code", [
    (dict(h=None), INVALID), (dict(w=None), INVALID), (dict(idx=None), INVALID), (dict(b=0), INVALID),
    (dict(d=4090), UNSUPPORTED), (dict(k=0), INVALID), (dict(it=0.0), INVALID), (dict(dt=3), INVALID),
    (dict(h=FAKE + 4), UNSUPPORTED), (dict(lp=FAKE + 2), INVALID),
    # 16 sequences x 121 rows need more scratch than the library's array holds
    (dict(b=16, gamma=121, k=32), WORKSPACE),
])
def test_marginal_topk_static_rejects(over, code):
    assert _static(**over) == code


def test_static_scratch_size():
    assert binding.lib().treeflash_static_scratch_bytes() == 16 << 20
