"""Thin Python binding of ``libtreeflash.so`` (argument marshalling only).

The functions carry the C names; they take torch tensors on the GPU, check
dtypes/devices/contiguity, allocate outputs with torch when none are given,
and pass raw device pointers plus the current HIP stream to the library.  All
arithmetic happens in the library's kernels; there is no fallback path: if
the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtreeflash.so")

TF_F32, TF_BF16 = 0, 1
STATUS = {0: "TF_OK", 1: "TF_ERR_INVALID_ARG", 2: "TF_ERR_UNSUPPORTED", 3: "TF_ERR_WORKSPACE", 4: "TF_ERR_HIP"}
EXPORTED = ("treeflash_workspace_bytes", "treeflash_marginal_topk", "treeflash_marginal_topk_timed",
            "treeflash_marginal_topk_static", "treeflash_static_scratch_bytes",
            "treeflash_arapprox_hidden", "treeflash_arapprox_linear_hidden", "treeflash_arapprox_expand",
            "treeflash_build_tree",
            "treeflash_build_tree_marginal", "treeflash_tree_attention_inputs", "treeflash_accept",
            "treeflash_workspace_bytes_2prev", "treeflash_arapprox_2prev_hidden", "treeflash_build_tree_2prev",
            "treeflash_status_string")

_lib = None


class TreeflashError(RuntimeError):
    def __init__(self, func: str, status: int):
        self.status = status
        super().__init__(f"{func} failed: {STATUS.get(status, status)} ({status_string(status)})")


def lib() -> ctypes.CDLL:
    """Load the library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_03819_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, I, F, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    L.treeflash_workspace_bytes.argtypes = [I, I, I, I, I, I, I, I]
    L.treeflash_workspace_bytes.restype = S
    L.treeflash_marginal_topk.argtypes = [P, P, I, I, I, I, I, F, I, P, P, P, P, S, P]
    L.treeflash_marginal_topk.restype = I
    L.treeflash_marginal_topk_timed.argtypes = [P, P, I, I, I, I, I, F, I, P, P, P, P, S, P, P, P]
    L.treeflash_marginal_topk_timed.restype = I
    L.treeflash_marginal_topk_static.argtypes = [P, P, I, I, I, I, I, F, I, P, P, P, P]
    L.treeflash_marginal_topk_static.restype = I
    L.treeflash_static_scratch_bytes.argtypes = []
    L.treeflash_static_scratch_bytes.restype = S
    L.treeflash_arapprox_hidden.argtypes = [P, P, P, P, P, P, P, P, P, I, I, I, I, I, I, F, I, P, P, S, P]
    L.treeflash_arapprox_hidden.restype = I
    L.treeflash_arapprox_linear_hidden.argtypes = [P, P, P, P, P, P, P, I, I, I, I, I, F, I, P, P, S, P]
    L.treeflash_arapprox_linear_hidden.restype = I
    L.treeflash_arapprox_expand.argtypes = [P, P, P, P, P, P, P, P, P, P, I, I, I, I, I, I, I, F, F, I,
                                            P, P, P, P, S, P]
    L.treeflash_arapprox_expand.restype = I
    L.treeflash_build_tree.argtypes = [P, P, P, I, I, I, I, I, P, P, P, P, P, P]
    L.treeflash_build_tree.restype = I
    L.treeflash_build_tree_marginal.argtypes = [P, P, I, I, I, I, P, P, P, P, P, P]
    L.treeflash_build_tree_marginal.restype = I
    L.treeflash_tree_attention_inputs.argtypes = [P, P, P, P, I, I, P, P, P, P]
    L.treeflash_tree_attention_inputs.restype = I
    L.treeflash_accept.argtypes = [P, P, P, I, I, I, P, P, P, P]
    L.treeflash_accept.restype = I
    L.treeflash_workspace_bytes_2prev.argtypes = [I, I, I, I, I, I, I, I]
    L.treeflash_workspace_bytes_2prev.restype = S
    L.treeflash_arapprox_2prev_hidden.argtypes = [P, P, P, P, P, P, P, P, P, P, I, I, I, I, I, I, F, I, P, P, S, P]
    L.treeflash_arapprox_2prev_hidden.restype = I
    L.treeflash_build_tree_2prev.argtypes = [P, P, P, I, I, I, I, I, P, P, P, P, P, P]
    L.treeflash_build_tree_2prev.restype = I
    L.treeflash_status_string.argtypes = [I]
    L.treeflash_status_string.restype = ctypes.c_char_p
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().treeflash_status_string(int(status)).decode()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return TF_BF16
    if t.dtype == torch.float32:
        return TF_F32
    raise TypeError(f"unsupported dtype {t.dtype}; expected bfloat16 or float32")


def _ptr(t: Optional[torch.Tensor], name: str, dtype=None, device=None) -> Optional[int]:
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _shapes(func: str, **want):
    """Raise unless every tensor has the shape the library will read it with."""
    for name, (t, shape) in want.items():
        if t is not None and tuple(t.shape) != tuple(shape):
            raise ValueError(f"{func}: {name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _check(func: str, status: int):
    if status != 0:
        raise TreeflashError(func, status)


def treeflash_workspace_bytes(b, gamma, d, I, V, k, topk2, dtype) -> int:
    code = dtype if isinstance(dtype, int) else (TF_BF16 if dtype == torch.bfloat16 else TF_F32)
    return int(lib().treeflash_workspace_bytes(b, gamma, d, I, V, k, topk2, code))


def alloc_workspace(nbytes: int, device) -> torch.Tensor:
    """Workspace as a torch byte buffer (PyTorch owns device memory)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def treeflash_marginal_topk(h: torch.Tensor, lm_head: torch.Tensor, k: int, inv_temperature: float = 1.0,
                            workspace: Optional[torch.Tensor] = None, topk_idx: Optional[torch.Tensor] = None,
                            topk_logprob: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                            events: Optional[tuple] = None):
    """Stage 1: top-k ids and log-probs of LMHead(h) per draft depth (any [b, rows, d]).

    `events`: optional pair of raw hipEvent_t handles recorded around the
    LM-head kernel (treeflash_marginal_topk_timed)."""
    b, gamma, d = h.shape
    V = lm_head.shape[0]
    dev = h.device
    dt = _dtype_code(h)
    if lm_head.shape != (V, d):
        raise ValueError("lm_head must be [V, d]")
    if topk_idx is None:
        topk_idx = torch.empty((b, gamma, k), dtype=torch.int32, device=dev)
    if topk_logprob is None:
        topk_logprob = torch.empty((b, gamma, k), dtype=torch.float32, device=dev)
    if workspace is None:
        # stage-1 scratch for b * gamma rows (gamma may count more rows than a draft depth)
        workspace = alloc_workspace(treeflash_workspace_bytes(b * gamma, 1, d, 16, V, k, min(k, V), dt), dev)
    args = (_ptr(h, "h", device=dev), _ptr(lm_head, "lm_head", h.dtype, dev), b, gamma, d, V, k,
            float(inv_temperature), dt, _ptr(topk_idx, "topk_idx", torch.int32, dev),
            _ptr(topk_logprob, "topk_logprob", torch.float32, dev), _ptr(lse, "lse", torch.float32, dev),
            _ptr(workspace, "workspace", device=dev), workspace.numel() * workspace.element_size(), _stream(dev))
    if events is None:
        _check("treeflash_marginal_topk", lib().treeflash_marginal_topk(*args))
    else:
        _check("treeflash_marginal_topk_timed", lib().treeflash_marginal_topk_timed(*args, events[0], events[1]))
    return topk_idx, topk_logprob


def treeflash_marginal_topk_static(h: torch.Tensor, lm_head: torch.Tensor, k: int, inv_temperature: float = 1.0,
                                   topk_idx: Optional[torch.Tensor] = None,
                                   topk_logprob: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None):
    """treeflash_marginal_topk with the library's own device scratch (no workspace)."""
    b, gamma, d = h.shape
    V = lm_head.shape[0]
    dev = h.device
    dt = _dtype_code(h)
    if lm_head.shape != (V, d):
        raise ValueError("lm_head must be [V, d]")
    if topk_idx is None:
        topk_idx = torch.empty((b, gamma, k), dtype=torch.int32, device=dev)
    if topk_logprob is None:
        topk_logprob = torch.empty((b, gamma, k), dtype=torch.float32, device=dev)
    _check("treeflash_marginal_topk_static", lib().treeflash_marginal_topk_static(
        _ptr(h, "h", device=dev), _ptr(lm_head, "lm_head", h.dtype, dev), b, gamma, d, V, k,
        float(inv_temperature), dt, _ptr(topk_idx, "topk_idx", torch.int32, dev),
        _ptr(topk_logprob, "topk_logprob", torch.float32, dev), _ptr(lse, "lse", torch.float32, dev), _stream(dev)))
    return topk_idx, topk_logprob


def treeflash_arapprox_hidden(h, root_token, topk_idx, emb, norm_h_gain, norm_e_gain, w_gate, w_up, w_down,
                              rms_eps: float = 1e-6, workspace: Optional[torch.Tensor] = None,
                              hprime: Optional[torch.Tensor] = None, V: Optional[int] = None):
    """Eq. 1 for every conditional row: h' [b, R, d] (w_up None: the plain SiLU MLP)."""
    b, gamma, d = h.shape
    k = topk_idx.shape[2]
    V = emb.shape[0] if V is None else V
    I = w_gate.shape[0]
    R = 1 + (gamma - 1) * k
    _shapes("treeflash_arapprox_hidden", root_token=(root_token, (b,)), topk_idx=(topk_idx, (b, gamma, k)),
            emb=(emb, (V, d)), w_gate=(w_gate, (I, 2 * d)), w_up=(w_up, (I, 2 * d)), w_down=(w_down, (d, I)),
            hprime=(hprime, (b, R, d)))
    dev = h.device
    dt = _dtype_code(h)
    if hprime is None:
        hprime = torch.empty((b, R, d), dtype=h.dtype, device=dev)
    if workspace is None:
        workspace = alloc_workspace(treeflash_workspace_bytes(b, gamma, d, I, V, k, 1, dt), dev)
    st = lib().treeflash_arapprox_hidden(
        _ptr(h, "h", device=dev), _ptr(root_token, "root_token", torch.int32, dev),
        _ptr(topk_idx, "topk_idx", torch.int32, dev), _ptr(emb, "emb", h.dtype, dev),
        _ptr(norm_h_gain, "norm_h_gain", h.dtype, dev), _ptr(norm_e_gain, "norm_e_gain", h.dtype, dev),
        _ptr(w_gate, "w_gate", h.dtype, dev), _ptr(w_up, "w_up", h.dtype, dev), _ptr(w_down, "w_down", h.dtype, dev),
        b, gamma, d, I, V, k, float(rms_eps), dt, _ptr(hprime, "hprime", h.dtype, dev),
        _ptr(workspace, "workspace", device=dev), workspace.numel() * workspace.element_size(), _stream(dev))
    _check("treeflash_arapprox_hidden", st)
    return hprime


def treeflash_arapprox_linear_hidden(h, root_token, topk_idx, emb, norm_h_gain, norm_e_gain, w_lin,
                                     rms_eps: float = 1e-6, workspace: Optional[torch.Tensor] = None,
                                     hprime: Optional[torch.Tensor] = None, V: Optional[int] = None):
    """The w/ Linear approximator for every conditional row: h' [b, R, d]."""
    b, gamma, d = h.shape
    k = topk_idx.shape[2]
    V = emb.shape[0] if V is None else V
    R = 1 + (gamma - 1) * k
    _shapes("treeflash_arapprox_linear_hidden", root_token=(root_token, (b,)), topk_idx=(topk_idx, (b, gamma, k)),
            emb=(emb, (V, d)), w_lin=(w_lin, (d, 2 * d)), hprime=(hprime, (b, R, d)))
    dev = h.device
    dt = _dtype_code(h)
    if hprime is None:
        hprime = torch.empty((b, R, d), dtype=h.dtype, device=dev)
    if workspace is None:
        workspace = alloc_workspace(treeflash_workspace_bytes(b, gamma, d, 16, V, k, 1, dt), dev)
    st = lib().treeflash_arapprox_linear_hidden(
        _ptr(h, "h", device=dev), _ptr(root_token, "root_token", torch.int32, dev),
        _ptr(topk_idx, "topk_idx", torch.int32, dev), _ptr(emb, "emb", h.dtype, dev),
        _ptr(norm_h_gain, "norm_h_gain", h.dtype, dev), _ptr(norm_e_gain, "norm_e_gain", h.dtype, dev),
        _ptr(w_lin, "w_lin", h.dtype, dev), b, gamma, d, V, k, float(rms_eps), dt,
        _ptr(hprime, "hprime", h.dtype, dev), _ptr(workspace, "workspace", device=dev),
        workspace.numel() * workspace.element_size(), _stream(dev))
    _check("treeflash_arapprox_linear_hidden", st)
    return hprime


def treeflash_workspace_bytes_2prev(b, gamma, d, I, V, k, topk2, dtype) -> int:
    code = dtype if isinstance(dtype, int) else (TF_BF16 if dtype == torch.bfloat16 else TF_F32)
    return int(lib().treeflash_workspace_bytes_2prev(b, gamma, d, I, V, k, topk2, code))


def treeflash_arapprox_2prev_hidden(h, context_token, root_token, topk_idx, emb, norm_h_gain, norm_e_gain, w_gate,
                                    w_up, w_down, rms_eps: float = 1e-6, workspace: Optional[torch.Tensor] = None,
                                    hprime: Optional[torch.Tensor] = None, V: Optional[int] = None):
    """The w/ 2-prev approximator for every bigram row: h' [b, R2, d]."""
    b, gamma, d = h.shape
    k = topk_idx.shape[2]
    V = emb.shape[0] if V is None else V
    I = w_gate.shape[0]
    R = 1 if gamma == 1 else 1 + k + (gamma - 2) * k * k
    _shapes("treeflash_arapprox_2prev_hidden", context_token=(context_token, (b,)), root_token=(root_token, (b,)),
            topk_idx=(topk_idx, (b, gamma, k)), emb=(emb, (V, d)), w_gate=(w_gate, (I, 3 * d)),
            w_up=(w_up, (I, 3 * d)), w_down=(w_down, (d, I)), hprime=(hprime, (b, R, d)))
    dev = h.device
    dt = _dtype_code(h)
    if hprime is None:
        hprime = torch.empty((b, R, d), dtype=h.dtype, device=dev)
    if workspace is None:
        workspace = alloc_workspace(treeflash_workspace_bytes_2prev(b, gamma, d, I, V, k, 1, dt), dev)
    st = lib().treeflash_arapprox_2prev_hidden(
        _ptr(h, "h", device=dev), _ptr(context_token, "context_token", torch.int32, dev),
        _ptr(root_token, "root_token", torch.int32, dev), _ptr(topk_idx, "topk_idx", torch.int32, dev),
        _ptr(emb, "emb", h.dtype, dev), _ptr(norm_h_gain, "norm_h_gain", h.dtype, dev),
        _ptr(norm_e_gain, "norm_e_gain", h.dtype, dev), _ptr(w_gate, "w_gate", h.dtype, dev),
        _ptr(w_up, "w_up", h.dtype, dev), _ptr(w_down, "w_down", h.dtype, dev), b, gamma, d, I, V, k,
        float(rms_eps), dt, _ptr(hprime, "hprime", h.dtype, dev), _ptr(workspace, "workspace", device=dev),
        workspace.numel() * workspace.element_size(), _stream(dev))
    _check("treeflash_arapprox_2prev_hidden", st)
    return hprime


def treeflash_arapprox_expand(h, root_token, topk_idx, emb, norm_h_gain, norm_e_gain, w_gate, w_up, w_down,
                              lm_head, topk2: int, inv_temperature: float = 1.0, rms_eps: float = 1e-6,
                              workspace: Optional[torch.Tensor] = None, cond_idx=None, cond_logprob=None,
                              cond_lse=None, want_lse: bool = True):
    """Stage 2: Eq. 1 on every conditional row (w_up None: the plain SiLU MLP),
    LM head, log-softmax, top-topk2."""
    b, gamma, d = h.shape
    k = topk_idx.shape[2]
    V = lm_head.shape[0]
    I = w_gate.shape[0]
    R = 1 + (gamma - 1) * k
    _shapes("treeflash_arapprox_expand", root_token=(root_token, (b,)), topk_idx=(topk_idx, (b, gamma, k)),
            emb=(emb, (V, d)), w_gate=(w_gate, (I, 2 * d)), w_up=(w_up, (I, 2 * d)), w_down=(w_down, (d, I)),
            lm_head=(lm_head, (V, d)), cond_idx=(cond_idx, (b, R, topk2)), cond_logprob=(cond_logprob, (b, R, topk2)))
    dev = h.device
    dt = _dtype_code(h)
    if cond_idx is None:
        cond_idx = torch.empty((b, R, topk2), dtype=torch.int32, device=dev)
    if cond_logprob is None:
        cond_logprob = torch.empty((b, R, topk2), dtype=torch.float32, device=dev)
    if cond_lse is None and want_lse:
        cond_lse = torch.empty((b, R), dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = alloc_workspace(treeflash_workspace_bytes(b, gamma, d, I, V, k, topk2, dt), dev)
    st = lib().treeflash_arapprox_expand(
        _ptr(h, "h", device=dev), _ptr(root_token, "root_token", torch.int32, dev),
        _ptr(topk_idx, "topk_idx", torch.int32, dev), _ptr(emb, "emb", h.dtype, dev),
        _ptr(norm_h_gain, "norm_h_gain", h.dtype, dev), _ptr(norm_e_gain, "norm_e_gain", h.dtype, dev),
        _ptr(w_gate, "w_gate", h.dtype, dev), _ptr(w_up, "w_up", h.dtype, dev), _ptr(w_down, "w_down", h.dtype, dev),
        _ptr(lm_head, "lm_head", h.dtype, dev), b, gamma, d, I, V, k, topk2, float(inv_temperature),
        float(rms_eps), dt, _ptr(cond_idx, "cond_idx", torch.int32, dev),
        _ptr(cond_logprob, "cond_logprob", torch.float32, dev), _ptr(cond_lse, "cond_lse", torch.float32, dev),
        _ptr(workspace, "workspace", device=dev), workspace.numel() * workspace.element_size(), _stream(dev))
    _check("treeflash_arapprox_expand", st)
    return cond_idx, cond_logprob, cond_lse


def _build_tree(func: str, rows_of, cond_idx, cond_logprob, topk_idx, B, out):
    b, R, topk2 = cond_idx.shape
    gamma, k = topk_idx.shape[1], topk_idx.shape[2]
    if R != rows_of(gamma, k) or cond_logprob.shape != cond_idx.shape or topk_idx.shape[0] != b:
        raise ValueError(f"{func}: rows {tuple(cond_idx.shape)} do not match candidates {tuple(topk_idx.shape)}")
    dev = cond_idx.device
    if out is None:
        out = _tree_buffers(b, B, dev)
    st = getattr(lib(), func)(
        _ptr(cond_idx, "cond_idx", torch.int32, dev), _ptr(cond_logprob, "cond_logprob", torch.float32, dev),
        _ptr(topk_idx, "topk_idx", torch.int32, dev), b, gamma, k, topk2, B,
        _ptr(out["token"], "token", torch.int32, dev), _ptr(out["parent"], "parent", torch.int32, dev),
        _ptr(out["depth"], "depth", torch.int32, dev), _ptr(out["score"], "score", torch.float32, dev),
        _ptr(out.get("child_row"), "child_row", torch.int32, dev), _stream(dev))
    _check(func, st)
    return out


def treeflash_build_tree(cond_idx, cond_logprob, topk_idx, B: int, out: Optional[Dict[str, torch.Tensor]] = None):
    """Part 2: best-first selection of B nodes per sequence (pop order)."""
    return _build_tree("treeflash_build_tree", lambda g, k: 1 + (g - 1) * k, cond_idx, cond_logprob, topk_idx, B,
                       out)


def treeflash_build_tree_2prev(cond_idx, cond_logprob, topk_idx, B: int,
                               out: Optional[Dict[str, torch.Tensor]] = None):
    """Part 2 over the bigram rows of the w/ 2-prev approximator."""
    return _build_tree("treeflash_build_tree_2prev", lambda g, k: 1 if g == 1 else 1 + k + (g - 2) * k * k,
                       cond_idx, cond_logprob, topk_idx, B, out)


def _tree_buffers(b: int, B: int, dev) -> Dict[str, torch.Tensor]:
    return {
        "token": torch.empty((b, B), dtype=torch.int32, device=dev),
        "parent": torch.empty((b, B), dtype=torch.int32, device=dev),
        "depth": torch.empty((b, B), dtype=torch.int32, device=dev),
        "score": torch.empty((b, B), dtype=torch.float32, device=dev),
        "child_row": torch.empty((b, B), dtype=torch.int32, device=dev),
    }


def treeflash_build_tree_marginal(marg_idx, marg_logprob, B: int, out: Optional[Dict[str, torch.Tensor]] = None):
    """Marginal OPT-Tree (the DDTree baseline) from stage-1 lists [b, gamma, K]."""
    b, gamma, K = marg_idx.shape
    dev = marg_idx.device
    if out is None:
        out = _tree_buffers(b, B, dev)
    st = lib().treeflash_build_tree_marginal(
        _ptr(marg_idx, "marg_idx", torch.int32, dev), _ptr(marg_logprob, "marg_logprob", torch.float32, dev),
        b, gamma, K, B, _ptr(out["token"], "token", torch.int32, dev),
        _ptr(out["parent"], "parent", torch.int32, dev), _ptr(out["depth"], "depth", torch.int32, dev),
        _ptr(out["score"], "score", torch.float32, dev), _ptr(out.get("child_row"), "child_row", torch.int32, dev),
        _stream(dev))
    _check("treeflash_build_tree_marginal", st)
    return out


def treeflash_tree_attention_inputs(root_token, tree: Dict[str, torch.Tensor], out: Optional[dict] = None):
    """Verifier input of each draft tree: tokens, positions [b, B+1], ancestor mask [b, B+1, B+1] (uint8)."""
    b, B = tree["token"].shape
    dev = tree["token"].device
    if out is None:
        out = {"tokens": torch.empty((b, B + 1), dtype=torch.int32, device=dev),
               "positions": torch.empty((b, B + 1), dtype=torch.int32, device=dev),
               "mask": torch.empty((b, B + 1, B + 1), dtype=torch.uint8, device=dev)}
    st = lib().treeflash_tree_attention_inputs(
        _ptr(root_token, "root_token", torch.int32, dev), _ptr(tree["token"], "token", torch.int32, dev),
        _ptr(tree["parent"], "parent", torch.int32, dev), _ptr(tree["depth"], "depth", torch.int32, dev), b, B,
        _ptr(out["tokens"], "tokens", torch.int32, dev), _ptr(out["positions"], "positions", torch.int32, dev),
        _ptr(out["mask"], "mask", torch.uint8, dev), _stream(dev))
    _check("treeflash_tree_attention_inputs", st)
    return out


def treeflash_accept(tree: Dict[str, torch.Tensor], target: torch.Tensor, gamma: int, out: Optional[dict] = None):
    """Greedy equality walk given the verifier's next token at every position [b, B+1]."""
    b, B = tree["token"].shape
    dev = tree["token"].device
    if target.shape != (b, B + 1):
        raise ValueError("target must be [b, B+1]")
    if out is None:
        out = {"accepted": torch.empty((b, gamma), dtype=torch.int32, device=dev),
               "accept_len": torch.empty((b,), dtype=torch.int32, device=dev),
               "bonus": torch.empty((b,), dtype=torch.int32, device=dev)}
    st = lib().treeflash_accept(
        _ptr(tree["token"], "token", torch.int32, dev), _ptr(tree["parent"], "parent", torch.int32, dev),
        _ptr(target, "target", torch.int32, dev), b, B, gamma,
        _ptr(out["accepted"], "accepted", torch.int32, dev), _ptr(out["accept_len"], "accept_len", torch.int32, dev),
        _ptr(out["bonus"], "bonus", torch.int32, dev), _stream(dev))
    _check("treeflash_accept", st)
    return out


class MarginalDrafter:
    """The marginal baseline over resident weights: stage 1 with K = min(B, V)
    entries per depth, then the marginal OPT-Tree.  Allocates nothing per step."""

    def __init__(self, lm_head: torch.Tensor, b: int, gamma: int, B: int, inv_temperature: float = 1.0):
        self.lm_head = lm_head
        self.dev = lm_head.device
        self.V, self.d = lm_head.shape
        self.b, self.gamma, self.B = b, gamma, B
        self.K = min(B, self.V)
        self.inv_t = inv_temperature
        nbytes = treeflash_workspace_bytes(b, gamma, self.d, 16, self.V, self.K, self.K, lm_head.dtype)
        if nbytes == 0:
            raise ValueError("invalid drafting shapes")
        self.workspace = alloc_workspace(nbytes, self.dev)
        self.idx = torch.empty((b, gamma, self.K), dtype=torch.int32, device=self.dev)
        self.lp = torch.empty((b, gamma, self.K), dtype=torch.float32, device=self.dev)
        self.tree = _tree_buffers(b, B, self.dev)

    def step(self, h, lm_head=None):
        treeflash_marginal_topk(h, self.lm_head if lm_head is None else lm_head, self.K, self.inv_t,
                                self.workspace, self.idx, self.lp)
        return treeflash_build_tree_marginal(self.idx, self.lp, self.B, self.tree)


class Drafter:
    """One drafting step over resident weights: the three C calls in order.

    Holds the workspace and output buffers so repeated steps allocate nothing.
    With a ``w_lin`` weight (the w/ Linear approximator) stage 2 is
    treeflash_arapprox_linear_hidden into a held h' buffer followed by
    treeflash_marginal_topk on its rows.
    """

    def __init__(self, weights: Dict[str, torch.Tensor], b: int, gamma: int, k: int, B: int,
                 inv_temperature: float = 1.0, rms_eps: float = 1e-6, topk2: Optional[int] = None):
        self.w = weights
        lm = weights["lm_head"]
        self.dev = lm.device
        self.V, self.d = lm.shape
        self.linear = "w_lin" in weights
        self.I = 16 if self.linear else weights["w_gate"].shape[0]
        self.b, self.gamma, self.k, self.B = b, gamma, k, B
        self.topk2 = min(B, self.V) if topk2 is None else topk2
        self.inv_t, self.eps = inv_temperature, rms_eps
        self.R = 1 + (gamma - 1) * k
        dt = lm.dtype
        nbytes = treeflash_workspace_bytes(b, gamma, self.d, self.I, self.V, k, self.topk2, dt)
        if nbytes == 0:
            raise ValueError("invalid drafting shapes")
        self.workspace = alloc_workspace(nbytes, self.dev)
        z = dict(device=self.dev)
        self.topk_idx = torch.empty((b, gamma, k), dtype=torch.int32, **z)
        self.topk_lp = torch.empty((b, gamma, k), dtype=torch.float32, **z)
        self.cond_idx = torch.empty((b, self.R, self.topk2), dtype=torch.int32, **z)
        self.cond_lp = torch.empty((b, self.R, self.topk2), dtype=torch.float32, **z)
        self.cond_lse = torch.empty((b, self.R), dtype=torch.float32, **z)
        self.hprime = torch.empty((b, self.R, self.d), dtype=dt, **z) if self.linear else None
        self.tree = {
            "token": torch.empty((b, B), dtype=torch.int32, **z),
            "parent": torch.empty((b, B), dtype=torch.int32, **z),
            "depth": torch.empty((b, B), dtype=torch.int32, **z),
            "score": torch.empty((b, B), dtype=torch.float32, **z),
            "child_row": torch.empty((b, B), dtype=torch.int32, **z),
        }

    def stage1(self, h, weights=None):
        w = weights or self.w
        return treeflash_marginal_topk(h, w["lm_head"], self.k, self.inv_t, self.workspace,
                                       self.topk_idx, self.topk_lp)

    def stage2(self, h, root, weights=None, topk_idx=None):
        w = weights or self.w
        tk = self.topk_idx if topk_idx is None else topk_idx
        if self.linear:
            treeflash_arapprox_linear_hidden(h, root, tk, w["emb"], w["norm_h_gain"], w["norm_e_gain"], w["w_lin"],
                                             self.eps, self.workspace, self.hprime, self.V)
            treeflash_marginal_topk(self.hprime, w["lm_head"], self.topk2, self.inv_t, self.workspace,
                                    self.cond_idx, self.cond_lp, self.cond_lse)
            return self.cond_idx, self.cond_lp, self.cond_lse
        return treeflash_arapprox_expand(
            h, root, self.topk_idx if topk_idx is None else topk_idx, w["emb"], w["norm_h_gain"],
            w["norm_e_gain"], w["w_gate"], w.get("w_up"), w["w_down"], w["lm_head"], self.topk2, self.inv_t,
            self.eps, self.workspace, self.cond_idx, self.cond_lp, self.cond_lse)

    def tree_build(self, cond_idx=None, cond_lp=None, topk_idx=None):
        return treeflash_build_tree(self.cond_idx if cond_idx is None else cond_idx,
                                    self.cond_lp if cond_lp is None else cond_lp,
                                    self.topk_idx if topk_idx is None else topk_idx, self.B, self.tree)

    def step(self, h, root, weights=None):
        """Stage 1, stage 2 and the tree for every sequence; returns the tree buffers."""
        self.stage1(h, weights)
        self.stage2(h, root, weights)
        return self.tree_build()

    def diagnostics(self) -> int:
        """Slices the last call re-evaluated on the exact slow path (synchronises)."""
        return int(self.workspace[:4].view(torch.int32).item())


class Drafter2Prev(Drafter):
    """A drafting step of the w/ 2-prev approximator (bigram rows): stage 1,
    treeflash_arapprox_2prev_hidden into a held h' buffer, the LM head on its
    rows, treeflash_build_tree_2prev.  The weights' w_gate / w_up are [I, 3d]."""

    def __init__(self, weights: Dict[str, torch.Tensor], b: int, gamma: int, k: int, B: int,
                 inv_temperature: float = 1.0, rms_eps: float = 1e-6, topk2: Optional[int] = None):
        lm = weights["lm_head"]
        V, d = lm.shape
        I = weights["w_gate"].shape[0]
        if weights["w_gate"].shape[1] != 3 * d:
            raise ValueError("w_gate must be [I, 3d] for the 2-prev approximator")
        self.w = weights
        self.dev = lm.device
        self.V, self.d, self.I = V, d, I
        self.linear = False
        self.b, self.gamma, self.k, self.B = b, gamma, k, B
        self.topk2 = min(B, V) if topk2 is None else topk2
        self.inv_t, self.eps = inv_temperature, rms_eps
        self.R = 1 if gamma == 1 else 1 + k + (gamma - 2) * k * k
        nbytes = treeflash_workspace_bytes_2prev(b, gamma, d, I, V, k, self.topk2, lm.dtype)
        if nbytes == 0:
            raise ValueError("invalid drafting shapes")
        self.workspace = alloc_workspace(nbytes, self.dev)
        z = dict(device=self.dev)
        self.topk_idx = torch.empty((b, gamma, k), dtype=torch.int32, **z)
        self.topk_lp = torch.empty((b, gamma, k), dtype=torch.float32, **z)
        self.cond_idx = torch.empty((b, self.R, self.topk2), dtype=torch.int32, **z)
        self.cond_lp = torch.empty((b, self.R, self.topk2), dtype=torch.float32, **z)
        self.cond_lse = torch.empty((b, self.R), dtype=torch.float32, **z)
        self.hprime = torch.empty((b, self.R, d), dtype=lm.dtype, **z)
        self.tree = _tree_buffers(b, B, self.dev)
        self.context = None

    def stage2(self, h, root, weights=None, topk_idx=None, context=None):
        w = weights or self.w
        ctx = self.context if context is None else context
        if ctx is None:
            raise ValueError("the 2-prev rows need the context token before each root")
        tk = self.topk_idx if topk_idx is None else topk_idx
        treeflash_arapprox_2prev_hidden(h, ctx, root, tk, w["emb"], w["norm_h_gain"], w["norm_e_gain"], w["w_gate"],
                                        w["w_up"], w["w_down"], self.eps, self.workspace, self.hprime, self.V)
        treeflash_marginal_topk(self.hprime, w["lm_head"], self.topk2, self.inv_t, self.workspace,
                                self.cond_idx, self.cond_lp, self.cond_lse)
        return self.cond_idx, self.cond_lp, self.cond_lse

    def tree_build(self, cond_idx=None, cond_lp=None, topk_idx=None):
        return treeflash_build_tree_2prev(self.cond_idx if cond_idx is None else cond_idx,
                                          self.cond_lp if cond_lp is None else cond_lp,
                                          self.topk_idx if topk_idx is None else topk_idx, self.B, self.tree)

    def step(self, h, root, weights=None, context=None):
        if context is not None:
            self.context = context
        return super().step(h, root, weights)
