"""Python binding of libptd.so, the MI355X (gfx950) Progressive Tree Drafting
hot path.

The functions named ``ptd_*`` mirror the C entry points of ``include/ptd.h``
one to one: they marshal arguments (torch tensors or raw integer device
addresses, a HIP stream) and raise :class:`PTDError` on a non-zero status.
Every step of the path runs in the library's HIP kernels; torch only provides
device memory and the stream.  There is no CPU fallback: without a built
``libptd.so`` the import fails.

The lower-case helpers (``tree_mask``, ``tree_attention``, ``topk_argmax``,
``verify``, ``expand``, ``verify_expand``, ``tree_rope``, ``kv_commit``,
``verify_sample``, ``step_prune``, the ``Pool`` class) allocate outputs with
torch and call the entry points.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch  # loads the HIP runtime that libptd.so then shares

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libptd.so")

PTD_F32, PTD_BF16 = 0, 1
PTD_ROPE_HALF, PTD_ROPE_INTERLEAVED = 0, 1
PTD_MAX_T, PTD_MAX_K, PTD_MAX_DEPTH = 1024, 16, 64
STATUS = {0: "PTD_OK", 1: "PTD_ERR_NULL", 2: "PTD_ERR_SHAPE", 3: "PTD_ERR_DTYPE",
          4: "PTD_ERR_ALIGN", 5: "PTD_ERR_WORKSPACE", 6: "PTD_ERR_HIP",
          7: "PTD_ERR_BAD_TREE", 8: "PTD_ERR_KV_LEN", 9: "PTD_ERR_BAD_PATH",
          10: "PTD_ERR_PAGE", 11: "PTD_ERR_SCRATCH"}
PTD_NOALLOC_SCRATCH_BYTES = 64 << 20


class PTDError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} "
                         f"({_lib.ptd_status_string(status).decode()})")


class AttnShape(ctypes.Structure):
    """ptd_attn_shape"""
    _fields_ = [("B", ctypes.c_int32), ("Hq", ctypes.c_int32),
                ("Hkv", ctypes.c_int32), ("D", ctypes.c_int32),
                ("L_cap", ctypes.c_int32), ("in_dtype", ctypes.c_int),
                ("out_dtype", ctypes.c_int), ("scale", ctypes.c_float)]


class KVPages(ctypes.Structure):
    """ptd_kv_pages"""
    _fields_ = [("k_pages", ctypes.c_void_p), ("v_pages", ctypes.c_void_p),
                ("page_table", ctypes.c_void_p), ("page_size", ctypes.c_int32),
                ("max_pages", ctypes.c_int32), ("num_pages", ctypes.c_int32)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                      "(hipcc --offload-arch=gfx950)")
_lib = ctypes.CDLL(LIB_PATH)

_vp, _i32, _i64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
_SIGS = {
    "ptd_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "ptd_version": ([], ctypes.c_int),
    "ptd_build_tree_mask": ([_vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp], ctypes.c_int),
    "ptd_tree_attention_workspace_bytes": ([ctypes.POINTER(AttnShape), _i32], _sz),
    "ptd_tree_attention": ([_vp, _vp, _vp, _vp, _vp, _i32, _vp, ctypes.POINTER(AttnShape),
                            _vp, _vp, _sz, _vp, _vp], ctypes.c_int),
    "ptd_tree_attention_ragged": ([_vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp,
                                   ctypes.POINTER(AttnShape), _vp, _vp, _sz, _vp, _vp],
                                  ctypes.c_int),
    "ptd_tree_attention_noalloc": ([_vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp,
                                    ctypes.POINTER(AttnShape), _vp, _vp, _vp], ctypes.c_int),
    "ptd_tree_attention_fp8kv": ([_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp,
                                  ctypes.POINTER(AttnShape), _vp, _sz, _vp, _vp], ctypes.c_int),
    "ptd_tree_attention_paged_fp8kv": ([_vp, ctypes.POINTER(KVPages), _vp, _vp, _vp, _vp, _vp,
                                        _i32, _vp, ctypes.POINTER(AttnShape), _vp, _sz, _vp,
                                        _vp], ctypes.c_int),
    "ptd_tree_attention_paged": ([_vp, ctypes.POINTER(KVPages), _vp, _vp, _vp, _i32, _vp,
                                  ctypes.POINTER(AttnShape), _vp, _vp, _sz, _vp, _vp],
                                 ctypes.c_int),
    "ptd_topk_workspace_bytes": ([_i32, _i32, _i32], _sz),
    "ptd_topk_argmax": ([_vp, ctypes.c_int, _i32, _i32, _i64, _i32, _vp, _vp, _vp, _vp,
                         _sz, _vp], ctypes.c_int),
    "ptd_verify": ([_vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
    "ptd_expand": ([_vp, _vp, _vp, _i32, _i32, _vp, _i32, _vp, _i32, _i32, _vp, _vp, _vp,
                    _vp, _vp], ctypes.c_int),
    "ptd_verify_expand": ([_vp, _vp, _vp, _vp, _i32, _i32, _vp, _i32, _vp, _i32, _i32, _vp,
                           _vp, _vp, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
    "ptd_tree_rope": ([_vp, _vp, _vp, _vp, _i32, ctypes.POINTER(AttnShape), ctypes.c_double,
                       _vp, _i32, _vp, _vp, _vp], ctypes.c_int),
    "ptd_kv_commit": ([_vp, _vp, _vp, _vp, _vp, _i32, ctypes.POINTER(AttnShape), _vp, _vp,
                       _vp], ctypes.c_int),
    "ptd_verify_sample_workspace_bytes": ([_i32, _i32, _i32], _sz),
    "ptd_step_prune": ([_vp, _vp, _vp, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp],
                       ctypes.c_int),
    "ptd_pool_bytes": ([_i32, _i32, _i32], _sz),
    "ptd_pool_init": ([_vp, _sz, _i32, _i32, _i32, _vp], ctypes.c_int),
    "ptd_pool_merge": ([_vp, _sz, _i32, _i32, _i32, _vp, _vp, _vp, _i32, _vp, _vp],
                       ctypes.c_int),
    "ptd_pool_retrieve": ([_vp, _sz, _i32, _i32, _i32, _vp, _i32, _vp, _vp, _vp, _vp],
                          ctypes.c_int),
    "ptd_verify_sample": ([_vp, ctypes.c_int, _i32, _i64, _vp, _vp, _vp, _i32, _i32,
                           ctypes.c_double, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp, _vp],
                          ctypes.c_int),
}
for _name, (_args, _res) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, torch.Tensor):
        return x.data_ptr()
    return int(x)


def _stream(s):
    if s is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, torch.cuda.Stream):
        return s.cuda_stream
    return int(s)


def _check(st: int, where: str):
    if st != 0:
        raise PTDError(st, where)


# ---------------------------------------------------------------------------
# entry points (same names and argument order as include/ptd.h)
# ---------------------------------------------------------------------------
def ptd_status_string(status: int) -> str:
    return _lib.ptd_status_string(status).decode()


def ptd_version() -> int:
    return _lib.ptd_version()


def ptd_build_tree_mask(parent, tree_len, B, T, mask, depth, dev_status=None, stream=None):
    _check(_lib.ptd_build_tree_mask(_ptr(parent), _ptr(tree_len), B, T, _ptr(mask),
                                    _ptr(depth), _ptr(dev_status), _stream(stream)),
           "ptd_build_tree_mask")


def ptd_tree_attention_workspace_bytes(shape: AttnShape, T: int) -> int:
    return _lib.ptd_tree_attention_workspace_bytes(ctypes.byref(shape), T)


def ptd_tree_attention(q, k_cache, v_cache, kv_len, parent, T, out, shape: AttnShape,
                       mask=None, workspace=None, workspace_bytes=0, dev_status=None,
                       stream=None):
    _check(_lib.ptd_tree_attention(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(kv_len),
                                   _ptr(parent), T, _ptr(out), ctypes.byref(shape),
                                   _ptr(mask), _ptr(workspace), workspace_bytes,
                                   _ptr(dev_status), _stream(stream)),
           "ptd_tree_attention")


def ptd_tree_attention_ragged(q, k_cache, v_cache, kv_len, tree_len, parent, T, out,
                              shape: AttnShape, mask=None, workspace=None, workspace_bytes=0,
                              dev_status=None, stream=None):
    _check(_lib.ptd_tree_attention_ragged(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(kv_len),
                                          _ptr(tree_len), _ptr(parent), T, _ptr(out),
                                          ctypes.byref(shape), _ptr(mask), _ptr(workspace),
                                          workspace_bytes, _ptr(dev_status), _stream(stream)),
           "ptd_tree_attention_ragged")


def ptd_tree_attention_noalloc(q, k_cache, v_cache, kv_len, tree_len, parent, T, out,
                               shape: AttnShape, mask=None, dev_status=None, stream=None):
    _check(_lib.ptd_tree_attention_noalloc(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(kv_len),
                                           _ptr(tree_len), _ptr(parent), T, _ptr(out),
                                           ctypes.byref(shape), _ptr(mask), _ptr(dev_status),
                                           _stream(stream)),
           "ptd_tree_attention_noalloc")


def ptd_tree_attention_fp8kv(q, k_cache, v_cache, k_scale, v_scale, kv_len, tree_len, parent, T,
                             out, shape: AttnShape, workspace=None, workspace_bytes=0,
                             dev_status=None, stream=None):
    _check(_lib.ptd_tree_attention_fp8kv(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_scale),
                                         _ptr(v_scale), _ptr(kv_len), _ptr(tree_len),
                                         _ptr(parent), T, _ptr(out), ctypes.byref(shape),
                                         _ptr(workspace), workspace_bytes, _ptr(dev_status),
                                         _stream(stream)),
           "ptd_tree_attention_fp8kv")


def ptd_tree_attention_paged_fp8kv(q, kv: KVPages, k_scale, v_scale, kv_len, tree_len, parent, T,
                                   out, shape: AttnShape, workspace=None, workspace_bytes=0,
                                   dev_status=None, stream=None):
    _check(_lib.ptd_tree_attention_paged_fp8kv(_ptr(q), ctypes.byref(kv), _ptr(k_scale),
                                               _ptr(v_scale), _ptr(kv_len), _ptr(tree_len),
                                               _ptr(parent), T, _ptr(out), ctypes.byref(shape),
                                               _ptr(workspace), workspace_bytes, _ptr(dev_status),
                                               _stream(stream)),
           "ptd_tree_attention_paged_fp8kv")


def ptd_tree_attention_paged(q, kv: KVPages, kv_len, tree_len, parent, T, out, shape: AttnShape,
                             mask=None, workspace=None, workspace_bytes=0, dev_status=None,
                             stream=None):
    _check(_lib.ptd_tree_attention_paged(_ptr(q), ctypes.byref(kv), _ptr(kv_len), _ptr(tree_len),
                                         _ptr(parent), T, _ptr(out), ctypes.byref(shape),
                                         _ptr(mask), _ptr(workspace), workspace_bytes,
                                         _ptr(dev_status), _stream(stream)),
           "ptd_tree_attention_paged")


def ptd_topk_workspace_bytes(R: int, V: int, k: int) -> int:
    return _lib.ptd_topk_workspace_bytes(R, V, k)


def ptd_topk_argmax(logits, dtype, R, V, ld, k, argmax, topk_idx=None, topk_val=None,
                    workspace=None, workspace_bytes=0, stream=None):
    _check(_lib.ptd_topk_argmax(_ptr(logits), dtype, R, V, ld, k, _ptr(argmax),
                                _ptr(topk_idx), _ptr(topk_val), _ptr(workspace),
                                workspace_bytes, _stream(stream)),
           "ptd_topk_argmax")


def ptd_verify(argmax, draft_tokens, parent, tree_len, B, T, accept_len, accept_nodes,
               out_tokens, dev_status=None, stream=None):
    _check(_lib.ptd_verify(_ptr(argmax), _ptr(draft_tokens), _ptr(parent), _ptr(tree_len),
                           B, T, _ptr(accept_len), _ptr(accept_nodes), _ptr(out_tokens),
                           _ptr(dev_status), _stream(stream)),
           "ptd_verify")


def ptd_expand(parent, tokens, tree_len, B, T, topk_idx, k, width_sched, d_max, T_max,
               parent_next, tokens_next, tree_len_next, dev_status=None, stream=None):
    ws = (ctypes.c_int32 * max(1, len(width_sched)))(*[int(x) for x in width_sched])
    if len(width_sched) < d_max:
        raise ValueError("width_sched needs d_max entries")
    _check(_lib.ptd_expand(_ptr(parent), _ptr(tokens), _ptr(tree_len), B, T, _ptr(topk_idx),
                           k, ctypes.cast(ws, _vp), d_max, T_max, _ptr(parent_next),
                           _ptr(tokens_next), _ptr(tree_len_next), _ptr(dev_status),
                           _stream(stream)),
           "ptd_expand")


def ptd_verify_expand(argmax, draft_tokens, parent, tree_len, B, T, topk_idx, k, width_sched,
                      d_max, T_max, accept_len, accept_nodes, out_tokens, parent_next,
                      tokens_next, tree_len_next, dev_status=None, stream=None):
    if len(width_sched) < d_max:
        raise ValueError("width_sched needs d_max entries")
    ws = (ctypes.c_int32 * max(1, len(width_sched)))(*[int(x) for x in width_sched])
    _check(_lib.ptd_verify_expand(_ptr(argmax), _ptr(draft_tokens), _ptr(parent),
                                  _ptr(tree_len), B, T, _ptr(topk_idx), k,
                                  ctypes.cast(ws, _vp), d_max, T_max, _ptr(accept_len),
                                  _ptr(accept_nodes), _ptr(out_tokens), _ptr(parent_next),
                                  _ptr(tokens_next), _ptr(tree_len_next), _ptr(dev_status),
                                  _stream(stream)),
           "ptd_verify_expand")


def ptd_tree_rope(q, k_cache, kv_len, parent, T, shape: AttnShape, theta=10000.0,
                  inv_freq: Optional[Sequence[float]] = None, pairing=PTD_ROPE_HALF,
                  pos_out=None, dev_status=None, stream=None):
    """inv_freq: host sequence of D/2 floats, or None for theta^(-2p/D)."""
    f = None
    if inv_freq is not None:
        if len(inv_freq) != shape.D // 2:
            raise ValueError("inv_freq needs D/2 entries")
        f = (ctypes.c_double * len(inv_freq))(*[float(x) for x in inv_freq])
    _check(_lib.ptd_tree_rope(_ptr(q), _ptr(k_cache), _ptr(kv_len), _ptr(parent), T,
                              ctypes.byref(shape), float(theta),
                              None if f is None else ctypes.cast(f, _vp), pairing,
                              _ptr(pos_out), _ptr(dev_status), _stream(stream)),
           "ptd_tree_rope")


def ptd_kv_commit(k_cache, v_cache, kv_len, accept_len, accept_nodes, T, shape: AttnShape,
                  kv_len_next, dev_status=None, stream=None):
    _check(_lib.ptd_kv_commit(_ptr(k_cache), _ptr(v_cache), _ptr(kv_len), _ptr(accept_len),
                              _ptr(accept_nodes), T, ctypes.byref(shape), _ptr(kv_len_next),
                              _ptr(dev_status), _stream(stream)),
           "ptd_kv_commit")


def ptd_verify_sample_workspace_bytes(B: int, T: int, V: int) -> int:
    return _lib.ptd_verify_sample_workspace_bytes(B, T, V)


def ptd_verify_sample(logits, dtype, V, ld, draft_tokens, parent, tree_len, B, T, temperature,
                      u_node, u_bonus, accept_len, accept_nodes, out_tokens, workspace=None,
                      workspace_bytes=0, dev_status=None, stream=None):
    _check(_lib.ptd_verify_sample(_ptr(logits), dtype, V, ld, _ptr(draft_tokens), _ptr(parent),
                                  _ptr(tree_len), B, T, float(temperature), _ptr(u_node),
                                  _ptr(u_bonus), _ptr(accept_len), _ptr(accept_nodes),
                                  _ptr(out_tokens), _ptr(workspace), workspace_bytes,
                                  _ptr(dev_status), _stream(stream)),
           "ptd_verify_sample")


def ptd_step_prune(parent, tokens, tree_len, B, T, d_max, T_max, parent_next, tokens_next,
                   tree_len_next, dev_status=None, stream=None):
    _check(_lib.ptd_step_prune(_ptr(parent), _ptr(tokens), _ptr(tree_len), B, T, d_max, T_max,
                               _ptr(parent_next), _ptr(tokens_next), _ptr(tree_len_next),
                               _ptr(dev_status), _stream(stream)),
           "ptd_step_prune")


def ptd_pool_bytes(B: int, e_max: int, n_cap: int) -> int:
    return _lib.ptd_pool_bytes(B, e_max, n_cap)


def ptd_pool_init(pool, pool_bytes, B, e_max, n_cap, stream=None):
    _check(_lib.ptd_pool_init(_ptr(pool), pool_bytes, B, e_max, n_cap, _stream(stream)),
           "ptd_pool_init")


def ptd_pool_merge(pool, pool_bytes, B, e_max, n_cap, parent, tokens, tree_len, T,
                   dev_status=None, stream=None):
    _check(_lib.ptd_pool_merge(_ptr(pool), pool_bytes, B, e_max, n_cap, _ptr(parent),
                               _ptr(tokens), _ptr(tree_len), T, _ptr(dev_status),
                               _stream(stream)),
           "ptd_pool_merge")


def ptd_pool_retrieve(pool, pool_bytes, B, e_max, n_cap, last_token, T_max, parent_out,
                      tokens_out, tree_len_out, stream=None):
    _check(_lib.ptd_pool_retrieve(_ptr(pool), pool_bytes, B, e_max, n_cap, _ptr(last_token),
                                  T_max, _ptr(parent_out), _ptr(tokens_out),
                                  _ptr(tree_len_out), _stream(stream)),
           "ptd_pool_retrieve")


# ---------------------------------------------------------------------------
# tensor helpers: allocate outputs, check device/dtype/contiguity, call
# ---------------------------------------------------------------------------
def _need_gpu(*ts):
    for t in ts:
        if t is not None and (not isinstance(t, torch.Tensor) or not t.is_cuda
                              or not t.is_contiguous()):
            raise ValueError("expected contiguous GPU tensors")


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return PTD_BF16
    if t.dtype == torch.float32:
        return PTD_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def attn_shape(q: torch.Tensor, k_cache: torch.Tensor, out_dtype=None,
               scale: float = 0.0) -> AttnShape:
    B, T, Hq, D = q.shape
    _, Hkv, L_cap, _ = k_cache.shape
    od = _dtype_code(q) if out_dtype is None else (
        PTD_BF16 if out_dtype == torch.bfloat16 else PTD_F32)
    return AttnShape(B, Hq, Hkv, D, L_cap, _dtype_code(q), od, float(scale))


def tree_mask(parent: torch.Tensor, tree_len: Optional[torch.Tensor] = None,
              dev_status: Optional[torch.Tensor] = None):
    _need_gpu(parent, tree_len)
    B, T = parent.shape
    mask = torch.empty((B, T, (T + 63) // 64), dtype=torch.int64, device=parent.device)
    depth = torch.empty((B, T), dtype=torch.int32, device=parent.device)
    ptd_build_tree_mask(parent, tree_len, B, T, mask, depth, dev_status)
    return mask, depth


def tree_attention(q, k_cache, v_cache, kv_len, parent, mask=None, out=None,
                   out_dtype=None, scale: float = 0.0, workspace=None,
                   dev_status=None, tree_len=None):
    """tree_len int32 [B] (optional): a padded batch of trees of different
    sizes (ptd_tree_attention_ragged); nodes >= tree_len[b] get zero rows."""
    _need_gpu(q, k_cache, v_cache, kv_len, parent, mask, tree_len)
    B, T, Hq, D = q.shape
    shape = attn_shape(q, k_cache, out_dtype, scale)
    if out is None:
        od = torch.bfloat16 if shape.out_dtype == PTD_BF16 else torch.float32
        out = torch.empty((B, T, Hq, D), dtype=od, device=q.device)
    nbytes = ptd_tree_attention_workspace_bytes(shape, T)
    if workspace is None and nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    wsb = 0 if workspace is None else workspace.numel()
    if tree_len is None:
        ptd_tree_attention(q, k_cache, v_cache, kv_len, parent, T, out, shape, mask,
                           workspace, wsb, dev_status)
    else:
        ptd_tree_attention_ragged(q, k_cache, v_cache, kv_len, tree_len, parent, T, out, shape,
                                  mask, workspace, wsb, dev_status)
    return out


def tree_attention_fp8kv(q, k_cache, v_cache, k_scale, v_scale, kv_len, parent, out=None,
                         out_dtype=None, scale: float = 0.0, workspace=None, dev_status=None,
                         tree_len=None):
    """k_cache, v_cache uint8 [B][Hkv][L_cap][D] E4M3 codes; k_scale, v_scale
    float32 [Hkv] (or None); q bf16; otherwise as tree_attention."""
    _need_gpu(q, k_cache, v_cache, k_scale, v_scale, kv_len, parent, tree_len)
    if k_cache.dtype != torch.uint8 or v_cache.dtype != torch.uint8:
        raise ValueError("expected uint8 E4M3 caches")
    B, T, Hq, D = q.shape
    _, Hkv, L, _ = k_cache.shape
    shape = AttnShape(B, Hq, Hkv, D, L, _dtype_code(q),
                      _dtype_code(q) if out_dtype is None else
                      (PTD_BF16 if out_dtype == torch.bfloat16 else PTD_F32), float(scale))
    if out is None:
        od = torch.bfloat16 if shape.out_dtype == PTD_BF16 else torch.float32
        out = torch.empty((B, T, Hq, D), dtype=od, device=q.device)
    nbytes = ptd_tree_attention_workspace_bytes(shape, T)
    if workspace is None and nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    ptd_tree_attention_fp8kv(q, k_cache, v_cache, k_scale, v_scale, kv_len, tree_len, parent, T,
                             out, shape, workspace, 0 if workspace is None else workspace.numel(),
                             dev_status)
    return out


def tree_attention_paged(q, k_pages, v_pages, page_table, kv_len, parent, out=None,
                         out_dtype=None, scale: float = 0.0, workspace=None, dev_status=None,
                         tree_len=None, k_scale=None, v_scale=None):
    """k_pages, v_pages [num_pages][Hkv][page_size][D] (bf16, or uint8 E4M3
    codes with optional k_scale / v_scale [Hkv]), page_table int32
    [B][max_pages]; otherwise as tree_attention."""
    _need_gpu(q, k_pages, v_pages, page_table, kv_len, parent, tree_len, k_scale, v_scale)
    B, T, Hq, D = q.shape
    num_pages, Hkv, ps, _ = k_pages.shape
    max_pages = page_table.shape[1]
    shape = AttnShape(B, Hq, Hkv, D, max_pages * ps, _dtype_code(q),
                      _dtype_code(q) if out_dtype is None else
                      (PTD_BF16 if out_dtype == torch.bfloat16 else PTD_F32), float(scale))
    if out is None:
        od = torch.bfloat16 if shape.out_dtype == PTD_BF16 else torch.float32
        out = torch.empty((B, T, Hq, D), dtype=od, device=q.device)
    nbytes = ptd_tree_attention_workspace_bytes(shape, T)
    if workspace is None and nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    kv = KVPages(k_pages.data_ptr(), v_pages.data_ptr(), page_table.data_ptr(), ps, max_pages,
                 num_pages)
    wsb = 0 if workspace is None else workspace.numel()
    if k_pages.dtype == torch.uint8:
        ptd_tree_attention_paged_fp8kv(q, kv, k_scale, v_scale, kv_len, tree_len, parent, T, out,
                                       shape, workspace, wsb, dev_status)
    else:
        ptd_tree_attention_paged(q, kv, kv_len, tree_len, parent, T, out, shape, None, workspace,
                                 wsb, dev_status)
    return out


def topk_argmax(logits: torch.Tensor, k: int, with_values: bool = True, workspace=None):
    """logits [R][V] with unit stride along V (a row stride ld >= V is allowed),
    or any contiguous [..][V]; returns (argmax [R], idx [R][k], val [R][k])."""
    if not logits.is_cuda:
        raise ValueError("expected GPU logits")
    if logits.dim() != 2:
        logits = logits.reshape(-1, logits.shape[-1])
    if logits.stride(1) != 1:
        raise ValueError("logits need unit stride along the vocabulary")
    R, V = logits.shape
    ld = logits.stride(0)
    dev = logits.device
    am = torch.empty(R, dtype=torch.int32, device=dev)
    idx = torch.empty((R, k), dtype=torch.int32, device=dev)
    val = torch.empty((R, k), dtype=torch.float32, device=dev) if with_values else None
    nbytes = ptd_topk_workspace_bytes(R, V, k)
    if workspace is None and nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    ptd_topk_argmax(logits, _dtype_code(logits), R, V, ld, k, am, idx, val, workspace,
                    0 if workspace is None else workspace.numel())
    return am, idx, val


def verify(argmax, draft_tokens, parent, tree_len=None, dev_status=None):
    _need_gpu(argmax, draft_tokens, parent, tree_len)
    B, T = parent.shape
    dev = parent.device
    al = torch.empty(B, dtype=torch.int32, device=dev)
    an = torch.empty((B, T), dtype=torch.int32, device=dev)
    ot = torch.empty((B, T + 1), dtype=torch.int32, device=dev)
    ptd_verify(argmax, draft_tokens, parent, tree_len, B, T, al, an, ot, dev_status)
    return al, an, ot


def expand(parent, tokens, topk_idx, width_sched: Sequence[int], d_max: int, T_max: int,
           tree_len=None, dev_status=None):
    _need_gpu(parent, tokens, topk_idx, tree_len)
    B, T = parent.shape
    k = topk_idx.shape[-1]
    dev = parent.device
    pn = torch.empty((B, T_max), dtype=torch.int32, device=dev)
    tn = torch.empty((B, T_max), dtype=torch.int32, device=dev)
    ln = torch.empty(B, dtype=torch.int32, device=dev)
    ptd_expand(parent, tokens, tree_len, B, T, topk_idx, k, width_sched, d_max, T_max,
               pn, tn, ln, dev_status)
    return pn, tn, ln


def verify_expand(argmax, draft_tokens, parent, topk_idx, width_sched: Sequence[int],
                  d_max: int, T_max: int, tree_len=None, dev_status=None):
    """Returns (accept_len, accept_nodes, out_tokens, parent_next, tokens_next,
    tree_len_next)."""
    _need_gpu(argmax, draft_tokens, parent, topk_idx, tree_len)
    B, T = parent.shape
    k = topk_idx.shape[-1]
    dev = parent.device
    al = torch.empty(B, dtype=torch.int32, device=dev)
    an = torch.empty((B, T), dtype=torch.int32, device=dev)
    ot = torch.empty((B, T + 1), dtype=torch.int32, device=dev)
    pn = torch.empty((B, T_max), dtype=torch.int32, device=dev)
    tn = torch.empty((B, T_max), dtype=torch.int32, device=dev)
    ln = torch.empty(B, dtype=torch.int32, device=dev)
    ptd_verify_expand(argmax, draft_tokens, parent, tree_len, B, T, topk_idx, k, width_sched,
                      d_max, T_max, al, an, ot, pn, tn, ln, dev_status)
    return al, an, ot, pn, tn, ln


def tree_rope(q, k_cache, kv_len, parent, theta: float = 10000.0, inv_freq=None,
              pairing: int = PTD_ROPE_HALF, dev_status=None):
    """Turns q [B][T][Hq][D] and the tree rows kv_len + i of k_cache
    [B][Hkv][L_cap][D] in place (either may be None); returns the positions
    int32 [B][T]."""
    _need_gpu(q, k_cache, kv_len, parent)
    B, T = parent.shape
    ref = q if q is not None else k_cache
    Hq, D = (q.shape[2], q.shape[3]) if q is not None else (1, k_cache.shape[3])
    Hkv, L_cap = (k_cache.shape[1], k_cache.shape[2]) if k_cache is not None else (1, T)
    dt = _dtype_code(ref)
    shape = AttnShape(B, Hq, Hkv, D, L_cap, dt, dt, 0.0)
    pos = torch.empty((B, T), dtype=torch.int32, device=parent.device)
    ptd_tree_rope(q, k_cache, kv_len, parent, T, shape, theta, inv_freq, pairing, pos,
                  dev_status)
    return pos


def kv_commit(k_cache, v_cache, kv_len, accept_len, accept_nodes, dev_status=None):
    """Moves the accepted nodes' rows in place; returns kv_len_next int32 [B]."""
    _need_gpu(k_cache, v_cache, kv_len, accept_len, accept_nodes)
    B, Hkv, L_cap, D = k_cache.shape
    T = accept_nodes.shape[-1]
    dt = _dtype_code(k_cache)
    shape = AttnShape(B, Hkv, Hkv, D, L_cap, dt, dt, 0.0)
    nxt = torch.empty(B, dtype=torch.int32, device=k_cache.device)
    ptd_kv_commit(k_cache, v_cache, kv_len, accept_len, accept_nodes, T, shape, nxt,
                  dev_status)
    return nxt


def verify_sample(logits, draft_tokens, parent, temperature: float, u_node, u_bonus,
                  tree_len=None, workspace=None, dev_status=None):
    """logits [B][T+1][V] or [B*(T+1)][V] (unit stride along V); uniforms
    u_node float64 [B][T], u_bonus float64 [B][T+1].
    Returns (accept_len, accept_nodes, out_tokens)."""
    _need_gpu(draft_tokens, parent, tree_len, u_node, u_bonus)
    if not logits.is_cuda:
        raise ValueError("expected GPU logits")
    B, T = parent.shape
    lg = logits.reshape(B * (T + 1), logits.shape[-1]) if logits.dim() != 2 else logits
    if lg.stride(1) != 1:
        raise ValueError("logits need unit stride along the vocabulary")
    if u_node.dtype != torch.float64 or u_bonus.dtype != torch.float64:
        raise TypeError("uniforms are float64")
    V, ld = lg.shape[1], lg.stride(0)
    dev = parent.device
    al = torch.empty(B, dtype=torch.int32, device=dev)
    an = torch.empty((B, T), dtype=torch.int32, device=dev)
    ot = torch.empty((B, T + 1), dtype=torch.int32, device=dev)
    nbytes = ptd_verify_sample_workspace_bytes(B, T, V)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    ptd_verify_sample(lg, _dtype_code(lg), V, ld, draft_tokens, parent, tree_len, B, T,
                      temperature, u_node, u_bonus, al, an, ot, workspace, workspace.numel(),
                      dev_status)
    return al, an, ot


def step_prune(parent, tokens, d_max: int, T_max: int, tree_len=None, dev_status=None):
    """Returns (parent_next, tokens_next, tree_len_next)."""
    _need_gpu(parent, tokens, tree_len)
    B, T = parent.shape
    dev = parent.device
    pn = torch.empty((B, T_max), dtype=torch.int32, device=dev)
    tn = torch.empty((B, T_max), dtype=torch.int32, device=dev)
    ln = torch.empty(B, dtype=torch.int32, device=dev)
    ptd_step_prune(parent, tokens, tree_len, B, T, d_max, T_max, pn, tn, ln, dev_status)
    return pn, tn, ln


class Pool:
    """A device candidate pool of B sequences (at most e_max trees of at
    most n_cap nodes per sequence), set up on construction."""

    def __init__(self, B: int, e_max: int, n_cap: int, device="cuda"):
        self.B, self.e_max, self.n_cap = B, e_max, n_cap
        self.nbytes = ptd_pool_bytes(B, e_max, n_cap)
        if not self.nbytes:
            raise ValueError("invalid pool sizes")
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
        ptd_pool_init(self.buf, self.nbytes, B, e_max, n_cap)

    def merge(self, parent, tokens, tree_len=None, dev_status=None):
        _need_gpu(parent, tokens, tree_len)
        ptd_pool_merge(self.buf, self.nbytes, self.B, self.e_max, self.n_cap, parent, tokens,
                       tree_len, parent.shape[1], dev_status)

    def retrieve(self, last_token, T_max: int):
        """Returns (parent, tokens, tree_len) of the candidate trees."""
        _need_gpu(last_token)
        dev = self.buf.device
        po = torch.empty((self.B, T_max), dtype=torch.int32, device=dev)
        to = torch.empty((self.B, T_max), dtype=torch.int32, device=dev)
        ln = torch.empty(self.B, dtype=torch.int32, device=dev)
        ptd_pool_retrieve(self.buf, self.nbytes, self.B, self.e_max, self.n_cap, last_token,
                          T_max, po, to, ln)
        return po, to, ln
