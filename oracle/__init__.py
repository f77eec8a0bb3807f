"""CPU oracle for the Progressive Tree Drafting hot path (fp64, plain C).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
CPU-baseline leg of the benchmark.  The product library never imports or links
it, and it shares no code with the GPU path.

Thin ctypes wrappers over ``libptd_oracle.so`` built from ``ptd_oracle.c``
(see ``oracle/build.py``).  Inputs are the workload arrays exactly as the GPU
receives them (bf16 as uint16 bits, or float32); the C code widens them to
fp64 exactly.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libptd_oracle.so")
_lib = None

_i32p = ctypes.POINTER(ctypes.c_int32)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, d = ctypes.c_void_p, ctypes.c_int, ctypes.c_double
    lib.oracle_tree_mask.argtypes = [vp, vp, i, i, vp, vp]
    lib.oracle_attention_row.argtypes = [vp, vp, vp, i, vp, vp, vp, i, i, i, i, i, i,
                                         d, i, i, i, vp]
    lib.oracle_tree_attention.argtypes = [vp, vp, vp, i, vp, vp, vp, i, i, i, i, i, i,
                                          d, vp]
    lib.oracle_topk.argtypes = [vp, i, i, i, ctypes.c_longlong, i, vp, vp, vp]
    lib.oracle_e4m3_decode.argtypes = [vp, ctypes.c_longlong, vp]
    lib.oracle_verify.argtypes = [vp, vp, vp, vp, i, i, vp, vp, vp]
    lib.oracle_expand.argtypes = [vp, vp, vp, i, i, vp, i, vp, i, i, vp, vp, vp]
    lib.oracle_tree_rope.argtypes = [vp, vp, i, vp, vp, i, i, i, i, i, i, vp, i, vp, vp,
                                     vp]
    lib.oracle_kv_commit.argtypes = [vp, vp, i, vp, vp, vp, i, i, i, i, i, vp]
    lib.oracle_verify_sample.argtypes = [vp, i, ctypes.c_longlong, i, vp, vp, vp, i, i, d,
                                         vp, vp, vp, vp, vp, vp]
    lib.oracle_step_prune.argtypes = [vp, vp, vp, i, i, i, i, vp, vp, vp]
    lib.oracle_pool_new.argtypes = [i, i, i]
    lib.oracle_pool_new.restype = vp
    lib.oracle_pool_free.argtypes = [vp]
    lib.oracle_pool_free.restype = None
    lib.oracle_pool_merge.argtypes = [vp, vp, vp, vp, i, i]
    lib.oracle_pool_retrieve.argtypes = [vp, vp, i, i, vp, vp, vp]
    lib.oracle_gather_pages.argtypes = [vp, i, vp, i, i, i, i, i, i, vp]
    for f in ("oracle_gather_pages", "oracle_step_prune", "oracle_pool_merge", "oracle_pool_retrieve",
              "oracle_verify_sample", "oracle_tree_mask", "oracle_attention_row", "oracle_tree_attention",
              "oracle_topk", "oracle_verify", "oracle_expand", "oracle_tree_rope",
              "oracle_kv_commit", "oracle_e4m3_decode"):
        getattr(lib, f).restype = ctypes.c_int
    _lib = lib
    return lib


class OracleError(RuntimeError):
    pass


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def _check(st: int):
    if st != 0:
        raise OracleError({2: "bad sizes", 7: "malformed tree", 8: "kv_len out of range",
                           9: "malformed accepted path", 10: "page id out of range"}.get(st, st))


def _dtype_code(arr: np.ndarray) -> int:
    if arr.dtype == np.uint16:
        return 1
    if arr.dtype == np.float32:
        return 0
    if arr.dtype == np.float64:
        return 2
    raise TypeError("oracle inputs are bf16 bits (uint16), float32 or float64")


def tree_mask(parent: np.ndarray, tree_len: Optional[np.ndarray] = None):
    """parent int32 [B][T] -> (mask uint64 [B][T][W], depth int32 [B][T])."""
    parent = _c(parent, np.int32)
    B, T = parent.shape
    W = (T + 63) // 64
    mask = np.zeros((B, T, W), np.uint64)
    depth = np.zeros((B, T), np.int32)
    tl = None if tree_len is None else _c(tree_len, np.int32)
    _check(_load().oracle_tree_mask(_p(parent), _p(tl), B, T, _p(mask), _p(depth)))
    return mask, depth


def _attn_args(q, k_cache, v_cache, kv_len, parent):
    q = np.ascontiguousarray(q)
    k_cache = np.ascontiguousarray(k_cache)
    v_cache = np.ascontiguousarray(v_cache)
    dt = _dtype_code(q)
    if _dtype_code(k_cache) != dt or _dtype_code(v_cache) != dt:
        raise TypeError("q/k/v dtypes differ")
    B, T, Hq, D = q.shape
    _, Hkv, L_cap, _ = k_cache.shape
    return (q, k_cache, v_cache, dt, _c(kv_len, np.int32), _c(parent, np.int32),
            B, T, Hq, Hkv, D, L_cap)


def tree_attention(q, k_cache, v_cache, kv_len, parent, scale: float,
                   tree_len=None) -> np.ndarray:
    """All outputs [B][T][Hq][D] in float64.  tree_len [B] (optional): nodes
    at index >= tree_len[b] are padding with zero outputs."""
    q, kc, vc, dt, kvl, par, B, T, Hq, Hkv, D, L = _attn_args(
        q, k_cache, v_cache, kv_len, parent)
    tl = None if tree_len is None else _c(tree_len, np.int32)
    out = np.zeros((B, T, Hq, D), np.float64)
    _check(_load().oracle_tree_attention(_p(q), _p(kc), _p(vc), dt, _p(kvl),
                                         _p(par), None if tl is None else _p(tl),
                                         B, T, Hq, Hkv, D, L, float(scale), _p(out)))
    return out


def attention_rows(q, k_cache, v_cache, kv_len, parent, scale: float, rows,
                   tree_len=None, threads: int = 1):
    """Selected outputs: rows is a list of (b, h, i); returns [len(rows)][D].
    threads > 1 spreads the rows over a thread pool (each row is computed
    alone, so the results do not depend on it)."""
    q, kc, vc, dt, kvl, par, B, T, Hq, Hkv, D, L = _attn_args(
        q, k_cache, v_cache, kv_len, parent)
    tl = None if tree_len is None else _c(tree_len, np.int32)
    lib = _load()
    out = np.zeros((len(rows), D), np.float64)

    def run(ns):
        for n in ns:
            b, h, i = rows[n]
            _check(lib.oracle_attention_row(
                _p(q), _p(kc), _p(vc), dt, _p(kvl), _p(par), None if tl is None else _p(tl),
                B, T, Hq, Hkv, D, L, float(scale), int(b), int(h), int(i),
                out[n].ctypes.data_as(ctypes.c_void_p)))

    if threads <= 1 or len(rows) < 2:
        run(range(len(rows)))
    else:
        import concurrent.futures as cf
        with cf.ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, [range(j, len(rows), threads) for j in range(threads)]))
    return out


def e4m3_decode(codes) -> np.ndarray:
    """OCP FP8 E4M3 codes (uint8) -> their values, float64, same shape."""
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    out = np.empty(c.shape, np.float64)
    _check(_load().oracle_e4m3_decode(_p(c), c.size, _p(out)))
    return out


def tree_attention_fp8kv(q, k_codes, v_codes, k_scale, v_scale, kv_len, parent,
                         scale: float, tree_len=None, rows=None, threads: int = 1):
    """Tree attention on E4M3 key/value caches [B][Hkv][L][D] with per-KV-head
    scales: key = value(code) * k_scale[g], likewise for values.  All outputs
    [B][T][Hq][D] (float64), or the selected (b, h, i) rows if given."""
    ks = np.asarray(k_scale, np.float64)[None, :, None, None]
    vs = np.asarray(v_scale, np.float64)[None, :, None, None]
    kc = e4m3_decode(k_codes) * ks   # exact: 4 significant bits times a float32
    vc = e4m3_decode(v_codes) * vs
    qd = np.ascontiguousarray(q)
    if qd.dtype == np.uint16:  # bf16 bits, widened exactly
        qd = (qd.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if rows is None:
        return tree_attention(qd, kc, vc, kv_len, parent, scale, tree_len=tree_len)
    return attention_rows(qd, kc, vc, kv_len, parent, scale, rows, tree_len=tree_len,
                          threads=threads)


def topk(logits: np.ndarray, k: int):
    """logits [R][V] (or [..][V]) -> (argmax int32 [R], idx int32 [R][k],
    val float64 [R][k])."""
    lg = np.ascontiguousarray(logits)
    V = lg.shape[-1]
    lg2 = lg.reshape(-1, V)
    R = lg2.shape[0]
    am = np.zeros(R, np.int32)
    idx = np.zeros((R, k), np.int32)
    val = np.zeros((R, k), np.float64)
    _check(_load().oracle_topk(_p(lg2), _dtype_code(lg2), R, V, V, k, _p(am),
                               _p(idx), _p(val)))
    return am, idx, val


def verify(argmax, tokens, parent, tree_len=None):
    """-> (accept_len [B], accept_nodes [B][T], out_tokens [B][T+1])."""
    tokens = _c(tokens, np.int32)
    parent = _c(parent, np.int32)
    B, T = parent.shape
    am = _c(argmax, np.int32).reshape(B, T + 1)
    al = np.zeros(B, np.int32)
    an = np.zeros((B, T), np.int32)
    ot = np.zeros((B, T + 1), np.int32)
    tl = None if tree_len is None else _c(tree_len, np.int32)
    _check(_load().oracle_verify(_p(am), _p(tokens), _p(parent), _p(tl), B, T,
                                 _p(al), _p(an), _p(ot)))
    return al, an, ot


def expand(parent, tokens, topk_idx, width_sched, d_max: int, T_max: int,
           tree_len=None):
    """-> (parent_next [B][T_max], tokens_next [B][T_max], tree_len_next [B])."""
    parent = _c(parent, np.int32)
    tokens = _c(tokens, np.int32)
    B, T = parent.shape
    ti = _c(topk_idx, np.int32)
    k = ti.shape[-1]
    ti = ti.reshape(B, T + 1, k)
    ws = _c(width_sched, np.int32)
    if ws.shape[0] < d_max:
        raise ValueError("width_sched needs d_max entries")
    pn = np.zeros((B, T_max), np.int32)
    tn = np.zeros((B, T_max), np.int32)
    ln = np.zeros(B, np.int32)
    tl = None if tree_len is None else _c(tree_len, np.int32)
    _check(_load().oracle_expand(_p(parent), _p(tokens), _p(tl), B, T, _p(ti), k,
                                 _p(ws), d_max, T_max, _p(pn), _p(tn), _p(ln)))
    return pn, tn, ln


def rope_inv_freq(D: int, theta: float) -> np.ndarray:
    """Rotary frequencies of RoFormer (Su et al., 2021): pair p of a head of
    D dimensions turns by theta^(-2p/D) radians per position, p < D/2."""
    p = np.arange(D // 2, dtype=np.float64)
    return np.power(float(theta), -2.0 * p / D)


def tree_rope(q, k_cache, kv_len, parent, theta: float = 10000.0, inv_freq=None,
              pairing: int = 0):
    """Positions kv_len + |pi(i)| - 1 of the tree nodes and the rotary
    embedding of their queries and keys (the tree rows kv_len + i of k_cache).
    pairing 0: pair p = (p, p + D/2); 1: pair p = (2p, 2p + 1).
    -> (q_out float64 [B][T][Hq][D], k_out float64 [B][Hkv][T][D],
        pos int32 [B][T])."""
    q = np.ascontiguousarray(q)
    k_cache = np.ascontiguousarray(k_cache)
    dt = _dtype_code(q)
    if _dtype_code(k_cache) != dt:
        raise TypeError("q/k dtypes differ")
    B, T, Hq, D = q.shape
    _, Hkv, L_cap, _ = k_cache.shape
    f = rope_inv_freq(D, theta) if inv_freq is None else _c(inv_freq, np.float64)
    if f.shape != (D // 2,):
        raise ValueError("inv_freq needs D/2 entries")
    qo = np.zeros((B, T, Hq, D), np.float64)
    ko = np.zeros((B, Hkv, T, D), np.float64)
    pos = np.zeros((B, T), np.int32)
    kvl = _c(kv_len, np.int32)
    par = _c(parent, np.int32)
    _check(_load().oracle_tree_rope(_p(q), _p(k_cache), dt, _p(kvl), _p(par), B, T, Hq, Hkv,
                                    D, L_cap, _p(f), int(pairing), _p(qo), _p(ko),
                                    _p(pos)))
    return qo, ko, pos


def kv_commit(k_cache, v_cache, kv_len, accept_len, accept_nodes):
    """Commit of the accepted path on copies of the caches
    ([B][Hkv][L_cap][D], bf16 bits or float32).
    -> (k_cache_new, v_cache_new, kv_len_next int32 [B])."""
    kc = np.array(k_cache, copy=True, order="C")
    vc = np.array(v_cache, copy=True, order="C")
    dt = _dtype_code(kc)
    if _dtype_code(vc) != dt:
        raise TypeError("k/v dtypes differ")
    B, Hkv, L_cap, D = kc.shape
    an = _c(accept_nodes, np.int32)
    T = an.shape[-1]
    an = an.reshape(B, T)
    nxt = np.zeros(B, np.int32)
    _check(_load().oracle_kv_commit(_p(kc), _p(vc), dt, _p(_c(kv_len, np.int32)),
                                    _p(_c(accept_len, np.int32)), _p(an), B, T, Hkv, D,
                                    L_cap, _p(nxt)))
    return kc, vc, nxt


def verify_sample(logits, tokens, parent, temperature: float, u_node, u_bonus, tree_len=None):
    """Sampling verification.  logits [B][T+1][V] (or [B*(T+1)][V]), uniforms
    u_node [B][T] (the draw made when node n is examined) and u_bonus [B][T+1]
    (the draw for the bonus token at each row).
    -> (accept_len [B], accept_nodes [B][T], out_tokens [B][T+1], margin [B])."""
    tokens = _c(tokens, np.int32)
    parent = _c(parent, np.int32)
    B, T = parent.shape
    lg = np.ascontiguousarray(logits)
    V = lg.shape[-1]
    lg = lg.reshape(B * (T + 1), V)
    un = _c(u_node, np.float64).reshape(B, T)
    ub = _c(u_bonus, np.float64).reshape(B, T + 1)
    al = np.zeros(B, np.int32)
    an = np.zeros((B, T), np.int32)
    ot = np.zeros((B, T + 1), np.int32)
    mg = np.zeros(B, np.float64)
    tl = None if tree_len is None else _c(tree_len, np.int32)
    _check(_load().oracle_verify_sample(_p(lg), _dtype_code(lg), V, V, _p(tokens), _p(parent),
                                        _p(tl), B, T, float(temperature), _p(un), _p(ub),
                                        _p(al), _p(an), _p(ot), _p(mg)))
    return al, an, ot, mg


def step_prune(parent, tokens, d_max: int, T_max: int, tree_len=None):
    """Stepping (depth control) of a draft forest.
    -> (parent_next [B][T_max], tokens_next [B][T_max], tree_len_next [B])."""
    parent = _c(parent, np.int32)
    tokens = _c(tokens, np.int32)
    B, T = parent.shape
    pn = np.zeros((B, T_max), np.int32)
    tn = np.zeros((B, T_max), np.int32)
    ln = np.zeros(B, np.int32)
    tl = None if tree_len is None else _c(tree_len, np.int32)
    _check(_load().oracle_step_prune(_p(parent), _p(tokens), _p(tl), B, T, int(d_max),
                                     int(T_max), _p(pn), _p(tn), _p(ln)))
    return pn, tn, ln


class Pool:
    """Candidate pool of B sequences: trees of tokens keyed by their root's
    token, at most e_max trees of at most n_cap nodes per sequence."""

    def __init__(self, B: int, e_max: int, n_cap: int):
        self.B = B
        self._lib = _load()
        self._h = self._lib.oracle_pool_new(B, e_max, n_cap)
        if not self._h:
            raise OracleError("bad sizes")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            self._lib.oracle_pool_free(h)
            self._h = None

    def merge(self, parent, tokens, tree_len=None):
        parent = _c(parent, np.int32)
        tokens = _c(tokens, np.int32)
        B, T = parent.shape
        tl = None if tree_len is None else _c(tree_len, np.int32)
        _check(self._lib.oracle_pool_merge(self._h, _p(parent), _p(tokens), _p(tl), B, T))

    def retrieve(self, last_token, T_max: int):
        """-> (parent [B][T_max], tokens [B][T_max], tree_len [B])."""
        lt = _c(last_token, np.int32)
        po = np.zeros((self.B, T_max), np.int32)
        to = np.zeros((self.B, T_max), np.int32)
        ln = np.zeros(self.B, np.int32)
        _check(self._lib.oracle_pool_retrieve(self._h, _p(lt), self.B, int(T_max), _p(po),
                                              _p(to), _p(ln)))
        return po, to, ln


def gather_pages(pages, page_table, page_size: int):
    """Paged cache pages [num_pages][Hkv][page_size][D] (bf16 bits or fp32)
    and page_table int32 [B][max_pages] -> the contiguous cache
    [B][Hkv][max_pages * page_size][D]."""
    pages = np.ascontiguousarray(pages)
    pt = _c(page_table, np.int32)
    num_pages, Hkv, ps, D = pages.shape
    if ps != page_size:
        raise ValueError("pages' second-to-last axis is the page size")
    B, max_pages = pt.shape
    cache = np.zeros((B, Hkv, max_pages * page_size, D), pages.dtype)
    _check(_load().oracle_gather_pages(_p(pages), _dtype_code(pages), _p(pt), B, Hkv, D,
                                       page_size, max_pages, num_pages, _p(cache)))
    return cache
