"""Whole-output GPU parity at the full workload sizes: every output row of the
attention call, element by element, against the fp64 oracle (its rows spread
over a thread pool).  The calls run as the step runs them (ancestor masks
from ptd_tree_mask, the same launch configuration).

fp32 outputs must be within 2e-3 of the oracle everywhere.  bf16 outputs are
the fp32 result rounded to nearest, which moves an element by at most 2^-9 of
its magnitude, so each must be within 2e-3 + 2^-9 |ref| of the oracle."""
import os

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

pytestmark = pytest.mark.gpu
TOL = 2e-3
THREADS = max(1, min(16, os.cpu_count() or 1))


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_10661_amd as lib
    return lib


def cu(a):
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def all_rows(w):
    return [(b, h, i) for b in range(w.B) for h in range(w.Hq) for i in range(w.T)]


def as_output(w, rows, vals):
    ref = np.zeros((w.B, w.T, w.Hq, w.D), np.float64)
    for n, (b, h, i) in enumerate(rows):
        ref[b, i, h] = vals[n]
    return ref


_REF = {}


def oracle_full(w, name):
    if name not in _REF:
        rows = all_rows(w)
        vals = O.attention_rows(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale, rows,
                                threads=THREADS)
        _REF[name] = as_output(w, rows, vals)
    return _REF[name]


def check(got32, got16, ref, what):
    err = np.abs(got32 - ref)
    assert err.max() <= TOL, (what, "fp32 out", float(err.max()), np.unravel_index(err.argmax(), err.shape))
    assert np.isfinite(got16).all()
    excess = np.abs(got16 - ref) - (TOL + 2.0 ** -9 * np.abs(ref))
    assert excess.max() <= 0.0, (what, "bf16 out", float(excess.max()))


@pytest.mark.parametrize("name", ["llama2-7b", "llama2-13b", "llama3-8b-long", "ragged-16"])
def test_attention_full_output(P, name):
    w = W.make_workload(name, logits=False)
    q, kc, vc, kvl, par = cu(w.q), cu(w.k_cache), cu(w.v_cache), cu(w.kv_len), cu(w.parent)
    mask = P.tree_mask(par)[0]
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    o32 = P.tree_attention(q, kc, vc, kvl, par, mask=mask, out_dtype=torch.float32, dev_status=st)
    o16 = P.tree_attention(q, kc, vc, kvl, par, mask=mask, dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    got32 = o32.cpu().numpy().astype(np.float64)
    got16 = o16.float().cpu().numpy().astype(np.float64)
    check(got32, got16, oracle_full(w, name), name)


def test_attention_full_output_paged_gqa_long(P):
    # the GQA long-context workload with its caches in 64-row pages scattered
    # through a random page table
    w = W.make_workload("llama3-8b-long", logits=False)
    ps = 64
    B, Hkv, L, D = w.k_cache.shape
    maxp = L // ps
    rng = np.random.default_rng(31)
    table = rng.permutation(B * maxp).reshape(B, maxp).astype(np.int32)

    def pages(c):
        out = np.empty((B * maxp, Hkv, ps, D), c.dtype)
        for b in range(B):
            for j in range(maxp):
                out[table[b, j]] = c[b, :, j * ps:(j + 1) * ps]
        return out

    kp, vp = pages(w.k_cache), pages(w.v_cache)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    args = (cu(w.q), cu(kp), cu(vp), cu(table), cu(w.kv_len), cu(w.parent))
    o32 = P.tree_attention_paged(*args, out_dtype=torch.float32, dev_status=st)
    o16 = P.tree_attention_paged(*args, dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    check(o32.cpu().numpy().astype(np.float64), o16.float().cpu().numpy().astype(np.float64),
          oracle_full(w, "llama3-8b-long"), "paged llama3-8b-long")


def test_attention_full_output_fp8_gqa_long(P):
    # the GQA long-context workload with E4M3 caches, one scale per KV head
    w = W.make_workload("llama3-8b-long", logits=False)
    kq, ks = W.quantize_kv_e4m3(W.bf16_bits_to_f32(w.k_cache))
    vq, vs = W.quantize_kv_e4m3(W.bf16_bits_to_f32(w.v_cache))
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    args = (cu(w.q), cu(kq), cu(vq), cu(ks), cu(vs), cu(w.kv_len), cu(w.parent))
    o32 = P.tree_attention_fp8kv(*args, out_dtype=torch.float32, dev_status=st)
    o16 = P.tree_attention_fp8kv(*args, dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    rows = all_rows(w)
    vals = O.tree_attention_fp8kv(w.q, kq, vq, ks, vs, w.kv_len, w.parent, w.scale, rows=rows,
                                  threads=THREADS)
    check(o32.cpu().numpy().astype(np.float64), o16.float().cpu().numpy().astype(np.float64),
          as_output(w, rows, vals), "fp8 llama3-8b-long")
