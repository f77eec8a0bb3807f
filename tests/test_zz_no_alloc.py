"""GPU check of ptd_tree_attention_noalloc, the allocation-free attention entry
point, through the C ABI: on the same seeded inputs its output equals that of
ptd_tree_attention_ragged with a caller workspace (same kernels, same plan:
bit for bit, which is within the 2e-3 attention tolerance), and it stays
within 2e-3 of the fp64 oracle on sampled rows.  Two calls in a row, the
second on a smaller problem, so the second call finds the first call's data
in the fixed scratch array; a third call builds masks in the scratch
(trees over 128 nodes)."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

pytestmark = pytest.mark.gpu
TOL = 2e-3


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


def make(rng, B, T, Hq, Hkv, D, kv_len, tree_len):
    kv_len = np.asarray(kv_len, np.int32)
    tl = np.asarray(tree_len, np.int32)
    L = int((kv_len + tl).max())
    par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)]).astype(np.int32)
    q = W.f32_to_bf16_bits(rng.standard_normal((B, T, Hq, D)).astype(np.float32))
    kc = W.f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D)).astype(np.float32))
    vc = W.f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D)).astype(np.float32))
    return q, kc, vc, kv_len, tl, par


def run_both(P, q, kc, vc, kv_len, tl, par):
    B, T, Hq, D = q.shape
    Hkv, L = kc.shape[1], kc.shape[2]
    tq, tk, tv, tkv, ttl, tpar = cu(q), cu(kc), cu(vc), cu(kv_len), cu(tl), cu(par)
    shape = P.AttnShape(B, Hq, Hkv, D, L, P.PTD_BF16, P.PTD_F32, 0.0)
    need = P.ptd_tree_attention_workspace_bytes(shape, T)
    assert 0 < need <= P.PTD_NOALLOC_SCRATCH_BYTES
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ref = torch.full((B, T, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
    got = torch.full((B, T, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
    P.ptd_tree_attention_ragged(tq, tk, tv, tkv, ttl, tpar, T, ref, shape, None, ws, need, st)
    P.ptd_tree_attention_noalloc(tq, tk, tv, tkv, ttl, tpar, T, got, shape, None, st)
    torch.cuda.synchronize()
    assert st.item() == 0, P.ptd_status_string(st.item())
    return ref.cpu().numpy(), got.cpu().numpy()


def check_oracle(got, q, kc, vc, kv_len, tl, par, rng, n=24):
    B, T, Hq, D = q.shape
    rows = []
    for _ in range(n):
        b = int(rng.integers(B))
        rows.append((b, int(rng.integers(Hq)), int(rng.integers(max(1, tl[b])))))
    refo = O.attention_rows(q, kc, vc, kv_len, par, 1.0 / np.sqrt(D), rows, tree_len=tl)
    for k, (b, h, i) in enumerate(rows):
        assert np.abs(got[b, i, h] - refo[k]).max() <= TOL, (b, h, i)


def test_noalloc_matches_workspace_call_twice(P):
    rng = np.random.default_rng(2024)
    # first call: a GQA batch of 4 sequences, split partials in the scratch
    a = make(rng, 4, 64, 32, 8, 128, [3000, 700, 5100, 1800], [64, 37, 1, 50])
    ref, got = run_both(P, *a)
    assert np.array_equal(ref, got)
    assert not np.isnan(got).any()
    check_oracle(got, *a, rng)
    # second call, smaller: one sequence, fewer keys and nodes, other heads
    b = make(rng, 1, 24, 8, 8, 128, [900], [24])
    ref2, got2 = run_both(P, *b)
    assert np.array_equal(ref2, got2)
    assert not np.isnan(got2).any()
    check_oracle(got2, *b, rng)
    # a tree of 200 nodes: ancestor masks are built into the scratch too
    c = make(rng, 2, 200, 4, 4, 64, [600, 1500], [200, 130])
    ref3, got3 = run_both(P, *c)
    assert np.array_equal(ref3, got3)
    check_oracle(got3, *c, rng)
