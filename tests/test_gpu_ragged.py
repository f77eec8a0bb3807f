"""GPU parity of tree attention over a padded batch of trees of different
sizes (ptd_tree_attention_ragged, and ptd_tree_attention_paged with tree_len),
through the C ABI, against the fp64 CPU oracle on the same seeded inputs.

Live rows: fp32 outputs within 2e-3 of the oracle (bf16 inputs, fp32
accumulation; 1e-5 for fp32 inputs).  Padding rows: exactly zero.  The
padding slots are filled with garbage (out-of-range parents, huge queries and
cache rows) that must not be read, and the caches end right after the
longest live tree where the cases allow it."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

pytestmark = pytest.mark.gpu
TOL_BF16 = 2e-3
TOL_F32 = 1e-5


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


def make_case(rng, B, T, Hq, Hkv, D, kv_len, tree_len, dtype="bf16", extra_rows=0, parents=None):
    """Seeded inputs; garbage in every padding slot; cache of
    max(kv_len + tree_len) + extra_rows rows."""
    kv_len = np.asarray(kv_len, np.int32)
    tl = np.asarray(tree_len, np.int32)
    L = int((kv_len + np.clip(tl, 0, T)).max()) + extra_rows
    L = max(L, 1)
    par = parents if parents is not None else np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    par = par.astype(np.int32).copy()
    q = rng.standard_normal((B, T, Hq, D)).astype(np.float32)
    kc = rng.standard_normal((B, Hkv, L, D)).astype(np.float32)
    vc = rng.standard_normal((B, Hkv, L, D)).astype(np.float32)
    for b in range(B):
        n = min(max(int(tl[b]), 0), T)
        par[b, n:] = [77, -9, T + 5][b % 3]
        q[b, n:] = 3e4
        kc[b, :, kv_len[b] + n:] = -3e4
        vc[b, :, kv_len[b] + n:] = 3e4
    if dtype == "bf16":
        q, kc, vc = W.f32_to_bf16_bits(q), W.f32_to_bf16_bits(kc), W.f32_to_bf16_bits(vc)
    return q, kc, vc, kv_len, tl, par


def check(P, q, kc, vc, kv_len, tl, par, rows=None, tol=TOL_BF16, out_dtype=torch.float32):
    B, T, Hq, D = q.shape
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = P.tree_attention(cu(q), cu(kc), cu(vc), cu(kv_len), cu(par), out_dtype=out_dtype,
                           dev_status=st, tree_len=cu(tl))
    torch.cuda.synchronize()
    assert st.item() == 0
    got = out.float().cpu().numpy()
    n_live = np.clip(tl, 0, T)
    for b in range(B):
        assert np.all(got[b, n_live[b]:] == 0.0), b
    scale = 1.0 / np.sqrt(D)
    if rows is None:
        ref = O.tree_attention(q, kc, vc, kv_len, par, scale, tree_len=tl)
        assert np.abs(got - ref).max() <= tol
    else:
        ref = O.attention_rows(q, kc, vc, kv_len, par, scale, rows, tree_len=tl)
        for n, (b, h, i) in enumerate(rows):
            assert np.abs(got[b, i, h] - ref[n]).max() <= tol, (b, h, i)
    return out


@pytest.mark.parametrize("D,Hq,Hkv", [(128, 8, 2), (64, 4, 4)])
def test_ragged_small_bf16(P, D, Hq, Hkv):
    rng = np.random.default_rng(D + Hq)
    q, kc, vc, kvl, tl, par = make_case(rng, 5, 13, Hq, Hkv, D, [0, 300, 20, 7, 1000],
                                        [13, 5, 0, 1, 9])
    check(P, q, kc, vc, kvl, tl, par)


def test_ragged_out_of_range_tree_len_is_clamped(P):
    rng = np.random.default_rng(2)
    q, kc, vc, kvl, tl, par = make_case(rng, 3, 10, 4, 2, 128, [40, 0, 5], [-3, 99, 10])
    check(P, q, kc, vc, kvl, tl, par)


def test_ragged_fp32_inputs(P):
    rng = np.random.default_rng(3)
    q, kc, vc, kvl, tl, par = make_case(rng, 4, 11, 4, 2, 64, [16, 0, 90, 3], [11, 2, 0, 6],
                                        dtype="f32")
    check(P, q, kc, vc, kvl, tl, par, tol=TOL_F32)


def test_ragged_tree_over_128_nodes_reads_built_masks(P):
    rng = np.random.default_rng(4)
    q, kc, vc, kvl, tl, par = make_case(rng, 2, 150, 4, 4, 128, [64, 500], [150, 70])
    rows = [(0, 1, 149), (0, 3, 0), (1, 2, 69), (1, 0, 33), (0, 2, 100), (1, 3, 5)]
    check(P, q, kc, vc, kvl, tl, par, rows=rows)


@pytest.mark.parametrize("extra", [0, 4000])
def test_ragged_all_padding_is_zero(P, extra):
    # no committed keys and no live node: nothing to attend to, zero rows
    # (a short cache gives one split, whose workgroups write the zeros; a
    # long one gives several splits and the combine writes them)
    rng = np.random.default_rng(5 + extra)
    q, kc, vc, kvl, tl, par = make_case(rng, 2, 16, 8, 8, 128, [0, 0], [0, 0], extra_rows=extra)
    for od in (torch.float32, torch.bfloat16):
        out = check(P, q, kc, vc, kvl, tl, par, out_dtype=od)
        assert not torch.isnan(out.float()).any()


def test_ragged_full_tree_len_equals_plain_call(P):
    rng = np.random.default_rng(6)
    B, T = 3, 24
    q, kc, vc, kvl, tl, par = make_case(rng, B, T, 8, 2, 128, [100, 3, 700], [T, T, T])
    a = P.tree_attention(cu(q), cu(kc), cu(vc), cu(kvl), cu(par))
    b = P.tree_attention(cu(q), cu(kc), cu(vc), cu(kvl), cu(par), tree_len=cu(tl))
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_ragged_bad_live_tree_reports(P):
    rng = np.random.default_rng(7)
    q, kc, vc, kvl, tl, par = make_case(rng, 1, 8, 4, 4, 128, [30], [5])
    par[0, 3] = 4  # a live node whose parent is not below it
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    P.tree_attention(cu(q), cu(kc), cu(vc), cu(kvl), cu(par), dev_status=st, tree_len=cu(tl))
    torch.cuda.synchronize()
    assert st.item() == 7


def test_ragged_kv_len_checked_against_live_rows(P):
    rng = np.random.default_rng(8)
    q, kc, vc, kvl, tl, par = make_case(rng, 2, 8, 4, 4, 128, [30, 10], [5, 8])
    L = kc.shape[2]  # = 38: sequence 0 needs 35 rows, sequence 1 needs 18
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    P.tree_attention(cu(q), cu(kc), cu(vc), cu(kvl), cu(par), dev_status=st, tree_len=cu(tl))
    torch.cuda.synchronize()
    assert st.item() == 0
    kvl2 = np.array([L - 4, 10], np.int32)  # 34 + 5 > 38
    P.tree_attention(cu(q), cu(kc), cu(vc), cu(kvl2), cu(par), dev_status=st, tree_len=cu(tl))
    torch.cuda.synchronize()
    assert st.item() == 8


def test_ragged_batch_of_16_sampled(P):
    # the batched ragged shape: 16 sequences, GQA 32/8, D = 128, committed
    # lengths 512..8192, each sequence with its own tree size 1..64
    w = W.make_workload("ragged-16")
    rng = np.random.default_rng(9)
    tl = rng.integers(1, w.T + 1, w.B).astype(np.int32)
    tl[3] = w.T
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = P.tree_attention(cu(w.q), cu(w.k_cache), cu(w.v_cache), cu(w.kv_len), cu(w.parent),
                           out_dtype=torch.float32, dev_status=st, tree_len=cu(tl))
    torch.cuda.synchronize()
    assert st.item() == 0
    got = out.cpu().numpy()
    for b in range(w.B):
        assert np.all(got[b, tl[b]:] == 0.0)
    rows = []
    for _ in range(16):
        b = int(rng.integers(0, w.B))
        rows.append((b, int(rng.integers(0, w.Hq)), int(rng.integers(0, tl[b]))))
    ref = O.attention_rows(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale, rows,
                           tree_len=tl)
    for n, (b, h, i) in enumerate(rows):
        assert np.abs(got[b, i, h] - ref[n]).max() <= TOL_BF16, (b, h, i)


def test_ragged_paged_matches_contiguous(P):
    # paged caches with tree_len: bit for bit the contiguous ragged call
    rng = np.random.default_rng(10)
    B, T, Hkv, D, ps = 3, 20, 4, 128, 64
    q, kc, vc, kvl, tl, par = make_case(rng, B, T, 8, Hkv, D, [200, 0, 64], [20, 7, 1])
    L = (kc.shape[2] + ps - 1) // ps * ps
    pad = ((0, 0), (0, 0), (0, L - kc.shape[2]), (0, 0))
    kc, vc = np.pad(kc, pad), np.pad(vc, pad)
    maxp = L // ps
    table = rng.permutation(B * maxp + 2)[:B * maxp].reshape(B, maxp).astype(np.int32)
    kp = np.zeros((B * maxp + 2, Hkv, ps, D), np.uint16)
    vp = np.zeros_like(kp)
    for b in range(B):
        for j in range(maxp):
            kp[table[b, j]] = kc[b, :, j * ps:(j + 1) * ps]
            vp[table[b, j]] = vc[b, :, j * ps:(j + 1) * ps]
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    paged = P.tree_attention_paged(cu(q), cu(kp), cu(vp), cu(table), cu(kvl), cu(par),
                                   dev_status=st, tree_len=cu(tl))
    contig = P.tree_attention(cu(q), cu(kc), cu(vc), cu(kvl), cu(par), dev_status=st,
                              tree_len=cu(tl))
    torch.cuda.synchronize()
    assert st.item() == 0
    assert torch.equal(paged.view(torch.int16), contig.view(torch.int16))
    got = contig.float().cpu().numpy()
    ref = O.tree_attention(q, kc, vc, kvl, par, 1.0 / np.sqrt(D), tree_len=tl)
    assert np.abs(got - ref).max() <= 8e-3  # bf16 outputs: half an ulp at |x| < 2


def test_ragged_fp32_tree_over_128_nodes(P):
    # vector-ALU path with masks built from tree_len
    rng = np.random.default_rng(11)
    q, kc, vc, kvl, tl, par = make_case(rng, 2, 140, 2, 2, 64, [30, 5], [140, 66], dtype="f32")
    rows = [(0, 1, 139), (0, 0, 70), (1, 1, 65), (1, 0, 0)]
    check(P, q, kc, vc, kvl, tl, par, rows=rows, tol=TOL_F32)


def test_ragged_paged_tree_over_128_nodes(P):
    # paged caches, masks built from tree_len, padding pages never read
    rng = np.random.default_rng(12)
    B, T, Hkv, D, ps = 2, 160, 2, 128, 32
    q, kc, vc, kvl, tl, par = make_case(rng, B, T, 4, Hkv, D, [64, 300], [160, 90])
    L = (kc.shape[2] + ps - 1) // ps * ps
    pad = ((0, 0), (0, 0), (0, L - kc.shape[2]), (0, 0))
    kc, vc = np.pad(kc, pad), np.pad(vc, pad)
    maxp = L // ps
    table = rng.permutation(B * maxp)[:B * maxp].reshape(B, maxp).astype(np.int32)
    kp = np.zeros((B * maxp, Hkv, ps, D), np.uint16)
    vp = np.zeros_like(kp)
    for b in range(B):
        for j in range(maxp):
            kp[table[b, j]] = kc[b, :, j * ps:(j + 1) * ps]
            vp[table[b, j]] = vc[b, :, j * ps:(j + 1) * ps]
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    paged = P.tree_attention_paged(cu(q), cu(kp), cu(vp), cu(table), cu(kvl), cu(par),
                                   out_dtype=torch.float32, dev_status=st, tree_len=cu(tl))
    torch.cuda.synchronize()
    assert st.item() == 0
    got = paged.cpu().numpy()
    assert np.all(got[1, 90:] == 0.0)
    rows = [(0, 3, 159), (0, 1, 128), (1, 2, 89), (1, 0, 3)]
    ref = O.attention_rows(q, kc, vc, kvl, par, 1.0 / np.sqrt(D), rows, tree_len=tl)
    for n, (b, h, i) in enumerate(rows):
        assert np.abs(got[b, i, h] - ref[n]).max() <= TOL_BF16, (b, h, i)
