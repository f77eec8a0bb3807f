"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle on
the same seeded inputs.  Integer results (masks, depths, indices, accepted
paths, expanded trees) must be bit-exact; attention must be within max-abs
2e-3 for bf16 inputs and 1e-5 for fp32 inputs (fp32 accumulation)."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-3, "f32": 1e-5}


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_10661_amd as lib
    return lib


def cu(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def status_buf():
    return torch.zeros(1, dtype=torch.int32, device="cuda")


# ---------------------------------------------------------------------------
# ancestor masks
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("T", [1, 2, 63, 64, 65, 130, 1024])
def test_mask_random_trees(P, T):
    rng = np.random.default_rng(T)
    par = np.stack([W.tree_uniform(rng, T)[0], W.tree_chain(T)[0], W.tree_star(T)[0]])
    tl = np.array([T, max(1, T // 2), T], np.int32)
    for tree_len in (None, tl):
        m_ref, d_ref = O.tree_mask(par, tree_len)
        st = status_buf()
        m, d = P.tree_mask(cu(par), None if tree_len is None else cu(tree_len), st)
        torch.cuda.synchronize()
        assert st.item() == 0
        assert np.array_equal(m.cpu().numpy().view(np.uint64), m_ref)
        assert np.array_equal(d.cpu().numpy(), d_ref)


def test_mask_reports_bad_tree(P):
    par = np.array([[-1, 0, 2, 1], [-1, -1, 0, 1]], np.int32)
    st = status_buf()
    P.tree_mask(cu(par), None, st)
    torch.cuda.synchronize()
    assert st.item() == 7


# ---------------------------------------------------------------------------
# top-k / argmax
# ---------------------------------------------------------------------------
def _topk_case(P, arr, k, ld=None):
    R, V = arr.shape
    if ld is not None and ld > V:
        buf = np.zeros((R, ld), arr.dtype)
        buf[:, :V] = arr
        t = cu(buf)[:, :V]
    else:
        t = cu(arr)
    am, idx, val = P.topk_argmax(t, k)
    torch.cuda.synchronize()
    r_am, r_idx, r_val = O.topk(arr, k)
    assert np.array_equal(am.cpu().numpy(), r_am)
    assert np.array_equal(idx.cpu().numpy(), r_idx)
    v = val.cpu().numpy().astype(np.float64)
    assert np.array_equal(v, r_val)
    assert np.array_equal(np.signbit(v), np.signbit(r_val))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("R,V,k", [(1, 1, 1), (3, 7, 5), (17, 1000, 4), (65, 32000, 4),
                                   (97, 32000, 5), (8, 32003, 16), (5, 128256, 8),
                                   (1100, 4099, 2), (3, 70001, 8), (2, 200003, 16),
                                   (2, 300007, 4), (1, 600001, 16), (300, 128256, 8),
                                   (70, 128256, 8), (16, 600001, 16)])
def test_topk_random(P, dtype, R, V, k):
    rng = np.random.default_rng(R * 7 + V + k)
    x = rng.standard_normal((R, V), dtype=np.float32) * np.float32(1.41)
    # injected ties (bf16 makes more on its own) and signed zeros
    cols = rng.integers(0, V, min(V, 50))
    x[:, cols] = x[:, cols[:1]]
    x[::2, rng.integers(0, V, min(V, 9))] = np.float32(-0.0)
    x[1::2, rng.integers(0, V, min(V, 9))] = np.float32(0.0)
    arr = W.f32_to_bf16_bits(x) if dtype == "bf16" else x
    _topk_case(P, arr, k)


def test_topk_all_equal_and_strided(P):
    x = np.full((6, 5000), 0.75, np.float32)
    x[3, 4999] = 0.8
    _topk_case(P, W.f32_to_bf16_bits(x), 8)
    rng = np.random.default_rng(1)
    x = W.f32_to_bf16_bits(rng.standard_normal((9, 3001), dtype=np.float32))
    _topk_case(P, x, 6, ld=3008)   # 16-byte aligned rows, vector loads
    _topk_case(P, x, 6, ld=3005)   # misaligned rows, scalar loads
    # rows where -inf entries must fill the list (fewer finite values than k)
    y = np.full((4, 4100), -np.inf, np.float32)
    y[0, 17] = 1.0
    y[1, [5, 4099]] = -3.0
    y[2, 0] = np.float32(-0.0)
    _topk_case(P, y, 5)
    _topk_case(P, W.f32_to_bf16_bits(y), 5)
    big = np.full((2, 200003), -np.inf, np.float32)  # sliced path
    big[0, 199999] = 2.0
    _topk_case(P, W.f32_to_bf16_bits(big), 3)


@pytest.mark.parametrize("k", [1, 4, 16])
def test_topk_many_ties_at_the_top(P, k):
    # more elements tie with the k-th best than the candidate list holds
    rng = np.random.default_rng(k)
    x = rng.standard_normal((5, 40000), dtype=np.float32)
    for r, n in enumerate([1500, 3000, 1025, 1024, 40000]):
        x[r, rng.choice(40000, n, replace=False)] = np.float32(9.0)
    _topk_case(P, x, k)
    _topk_case(P, W.f32_to_bf16_bits(x), k)


def test_topk_many_slices_with_ties(P):
    # enough slices for the 512-thread workgroups (four or more per CU), some
    # rows with more ties at the top than the candidate lists hold
    rng = np.random.default_rng(77)
    R, V = 1100, 5000
    x = rng.standard_normal((R, V), dtype=np.float32)
    for r in range(0, R, 7):
        x[r, rng.choice(V, 300 + r % 900, replace=False)] = np.float32(6.0)
    for k in (1, 8, 16):
        _topk_case(P, x, k)
        _topk_case(P, W.f32_to_bf16_bits(x), k)


@pytest.mark.parametrize("V", [32000, 3001])
def test_topk_signed_zero_ties(P, V):
    # the best values are zeros of both signs: they tie, lower index first
    rng = np.random.default_rng(V)
    x = -np.abs(rng.standard_normal((4, V), dtype=np.float32)) - np.float32(0.5)
    for r in range(4):
        pos = rng.choice(V, 12, replace=False)
        x[r, pos] = np.where(np.arange(12) % 2 == r % 2, np.float32(-0.0), np.float32(0.0))
    for k in (1, 5, 16):
        _topk_case(P, x, k)
        _topk_case(P, W.f32_to_bf16_bits(x), k)


@pytest.mark.parametrize("n", [63, 64, 65, 100, 700])
def test_topk_candidate_counts(P, n):
    # n values tie at the top: ranked by counting up to 64, merged above
    rng = np.random.default_rng(n)
    x = rng.standard_normal((3, 32000), dtype=np.float32)
    for r in range(3):
        x[r, rng.choice(32000, n, replace=False)] = np.float32(7.5)
    for k in (4, 16):
        _topk_case(P, x, k)
        _topk_case(P, W.f32_to_bf16_bits(x), k)


def test_topk_golden(P):
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "topk_ties.json")))
    rows = np.array(g["rows"], np.float32)
    am, idx, val = P.topk_argmax(cu(rows), g["k"])
    assert am.cpu().tolist() == g["argmax"]
    assert idx.cpu().tolist() == g["topk_idx"]
    assert np.signbit(val.cpu().numpy()[0, 4])


# ---------------------------------------------------------------------------
# verification
# ---------------------------------------------------------------------------
def test_verify_random(P):
    rng = np.random.default_rng(3)
    for T in (1, 5, 64, 96, 1024):
        B = 6
        par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
        tok = rng.integers(0, 3, (B, T)).astype(np.int32)
        am = rng.integers(0, 3, (B, T + 1)).astype(np.int32)
        tl = rng.integers(0, T + 1, B).astype(np.int32)
        for tree_len in (None, tl):
            ref = O.verify(am, tok, par, tree_len)
            st = status_buf()
            got = P.verify(cu(am), cu(tok), cu(par), None if tree_len is None else cu(tree_len), st)
            torch.cuda.synchronize()
            assert st.item() == 0
            for g, r in zip(got, ref):
                assert np.array_equal(g.cpu().numpy(), r), T


def test_verify_golden_and_bad_tree(P):
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "verify_example.json")))
    for c in g["cases"]:
        al, an, ot = P.verify(cu(np.array([c["argmax"]], np.int32)),
                              cu(np.array([c["tokens"]], np.int32)),
                              cu(np.array([c["parent"]], np.int32)))
        assert al.item() == c["accept_len"]
        assert an.cpu().tolist()[0] == c["accept_nodes"]
        assert ot.cpu().tolist()[0] == c["out_tokens"]
    st = status_buf()
    P.verify(cu(np.zeros((1, 4), np.int32)), cu(np.zeros((1, 3), np.int32)),
             cu(np.array([[-1, 1, 0]], np.int32)), None, st)
    torch.cuda.synchronize()
    assert st.item() == 7


# ---------------------------------------------------------------------------
# expansion
# ---------------------------------------------------------------------------
def test_expand_random(P):
    rng = np.random.default_rng(4)
    for trial in range(40):
        B = 3
        T = int(rng.choice([1, 7, 33, 64, 200]))
        k = int(rng.integers(1, 9))
        d_max = int(rng.integers(1, 8))
        width = rng.integers(1, 5, d_max).astype(np.int32)
        T_max = int(rng.choice([1, T, 2 * T, 1024]))
        par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
        tok = np.stack([W.sibling_distinct_tokens(rng, par[b], 20) for b in range(B)])
        ti = rng.integers(0, 20, (B, T + 1, k)).astype(np.int32)
        tl = rng.integers(1, T + 1, B).astype(np.int32) if trial % 2 else None
        ref = O.expand(par, tok, ti, width, d_max, T_max, tl)
        got = P.expand(cu(par), cu(tok), cu(ti), width.tolist(), d_max, T_max,
                       None if tl is None else cu(tl))
        for g, r in zip(got, ref):
            assert np.array_equal(g.cpu().numpy(), r), (trial, T, k, d_max, T_max)


def test_verify_expand_fused(P):
    rng = np.random.default_rng(14)
    for trial in range(20):
        B = 4
        T = int(rng.choice([1, 16, 64, 96, 300]))
        k = int(rng.integers(1, 9))
        d_max = int(rng.integers(1, 7))
        width = rng.integers(1, 5, d_max).astype(np.int32)
        T_max = int(rng.choice([T, 2 * T, 1024]))
        par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
        tok = rng.integers(0, 6, (B, T)).astype(np.int32)  # duplicate siblings allowed
        am = rng.integers(0, 6, (B, T + 1)).astype(np.int32)
        ti = rng.integers(0, 6, (B, T + 1, k)).astype(np.int32)
        tl = rng.integers(1, T + 1, B).astype(np.int32) if trial % 2 else None
        ref = O.verify(am, tok, par, tl) + O.expand(par, tok, ti, width, d_max, T_max, tl)
        got = P.verify_expand(cu(am), cu(tok), cu(par), cu(ti), width.tolist(), d_max, T_max,
                              None if tl is None else cu(tl))
        for g, r in zip(got, ref):
            assert np.array_equal(g.cpu().numpy(), r), (trial, T, k)


def _small_tree(rng, T):
    kind = int(rng.integers(4))
    if kind == 0:
        return W.tree_chain(T)[0]
    if kind == 1:
        return W.tree_star(T)[0]
    if kind == 2:
        br = [int(x) for x in rng.integers(1, 5, 8)]
        par = W.tree_branching(br, T)[0]
        if par.shape[0] == T:
            return par
    return W.tree_uniform(rng, T)[0]


@pytest.mark.parametrize("seed", range(4))
def test_verify_expand_small_trees(P, seed):
    # trees of <= 64 nodes (one wave per sequence): chains, stars, level-built
    # and uniform trees, k up to 16, deep depth caps, cuts below T
    rng = np.random.default_rng(200 + seed)
    for trial in range(25):
        B = int(rng.integers(1, 5))
        T = int(rng.choice([1, 2, 5, 31, 63, 64]))
        k = int(rng.integers(1, 17))
        d_max = int(rng.integers(1, 65))
        width = rng.integers(1, 6, d_max).astype(np.int32)
        T_max = int(rng.integers(1, 65))
        par = np.stack([_small_tree(rng, T) for _ in range(B)])
        V = int(rng.choice([3, 8, 1000]))
        tok = rng.integers(0, V, (B, T)).astype(np.int32)
        am = rng.integers(0, V, (B, T + 1)).astype(np.int32)
        if trial % 3 == 0:  # plant accepted chains: every node's token is its parent's argmax
            for b in range(B):
                for i in range(T):
                    tok[b, i] = am[b, par[b, i] + 1]
        ti = rng.integers(0, V, (B, T + 1, k)).astype(np.int32)
        tl = rng.integers(0, T + 1, B).astype(np.int32) if trial % 2 else None
        ref_v = O.verify(am, tok, par, tl)
        ref_e = O.expand(par, tok, ti, width, d_max, T_max, tl)
        got = P.verify_expand(cu(am), cu(tok), cu(par), cu(ti), width.tolist(), d_max, T_max,
                              None if tl is None else cu(tl))
        for g, r in zip(got, ref_v + ref_e):
            assert np.array_equal(g.cpu().numpy(), r), (seed, trial, T, k, d_max, T_max)
        got_v = P.verify(cu(am), cu(tok), cu(par), None if tl is None else cu(tl))
        got_e = P.expand(cu(par), cu(tok), cu(ti), width.tolist(), d_max, T_max,
                         None if tl is None else cu(tl))
        for g, r in zip(tuple(got_v) + tuple(got_e), ref_v + ref_e):
            assert np.array_equal(g.cpu().numpy(), r), (seed, trial, T, k, d_max, T_max)


@pytest.mark.parametrize("seed", range(4))
def test_verify_expand_mid_trees(P, seed):
    # trees of 65-128 nodes and cuts up to 128 (one wave, two nodes per
    # lane), and small trees cut above 64: chains, stars, level-built and
    # uniform trees, k up to 16, deep depth caps
    rng = np.random.default_rng(300 + seed)
    for trial in range(25):
        B = int(rng.integers(1, 5))
        T = int(rng.choice([7, 64, 65, 96, 127, 128]))
        k = int(rng.integers(1, 17))
        d_max = int(rng.integers(1, 65))
        width = rng.integers(1, 6, d_max).astype(np.int32)
        T_max = int(rng.integers(65, 129)) if T <= 64 else int(rng.integers(1, 129))
        par = np.stack([_small_tree(rng, T) for _ in range(B)])
        V = int(rng.choice([3, 8, 1000]))
        tok = rng.integers(0, V, (B, T)).astype(np.int32)
        am = rng.integers(0, V, (B, T + 1)).astype(np.int32)
        if trial % 3 == 0:  # plant accepted chains: every node's token is its parent's argmax
            for b in range(B):
                for i in range(T):
                    tok[b, i] = am[b, par[b, i] + 1]
        ti = rng.integers(0, V, (B, T + 1, k)).astype(np.int32)
        tl = rng.integers(0, T + 1, B).astype(np.int32) if trial % 2 else None
        ref_v = O.verify(am, tok, par, tl)
        ref_e = O.expand(par, tok, ti, width, d_max, T_max, tl)
        got = P.verify_expand(cu(am), cu(tok), cu(par), cu(ti), width.tolist(), d_max, T_max,
                              None if tl is None else cu(tl))
        for j, (g, r) in enumerate(zip(got, ref_v + ref_e)):
            g = g.cpu().numpy()
            assert np.array_equal(g, r), f"{(seed, trial, T, k, d_max, T_max)} output {j}: {_diff(g, r)}"
        got_v = P.verify(cu(am), cu(tok), cu(par), None if tl is None else cu(tl))
        got_e = P.expand(cu(par), cu(tok), cu(ti), width.tolist(), d_max, T_max,
                         None if tl is None else cu(tl))
        for j, (g, r) in enumerate(zip(tuple(got_v) + tuple(got_e), ref_v + ref_e)):
            g = g.cpu().numpy()
            assert np.array_equal(g, r), f"{(seed, trial, T, k, d_max, T_max)} output {j}: {_diff(g, r)}"


@pytest.mark.parametrize("T,top", [(40, 31), (64, 31), (110, 95), (128, 95)])
def test_verify_path_through_bit_31(P, T, top):
    # accepted chain 0..top (top = 31 or 95: bit 31 of a path-mask word) and
    # live roots above it that are not accepted: the path mask of the
    # terminal must not leak into the nodes above top
    par = np.full((1, T), -1, np.int32)
    par[0, 1:top + 1] = np.arange(top)
    am = np.arange(1, T + 2, dtype=np.int32)[None, :] % 7
    tok = np.empty((1, T), np.int32)
    for i in range(T):
        tok[0, i] = am[0, par[0, i] + 1] if i <= top else (am[0, 0] + 1) % 7
    ref = O.verify(am, tok, par)
    assert ref[0][0] == top + 1
    got = P.verify(cu(am), cu(tok), cu(par))
    for j, (g, r) in enumerate(zip(got, ref)):
        g = g.cpu().numpy()
        assert np.array_equal(g, r), f"output {j}: {_diff(g, r)}"
    ti = np.zeros((1, T + 1, 2), np.int32)
    ref_e = O.expand(par, tok, ti, np.array([2] * 8, np.int32), 8, T)
    got = P.verify_expand(cu(am), cu(tok), cu(par), cu(ti), [2] * 8, 8, T)
    for j, (g, r) in enumerate(zip(got, ref + ref_e)):
        g = g.cpu().numpy()
        assert np.array_equal(g, r), f"output {j}: {_diff(g, r)}"


def _diff(got, ref):
    """The first few differing positions as (index, got, expected)."""
    if got.shape != ref.shape:
        return ("shape", got.shape, ref.shape)
    idx = np.argwhere(got != ref)[:6]
    return [(tuple(int(v) for v in i), int(got[tuple(i)]), int(ref[tuple(i)])) for i in idx]


@pytest.mark.parametrize("T", [9, 64, 100, 128, 129])
def test_verify_expand_bad_tree_rejects(P, T):
    par = W.tree_chain(T)[0][None, :].copy()
    par[0, T // 2] = T // 2  # its own parent
    st = status_buf()
    z = np.zeros((1, T + 1), np.int32)
    got = P.verify_expand(cu(z), cu(z[:, :T]), cu(par), cu(np.zeros((1, T + 1, 2), np.int32)),
                          [2] * 4, 4, T, None, st)
    torch.cuda.synchronize()
    assert st.item() == 7
    al, an, ot, pn, tn, ln = (g.cpu().numpy() for g in got)
    assert al[0] == 0 and ln[0] == 0
    assert (an == -1).all() and (ot == -1).all() and (pn == -1).all() and (tn == -1).all()


def test_expand_golden(P):
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "expand_example.json")))
    for c in g["cases"]:
        pn, tn, ln = P.expand(cu(np.array([g["parent"]], np.int32)),
                              cu(np.array([g["tokens"]], np.int32)),
                              cu(np.array([g["topk_idx"]], np.int32)),
                              g["width_sched"], c["d_max"], c["T_max"])
        assert pn.cpu().tolist()[0] == c["parent_next"]
        assert tn.cpu().tolist()[0] == c["tokens_next"]
        assert ln.item() == c["tree_len_next"]


# ---------------------------------------------------------------------------
# tree attention
# ---------------------------------------------------------------------------
def _attn_gpu(P, w, out_dtype=None, with_mask=False):
    q, kc, vc = cu(w.q), cu(w.k_cache), cu(w.v_cache)
    kvl, par = cu(w.kv_len), cu(w.parent)
    mask = P.tree_mask(par)[0] if with_mask else None
    st = status_buf()
    out = P.tree_attention(q, kc, vc, kvl, par, mask=mask, out_dtype=out_dtype,
                           dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    return out.float().cpu().numpy().astype(np.float64)


def _spec(**kw):
    base = dict(B=1, Hq=4, Hkv=4, D=128, kv_len=100, T=16, tree="uniform", V=16,
                dtype="bf16", plant=None, k=2)
    base.update(kw)
    return base


SMALL = [
    _spec(),
    _spec(D=64, Hq=2, Hkv=2, T=33, kv_len=0),
    _spec(tree="chain", T=65, kv_len=7),
    _spec(tree="star", T=64, kv_len=300, V=1000),
    _spec(B=3, Hq=8, Hkv=2, T=20, kv_len=[0, 129, 640]),
    _spec(Hq=32, Hkv=8, T=64, kv_len=1000),          # 256 query rows per KV head
    _spec(Hq=6, Hkv=1, T=96, kv_len=255),            # 576 rows: several row passes
    _spec(T=1, kv_len=2047),                         # plain decode
    _spec(T=130, kv_len=33, Hq=2, Hkv=2),            # three mask words
    _spec(D=64, Hq=4, Hkv=2, T=9, kv_len=5000, L_pad=40),
    _spec(tree="chain", T=128, kv_len=40, Hq=2, Hkv=2),  # walks of 128 nodes
    _spec(Hq=2, Hkv=2, T=100, kv_len=3000),          # two words, many KV splits
    _spec(Hq=1, Hkv=1, T=8, kv_len=12000),           # 47 KV splits: three combine groups
    # batches taken largest first: 64 sequences (every lane ranks one; 64
    # (b, g) pairs dealt over the XCDs), 12 with equal sizes (ties in index
    # order; 24 pairs), 5 (pairs not a multiple of 8: contiguous XCD ranges),
    # and 65 (beyond one wave: index order)
    _spec(B=64, Hq=2, Hkv=1, T=8, kv_len=[(37 * i) % 300 for i in range(64)]),
    _spec(B=12, Hq=4, Hkv=2, T=16, kv_len=[200, 50, 200, 200, 0, 50, 700, 700, 3, 200, 50, 700]),
    _spec(B=5, Hq=2, Hkv=1, T=20, kv_len=[10, 900, 300, 900, 1]),
    _spec(B=65, Hq=2, Hkv=1, T=4, kv_len=[(53 * i) % 400 for i in range(65)]),
    # batches in 128-row passes (256-thread workgroups, two per CU), D = 64 too
    _spec(B=2, Hq=8, Hkv=2, T=40, kv_len=[300, 1200]),
    _spec(D=64, B=3, Hq=8, Hkv=2, T=40, kv_len=[1200, 0, 450]),
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_attention_small_full(P, case):
    w = W.make_workload(SMALL[case], seed=100 + case, logits=False)
    ref = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale)
    for od in (torch.float32, torch.bfloat16):
        got = _attn_gpu(P, w, out_dtype=od, with_mask=(case % 2 == 0))
        tol = TOL["bf16"] if od == torch.float32 else TOL["bf16"] + 2 ** -8 * np.abs(ref).max()
        err = np.abs(got - ref).max()
        assert err <= tol, (case, od, err)


@pytest.mark.parametrize("spec", [
    _spec(dtype="f32", D=64, Hq=2, Hkv=2, T=16, kv_len=128),
    _spec(dtype="f32", D=128, Hq=4, Hkv=2, T=40, kv_len=[77], tree="chain"),
    _spec(dtype="f32", D=64, Hq=3, Hkv=3, B=2, T=70, kv_len=[0, 200]),
])
def test_attention_fp32_full(P, spec):
    w = W.make_workload(spec, seed=7, logits=False)
    ref = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale)
    got = _attn_gpu(P, w, out_dtype=torch.float32)
    assert np.abs(got - ref).max() <= TOL["f32"]


def test_attention_tiny_config(P):
    w = W.make_workload("tiny", logits=False)
    ref = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale)
    got = _attn_gpu(P, w)
    assert np.abs(got - ref).max() <= TOL["f32"]


def _sample_rows(w, n, seed):
    rng = np.random.default_rng(seed)
    rows = {(0, 0, 0), (w.B - 1, w.Hq - 1, w.T - 1), (0, w.Hq // 2, w.T // 2)}
    while len(rows) < n:
        rows.add((int(rng.integers(w.B)), int(rng.integers(w.Hq)), int(rng.integers(w.T))))
    return sorted(rows)


@pytest.mark.parametrize("name", ["llama2-7b", "llama2-13b", "llama3-8b-long", "ragged-16"])
def test_attention_configs_sampled(P, name):
    w = W.make_workload(name, logits=False)
    got = _attn_gpu(P, w, with_mask=True)  # bf16 out, as the step runs it
    got32 = _attn_gpu(P, w, out_dtype=torch.float32, with_mask=True)
    rows = _sample_rows(w, 40, 1)
    ref = O.attention_rows(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale, rows)
    for n, (b, h, i) in enumerate(rows):
        assert np.abs(got32[b, i, h] - ref[n]).max() <= TOL["bf16"], (b, h, i)
        assert np.abs(got[b, i, h] - ref[n]).max() <= TOL["bf16"] + 2 ** -8 * np.abs(ref[n]).max()
    assert np.isfinite(got).all()


def _dominant_case(seed, B, kvl, Hq, Hkv, T, n_dom, extra):
    """Inputs where n_dom keys per KV head hold much of the softmax weight of
    the head's query rows: the keys point along the mean query direction,
    scaled so that for the median row their scores lead the unit-variance
    scores of the other keys by log(1.65 kv_len) + extra (a lead of
    log(1.65 kv_len) alone gives one such key about half the weight)."""
    rng = np.random.default_rng(seed)
    D, G = 128, Hq // Hkv
    par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)]).astype(np.int32)
    q = rng.standard_normal((B, T, Hq, D)).astype(np.float32)
    kc = rng.standard_normal((B, Hkv, kvl + T, D)).astype(np.float32)
    vc = (rng.standard_normal((B, Hkv, kvl + T, D)) * 2.0).astype(np.float32)
    lead = np.log(1.65 * kvl) + extra
    for b in range(B):
        for g in range(Hkv):
            rows = q[b, :, g * G:(g + 1) * G].reshape(-1, D)
            qs = rows.sum(0)
            qs /= np.linalg.norm(qs)
            alpha = lead / np.median(rows @ qs / np.sqrt(D))
            for d in range(n_dom):
                j = int(rng.integers(40, kvl))
                kc[b, g, j] = qs * alpha * (1.0 + 0.02 * d)
    return (W.f32_to_bf16_bits(q), W.f32_to_bf16_bits(kc), W.f32_to_bf16_bits(vc),
            np.full(B, kvl, np.int32), par)


# (seed, B, kv_len, Hq, Hkv, T, keys holding the weight, extra lead).  Some
# run through several KV splits (long sequences, few heads).
DOMINANT = [(1, 1, 1024, 8, 8, 16, 1, 0.0), (3, 2, 1024, 8, 8, 16, 2, 1.0),
            (5, 3, 700, 8, 8, 32, 2, 0.0), (2, 1, 2000, 32, 8, 64, 1, 1.0),
            (6, 1, 1024, 4, 4, 4, 4, 2.0), (4, 2, 4096, 32, 8, 64, 2, 0.5),
            (7, 1, 20000, 8, 8, 16, 1, 0.0), (8, 1, 30000, 8, 1, 1, 2, 1.0)]


@pytest.mark.parametrize("case", DOMINANT)
def test_attention_dominant_keys(P, case):
    q, kc, vc, kvl, par = _dominant_case(*case)
    ref = O.tree_attention(q, kc, vc, kvl, par, 1 / np.sqrt(128))
    st = status_buf()
    out = P.tree_attention(cu(q), cu(kc), cu(vc), cu(kvl), cu(par), out_dtype=torch.float32,
                           dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    err = np.abs(out.cpu().numpy().astype(np.float64) - ref).max()
    assert err <= TOL["bf16"], (case, err)


def test_attention_deterministic(P):
    w = W.make_workload(_spec(Hq=32, Hkv=8, T=64, kv_len=3000), seed=9, logits=False)
    a = _attn_gpu(P, w, out_dtype=torch.float32)
    b = _attn_gpu(P, w, out_dtype=torch.float32)
    assert np.array_equal(a, b)


def test_attention_workspace_reuse(P):
    # one workspace (not initialised) through calls of different shapes: the
    # split arrival words must neither need zeroing nor leak between calls
    specs = [_spec(Hq=8, Hkv=8, T=64, kv_len=2000), _spec(Hq=2, Hkv=2, T=100, kv_len=3000),
             _spec(Hq=8, Hkv=8, T=64, kv_len=2000)]
    ws = torch.full((1 << 24,), 0x5A, dtype=torch.uint8, device="cuda")
    for n, sp in enumerate(specs):
        w = W.make_workload(sp, seed=40 + n, logits=False)
        ref = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale)
        for rep in range(2):
            st = status_buf()
            out = P.tree_attention(cu(w.q), cu(w.k_cache), cu(w.v_cache), cu(w.kv_len),
                                   cu(w.parent), out_dtype=torch.float32, workspace=ws,
                                   dev_status=st)
            torch.cuda.synchronize()
            assert st.item() == 0
            err = np.abs(out.cpu().numpy().astype(np.float64) - ref).max()
            assert err <= TOL["bf16"], (n, rep, err)


@pytest.mark.parametrize("T", [20, 130])
def test_attention_bad_tree_reports(P, T):
    w = W.make_workload(_spec(T=T, kv_len=50), seed=5, logits=False)
    w.parent[0, T // 2] = T // 2 + 3  # not topological
    st = status_buf()
    P.tree_attention(cu(w.q), cu(w.k_cache), cu(w.v_cache), cu(w.kv_len), cu(w.parent),
                     dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 7


def test_attention_kv_len_too_long_reports(P):
    w = W.make_workload(_spec(T=8, kv_len=50), seed=3, logits=False)
    w.kv_len[0] = w.L_cap  # kv_len + T > L_cap
    q, kc, vc = cu(w.q), cu(w.k_cache), cu(w.v_cache)
    st = status_buf()
    P.tree_attention(q, kc, vc, cu(w.kv_len), cu(w.parent), dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 8


@pytest.mark.parametrize("bad", [-5, 2 ** 31 - 1])
def test_attention_bad_kv_len_in_a_batch(P, bad):
    # a batch taken largest first with one invalid length (negative, or near
    # the int range): reported, and the other sequences are still right
    spec = _spec(B=4, Hq=32, Hkv=8, T=40, kv_len=[300, 40, 900, 120])
    w = W.make_workload(spec, seed=11, logits=False)
    ref = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale)
    kvl = w.kv_len.copy()
    kvl[1] = bad
    st = status_buf()
    got = P.tree_attention(cu(w.q), cu(w.k_cache), cu(w.v_cache), cu(kvl), cu(w.parent),
                           out_dtype=torch.float32, dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 8
    got = got.cpu().numpy()
    for b in (0, 2, 3):
        assert np.abs(got[b] - ref[b]).max() <= TOL["bf16"], b


# ---------------------------------------------------------------------------
# one whole step through the C ABI
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["tiny", "llama2-7b"])
def test_full_step(P, name):
    w = W.make_workload(name)
    B, T = w.B, w.T
    par, tok = cu(w.parent), cu(w.tokens)
    mask, depth = P.tree_mask(par)
    out = P.tree_attention(cu(w.q), cu(w.k_cache), cu(w.v_cache), cu(w.kv_len), par, mask=mask)
    am, idx, val = P.topk_argmax(cu(w.logits), w.k)
    al, an, ot = P.verify(am.view(B, T + 1), tok, par)
    pn, tn, ln = P.expand(par, tok, idx.view(B, T + 1, w.k), w.width, w.d_max, w.T_max)
    torch.cuda.synchronize()
    r_am, r_idx, _ = O.topk(w.logits, w.k)
    assert np.array_equal(am.cpu().numpy(), r_am)
    r_al, r_an, r_ot = O.verify(r_am.reshape(B, -1), w.tokens, w.parent)
    assert al.cpu().tolist() == r_al.tolist() == w.planted_depth.tolist()
    assert np.array_equal(an.cpu().numpy(), r_an) and np.array_equal(ot.cpu().numpy(), r_ot)
    r_pn, r_tn, r_ln = O.expand(w.parent, w.tokens, r_idx.reshape(B, T + 1, w.k), w.width,
                                w.d_max, w.T_max)
    assert np.array_equal(pn.cpu().numpy(), r_pn) and np.array_equal(tn.cpu().numpy(), r_tn)
    assert np.array_equal(ln.cpu().numpy(), r_ln)
    rows = _sample_rows(w, 12, 2)
    ref = O.attention_rows(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale, rows)
    o = out.float().cpu().numpy()
    for n, (b, h, i) in enumerate(rows):
        assert np.abs(o[b, i, h] - ref[n]).max() <= TOL[w.dtype] + (
            2 ** -8 * np.abs(ref[n]).max() if w.dtype == "bf16" else 0)
