"""GPU parity of tree attention on paged key/value caches
(ptd_tree_attention_paged), through the C ABI.  The oracle gathers the pages
into the contiguous cache and runs its attention on that; fp32 outputs must be
within 2e-3 of it (bf16 inputs, fp32 accumulation).  The paged kernel does the
same arithmetic as the contiguous one, so their bf16 outputs are also
compared bit for bit on the same data."""
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


def paginate(rng, cache, ps, spare=3):
    """Scatter a contiguous cache [B][Hkv][L][D] into pages through a random
    page table; unused pages hold noise."""
    B, Hkv, L, D = cache.shape
    maxp = L // ps
    num = B * maxp + spare
    table = rng.permutation(num)[:B * maxp].reshape(B, maxp).astype(np.int32)
    pages = W.f32_to_bf16_bits(rng.standard_normal((num, Hkv, ps, D)).astype(np.float32))
    for b in range(B):
        for j in range(maxp):
            pages[table[b, j]] = cache[b, :, j * ps:(j + 1) * ps]
    return pages, table


def run_paged(P, q, kp, vp, table, kv_len, parent, st=None, out_dtype=None):
    return P.tree_attention_paged(cu(q), cu(kp), cu(vp), cu(table), cu(kv_len), cu(parent),
                                  out_dtype=out_dtype, dev_status=st)


def case(P, rng, B, T, Hq, Hkv, D, L, ps, kv_len, parent, rows=None):
    q = W.f32_to_bf16_bits(rng.standard_normal((B, T, Hq, D)).astype(np.float32))
    kc = W.f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D)).astype(np.float32))
    vc = W.f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D)).astype(np.float32))
    kp, table = paginate(rng, kc, ps)
    vp = kp.copy()
    for b in range(B):  # V pages through the same table
        for j in range(L // ps):
            vp[table[b, j]] = vc[b, :, j * ps:(j + 1) * ps]
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = run_paged(P, q, kp, vp, table, kv_len, parent, st)
    out32 = run_paged(P, q, kp, vp, table, kv_len, parent, st, out_dtype=torch.float32)
    ref_contig = P.tree_attention(cu(q), cu(kc), cu(vc), cu(kv_len), cu(parent))
    torch.cuda.synchronize()
    assert st.item() == 0
    assert torch.equal(out.view(torch.int16), ref_contig.view(torch.int16))  # same arithmetic
    kg, vg = O.gather_pages(kp, table, ps), O.gather_pages(vp, table, ps)
    assert np.array_equal(kg, kc) and np.array_equal(vg, vc)
    got = out32.cpu().numpy()
    scale = 1.0 / np.sqrt(D)
    if rows is None:
        ref = O.tree_attention(q, kg, vg, kv_len, parent, scale)
        assert np.abs(got - ref).max() <= TOL
    else:
        ref = O.attention_rows(q, kg, vg, kv_len, parent, scale, rows)
        for n, (b, h, i) in enumerate(rows):
            assert np.abs(got[b, i, h] - ref[n]).max() <= TOL, (b, h, i)


@pytest.mark.parametrize("ps", [32, 64, 256])
@pytest.mark.parametrize("D,Hq,Hkv", [(128, 8, 2), (64, 4, 4)])
def test_paged_small(P, ps, D, Hq, Hkv):
    rng = np.random.default_rng(ps + D)
    B, T = 3, 13
    L = 1024
    parent = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    kv_len = np.array([0, 300, L - T], np.int32)
    case(P, rng, B, T, Hq, Hkv, D, L, ps, kv_len, parent)


@pytest.mark.parametrize("T", [1, 64, 130])
def test_paged_tree_sizes(P, T):
    rng = np.random.default_rng(T)
    B, L, ps = 2, 768, 64
    parent = np.stack([W.tree_chain(T)[0], W.tree_uniform(rng, T)[0]])
    kv_len = np.array([200, L - T], np.int32)
    case(P, rng, B, T, 8, 8, 128, L, ps, kv_len, parent)


@pytest.mark.parametrize("name,ps", [("llama2-7b", 64), ("llama3-8b-long", 32), ("ragged-16", 128)])
def test_paged_configs_sampled(P, name, ps):
    w = W.make_workload(name)
    rng = np.random.default_rng(7)
    L = w.L_cap
    L_pad = (L + ps - 1) // ps * ps
    kc, vc = w.k_cache, w.v_cache
    if L_pad != L:
        pad = ((0, 0), (0, 0), (0, L_pad - L), (0, 0))
        kc, vc = np.pad(kc, pad), np.pad(vc, pad)
    kp, table = paginate(rng, kc, ps, spare=1)
    vp = kp.copy()
    for b in range(w.B):
        for j in range(L_pad // ps):
            vp[table[b, j]] = vc[b, :, j * ps:(j + 1) * ps]
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = run_paged(P, w.q, kp, vp, table, w.kv_len, w.parent, st)
    out32 = run_paged(P, w.q, kp, vp, table, w.kv_len, w.parent, st, out_dtype=torch.float32)
    contig = P.tree_attention(cu(w.q), cu(kc), cu(vc), cu(w.kv_len), cu(w.parent))
    torch.cuda.synchronize()
    assert st.item() == 0
    assert torch.equal(out.view(torch.int16), contig.view(torch.int16))
    rows = [(int(rng.integers(0, w.B)), int(rng.integers(0, w.Hq)), int(rng.integers(0, w.T)))
            for _ in range(12)]
    ref = O.attention_rows(w.q, kc, vc, w.kv_len, w.parent, w.scale, rows)
    got = out32.cpu().numpy()
    for n, (b, h, i) in enumerate(rows):
        assert np.abs(got[b, i, h] - ref[n]).max() <= TOL, (b, h, i)


def test_paged_split_over_256_pages(P):
    # one split per (sequence, KV head) spans more than 256 pages of 32 rows:
    # page ids past the staged ones are read one by one
    rng = np.random.default_rng(8)
    B, Hkv, T, D, ps = 2, 128, 4, 64, 32
    L = 8320
    parent = np.stack([W.tree_chain(T)[0], W.tree_star(T)[0]])
    kv_len = np.array([L - T, 8300], np.int32)
    case(P, rng, B, T, Hkv, Hkv, D, L, ps, kv_len, parent,
         rows=[(0, 5, 3), (1, 127, 0), (0, 64, 1), (1, 0, 2)])


def test_paged_bad_page_id_reports(P):
    rng = np.random.default_rng(9)
    B, T, Hkv, D, ps, L = 1, 8, 2, 64, 32, 256
    kc = W.f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D)).astype(np.float32))
    kp, table = paginate(rng, kc, ps)
    table[0, 2] = kp.shape[0] + 5  # past the pages
    q = W.f32_to_bf16_bits(rng.standard_normal((B, T, Hkv, D)).astype(np.float32))
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    run_paged(P, q, kp, kp, table, np.array([100], np.int32), W.tree_chain(T)[0][None], st)
    torch.cuda.synchronize()
    assert st.item() == 10
