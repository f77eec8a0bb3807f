"""GPU parity of tree attention on 8-bit (OCP E4M3) key/value caches with
per-KV-head scales (ptd_tree_attention_fp8kv), through the C ABI, against the
fp64 CPU oracle (which decodes the codes from the format's definition).

The kernel widens the codes to bf16 exactly and runs the bf16 path's
arithmetic, so the bar is the bf16 path's: fp32 outputs within 2e-3 of the
oracle; with unit scales its outputs equal, bit for bit, the bf16 kernel's on
caches holding the decoded values."""
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


def make(rng, B, T, Hq, Hkv, L, amp=1.0):
    q = W.f32_to_bf16_bits(rng.standard_normal((B, T, Hq, 128)).astype(np.float32))
    kq, ks = W.quantize_kv_e4m3(rng.standard_normal((B, Hkv, L, 128)) * amp)
    vq, vs = W.quantize_kv_e4m3(rng.standard_normal((B, Hkv, L, 128)) * amp)
    return q, kq, ks, vq, vs


def run(P, q, kq, ks, vq, vs, kv_len, parent, tree_len=None, out_dtype=torch.float32):
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = P.tree_attention_fp8kv(cu(q), cu(kq), cu(vq), None if ks is None else cu(ks),
                                 None if vs is None else cu(vs), cu(kv_len), cu(parent),
                                 out_dtype=out_dtype, dev_status=st,
                                 tree_len=None if tree_len is None else cu(tree_len))
    torch.cuda.synchronize()
    assert st.item() == 0
    return out


@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (4, 4), (32, 8)])
def test_fp8kv_small_vs_oracle(P, Hq, Hkv):
    rng = np.random.default_rng(Hq + Hkv)
    B, T, L = 3, 13, 1100
    q, kq, ks, vq, vs = make(rng, B, T, Hq, Hkv, L)
    kv_len = np.array([0, 300, L - T], np.int32)
    parent = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    got = run(P, q, kq, ks, vq, vs, kv_len, parent).cpu().numpy()
    ref = O.tree_attention_fp8kv(q, kq, vq, ks, vs, kv_len, parent, 1.0 / np.sqrt(128))
    assert np.abs(got - ref).max() <= TOL


@pytest.mark.parametrize("T", [1, 64, 150])
def test_fp8kv_tree_sizes(P, T):
    rng = np.random.default_rng(T)
    B, L = 2, 900 + T
    q, kq, ks, vq, vs = make(rng, B, T, 8, 8, L)
    kv_len = np.array([200, L - T], np.int32)
    parent = np.stack([W.tree_chain(T)[0], W.tree_uniform(rng, T)[0]])
    got = run(P, q, kq, ks, vq, vs, kv_len, parent).cpu().numpy()
    if T <= 64:
        ref = O.tree_attention_fp8kv(q, kq, vq, ks, vs, kv_len, parent, 1.0 / np.sqrt(128))
        assert np.abs(got - ref).max() <= TOL
    else:
        rows = [(0, 3, T - 1), (1, 7, 0), (1, 0, T // 2), (0, 5, 77)]
        ref = O.tree_attention_fp8kv(q, kq, vq, ks, vs, kv_len, parent, 1.0 / np.sqrt(128),
                                     rows=rows)
        for n, (b, h, i) in enumerate(rows):
            assert np.abs(got[b, i, h] - ref[n]).max() <= TOL, (b, h, i)


def test_fp8kv_unit_scales_equal_bf16_kernel_on_decoded_caches(P):
    rng = np.random.default_rng(20)
    B, T, L = 2, 64, 2112
    q, kq, _, vq, _ = make(rng, B, T, 32, 32, L)
    kv_len = np.array([L - T, 700], np.int32)
    parent = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    a = run(P, q, kq, None, vq, None, kv_len, parent, out_dtype=torch.bfloat16)
    kb = W.f32_to_bf16_bits(O.e4m3_decode(kq).astype(np.float32))
    vb = W.f32_to_bf16_bits(O.e4m3_decode(vq).astype(np.float32))
    b = P.tree_attention(cu(q), cu(kb), cu(vb), cu(kv_len), cu(parent))
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_fp8kv_unit_scales_equal_bf16_kernel_batch_of_long_groups(P):
    # 256 query rows per KV head in a batch: the 256-thread workgroups, two
    # per CU, for both kernels
    rng = np.random.default_rng(22)
    B, T, L = 3, 64, 1500
    q, kq, _, vq, _ = make(rng, B, T, 32, 8, L)
    kv_len = np.array([L - T, 333, 1000], np.int32)
    parent = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    a = run(P, q, kq, None, vq, None, kv_len, parent, out_dtype=torch.bfloat16)
    kb = W.f32_to_bf16_bits(O.e4m3_decode(kq).astype(np.float32))
    vb = W.f32_to_bf16_bits(O.e4m3_decode(vq).astype(np.float32))
    b = P.tree_attention(cu(q), cu(kb), cu(vb), cu(kv_len), cu(parent))
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    # unit scales leave the codes' own range (up to 448): the bound relative
    # to the values' scale, as for scaled caches
    ref = O.tree_attention(q, kb, vb, kv_len, parent, 1.0 / np.sqrt(128))
    got = run(P, q, kq, None, vq, None, kv_len, parent).cpu().numpy()
    assert np.abs(got - ref).max() <= TOL * np.abs(ref).max() / 4


def test_fp8kv_ragged_and_scales(P):
    rng = np.random.default_rng(21)
    B, T, L = 4, 20, 600
    q, kq, ks, vq, vs = make(rng, B, T, 8, 2, L, amp=30.0)
    kv_len = np.array([100, 0, 500, 7], np.int32)
    tl = np.array([20, 3, 0, 11], np.int32)
    parent = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    got = run(P, q, kq, ks, vq, vs, kv_len, parent, tree_len=tl).cpu().numpy()
    ref = O.tree_attention_fp8kv(q, kq, vq, ks, vs, kv_len, parent, 1.0 / np.sqrt(128),
                                 tree_len=tl)
    # values of amplitude ~30: the bf16-path bound relative to that scale
    assert np.abs(got - ref).max() <= TOL * 30
    for b in range(B):
        assert np.all(got[b, tl[b]:] == 0.0)


def test_fp8kv_gqa_long_context_sampled(P):
    # the GQA long-context shape (32 query / 8 KV heads, 32768 committed keys)
    # with its caches quantized to E4M3 per KV head
    w = W.make_workload("llama3-8b-long")
    kq, ks = W.quantize_kv_e4m3(W.bf16_bits_to_f32(w.k_cache))
    vq, vs = W.quantize_kv_e4m3(W.bf16_bits_to_f32(w.v_cache))
    got = run(P, w.q, kq, ks, vq, vs, w.kv_len, w.parent).cpu().numpy()
    rng = np.random.default_rng(22)
    rows = [(0, int(rng.integers(0, w.Hq)), int(rng.integers(0, w.T))) for _ in range(10)]
    ref = O.tree_attention_fp8kv(w.q, kq, vq, ks, vs, w.kv_len, w.parent, w.scale, rows=rows)
    for n, (b, h, i) in enumerate(rows):
        assert np.abs(got[b, i, h] - ref[n]).max() <= TOL, (b, h, i)


@pytest.mark.parametrize("ps", [32, 128])
def test_fp8kv_paged_matches_contiguous(P, ps):
    # E4M3 caches scattered over pages through a random table: bit for bit the
    # contiguous 8-bit call (same arithmetic), and within the bound of the oracle
    rng = np.random.default_rng(30 + ps)
    B, T, Hkv, L = 3, 24, 4, 1024
    q, kq, ks, vq, vs = make(rng, B, T, 16, Hkv, L)
    kv_len = np.array([0, 500, L - T], np.int32)
    tl = np.array([24, 9, 17], np.int32)
    parent = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    maxp = L // ps
    table = rng.permutation(B * maxp + 3)[:B * maxp].reshape(B, maxp).astype(np.int32)
    kp = rng.integers(0, 0x7E, (B * maxp + 3, Hkv, ps, 128)).astype(np.uint8)  # noise pages
    vp = kp.copy()
    for b in range(B):
        for j in range(maxp):
            kp[table[b, j]] = kq[b, :, j * ps:(j + 1) * ps]
            vp[table[b, j]] = vq[b, :, j * ps:(j + 1) * ps]
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    paged = P.tree_attention_paged(cu(q), cu(kp), cu(vp), cu(table), cu(kv_len), cu(parent),
                                   out_dtype=torch.float32, dev_status=st, tree_len=cu(tl),
                                   k_scale=cu(ks), v_scale=cu(vs))
    contig = run(P, q, kq, ks, vq, vs, kv_len, parent, tree_len=tl)
    torch.cuda.synchronize()
    assert st.item() == 0
    assert torch.equal(paged, contig)
    ref = O.tree_attention_fp8kv(q, kq, vq, ks, vs, kv_len, parent, 1.0 / np.sqrt(128),
                                 tree_len=tl)
    assert np.abs(paged.cpu().numpy() - ref).max() <= TOL


def test_fp8kv_tree_over_128_nodes_with_tree_len(P):
    rng = np.random.default_rng(40)
    B, T, L = 2, 144, 700
    q, kq, ks, vq, vs = make(rng, B, T, 8, 2, L)
    kv_len = np.array([300, 0], np.int32)
    tl = np.array([144, 100], np.int32)
    parent = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    parent[1, 100:] = 500  # padding parents: never read
    got = run(P, q, kq, ks, vq, vs, kv_len, parent, tree_len=tl).cpu().numpy()
    assert np.all(got[1, 100:] == 0.0)
    rows = [(0, 7, 143), (0, 2, 129), (1, 5, 99), (1, 0, 1)]
    ref = O.tree_attention_fp8kv(q, kq, vq, ks, vs, kv_len, parent, 1.0 / np.sqrt(128),
                                 tree_len=tl, rows=rows)
    for n, (b, h, i) in enumerate(rows):
        assert np.abs(got[b, i, h] - ref[n]).max() <= TOL, (b, h, i)
