"""GPU parity of stepping (ptd_step_prune) and of the candidate pool
(ptd_pool_init / ptd_pool_merge / ptd_pool_retrieve) against the CPU oracle,
through the C ABI.  Every output is integer and must be bit-exact: the
stepped trees, and the candidate trees retrieved after every merge."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_10661_amd as lib
    return lib


def cu(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def trees(rng, B, T, kind):
    out = []
    for b in range(B):
        k = kind if kind != "mix" else ["uniform", "chain", "star", "branch"][b % 4]
        if k == "uniform":
            out.append(W.tree_uniform(rng, T)[0])
        elif k == "chain":
            out.append(W.tree_chain(T)[0])
        elif k == "star":
            out.append(W.tree_star(T)[0])
        else:
            out.append(W.tree_branching([3, 3, 2, 2, 2, 2], T)[0])
    return np.stack(out)


@pytest.mark.parametrize("T", [1, 7, 33, 64, 65, 96, 128])
@pytest.mark.parametrize("d_max", [1, 2, 3, 5])
def test_step_prune_random(P, T, d_max):
    rng = np.random.default_rng(T * 10 + d_max)
    B = 8
    par = trees(rng, B, T, "mix")
    tok = rng.integers(0, 50, (B, T)).astype(np.int32)
    tl = rng.integers(0, T + 1, B).astype(np.int32)
    for tree_len, T_max in ((None, T), (tl, max(1, T // 2)), (None, 64)):
        ref = O.step_prune(par, tok, d_max, T_max, tree_len)
        st = torch.zeros(1, dtype=torch.int32, device="cuda")
        got = P.step_prune(cu(par), cu(tok), d_max, T_max,
                           None if tree_len is None else cu(tree_len), st)
        torch.cuda.synchronize()
        assert st.item() == 0
        for r, g in zip(ref, got):
            assert np.array_equal(g.cpu().numpy(), r)


def test_step_prune_bad_tree(P):
    par = np.array([[-1, 0, 2, 1], [-1, 0, 1, 2]], np.int32)
    tok = np.arange(8, dtype=np.int32).reshape(2, 4)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    pn, tn, ln = P.step_prune(cu(par), cu(tok), 2, 4, None, st)
    torch.cuda.synchronize()
    assert st.item() == 7
    assert ln[0].item() == 0 and (pn[0] == -1).all()
    r = O.step_prune(par[1:], tok[1:], 2, 4)
    assert np.array_equal(pn[1].cpu().numpy(), r[0][0]) and ln[1].item() == r[2][0]


def pool_case(P, rng, B, T, V, e_max, n_cap, steps, T_max=64, kinds="mix"):
    ref = O.Pool(B, e_max, n_cap)
    gpu = P.Pool(B, e_max, n_cap)
    keys = np.arange(V + 1, dtype=np.int32)  # token V never occurs: always absent
    for step in range(steps):
        par = trees(rng, B, T, kinds)
        tok = rng.integers(0, V, (B, T)).astype(np.int32)
        tl = rng.integers(1, T + 1, B).astype(np.int32)
        ref.merge(par, tok, tl)
        st = torch.zeros(1, dtype=torch.int32, device="cuda")
        gpu.merge(cu(par), cu(tok), cu(tl), st)
        torch.cuda.synchronize()
        assert st.item() == 0
        for key in keys:
            last = np.full(B, key, np.int32)
            r = ref.retrieve(last, T_max)
            g = gpu.retrieve(cu(last), T_max)
            for a, c in zip(r, g):
                assert np.array_equal(c.cpu().numpy(), a), (step, key)


def test_pool_few_tokens_many_merges(P):
    # few token values: most sub-trees meet existing trees and nodes
    pool_case(P, np.random.default_rng(1), B=3, T=24, V=6, e_max=64, n_cap=64, steps=5)


def test_pool_bounds_drop_deterministically(P):
    # small trees and few of them: both bounds are hit
    pool_case(P, np.random.default_rng(2), B=4, T=40, V=12, e_max=5, n_cap=6, steps=4, T_max=8)


def test_pool_many_tokens_full_trees(P):
    pool_case(P, np.random.default_rng(3), B=2, T=64, V=500, e_max=2048, n_cap=64, steps=3)


@pytest.mark.parametrize("T,n_cap,V", [(65, 66, 30), (96, 97, 300), (128, 129, 40)])
def test_pool_large_trees(P, T, n_cap, V):
    # drafts of more than 64 nodes into trees of more than 64 nodes
    pool_case(P, np.random.default_rng(T), B=3, T=T, V=V, e_max=2048, n_cap=n_cap, steps=3,
              T_max=n_cap - 1)


def test_pool_more_touched_trees_than_staged(P):
    # about 120 distinct tokens per draft: the touched trees are staged in
    # two batches
    pool_case(P, np.random.default_rng(6), B=2, T=128, V=5000, e_max=2048, n_cap=129, steps=2,
              T_max=128)


def test_step_and_pool_13b_expanded_tree(P):
    # the 96-node trees that expansion builds for the 13B workload: stepped,
    # merged into a pool and retrieved by every token they hold
    w = W.make_workload("llama2-13b")
    B = w.B
    _, idx, _ = O.topk(w.logits, w.k)
    pn, tn, ln = O.expand(w.parent, w.tokens, idx.reshape(B, w.T + 1, w.k), w.width, w.d_max,
                          w.T_max)
    assert w.T_max == 96 and ln.max() > 64
    for d_max in (1, 2, 3, w.d_max - 1):
        ref = O.step_prune(pn, tn, d_max, w.T_max, ln)
        st = torch.zeros(1, dtype=torch.int32, device="cuda")
        got = P.step_prune(cu(pn), cu(tn), d_max, w.T_max, cu(ln), st)
        torch.cuda.synchronize()
        assert st.item() == 0
        for r, g in zip(ref, got):
            assert np.array_equal(g.cpu().numpy(), r), d_max
    ref = O.Pool(B, 2048, w.T_max + 1)
    gpu = P.Pool(B, 2048, w.T_max + 1)
    for step in range(2):
        ref.merge(pn, tn, ln)
        st = torch.zeros(1, dtype=torch.int32, device="cuda")
        gpu.merge(cu(pn), cu(tn), cu(ln), st)
        torch.cuda.synchronize()
        assert st.item() == 0
        for key in np.unique(tn[tn >= 0])[:64]:
            last = np.full(B, key, np.int32)
            r = ref.retrieve(last, w.T_max)
            g = gpu.retrieve(cu(last), w.T_max)
            for a, c in zip(r, g):
                assert np.array_equal(c.cpu().numpy(), a), (step, key)


def test_pool_bad_tree_leaves_pool(P):
    rng = np.random.default_rng(4)
    par = trees(rng, 2, 10, "uniform")
    tok = rng.integers(0, 5, (2, 10)).astype(np.int32)
    ref = O.Pool(2, 32, 16)
    gpu = P.Pool(2, 32, 16)
    ref.merge(par, tok)
    gpu.merge(cu(par), cu(tok))
    bad = par.copy()
    bad[0, 5] = 7  # not topological: sequence 0 is rejected, sequence 1 merges
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    gpu.merge(cu(bad), cu(tok), None, st)
    torch.cuda.synchronize()
    assert st.item() == 7
    ref_only1 = O.Pool(2, 32, 16)
    ref_only1.merge(par, tok)
    ref_only1.merge(par, tok, np.array([0, 10], np.int32))  # sequence 0: nothing merged
    for key in range(6):
        last = np.full(2, key, np.int32)
        r = ref_only1.retrieve(last, 16)
        g = gpu.retrieve(cu(last), 16)
        for a, c in zip(r, g):
            assert np.array_equal(c.cpu().numpy(), a), key


def test_pool_merge_deterministic(P):
    # the pool's internal layout (hash slots claimed concurrently, node records
    # past a tree's count) may differ between runs; every retrieval may not
    rng = np.random.default_rng(5)
    par = trees(rng, 4, 64, "mix")
    tok = rng.integers(0, 40, (4, 64)).astype(np.int32)
    outs = []
    for _ in range(2):
        gpu = P.Pool(4, 256, 32)
        gpu.merge(cu(par), cu(tok))
        res = []
        for key in range(41):
            res += [t.cpu() for t in gpu.retrieve(cu(np.full(4, key, np.int32)), 32)]
        outs.append(res)
    assert all(torch.equal(a, b) for a, b in zip(*outs))
