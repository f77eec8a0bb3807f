"""Pins for the CPU oracle: each check compares it with something other than
itself (closed forms, torch SDPA / numpy library routines on special cases,
brute force on tiny inputs, the generator's planted path, hand-derived
fixtures in tests/golden/).  CPU only."""
import itertools
import json
import os

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _bits(mask_row):
    out = set()
    for w, word in enumerate(mask_row):
        word = int(word)
        for j in range(64):
            if word >> j & 1:
                out.add(64 * w + j)
    return out


# ---------------------------------------------------------------------------
# ancestor masks
# ---------------------------------------------------------------------------
def test_mask_chain_closed_form():
    T = 130  # spans three 64-bit words
    parent, _ = W.tree_chain(T)
    mask, depth = O.tree_mask(parent[None])
    for i in range(T):
        assert _bits(mask[0, i]) == set(range(i + 1))
    assert (depth[0] == np.arange(1, T + 1)).all()


def test_mask_star_identity():
    T = 70
    parent, _ = W.tree_star(T)
    mask, depth = O.tree_mask(parent[None])
    for i in range(T):
        assert _bits(mask[0, i]) == {i}
    assert (depth == 1).all()


def test_mask_heap_binary_tree_closed_form():
    # heap numbering: node i > 0 has parent (i-1)//2; the ancestors of i are
    # ((i+1) >> s) - 1 for s = 0..bit_length(i+1)-1
    T = 127
    parent = np.array([-1] + [(i - 1) // 2 for i in range(1, T)], np.int32)
    mask, depth = O.tree_mask(parent[None])
    for i in range(T):
        n = i + 1
        expect = {(n >> s) - 1 for s in range(n.bit_length())}
        assert _bits(mask[0, i]) == expect
        assert depth[0, i] == n.bit_length()


def test_mask_golden_and_tree_len():
    g = _golden("verify_example.json")
    for case in g["cases"]:
        par = np.array(case["parent"], np.int32)[None]
        mask, depth = O.tree_mask(par)
        assert mask[0, :, 0].tolist() == case["mask"]
        assert depth[0].tolist() == case["depth"]
    par = np.array([[-1, 0, 1, 2]], np.int32)
    mask, depth = O.tree_mask(par, tree_len=np.array([2], np.int32))
    assert mask[0, :, 0].tolist() == [1, 3, 0, 0]
    assert depth[0].tolist() == [1, 2, 0, 0]


@pytest.mark.parametrize("bad", [[-1, 1], [0, -1], [-1, -2], [-1, 0, 5]])
def test_mask_rejects_bad_tree(bad):
    with pytest.raises(O.OracleError):
        O.tree_mask(np.array([bad], np.int32))


def test_mask_random_invariants():
    rng = np.random.default_rng(5)
    for T in (1, 2, 63, 64, 65, 200):
        par, level = W.tree_uniform(rng, T)
        mask, depth = O.tree_mask(par[None])
        assert (depth[0] == level).all()  # generator's own level count
        for i in range(T):
            s = _bits(mask[0, i])
            assert i in s and max(s) == i
            if par[i] >= 0:
                assert _bits(mask[0, par[i]]) < s


# ---------------------------------------------------------------------------
# tree attention: special cases that reduce to plain decode attention
# (torch SDPA in fp64 on the CPU, no mask, keys selected per query)
# ---------------------------------------------------------------------------
def _sdpa_one(q, K, V, scale):
    # q [D], K/V [n][D] -> [D]
    qt = torch.from_numpy(q)[None, None, None]
    kt = torch.from_numpy(np.ascontiguousarray(K))[None, None]
    vt = torch.from_numpy(np.ascontiguousarray(V))[None, None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
    return o[0, 0, 0].numpy()


def _spec(**kw):
    base = dict(B=1, Hq=2, Hkv=2, D=16, kv_len=20, T=6, tree="uniform", V=50,
                dtype="f32", plant=None, k=2)
    base.update(kw)
    return base


def _check_against_key_sets(w, keysets, scale=None, tol=1e-12):
    """keysets(b, i) -> list of cache rows node i of sequence b sees."""
    scale = w.scale if scale is None else scale
    out = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, scale)
    q = W.to_f64(w.q, w.dtype)
    kc = W.to_f64(w.k_cache, w.dtype)
    vc = W.to_f64(w.v_cache, w.dtype)
    G = w.Hq // w.Hkv
    for b in range(w.B):
        for i in range(w.T):
            rows = keysets(b, i)
            for h in range(w.Hq):
                g = h // G
                ref = _sdpa_one(q[b, i, h], kc[b, g, rows], vc[b, g, rows], scale)
                np.testing.assert_allclose(out[b, i, h], ref, rtol=0, atol=tol)


def test_attention_chain_is_causal_decode():
    w = W.make_workload(_spec(tree="chain", T=9, kv_len=17), seed=1)
    n = int(w.kv_len[0])
    _check_against_key_sets(w, lambda b, i: list(range(n + i + 1)))


def test_attention_single_node_is_decode():
    w = W.make_workload(_spec(tree="chain", T=1, kv_len=33, Hq=4, Hkv=4), seed=2)
    n = int(w.kv_len[0])
    _check_against_key_sets(w, lambda b, i: list(range(n + 1)))


def test_attention_star_is_independent_queries():
    w = W.make_workload(_spec(tree="star", T=7, kv_len=12), seed=3)
    n = int(w.kv_len[0])
    _check_against_key_sets(w, lambda b, i: list(range(n)) + [n + i])


def test_attention_gqa_ragged_bf16_chain():
    # 4 query heads share 2 KV heads; two sequences with different prefixes;
    # bf16 inputs widened exactly; non-default scale
    w = W.make_workload(_spec(B=2, Hq=4, Hkv=2, tree="chain", T=5,
                              kv_len=[9, 0], dtype="bf16"), seed=4)
    _check_against_key_sets(
        w, lambda b, i: list(range(int(w.kv_len[b]) + i + 1)), scale=0.37)


def test_attention_heap_tree_selected_keys():
    # binary heap tree: node i sees the prefix and its heap ancestors
    T = 15
    w = W.make_workload(_spec(tree="star", T=T, kv_len=5), seed=6)
    w.parent[0] = np.array([-1] + [(i - 1) // 2 for i in range(1, T)], np.int32)
    n = int(w.kv_len[0])

    def rows(b, i):
        m = i + 1
        return list(range(n)) + sorted(n + (m >> s) - 1 for s in range(m.bit_length()))
    _check_against_key_sets(w, rows)


def test_attention_relabel_invariance():
    # renumbering the tree in another topological order (and moving the tree
    # rows of the cache with it) permutes the outputs the same way
    w = W.make_workload(_spec(T=12, kv_len=8, Hq=4, Hkv=2), seed=7)
    par = w.parent[0]
    T = w.T
    # random topological order: repeatedly pick a random node whose parent is placed
    rng = np.random.default_rng(0)
    placed, order = set(), []
    while len(order) < T:
        ready = [i for i in range(T) if i not in placed and (par[i] < 0 or par[i] in placed)]
        c = ready[rng.integers(len(ready))]
        order.append(c)
        placed.add(c)
    new_of = {old: new for new, old in enumerate(order)}
    par2 = np.array([-1 if par[o] < 0 else new_of[int(par[o])] for o in order], np.int32)
    n = int(w.kv_len[0])
    q2 = w.q[:, order]
    k2 = w.k_cache.copy()
    v2 = w.v_cache.copy()
    k2[:, :, n:n + T] = w.k_cache[:, :, n + np.array(order)]
    v2[:, :, n:n + T] = w.v_cache[:, :, n + np.array(order)]
    o1 = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale)
    o2 = O.tree_attention(q2, k2, v2, w.kv_len, par2[None], w.scale)
    np.testing.assert_allclose(o2[0], o1[0, order], rtol=0, atol=1e-13)


def test_attention_rows_match_full():
    w = W.make_workload(_spec(B=2, kv_len=[4, 11], Hq=4, Hkv=1), seed=8)
    full = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale)
    rows = [(0, 3, 2), (1, 0, 5), (1, 2, 0)]
    part = O.attention_rows(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale, rows)
    for n, (b, h, i) in enumerate(rows):
        assert np.array_equal(part[n], full[b, i, h])


def _ancestor_rows(par, n, i):
    rows, a = [], i
    while a != -1:
        rows.append(n + a)
        a = int(par[a])
    return list(range(n)) + sorted(rows)


def test_attention_tree_len_live_rows_are_decode_and_padding_is_ignored():
    # a padded batch of trees of sizes 10, 4, 0 and 7: every live node sees its
    # prefix and ancestors (plain SDPA over that key set), padding rows are zero,
    # and garbage in the padding (parents, queries, cache rows) changes nothing
    T = 10
    w = W.make_workload(_spec(B=4, Hq=4, Hkv=2, T=T, kv_len=[5, 0, 12, 3]), seed=9)
    tl = np.array([10, 4, 0, 7], np.int32)
    q = w.q.copy()
    kc, vc = w.k_cache.copy(), w.v_cache.copy()
    par = w.parent.copy()
    for b in range(w.B):
        n = int(w.kv_len[b])
        q[b, tl[b]:] = 1e6
        kc[b, :, n + tl[b]:] = -1e6
        vc[b, :, n + tl[b]:] = 1e6
        par[b, tl[b]:] = [99, -7, 3][b % 3] if tl[b] < T else par[b, tl[b]:]
    out = O.tree_attention(q, kc, vc, w.kv_len, par, w.scale, tree_len=tl)
    clean = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale)
    qf, kf, vf = (W.to_f64(x, w.dtype) for x in (w.q, w.k_cache, w.v_cache))
    G = w.Hq // w.Hkv
    for b in range(w.B):
        n = int(w.kv_len[b])
        assert np.all(out[b, tl[b]:] == 0.0)
        for i in range(tl[b]):
            rows = _ancestor_rows(w.parent[b], n, i)
            for h in range(w.Hq):
                ref = _sdpa_one(qf[b, i, h], kf[b, h // G, rows], vf[b, h // G, rows], w.scale)
                np.testing.assert_allclose(out[b, i, h], ref, rtol=0, atol=1e-12)
            # a live node's result does not depend on the tree's size
            assert np.array_equal(out[b, i], clean[b, i])


def test_attention_tree_len_full_is_no_tree_len_and_cache_may_end_at_the_tree():
    w = W.make_workload(_spec(B=2, T=8, kv_len=[6, 2]), seed=10)
    full = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale)
    same = O.tree_attention(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale,
                            tree_len=np.array([8, 8], np.int32))
    assert np.array_equal(full, same)
    # sizes 3 and 5: the cache needs only kv_len + tree_len rows
    tl = np.array([3, 5], np.int32)
    L = int((w.kv_len + tl).max())
    out = O.tree_attention(w.q, w.k_cache[:, :, :L], w.v_cache[:, :, :L], w.kv_len, w.parent,
                           w.scale, tree_len=tl)
    for b in range(2):
        assert np.array_equal(out[b, :tl[b]], full[b, :tl[b]])
    with pytest.raises(RuntimeError):
        O.tree_attention(w.q, w.k_cache[:, :, :L], w.v_cache[:, :, :L], w.kv_len, w.parent,
                         w.scale)


# ---------------------------------------------------------------------------
# 8-bit (OCP E4M3) key/value caches
# ---------------------------------------------------------------------------
def test_e4m3_decode_matches_torch_float8_e4m3fn():
    codes = np.arange(256, dtype=np.uint8)
    got = O.e4m3_decode(codes)
    ref = torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).double().numpy()
    assert np.array_equal(np.isnan(got), np.isnan(ref)) and np.isnan(got).sum() == 2
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])
    assert np.array_equal(np.signbit(got[ok]), np.signbit(ref[ok]))


def test_e4m3_decode_closed_forms():
    pairs = {0x38: 1.0, 0x40: 2.0, 0x30: 0.5, 0x3C: 1.5, 0x7E: 448.0, 0xFE: -448.0,
             0x78: 256.0, 0x08: 2.0 ** -6, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9,
             0x00: 0.0, 0xB8: -1.0}
    got = O.e4m3_decode(np.array(list(pairs), np.uint8))
    assert got.tolist() == list(pairs.values())
    z = O.e4m3_decode(np.array([0x80], np.uint8))[0]
    assert z == 0.0 and np.signbit(z)
    assert np.isnan(O.e4m3_decode(np.array([0x7F, 0xFF], np.uint8))).all()


def _e4m3_codes(rng, shape):
    # random finite codes (no NaN)
    c = rng.integers(0, 256, shape).astype(np.uint8)
    c[(c & 0x7F) == 0x7F] = 0x3F
    return c


def test_e4m3_input_encoder_rounds_like_torch():
    # the seeded generator's quantizer (input side, not the oracle)
    rng = np.random.default_rng(12)
    x = (rng.standard_normal(50000) * np.exp(rng.uniform(-12, 7, 50000))).astype(np.float32)
    x = np.clip(x, -448, 448)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(W.f32_to_e4m3_bits(x), ref)


def test_fp8kv_attention_is_the_attention_of_the_decoded_caches():
    # every E4M3 value is a bf16 value: with unit scales the fp8 path equals
    # the bf16 oracle on caches holding the same values
    rng = np.random.default_rng(11)
    w = W.make_workload(_spec(B=2, Hq=4, Hkv=2, T=7, kv_len=[9, 3], dtype="bf16"), seed=11)
    kq = _e4m3_codes(rng, w.k_cache.shape)
    vq = _e4m3_codes(rng, w.v_cache.shape)
    one = np.ones(w.Hkv, np.float32)
    out8 = O.tree_attention_fp8kv(w.q, kq, vq, one, one, w.kv_len, w.parent, w.scale)
    as_bf16 = lambda c: W.f32_to_bf16_bits(O.e4m3_decode(c).astype(np.float32))
    ref = O.tree_attention(w.q, as_bf16(kq), as_bf16(vq), w.kv_len, w.parent, w.scale)
    assert np.array_equal(out8, ref)
    # a key scale multiplies every score (= a larger softmax scale); a value
    # scale multiplies the output
    ks = np.array([2.0, 0.25], np.float32)
    vs = np.array([0.5, 3.0], np.float32)
    out_s = O.tree_attention_fp8kv(w.q, kq, vq, ks, vs, w.kv_len, w.parent, w.scale)
    G = w.Hq // w.Hkv
    for g in range(w.Hkv):
        ref_g = O.tree_attention(w.q, as_bf16(kq), as_bf16(vq), w.kv_len, w.parent,
                                 w.scale * float(ks[g]))
        np.testing.assert_allclose(out_s[:, :, g * G:(g + 1) * G],
                                   float(vs[g]) * ref_g[:, :, g * G:(g + 1) * G],
                                   rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------------------
# top-k / argmax
# ---------------------------------------------------------------------------
def test_topk_golden_ties():
    g = _golden("topk_ties.json")
    rows = np.array(g["rows"], np.float32)
    am, idx, val = O.topk(rows, g["k"])
    assert am.tolist() == g["argmax"]
    assert idx.tolist() == g["topk_idx"]
    assert np.array_equal(val, np.array(g["topk_val"]))
    assert np.signbit(val[0, 4])  # the row's own -0.0 is returned


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_topk_matches_lexsort_and_argmax(dtype):
    rng = np.random.default_rng(11)
    R, V, k = 9, 3001, 16
    x = rng.standard_normal((R, V), dtype=np.float32) * np.float32(1.4)
    x[:, rng.integers(0, V, 40)] = np.float32(0.0)  # ties, incl. signed zeros
    x[2, 100:140] = np.float32(-0.0)
    x[4, :] = np.float32(1.0)
    arr = W.f32_to_bf16_bits(x) if dtype == "bf16" else x
    am, idx, val = O.topk(arr, k)
    xv = W.to_f64(arr, dtype)
    for r in range(R):
        order = np.lexsort((np.arange(V), -xv[r]))
        assert idx[r].tolist() == order[:k].tolist()
        assert am[r] == np.argmax(xv[r])
        assert np.array_equal(val[r], xv[r, order[:k]])


# ---------------------------------------------------------------------------
# verification
# ---------------------------------------------------------------------------
def _brute_accept(parent, tokens, argmax):
    """Enumerate every root-to-leaf path; along each path count the eligible
    prefix; the answer is the longest, lowest terminal index on ties."""
    T = len(parent)
    children = {p: [c for c in range(T) if parent[c] == p] for p in range(-1, T)}
    best = (0, None)
    paths = []

    def walk(node, path):
        kids = children[node]
        if not kids:
            paths.append(path)
        for c in kids:
            walk(c, path + [c])
    walk(-1, [])
    for path in paths:
        depth, prev = 0, -1
        for c in path:
            if tokens[c] != argmax[prev + 1]:
                break
            depth += 1
            prev = c
        if depth == 0:
            continue
        term = path[depth - 1]
        if depth > best[0] or (depth == best[0] and term < best[1]):
            best = (depth, term)
    return best


def test_verify_golden():
    g = _golden("verify_example.json")
    for c in g["cases"]:
        par = np.array([c["parent"]], np.int32)
        tok = np.array([c["tokens"]], np.int32)
        am = np.array([c["argmax"]], np.int32)
        al, an, ot = O.verify(am, tok, par)
        assert al[0] == c["accept_len"]
        assert an[0].tolist() == c["accept_nodes"]
        assert ot[0].tolist() == c["out_tokens"]


def test_verify_brute_force_small_trees():
    rng = np.random.default_rng(21)
    for trial in range(400):
        T = int(rng.integers(1, 9))
        par, _ = W.tree_uniform(rng, T)
        V = 3  # tiny vocabulary: many eligible edges and duplicate siblings
        tok = rng.integers(0, V, T).astype(np.int32)
        am = rng.integers(0, V, T + 1).astype(np.int32)
        al, an, ot = O.verify(am[None], tok[None], par[None])
        depth, term = _brute_accept(par, tok, am)
        assert al[0] == depth, trial
        if depth:
            path = []
            a = term
            while a != -1:
                path.append(a)
                a = par[a]
            assert an[0, :depth].tolist() == path[::-1]
            assert ot[0, depth] == am[term + 1]
        else:
            assert ot[0, 0] == am[0]


@pytest.mark.parametrize("name", ["tiny", "llama2-7b", "llama2-13b"])
def test_verify_planted_paths(name):
    w = W.make_workload(name, kv=False)
    am, idx, _ = O.topk(w.logits, w.k)
    al, an, ot = O.verify(am.reshape(w.B, -1), w.tokens, w.parent)
    for b in range(w.B):
        d = int(w.planted_depth[b])
        assert al[b] == d
        assert an[b, :d].tolist() == w.planted_path[b]
        assert ot[b, d] == w.planted_bonus[b]


def test_verify_ragged_planted():
    spec = dict(W.CONFIGS["ragged-16"], V=5000, kv_len=4)
    w = W.make_workload(spec, kv=False)
    am, _, _ = O.topk(w.logits, 1)
    al, an, _ = O.verify(am.reshape(w.B, -1), w.tokens, w.parent)
    assert al.tolist() == w.planted_depth.tolist()


def test_verify_tree_len_ignores_tail():
    par = np.array([[-1, 0, 1, 2]], np.int32)
    tok = np.array([[1, 2, 3, 4]], np.int32)
    am = np.array([[1, 2, 3, 4, 9]], np.int32)
    al, _, ot = O.verify(am, tok, par)
    assert al[0] == 4 and ot[0, 4] == 9
    al, an, ot = O.verify(am, tok, par, tree_len=np.array([2], np.int32))
    assert al[0] == 2 and an[0].tolist() == [0, 1, -1, -1] and ot[0, 2] == 3


# ---------------------------------------------------------------------------
# expansion
# ---------------------------------------------------------------------------
def test_expand_golden():
    g = _golden("expand_example.json")
    par = np.array([g["parent"]], np.int32)
    tok = np.array([g["tokens"]], np.int32)
    ti = np.array([g["topk_idx"]], np.int32)
    for c in g["cases"]:
        pn, tn, ln = O.expand(par, tok, ti, g["width_sched"], c["d_max"], c["T_max"])
        assert pn[0].tolist() == c["parent_next"]
        assert tn[0].tolist() == c["tokens_next"]
        assert ln[0] == c["tree_len_next"]


def _token_paths(parent, tokens, n):
    paths = set()
    for i in range(n):
        p, a = [], i
        while a != -1:
            p.append(int(tokens[a]))
            a = int(parent[a])
        paths.add(tuple(p[::-1]))
    return paths


def test_expand_top1_unbounded_is_progressive_expansion():
    # k=1 with no width or depth limit: every node v gains exactly the child
    # d_v (its top-1 token) -- V^t = V^{t-1} u {d_v} -- unless a child with
    # that token exists already; compared as sets of root-to-node token paths
    rng = np.random.default_rng(31)
    for trial in range(200):
        T = int(rng.integers(1, 12))
        par, _ = W.tree_uniform(rng, T)
        tok = W.sibling_distinct_tokens(rng, par, 6)
        d_v = rng.integers(0, 6, T + 1).astype(np.int32)
        ti = d_v[:, None][None]
        pn, tn, ln = O.expand(par[None], tok[None], ti, [1000] * 64, 64, 4 * T)
        n = int(ln[0])
        old = _token_paths(par, tok, T)
        grown = set(old)
        for v in range(T):
            pv, a = [], v
            while a != -1:
                pv.append(int(tok[a]))
                a = int(par[a])
            grown.add(tuple(pv[::-1]) + (int(d_v[v + 1]),))
        assert _token_paths(pn[0], tn[0], n) == grown, trial
        assert n == len(grown)  # merged-by-value: one node per token path


def test_expand_bfs_order_caps_and_truncation():
    rng = np.random.default_rng(41)
    for trial in range(200):
        T = int(rng.integers(1, 14))
        par, lev = W.tree_uniform(rng, T)
        tok = W.sibling_distinct_tokens(rng, par, 9)
        k = int(rng.integers(1, 5))
        ti = rng.integers(0, 9, (1, T + 1, k)).astype(np.int32)
        d_max = int(rng.integers(1, 6))
        width = rng.integers(1, 4, d_max).astype(np.int32)
        pn, tn, ln = O.expand(par[None], tok[None], ti, width, d_max, 10 * T)
        n = int(ln[0])
        p, t = pn[0, :n], tn[0, :n]
        assert (pn[0, n:] == -1).all() and (tn[0, n:] == -1).all()
        # parents precede children; parents are non-decreasing (breadth-first)
        assert all(p[i] < i for i in range(n))
        assert (np.diff(p) >= 0).all()
        depth = np.zeros(n, int)
        for i in range(n):
            depth[i] = 1 if p[i] < 0 else depth[p[i]] + 1
        assert (np.diff(depth) >= 0).all()
        old = _token_paths(par, tok, T)
        assert old <= _token_paths(p, t, n)
        for i in range(n):  # depth and width caps hold wherever a node grew
            kids = [c for c in range(n) if p[c] == i]
            added = [c for c in kids if tuple(_path_tokens(p, t, c)) not in old]
            if added:
                assert depth[i] + 1 <= d_max
                assert len(kids) <= width[depth[i]]
        # truncation keeps a breadth-first prefix
        for T_max in (1, max(1, n // 2), n):
            pn2, tn2, ln2 = O.expand(par[None], tok[None], ti, width, d_max, T_max)
            assert ln2[0] == min(n, T_max)
            assert pn2[0].tolist() == pn[0, :T_max].tolist()
            assert tn2[0].tolist() == tn[0, :T_max].tolist()


def _path_tokens(parent, tokens, i):
    out, a = [], i
    while a != -1:
        out.append(int(tokens[a]))
        a = int(parent[a])
    return out[::-1]


# ---------------------------------------------------------------------------
# generator invariants
# ---------------------------------------------------------------------------
def test_generator_shapes_and_bfs_truncation():
    for name, levels in [("llama2-7b", [4, 12, 24, 24]), ("llama2-13b", [5, 20, 60, 11])]:
        w = W.make_workload(name, kv=False, logits=False)
        _, depth = O.tree_mask(w.parent)
        counts = np.bincount(depth[0])[1:]
        assert counts.tolist() == levels
    w = W.make_workload("tiny")
    assert w.q.dtype == np.float32 and w.k_cache.shape == (1, 2, 144, 64)
    w = W.make_workload(dict(W.CONFIGS["ragged-16"], V=64), logits=True)
    assert w.kv_len.min() >= 512 and w.kv_len.max() <= 8192
    assert w.k_cache.dtype == np.uint16


def test_bf16_rounding_is_rne():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.0e-3], np.float32)
    b = W.f32_to_bf16_bits(x)
    back = W.bf16_bits_to_f32(b)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: rounds to even (1.0);
    # 1 + 3*2^-8 is a tie between 1+2^-7 and 1+2^-6: rounds to even (1+2^-6)
    assert back.tolist()[:4] == [1.0, 1.0, 1.015625, -2.5]
    assert abs(back[4] - 3.0e-3) <= 3.0e-3 * 2 ** -8
    assert np.array_equal(W.f32_to_bf16_bits(
        torch.from_numpy(x).to(torch.bfloat16).float().numpy()), b)


# ---------------------------------------------------------------------------
# positions and rotary embedding of the tree rows
# ---------------------------------------------------------------------------
def _rope_inputs(rng, B, T, Hq, Hkv, D, L_cap):
    q = rng.standard_normal((B, T, Hq, D)).astype(np.float32)
    k = rng.standard_normal((B, Hkv, L_cap, D)).astype(np.float32)
    return q, k


def test_rope_inv_freq_closed_form():
    # RoFormer: theta_p = base^(-2p/D)
    assert np.array_equal(O.rope_inv_freq(4, 10000.0), [1.0, 0.01])
    assert np.allclose(O.rope_inv_freq(8, 256.0), [1.0, 0.25, 1 / 16, 1 / 64], rtol=0, atol=1e-15)


def test_rope_positions_closed_forms():
    rng = np.random.default_rng(11)
    T = 15
    chain, _ = W.tree_chain(T)
    star, _ = W.tree_star(T)
    heap = np.array([-1] + [(i - 1) // 2 for i in range(1, T)], np.int32)
    parent = np.stack([chain, star, heap])
    kv_len = np.array([0, 7, 40], np.int32)
    q, k = _rope_inputs(rng, 3, T, 1, 1, 4, 64)
    _, _, pos = O.tree_rope(q, k, kv_len, parent)
    i = np.arange(T)
    assert (pos[0] == kv_len[0] + i).all()                            # chain: depth i + 1
    assert (pos[1] == kv_len[1]).all()                                # star: every node a root
    assert (pos[2] == kv_len[2] + np.floor(np.log2(i + 1))).all()     # heap: depth bit_length(i+1)


def test_rope_position_zero_is_identity():
    rng = np.random.default_rng(12)
    T, D = 6, 16
    star, _ = W.tree_star(T)
    q, k = _rope_inputs(rng, 1, T, 3, 2, D, T)
    for pairing in (0, 1):
        qo, ko, pos = O.tree_rope(q, k, np.array([0], np.int32), star[None], pairing=pairing)
        assert (pos == 0).all()
        assert np.array_equal(qo, q.astype(np.float64))
        assert np.array_equal(ko, k[:, :, :T].astype(np.float64))


def test_rope_turns_e1_counterclockwise():
    # D = 2, one pair with frequency 1: e1 at position a becomes (cos a, sin a),
    # e2 becomes (-sin a, cos a) (the textbook plane rotation by a).
    T = 4
    chain, _ = W.tree_chain(T)
    q = np.zeros((1, T, 2, 2), np.float32)
    q[0, :, 0] = [1.0, 0.0]
    q[0, :, 1] = [0.0, 1.0]
    k = np.zeros((1, 1, T + 1, 2), np.float32)
    qo, _, pos = O.tree_rope(q, k, np.array([1], np.int32), chain[None],
                             inv_freq=np.array([1.0]))
    for i in range(T):
        a = float(pos[0, i])
        assert a == 1 + i
        assert np.allclose(qo[0, i, 0], [np.cos(a), np.sin(a)], rtol=0, atol=1e-15)
        assert np.allclose(qo[0, i, 1], [-np.sin(a), np.cos(a)], rtol=0, atol=1e-15)


def test_rope_preserves_pair_norms():
    rng = np.random.default_rng(13)
    B, T, Hq, Hkv, D, L = 2, 9, 2, 1, 32, 40
    parent = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    q, k = _rope_inputs(rng, B, T, Hq, Hkv, D, L)
    kv_len = np.array([3, 31], np.int32)
    for pairing in (0, 1):
        qo, ko, _ = O.tree_rope(q, k, kv_len, parent, theta=500000.0, pairing=pairing)
        p = np.arange(D // 2)
        a, b2 = (p, p + D // 2) if pairing == 0 else (2 * p, 2 * p + 1)
        n_in = q[..., a].astype(np.float64) ** 2 + q[..., b2].astype(np.float64) ** 2
        n_out = qo[..., a] ** 2 + qo[..., b2] ** 2
        assert np.allclose(n_out, n_in, rtol=1e-12, atol=0)
        kin = np.stack([k[b, :, kv_len[b]:kv_len[b] + T] for b in range(B)]).astype(np.float64)
        assert np.allclose(ko[..., a] ** 2 + ko[..., b2] ** 2, kin[..., a] ** 2 + kin[..., b2] ** 2,
                           rtol=1e-12, atol=0)


def test_rope_scores_depend_on_relative_position_only():
    # the same query and key vectors at every node of a chain: the rotated
    # score of node i against node j is a function of i - j alone
    rng = np.random.default_rng(14)
    T, D, kv = 10, 16, 5
    chain, _ = W.tree_chain(T)
    q0 = rng.standard_normal(D).astype(np.float32)
    k0 = rng.standard_normal(D).astype(np.float32)
    q = np.broadcast_to(q0, (1, T, 1, D)).copy()
    k = np.zeros((1, 1, kv + T, D), np.float32)
    k[0, 0, kv:] = k0
    for pairing in (0, 1):
        qo, ko, _ = O.tree_rope(q, k, np.array([kv], np.int32), chain[None], theta=100.0,
                                pairing=pairing)
        s = qo[0, :, 0] @ ko[0, 0].T               # [i][j]
        for d in range(-T + 1, T):
            diag = np.diagonal(s, offset=-d)       # entries with i - j = d
            assert np.allclose(diag, diag[0], rtol=0, atol=1e-12)
        assert np.ptp([np.diagonal(s, -d)[0] for d in range(T)]) > 1e-3


def test_rope_interleaved_is_half_on_permuted_dims():
    rng = np.random.default_rng(15)
    B, T, Hq, Hkv, D, L = 1, 7, 2, 2, 16, 20
    parent = W.tree_uniform(rng, T)[0][None]
    q, k = _rope_inputs(rng, B, T, Hq, Hkv, D, L)
    perm = np.concatenate([np.arange(0, D, 2), np.arange(1, D, 2)])   # half slot -> x index
    kv_len = np.array([9], np.int32)
    qi, ki, _ = O.tree_rope(q, k, kv_len, parent, pairing=1)
    qh, kh, _ = O.tree_rope(q[..., perm], k[..., perm], kv_len, parent, pairing=0)
    inv = np.argsort(perm)
    assert np.allclose(qi, qh[..., inv], rtol=0, atol=1e-14)
    assert np.allclose(ki, kh[..., inv], rtol=0, atol=1e-14)


def test_rope_rejects_bad_tree_and_kv_len():
    rng = np.random.default_rng(16)
    q, k = _rope_inputs(rng, 1, 4, 1, 1, 4, 8)
    with pytest.raises(O.OracleError):
        O.tree_rope(q, k, np.array([0], np.int32), np.array([[-1, 0, 2, 1]], np.int32))
    with pytest.raises(O.OracleError):
        O.tree_rope(q, k, np.array([5], np.int32), np.array([[-1, 0, 1, 2]], np.int32))


# ---------------------------------------------------------------------------
# commit of the accepted path
# ---------------------------------------------------------------------------
def test_kv_commit_golden():
    g = _golden("kv_commit_example.json")
    L = g["L_cap"]
    r = np.arange(L, dtype=np.float32)
    k = np.stack([10 * r, 10 * r + 1], -1)[None, None]
    v = np.stack([-10 * r, -10 * r - 1], -1)[None, None]
    kn, vn, nxt = O.kv_commit(k, v, np.array(g["kv_len"], np.int32),
                              np.array(g["accept_len"], np.int32),
                              np.array(g["accept_nodes"], np.int32))
    assert np.array_equal(kn[0, 0], np.array(g["k_after_rows"], np.float32))
    assert np.array_equal(vn[0, 0], np.array(g["v_after_rows"], np.float32))
    assert nxt.tolist() == g["kv_len_next"]


def test_kv_commit_chain_prefix_and_empty_are_identity():
    rng = np.random.default_rng(17)
    B, Hkv, L, D, T = 2, 3, 30, 8, 6
    k = W.f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D)).astype(np.float32))
    v = W.f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D)).astype(np.float32))
    nodes = np.full((B, T), -1, np.int32)
    nodes[0, :4] = np.arange(4)                 # the first four nodes of a chain
    kn, vn, nxt = O.kv_commit(k, v, np.array([5, 9], np.int32), np.array([4, 0], np.int32),
                              nodes)
    assert np.array_equal(kn, k) and np.array_equal(vn, v)
    assert nxt.tolist() == [9, 9]


def test_rope_then_commit_matches_rope_at_committed_rows():
    # Rotating the tree keys at kv_len + |pi(i)| - 1 and committing the
    # accepted path leaves committed row kv_len + j - 1 rotated at exactly that
    # row's position, as if the path had been decoded one token at a time.
    rng = np.random.default_rng(18)
    B, T, Hkv, D, L = 3, 24, 2, 8, 64
    parent = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    kv_len = np.array([0, 11, 30], np.int32)
    k = rng.standard_normal((B, Hkv, L, D)).astype(np.float32)
    q = np.zeros((B, T, 1, D), np.float32)
    _, ko, _ = O.tree_rope(q, k, kv_len, parent, theta=1000.0)
    k_rot = k.copy()
    for b in range(B):
        k_rot[b, :, kv_len[b]:kv_len[b] + T] = ko[b].astype(np.float32)
    # an accepted path: the root path of the deepest node (lowest index on ties)
    _, depth = O.tree_mask(parent)
    al = np.zeros(B, np.int32)
    an = np.full((B, T), -1, np.int32)
    for b in range(B):
        t = int(np.argmax(depth[b]))
        path = []
        while t >= 0:
            path.append(t)
            t = int(parent[b, t])
        path = path[::-1]
        al[b] = len(path)
        an[b, :len(path)] = path
    kn, _, nxt = O.kv_commit(k_rot, k_rot, kv_len, al, an)
    assert (nxt == kv_len + al).all()
    for b in range(B):
        n = int(al[b])
        src = k[b][:, kv_len[b] + an[b, :n]]                      # un-rotated keys of the path
        chain, _ = W.tree_chain(n)
        kk = np.zeros((1, Hkv, kv_len[b] + n, D), np.float32)
        kk[0, :, kv_len[b]:] = src
        _, want, pos = O.tree_rope(np.zeros((1, n, 1, D), np.float32), kk, kv_len[b:b + 1],
                                   chain[None], theta=1000.0)
        assert (pos[0] == kv_len[b] + np.arange(n)).all()
        assert np.allclose(kn[b, :, kv_len[b]:kv_len[b] + n], want[0], rtol=0, atol=1e-6)


@pytest.mark.parametrize("al,nodes,kv", [
    ([2], [[3, 1, -1, -1]], [0]),    # not increasing
    ([2], [[1, 4, -1, -1]], [0]),    # node id >= T
    ([5], [[0, 1, 2, 3]], [0]),      # longer than the tree
    ([-1], [[0, 1, 2, 3]], [0]),     # negative length
    ([1], [[0, 1, 2, 3]], [5]),      # kv_len + T > L_cap
])
def test_kv_commit_rejects_bad_paths(al, nodes, kv):
    k = np.zeros((1, 1, 8, 2), np.float32)
    with pytest.raises(O.OracleError):
        O.kv_commit(k, k, np.array(kv, np.int32), np.array(al, np.int32),
                    np.array(nodes, np.int32))


# ---------------------------------------------------------------------------
# sampling verification (App. E / App. F)
# ---------------------------------------------------------------------------
def _chi2_ok(counts, probs, n):
    """Pearson chi-square of observed counts against n * probs; accepts at a
    p-value above 1e-6 (fixed seeds: the outcome is deterministic)."""
    from scipy.stats import chi2
    exp_ = n * np.asarray(probs, np.float64)
    keep = exp_ > 0
    assert (np.asarray(counts)[~keep] == 0).all()
    stat = float((((np.asarray(counts) - exp_) ** 2)[keep] / exp_[keep]).sum())
    return chi2.sf(stat, keep.sum() - 1) > 1e-6


def _replicate(parent, tokens, rows, n):
    B = n
    T = len(parent)
    par = np.broadcast_to(np.asarray(parent, np.int32), (B, T)).copy()
    tok = np.broadcast_to(np.asarray(tokens, np.int32), (B, T)).copy()
    lg = np.broadcast_to(np.asarray(rows, np.float32), (B, T + 1, len(rows[0]))).copy()
    return par, tok, lg


def test_sample_first_token_follows_the_model_distribution():
    # App. F: every candidate is selected with its own probability, and the
    # fallback draw covers the rest, so the first emitted token ~ P_root.
    # Logits are logs of chosen probabilities (temperature 1).
    P0 = np.array([0.30, 0.25, 0.20, 0.10, 0.10, 0.05])
    n = 200_000
    rng = np.random.default_rng(21)
    rows = [np.log(P0)] + [np.log(np.full(6, 1 / 6))] * 3
    # three root children with tokens 1, 4, 2 (one likely, one unlikely, one middling)
    par, tok, lg = _replicate([-1, -1, -1], [1, 4, 2], rows, n)
    al, an, ot, _ = O.verify_sample(lg, tok, par, 1.0, rng.random((n, 3)), rng.random((n, 4)))
    first = ot[:, 0]
    assert (first >= 0).all()
    assert _chi2_ok(np.bincount(first, minlength=6), P0, n)
    # which child was accepted: child i with probability P0[token_i]
    acc = np.where(al > 0, an[:, 0], 3)
    assert _chi2_ok(np.bincount(acc, minlength=4), [P0[1], P0[4], P0[2], 1 - P0[[1, 4, 2]].sum()], n)


def test_sample_second_token_follows_the_childs_distribution():
    # after accepting root child A (token 0), the next emitted token ~ P_A
    P0 = np.array([0.4, 0.3, 0.2, 0.1])
    PA = np.array([0.1, 0.2, 0.3, 0.4])
    n = 200_000
    rng = np.random.default_rng(22)
    uniform = np.log(np.full(4, 0.25))
    # nodes: 0 = A (token 0, root child), 1 = B (token 1, root child),
    #        2 = C (token 2, child of A), 3 = D (token 3, child of A)
    rows = [np.log(P0), np.log(PA), uniform, uniform, uniform]
    par, tok, lg = _replicate([-1, -1, 0, 0], [0, 1, 2, 3], rows, n)
    al, an, ot, _ = O.verify_sample(lg, tok, par, 1.0, rng.random((n, 4)), rng.random((n, 5)))
    via_a = (al >= 1) & (an[:, 0] == 0)
    m = int(via_a.sum())
    assert abs(m / n - P0[0]) < 5 * np.sqrt(P0[0] * (1 - P0[0]) / n)
    assert _chi2_ok(np.bincount(ot[via_a, 1], minlength=4), PA, m)


def test_sample_duplicate_sibling_never_accepted():
    P0 = np.array([0.5, 0.3, 0.2])
    n = 50_000
    rng = np.random.default_rng(23)
    rows = [np.log(P0)] + [np.log(np.full(3, 1 / 3))] * 2
    par, tok, lg = _replicate([-1, -1], [1, 1], rows, n)
    al, an, ot, _ = O.verify_sample(lg, tok, par, 1.0, rng.random((n, 2)), rng.random((n, 3)))
    assert not ((al > 0) & (an[:, 0] == 1)).any()
    assert _chi2_ok(np.bincount(ot[:, 0], minlength=3), P0, n)


def test_sample_temperature_scales_logits():
    # softmax(l / t) with l = t * log(P): the model distribution is P again
    P0 = np.array([0.5, 0.25, 0.125, 0.125])
    n = 100_000
    rng = np.random.default_rng(24)
    t = 0.37
    rows = [t * np.log(P0), t * np.log(np.full(4, 0.25))]
    par, tok, lg = _replicate([-1], [2], rows, n)
    al, an, ot, _ = O.verify_sample(lg, tok, par, t, rng.random((n, 1)), rng.random((n, 2)))
    assert _chi2_ok(np.bincount(ot[:, 0], minlength=4), P0, n)


def test_sample_low_temperature_is_greedy():
    # as the temperature goes to 0 the model distribution becomes the argmax:
    # sampling verification reduces to greedy verification (pinned above)
    rng = np.random.default_rng(25)
    B, T, V = 8, 30, 50
    par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    # distinct integer logits: gaps >= 1, so at temperature 1e-3 every
    # probability but the argmax's is below exp(-1000)
    lg = np.stack([rng.permutation(V) for _ in range(B * (T + 1))]).astype(np.float32)
    lg = lg.reshape(B, T + 1, V)
    am, _, _ = O.topk(lg.reshape(-1, V), 1)
    am = am.reshape(B, T + 1)
    # tokens: half the children follow the argmax of their parent's row
    tok = rng.integers(0, V, (B, T)).astype(np.int32)
    for b in range(B):
        for i in range(T):
            if rng.random() < 0.6:
                tok[b, i] = am[b, par[b, i] + 1]
    g_al, g_an, g_ot = O.verify(am, tok, par)
    u1 = rng.uniform(0.01, 0.99, (B, T))
    u2 = rng.uniform(0.01, 0.99, (B, T + 1))
    al, an, ot, _ = O.verify_sample(lg, tok, par, 1e-3, u1, u2)
    # greedy takes the deepest accepted path; the sampling walk stops at the
    # first accepted child, which is the only child carrying the argmax token
    # unless siblings repeat it (then the earliest one is taken).
    for b in range(B):
        k = int(al[b])
        path = an[b, :k]
        # every step of the sampled path is an argmax match
        prev = -1
        for c in path:
            assert par[b, c] == prev and tok[b, c] == am[b, prev + 1]
            prev = c
        # the walk stopped where no child carries the argmax
        kids = [c for c in range(T) if par[b, c] == prev]
        assert all(tok[b, c] != am[b, prev + 1] for c in kids)
        assert ot[b, k] == am[b, prev + 1]
        assert k <= g_al[b]
    # with distinct tokens among siblings the two agree exactly
    par2 = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    tok2 = np.stack([W.sibling_distinct_tokens(rng, par2[b], V) for b in range(B)])
    for b in range(B):
        for i in range(T):
            if rng.random() < 0.7:
                p = par2[b, i]
                sib = [c for c in range(T) if par2[b, c] == p]
                if all(tok2[b, c] != am[b, p + 1] for c in sib):
                    tok2[b, i] = am[b, p + 1]
    g_al, g_an, g_ot = O.verify(am, tok2, par2)
    al, an, ot, _ = O.verify_sample(lg, tok2, par2, 1e-3, u1, u2)
    assert np.array_equal(al, g_al) and np.array_equal(an, g_an) and np.array_equal(ot, g_ot)


def test_sample_empty_tree_draws_from_the_root_row():
    P0 = np.array([0.2, 0.2, 0.6])
    n = 60_000
    rng = np.random.default_rng(26)
    rows = [np.log(P0), np.log(P0)]
    par, tok, lg = _replicate([-1], [0], rows, n)
    al, an, ot, _ = O.verify_sample(lg, tok, par, 1.0, rng.random((n, 1)), rng.random((n, 2)),
                                    tree_len=np.zeros(n, np.int32))
    assert (al == 0).all() and (an == -1).all()
    assert _chi2_ok(np.bincount(ot[:, 0], minlength=3), P0, n)


# ---------------------------------------------------------------------------
# stepping (depth control) and the candidate pool
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("L,d_max", [(1, 1), (5, 1), (8, 3), (8, 8), (20, 6)])
def test_step_prune_chain_is_a_sliding_window(L, d_max):
    par, _ = W.tree_chain(L)
    tok = (np.arange(L) * 7 + 3).astype(np.int32)
    pn, tn, ln = O.step_prune(par[None], tok[None], d_max, L)
    keep = min(L, d_max)
    assert ln[0] == keep
    assert tn[0, :keep].tolist() == tok[L - keep:].tolist()
    assert pn[0, :keep].tolist() == [-1] + list(range(keep - 1))
    assert (pn[0, keep:] == -1).all() and (tn[0, keep:] == -1).all()


def test_step_prune_heap_tree_closed_form():
    # heap numbering, 5 levels: the root steps to node 1 (depth 4 > 3), then
    # to node 3 (depth 3); node 3's sub-tree is {3, 7, 8, 15, 16, 17, 18}
    T = 31
    par = np.array([-1] + [(i - 1) // 2 for i in range(1, T)], np.int32)
    pn, tn, ln = O.step_prune(par[None], np.arange(T, dtype=np.int32)[None], 3, T)
    assert ln[0] == 7
    assert tn[0, :7].tolist() == [3, 7, 8, 15, 16, 17, 18]
    assert pn[0, :7].tolist() == [-1, 0, 0, 1, 1, 2, 2]


def test_step_prune_shallow_bfs_forest_is_unchanged():
    par, _ = W.tree_branching([3, 2, 2], 20)
    tok = np.arange(20, dtype=np.int32) + 100
    pn, tn, ln = O.step_prune(par[None], tok[None], 3, 20)
    assert ln[0] == 20 and np.array_equal(pn[0], par) and np.array_equal(tn[0], tok)


@pytest.mark.parametrize("d_max", [1, 2, 3, 5])
def test_step_prune_invariants(d_max):
    rng = np.random.default_rng(30 + d_max)
    B, T = 6, 40
    par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    tok = np.broadcast_to(np.arange(T, dtype=np.int32), (B, T)).copy()   # token = old id
    pn, tn, ln = O.step_prune(par, tok, d_max, T)
    _, depth = O.tree_mask(pn, ln)
    for b in range(B):
        n = int(ln[b])
        assert depth[b, :n].max() <= d_max
        kids = {v: [c for c in range(T) if par[b, c] == v] for v in range(T)}
        roots_in = [r for r in range(T) if par[b, r] == -1]
        roots_out = [int(tn[b, i]) for i in range(n) if pn[b, i] == -1]
        # one new root per old sub-tree, in the old roots' order, each on the
        # old root's chain of lowest-index children
        assert len(roots_out) == len(roots_in)
        for r, x in zip(roots_in, roots_out):
            chain = [r]
            while kids[chain[-1]]:
                chain.append(kids[chain[-1]][0])
            assert x in chain
        for i in range(n):
            # an output node's root path is the tail of its old root path
            path_out = []
            j = i
            while j >= 0:
                path_out.append(int(tn[b, j]))
                j = int(pn[b, j])
            path_in = []
            v = int(tn[b, i])
            while v >= 0:
                path_in.append(v)
                v = int(par[b, v])
            assert path_in[:len(path_out)] == path_out
        # the kept node set is closed under children
        kept = set(tn[b, :n].tolist())
        for v in kept:
            assert all(c in kept for c in kids[v])


def _subtree_paths(par, tok, n):
    """key token -> set of token tuples, one per (node u, proper descendant v):
    the tokens from u's child down to v (every sub-tree of the draft)."""
    out = {}
    for v in range(n):
        chain = []
        a = v
        while a >= 0:
            chain.append(a)
            a = int(par[a])
        chain = chain[::-1]                       # root .. v
        for i in range(len(chain) - 1):           # u = chain[i]
            out.setdefault(int(tok[chain[i]]), set()).add(tuple(int(tok[x]) for x in chain[i + 1:]))
    return out


def _retrieved_paths(pn, tn, n):
    paths = set()
    for i in range(n):
        p = []
        j = i
        while j >= 0:
            p.append(int(tn[j]))
            j = int(pn[j])
        paths.add(tuple(p[::-1]))
    return paths


def test_pool_merge_is_the_union_of_token_paths():
    # M adds the children missing by value and merges the common ones, so a
    # pool tree's root paths are the union of those of the merged sub-trees
    rng = np.random.default_rng(40)
    B, T, V = 3, 24, 6                      # few token values: many merges hit
    pool = O.Pool(B, 512, 1024)
    want = [dict() for _ in range(B)]
    for step in range(4):
        par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
        tok = rng.integers(0, V, (B, T)).astype(np.int32)
        tl = rng.integers(1, T + 1, B).astype(np.int32)
        pool.merge(par, tok, tl)
        for b in range(B):
            for k, ps in _subtree_paths(par[b], tok[b], int(tl[b])).items():
                want[b].setdefault(k, set()).update(ps)
    for key in range(V + 1):
        pn, tn, ln = pool.retrieve(np.full(B, key, np.int32), 1024)
        for b in range(B):
            n = int(ln[b])
            assert _retrieved_paths(pn[b], tn[b], n) == want[b].get(key, set())
            # siblings carry distinct tokens, parents come first
            for i in range(n):
                assert pn[b, i] < i
                sib = [tn[b, j] for j in range(n) if pn[b, j] == pn[b, i]]
                assert len(sib) == len(set(sib))


def test_pool_golden():
    g = _golden("pool_example.json")
    par = np.array([g["draft"]["parent"]], np.int32)
    tok = np.array([g["draft"]["tokens"]], np.int32)
    for case in ("small", "large"):
        c = g[case]
        pool = O.Pool(1, c["e_max"], c["n_cap"])
        pool.merge(par, tok)
        for last, wp, wt in zip(c["last"], c["parent"], c["tokens"]):
            pn, tn, ln = pool.retrieve(np.array([last], np.int32), 8)
            assert ln[0] == len(wt), (case, last)
            assert pn[0, :ln[0]].tolist() == wp and tn[0, :ln[0]].tolist() == wt, (case, last)
            assert (pn[0, ln[0]:] == -1).all() and (tn[0, ln[0]:] == -1).all()


# ---------------------------------------------------------------------------
# paged caches
# ---------------------------------------------------------------------------
def test_gather_pages_inverts_a_scatter():
    # scatter a contiguous cache into pages through a random page table (numpy
    # indexing), then gather it back
    rng = np.random.default_rng(50)
    B, Hkv, D, ps, maxp = 3, 2, 8, 32, 5
    cache = rng.standard_normal((B, Hkv, maxp * ps, D)).astype(np.float32)
    num_pages = B * maxp + 4
    perm = rng.permutation(num_pages)[:B * maxp].reshape(B, maxp).astype(np.int32)
    pages = np.zeros((num_pages, Hkv, ps, D), np.float32)
    for b in range(B):
        for j in range(maxp):
            pages[perm[b, j]] = cache[b, :, j * ps:(j + 1) * ps]
    assert np.array_equal(O.gather_pages(pages, perm, ps), cache)
    # bf16 bits are moved as they are
    bits = W.f32_to_bf16_bits(pages)
    assert np.array_equal(O.gather_pages(bits, perm, ps), W.f32_to_bf16_bits(cache))


def test_gather_pages_identity_table_is_the_page_layout():
    rng = np.random.default_rng(51)
    Hkv, D, ps, maxp = 2, 4, 32, 3
    pages = rng.standard_normal((maxp, Hkv, ps, D)).astype(np.float32)
    got = O.gather_pages(pages, np.arange(maxp, dtype=np.int32)[None], ps)
    assert np.array_equal(got[0], pages.transpose(1, 0, 2, 3).reshape(Hkv, maxp * ps, D))
    with pytest.raises(O.OracleError):
        O.gather_pages(pages, np.array([[0, 1, 3]], np.int32), ps)
