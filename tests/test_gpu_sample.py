"""GPU parity of sampling verification (ptd_verify_sample) against the fp64
CPU oracle, through the C ABI, on the same seeded logits, trees and uniforms.

Accepted lengths, paths and emitted tokens are integers decided by comparing
uniforms with probabilities.  The kernel computes the normalizer and the bonus
CDF from fp32 exponentials taken per block of 2048 entries and rescaled to
the row maximum (each factor within ~1.2e-7 relative: one ulp of the hardware
exp2, argument rounding compensated) summed in fp64, the oracle in fp64
throughout, so a probability or cumulative probability may differ by ~5e-7
at most.  The oracle reports, per sequence, the smallest distance of a
uniform from a boundary it was compared with (its margin).  A sequence whose
margin exceeds DELTA must equal the oracle's result exactly; one with a
smaller margin must equal it for the given uniforms, or for the same
uniforms all shifted by +DELTA or -DELTA (a decision within rounding of its
boundary going either way).
"""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

pytestmark = pytest.mark.gpu
DELTA = 6e-7


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


def likely_tokens(rng, logits_f32, parent, top=3, p_random=0.2):
    """Child tokens drawn among the top few of the parent's row (so walks go
    deep), sometimes uniformly at random."""
    B, T = parent.shape
    V = logits_f32.shape[-1]
    tok = np.empty((B, T), np.int32)
    for b in range(B):
        order = np.argsort(-logits_f32[b], axis=-1, kind="stable")[:, :top]
        for i in range(T):
            if rng.random() < p_random:
                tok[b, i] = rng.integers(0, V)
            else:
                tok[b, i] = order[parent[b, i] + 1, rng.integers(0, top)]
    return tok


def sample_case(P, lg, tok, par, temp, u1, u2, tree_len=None, ld=None):
    B, T = par.shape
    al_r, an_r, ot_r, mg_r = O.verify_sample(lg, tok, par, temp, u1, u2, tree_len)
    V = lg.shape[-1]
    flat = lg.reshape(B * (T + 1), V)
    if ld is not None and ld > V:
        buf = np.zeros((B * (T + 1), ld), flat.dtype)
        buf[:, :V] = flat
        t = cu(buf)[:, :V]
    else:
        t = cu(flat)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    al, an, ot = P.verify_sample(t, cu(tok), cu(par), temp, cu(u1), cu(u2),
                                 None if tree_len is None else cu(tree_len), dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    al, an, ot = al.cpu().numpy(), an.cpu().numpy(), ot.cpu().numpy()
    lgb = lg.reshape(B, T + 1, V)
    for b in range(B):
        if al[b] == al_r[b] and np.array_equal(an[b], an_r[b]) and np.array_equal(ot[b], ot_r[b]):
            continue
        assert mg_r[b] <= DELTA, (b, "differs although every decision is %.3g from its boundary"
                                  % mg_r[b])
        ok = False
        for sgn in (1.0, -1.0):
            sl = slice(b, b + 1)
            r = O.verify_sample(lgb[sl], tok[sl], par[sl], temp,
                                np.clip(u1[sl] + sgn * DELTA, 0.0, 1.0 - 2 ** -53),
                                np.clip(u2[sl] + sgn * DELTA, 0.0, 1.0 - 2 ** -53),
                                None if tree_len is None else tree_len[sl])
            if r[0][0] == al[b] and np.array_equal(r[1][0], an[b]) and np.array_equal(r[2][0], ot[b]):
                ok = True
        assert ok, (b, al[b], al_r[b], ot[b][:al[b] + 2], ot_r[b][:al_r[b] + 2])
    return al_r, ot_r


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("temp", [0.6, 1.0, 1.7])
def test_sample_random_trees(P, dtype, temp):
    rng = np.random.default_rng(int(temp * 10) + (dtype == "bf16"))
    B, T, V = 24, 20, 1000
    par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    x = (rng.standard_normal((B, T + 1, V)) * 2.0).astype(np.float32)
    # a dominant token per row (+8 nats) so that accepted chains form
    np.put_along_axis(x, np.argmax(x, axis=-1)[..., None],
                      np.max(x, axis=-1, keepdims=True) + 8.0, axis=-1)
    lg = W.f32_to_bf16_bits(x) if dtype == "bf16" else x
    lf = W.bf16_bits_to_f32(lg) if dtype == "bf16" else lg
    tok = likely_tokens(rng, lf, par)
    al, _ = sample_case(P, lg, tok, par, temp, rng.random((B, T)), rng.random((B, T + 1)))
    assert al.max() >= 2  # the walks do go below the roots


@pytest.mark.parametrize("name", ["llama2-7b", "llama2-13b", "llama3-8b-long", "ragged-16"])
def test_sample_configs(P, name):
    w = W.make_workload(name)
    rng = np.random.default_rng(5)
    B, T = w.B, w.T
    lf = W.bf16_bits_to_f32(w.logits).reshape(B, T + 1, w.V)
    tok = likely_tokens(rng, lf, w.parent, top=2, p_random=0.1)
    for draw in range(4):  # several draws of the uniforms
        sample_case(P, w.logits.reshape(B, T + 1, w.V), tok, w.parent, 1.0, rng.random((B, T)),
                    rng.random((B, T + 1)))


@pytest.mark.parametrize("B,T", [(2, 8), (8, 63)])
def test_sample_wide_rows_f32(P, B, T):
    # fp32 rows of more than 32 statistics blocks (the walk's wave-per-row
    # forms), with few blocks per call and with many (8192 or more: the
    # wave-per-block statistics)
    rng = np.random.default_rng(11 + B)
    V = 70001
    par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    x = (rng.standard_normal((B, T + 1, V)) * 2.0).astype(np.float32)
    np.put_along_axis(x, np.argmax(x, axis=-1)[..., None],
                      np.max(x, axis=-1, keepdims=True) + 6.0, axis=-1)
    tok = likely_tokens(rng, x, par, top=2, p_random=0.1)
    sample_case(P, x, tok, par, 1.0, rng.random((B, T)), rng.random((B, T + 1)))


def test_sample_wide_star_with_duplicates(P):
    # one node with 1000 children (many rejections, repeated tokens): the
    # rejected-token bitmap and the residual CDF
    rng = np.random.default_rng(6)
    B, T, V = 4, 1000, 5000
    par = np.full((B, T), -1, np.int32)
    x = rng.standard_normal((B, T + 1, V)).astype(np.float32)
    top = np.argsort(-x[:, 0], axis=-1)[:, :50]
    tok = np.stack([top[b, rng.integers(0, 50, T)] for b in range(B)]).astype(np.int32)
    u1 = rng.uniform(0.3, 1.0, (B, T))   # mostly rejections
    sample_case(P, x, tok, par, 1.0, u1, rng.random((B, T + 1)))


def test_sample_chain_padding_and_strided_rows(P):
    rng = np.random.default_rng(7)
    B, T, V = 6, 40, 3001
    par = np.stack([W.tree_chain(T)[0]] * 3 + [W.tree_uniform(rng, T)[0] for _ in range(3)])
    x = (rng.standard_normal((B, T + 1, V)) * 3.0).astype(np.float32)
    tok = likely_tokens(rng, x, par, top=1, p_random=0.0)
    tl = np.array([T, 7, 0, T, 1, 25], np.int32)
    sample_case(P, x, tok, par, 0.8, rng.random((B, T)) * 0.5, rng.random((B, T + 1)),
                tree_len=tl, ld=V + 5)


def test_sample_single_node_and_low_temperature(P):
    rng = np.random.default_rng(8)
    B, V = 32, 777
    x = rng.standard_normal((B, 2, V)).astype(np.float32)
    par = np.full((B, 1), -1, np.int32)
    tok = np.argmax(x[:, 0], axis=-1).astype(np.int32)[:, None]
    tok[::3] = (tok[::3] + 1) % V
    sample_case(P, x, tok, par, 0.05, rng.uniform(0.01, 0.99, (B, 1)), rng.random((B, 2)))


def test_sample_bad_tree_reports(P):
    rng = np.random.default_rng(9)
    par = np.array([[-1, 0, 2, 1], [-1, -1, 0, 1]], np.int32)
    x = rng.standard_normal((2, 5, 64)).astype(np.float32)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    al, an, ot = P.verify_sample(cu(x), cu(np.zeros((2, 4), np.int32)), cu(par), 1.0,
                                 cu(rng.random((2, 4))), cu(rng.random((2, 5))), dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 7
    assert al[0].item() == 0 and (an[0] == -1).all() and (ot[0] == -1).all()


def test_sample_deterministic(P):
    rng = np.random.default_rng(10)
    B, T, V = 8, 64, 32000
    par = np.stack([W.tree_uniform(rng, T)[0] for _ in range(B)])
    x = W.f32_to_bf16_bits(rng.standard_normal((B, T + 1, V)).astype(np.float32))
    tok = likely_tokens(rng, W.bf16_bits_to_f32(x), par)
    args = (cu(x), cu(tok), cu(par), 1.0, cu(rng.random((B, T))), cu(rng.random((B, T + 1))))
    r1 = [t.cpu() for t in P.verify_sample(*args)]
    r2 = [t.cpu() for t in P.verify_sample(*args)]
    assert all(torch.equal(a, b) for a, b in zip(r1, r2))
