"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol include/ptd.h declares, sizes workspaces, and rejects bad
arguments before launching anything (all calls here fail validation, so no
kernel is launched and no device pointer is touched)."""
import ctypes
import os
import re

import pytest

import paper_2607_10661_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "ptd.h")).read()
    return sorted(set(re.findall(r"^(?:int|size_t|const char\*)\s+(ptd_\w+)\(", src, re.M)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert "ptd_tree_attention" in names and len(names) >= 9
    lib = ctypes.CDLL(P.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
        assert hasattr(P, n), f"binding lacks {n}"


def test_status_strings():
    for code in range(0, 12):
        assert P.ptd_status_string(code) != "unknown status"
    assert P.ptd_status_string(99) == "unknown status"
    assert P.ptd_version() >= 100


def _shape(B=1, Hq=32, Hkv=32, D=128, L=2112, dt=P.PTD_BF16, od=P.PTD_BF16):
    return P.AttnShape(B, Hq, Hkv, D, L, dt, od, 0.0)


def test_attention_workspace_sizes():
    # splits * rows * (D + 2) fp32 partials, plus the masks, each 256-aligned
    n = P.ptd_tree_attention_workspace_bytes(_shape(), 64)
    assert n > 0 and n % 256 == 0
    assert n >= 64 * 32 * 130 * 4  # at least one split's partials
    assert P.ptd_tree_attention_workspace_bytes(_shape(dt=P.PTD_F32, D=64, Hq=2, Hkv=2, L=144),
                                                16) == 256  # masks only (no split)
    assert P.ptd_tree_attention_workspace_bytes(_shape(Hq=30, Hkv=8), 64) == 0  # Hq % Hkv
    assert P.ptd_tree_attention_workspace_bytes(_shape(D=96), 64) == 0
    assert P.ptd_tree_attention_workspace_bytes(_shape(), 0) == 0
    assert P.ptd_tree_attention_workspace_bytes(_shape(), P.PTD_MAX_T + 1) == 0
    # a cache shorter than T is valid for trees of fewer live nodes (ragged calls)
    assert P.ptd_tree_attention_workspace_bytes(_shape(dt=P.PTD_F32, D=64, Hq=2, Hkv=2, L=8),
                                                16) == 256
    assert P.ptd_tree_attention_workspace_bytes(_shape(L=0), 64) == 0


def test_attention_workspace_split_plans():
    # the partial bytes follow the plan's KV splits: one sequence of 256-row
    # groups: 16 splits (256 workgroups of 512 threads); a batch of them:
    # three splits per sequence (two 256-thread workgroups per CU)
    per = lambda B, splits: -(-splits * B * 8 * 256 * 130 * 4 // 256) * 256
    one = P.ptd_tree_attention_workspace_bytes(_shape(B=1, Hq=32, Hkv=8, L=32832), 64)
    assert one == per(1, 16)
    batch = P.ptd_tree_attention_workspace_bytes(_shape(B=16, Hq=32, Hkv=8, L=7798), 64)
    assert batch == per(16, 3)


def test_topk_workspace_sizes():
    assert P.ptd_topk_workspace_bytes(65, 300000, 4) > 0    # several slices per row
    assert P.ptd_topk_workspace_bytes(65, 128256, 4) == 65 * 8 * 4 * 16   # 8 fp32 slices (bf16: 4)
    assert P.ptd_topk_workspace_bytes(65, 32768, 4) == 65 * 2 * 4 * 16    # 2 fp32 slices
    assert P.ptd_topk_workspace_bytes(65, 16384, 4) == 0    # one slice per row
    assert P.ptd_topk_workspace_bytes(2048, 4000, 4) == 0   # one slice per row
    assert P.ptd_topk_workspace_bytes(4, 10, 11) == 0       # k > V
    assert P.ptd_topk_workspace_bytes(4, 100, 17) == 0      # k > PTD_MAX_K


FAKE = 1 << 20  # aligned non-null address; every call below fails validation first


def _err(fn, *a, **kw):
    with pytest.raises(P.PTDError) as e:
        fn(*a, stream=0, **kw)
    return e.value.status


def test_attention_validation():
    s = _shape()
    assert _err(P.ptd_tree_attention, None, FAKE, FAKE, FAKE, FAKE, 64, FAKE, s) == 1
    assert _err(P.ptd_tree_attention, FAKE, FAKE, FAKE, FAKE, FAKE, 0, FAKE, s) == 2
    assert _err(P.ptd_tree_attention, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE,
                _shape(L=32)) == 2                                      # L_cap < T
    assert _err(P.ptd_tree_attention, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE,
                _shape(Hq=3, Hkv=2)) == 2
    bad = _shape()
    bad.in_dtype = 7
    assert _err(P.ptd_tree_attention, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, bad) == 3
    assert _err(P.ptd_tree_attention, FAKE + 2, FAKE, FAKE, FAKE, FAKE, 64, FAKE, s) == 4
    # workspace missing / too small
    assert _err(P.ptd_tree_attention, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, s) == 5
    assert _err(P.ptd_tree_attention, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, s,
                workspace=FAKE, workspace_bytes=16) == 5


def test_ragged_attention_validation():
    s = _shape()
    A = P.ptd_tree_attention_ragged
    assert _err(A, None, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, s) == 1
    assert _err(A, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, FAKE, s) == 2
    assert _err(A, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, _shape(Hq=3, Hkv=2)) == 2
    assert _err(A, FAKE + 2, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, s) == 4
    assert _err(A, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, s) == 5  # no workspace


def test_noalloc_attention_validation():
    s = _shape()
    A = P.ptd_tree_attention_noalloc
    assert _err(A, None, FAKE, FAKE, FAKE, None, FAKE, 64, FAKE, s) == 1
    assert _err(A, FAKE, FAKE, FAKE, FAKE, None, FAKE, 0, FAKE, s) == 2
    assert _err(A, FAKE, FAKE, FAKE, FAKE, None, FAKE, 64, FAKE, _shape(Hq=3, Hkv=2)) == 2
    assert _err(A, FAKE + 2, FAKE, FAKE, FAKE, None, FAKE, 64, FAKE, s) == 4
    # 600 trees of 1024 nodes: their ancestor masks alone (78.6 MB) exceed the
    # fixed scratch; rejected before anything is looked up or launched
    big = _shape(B=600, Hq=1, Hkv=1, D=64, L=2048)
    assert P.ptd_tree_attention_workspace_bytes(big, 1024) > P.PTD_NOALLOC_SCRATCH_BYTES
    assert _err(A, FAKE, FAKE, FAKE, FAKE, None, FAKE, 1024, FAKE, big) == 11
    # the workloads' own problems fit (ragged-16's split partials: 34 MB)
    for shp, T in ((_shape(), 64), (_shape(B=16, Hkv=8, L=8256), 64),
                   (_shape(Hkv=8, L=32832), 64), (_shape(Hq=40, Hkv=40, L=4192), 96)):
        assert 0 < P.ptd_tree_attention_workspace_bytes(shp, T) <= P.PTD_NOALLOC_SCRATCH_BYTES


def test_fp8kv_attention_validation():
    s = _shape()
    A = P.ptd_tree_attention_fp8kv
    assert _err(A, None, FAKE, FAKE, None, None, FAKE, None, FAKE, 64, FAKE, s) == 1
    assert _err(A, FAKE, FAKE, FAKE, None, None, FAKE, None, FAKE, 64, FAKE,
                _shape(dt=P.PTD_F32, od=P.PTD_F32)) == 3               # bf16 queries only
    assert _err(A, FAKE, FAKE, FAKE, None, None, FAKE, None, FAKE, 64, FAKE, _shape(D=64)) == 2
    assert _err(A, FAKE, FAKE, FAKE, None, None, FAKE, None, FAKE, 64, FAKE, s) == 5
    assert _err(A, FAKE, FAKE, FAKE, FAKE + 2, None, FAKE, None, FAKE, 64, FAKE, s) == 4


def test_paged_fp8kv_attention_validation():
    s = _shape(L=2048)
    kv = P.KVPages(FAKE, FAKE, FAKE, 64, 32, 64)
    A = P.ptd_tree_attention_paged_fp8kv
    assert _err(A, FAKE, P.KVPages(FAKE, None, FAKE, 64, 32, 64), None, None, FAKE, None, FAKE,
                64, FAKE, s) == 1
    assert _err(A, FAKE, kv, None, None, FAKE, None, FAKE, 64, FAKE,
                _shape(L=2048, dt=P.PTD_F32, od=P.PTD_F32)) == 3
    assert _err(A, FAKE, P.KVPages(FAKE, FAKE, FAKE, 48, 2048 // 48, 64), None, None, FAKE, None,
                FAKE, 64, FAKE, s) == 2
    assert _err(A, FAKE, P.KVPages(FAKE, FAKE, FAKE, 64, 16, 64), None, None, FAKE, None, FAKE,
                64, FAKE, _shape(L=1024, D=64)) == 2
    assert _err(A, FAKE, kv, FAKE + 2, None, FAKE, None, FAKE, 64, FAKE, s) == 4
    assert _err(A, FAKE, kv, None, None, FAKE, None, FAKE, 64, FAKE, s) == 5


def test_topk_verify_expand_mask_validation():
    assert _err(P.ptd_topk_argmax, None, P.PTD_BF16, 4, 100, 100, 4, FAKE) == 1
    assert _err(P.ptd_topk_argmax, FAKE, 5, 4, 100, 100, 4, FAKE) == 3
    assert _err(P.ptd_topk_argmax, FAKE, P.PTD_BF16, 4, 100, 99, 4, FAKE) == 2   # ld < V
    assert _err(P.ptd_topk_argmax, FAKE, P.PTD_BF16, 4, 100, 100, 17, FAKE) == 2
    assert _err(P.ptd_topk_argmax, FAKE + 1, P.PTD_BF16, 4, 100, 100, 4, FAKE) == 4
    # a row beyond one workgroup's slice is split over slices, which needs a workspace
    assert _err(P.ptd_topk_argmax, FAKE, P.PTD_BF16, 65, 300000, 300000, 4, FAKE) == 5
    assert _err(P.ptd_topk_argmax, FAKE, P.PTD_F32, 65, 200000, 200000, 4, FAKE) == 5
    assert _err(P.ptd_verify, FAKE, FAKE, None, None, 1, 4, FAKE, FAKE, FAKE) == 1
    assert _err(P.ptd_verify, FAKE, FAKE, FAKE, None, 1, 0, FAKE, FAKE, FAKE) == 2
    assert _err(P.ptd_verify, FAKE, FAKE, FAKE, None, 1, P.PTD_MAX_T + 1, FAKE, FAKE, FAKE) == 2
    assert _err(P.ptd_expand, FAKE, FAKE, None, 1, 4, FAKE, 0, [4], 1, 8, FAKE, FAKE, FAKE) == 2
    assert _err(P.ptd_expand, FAKE, FAKE, None, 1, 4, FAKE, 2, [4] * 65, 65, 8, FAKE, FAKE,
                FAKE) == 2
    assert _err(P.ptd_build_tree_mask, FAKE, None, 0, 4, FAKE, FAKE) == 2
    assert _err(P.ptd_build_tree_mask, None, None, 1, 4, FAKE, FAKE) == 1


def test_rope_commit_validation():
    s = _shape(Hq=32, Hkv=8, L=4096)
    R = P.ptd_tree_rope
    assert _err(R, None, None, FAKE, FAKE, 64, s) == 1                 # nothing to turn or write
    assert _err(R, FAKE, FAKE, None, FAKE, 64, s) == 1
    assert _err(R, FAKE, FAKE, FAKE, FAKE, 0, s) == 2
    assert _err(R, FAKE, FAKE, FAKE, FAKE, 64, _shape(L=32)) == 2      # L_cap < T
    assert _err(R, FAKE, FAKE, FAKE, FAKE, 64, _shape(D=96)) == 2
    assert _err(R, FAKE, FAKE, FAKE, FAKE, 64, s, pairing=2) == 2
    assert _err(R, FAKE, FAKE, FAKE, FAKE, 64, s, theta=0.0) == 2
    assert _err(R, FAKE, FAKE, FAKE, FAKE, 64, s, theta=float("inf")) == 2
    bad = _shape()
    bad.in_dtype = 7
    assert _err(R, FAKE, FAKE, FAKE, FAKE, 64, bad) == 3
    assert _err(R, FAKE + 8, FAKE, FAKE, FAKE, 64, s) == 4
    assert _err(R, FAKE, FAKE + 4, FAKE, FAKE, 64, s) == 4
    with pytest.raises(ValueError):
        R(FAKE, FAKE, FAKE, FAKE, 64, s, inv_freq=[1.0] * 3, stream=0)
    C = P.ptd_kv_commit
    assert _err(C, FAKE, None, FAKE, FAKE, FAKE, 64, s, FAKE) == 1
    assert _err(C, FAKE, FAKE, FAKE, FAKE, FAKE, 64, s, None) == 1
    assert _err(C, FAKE, FAKE, FAKE, FAKE, FAKE, 64, s, FAKE) == 2    # kv_len_next aliases kv_len
    assert _err(C, FAKE, FAKE, FAKE, FAKE, FAKE, 0, s, FAKE * 2) == 2
    assert _err(C, FAKE, FAKE, FAKE, FAKE, FAKE, P.PTD_MAX_T + 1, _shape(L=8192), FAKE * 2) == 2
    assert _err(C, FAKE, FAKE, FAKE, FAKE, FAKE, 64, bad, FAKE * 2) == 3
    assert _err(C, FAKE, FAKE + 2, FAKE, FAKE, FAKE, 64, s, FAKE * 2) == 4


def test_verify_sample_validation():
    # 65 rows x 16 blocks of 2048 entries x 16 B, 256-rounded
    assert P.ptd_verify_sample_workspace_bytes(1, 64, 32000) == 65 * 16 * 16
    assert P.ptd_verify_sample_workspace_bytes(1, 64, 100) == 1280
    assert P.ptd_verify_sample_workspace_bytes(0, 64, 100) == 0
    assert P.ptd_verify_sample_workspace_bytes(1, P.PTD_MAX_T + 1, 100) == 0
    assert P.ptd_verify_sample_workspace_bytes(1, 64, 262145) == 0
    S = P.ptd_verify_sample
    args = dict(workspace=FAKE, workspace_bytes=1 << 20)
    assert _err(S, None, P.PTD_BF16, 100, 100, FAKE, FAKE, None, 1, 4, 1.0, FAKE, FAKE, FAKE,
                FAKE, FAKE, **args) == 1
    assert _err(S, FAKE, 5, 100, 100, FAKE, FAKE, None, 1, 4, 1.0, FAKE, FAKE, FAKE, FAKE,
                FAKE, **args) == 3
    assert _err(S, FAKE, P.PTD_BF16, 100, 99, FAKE, FAKE, None, 1, 4, 1.0, FAKE, FAKE, FAKE,
                FAKE, FAKE, **args) == 2                                     # ld < V
    assert _err(S, FAKE, P.PTD_BF16, 262145, 262145, FAKE, FAKE, None, 1, 4, 1.0, FAKE, FAKE,
                FAKE, FAKE, FAKE, **args) == 2                               # V above the bitmap
    for t in (0.0, -1.0, float("inf"), float("nan")):
        assert _err(S, FAKE, P.PTD_BF16, 100, 100, FAKE, FAKE, None, 1, 4, t, FAKE, FAKE, FAKE,
                    FAKE, FAKE, **args) == 2
    assert _err(S, FAKE, P.PTD_BF16, 100, 100, FAKE, FAKE, None, 1, 4, 1.0, FAKE, FAKE, FAKE,
                FAKE, FAKE, workspace=FAKE, workspace_bytes=16) == 5
    assert _err(S, FAKE, P.PTD_BF16, 100, 100, FAKE, FAKE, None, 1, 4, 1.0, FAKE, FAKE, FAKE,
                FAKE, FAKE, workspace=FAKE + 4, workspace_bytes=1 << 20) == 4
    assert _err(S, FAKE, P.PTD_BF16, 100, 100, FAKE, FAKE, None, 1000, 65, 1.0, FAKE, FAKE,
                FAKE, FAKE, FAKE, **args) == 2                               # rows > 65535


def test_step_prune_and_pool_validation():
    assert P.ptd_pool_bytes(1, 0, 8) == 0 and P.ptd_pool_bytes(1, 2049, 8) == 0
    assert P.ptd_pool_bytes(1, 8, 130) == 0 and P.ptd_pool_bytes(0, 8, 8) == 0
    # 16-byte header, 64 hash slots (key + tree), 8 counts, 8 x 8 nodes, 256-rounded
    assert P.ptd_pool_bytes(1, 8, 8) == 1280 and P.ptd_pool_bytes(3, 8, 8) == 3 * 1280
    assert _err(P.ptd_step_prune, None, FAKE, None, 1, 8, 2, 8, FAKE, FAKE, FAKE) == 1
    assert _err(P.ptd_step_prune, FAKE, FAKE, None, 1, 129, 2, 8, FAKE, FAKE, FAKE) == 2
    assert _err(P.ptd_step_prune, FAKE, FAKE, None, 1, 8, 0, 8, FAKE, FAKE, FAKE) == 2
    nb = P.ptd_pool_bytes(2, 16, 8)
    assert _err(P.ptd_pool_init, None, nb, 2, 16, 8) == 1
    assert _err(P.ptd_pool_init, FAKE, nb - 1, 2, 16, 8) == 5
    assert _err(P.ptd_pool_init, FAKE + 16, nb, 2, 16, 8) == 4
    assert _err(P.ptd_pool_merge, FAKE, nb, 2, 16, 8, FAKE, FAKE, None, 129) == 2
    assert _err(P.ptd_pool_merge, FAKE, nb, 2, 16, 8, None, FAKE, None, 8) == 1
    assert _err(P.ptd_pool_retrieve, FAKE, nb, 2, 16, 8, FAKE, 0, FAKE, FAKE, FAKE) == 2
    assert _err(P.ptd_pool_retrieve, FAKE, nb, 2, 16, 130, FAKE, 8, FAKE, FAKE, FAKE) == 2


def test_paged_attention_validation():
    s = _shape(L=2048)
    kv = P.KVPages(FAKE, FAKE, FAKE, 64, 32, 64)
    A = P.ptd_tree_attention_paged
    bad_null = P.KVPages(FAKE, None, FAKE, 64, 32, 64)
    assert _err(A, FAKE, bad_null, FAKE, None, FAKE, 64, FAKE, s) == 1
    f32 = _shape(L=2048, dt=P.PTD_F32, od=P.PTD_F32)
    assert _err(A, FAKE, kv, FAKE, None, FAKE, 64, FAKE, f32) == 3            # bf16 only
    for ps in (16, 48, 96):                                              # power of two >= 32
        assert _err(A, FAKE, P.KVPages(FAKE, FAKE, FAKE, ps, 2048 // ps, 64), FAKE, None, FAKE, 64,
                    FAKE, s) == 2
    assert _err(A, FAKE, P.KVPages(FAKE, FAKE, FAKE, 64, 31, 64), FAKE, None, FAKE, 64, FAKE, s) == 2
    assert _err(A, FAKE, P.KVPages(FAKE, FAKE, FAKE, 64, 32, 0), FAKE, None, FAKE, 64, FAKE, s) == 2
