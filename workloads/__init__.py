"""Seeded synthetic inputs for one Progressive Tree Drafting step.

This module is shared by the CPU oracle side (tests) and the GPU side (tests,
bench).  It only draws random numbers and builds input *structure* (tree shapes,
token ids, a planted accepted path); it contains none of the method's
arithmetic: no attention, no argmax/top-k, no verification, no expansion.

Workload shapes follow the paper's setting (Sec. 4.1: batch 1, BF16, Llama-2/3
shaped models; Sec. 4.2.2: tree width 4, depth 6; App. H Table 5: 48-73 extra
tree tokens per forward).  The datasets the paper measures on (MT-Bench,
GSM-100, HumanEval, MBPP-100) are not available; these seeded inputs stand in
for them.

Planting an accepted path without computing any argmax: along a chosen
root-to-node path n_1..n_d, the logit of token[n_j] in the row of n_j's parent
is overwritten with PLANT_VALUE, which exceeds every drawn logit (draws are
clipped to +-CLIP).  The row of the terminal node gets PLANT_VALUE at a "bonus"
token that no child of the terminal carries.  Sibling tokens are distinct, so
no other node can join the accepted path: the greedy accepted length is exactly
d by construction.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Union

import numpy as np

PLANT_VALUE = 16.0   # exactly representable in bf16 and fp32
CLIP = 12.0          # |drawn logit| <= CLIP < PLANT_VALUE

# ---------------------------------------------------------------------------
# Named configurations (sizes of the paper-shaped workloads)
# ---------------------------------------------------------------------------
CONFIGS: Dict[str, dict] = {
    # 2 heads, head_dim 64, committed KV 128, 16 nodes, parent uniform over
    # {-1, 0..i-1}; fp32; vocab 1000; planted accepted depth 3.
    "tiny": dict(B=1, Hq=2, Hkv=2, D=64, kv_len=128, T=16, tree="uniform",
                 V=1000, logit_std=1.0, dtype="f32", plant=3, k=4,
                 width=[4, 4, 4, 4, 4, 4], seed=0),
    # Llama-2-7B attention shape: 32 heads, head_dim 128, KV 2048, T=64.
    "llama2-7b": dict(B=1, Hq=32, Hkv=32, D=128, kv_len=2048, T=64,
                      tree=[4, 3, 2, 2, 1], V=32000, logit_std=math.sqrt(2.0),
                      dtype="bf16", plant=4, k=4, width=[4, 3, 2, 2, 1], seed=1),
    # Llama-2-13B attention shape: 40 heads, KV 4096, T=96.
    "llama2-13b": dict(B=1, Hq=40, Hkv=40, D=128, kv_len=4096, T=96,
                       tree=[5, 4, 3, 2, 1, 1], V=32000, logit_std=math.sqrt(2.0),
                       dtype="bf16", plant=("uniform", 6), k=5,
                       width=[5, 4, 3, 2, 1, 1], seed=2),
    # Llama-3-8B GQA (32 query / 8 KV heads), long context 32768, T=64,
    # vocab 128256, top-8 child expansion.
    "llama3-8b-long": dict(B=1, Hq=32, Hkv=8, D=128, kv_len=32768, T=64,
                           tree=[4, 3, 2, 2, 1], V=128256,
                           logit_std=math.sqrt(2.0), dtype="bf16", plant=4, k=8,
                           width=[4, 3, 2, 2, 1], seed=3),
    # 16 sequences, KV length uniform in [512, 8192], Llama-3-8B GQA shape.
    "ragged-16": dict(B=16, Hq=32, Hkv=8, D=128, kv_len=("uniform", 512, 8192),
                      T=64, tree=[4, 3, 2, 2, 1], V=128256,
                      logit_std=math.sqrt(2.0), dtype="bf16",
                      plant=("uniform", 5), k=8, width=[4, 3, 2, 2, 1], seed=4),
}


# ---------------------------------------------------------------------------
# dtype helpers (bit-level conversions, no arithmetic of the method)
# ---------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even), returning uint16 bits.
    Inputs are finite (no NaN handling needed)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bits to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


# The 127 non-negative finite OCP E4M3 values, indexed by their code (0x00 ..
# 0x7E): (1 + m/8) * 2^(e-7), subnormals (m/8) * 2^-6 at e = 0.
_E4M3_POS = np.array([(m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
                      for e in range(16) for m in range(8)][:127], np.float64)


def f32_to_e4m3_bits(x: np.ndarray) -> np.ndarray:
    """Round to the nearest OCP E4M3 value (ties to the even code, i.e. even
    mantissa), saturating at +-448; returns uint8 codes.  Inputs are finite."""
    a = np.abs(np.asarray(x, np.float64))
    a = np.minimum(a, 448.0)
    hi = np.clip(np.searchsorted(_E4M3_POS, a, side="left"), 0, 126)
    lo = np.clip(hi - 1, 0, 126)
    d_hi = _E4M3_POS[hi] - a
    d_lo = a - _E4M3_POS[lo]
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (lo % 2 == 0))
    code = np.where(pick_lo, lo, hi).astype(np.uint8)
    return code | np.where(np.signbit(np.asarray(x, np.float64)), 0x80, 0).astype(np.uint8)


def quantize_kv_e4m3(cache: np.ndarray):
    """A float cache [B][Hkv][L][D] -> (E4M3 codes, float32 scale per KV head):
    scale_g = max |x| over the head / 448, codes = e4m3(x / scale_g)."""
    x = np.asarray(cache, np.float64)
    amax = np.abs(x).max(axis=(0, 2, 3))
    scale = np.where(amax > 0, amax / 448.0, 1.0).astype(np.float32)
    codes = f32_to_e4m3_bits(x / scale.astype(np.float64)[None, :, None, None])
    return codes, scale


def to_f64(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of a workload array ("bf16" bits or "f32") to float64."""
    if dtype == "bf16":
        return bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float32).astype(np.float64)


def _draw(rng: np.random.Generator, shape, dtype: str, std: float = 1.0,
          clip: Optional[float] = None) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    if clip is not None:
        np.clip(x, -clip, clip, out=x)
    return f32_to_bf16_bits(x) if dtype == "bf16" else x


# ---------------------------------------------------------------------------
# Tree shapes (parent arrays in topological order: parent[i] in [-1, i))
# ---------------------------------------------------------------------------
def tree_uniform(rng: np.random.Generator, T: int):
    """parent[i] uniform over {-1, 0, .., i-1}.  Returns (parent, level) where
    level[i] is the number of nodes on the root path of i (built while drawing)."""
    parent = np.empty(T, np.int32)
    level = np.empty(T, np.int32)
    for i in range(T):
        p = int(rng.integers(-1, i)) if i > 0 else -1
        parent[i] = p
        level[i] = 1 if p < 0 else level[p] + 1
    return parent, level


def tree_branching(branching: Sequence[int], T: int):
    """Level-by-level tree: branching[0] roots, every node on level d gets
    branching[d] children; nodes numbered in BFS order and truncated to T."""
    parent: List[int] = []
    level: List[int] = []
    frontier = [-1]
    for d, w in enumerate(branching):
        nxt = []
        for p in frontier:
            for _ in range(w):
                if len(parent) == T:
                    break
                parent.append(p)
                level.append(d + 1)
                nxt.append(len(parent) - 1)
        frontier = nxt
        if len(parent) == T:
            break
    if len(parent) < T:
        raise ValueError("branching schedule yields fewer than T nodes")
    return np.asarray(parent, np.int32), np.asarray(level, np.int32)


def tree_chain(T: int):
    parent = np.arange(-1, T - 1, dtype=np.int32)
    return parent, np.arange(1, T + 1, dtype=np.int32)


def tree_star(T: int):
    return np.full(T, -1, np.int32), np.ones(T, np.int32)


def make_tree(rng: np.random.Generator, kind, T: int):
    if isinstance(kind, (list, tuple)):
        return tree_branching(kind, T)
    if kind == "uniform":
        return tree_uniform(rng, T)
    if kind == "chain":
        return tree_chain(T)
    if kind == "star":
        return tree_star(T)
    raise ValueError(f"unknown tree kind {kind!r}")


def sibling_distinct_tokens(rng: np.random.Generator, parent: np.ndarray, V: int):
    """Token ids uniform in [0, V), pairwise distinct among siblings (nodes
    with the same parent, roots being siblings of each other)."""
    T = parent.shape[0]
    tokens = np.empty(T, np.int32)
    groups: Dict[int, List[int]] = {}
    for i in range(T):
        groups.setdefault(int(parent[i]), []).append(i)
    for p in sorted(groups):
        members = groups[p]
        if len(members) > V:
            raise ValueError("more siblings than vocabulary entries")
        tokens[members] = rng.choice(V, size=len(members), replace=False)
    return tokens


# ---------------------------------------------------------------------------
# Workload container
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    D: int
    T: int
    V: int
    L_cap: int
    dtype: str                  # "bf16" (uint16 bits) or "f32"
    scale: float                # softmax scale 1/sqrt(D)
    q: np.ndarray               # [B][T][Hq][D]
    k_cache: np.ndarray         # [B][Hkv][L_cap][D]; node i at row kv_len[b]+i
    v_cache: np.ndarray         # [B][Hkv][L_cap][D]
    kv_len: np.ndarray          # int32 [B]
    parent: np.ndarray          # int32 [B][T]
    tokens: np.ndarray          # int32 [B][T]
    logits: np.ndarray          # [B][T+1][V]; row 0 = last committed token
    k: int                      # top-k for child expansion
    width: List[int]            # width_sched[d] = max children of a depth-d node
    d_max: int
    T_max: int
    level: np.ndarray           # int32 [B][T], root-path node count (generator's own)
    planted_depth: np.ndarray   # int32 [B]
    planted_path: List[List[int]]
    planted_bonus: np.ndarray   # int32 [B]

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    def nbytes_inputs(self) -> int:
        return sum(a.nbytes for a in (self.q, self.k_cache, self.v_cache,
                                      self.logits, self.parent, self.tokens))


def _resolve(spec, rng, key):
    v = spec[key]
    if isinstance(v, tuple) and v and v[0] == "uniform":
        if len(v) == 2:
            return int(rng.integers(0, v[1] + 1))
        return int(rng.integers(v[1], v[2] + 1))
    return v


def make_workload(spec: Union[str, dict], seed: Optional[int] = None,
                  logits: bool = True, kv: bool = True) -> Workload:
    """Build the seeded workload for a named config or an explicit spec dict.

    spec keys: B, Hq, Hkv, D, kv_len (int, list, or ("uniform", lo, hi)),
    T, tree ("uniform" | "chain" | "star" | branching list), V, logit_std,
    dtype, plant (int depth, ("uniform", max), or None), k, width.
    Optional: L_pad (extra unused cache rows), d_max, T_max.
    With B > 1 every sequence draws from its own child seed stream.
    """
    name = spec if isinstance(spec, str) else spec.get("name", "custom")
    spec = dict(CONFIGS[spec]) if isinstance(spec, str) else dict(spec)
    if seed is None:
        seed = spec.get("seed", 0)
    B, Hq, Hkv, D, T, V = (spec[x] for x in ("B", "Hq", "Hkv", "D", "T", "V"))
    dtype = spec["dtype"]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    if B == 1:
        rngs = [np.random.Generator(np.random.PCG64(seed))]
    else:
        rngs = [np.random.Generator(np.random.PCG64(s))
                for s in np.random.SeedSequence(seed).spawn(B)]

    kvl = spec["kv_len"]
    kv_len = np.empty(B, np.int32)
    for b in range(B):
        if isinstance(kvl, (list, np.ndarray)):
            kv_len[b] = kvl[b]
        else:
            kv_len[b] = _resolve(spec, rngs[b], "kv_len")
    L_cap = int(kv_len.max()) + T + int(spec.get("L_pad", 0))

    edt = np.uint16 if dtype == "bf16" else np.float32
    q = np.zeros((B, T, Hq, D), edt)
    kc = np.zeros((B, Hkv, L_cap, D), edt)
    vc = np.zeros((B, Hkv, L_cap, D), edt)
    parent = np.empty((B, T), np.int32)
    tokens = np.empty((B, T), np.int32)
    level = np.empty((B, T), np.int32)
    lg = np.zeros((B, T + 1, V), edt) if logits else np.zeros((B, T + 1, 0), edt)
    pdepth = np.zeros(B, np.int32)
    pbonus = np.zeros(B, np.int32)
    ppath: List[List[int]] = []

    for b in range(B):
        rng = rngs[b]
        # tree first (so that "uniform" trees can be redrawn until the planted
        # depth exists)
        plant = spec.get("plant")
        while True:
            par, lev = make_tree(rng, spec["tree"], T)
            if plant is None:
                d = 0
                break
            if isinstance(plant, tuple):
                d = int(rng.integers(0, min(plant[1], int(lev.max())) + 1))
                break
            d = int(plant)
            if d == 0 or (lev == d).any():
                break
            if spec["tree"] != "uniform":
                raise ValueError("tree has no node at the planted depth")
        parent[b], level[b] = par, lev
        tokens[b] = sibling_distinct_tokens(rng, par, V)
        n = int(kv_len[b])
        if kv:
            q[b] = _draw(rng, (T, Hq, D), dtype)
            kc[b, :, : n + T] = _draw(rng, (Hkv, n + T, D), dtype)
            vc[b, :, : n + T] = _draw(rng, (Hkv, n + T, D), dtype)
        if logits:
            lg[b] = _draw(rng, (T + 1, V), dtype, spec.get("logit_std", 1.0), CLIP)
        # planted accepted path of depth d
        path: List[int] = []
        if plant is not None:
            if d > 0:
                cands = np.flatnonzero(lev == d)
                a = int(cands[rng.integers(0, cands.size)])
                while a != -1:
                    path.append(a)
                    a = int(par[a])
                path.reverse()
            term_row = path[-1] + 1 if path else 0
            term = path[-1] if path else -1
            taken = set(int(tokens[b, c]) for c in np.flatnonzero(par == term))
            while True:
                bonus = int(rng.integers(0, V))
                if bonus not in taken:
                    break
            if logits:
                pv = (f32_to_bf16_bits(np.array([PLANT_VALUE], np.float32))[0]
                      if dtype == "bf16" else np.float32(PLANT_VALUE))
                for a in path:
                    lg[b, int(par[a]) + 1, int(tokens[b, a])] = pv
                lg[b, term_row, bonus] = pv
            pbonus[b] = bonus
        pdepth[b] = len(path)
        ppath.append(path)

    width = list(spec.get("width", [4] * 6))
    return Workload(
        name=name, B=B, Hq=Hq, Hkv=Hkv, D=D, T=T, V=V, L_cap=L_cap, dtype=dtype,
        scale=1.0 / math.sqrt(D), q=q, k_cache=kc, v_cache=vc, kv_len=kv_len,
        parent=parent, tokens=tokens, logits=lg, k=int(spec.get("k", 4)),
        width=width, d_max=int(spec.get("d_max", len(width))),
        T_max=int(spec.get("T_max", T)), level=level, planted_depth=pdepth,
        planted_path=ppath, planted_bonus=pbonus)


def algorithmic_bytes(w: Workload) -> Dict[str, int]:
    """Bytes one step must move at least once (committed K/V read once, tree
    K/V, q, out, logits; int arrays are negligible and left out)."""
    es = 2 if w.dtype == "bf16" else 4
    committed = int(w.kv_len.sum()) * w.Hkv * w.D * 2 * es
    tree_kv = w.B * w.T * w.Hkv * w.D * 2 * es
    q_out = 2 * w.B * w.T * w.Hq * w.D * es
    logits = w.B * (w.T + 1) * w.V * es
    attn = committed + tree_kv + q_out
    return dict(committed_kv=committed, tree_kv=tree_kv, q_out=q_out,
                attention=attn, logits=logits, step=attn + logits)


def ragged_attention_bytes(w: Workload, tree_len: np.ndarray) -> int:
    """Algorithmic bytes of the attention over trees of tree_len[b] live
    nodes: committed K/V, the live tree rows' K/V, q and out of live rows."""
    es = 2 if w.dtype == "bf16" else 4
    live = int(np.clip(np.asarray(tree_len), 0, w.T).sum())
    return (int(w.kv_len.sum()) * w.Hkv * w.D * 2 * es + live * w.Hkv * w.D * 2 * es
            + 2 * live * w.Hq * w.D * es)


def fp8kv_attention_bytes(w: Workload) -> int:
    """Algorithmic bytes of the attention on 8-bit key/value caches: committed
    and tree K/V at one byte per element, q and out at the workload's width."""
    es = 2 if w.dtype == "bf16" else 4
    kv = (int(w.kv_len.sum()) + w.B * w.T) * w.Hkv * w.D * 2
    return kv + 2 * w.B * w.T * w.Hq * w.D * es


def rope_bytes(w: Workload) -> int:
    """Bytes the rotary embedding of the tree rows moves: every query head
    and tree key row of every node read and written once."""
    es = 2 if w.dtype == "bf16" else 4
    return 2 * w.B * w.T * (w.Hq + w.Hkv) * w.D * es


def commit_bytes(w: Workload, accept_nodes: np.ndarray, accept_len: np.ndarray) -> int:
    """Bytes the commit of the accepted paths moves: each K and V row that
    changes place (node n_j != j - 1) read and written once, in every KV head."""
    es = 2 if w.dtype == "bf16" else 4
    moved = sum(int((np.asarray(accept_nodes[b][:int(accept_len[b])]) !=
                     np.arange(int(accept_len[b]))).sum()) for b in range(w.B))
    return 2 * 2 * moved * w.Hkv * w.D * es


def sample_bytes(w: Workload) -> int:
    """Bytes sampling verification reads at least: every logits row once (its
    maximum and normalizer); the gathered candidates and the terminal row's
    second pass are left out."""
    es = 2 if w.dtype == "bf16" else 4
    return w.B * (w.T + 1) * w.V * es


def attention_flops(w: Workload) -> int:
    """4 * T * Hq * (kv_len + T) * D per sequence (QK^T and PV over every key
    position a node could see, counted densely over the tree block)."""
    return int(sum(4 * w.T * w.Hq * (int(n) + w.T) * w.D for n in w.kv_len))
