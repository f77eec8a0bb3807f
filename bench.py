#!/usr/bin/env python3
"""Benchmark of one Progressive Tree Drafting step on one MI355X.

A step = the whole hot path over one batch of synthetic inputs, on one stream:
ptd_tree_attention (one layer; ancestor masks derived in the kernel for trees
of <= 128 nodes, built into the workspace otherwise) -> ptd_topk_argmax ->
ptd_verify_expand (verification and expansion in one launch).  The positions
with rotary embedding of the tree rows (ptd_tree_rope), the commit of the
accepted path (ptd_kv_commit) and sampling verification (ptd_verify_sample)
are timed on their own after the step, on the same inputs, and reported under
"next_rows".  Inputs are seeded synthetic tensors shaped like the
paper's workloads (Llama-2-7B attention shape by default), resident in HBM
before timing starts; R input sets totalling >= 1 GiB are rotated so the
256 MB MALL cannot serve the KV cache from one step to the next.

Prints one JSON line: tree tokens/s (value), us/step, the attention stage's
achieved HBM bandwidth against the 8 TB/s peak, and the CPU oracle's rate on a
bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
DEFAULT_WORKLOAD = "ragged-16"
# measured in the same run and reported as fields of the same line
COMPANION_WORKLOADS = "llama3-8b-long"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--also", default=COMPANION_WORKLOADS,
                    help="comma-separated workloads whose step and attention figures are "
                         "measured after the main one and added to the line ('' for none)")
    ap.add_argument("--plain", action="store_true",
                    help="time only the step and the plain attention call of --workload (no "
                         "next rows, companion workloads, decode shapes or CPU baseline): the "
                         "run that kernel traces and counters are taken on")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the decode-shaped attention calls")
    ap.add_argument("--rotate-bytes", type=float, default=1.0 * 2**30,
                    help="total bytes of rotated input sets (cold-cache timing)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU time of the oracle sample (0 disables)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run only a plain 512 MiB device copy, 5 times: the reference "
                         "kernel whose FETCH_SIZE / WRITE_SIZE counters scale the "
                         "attention kernel's traffic counts")
    return ap.parse_args()


def calibrate_copy():
    import torch
    n = 512 << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n,
                      "launches": 5}), flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    src = os.path.join(ROOT, "paper_2607_10661_amd", "csrc", "tree_attention.hip")
    with open(src, "rb") as f:
        h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(workload, per_launch_alg):
    """HBM bytes per attention launch from committed rocprofv3 --pmc summaries
    (FETCH_SIZE + WRITE_SIZE, scaled by the copy-kernel calibration); None if
    absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_tree_attention_{workload}.json")
    try:
        with open(path) as f:
            d = json.load(f)
    except OSError:
        return None
    if d.get("kernel_source_sha") != kernel_source_hash():
        return None
    return d.get("bytes_per_launch")


def host_cpu():
    """CPU model and the CPUs this process may run on (Linux)."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        cpus = sorted(os.sched_getaffinity(0))
    except AttributeError:
        cpus = list(range(os.cpu_count() or 1))
    ranges, start = [], None
    for i, c in enumerate(cpus):
        if start is None:
            start = c
        if i + 1 == len(cpus) or cpus[i + 1] != c + 1:
            ranges.append(f"{start}-{c}" if c != start else f"{start}")
            start = None
    return model, ",".join(ranges), len(cpus)


def cpu_baseline(args, name, w):
    """The oracle timed on this host: whole steps (ancestor masks, attention
    rows over a thread pool, top-k, verification, expansion) for at least
    --cpu-seconds; and a one-thread rate estimated from a sample of the
    attention rows (every 16th) plus the rest of a step."""
    import concurrent.futures as cf

    import numpy as np

    import oracle as O
    B, T, k = w.B, w.T, w.k
    model, affinity, ncpu = host_cpu()
    nth = max(1, min(16, ncpu))
    rows_all = [(b, h, i) for b in range(B) for h in range(w.Hq) for i in range(T)]
    chunks = [rows_all[j::nth] for j in range(nth)]

    def rows_of(ch):
        return O.attention_rows(w.q, w.k_cache, w.v_cache, w.kv_len, w.parent, w.scale, ch)

    lg_rows = w.logits.reshape(-1, w.V)
    lg_chunks = [lg_rows[j::nth] for j in range(nth)]

    def rest(ex=None):
        if ex is None:
            r_am, r_idx, _ = O.topk(lg_rows, k)
        else:  # logits rows over the pool, reassembled in row order
            parts = list(ex.map(lambda c: O.topk(c, k), lg_chunks))
            r_am = np.empty(lg_rows.shape[0], np.int32)
            r_idx = np.empty((lg_rows.shape[0], k), np.int32)
            for j, (a, ix, _) in enumerate(parts):
                r_am[j::nth] = a
                r_idx[j::nth] = ix
        O.verify(r_am.reshape(B, -1), w.tokens, w.parent)
        O.expand(w.parent, w.tokens, r_idx.reshape(B, T + 1, k), w.width, w.d_max, w.T_max)

    with cf.ThreadPoolExecutor(nth) as ex:
        done, t0 = 0, time.perf_counter()
        while True:
            O.tree_mask(w.parent)
            list(ex.map(rows_of, chunks))
            rest(ex)
            done += 1
            el = time.perf_counter() - t0
            if el >= args.cpu_seconds or el * (done + 1) / done > 3 * args.cpu_seconds:
                break
    sample = rows_all[::16]
    t0 = time.perf_counter()
    O.tree_mask(w.parent)
    rows_of(sample)
    t_rows = time.perf_counter() - t0
    t0 = time.perf_counter()
    rest()
    t_rest = time.perf_counter() - t0
    est = t_rows * len(rows_all) / len(sample) + t_rest
    return {"value": round(B * T * done / el, 3), "unit": "tree tokens/s", "cores": nth,
            "kind": "oracle",
            "sample": f"{done} whole {name} step(s) (all {B * T} nodes x {w.Hq} heads; "
                      f"attention rows and top-k rows over {nth} threads), {el:.1f} s",
            "us_per_step": round(el / done * 1e6, 1),
            "cpu_model": model, "affinity": affinity, "cpus_available": ncpu,
            "single_thread": {"value": round(B * T / est, 3), "unit": "tree tokens/s",
                              "cores": 1,
                              "sample": f"every 16th attention row ({len(sample)} of "
                                        f"{len(rows_all)}, {t_rows:.1f} s, scaled) + top-k, "
                                        f"verify and expand ({t_rest:.2f} s)"}}


def load_mfma(workload):
    """MFMA busy share of the attention kernel from a committed rocprofv3
    counter summary (None if absent or taken on another kernel source)."""
    path = os.path.join(ROOT, "profiles", f"mfma_tree_attention_{workload}.json")
    try:
        with open(path) as f:
            d = json.load(f)
    except OSError:
        return None
    if d.get("kernel_source_sha") != kernel_source_hash():
        return None
    return {k: d[k] for k in ("mfma_util_pct", "kernel", "counters", "file") if k in d}


# Decode-shaped attention calls: (name, B, T, Hq, Hkv, kv_len)
DECODE_SHAPES = [("T1_mha_4096", 1, 1, 32, 32, 4096), ("T1_gqa_32768", 1, 1, 32, 8, 32768),
                 ("T3_gqa_32768", 1, 3, 32, 8, 32768), ("T1_gqa_B16_8192", 16, 1, 32, 8, 8192)]


def decode_calls(args):
    """ptd_tree_attention on decode-sized calls (T = 1 to 3, fewer than 16 query
    rows per KV head), against a device copy of the same key/value bytes
    (each cold: input sets rotated).  The copy moves the bytes twice (read
    and write); its rate is read + write bytes per second."""
    import numpy as np
    import torch

    import paper_2607_10661_amd as P
    import workloads as W
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    out = {}
    for nm, B, T, Hq, Hkv, kvl in DECODE_SHAPES:
        w = W.make_workload(dict(B=B, Hq=Hq, Hkv=Hkv, D=128, kv_len=kvl, T=T, tree="uniform",
                                 V=16, dtype="bf16", plant=None, k=2), seed=3, logits=False)
        def cu(a):
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(
                torch.bfloat16)
        q0, k0, v0 = cu(w.q), cu(w.k_cache), cu(w.v_cache)
        set_b = (q0.numel() + k0.numel() + v0.numel()) * 2
        R = max(2, min(64, math.ceil(args.rotate_bytes / set_b)))
        sets = [(q0, k0, v0)] + [(q0.clone(), k0.clone(), v0.clone()) for _ in range(R - 1)]
        kv_len, parent = cu_i(w.kv_len, dev), cu_i(w.parent, dev)
        shape = P.attn_shape(q0, k0, out_dtype=q0.dtype)
        ws = torch.empty(max(1, P.ptd_tree_attention_workspace_bytes(shape, T)),
                         dtype=torch.uint8, device=dev)
        o = torch.empty_like(q0)
        st = torch.zeros(1, dtype=torch.int32, device=dev)
        n = max(20, args.steps)

        def att(i):
            q, kc, vc = sets[i % R]
            P.ptd_tree_attention(q, kc, vc, kv_len, parent, T, o, shape, None, ws, ws.numel(), st,
                                 sp)
        kv_bytes = 2 * B * Hkv * (kvl + T) * 128 * 2
        dsts = [torch.empty(kv_bytes // 2, dtype=torch.bfloat16, device=dev) for _ in range(2)]
        srcs = [torch.cat([s[1].view(-1)[:kv_bytes // 4], s[2].view(-1)[:kv_bytes // 4]])
                for s in sets[:R]]

        def cp(i):
            dsts[i % 2].copy_(srcs[i % R])
        res = {}
        for fn, key in ((att, "attention"), (cp, "copy")):
            for i in range(5):
                fn(i)
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(20_000_000)
            e0.record(stream)
            for i in range(n):
                fn(i)
            e1.record(stream)
            torch.cuda.synchronize()
            res[key] = e0.elapsed_time(e1) * 1e-3 / n
        assert st.item() == 0, P.ptd_status_string(st.item())
        alg = W.algorithmic_bytes(w)["attention"]
        out[nm] = {"B": B, "T": T, "Hq": Hq, "Hkv": Hkv, "kv_len": kvl,
                   "attention_us": round(res["attention"] * 1e6, 3), "alg_bytes": alg,
                   "attention_GBps": round(alg / res["attention"] / 1e9, 1),
                   "copy_us": round(res["copy"] * 1e6, 3),
                   "copy_GBps": round(2 * kv_bytes / res["copy"] / 1e9, 1)}
        del sets, srcs, dsts
        torch.cuda.empty_cache()
    return out


def cu_i(a, dev):
    import numpy as np
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)



def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    line = run(args, args.workload, "plain" if args.plain else "full")
    if not args.plain:
        for wl in [x for x in args.also.split(",") if x and x != args.workload]:
            line[wl] = run(args, wl, "companion")
        if not args.no_decode:
            line["decode"] = decode_calls(args)
    print(json.dumps(line), flush=True)


def run(args, name, mode):
    """Measure one workload.  mode "full": the step, the attention call, every
    next row and the CPU baseline; "plain": the step and the attention call
    only; "companion": the same, returned as a field of the main line."""

    import numpy as np
    import torch

    import paper_2607_10661_amd as P
    import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = W.make_workload(name)
    B, T, k = w.B, w.T, w.k

    def cu(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    base = dict(q=cu(w.q), k=cu(w.k_cache), v=cu(w.v_cache), logits=cu(w.logits))
    set_bytes = sum(t.numel() * t.element_size() for t in base.values())
    R = max(1, min(64, math.ceil(args.rotate_bytes / set_bytes)))
    sets = [base] + [{n: t.clone() for n, t in base.items()} for _ in range(R - 1)]
    parent, tokens, kv_len = cu(w.parent), cu(w.tokens), cu(w.kv_len)

    shape = P.attn_shape(base["q"], base["k"], out_dtype=base["q"].dtype)
    ws_attn = torch.empty(max(1, P.ptd_tree_attention_workspace_bytes(shape, T)),
                          dtype=torch.uint8, device=dev)
    R_rows = B * (T + 1)
    ws_topk = torch.empty(max(1, P.ptd_topk_workspace_bytes(R_rows, w.V, k)),
                          dtype=torch.uint8, device=dev)
    out = torch.empty_like(base["q"])
    am = torch.empty(R_rows, dtype=torch.int32, device=dev)
    tidx = torch.empty((R_rows, k), dtype=torch.int32, device=dev)
    tval = torch.empty((R_rows, k), dtype=torch.float32, device=dev)
    al = torch.empty(B, dtype=torch.int32, device=dev)
    an = torch.empty((B, T), dtype=torch.int32, device=dev)
    ot = torch.empty((B, T + 1), dtype=torch.int32, device=dev)
    pn = torch.empty((B, w.T_max), dtype=torch.int32, device=dev)
    tn = torch.empty((B, w.T_max), dtype=torch.int32, device=dev)
    ln = torch.empty(B, dtype=torch.int32, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    dt_code = P.PTD_BF16 if w.dtype == "bf16" else P.PTD_F32

    def attention(i):
        s = sets[i % R]
        P.ptd_tree_attention(s["q"], s["k"], s["v"], kv_len, parent, T, out, shape, None,
                             ws_attn, ws_attn.numel(), status, sp)

    def step(i):
        s = sets[i % R]
        attention(i)
        P.ptd_topk_argmax(s["logits"], dt_code, R_rows, w.V, w.V, k, am, tidx, tval,
                          ws_topk, ws_topk.numel(), sp)
        P.ptd_verify_expand(am, tokens, parent, None, B, T, tidx, k, w.width, w.d_max, w.T_max,
                            al, an, ot, pn, tn, ln, status, sp)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    assert status.item() == 0, P.ptd_status_string(status.item())
    assert al.cpu().tolist() == w.planted_depth.tolist(), "accepted length mismatch"

    def timed(fn, n):
        """Back-to-back GPU time of n calls of fn on the launch stream.  A GPU
        spin kernel is queued first so the host enqueues all n calls before the
        GPU reaches them: the region measures GPU execution, not Python launch
        speed."""
        torch.cuda.synchronize()
        h0 = time.perf_counter()
        for i in range(min(n, 10)):
            fn(args.warmup + i)
        host_s = (time.perf_counter() - h0) / min(n, 10)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        if hasattr(torch.cuda, "_sleep"):
            torch.cuda._sleep(int(host_s * n * 1.5 * 2.5e9) + 10_000_000)
        e0.record(stream)
        for i in range(n):
            fn(args.warmup + i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n, host_s

    K = args.steps
    ms_step, host_step_s = timed(step, K)
    assert status.item() == 0, P.ptd_status_string(status.item())
    # the roofline's kernel: ptd_tree_attention alone, back to back, same inputs
    att_ms, _ = timed(attention, K)
    att_avg_s = att_ms * 1e-3
    alg = W.algorithmic_bytes(w)
    achieved = alg["attention"] / att_avg_s / 1e9
    flops = W.attention_flops(w)
    tokens_per_s = B * T / (ms_step * 1e-3)
    traffic = load_traffic(name, alg["attention"])
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                "kernel": "ptd_tree_attention (k_attn_mfma + k_attn_combine)",
                "alg_bytes_per_launch": alg["attention"],
                "basis": "algorithmic bytes of one call / average duration of %d back-to-back "
                         "calls (HIP events on the launch stream); the kernel trace of "
                         "bench.py --plain gives the two kernels' average durations, whose "
                         "sum is this duration" % K}
    config = {"workload": name, "B": B, "T": T, "Hq": w.Hq, "Hkv": w.Hkv, "D": w.D,
              "kv_len": int(w.kv_len.max()) if B == 1 else w.kv_len.tolist(), "V": w.V, "k": k}
    if mode != "full":
        torch.cuda.synchronize()
        res = {"config": config, "us_per_step": round(ms_step * 1e3, 3),
               "tree_tokens_per_s": round(tokens_per_s, 1),
               "attention_us": round(att_avg_s * 1e6, 3),
               "attention_TBps": round(achieved / 1000, 3), "roofline": roofline,
               "mfma_counters": load_mfma(name)}
        del sets, base
        torch.cuda.empty_cache()
        return res

    # ptd_tree_rope and ptd_kv_commit on their own, after the step timings:
    # the rope turns q and the tree key rows of the rotated sets in place, the
    # commit moves the accepted rows (kv_len is not advanced, so every call
    # moves the same rows).  Neither changes the bytes a later call moves.
    acc_len = al.clone()
    acc_nodes = an.clone()
    kv_next = torch.empty_like(kv_len)
    rope_shape = P.AttnShape(B, w.Hq, w.Hkv, w.D, w.L_cap, shape.in_dtype, shape.in_dtype, 0.0)
    theta = 10000.0

    def rope(i):
        s = sets[i % R]
        P.ptd_tree_rope(s["q"], s["k"], kv_len, parent, T, rope_shape, theta, None,
                        P.PTD_ROPE_HALF, None, status, sp)

    def commit(i):
        s = sets[i % R]
        P.ptd_kv_commit(s["k"], s["v"], kv_len, acc_len, acc_nodes, T, rope_shape, kv_next,
                        status, sp)

    # sampling verification of the same trees and logits, uniforms drawn once
    g = torch.Generator(device="cpu").manual_seed(1234)
    u_node = torch.rand((B, T), generator=g, dtype=torch.float64).to(dev)
    u_bonus = torch.rand((B, T + 1), generator=g, dtype=torch.float64).to(dev)
    ws_samp = torch.empty(max(1, P.ptd_verify_sample_workspace_bytes(B, T, w.V)), dtype=torch.uint8,
                          device=dev)
    s_al = torch.empty(B, dtype=torch.int32, device=dev)
    s_an = torch.empty((B, T), dtype=torch.int32, device=dev)
    s_ot = torch.empty((B, T + 1), dtype=torch.int32, device=dev)

    def sample(i):
        s = sets[i % R]
        P.ptd_verify_sample(s["logits"], dt_code, w.V, w.V, tokens, parent, None, B, T, 1.0,
                            u_node, u_bonus, s_al, s_an, s_ot, ws_samp, ws_samp.numel(), status,
                            sp)

    # stepping of the expanded tree, its merge into a candidate pool, and the
    # retrieval of the next candidate tree by the bonus token
    d_prune = max(1, w.d_max - 1)
    sp_pn = torch.empty((B, w.T_max), dtype=torch.int32, device=dev)
    sp_tn = torch.empty((B, w.T_max), dtype=torch.int32, device=dev)
    sp_ln = torch.empty(B, dtype=torch.int32, device=dev)
    pool_e, pool_n = 2048, w.T_max + 1  # a retrieved tree can fill the draft
    pool_bytes = P.ptd_pool_bytes(B, pool_e, pool_n)
    pool = torch.empty(pool_bytes, dtype=torch.uint8, device=dev)
    P.ptd_pool_init(pool, pool_bytes, B, pool_e, pool_n, stream=sp)
    bonus = torch.gather(ot, 1, al.long().view(B, 1)).view(B).contiguous()
    rt_pn = torch.empty((B, w.T_max), dtype=torch.int32, device=dev)
    rt_tn = torch.empty((B, w.T_max), dtype=torch.int32, device=dev)
    rt_ln = torch.empty(B, dtype=torch.int32, device=dev)

    def prune(i):
        P.ptd_step_prune(pn, tn, ln, B, w.T_max, d_prune, w.T_max, sp_pn, sp_tn, sp_ln, status, sp)

    def merge(i):
        P.ptd_pool_merge(pool, pool_bytes, B, pool_e, pool_n, pn, tn, ln, w.T_max, status, sp)

    def retrieve(i):
        P.ptd_pool_retrieve(pool, pool_bytes, B, pool_e, pool_n, bonus, w.T_max, rt_pn, rt_tn,
                            rt_ln, sp)

    # attention on paged caches: 64-row pages scattered through a random page
    # table (one table for all rotated sets), same inputs otherwise
    PS = 64
    paged_ms = None
    if w.dtype == "bf16" and w.L_cap % PS == 0:
        maxp = w.L_cap // PS
        num_pages = B * maxp
        gtab = torch.Generator(device="cpu").manual_seed(99)
        table = torch.randperm(num_pages, generator=gtab).to(torch.int32).view(B, maxp).to(dev)

        def paginate(c):
            pages = torch.empty((num_pages, w.Hkv, PS, w.D), dtype=c.dtype, device=dev)
            pages[table.view(-1).long()] = (c.view(B, w.Hkv, maxp, PS, w.D).permute(0, 2, 1, 3, 4)
                                            .reshape(B * maxp, w.Hkv, PS, w.D))
            return pages

        paged_sets = [(paginate(st_["k"]), paginate(st_["v"])) for st_ in sets]
        kvps = [P.KVPages(kp.data_ptr(), vp.data_ptr(), table.data_ptr(), PS, maxp, num_pages)
                for kp, vp in paged_sets]

        def attention_paged(i):
            s = sets[i % R]
            P.ptd_tree_attention_paged(s["q"], kvps[i % R], kv_len, None, parent, T, out, shape, None,
                                       ws_attn, ws_attn.numel(), status, sp)

        paged_ms, _ = timed(attention_paged, K)

    # a padded batch of trees of different sizes: per-sequence tree sizes drawn
    # uniformly from 1..T (seeded), the rest of each sequence's T slots padding
    gtl = torch.Generator(device="cpu").manual_seed(98)
    tree_len_r = torch.randint(1, T + 1, (B,), generator=gtl, dtype=torch.int32)
    tree_len_d = tree_len_r.to(dev)

    def attention_ragged(i):
        s = sets[i % R]
        P.ptd_tree_attention_ragged(s["q"], s["k"], s["v"], kv_len, tree_len_d, parent, T, out,
                                    shape, None, ws_attn, ws_attn.numel(), status, sp)

    ragged_ms, _ = timed(attention_ragged, K)

    # 8-bit (E4M3) key/value caches with one scale per KV head, quantized on
    # the GPU from each rotated set before timing (D = 128, bf16 queries)
    fp8_ms = None
    if w.dtype == "bf16" and w.D == 128:
        def quant(c):
            amax = c.float().abs().amax(dim=(0, 2, 3)).clamp_min(1e-30)
            sc = (amax / 448.0).contiguous()
            codes = (c.float() / sc[None, :, None, None]).to(torch.float8_e4m3fn)
            return codes.view(torch.uint8).contiguous(), sc

        fp8_sets = []
        for st_ in sets:
            kq, ksc = quant(st_["k"])
            vq, vsc = quant(st_["v"])
            fp8_sets.append((kq, vq, ksc, vsc))

        def attention_fp8(i):
            s = sets[i % R]
            kq, vq, ksc, vsc = fp8_sets[i % R]
            P.ptd_tree_attention_fp8kv(s["q"], kq, vq, ksc, vsc, kv_len, None, parent, T, out,
                                       shape, ws_attn, ws_attn.numel(), status, sp)

        fp8_ms, _ = timed(attention_fp8, K)
    sample_ms, _ = timed(sample, K)
    prune_ms, _ = timed(prune, K)
    merge_ms, _ = timed(merge, K)
    retrieve_ms, _ = timed(retrieve, K)
    rope_ms, _ = timed(rope, K)
    commit_ms, _ = timed(commit, K)
    torch.cuda.synchronize()
    assert status.item() == 0, P.ptd_status_string(status.item())
    rope_b = W.rope_bytes(w)
    commit_b = W.commit_bytes(w, acc_nodes.cpu().numpy(), acc_len.cpu().numpy())

    def next_row(ms, nbytes, what):
        gbps = nbytes / (ms * 1e-3) / 1e9
        return {"us": round(ms * 1e3, 3), "alg_bytes": nbytes, "GBps": round(gbps, 1),
                "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4), "what": what}

    # CPU oracle on a bounded sample of the same workload: whole steps
    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(args, name, w)

    line = {
        "metric": "tree tokens/s (tree-attn + top-k + verify + expand step)",
        "value": round(tokens_per_s, 1),
        "unit": "tree tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6),
        "us_per_step": round(ms_step * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded), cold cache: %d rotated input sets" % R,
        "config": config,
        "attention_us": round(att_avg_s * 1e6, 3),
        "host_enqueue_us_per_step": round(host_step_s * 1e6, 1),
        "attention_timing": "ptd_tree_attention alone, %d back-to-back calls on the launch stream "
                            "(HIP events)" % K,
        "attention_TBps": round(achieved / 1000, 3),
        "attention_dense_flops_frac": round(flops / att_avg_s / 2.5e15, 4),
        "attention_dense_flops_note": "4*T*Hq*(kv_len+T)*D per sequence (tree block counted "
                                      "densely) / attention_us / 2.5 PFLOP/s; the MFMA busy "
                                      "counter is under mfma_counters",
        "mfma_counters": load_mfma(name),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "next_rows": {
            "tree_rope": next_row(rope_ms, rope_b, "ptd_tree_rope: positions kv_len+|pi(i)|-1, "
                                  "rotary embedding of q and the tree key rows (theta 1e4, "
                                  "half pairing), %d back-to-back calls" % K),
            "kv_commit": next_row(commit_ms, commit_b, "ptd_kv_commit of the accepted paths "
                                  "(accept_len %s), %d back-to-back calls"
                                  % (acc_len.cpu().tolist(), K)),
            "verify_sample": next_row(sample_ms, W.sample_bytes(w), "ptd_verify_sample at "
                                      "temperature 1 (row statistics of all %d logits rows + "
                                      "walk + bonus draw), %d back-to-back calls"
                                      % (B * (T + 1), K)),
        },
    }
    line["next_rows"]["ragged_attention"] = next_row(
        ragged_ms, W.ragged_attention_bytes(w, tree_len_r.numpy()),
        "ptd_tree_attention_ragged: per-sequence tree sizes %s of T = %d slots, %d back-to-back "
        "calls" % (tree_len_r.tolist() if B <= 16 else "1..%d" % T, T, K))
    if fp8_ms is not None:
        line["next_rows"]["fp8kv_attention"] = next_row(
            fp8_ms, W.fp8kv_attention_bytes(w), "ptd_tree_attention_fp8kv: the attention call "
            "on E4M3 key/value caches (one scale per KV head), %d back-to-back calls; bf16 "
            "caches: %.3f us" % (K, att_avg_s * 1e6))
    if paged_ms is not None:
        line["next_rows"]["paged_attention"] = next_row(
            paged_ms, alg["attention"], "ptd_tree_attention_paged: the attention call on %d-row "
            "pages through a random page table (%d pages), %d back-to-back calls; contiguous: "
            "%.3f us" % (PS, num_pages, K, att_avg_s * 1e6))
    tree_b = B * w.T_max * 4 * 2
    line["next_rows"].update({
        "step_prune": next_row(prune_ms, 2 * tree_b, "ptd_step_prune of the expanded trees "
                               "(T_max %d) at d_max %d, %d back-to-back calls"
                               % (w.T_max, d_prune, K)),
        "pool_merge": next_row(merge_ms, tree_b, "ptd_pool_merge of the expanded trees into "
                               "a pool of %d trees x %d nodes per sequence (first call grows "
                               "it, later calls find every node), %d back-to-back calls"
                               % (pool_e, pool_n, K)),
        "pool_retrieve": next_row(retrieve_ms, tree_b, "ptd_pool_retrieve of the candidate "
                                  "trees keyed by the bonus tokens, %d back-to-back calls" % K),
    })
    del sets, base
    torch.cuda.empty_cache()
    return line


if __name__ == "__main__":
    main()
