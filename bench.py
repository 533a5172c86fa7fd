#!/usr/bin/env python3
"""Verify-step benchmark on one MI355X.

One step = the whole verify hot path at one verifier level for one batch:
verification attention, then accept-and-diverge with the rollback applied by
its finishing kernel (two C-ABI calls on one stream:
specrouter_verify_attention, specrouter_accept_and_rollback). The standalone
rollback call is timed on its own as well. `value` comes from K steps timed
with events at the two ends only; each entry point's average duration (and
the roofline) from K back-to-back calls of that entry point alone, again with
events at the two ends only. Inputs are seeded synthetic data of the named
workload and are resident in HBM before timing starts. To keep the 256 MB
last-level cache from serving repeated steps, R copies of the inputs live at
different HBM addresses and step s uses copy s mod R. Every step rolls back a
fresh copy of the cache lengths and validity mask (staged before the timed
region), so the fused rollback clears the rejected rows on every step.

Default workload: the ragged 256-sequence batch (B = 256, bf16 logits), the
largest single-GPU configuration; --config 2 is the Llama-3-8B-shaped
16-sequence batch, --config 3 the three-level chain.

Prints ONE JSON line (rank 0) with the throughput in verified draft tokens/s,
the roofline of the dominant kernel (HIP events over the timed region), and
the CPU reference timed on a bounded sample of the same workload.

  python bench.py [--steps K] [--warmup W] [--config 2|5|...] [--no-cpu]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

PEAK_HBM_GBS = 8000.0
PROFILE_COUNTERS = os.path.join(HERE, "profiles", "counters.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--rotate", type=int, default=0, help="input copies (0 = enough to exceed 1 GB)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-seqs", type=int, default=0, help="sequences in the CPU-baseline sample")
    return ap.parse_args()


# Sources whose kernels each entry point launches: HBM byte counters taken
# for an older version of them no longer describe the code that runs.
KERNEL_SOURCES = {
    "verify_attention": ["attention.hip", "sr_internal.h"],
    "accept_and_diverge": ["accept.hip", "sr_internal.h"],
    "rollback": ["rollback.hip", "sr_internal.h"],
    "accept_filter": ["accept.hip", "filter.inc", "sr_internal.h"],
}


def kernel_source_hash(entry):
    h = hashlib.sha256()
    for n in KERNEL_SOURCES[entry]:
        with open(os.path.join(HERE, "paper_2505_07680_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def calibration_copy(dev):
    """A device copy of known size (256 MiB), made right before the first
    verify-step kernel: profile_bench.py scales the rocprofv3 HBM byte
    counters by what they read for the last copy before that kernel."""
    import torch

    src = torch.empty(256 << 20, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()


def hbm_probe(sr, dev, ev, gib=1, copies=3, reps=9):
    """Read bandwidth of the library's streaming-read probe and copy
    bandwidth (bytes read + written, a device copy) over `copies` rotated
    buffers of `gib` GiB each, so neither the 256 MB Infinity Cache nor the
    L2s serve the repeats: the practical ceiling the kernels are compared
    with."""
    import torch

    n = (gib << 30) // 4
    bufs = [torch.full((n,), 1.0, dtype=torch.float32, device=dev) for _ in range(copies)]
    dst = torch.empty(n, dtype=torch.float32, device=dev)
    out = {}
    for name, fn, bytes_per in (("read", lambda x: sr.specrouter_hbm_read_probe(x), n * 4),
                                ("copy", lambda x: dst.copy_(x), 2 * n * 4)):
        for i in range(copies):
            fn(bufs[i])
        torch.cuda.synchronize()
        e0, e1 = ev(), ev()
        e0.record()
        for i in range(reps):
            fn(bufs[i % copies])
        e1.record()
        torch.cuda.synchronize()
        out[f"{name}_GB/s"] = round(reps * bytes_per / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    del bufs, dst
    torch.cuda.empty_cache()
    out["note"] = (f"specrouter_hbm_read_probe and a device copy over {copies} rotated {gib} GiB buffers "
                   "(HIP events)")
    return out


def measured_traffic(entry, workload):
    """HBM bytes per call from the rocprofv3 FETCH_SIZE + WRITE_SIZE passes
    (calibrated against a copy of known size), or None when they were taken
    for other sources or not at all."""
    try:
        with open(PROFILE_COUNTERS) as f:
            ent = json.load(f).get(entry, {}).get(workload)
    except (OSError, ValueError):
        return None
    if not ent or ent.get("source_hash") != kernel_source_hash(entry):
        return None
    return ent.get("bytes_per_call")


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: this implementation runs on exactly one GPU (the verify step shards by sequence with "
              "no cross-GPU exchange). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2505_07680_amd as sr
    from workloads import CONFIGS, level_inputs

    sr.load()
    if not torch.cuda.is_available():
        print("bench.py: no HIP device visible", file=sys.stderr)
        sys.exit(3)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    shape = CONFIGS[args.config]
    if not hasattr(shape, "gmax"):
        chain_bench(args, sr, shape)
        return
    t0 = time.time()
    inp = level_inputs(shape)
    gen_s = time.time() - t0

    B, G1, Hq, D = inp.q.shape
    gmax = G1 - 1
    Hkv, cap = inp.k.shape[1], inp.k.shape[2]
    V = inp.p_logits.shape[2]
    code = sr.SR_BF16 if shape.logits == "bf16" else sr.SR_F32
    esz = 2 if code == sr.SR_BF16 else 4

    def up(x):
        x = np.ascontiguousarray(x)
        if x.dtype == np.uint16:
            x = x.view(np.int16)
        return torch.from_numpy(x).to(dev)

    # bytes the method must move per step (algorithmic): each entry point's
    # compulsory HBM reads and writes
    kv_len = inp.kv_len.astype(np.int64)
    gam = inp.gamma.astype(np.int64)
    att_bytes = int((2 * Hkv * kv_len * D * 2).sum()          # K and V rows below kv_len (bf16)
                    + ((gam + 1) * Hq * D * 2).sum()           # live query rows (bf16)
                    + ((gam + 1) * Hq * D * 4).sum()           # live output rows (fp32)
                    + kv_len.sum())                            # cache-mask bytes
    acc_bytes = int(((2 * gam + 1) * V * esz).sum())           # live verifier and draft logit rows
    set_bytes = inp.k.nbytes + inp.v.nbytes + inp.p_logits.nbytes + inp.q_logits.nbytes
    R = args.rotate or max(2, int(np.ceil(1.2e9 / set_bytes)))

    sets = []
    base_mask = np.zeros((B, cap), np.uint8)
    for b in range(B):
        base_mask[b, : inp.kv_len[b]] = 1
    for r in range(R):
        s = dict(
            q=up(inp.q), k=up(inp.k), v=up(inp.v), kv_in=up(inp.kv_len),
            gamma=up(inp.gamma), mask_in=up(base_mask),
            p=up(inp.p_logits), ql=up(inp.q_logits), drafts=up(inp.drafts),
            u_acc=up(inp.u_acc), u_res=up(inp.u_res),
            out=torch.empty((B, G1, Hq, D), dtype=torch.float32, device=dev),
            ws=sr.attention_workspace(B, gmax, Hq, Hkv, D, cap, device=dev),
            acc=sr.AcceptBuffers(B, gmax, V, code, device=dev),
            phys=torch.zeros(1, dtype=torch.int32, device=dev),
            st=torch.zeros(1, dtype=torch.int32, device=dev),
        )
        sets.append(s)


    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    K = args.steps
    # One fresh (cache lengths, validity mask) pair per rolled-back call, so
    # every timed call's rollback clears the rejected rows; refilled from the
    # pristine state outside the timed regions.
    n_work = max(K, args.warmup, 1)
    work = [(torch.empty(B, dtype=torch.int32, device=dev), torch.empty((B, cap), dtype=torch.uint8, device=dev))
            for _ in range(n_work)]

    def refill():
        for kw, mw in work:
            kw.copy_(sets[0]["kv_in"])
            mw.copy_(sets[0]["mask_in"])
        torch.cuda.synchronize()

    def attention(s):
        sr.specrouter_verify_attention(s["q"], s["k"], s["v"], s["mask_in"], s["kv_in"], s["gamma"],
                                       s["out"], inp.scale, s["ws"], s["st"])

    def accept(s, w):
        a = s["acc"]
        sr.specrouter_accept_and_rollback(s["p"], s["ql"], s["drafts"], s["gamma"], s["u_acc"], s["u_res"],
                                          s["kv_in"], a.accept_len, a.out_tokens, a.new_len, a.accept_prob,
                                          a.p_tok, a.q_tok, a.kl, a.tv, w[0], w[1], s["phys"], a.workspace, s["st"])

    def step(s, w):
        attention(s)
        accept(s, w)

    refill()
    calibration_copy(dev)
    for i in range(args.warmup):
        step(sets[i % R], work[i % n_work])
    refill()

    def timed(fn):
        """ms for K calls of fn(i), events at the two ends only."""
        e0, e1 = ev(), ev()
        torch.cuda.synchronize()
        e0.record()
        for i in range(K):
            fn(i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    # Timed region 1 (the metric): K whole steps.
    t_wall = time.perf_counter()
    total_ms = timed(lambda i: step(sets[i % R], work[i]))
    wall = time.perf_counter() - t_wall
    # Each entry point's average duration (the roofline): K back-to-back calls
    # of it alone on the same rotated inputs.
    att_ms = timed(lambda i: attention(sets[i % R])) / K
    refill()
    acc_ms = timed(lambda i: accept(sets[i % R], work[i])) / K
    # the mask bytes the rollback clears: the rejected rows of every sequence
    acc_k = sets[0]["acc"].accept_len.cpu().numpy().astype(np.int64)
    rb_bytes = int(B * 12 + (gam - np.maximum(acc_k, 0)).sum())

    status = int(sum(int(s["st"].item()) for s in sets))
    acc0 = sets[0]["acc"]
    mean_accept = float(acc0.accept_len.float().mean().item())
    drafts_per_step = int(gam.sum())
    ms_per_step = total_ms / K
    value = drafts_per_step * K / (total_ms / 1e3)

    att_gbs = att_bytes / (att_ms / 1e3) / 1e9
    acc_gbs = (acc_bytes + rb_bytes) / (acc_ms / 1e3) / 1e9
    # the roofline is reported for the entry point that takes the longest
    dominant = "verify_attention" if att_ms >= acc_ms else "accept_and_rollback"
    dom_bytes, dom_ms = (att_bytes, att_ms) if dominant == "verify_attention" else (acc_bytes + rb_bytes, acc_ms)
    dom_gbs = dom_bytes / (dom_ms / 1e3) / 1e9
    roofline = {
        "bound": "hbm", "kernel": "specrouter_" + dominant,
        "achieved": round(dom_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
        "frac": round(dom_gbs / PEAK_HBM_GBS, 4),
        "traffic": measured_traffic("verify_attention" if dominant == "verify_attention" else "accept_and_diverge",
                                    shape.name),
        "algorithmic_bytes": dom_bytes, "avg_launch_us": round(dom_ms * 1e3, 2),
    }

    # sampling variants of the accept call on the same inputs (greedy drafts
    # are the workload's drafts; only the timing is reported)
    variants = {}
    for T, tk, tp in ((0.0, 0, 1.0), (0.7, 0, 1.0), (0.7, 50, 1.0), (0.7, 0, 0.9), (0.7, 50, 0.9)):
        for i in range(args.warmup):
            s = sets[i % R]
            a = s["acc"]
            sr.specrouter_accept_and_diverge_sampled(
                s["p"], s["ql"], s["drafts"], s["gamma"], s["u_acc"], s["u_res"], s["kv_in"], a.accept_len,
                a.out_tokens, a.new_len, a.accept_prob, a.p_tok, a.q_tok, a.kl, a.tv, a.workspace, s["st"],
                temperature=T, top_k=tk, top_p=tp)
        e0, e1 = ev(), ev()
        torch.cuda.synchronize()
        e0.record()
        for i in range(K):
            s = sets[i % R]
            a = s["acc"]
            sr.specrouter_accept_and_diverge_sampled(
                s["p"], s["ql"], s["drafts"], s["gamma"], s["u_acc"], s["u_res"], s["kv_in"], a.accept_len,
                a.out_tokens, a.new_len, a.accept_prob, a.p_tok, a.q_tok, a.kl, a.tv, a.workspace, s["st"],
                temperature=T, top_k=tk, top_p=tp)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / K * 1e3
        name = "accept_greedy" if T == 0 else f"accept_temperature_{T}"
        name += (f"_top_k_{tk}" if tk else "") + (f"_top_p_{tp}" if tp < 1 else "")
        variants[name] = {"us": round(us, 2), "GB/s": round(acc_bytes / us / 1e3, 1)}
    # chain glue between two verifier levels (window of a gamma-4 upper level
    # and the consensus), on this step's accept outputs as the lower level
    s = sets[0]
    a = s["acc"]
    cap4 = 4
    g_n = torch.empty(B, dtype=torch.int32, device=dev)
    d_n = torch.empty((B, cap4), dtype=torch.int32, device=dev)
    kv_n = torch.empty(B, dtype=torch.int32, device=dev)
    ctx_n = (s["kv_in"] - s["gamma"] - 1).contiguous()
    lu, ll = torch.empty_like(g_n), torch.empty_like(g_n)
    pend, npend = torch.empty((B, 2), dtype=torch.int32, device=dev), torch.empty_like(g_n)
    ku = torch.zeros(B, dtype=torch.int32, device=dev)
    ou = torch.zeros((B, cap4 + 1), dtype=torch.int32, device=dev)
    def graph_us(fn, n=50):
        """GPU time per call of a short launch sequence, replayed from a HIP
        graph (the host's enqueue time is not part of it)."""
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(n):
                fn()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = ev(), ev()
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n * 1e3

    glue = {
        "window_us": round(graph_us(lambda: sr.specrouter_chain_window(a.accept_len, a.out_tokens, cap4, g_n, d_n,
                                                                       ctx_len=ctx_n, kv_len_next=kv_n)), 2),
        "consensus_us": round(graph_us(lambda: sr.specrouter_chain_consensus(ctx_n, a.accept_len, a.out_tokens, ku,
                                                                             ou, lu, ll, pend, npend, s["st"])), 2),
        "note": "GPU time per call (HIP graph replay)",
    }
    variants["chain_glue"] = glue
    # the standalone entry points the step fuses: rollback alone (graph
    # replay) and accept-and-diverge alone (HIP events)
    kv_rb, mask_rb = s["kv_in"].clone(), s["mask_in"].clone()  # new_len <= kv_in: a pure rollback
    rb_us = graph_us(lambda: sr.specrouter_rollback(kv_rb, mask_rb, a.new_len, s["phys"], s["st"]))
    e0, e1 = ev(), ev()
    torch.cuda.synchronize()
    e0.record()
    for i in range(K):
        s2 = sets[i % R]
        a2 = s2["acc"]
        sr.specrouter_accept_and_diverge(s2["p"], s2["ql"], s2["drafts"], s2["gamma"], s2["u_acc"], s2["u_res"],
                                         s2["kv_in"], a2.accept_len, a2.out_tokens, a2.new_len, a2.accept_prob,
                                         a2.p_tok, a2.q_tok, a2.kl, a2.tv, a2.workspace, s2["st"])
    e1.record()
    torch.cuda.synchronize()
    acc_only_us = e0.elapsed_time(e1) / K * 1e3
    variants["accept_alone"] = {"us": round(acc_only_us, 2), "GB/s": round(acc_bytes / acc_only_us / 1e3, 1),
                                "note": "specrouter_accept_and_diverge without the rollback"}

    # KV-cache state: append this step's rows (per-sequence cursors) and
    # compact a cache with 2% holes, on scratch caches of the workload's shape
    kc = torch.empty_like(sets[0]["k"])
    vc = torch.empty_like(sets[0]["v"])
    kn = torch.empty((B, G1, Hkv, D), dtype=torch.int16, device=dev).random_(-(1 << 14), 1 << 14)
    vn = torch.empty_like(kn)
    ctx_len = (s["kv_in"] - s["gamma"] - 1).contiguous()
    kvw = ctx_len.clone()
    mk = s["mask_in"].clone()
    def append_once():
        kvw.copy_(ctx_len)
        sr.specrouter_kv_append(kn, vn, s["gamma"], kc, vc, mk, kvw, status=s["st"])

    app_us = graph_us(append_once) - graph_us(lambda: kvw.copy_(ctx_len))
    holes = torch.rand((B, cap), device=dev) < 0.02
    mask_h = (s["mask_in"].bool() & ~holes).to(torch.uint8)
    first = [int(np.argmax(~(mask_h[b, : inp.kv_len[b]].cpu().numpy().astype(bool)))) for b in range(B)]
    moved = int(sum(int(inp.kv_len[b]) - first[b] for b in range(B)))  # rows from the first hole on (upper bound)
    comp_ms = []
    for i in range(max(3, K // 20)):
        mk.copy_(mask_h)
        kvw.copy_(s["kv_in"])
        c0, c1 = ev(), ev()
        c0.record()
        sr.specrouter_kv_compact(kc, vc, mk, kvw, s["st"])
        c1.record()
        torch.cuda.synchronize()
        comp_ms.append(c0.elapsed_time(c1))
    comp_us = float(np.median(comp_ms)) * 1e3
    comp_bytes = moved * Hkv * D * 2 * 2 * 2  # K and V rows, read and written
    variants["kv_state"] = {
        "append_us": round(app_us, 2), "append_bytes": int(B * G1 * Hkv * D * 2 * 2 * 2),
        "compact_us": round(comp_us, 2), "compact_GB/s": round(comp_bytes / comp_us / 1e3, 1),
        "compact_note": "2% random holes; bytes = rows from each sequence's first hole, read and written",
    }
    status |= int(sum(int(s["st"].item()) for s in sets))

    cpu = None
    boundary = None
    if not args.no_cpu:
        cpu = cpu_baseline(inp, args.cpu_seqs)
        boundary = boundary_check(inp, acc0)
    sched = scheduler_timing(sr, sets[0]["gamma"], acc0.accept_len, acc0.tv)
    probe = hbm_probe(sr, dev, ev)

    line = {
        "metric": "verified draft tokens/s per verify step; HBM GB/s (KV + logits) vs MI355X peak",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 KV / fp32 logits" if code == sr.SR_F32 else "bf16 KV / bf16 logits",
        "data": "synthetic (seeded Philox; Q,K,V ~ N(0,1) bf16; logits N(0,9) + draft noise)",
        "config": {
            "workload": f"{shape.name}: {shape.note}",
            "B": B, "gamma": int(gam.max()), "heads": f"{Hq}/{Hkv}", "head_dim": D,
            "cache_len": int(kv_len.max()), "vocab": V, "input_copies": R,
            "parallelism": "single GPU",
        },
        "roofline": roofline,
        "kernels": {
            "verify_attention": {"us": round(att_ms * 1e3, 2), "GB/s": round(att_gbs, 1),
                                 "frac": round(att_gbs / PEAK_HBM_GBS, 4),
                                 "frac_of_probe": round(att_gbs / probe["read_GB/s"], 4), "algorithmic_bytes": att_bytes,
                                 "traffic": measured_traffic("verify_attention", shape.name)},
            "accept_and_rollback": {"us": round(acc_ms * 1e3, 2), "GB/s": round(acc_gbs, 1),
                                    "frac": round(acc_gbs / PEAK_HBM_GBS, 4),
                                    "frac_of_probe": round(acc_gbs / probe["read_GB/s"], 4),
                                    "algorithmic_bytes": acc_bytes + rb_bytes,
                                    "traffic": measured_traffic("accept_and_diverge", shape.name),
                                    "note": "accept-and-diverge with the rollback done by its finish kernel"},
            "rollback": {"us": round(rb_us, 2), "algorithmic_bytes": rb_bytes,
                         "note": "the standalone rollback call (not part of the step), HIP graph replay"},
        },
        "hbm_probe": probe,
        "sampling_variants": variants,
        "mean_accept_len": round(mean_accept, 3),
        "status_bits": status,
        "boundary": boundary,
        "cpu_baseline": cpu,
        "scheduler": sched,
        "host_wall_s": round(wall, 4),
        "input_gen_s": round(gen_s, 2),
    }
    print(json.dumps(line), flush=True)


def chain_bench(args, sr, shape):
    """One step of the three-level chain (draft -> intermediate -> target),
    all on the device: the intermediate level's attention and accept, the
    target's draft window (the first min(k + 1, gamma_tgt) tokens the
    intermediate level emitted), the target level's attention and accept
    (its draft rows are the intermediate level's verifier rows, a strided
    view), the consensus and both levels' rollbacks. The draft level's
    decode attention (gamma = 0, once per drafted token) is timed apart.
    The step's working set is far above the 256 MB Infinity Cache, so the
    inputs are not rotated."""
    import torch

    from workloads import chain_inputs

    dev = torch.device("cuda:0")
    t0 = time.time()
    ci = chain_inputs(shape)
    gen_s = time.time() - t0
    B, ctx, gi, gt = shape.B, shape.ctx, shape.gamma_int, shape.gamma_tgt
    inter, tg, dr = ci["inter"], ci["target"], ci["draft"]
    z1, z2, _ = ci["z"]
    V = z2.shape[2]

    def up(x):
        x = np.ascontiguousarray(x)
        return torch.from_numpy(x.view(np.int16) if x.dtype == np.uint16 else x).to(dev)

    def i32(shape_):
        return torch.zeros(shape_, dtype=torch.int32, device=dev)

    Hq_i, D_i, Hkv_i = inter.q.shape[2], inter.q.shape[3], inter.k.shape[1]
    Hq_t, D_t, Hkv_t = tg["q"].shape[2], tg["q"].shape[3], tg["k"].shape[1]
    q_i, k_i, v_i, kv_i, g_i = up(inter.q), up(inter.k), up(inter.v), up(inter.kv_len), up(inter.gamma)
    p2, q1, d_i = up(z2), up(z1), up(inter.drafts)
    ua_i, ur_i = up(inter.u_acc), up(inter.u_res)
    q_t, k_t, v_t, p3 = up(tg["q"]), up(tg["k"]), up(tg["v"]), up(tg["p_logits"])
    ua_t, ur_t = up(tg["u_acc"]), up(tg["u_res"])
    out_i = torch.empty((B, gi + 1, Hq_i, D_i), dtype=torch.float32, device=dev)
    out_t = torch.empty((B, gt + 1, Hq_t, D_t), dtype=torch.float32, device=dev)
    cap_i, cap_t = inter.k.shape[2], tg["k"].shape[2]
    ws_i = sr.attention_workspace(B, gi, Hq_i, Hkv_i, D_i, cap_i, device=dev)
    ws_t = sr.attention_workspace(B, gt, Hq_t, Hkv_t, D_t, cap_t, device=dev)
    ab_i = sr.AcceptBuffers(B, gi, V, sr.SR_F32, device=dev)
    ab_t = sr.AcceptBuffers(B, gt, V, sr.SR_F32, device=dev)
    ctx_t = torch.full((B,), ctx, dtype=torch.int32, device=dev)
    g3, d3, kv3 = i32(B), i32((B, gt)), i32(B)
    upl, lol, pend, npend = i32(B), i32(B), i32((B, 2)), i32(B)
    st = i32(1)
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    K, W = args.steps, args.warmup
    # one fresh copy of the intermediate level's cache lengths per step (its
    # rollback rewrites them), restored outside the timed regions
    kv_work = [kv_i.clone() for _ in range(max(K, W, 1))]

    def refill():
        for kw in kv_work:
            kw.copy_(kv_i)
        torch.cuda.synchronize()

    def step(i, evs=None):
        mark = (lambda i: evs[i].record()) if evs else (lambda i: None)  # noqa: E731
        mark(0)
        sr.specrouter_verify_attention(q_i, k_i, v_i, None, kv_i, g_i, out_i, inter.scale, ws_i, st)
        mark(1)
        sr.specrouter_accept_and_diverge(p2, q1, d_i, g_i, ua_i, ur_i, kv_i, ab_i.accept_len, ab_i.out_tokens,
                                         ab_i.new_len, ab_i.accept_prob, ab_i.p_tok, ab_i.q_tok, ab_i.kl, ab_i.tv,
                                         ab_i.workspace, st)
        mark(2)
        sr.specrouter_chain_window(ab_i.accept_len, ab_i.out_tokens, gt, g3, d3, ctx_len=ctx_t, kv_len_next=kv3)
        sr.specrouter_verify_attention(q_t, k_t, v_t, None, kv3, g3, out_t, tg["scale"], ws_t, st)
        mark(3)
        sr.specrouter_accept_and_diverge(p3, p2[:, :gt], d3, g3, ua_t, ur_t, kv3, ab_t.accept_len, ab_t.out_tokens,
                                         ab_t.new_len, ab_t.accept_prob, ab_t.p_tok, ab_t.q_tok, ab_t.kl, ab_t.tv,
                                         ab_t.workspace, st)
        mark(4)
        sr.specrouter_chain_consensus(ctx_t, ab_i.accept_len, ab_i.out_tokens, ab_t.accept_len, ab_t.out_tokens,
                                      upl, lol, pend, npend, st)
        sr.specrouter_rollback(kv3, None, upl, None, st, L_cap=cap_t)
        sr.specrouter_rollback(kv_work[i], None, lol, None, st, L_cap=cap_i)
        mark(5)

    calibration_copy(dev)
    for i in range(max(W, 1)):
        step(i)
    refill()
    status = int(st.item())
    drafts = int(inter.gamma.sum()) + int(g3.sum().item())  # the same every step (fixed inputs)
    e0, e1 = ev(), ev()
    e0.record()
    for i in range(K):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / K
    refill()
    # per-phase durations from a second run with events between the phases
    names = ("intermediate_attention", "intermediate_accept", "window_and_target_attention", "target_accept",
             "consensus_and_rollbacks")
    tot = np.zeros(len(names))
    for i in range(K):
        evs = [ev() for _ in range(6)]
        step(i, evs)
        torch.cuda.synchronize()
        tot += [evs[p].elapsed_time(evs[p + 1]) for p in range(len(names))]
    phase_us = {n: round(t / K * 1e3, 2) for n, t in zip(names, tot)}
    # draft level: one decode-attention call (gamma = 0), made once per drafted token
    Hq_d, D_d, Hkv_d = dr["q"].shape[2], dr["q"].shape[3], dr["k"].shape[1]
    q_d, k_d, v_d, kv_d = up(dr["q"]), up(dr["k"]), up(dr["v"]), up(dr["kv_len"])
    g0 = i32(B)
    out_d = torch.empty((B, 1, Hq_d, D_d), dtype=torch.float32, device=dev)
    ws_d = sr.attention_workspace(B, 0, Hq_d, Hkv_d, D_d, dr["k"].shape[2], device=dev)
    for _ in range(3):
        sr.specrouter_verify_attention(q_d, k_d, v_d, None, kv_d, g0, out_d, dr["scale"], ws_d, st)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(K):
        sr.specrouter_verify_attention(q_d, k_d, v_d, None, kv_d, g0, out_d, dr["scale"], ws_d, st)
    e1.record()
    torch.cuda.synchronize()
    draft_us = e0.elapsed_time(e1) / K * 1e3
    status |= int(st.item())

    kv_len = inter.kv_len.astype(np.int64)
    att_bytes = int((2 * Hkv_i * kv_len * D_i * 2).sum() + B * (gi + 1) * Hq_i * D_i * (2 + 4))
    att_us = phase_us["intermediate_attention"]
    att_gbs = att_bytes / (att_us * 1e-6) / 1e9
    line = {
        "metric": "verified draft tokens/s per verify step; HBM GB/s (KV + logits) vs MI355X peak",
        "value": round(drafts / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 KV / fp32 logits",
        "data": "synthetic (seeded Philox; Q,K,V ~ N(0,1) bf16; chained logits z3, z2 = z3 + noise, z1 = z2 + noise)",
        "config": {"workload": f"{shape.name}: {shape.note}", "B": B, "ctx": ctx, "gamma_int": gi,
                   "gamma_tgt": gt, "heads_int": f"{Hq_i}/{Hkv_i}x{D_i}", "heads_tgt": f"{Hq_t}/{Hkv_t}x{D_t}",
                   "vocab": V, "drafts_per_step": drafts, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": "specrouter_verify_attention (intermediate level)",
                     "achieved": round(att_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(att_gbs / PEAK_HBM_GBS, 4), "traffic": None, "algorithmic_bytes": att_bytes,
                     "avg_launch_us": att_us},
        "phases_us": phase_us,
        "draft_decode_attention_us": round(draft_us, 2),
        "mean_k_int": round(float(ab_i.accept_len.float().mean().item()), 3),
        "mean_k_tgt": round(float(ab_t.accept_len.float().mean().item()), 3),
        "status_bits": status,
        "cpu_baseline": None if args.no_cpu else chain_cpu_baseline(ci, shape),
        "boundary": None if args.no_cpu else chain_boundary_check(ci, shape, ab_i, ab_t, g3),
        "note": "three-level chain step (intermediate and target levels); the draft level's decode attention apart",
        "input_gen_s": round(gen_s, 2),
    }
    print(json.dumps(line), flush=True)


def chain_boundary_check(ci, shape, ab_i, ab_t, g3):
    """Both accept levels of the timed chain steps against the CPU reference
    on every sequence: the intermediate level on its own inputs, the target
    level on the window the reference derives from the intermediate level's
    outcome (so a different intermediate outcome shows as a mismatch at both
    levels). Decisions must agree exactly except on boundary cases (a uniform
    within 1e-6 of a CDF breakpoint or acceptance threshold)."""
    import oracle

    inter, t = ci["inter"], ci["target"]
    z2 = ci["z"][1]
    ctx, gt = shape.ctx, shape.gamma_tgt
    r2 = oracle.accept_and_diverge(inter.p_logits, inter.q_logits, inter.drafts, inter.gamma, inter.u_acc,
                                   inter.u_res, kv_len=inter.kv_len)
    w3 = oracle.chain.target_window(r2["accept_len"], gt)
    d3 = oracle.chain.target_drafts(r2["out_tokens"], w3, gt)
    kv3 = (ctx + w3 + 1).astype(np.int32)
    r3 = oracle.accept_and_diverge(t["p_logits"], z2[:, :gt], d3, w3, t["u_acc"], t["u_res"], kv_len=kv3)
    out = {}
    for name, acc, ref, extra in (("intermediate", ab_i, r2, None), ("target", ab_t, r3, (g3, w3))):
        k = acc.accept_len.cpu().numpy()
        toks = acc.out_tokens.cpu().numpy()
        same = (k == ref["accept_len"]) & (toks == ref["out_tokens"]).all(axis=1)
        if extra is not None:
            same &= extra[0].cpu().numpy() == extra[1]
        bd = ref["boundary"].astype(bool)
        out[name] = {"sequences": int(k.shape[0]), "boundary_cases": int(bd.sum()),
                     "boundary_mismatches": int((bd & ~same).sum()),
                     "mismatches_outside_boundary": int((~bd & ~same).sum()),
                     "min_margin": float(np.min(ref["margin"]))}
    out["note"] = ("GPU accept lengths, tokens (and the target window) vs the CPU reference on every sequence "
                   "(margin < 1e-6 = boundary)")
    return out


def chain_cpu_baseline(ci, shape, target_s=10.0):
    """The CPU reference on whole chain steps of a prefix of the batch, one
    sequence at a time until about target_s has elapsed: the intermediate
    level's attention and accept, the target's window, attention and accept
    (its draft rows the intermediate level's verifier rows), and both
    rollbacks; counts the drafts of both levels."""
    import oracle

    inter, t = ci["inter"], ci["target"]
    z2 = ci["z"][1]
    B, ctx, gt = shape.B, shape.ctx, shape.gamma_tgt
    dt, done, drafts = 0.0, 0, 0
    for b in range(B):
        t0 = time.perf_counter()
        oracle.verify_attention(inter.q, inter.k, inter.v, inter.kv_len, inter.gamma, inter.scale, seqs=[b])
        r2 = oracle.accept_and_diverge(inter.p_logits, inter.q_logits, inter.drafts, inter.gamma, inter.u_acc,
                                       inter.u_res, kv_len=inter.kv_len, seqs=[b])
        g3 = oracle.chain.target_window(r2["accept_len"], gt)
        d3 = oracle.chain.target_drafts(r2["out_tokens"], g3, gt)
        kv3 = (ctx + g3 + 1).astype(np.int32)
        oracle.verify_attention(t["q"], t["k"], t["v"], kv3, g3, t["scale"], seqs=[b])
        r3 = oracle.accept_and_diverge(t["p_logits"], z2[:, :gt], d3, g3, t["u_acc"], t["u_res"], kv_len=kv3,
                                       seqs=[b])
        up_len, lo_len, _ = oracle.chain.rollback_targets(ctx, r2["accept_len"][[b]], r3["accept_len"][[b]])
        oracle.rollback(kv3[[b]], None, up_len)
        oracle.rollback(inter.kv_len[[b]], None, lo_len)
        dt += time.perf_counter() - t0
        done += 1
        drafts += int(inter.gamma[b]) + int(g3[b])
        if dt >= target_s:
            break
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        cores = os.cpu_count()
    threads = os.environ.get("OPENBLAS_NUM_THREADS") or os.environ.get("OMP_NUM_THREADS") or str(cores)
    return {
        "value": round(drafts / dt, 2), "unit": "tokens/s", "cores": int(min(cores, int(threads))), "kind": "oracle",
        "sample": f"{done} of {B} sequences, whole two-level chain steps one sequence at a time (fp64 numpy), "
                  f"{dt:.1f} s",
    }


def scheduler_timing(sr, gamma, accept_len, tv, reps=2000):
    """Host cost of the chain scheduler around this step: one observation of
    the step's accept outputs (gamma, accept_len, tv; copied to the host once,
    outside the timing) and one Algorithm 1 selection, over a five-model pool
    shaped like the paper's Llama family (68M, 1.1B, 7B, 13B, 70B parameters;
    target 70B; window = the workload's gamma_max)."""
    g = gamma.cpu().numpy()
    k = accept_len.cpu().numpy()
    t = tv.cpu().numpy()
    cap = [0.068, 1.1, 7.0, 13.0, 70.0]
    s = sr.ChainScheduler(cap, 4, max(1, t.shape[1]))
    for m, c in enumerate(cap):
        s.observe_time(m, 2e-4 * c ** 0.5)  # synthetic per-token times
    for i in range(5):
        for j in range(i + 1, 5):
            s.set_similarity(i, j, 0.5 + 0.08 * i)
    t0 = time.perf_counter()
    for _ in range(reps):
        s.observe_step(3, 4, g, k, t)
    obs_us = (time.perf_counter() - t0) / reps * 1e6
    t0 = time.perf_counter()
    for _ in range(reps):
        chain, t_eff, n_cand = s.optimal_chain()
    sel_us = (time.perf_counter() - t0) / reps * 1e6
    s.close()
    return {"observe_step_us": round(obs_us, 2), "optimal_chain_us": round(sel_us, 2), "models": len(cap),
            "candidates": n_cand, "chain": chain, "note": "host C++ via the ctypes binding, per call"}


def boundary_check(inp, acc):
    """The accept outputs of the timed calls against the CPU reference on every
    sequence of the batch: decisions must agree exactly except on boundary
    cases (a uniform within 1e-6 of a CDF breakpoint or acceptance threshold),
    which are counted, with the mismatches among them."""
    import oracle

    ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res,
                                    kv_len=inp.kv_len)
    k = acc.accept_len.cpu().numpy()
    toks = acc.out_tokens.cpu().numpy()
    same = (k == ref["accept_len"]) & (toks == ref["out_tokens"]).all(axis=1)
    bd = ref["boundary"].astype(bool)
    return {
        "sequences": int(k.shape[0]),
        "boundary_cases": int(bd.sum()),
        "boundary_mismatches": int((bd & ~same).sum()),
        "mismatches_outside_boundary": int((~bd & ~same).sum()),
        "min_margin": float(np.min(ref["margin"])),
        "note": "GPU accept lengths and tokens vs the CPU reference on every sequence (margin < 1e-6 = boundary)",
    }


def cpu_baseline(inp, n_seqs, target_s=10.0, cap_s=30.0):
    """The CPU reference, untuned, on a bounded sample of the same workload:
    whole verify steps (attention, accept-and-diverge, rollback), one
    sequence after another in batch order until about target_s has elapsed
    (whole passes over the batch again if it finishes sooner, never starting
    one that would pass cap_s)."""
    import oracle

    B = inp.B

    def run(b):
        t0 = time.perf_counter()
        oracle.verify_attention(inp.q, inp.k, inp.v, inp.kv_len, inp.gamma, inp.scale, seqs=[b])
        r = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res,
                                      kv_len=inp.kv_len, seqs=[b])
        oracle.rollback(inp.kv_len[[b]], None, r["new_len"][[b]])
        return time.perf_counter() - t0

    limit = n_seqs or B
    dt, done, drafts, passes = 0.0, 0, 0, 0
    while True:
        for b in range(min(limit, B)):
            dt += run(b)
            done += 1
            drafts += int(inp.gamma[b])
            if passes == 0 and dt >= target_s:
                break
        passes += 1
        if dt >= target_s or done < min(limit, B) or dt + dt / passes > cap_s:
            break
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        cores = os.cpu_count()
    threads = os.environ.get("OPENBLAS_NUM_THREADS") or os.environ.get("OMP_NUM_THREADS") or str(cores)
    sample = (f"{done} of {B} sequences" if done < B else f"all {B} sequences x {done // B} pass(es)")
    return {
        "value": round(drafts / dt, 2), "unit": "tokens/s", "cores": int(min(cores, int(threads))),
        "kind": "oracle",
        "sample": f"{sample}, whole verify steps one sequence at a time (fp64 numpy), {dt:.1f} s",
    }


if __name__ == "__main__":
    main()
