#!/usr/bin/env python3
"""Benchmark of the KV-COBRA hot path on one MI355X.

Workload (default): Llama-3-8B-shaped compressed cache, 32 layers x 8 KV heads
x batch 8, 32 768 cached tokens per sequence, 4 query heads per KV head,
head_dim 128, joint K+V at 2 bits per dimension (K: attention-KL weights with
C1 + C2; V: MSE weights, C1 only), synthetic power-law KV. Other workloads:
--workload (the long-context 0.5 bpd, the bit-rate sweep with --bpd, the
70B-shaped one).

A step is one serving decode step, one kvc_decode_step call: append the new
token's K and V to every unit's compressed stream and run decode attention over
all T + 1 tokens of every unit. `value` is the step's algorithmic HBM bytes
divided by the step time. Separately timed: the on-device calibration (table
step 1), the bulk prefill encode of the whole cache (median of five), the
decode-attention call alone (the roofline entry), and the same step as two
calls and as one call per layer (context).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn HBM GB/s + encode tokens/s, 8B-shape KV @32k ctx, 2 bpd"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0  # dense fp16 matrix-core peak (the bulk encoder's projection)


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def decode_alg_bytes(cache, n_tok: int) -> int:
    """Code bytes actually needed (r*b/8 per token), bases once per (layer, head, side), q and out."""
    w = cache.w
    K, V = cache.K, cache.V
    per_tok = int(np.sum(K.r_h.astype(np.int64) * K.b_h + V.r_h.astype(np.int64) * V.b_h))  # bits per token
    codes = per_tok * n_tok // 8
    basis = sum(p.size * 2 for p in cache.k_tab.P) + sum(p.size * 2 for p in cache.v_tab.P)
    qo = w.n_units * w.group * w.d * (2 + 4)
    return codes + basis + qo


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("kvc_kernels.hip", "kvc_decode.hip", "kvc_decode_g4.hip", "kvc_decode_g8.hip", "kvc_device.h",
              "kvc_append.h"):
        with open(os.path.join(ROOT, "paper_2609_24298_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(per_launch_alg: int, workload: str):
    """HBM bytes per decode call from the committed rocprofv3 counter summary, if it is current and of
    this workload."""
    path = os.path.join(ROOT, "profiles", f"decode_attn_{workload}_traffic.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha") != kernel_source_hash() or t.get("workload") != workload:
        return None
    return t.get("hbm_bytes_per_call")


def host_info():
    """CPU model and the cores this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count()
    return {"cpu_model": model, "nproc": avail, "os_cpu_count": os.cpu_count()}


def cpu_baseline(w, stats, seed: int, units, n_tok: int, mse_tokens: int = 0):
    """The oracle, untuned, on a bounded sample: its own calibration of every head (the allocation
    couples them), its tables and bases, exact codes for `units` (C, threaded over tokens), then its
    fp64 decode attention (numpy) timed over those units. With mse_tokens, also the oracle's
    reconstruction MSE of the first mse_tokens tokens of each sampled unit and side."""
    import torch
    from threadpoolctl import threadpool_info

    from oracle import alloc as oa
    from oracle import attention as oatt
    from oracle import basis as ob
    from oracle import calib
    from oracle import native as onat
    from paper_2609_24298_amd import kvc, pipeline

    t_cal = time.perf_counter()
    cal = calib.calibrate_heads(np.stack([s.cov.S_k for s in stats]), np.stack([s.cov.S_v for s in stats]),
                                np.stack([np.stack(s.cov.S_q) for s in stats]))
    t_cal = time.perf_counter() - t_cal
    stats = [pipeline.HeadStats(s.cov, cal["lam_k"][h], cal["U_k"][h], cal["sigma2_q"][h], cal["lam_v"][h],
                                cal["U_v"][h]) for h, s in enumerate(stats)]
    ak = oa.allocate(cal["lam_k"], cal["sigma2_q"], oa.AllocOpts(bpd=w.bpd))
    av = oa.allocate(cal["lam_v"], None, oa.AllocOpts(bpd=w.bpd, solver=oa.SOLVER_C1_ONLY))
    prepared = []
    code_bytes = 0
    t_enc = 0.0
    n_vec = 0
    mse = {"K": [], "V": []}
    for u in units:
        h = w.head_of_unit(u)
        s = stats[h]
        rk, bk, rv, bv = int(ak["r"][h]), int(ak["b"][h]), int(av["r"][h]), int(av["b"][h])
        Pk, dk = ob.make_basis(s.U_k, ak["order"][h], s.lam_k, rk, bk, s.sign_k)
        Pv, dv = ob.make_basis(s.U_v, av["order"][h], s.lam_v, rv, bv, s.sign_v)
        xk = pipeline.draw_unit_tokens(w, stats, kvc.SIDE_K, n_tok, seed, "cuda", units=[u])[0]
        xv = pipeline.draw_unit_tokens(w, stats, kvc.SIDE_V, n_tok, seed, "cuda", units=[u])[0]
        xkb = xk.view(torch.int16).cpu().numpy().view(np.uint16)
        xvb = xv.view(torch.int16).cpu().numpy().view(np.uint16)
        t = time.perf_counter()
        ck = onat.encode_codes(Pk, dk, bk, xkb)
        cv = onat.encode_codes(Pv, dv, bv, xvb)
        t_enc += time.perf_counter() - t
        n_vec += 2 * n_tok
        if mse_tokens:
            for name, c, P, dl, b, xb in (("K", ck, Pk, dk, bk, xkb), ("V", cv, Pv, dv, bv, xvb)):
                rec = oatt.reconstruct(c[:mse_tokens], P, dl, b)
                x64 = xb[:mse_tokens].view(np.float16).astype(np.float64)
                mse[name].append(float(np.mean((rec - x64) ** 2)))
        sk = onat.pack(ck, rk, bk, kvc.SIDE_K)
        sv = onat.pack(cv, rv, bv, kvc.SIDE_V)
        q = pipeline.draw_queries(w, stats, seed + 1, "cpu")[u].view(torch.int16).numpy().view(np.uint16)
        prepared.append((sk, sv, rk, bk, rv, bv, Pk, Pv, dk, dv, q))
        code_bytes += (rk * bk + rv * bv) * n_tok // 8
    reps = 0
    t0 = time.perf_counter()
    while True:
        for sk, sv, rk, bk, rv, bv, Pk, Pv, dk, dv, q in prepared:
            ck = onat.unpack(sk, n_tok, rk, bk, kvc.SIDE_K)
            cv = onat.unpack(sv, n_tok, rv, bv, kvc.SIDE_V)
            oatt.decode_attention(ck, cv, Pk, Pv, dk, dv, bk, bv, q, n_tok)
        reps += 1
        el = time.perf_counter() - t0
        if el > 10.0 or reps >= 200:
            break
    blas = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] + [1])
    omp = int(os.environ.get("OMP_NUM_THREADS", "0")) or host_info()["nproc"]
    out = {
        "value": round(code_bytes * reps / el / 1e9, 4), "unit": "GB/s", "cores": int(max(blas, omp)), "kind": "oracle",
        "sample": f"{len(units)} units x {n_tok} tokens of the workload: fp64 decode attention from packed codes "
                  f"(numpy, {blas} BLAS threads), {reps} reps in {el:.1f} s; exact encode of the same sample "
                  f"(C, {omp} OpenMP threads over tokens) {n_vec / t_enc:.0f} vectors/s; fp64 Jacobi calibration "
                  f"of all {len(stats)} heads {t_cal:.2f} s",
        "encode_vectors_per_s": round(n_vec / t_enc, 1),
        "calibration_s": round(t_cal, 3),
        "threads": {"blas": int(blas), "openmp": int(omp)},
    }
    out.update(host_info())
    if mse_tokens:
        out["mse_oracle"] = {k: float(np.mean(v)) for k, v in mse.items()}
    return out


def calibration_timing(w, covs, dev, n_cal: int, seed: int):
    """Table step 1 on the device for every head of the workload: covariances of n_cal calibration
    activations per key, value and query head (kvc_covariance), eigendecompositions of the key and value
    covariances (kvc_eigh) and the query variance (kvc_query_variance), each timed with events on the
    launch stream."""
    import torch

    from paper_2609_24298_amd import kvc, synth

    H, G, d = len(covs), w.group, w.d
    ev = lambda: torch.cuda.Event(enable_timing=True)
    cov_ms = 0.0
    mats = {}
    for name, n_heads, factor in (("k", H, lambda c: [c.F_k]), ("v", H, lambda c: [c.F_v]),
                                  ("q", H * G, lambda c: c.F_q)):
        F = [f for c in covs for f in factor(c)]
        x = torch.empty((n_heads, n_cal, d), dtype=torch.float16, device=dev)
        for i, f in enumerate(F):
            x[i] = synth.draw_tokens_torch(f, n_cal, (seed, 9000 + i, ord(name)), dev)
        cov = torch.empty((n_heads, d, d), dtype=torch.float32, device=dev)
        kvc.kvc_covariance(x, n_cal, cov)
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record()
        kvc.kvc_covariance(x, n_cal, cov)
        b.record()
        torch.cuda.synchronize()
        cov_ms += a.elapsed_time(b)
        del x
        mats[name] = cov
    S = torch.cat([mats["k"], mats["v"]])
    lam = torch.empty((2 * H, d), dtype=torch.float32, device=dev)
    U = torch.empty((2 * H, d, d), dtype=torch.float32, device=dev)
    sw = torch.empty(2 * H, dtype=torch.int32, device=dev)
    a, b = ev(), ev()
    a.record()
    kvc.kvc_eigh(S, lam, U, sw)
    b.record()
    torch.cuda.synchronize()
    eigh_ms = a.elapsed_time(b)
    sig = torch.empty((H, d), dtype=torch.float32, device=dev)
    Sq = mats["q"].view(H, G, d, d)
    a, b = ev(), ev()
    a.record()
    kvc.kvc_query_variance(U[:H].contiguous(), Sq, sig)
    b.record()
    torch.cuda.synchronize()
    qv_ms = a.elapsed_time(b)
    res = {"kv_heads": H, "query_heads": H * G, "cal_tokens_per_head": n_cal, "covariance_ms": round(cov_ms, 3),
           "eigh_ms": round(eigh_ms, 3), "eigh_matrices": 2 * H, "eigh_sweeps_max": int(sw.max().item()),
           "query_variance_ms": round(qv_ms, 3), "total_ms": round(cov_ms + eigh_ms + qv_ms, 3)}
    log(f"calibration on the device: {res}")
    return res


def per_layer_loop(cache, w, q, seq, n_att: int, steps: int):
    """The same decode step issued as one kvc_decode_attn call per layer (the paper times its
    primitive per layer under CUDA graphs): eager launches, then the whole loop captured in one
    HIP graph and replayed. Context for the all-layers call, not the headline value."""
    import torch

    from paper_2609_24298_amd import kvc

    upl = w.batch * w.kv_heads
    sides = [cache.layer_sides(l) for l in range(w.layers)]
    nbytes = max(kvc.kvc_decode_attn_workspace(k, v, w.group, n_att) for k, v in sides)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    out = torch.empty((w.n_units, w.group, w.d), dtype=torch.float32, device=q.device)
    views = [(k, v, q[l * upl:(l + 1) * upl], seq[l * upl:(l + 1) * upl], out[l * upl:(l + 1) * upl])
             for l, (k, v) in enumerate(sides)]

    def loop():
        for k, v, ql, sl, ol in views:
            kvc.kvc_decode_attn(k, v, ql, w.group, sl, n_att, ol, ws)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    ms_eager = timed(loop)
    eager_out = out.clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        loop()  # warm the launch path on the capture stream before capturing
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        loop()
    ms_graph = timed(g.replay)
    same = bool(torch.equal(out, eager_out))
    dec_bytes = decode_alg_bytes(cache, n_att)
    log(f"per-layer loop ({w.layers} calls): eager {ms_eager:.3f} ms, graph {ms_graph:.3f} ms "
        f"({dec_bytes / (ms_graph / 1e3) / 1e9:.1f} GB/s), graph output equals eager: {same}")
    del g
    return {"calls": w.layers, "eager_ms": round(ms_eager, 4), "graph_ms": round(ms_graph, 4),
            "graph_GBs": round(dec_bytes / (ms_graph / 1e3) / 1e9, 2), "graph_equals_eager": same}


def allocator_timing(w, stats):
    """Host allocator (kvc_allocate, one CPU thread) on the workload's K heads: the damped C1 + C2 solve
    (the paper's default, best of three runs) and the exact DP (one run)."""
    from paper_2609_24298_amd import kvc
    lam = np.stack([s.lam_k for s in stats])
    sq = np.stack([s.sigma2_q for s in stats])
    out = {"heads": len(stats), "bpd": w.bpd}
    for name, solver, reps in (("damped_ms", kvc.SOLVER_DAMPED, 3), ("dp_ms", kvc.SOLVER_DP, 1)):
        best = None
        for _ in range(reps):
            t = time.perf_counter()
            kvc.kvc_allocate(lam, sq, kvc.alloc_opts(w.bpd, solver))
            el = (time.perf_counter() - t) * 1e3
            best = el if best is None else min(best, el)
        out[name] = round(best, 2)
    log(f"allocator on {len(stats)} heads at {w.bpd} bpd: damped {out['damped_ms']} ms, DP {out['dp_ms']} ms")
    return out


def rope_flop(cache, n_tok: int) -> int:
    """Matrix-core flops of one RoPE-aware decode call: per 64-token tile of a unit, the key reconstruction
    (2 x 128 x (r_K rounded up to 32) x 64) and the logits on hi + lo halves (2 x 2 x 16 x 128 x 64)."""
    tiles = (n_tok + 63) // 64
    r32 = (cache.K.r_h.astype(np.int64) + 31) // 32 * 32
    return int(tiles * np.sum(2 * 128 * r32 * 64 + 2 * 2 * 16 * 128 * 64))


def model_mse(cache, side: int, units) -> float:
    """Mean of the distortion model D(r, b) / d (MSE weights, Lemma lem:head-dist) over `units`, from the
    product's own calibration and table: the figure the measured MSE is compared with."""
    from paper_2609_24298_amd import kvc
    w = cache.w
    tab = cache.k_tab if side == kvc.SIDE_K else cache.v_tab
    vals = []
    for u in units:
        h = w.head_of_unit(u)
        lam = (cache.stats[h].lam_k if side == kvc.SIDE_K else cache.stats[h].lam_v)[tab.order[h]]
        r, b = int(tab.r[h]), int(tab.b[h])
        vals.append((np.sum(lam[r:]) + 2.0 ** (-2 * b) / 12.0 * np.sum(lam[:r])) / w.d)
    return float(np.mean(vals))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama8b_b8_t32k_2bpd")
    ap.add_argument("--bpd", type=float, default=None, help="budget per side instead of the workload's (bit-rate sweep)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cal-tokens", type=int, default=32768,
                    help="calibration activations per head for the timed on-device calibration (0: skip)")
    ap.add_argument("--mse-units", type=int, default=None,
                    help="units whose reconstruction MSE is measured (default: 8 for the bit-rate sweep, else 0)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-per-layer", action="store_true",
                    help="skip the per-layer loop (profiling runs that summarise the all-layers call)")
    ap.add_argument("--uniform", type=int, nargs=4, metavar=("RK", "BK", "RV", "BV"), default=None,
                    help="measurement case: one (r, b) pair per side for every head instead of the allocator's "
                         "(the workload name gets the pairs appended; never the headline line)")
    ap.add_argument("--copy-calib", action="store_true",
                    help="after the timed region, run one plain 1 GiB device-to-device copy (the reference kernel "
                         "for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {args.gpus}); the multi-GPU path is not part of "
              "this build", file=sys.stderr)
        sys.exit(2)

    import dataclasses

    import torch

    from paper_2609_24298_amd import kvc, pipeline, synth

    w = synth.WORKLOADS[args.workload]
    if args.bpd is not None:
        w = dataclasses.replace(w, name=f"{w.name}@{args.bpd:g}bpd", bpd=float(args.bpd))
    T = w.tokens
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"workload {w}")
    t_setup = time.perf_counter()
    covs = synth.workload_covs(w, args.seed)
    calib = None
    if args.cal_tokens > 0 and args.uniform is None:
        calib = calibration_timing(w, covs, dev, args.cal_tokens, args.seed)
        torch.cuda.empty_cache()
    stats = pipeline.calibrate(covs, dev)
    alloc_t = allocator_timing(w, stats)
    cache = pipeline.Cache(w, seed=args.seed, device=dev, capacity=T + kvc.TILE, uniform=args.uniform, stats=stats)
    log(f"calibration + tables + bases in {time.perf_counter() - t_setup:.1f} s; "
        f"K (r,b) spread {len(set(zip(cache.k_tab.r.tolist(), cache.k_tab.b.tolist())))} pairs")

    # ---- bulk prefill encode of the whole cache: one untimed run, then the median of five
    xk = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_K, T, args.seed, dev)
    xv = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_V, T, args.seed, dev)
    torch.cuda.synchronize()
    log(f"drew {2 * w.n_units * T} fp16 vectors")
    enc_times = []
    for rep in range(6):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        cache.encode(xk, xv, 0, T)
        e1.record()
        torch.cuda.synchronize()
        if rep:
            enc_times.append(e0.elapsed_time(e1) / 1e3)
    t_enc = float(np.median(enc_times))
    log(f"bulk encode: median {t_enc * 1e3:.2f} ms of {len(enc_times)} ({min(enc_times) * 1e3:.2f}..{max(enc_times) * 1e3:.2f})")
    enc_vectors = 2 * w.n_units * T
    enc_read = enc_vectors * w.d * 2
    bits_per_tok = int(np.sum(cache.K.r_h.astype(np.int64) * cache.K.b_h + cache.V.r_h.astype(np.int64) * cache.V.b_h))
    enc_write = bits_per_tok * T // 8
    enc_flop = 2 * w.d * T * int(np.sum(cache.K.r_h.astype(np.int64) + cache.V.r_h.astype(np.int64)))

    # ---- reconstruction MSE of sampled units (bit-rate sweep): GPU against the input and the model
    n_mse = (8 if "sweep" in args.workload else 0) if args.mse_units is None else args.mse_units
    mse = None
    mse_tokens = min(T, 4096)
    if n_mse:
        mse = {}
        for side, S, x in ((kvc.SIDE_K, cache.K, xk), (kvc.SIDE_V, cache.V, xv)):
            sub = kvc.SideRange(S, 0, n_mse)
            rec = torch.empty((n_mse, mse_tokens, w.d), dtype=torch.float32, device=dev)
            kvc.kvc_reconstruct(sub, 0, mse_tokens, rec)
            torch.cuda.synchronize()
            err = (rec.double() - x[:n_mse, :mse_tokens].double()).pow(2).mean().item()
            mse["KV"[side]] = {"gpu": err, "model_D_over_d": model_mse(cache, side, range(n_mse))}
        mse["units"], mse["tokens"] = n_mse, mse_tokens
        log(f"reconstruction MSE: {mse}")
    del xk, xv
    torch.cuda.empty_cache()

    # ---- decode step: append one token per unit and attend over T + 1 tokens, fused in one call
    xk1 = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_K, 1, args.seed + 100, dev)
    xv1 = pipeline.draw_unit_tokens(w, cache.stats, kvc.SIDE_V, 1, args.seed + 100, dev)
    q = pipeline.draw_queries(w, cache.stats, args.seed + 1, dev)
    n_att = T + 1
    seq = torch.full((w.n_units,), n_att, dtype=torch.int32, device=dev)
    ws, out = cache.decode_buffers(n_att)

    def step():
        cache.step(xk1, xv1, T, q, seq, n_att, out, ws)

    def step_two_calls():
        cache.encode(xk1, xv1, T, 1)
        cache.decode(q, seq, n_att, out, ws)

    def time_steps(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        for _ in range(args.steps):
            fn()
        s1.record()
        torch.cuda.synchronize()
        return s0.elapsed_time(s1) / args.steps

    ms_two = time_steps(step_two_calls)
    ms_step = time_steps(step)
    log(f"{args.steps} steps: {ms_step:.3f} ms/step fused (kvc_decode_step), {ms_two:.3f} ms as two calls")

    # decode call alone, events on the launch stream, for the roofline entry: back to back, and with the
    # 256 MB MALL flushed before each call, outside the events; the roofline takes the mean of the
    # flushed calls. The flush reads a 512 MB buffer (a reduction on the same stream, which ends before
    # the first event): the MALL then holds other, clean lines, so the call reads its codes from HBM. A
    # flush by writing the buffer leaves the MALL full of dirty lines whose write-back overlaps the next
    # call and takes HBM time from it (about 55 us per call on the 8B-shaped 32k workload); that variant
    # is reported as well, with the device idle before each call (an idle device also starts the call
    # at lower clocks, which the issue-bound workloads feel).
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in evs:
        a.record()
        cache.decode(q, seq, n_att, out, ws)
        b.record()
    torch.cuda.synchronize()
    t_b2b = float(np.mean([a.elapsed_time(b) for a, b in evs])) / 1e3
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    flush.fill_(1)
    flush_words = flush.view(torch.int32)

    def flushed(call, write=False):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for i, (a, b) in enumerate(evs):
            if write:
                flush.fill_(i & 0xFF)
                torch.cuda.synchronize()
            else:
                flush_words.sum()
            a.record()
            call()
            b.record()
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in evs])) / 1e3

    t_dec = flushed(lambda: cache.decode(q, seq, n_att, out, ws))
    t_dec_wflush = flushed(lambda: cache.decode(q, seq, n_att, out, ws), write=True)
    # the same decode with rotary position embeddings (keys cached pre-RoPE, rotated after reconstruction):
    # same bytes, plus the reconstruction of every key on the matrix cores
    t_rope = flushed(lambda: kvc.kvc_decode_attn_rope(cache.K, cache.V, q, w.group, seq, n_att, 500000.0, out, ws))
    del flush, flush_words
    assert torch.isfinite(out).all().item()

    # achievable HBM read rate on this device: the library's streaming-read probe over 2 GiB (best of 5)
    probe = torch.ones(2 << 30, dtype=torch.uint8, device=dev)
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    kvc.kvc_read_probe(probe, sink)
    p_ms = []
    for _ in range(5):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        kvc.kvc_read_probe(probe, sink)
        b.record()
        torch.cuda.synchronize()
        p_ms.append(a.elapsed_time(b))
    read_gbs = probe.numel() / (min(p_ms) / 1e3) / 1e9
    del probe, sink
    torch.cuda.empty_cache()

    per_layer = None if args.no_per_layer else per_layer_loop(cache, w, q, seq, n_att, args.steps)

    dec_bytes = decode_alg_bytes(cache, n_att)
    # append: read the new token's fp16 K and V, write r*b bits per unit and side
    append_bytes = 2 * w.n_units * w.d * 2 + bits_per_tok // 8
    step_bytes = dec_bytes + append_bytes
    value = step_bytes / (ms_step / 1e3) / 1e9
    achieved = dec_bytes / t_dec / 1e9
    log(f"decode call {t_dec * 1e3:.3f} ms, {achieved:.1f} GB/s algorithmic ({dec_bytes / 1e9:.3f} GB); "
        f"back to back {t_b2b * 1e3:.3f} ms; after a write flush {t_dec_wflush * 1e3:.3f} ms; "
        f"read probe {read_gbs:.1f} GB/s")

    res_workload = w.name + ("" if args.uniform is None else "@uniform_k{}_{}_v{}_{}".format(*args.uniform))
    res = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "i8/f32", "data": "synthetic",
        "config": {"workload": res_workload,
                   "layers": w.layers, "kv_heads": w.kv_heads, "q_per_kv": w.group,
                   "batch": w.batch, "context": T, "bpd_per_side": w.bpd, "head_dim": w.d},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(dec_bytes, res_workload),
                     "kernel": "kvc_decode_attn (qproj + decode_partial + combine)",
                     "alg_bytes_per_launch": dec_bytes, "avg_launch_ms": round(t_dec * 1e3, 4),
                     "launch_ms_back_to_back": round(t_b2b * 1e3, 4),
                     "launch_ms_after_write_flush": round(t_dec_wflush * 1e3, 4),
                     "flush": "512 MB read on the same stream before each timed call",
                     "achievable_read_GBs": round(read_gbs, 1),
                     "frac_of_achievable": round(achieved / read_gbs, 4)},
        "step": {"fused_ms": round(ms_step, 4), "two_calls_ms": round(ms_two, 4),
                 "bytes": step_bytes, "note": "append of the new token + decode attention over T + 1 tokens"},
        "per_layer_decode": per_layer,
        "rope_decode": {"ms": round(t_rope * 1e3, 4), "GBs": round(dec_bytes / t_rope / 1e9, 2),
                        "frac": round(dec_bytes / t_rope / 1e9 / HBM_PEAK_GBS, 4),
                        "mfma_TFLOPs": round(rope_flop(cache, n_att) / t_rope / 1e12, 2),
                        "note": "kvc_decode_attn_rope, rotary base 500000: K reconstructed per tile on fp16 matrix "
                                "cores, rotated, scored; MALL flushed before each call"},
        "encode": {"vectors_per_s": round(enc_vectors / t_enc, 1), "model_tokens_per_s": round(w.batch * T / t_enc, 1),
                   "ms_median": round(t_enc * 1e3, 3), "ms_min": round(min(enc_times) * 1e3, 3),
                   "ms_max": round(max(enc_times) * 1e3, 3), "runs": len(enc_times),
                   "hbm_GBs": round((enc_read + enc_write) / t_enc / 1e9, 2),
                   "hbm_frac": round((enc_read + enc_write) / t_enc / 1e9 / HBM_PEAK_GBS, 4),
                   "mfma_TFLOPs": round(enc_flop / t_enc / 1e12, 2),
                   "mfma_frac": round(enc_flop / t_enc / 1e12 / MFMA_F16_PEAK_TFLOPS, 4)},
        "calibration": calib,
        "allocator": alloc_t,
        "mse": mse,
    }
    if args.copy_calib:
        n = 1 << 30
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: {n} bytes read and written")
        del src, dst
    if not args.no_cpu_baseline and args.uniform is None:  # the oracle sample builds its own allocation
        log("cpu baseline (oracle) ...")
        try:
            units = list(range(n_mse)) if n_mse else [0, w.n_units // 2 + 3]
            res["cpu_baseline"] = cpu_baseline(w, cache.stats, args.seed, units, T, mse_tokens if n_mse else 0)
        except Exception as e:  # the baseline is context, never a reason to lose the GPU line
            res["cpu_baseline"] = {"error": repr(e)}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
