#!/usr/bin/env python3
"""Benchmark of one BRISK-DLM decoding step on one MI355X.

A step is the whole hot path over one block batch: brisk_propose_block (LM
head + fused top-K) and brisk_rerank_verify (the prefix-conditioned corrector
followed by greedy verification of its selections).  Inputs are synthetic, drawn once
on the GPU and resident in HBM before timing starts.

Prints one JSON line: block positions per second, the propose stage's
achieved HBM bandwidth (or MFMA rate) against the MI355X peak, per-stage
times, and the CPU oracle timed on the host on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2516.6      # dense bf16 MFMA: 256 CU x 4096 flop/clk x 2.4 GHz
METRIC = "block positions/sec (propose+rerank+verify) and % HBM/MFMA roofline"
DEFAULT_WORKLOAD = "llada8b-b1-l32"
ROOT = os.path.dirname(os.path.abspath(__file__))


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    # Eager launches are the default: on the decode shape a replayed hipGraph
    # of the step measured slower (about 3%), on the 2048-row shape 1% faster.
    ap.add_argument("--graph", dest="graph", action="store_true", default=False,
                    help="time hipGraph replay of the step instead of eager launches")
    ap.add_argument("--eager", dest="graph", action="store_false",
                    help="time eager launches of the step on one stream (the default)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the side timings of the verifier, profile, loss and sampling calls "
                         "(the timed step is unchanged), so a counter run sees only the step's kernels")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB streaming copy (for scaling HBM byte counters)")
    return ap.parse_args()


def propose_cost(wl):
    """Algorithmic bytes and flops of brisk_propose_block for one step."""
    rows = wl.B * wl.L
    bytes_ = 2 * wl.V * wl.d + 2 * rows * wl.d + rows * wl.K * 8
    flops = 2 * rows * wl.d * wl.V
    return bytes_, flops


def cpu_baseline(blk, budget_s):
    """The oracle, as is, on host cores, over a bounded sample of the same
    workload: whole sequences of the batch (all L positions, propose + rerank +
    verify), taken in order and repeated until the time budget is spent."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import oracle
    from synth import PSI_FIELDS, bf16_bits

    wl = blk.wl
    H_bits, W_bits, E_bits = bf16_bits(blk.H), bf16_bits(blk.W), bf16_bits(blk.E)
    H = oracle.bf16_to_f64(H_bits)
    h_c = oracle.bf16_to_f64(bf16_bits(blk.h_c))
    x0 = blk.x0.cpu().numpy().astype(np.int64)
    ver = blk.verifier.cpu().numpy()
    psi = {k: oracle.bf16_to_f64(bf16_bits(blk.psi[k])) for k in PSI_FIELDS}
    n_seq, positions, spent = 0, 0, 0.0
    while True:
        b = n_seq % wl.B
        rs = slice(b * wl.L, (b + 1) * wl.L)
        t0 = time.perf_counter()
        cl, ci = oracle.propose_block(H_bits[rs], W_bits, wl.K)
        out = oracle.rerank(psi, blk.alpha, blk.b_g, H[rs], h_c[b:b + 1], x0[b:b + 1], W_bits, E_bits,
                            cl, ci, 1, wl.L)
        oracle.verify_accept(out["selected"], ver[b:b + 1])
        spent += time.perf_counter() - t0
        n_seq += 1
        positions += wl.L
        if spent >= budget_s:
            break
    blas = [p.get("num_threads", 0) for p in threadpool_info() if p.get("user_api") == "blas"]
    cores = max(blas) if blas else 1
    return {"value": round(positions / spent, 2), "unit": "block positions/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{n_seq} sequence(s) of {wl.name} ({positions} positions: propose + rerank + "
                      f"verify, {spent:.1f} s); float64 numpy, host has {os.cpu_count()} logical CPUs"}


def time_accept_profile(brisk, dev, M, n_blocks=1 << 20, reps=50):
    """brisk_accept_profile over n_blocks accepted-prefix lengths (the
    statistics that feed the position weights), timed with HIP events."""
    import torch

    g = torch.Generator(device=dev).manual_seed(0)
    lens = torch.randint(0, M + 1, (n_blocks,), generator=g, device=dev, dtype=torch.int32)
    for _ in range(3):
        brisk.accept_profile(lens, M)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        brisk.accept_profile(lens, M)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    return {"n_blocks": n_blocks, "M": M, "us_per_call": round(us, 2),
            "read_GB_per_s": round(4 * n_blocks / (us * 1e-6) / 1e9, 1)}


def time_fused_verify(brisk, blk, wl, reps=20):
    """One LM-head pass over this block's proposal rows plus the previous
    block's verifier rows (bf16 of the hidden states plus sigma-scaled noise),
    against two separate passes, timed with HIP events."""
    import torch

    g = torch.Generator(device=blk.H.device).manual_seed(1)
    noise = torch.randn(blk.H.shape, generator=g, device=blk.H.device, dtype=torch.float32)
    Hv = (blk.H.float() + 0.3 * noise).to(torch.bfloat16)
    both = torch.cat([blk.H, Hv], dim=0).contiguous()
    rows = wl.B * wl.L

    def fused():
        brisk.propose_verify(both, blk.W, rows, wl.K)

    def separate():
        brisk.propose_block(blk.H, blk.W, wl.K)
        brisk.propose_verify(Hv, blk.W, 0, wl.K)

    out = {"rows": f"{rows} proposal + {rows} verifier"}
    for name, fn in (("fused_us", fused), ("separate_us", separate)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        out[name] = round(e0.elapsed_time(e1) * 1e3 / reps, 2)
    return out


def time_corrector_loss(brisk, blk, wl, corr, cl, ci, acc, reps=50):
    """brisk_corrector_loss on this step's candidates, refined logits and
    accept lengths, with verifier rows = bf16(hidden + 0.3 noise)."""
    import torch

    rr = brisk.rerank(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl, ci, wl.B, wl.L, want_scores=True)
    g = torch.Generator(device=blk.H.device).manual_seed(2)
    Hv = (blk.H.float() + 0.3 * torch.randn(blk.H.shape, generator=g, device=blk.H.device)).to(torch.bfloat16)
    fn = lambda: brisk.corrector_loss(Hv, blk.W, ci, cl, rr["refined"], acc, wl.B, wl.L)
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return {"positions": wl.B * wl.L, "us_per_call": round(e0.elapsed_time(e1) * 1e3 / reps, 2)}


def time_spec_verify(brisk, blk, wl, cl, ci, reps=20):
    """brisk_spec_verify on verifier rows bf16(hidden + 0.3 noise), proposals
    drawn from the softmax of the candidate logits mixed with the uniform law
    (weight 0.3), temperature 1, fresh seed per call."""
    import torch

    g = torch.Generator(device=blk.H.device).manual_seed(3)
    Hv = (blk.H.float() + 0.3 * torch.randn(blk.H.shape, generator=g, device=blk.H.device)).to(torch.bfloat16)
    prob = (0.7 * torch.softmax(cl.float(), dim=1) + 0.3 / wl.K).contiguous()
    pick = torch.multinomial(prob, 1, generator=g).view(-1)
    x = ci.gather(1, pick[:, None]).view(wl.B, wl.L).contiguous()
    u = torch.rand(wl.B * wl.L, generator=g, device=blk.H.device)
    calls = [0]

    def fn():
        calls[0] += 1
        return brisk.spec_verify(Hv, blk.W, x, ci, prob, u, 1000 + calls[0], 1.0)

    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        out = fn()
    e1.record()
    torch.cuda.synchronize()
    return {"positions": wl.B * wl.L, "us_per_call": round(e0.elapsed_time(e1) * 1e3 / reps, 2),
            "mean_accept_len": round(out["accept_len"].float().mean().item(), 3)}


def copy_calibration(n_bytes=1 << 30, reps=3):
    """A plain streaming kernel of known size (read n_bytes, write n_bytes),
    run so that HBM byte counters can be scaled against it."""
    import torch

    src = torch.ones(n_bytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(reps):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": {"kernel": "torch.neg (float32)", "read_bytes": n_bytes,
                                           "write_bytes": n_bytes, "launches": reps}}), flush=True)


def counter_traffic(wl):
    """HBM bytes per launch of the LM-head pass from the committed counter
    summary of this workload, or None when it is missing or was taken on a
    different version of the LM-head kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_propose_{wl.name}.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        return round(float(vals["hbm_bytes_lmhead_pass"]))
    except (KeyError, ValueError):
        return None


def kernel_source_hash():
    import hashlib

    h = hashlib.sha256()
    for name in ("lmhead_topk.hip", "device_common.h"):
        with open(os.path.join(ROOT, "paper_2609_33390_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the hot path is data parallel over sequences: each GPU would run this same step "
              "on its own share of the batch)", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    import torch

    import paper_2609_33390_amd as brisk
    import synth

    wl = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    blk = synth.make_block(wl, dev)
    corr = brisk.Corrector(blk.psi, blk.alpha, blk.b_g)
    rows, K = wl.B * wl.L, wl.K
    cl = torch.empty(rows, K, dtype=torch.float32, device=dev)
    ci = torch.empty(rows, K, dtype=torch.int32, device=dev)
    sel = torch.empty(wl.B, wl.L, dtype=torch.int32, device=dev)
    acc = torch.empty(wl.B, dtype=torch.int32, device=dev)
    cor = torch.empty(wl.B, dtype=torch.int32, device=dev)
    ws_p = torch.empty(brisk.propose_workspace_size(rows, wl.d, wl.V, K), dtype=torch.uint8, device=dev)
    ws_r = torch.empty(brisk.rerank_workspace_size(corr, wl.B, wl.L, K), dtype=torch.uint8, device=dev)

    # brisk_propose_block as its two launches, so that the LM-head pass (the
    # dominant kernel) is timed on its own
    def lmhead():
        brisk.propose_lmhead(blk.H, blk.W, K, ws_p)

    def merge():
        brisk.propose_merge(rows, wl.V, K, ws_p, cl, ci)

    def propose():
        lmhead()
        merge()

    def rest():
        brisk.rerank_verify(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl, ci, blk.verifier, wl.B, wl.L,
                            selected=sel, accept_len=acc, correction=cor, workspace=ws_r)

    for _ in range(args.warmup):
        propose()
        rest()
    torch.cuda.synchronize()

    n = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n)]
    def eager_total():
        """n eager steps back to back; returns their total time in ms."""
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record()
        for _ in range(n):
            propose()
            rest()
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1)

    def eager_stages():
        """n more eager steps with HIP events around each launch group (the
        events themselves add stream work, so these steps are not the timed
        ones); returns the per-step LM-head, propose and rerank+verify times."""
        torch.cuda.synchronize()
        for i in range(n):
            ev[i][0].record()
            lmhead()
            ev[i][1].record()
            merge()
            ev[i][2].record()
            rest()
            ev[i][3].record()
        torch.cuda.synchronize()
        return ([ev[i][0].elapsed_time(ev[i][1]) for i in range(n)],
                [ev[i][0].elapsed_time(ev[i][2]) for i in range(n)],
                [ev[i][2].elapsed_time(ev[i][3]) for i in range(n)])

    if args.graph:
        # the whole step captured once and replayed: one launch per step
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                propose()
                rest()
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(n):
            g.replay()
        t1.record()
        torch.cuda.synchronize()
        total_ms = t0.elapsed_time(t1)
        # per-launch figures (the roofline of the LM-head pass) from the same
        # steps launched eagerly with events between them
        lm_ms, prop_ms, rest_ms = eager_stages()
    else:
        total_ms = eager_total()
        lm_ms, prop_ms, rest_ms = eager_stages()

    ms_step = total_ms / n
    value = rows / (ms_step * 1e-3)
    bytes_, flops = propose_cost(wl)
    t_lm = statistics.mean(lm_ms) * 1e-3
    t_prop = statistics.mean(prop_ms) * 1e-3
    ai = flops / bytes_
    ridge = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)

    def roofline(b, t):
        if ai < ridge:
            a = b / t / 1e9
            return {"bound": "hbm", "achieved": round(a, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(a / HBM_PEAK_GBS, 4)}
        a = flops / t / 1e12
        return {"bound": "mfma", "achieved": round(a, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(a / BF16_PEAK_TFLOPS, 4)}

    # the dominant kernel: the LM-head pass (its candidates leave through the
    # merge launch, so its algorithmic bytes are the two operands it reads)
    roof = roofline(bytes_ - rows * wl.K * 8, t_lm)
    roof["traffic"] = counter_traffic(wl)
    roof["kernel"] = "lmhead_topk_kernel (brisk_propose_lmhead, the LM-head pass of brisk_propose_block)"
    roof["launch_us"] = round(t_lm * 1e6, 2)
    call = roofline(bytes_, t_prop)
    roof["propose_call"] = {"kernels": "lmhead_topk_kernel + topk_merge_kernel", "launch_us": round(t_prop * 1e6, 2),
                            "achieved": call["achieved"], "frac": call["frac"]}

    torch.cuda.synchronize()
    hist = torch.bincount(acc.long(), minlength=wl.L + 1).cpu().tolist()
    if args.no_extras:
        prof = fused = loss = spec = None
    else:
        prof = time_accept_profile(brisk, dev, wl.L)
        fused = time_fused_verify(brisk, blk, wl)
        loss = time_corrector_loss(brisk, blk, wl, corr, cl, ci, acc)
        spec = time_spec_verify(brisk, blk, wl, cl, ci)
    res = {
        "metric": METRIC, "value": round(value, 1), "unit": "block positions/s", "n_gpus": 1,
        "steps": n, "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; LLaDA/Dream-shaped random blocks, random-init corrector)",
        "config": {"workload": wl.name, "B": wl.B, "L": wl.L, "d": wl.d, "V": wl.V, "K": wl.K,
                   "r": wl.r, "timing": "hipGraph replay" if args.graph else "eager, one stream"},
        "roofline": roof,
        "stages_ms": {"lmhead": round(statistics.mean(lm_ms), 5), "propose": round(statistics.mean(prop_ms), 5),
                      "rerank+verify": round(statistics.mean(rest_ms), 5)},
        "accept_hist": hist,
        "accept_profile": prof,
        "propose_verify": fused,
        "corrector_loss": loss,
        "spec_verify": spec,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(blk, args.cpu_budget_s)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
