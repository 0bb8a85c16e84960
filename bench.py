#!/usr/bin/env python3
"""Benchmark of the SD1.4 UNet attention hot path on one MI355X.

A step is the attention of one 64x64-level transformer block of SD1.4's UNet
with classifier-free guidance: self-attention B=2, H=8, Lq=Lk=4096, D=40,
then cross-attention over the 77-token text context (Lq=4096, Lk=77, D=40),
both through the C ABI of libsdattn on fp16 N(0,1) inputs already resident
in HBM.  `value` is the useful attention work of the step (4*B*H*Lq*Lk*D
flops per call) divided by the wall time per step.

Also reported, on the same stream with HIP events:
  roofline      the self-attention kernel against the fp16 dense MFMA peak
  cross         the cross-attention kernel's algorithmic bytes against HBM,
                warm and with inputs rotated over more buffers than the
                256 MiB Infinity Cache holds ("cold")
  softmax_rows  Eq. 4's row reduction over A = Q K^T of the 64x64 level
                (65536 rows x 4096 fp16), which the fused kernels never
                materialise; timed alone, not part of the step
  cpu_baseline  the fp64 oracle on a bounded row sample of the same step
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "attention TFLOP/s and % fp16 MFMA peak, SD1.4 64×64 self-attn (B2,H8,L4096,D40)"
PEAK_F16_TFLOPS = 2500.0      # MI355X dense fp16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing")
    ap.add_argument("--no-extras", action="store_true",
                    help="time only the step (no cold cross or softmax_rows legs)")
    ap.add_argument("--cpu-rows-per-head", type=int, default=5120,
                    help="self-attention rows per (b, h) the oracle times")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 256 MiB device copy (scales the HBM traffic counters)")
    return ap.parse_args()


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; the attention "
                                   "path has no multi-GPU mode (--gpus must be 1)"}), flush=True)
        sys.exit(2)

    import torch
    import paper_2304_11267_amd as sd
    from paper_2304_11267_amd import workloads as wl

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}), flush=True)
        sys.exit(1)
    sd.load_library()
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()

    self_case = wl.CASES["l64_self"]
    cross_case = wl.CASES["l64_cross"]

    def upload(case):
        q, k, v = wl.case_inputs(case)
        qd, kd, vd = (torch.from_numpy(t).to(dev) for t in (q, k, v))
        return qd, kd, vd, torch.empty_like(qd)

    sq, sk, sv, so = upload(self_case)
    cq, ck, cv, co = upload(cross_case)

    def step():
        sd.forward(sq, sk, sv, so, self_case.scale, stream)
        sd.forward(cq, ck, cv, co, cross_case.scale, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # The timed steps: nothing else on the stream.  An event pair around
    # every launch would add its own dispatch gaps (a few microseconds per
    # pair on this runtime), so events bracket only the whole region.
    e_start, e_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e_start.record(stream)
    for _ in range(args.steps):
        step()
    e_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms_per_step = e_start.elapsed_time(e_end) / args.steps

    # Each kernel's average launch duration, on the same stream with the same
    # inputs and launch configuration: back-to-back launches between one event
    # pair (the figure rocprofv3's kernel trace reports for the same launches).
    self_ms = back_to_back_ms(torch, sd, stream, [(sq, sk, sv, so)], self_case.scale,
                              launches=max(1, min(args.steps, 100)))
    ms_per_step = wall * 1e3 / args.steps
    step_flops = self_case.flops + cross_case.flops
    value = step_flops / (ms_per_step * 1e-3) / 1e12

    self_tflops = self_case.flops / (self_ms * 1e-3) / 1e12
    roofline = {
        "kernel": "attn_fwd_lds_kernel<f16, D=40> (self-attention)",
        "bound": "mfma",
        "achieved": round(self_tflops, 2),
        "peak": PEAK_F16_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(self_tflops / PEAK_F16_TFLOPS, 4),
        "traffic": recorded_traffic(),
        "avg_kernel_us": round(self_ms * 1e3, 3),
        "flops_per_launch": self_case.flops,
    }
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "gpu_ms_per_step": round(gpu_ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic: seeded N(0,1) fp16 Q/K/V at SD1.4 shapes (no weights or text encoder)",
        "config": {
            "workload": "SD1.4 UNet 64x64-level attention block, CFG batch: self B2 H8 Lq=Lk=4096 D40 "
                        "+ cross B2 H8 Lq=4096 Lk=77 D40",
            "B": 2, "H": 8, "Lq": 4096, "Lk_self": 4096, "Lk_cross": 77, "D": 40,
            "step_flops": step_flops,
        },
        "roofline": roofline,
        "self_attention": {"avg_kernel_us": round(self_ms * 1e3, 3), "tflops": round(self_tflops, 2),
                           "frac_f16_peak": round(self_tflops / PEAK_F16_TFLOPS, 4)},
    }
    warm_ms = back_to_back_ms(torch, sd, stream, [(cq, ck, cv, co)], cross_case.scale)
    cross_gbs = cross_case.bytes / (warm_ms * 1e-3) / 1e9
    out["cross"] = {"avg_kernel_us": round(warm_ms * 1e3, 3), "bytes_per_launch": cross_case.bytes,
                    "warm_gbs": round(cross_gbs, 1), "warm_frac_hbm": round(cross_gbs / PEAK_HBM_GBS, 4),
                    "tflops": round(cross_case.flops / (warm_ms * 1e-3) / 1e12, 2)}

    if not args.no_extras:
        out["cross"].update(cold_cross(torch, sd, wl, dev, stream, cross_case))
        out["softmax_rows"] = bench_softmax_rows(torch, sd, dev, stream)
        out["two_pass"] = bench_two_pass(torch, sd, stream, self_case, (sq, sk, sv), self_ms)
        out["attention_block"] = bench_block(torch, sd, wl, dev, stream,
                                             {"self": self_ms, "cross": warm_ms})
        out["norm_act"] = bench_norm_act(torch, sd, wl, dev, stream)
        out["conv3x3_winograd"] = bench_conv(torch, sd, wl, dev, stream)

    if args.copy_calibration:
        out["copy_calibration"] = copy_calibration(torch, dev, stream)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, self_case, cross_case, args.cpu_rows_per_head)

    print(json.dumps(out), flush=True)


def back_to_back_ms(torch, sd, stream, sets, scale, launches=200, reps=3):
    """Average duration of one launch over `reps` batches of `launches` back-to-back
    calls cycling through `sets`, each batch queued behind a busy GPU so the events
    time the kernels, not the host."""
    for s in sets:
        sd.forward(*s, scale, stream)
    torch.cuda.synchronize()
    total = 0.0
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(20_000_000)
        e0.record(stream)
        for i in range(launches):
            sd.forward(*sets[i % len(sets)], scale, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        total += e0.elapsed_time(e1)
    return total / (reps * launches)


def cold_cross(torch, sd, wl, dev, stream, case, nsets=40):
    """Cross-attention with inputs rotated over nsets buffers (> 256 MiB in total)."""
    sets = []
    for i in range(nsets):
        q, k, v = wl.make_qkv(case.B, case.H, case.Lq, case.Lk, case.D, case.seed + 100 + i)
        qd, kd, vd = (torch.from_numpy(t).to(dev) for t in (q, k, v))
        sets.append((qd, kd, vd, torch.empty_like(qd)))
    ms = back_to_back_ms(torch, sd, stream, sets, case.scale, launches=5 * nsets)
    gbs = case.bytes / (ms * 1e-3) / 1e9
    return {"cold_avg_kernel_us": round(ms * 1e3, 3), "cold_gbs": round(gbs, 1),
            "cold_frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
            "cold_protocol": f"{nsets} input sets of {case.bytes} B rotated ({nsets * case.bytes / 2**20:.0f} MiB), "
                             "back-to-back launches"}


def bench_two_pass(torch, sd, stream, case, qkv, fused_ms, reps=5):
    """The partially fused softmax as three launches at the 64x64 level (logits
    in fp16 -> Eq. 4's (L, S) -> exp/normalise times V), against the fused kernel."""
    q, k, v = qkv
    B, H, Lq, Lk, D = case.B, case.H, case.Lq, case.Lk, case.D
    a = torch.empty(B, H, Lq, Lk, dtype=torch.float16, device=q.device)
    ls = torch.empty(B, H, Lq, 2, dtype=torch.float32, device=q.device)
    o = torch.empty_like(q)
    a2, ls2 = a.view(B * H * Lq, Lk), ls.view(B * H * Lq, 2)
    calls = [lambda: sd.logits(q, k, a, case.scale, stream),
             lambda: sd.softmax_rows(a2, ls2, None, 1.0, stream),
             lambda: sd.softmax_pv(a, ls, v, o, stream)]
    for c in calls:
        c()
    torch.cuda.synchronize()
    t = [[] for _ in calls]
    for _ in range(reps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
        ev[0].record(stream)
        for i, c in enumerate(calls):
            c()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        for i in range(len(calls)):
            t[i].append(ev[i].elapsed_time(ev[i + 1]))
    ms = [float(np.median(x)) for x in t]
    a_bytes = a.numel() * 2
    qkv_bytes = 2 * B * H * D * 2 * (Lq + Lk)
    total = sum(ms)
    return {
        "logits_us": round(ms[0] * 1e3, 2), "logits_gbs": round((a_bytes + qkv_bytes / 2) / (ms[0] * 1e-3) / 1e9, 1),
        "softmax_rows_us": round(ms[1] * 1e3, 2), "softmax_rows_gbs": round(a_bytes / (ms[1] * 1e-3) / 1e9, 1),
        "softmax_pv_us": round(ms[2] * 1e3, 2), "softmax_pv_gbs": round((a_bytes + qkv_bytes / 2) / (ms[2] * 1e-3) / 1e9, 1),
        "total_us": round(total * 1e3, 2),
        "fused_us": round(fused_ms * 1e3, 2),
        "fused_speedup": round(total / fused_ms, 2),
        "a_bytes": a_bytes,
        "config": "self B2 H8 L4096 D40, logits stored in fp16 (537 MB, written once, read twice)",
    }


def bench_softmax_rows(torch, sd, dev, stream, reps=10):
    rows, cols = 2 * 8 * 4096, 4096
    g = torch.Generator(device=dev)
    g.manual_seed(230411267)
    a = torch.randn(rows, cols, device=dev, dtype=torch.float32, generator=g).mul_(2.0).to(torch.float16)
    ls = torch.empty(rows, 2, device=dev, dtype=torch.float32)
    p = torch.empty_like(a)
    res = {}
    for name, pp in (("stats_only", None), ("with_p", p)):
        for _ in range(2):
            sd.softmax_rows(a, ls, pp, scale=1.0, stream=stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            sd.softmax_rows(a, ls, pp, scale=1.0, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        nbytes = rows * cols * 2 * (2 if pp is not None else 1) + rows * 8
        gbs = nbytes / (ms * 1e-3) / 1e9
        res[name] = {"avg_kernel_us": round(ms * 1e3, 2), "bytes": nbytes, "gbs": round(gbs, 1),
                     "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)}
    res["shape"] = f"{rows}x{cols} fp16 (A = Q K^T of the 64x64 level; A is L2/MALL-cold at 537 MB)"
    return res


def bench_block(torch, sd, wl, dev, stream, attn_ms, launches=50, reps=3):
    """SD's attention block at the 64x64 level (Q/K/V projections, the fused
    attention, the output projection with bias), launched back to back behind
    a busy GPU; weights N(0, 1/fan_in) standing in for trained ones.  Cross-
    attention is timed both as one call and as the per-step part alone, with
    the text context's K and V computed once beforehand (they do not change
    across denoising steps)."""

    def timed(call):
        call()
        torch.cuda.synchronize()
        best = None
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(20_000_000)
            e0.record(stream)
            for _ in range(launches):
                call()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / launches
            best = ms if best is None else min(best, ms)
        return best

    res = {}
    for kind in ("self", "cross"):
        case = wl.BLOCK_CASES["blk64_" + kind]
        x, ctx, wq, wk, wv, wo, bo = (torch.from_numpy(t).to(dev) for t in wl.block_inputs(case))
        ws = torch.empty(sd.attention_block_workspace(case.B, case.Lq, case.Lk, case.C),
                         dtype=torch.uint8, device=dev)
        out = torch.empty_like(x)
        ms = timed(lambda: sd.attention_block(x, ctx, wq, wk, wv, wo, bo, out, ws, case.H,
                                              case.scale, stream))
        res[kind] = {"us": round(ms * 1e3, 2), "flops": case.flops,
                     "tflops": round(case.flops / (ms * 1e-3) / 1e12, 1),
                     "attention_us": round(attn_ms[kind] * 1e3, 2),
                     "projections_us": round((ms - attn_ms[kind]) * 1e3, 2),
                     "shape": f"x [{case.B},{case.Lq},{case.C}] ctx [{case.B},{case.Lk},{case.Cc}] H{case.H}"}
        if kind == "cross":
            D = case.C // case.H
            k = torch.empty(case.B, case.H, case.Lk, D, dtype=x.dtype, device=dev)
            v = torch.empty_like(k)
            kv_ms = timed(lambda: sd.project_kv(ctx, wk, wv, k, v, case.H, stream))
            step_ms = timed(lambda: sd.attention_block_kv(x, wq, k, v, wo, bo, out, ws, case.scale,
                                                          stream))
            res["cross_cached_context"] = {
                "per_step_us": round(step_ms * 1e3, 2),
                "per_prompt_kv_us": round(kv_ms * 1e3, 2),
                "per_step_flops": case.flops - 4 * case.B * case.Lk * case.Cc * case.C}
    return res


def bench_norm_act(torch, sd, wl, dev, stream, launches=50, reps=3):
    """The specialised kernels of Sec. 3.1 at the 64x64 level: group
    normalisation of [2, 320, 64x64] (32 groups) and GEGLU of [8192, 2560] ->
    [8192, 1280], launched back to back behind a busy GPU."""

    def timed(call):
        call()
        torch.cuda.synchronize()
        best = None
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(20_000_000)
            e0.record(stream)
            for _ in range(launches):
                call()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / launches
            best = ms if best is None else min(best, ms)
        return best

    gc = wl.NORM_CASES["gn64"]
    x, gamma, beta = (torch.from_numpy(t).to(dev) for t in wl.norm_inputs(gc))
    y = torch.empty_like(x)
    gn_ms = timed(lambda: sd.group_norm(x, wl.GN_GROUPS, y, gamma, beta, wl.GN_EPS, stream))
    ec = wl.GEGLU_CASES["geglu64"]
    h = torch.from_numpy(wl.geglu_inputs(ec)).to(dev)
    o = torch.empty(ec.M, ec.F, dtype=h.dtype, device=dev)
    ge_ms = timed(lambda: sd.geglu(h, o, stream))
    res = {}
    for name, ms, nbytes, shape in (("group_norm", gn_ms, gc.bytes, f"[{gc.B},{gc.C},{gc.HW}] G{wl.GN_GROUPS}"),
                                    ("geglu", ge_ms, ec.bytes, f"[{ec.M},{2 * ec.F}] -> [{ec.M},{ec.F}]")):
        gbs = nbytes / (ms * 1e-3) / 1e9
        res[name] = {"us": round(ms * 1e3, 2), "bytes": nbytes, "gbs": round(gbs, 1),
                     "frac_hbm": round(gbs / PEAK_HBM_GBS, 4), "shape": shape}
    return res


def bench_conv(torch, sd, wl, dev, stream, launches=30, reps=3):
    """The UNet's 3x3 convolution at the 64x64 level (2 x 320 x 64 x 64 -> 320
    channels) by Winograd F(4x4, 3x3), launched back to back behind a busy GPU;
    the kernel transform (once per layer) is timed separately.  Also the same
    convolution through torch.nn.functional.conv2d (MIOpen) for reference."""

    def timed(call):
        call()
        torch.cuda.synchronize()
        best = None
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(20_000_000)
            e0.record(stream)
            for _ in range(launches):
                call()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / launches
            best = ms if best is None else min(best, ms)
        return best

    B, C, L = 2, wl.CONV_LEVELS[64], 64
    x, w, b = (torch.from_numpy(t).to(dev) for t in wl.make_conv(B, C, C, L, L, wl.SEED0 + 51))
    u = torch.empty(36, C, C, dtype=x.dtype, device=dev)
    ws = torch.empty(sd.conv3x3_workspace(B, C, C, L, L), dtype=torch.uint8, device=dev)
    y = torch.empty(B, C, L, L, dtype=x.dtype, device=dev)
    wt_ms = timed(lambda: sd.winograd_weights(w, u, stream))
    ms = timed(lambda: sd.conv3x3(x, u, y, ws, b, stream))
    ref_ms = timed(lambda: torch.nn.functional.conv2d(x, w, b, padding=1))
    direct = 2 * 9 * C * C * L * L * B
    tiles = B * (L // 4) * (L // 4)
    wino = 2 * 36 * tiles * C * C
    return {"us": round(ms * 1e3, 2), "direct_equivalent_tflops": round(direct / (ms * 1e-3) / 1e12, 1),
            "winograd_product_tflops": round(wino / (ms * 1e-3) / 1e12, 1),
            "direct_flops": direct, "winograd_product_flops": wino,
            "weight_transform_us": round(wt_ms * 1e3, 2),
            "torch_conv2d_us": round(ref_ms * 1e3, 2),
            "shape": f"x [{B},{C},{L},{L}] w [{C},{C},3,3]"}


def copy_calibration(torch, dev, stream, nbytes=256 << 20, reps=3):
    """A plain device copy of known size: its FETCH_SIZE / WRITE_SIZE counter
    readings give the scale between those counters and bytes moved."""
    src = torch.ones(nbytes // 2, dtype=torch.float16, device=dev)
    dst = torch.empty_like(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    dst.copy_(src)
    e0.record(stream)
    for _ in range(reps):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"bytes_read": nbytes, "bytes_written": nbytes, "avg_kernel_us": round(ms * 1e3, 2),
            "gbs": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)}


def recorded_traffic():
    """HBM bytes per launch of the 64x64 self-attention kernel from the
    committed rocprofv3 counter runs (FETCH_SIZE, WRITE_SIZE, scaled by a plain
    copy's readings), or None when the kernel source changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "attn_l64_self_hbm_traffic.json")
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    h = hashlib.sha256()
    for f in rec["sources"]:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    if h.hexdigest() != rec["sources_sha256"]:
        return None
    return int(rec["fetch_kib"] * rec["fetch_scale"] * 1024 + rec["write_kib"] * rec["write_scale"] * 1024)


def cpu_baseline(wl, self_case, cross_case, rows_per_head):
    import oracle
    q, k, v = wl.case_inputs(self_case)
    rows = wl.sample_rows(self_case.B, self_case.H, self_case.Lq, rows_per_head, seed=1)
    t0 = time.perf_counter()
    oracle.attention(q, k, v, self_case.scale, rows=rows)
    t_self = time.perf_counter() - t0
    cq, ck, cv = wl.case_inputs(cross_case)
    crows = wl.sample_rows(cross_case.B, cross_case.H, cross_case.Lq, cross_case.Lq, seed=2)
    t0 = time.perf_counter()
    oracle.attention(cq, ck, cv, cross_case.scale, rows=crows)
    t_cross = time.perf_counter() - t0
    flops = 4 * (rows.size * self_case.Lk + crows.size * cross_case.Lk) * self_case.D
    cpu = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"value": round(flops / (t_self + t_cross) / 1e12, 8), "unit": "TFLOP/s",
            "cores": oracle.num_threads(), "kind": "oracle", "cpu": cpu,
            "sample": f"{rows.size} self-attention rows and {crows.size} cross-attention rows of the step "
                      f"(fp64 three-pass, {t_self + t_cross:.1f} s)",
            "seconds": round(t_self + t_cross, 3)}


if __name__ == "__main__":
    main()
