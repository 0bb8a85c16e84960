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
  sweep         one UNet evaluation (16 blocks, self- then cross-attention)
                per denoising step over 20 steps with per-step inputs, and
                each level's kernels against their rooflines
  peaks_measured  what the chip sustains, from the measurement kernels of
                libsdattn_probes.so: fp16 MFMA rate and shader clock under
                that load, v_exp_f32 / v_fma_f32 rates and their overlap with
                the matrix core, HBM streaming, and a plain copy with the
                cross-attention kernel's grid and bytes (cold)
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
    ap.add_argument("--cpu-rows-per-head", type=int, default=1536,
                    help="self-attention rows per (b, h) the oracle times")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 256 MiB device copy (scales the HBM traffic counters)")
    ap.add_argument("--no-sweep", action="store_true", help="skip the 20-step UNet sweep")
    ap.add_argument("--no-probes", action="store_true", help="skip the measured-peak probes")
    ap.add_argument("--lk-scaling", action="store_true",
                    help="also time the 64x64 self-attention kernel at Lk = 256 .. 4096 (fixed cost and "
                         "cost per 128-key tile by a least-squares line)")
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

    if not args.no_probes:
        peaks = measured_peaks(torch, dev, stream)
        out["peaks_measured"] = peaks
        mp = peaks["mfma_f16_tflops"]
        roofline["peak_measured"] = mp
        roofline["frac_measured"] = round(self_tflops / mp, 4)
        # the matrix core alone on random operands: the ceiling with data that toggles
        mpn = peaks["mfma_f16_noise_tflops"]
        roofline["peak_measured_random_operands"] = mpn
        roofline["frac_measured_random_operands"] = round(self_tflops / mpn, 4)
        hp = peaks["hbm_copy_gbs"]
        out["cross"]["peak_measured_gbs"] = hp
        out["cross"]["warm_frac_measured"] = round(cross_gbs / hp, 4)
        if "cold_gbs" in out["cross"]:
            out["cross"]["cold_frac_measured"] = round(out["cross"]["cold_gbs"] / hp, 4)
        out["cross"]["floor"] = cross_floor(torch, wl, dev, stream, cross_case)

    if not args.no_sweep:
        out["sweep"] = bench_sweep(torch, sd, wl, dev, stream)

    if args.lk_scaling:
        out["lk_scaling"] = lk_scaling(torch, sd, wl, dev, stream, self_case)

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
        if kind == "self":
            # the same projections through torch (hipBLASLt), for comparison only:
            # Q, K, V as one [C, 3C] product and the output projection with bias
            x2 = x.reshape(-1, case.C)
            w3 = torch.cat([wq, wk, wv], 0).contiguous()
            qkv_ms = timed(lambda: torch.nn.functional.linear(x2, w3))
            out_ms = timed(lambda: torch.nn.functional.linear(x2, wo, bo))
            res[kind]["torch_projections_us"] = {"qkv": round(qkv_ms * 1e3, 2), "out": round(out_ms * 1e3, 2),
                                                 "total": round((qkv_ms + out_ms) * 1e3, 2)}
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


def _events_ms(torch, stream, call, reps=3):
    """Best of `reps` single timed calls (after one untimed call), events on `stream`."""
    call()
    torch.cuda.synchronize()
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        call()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    return best


def measured_peaks(torch, dev, stream):
    """Sustained rates from the measurement kernels (libsdattn_probes.so).

    mfma_f16_tflops    back-to-back v_mfma_f32_32x32x16_f16, two waves per SIMD
    shader_clock_ghz   the shader-clock counter against the 100 MHz counter
                       during that stream (clock under matrix-core load)
    *_noise_*          the same on random operands (bits toggling like real
                       activations) and the clock it sustains
    exp / fma          wave64 instructions per SIMD per shader cycle, alone
    overlap_*          time of one MFMA wave + one VALU wave per SIMD against
                       each alone: 0 = the sum of both (no overlap), 1 = the
                       longer of the two (full overlap)
    tile_mix_*         the D = 40 self-attention tile's instructions without
                       data movement, per 32x32 pair and SIMD, with and without
                       exponentials, near-constant or toggling operands, the
                       two waves of a SIMD in step or half an iteration apart;
                       the shader clock during each and the cycles per pair
    hbm_*_gbs          1 GiB copy (read + write bytes / time) and 2 GiB read
    """
    from paper_2304_11267_amd import probes
    blocks = 512                                   # 2 workgroups of 8 waves per CU
    out = torch.empty(blocks * 512, dtype=torch.float32, device=dev)
    clk = torch.zeros(4, dtype=torch.int64, device=dev)
    it_m, it_v = 8000, 8000

    def run(mode, im, iv, c=None):
        return _events_ms(torch, stream, lambda: probes.mix(mode, blocks, im, iv, out, c, stream))

    t_mfma = run(probes.MIX_MFMA, it_m, 0, clk)
    torch.cuda.synchronize()
    t0, t1, r0, r1 = (int(x) for x in clk.cpu().tolist())
    clock_ghz = (t1 - t0) / ((r1 - r0) / 100e6) / 1e9 if r1 > r0 else None
    mfma_tf = blocks * 8 * it_m * probes.MFMA_FLOPS_PER_ITER / (t_mfma * 1e-3) / 1e12
    # the same stream on random operands (a realistic matrix-core ceiling: the
    # clock it sustains drops with the bits that toggle)
    clk.zero_()
    t_mfma_n = run(probes.MIX_MFMA_NOISE, it_m, 0, clk)
    t0, t1, r0, r1 = (int(x) for x in clk.cpu().tolist())
    clock_n = (t1 - t0) / ((r1 - r0) / 100e6) / 1e9 if r1 > r0 else None
    mfma_tf_n = blocks * 8 * it_m * probes.MFMA_FLOPS_PER_ITER / (t_mfma_n * 1e-3) / 1e12
    t_fma = run(probes.MIX_FMA, 0, it_v)
    t_exp = run(probes.MIX_EXP, 0, it_v // 2)
    simds = 256 * 4
    waves_per_simd = blocks * 8 / simds
    res = {"mfma_f16_tflops": round(mfma_tf, 1),
           "mfma_f16_frac_of_datasheet": round(mfma_tf / PEAK_F16_TFLOPS, 4),
           "shader_clock_ghz": round(clock_ghz, 3) if clock_ghz else None,
           "mfma_f16_noise_tflops": round(mfma_tf_n, 1),
           "mfma_f16_noise_frac_of_datasheet": round(mfma_tf_n / PEAK_F16_TFLOPS, 4),
           "shader_clock_noise_ghz": round(clock_n, 3) if clock_n else None}
    if clock_ghz:
        cyc = lambda ms: ms * 1e-3 * clock_ghz * 1e9
        res["fma_cycles_per_wave64_op"] = round(cyc(t_fma) / (waves_per_simd * it_v * 16), 2)
        res["exp_cycles_per_wave64_op"] = round(cyc(t_exp) / (waves_per_simd * (it_v // 2) * 16), 2)
        res["mfma32x32x16_cycles"] = round(cyc(t_mfma) / (waves_per_simd * it_m * 4), 2)
    # one MFMA wave and one VALU wave per SIMD (waves 0-3 and 4-7 of each workgroup)
    half_m = run(probes.MIX_MFMA_HALF, it_m // 2, 0)
    for name, both_mode, alone_mode, iv in (("fma", probes.MIX_MFMA_FMA, probes.MIX_FMA_HALF, it_v),
                                            ("exp", probes.MIX_MFMA_EXP, probes.MIX_EXP_HALF, it_v // 2)):
        alone_v = run(alone_mode, 0, iv)
        both = run(both_mode, it_m // 2, iv)
        lo, hi = max(half_m, alone_v), half_m + alone_v
        res[f"overlap_mfma_{name}"] = round((hi - both) / (hi - lo), 3) if hi > lo else None
        res[f"mfma_{name}_us"] = {"mfma_alone": round(half_m * 1e3, 1), f"{name}_alone": round(alone_v * 1e3, 1),
                                  "together": round(both * 1e3, 1)}
    # the D = 40 tile's instruction mix without data movement: ns per 32x32 pair per SIMD,
    # the shader clock during it, and the shader cycles per pair at that clock
    ti = 4000
    pairs_per_simd = 2 * ti * 2           # two waves per SIMD, two pairs per iteration
    tile_clock, tile_cycles = {}, {}
    for key, exps, noise in (("tile_mix_ns_per_pair", True, False), ("tile_mix_no_exp_ns_per_pair", False, False),
                             ("tile_mix_noise_ns_per_pair", True, True),
                             ("tile_mix_noise_no_exp_ns_per_pair", False, True)):
        clk.zero_()
        t = _events_ms(torch, stream, lambda: probes.tile(256, ti, exps, out, noise, clk, stream))
        res[key] = round(t * 1e6 / pairs_per_simd, 2)
        t0, t1, r0, r1 = (int(x) for x in clk.cpu().tolist())
        if r1 > r0:
            ghz = (t1 - t0) / ((r1 - r0) / 100e6) / 1e9
            name = key[len("tile_mix_"):-len("_ns_per_pair")] or "plain"
            tile_clock[name] = round(ghz, 3)
            tile_cycles[name] = round(res[key] * ghz, 1)
    # the same with the second wave of each SIMD started half an iteration late
    clk.zero_()
    t = _events_ms(torch, stream, lambda: probes.tile(256, ti, True, out, True, clk, stream, stagger=13))
    res["tile_mix_noise_staggered_ns_per_pair"] = round(t * 1e6 / pairs_per_simd, 2)
    t0, t1, r0, r1 = (int(x) for x in clk.cpu().tolist())
    if r1 > r0:
        ghz = (t1 - t0) / ((r1 - r0) / 100e6) / 1e9
        tile_clock["noise_staggered"] = round(ghz, 3)
        tile_cycles["noise_staggered"] = round(res["tile_mix_noise_staggered_ns_per_pair"] * ghz, 1)
    res["tile_mix_clock_ghz"] = tile_clock
    res["tile_mix_cycles_per_pair"] = tile_cycles
    # HBM streaming (buffers far beyond the 256 MB Infinity Cache)
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device=dev)
    dst = torch.empty(n, dtype=torch.uint8, device=dev)
    src.fill_(1)
    cblocks = 256 * 32
    t_copy = _events_ms(torch, stream, lambda: probes.copy(src, dst, n, cblocks, stream))
    big = torch.empty(2 * n, dtype=torch.uint8, device=dev)
    big.fill_(3)
    sink = torch.empty(cblocks * 256, dtype=torch.int32, device=dev)
    t_read = _events_ms(torch, stream, lambda: probes.read(big, 2 * n, sink, cblocks, stream))
    res["hbm_copy_gbs"] = round(2 * n / (t_copy * 1e-3) / 1e9, 1)
    res["hbm_read_gbs"] = round(2 * n / (t_read * 1e-3) / 1e9, 1)
    res["hbm_copy_frac_of_datasheet"] = round(res["hbm_copy_gbs"] / PEAK_HBM_GBS, 4)
    del src, dst, big
    return res


def cross_floor(torch, wl, dev, stream, case, nsets=40):
    """The cross-attention kernel's bytes moved by a plain copy with its grid
    (workgroups of 8, 4 or 2 waves of 32 query rows, each reading its head's K
    and V and copying its Q rows to O), inputs rotated over `nsets` sets as in
    the cold protocol: the floor for any kernel that moves those bytes that
    way; and Q to O as one plain copy, the floor for moving them at all."""
    from paper_2304_11267_amd import probes
    sets = []
    g = torch.Generator(device=dev)
    g.manual_seed(case.seed)
    for _ in range(nsets):
        q = torch.randn(case.B, case.H, case.Lq, case.D, device=dev, generator=g).half()
        k = torch.randn(case.B, case.H, case.Lk, case.D, device=dev, generator=g).half()
        v = torch.randn(case.B, case.H, case.Lk, case.D, device=dev, generator=g).half()
        sets.append((q, k, v, torch.empty_like(q)))
    sink = torch.empty(case.B * case.H * ((case.Lq + 63) // 64), dtype=torch.int32, device=dev)
    launches = 5 * nsets

    def batch(rot, waves):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(20_000_000)
        e0.record(stream)
        for i in range(launches):
            s = sets[i % nsets] if rot else sets[0]
            probes.strip_copy(*s, sink, waves, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / launches

    res = {}
    for waves in (8, 4, 2):
        for s in sets:
            probes.strip_copy(*s, sink, waves, stream)
        torch.cuda.synchronize()
        cold = min(batch(True, waves) for _ in range(3))
        warm = min(batch(False, waves) for _ in range(3))
        res[f"waves{waves}"] = {"cold_us": round(cold * 1e3, 3),
                                "cold_gbs": round(case.bytes / (cold * 1e-3) / 1e9, 1),
                                "warm_us": round(warm * 1e3, 3),
                                "warm_gbs": round(case.bytes / (warm * 1e-3) / 1e9, 1)}
    # Q -> O as one plain grid-stride copy (no K, V; 2048 workgroups of 256
    # threads, 16 bytes per lane): what the chip does with these bytes at best
    qbytes = case.B * case.H * case.Lq * case.D * 2
    blocks = 2048

    def plain(rot):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(20_000_000)
        e0.record(stream)
        for i in range(launches):
            s = sets[i % nsets] if rot else sets[0]
            probes.copy(s[0], s[3], qbytes, blocks, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / launches

    for s in sets:
        probes.copy(s[0], s[3], qbytes, blocks, stream)
    torch.cuda.synchronize()
    cold = min(plain(True) for _ in range(3))
    warm = min(plain(False) for _ in range(3))
    res["plain_copy"] = {"cold_us": round(cold * 1e3, 3), "cold_gbs": round(2 * qbytes / (cold * 1e-3) / 1e9, 1),
                         "warm_us": round(warm * 1e3, 3), "warm_gbs": round(2 * qbytes / (warm * 1e-3) / 1e9, 1),
                         "bytes": 2 * qbytes}
    res["what"] = ("plain copy of Q to O plus reads of K, V in workgroups of 8, 4 or 2 strips of 32 rows "
                   f"(the cross kernel launches 4), {nsets} rotated input sets (cold) or one (warm), "
                   "back-to-back launches; plain_copy: Q to O alone, grid-stride over 2048 workgroups")
    return res


def bench_sweep(torch, sd, wl, dev, stream, steps=20, launches=20):
    """Config 5: the 32 attention calls of one UNet evaluation (16 blocks,
    self- then cross-attention) at each of 20 denoising steps, every call on
    its own inputs (N(0,1) drawn on the GPU from that call's seed; the timing
    does not depend on the values on the fast path).  Reported: ms per UNet
    evaluation over the 20 steps (one event pair around all 640 calls), and
    per level and kind the average kernel time from back-to-back launches
    with its roofline fraction."""
    calls = []
    for t in range(steps):
        for case in wl.sweep_cases(t):
            g = torch.Generator(device=dev)
            g.manual_seed(case.seed)
            q = torch.randn(case.B, case.H, case.Lq, case.D, device=dev, generator=g).half()
            k = torch.randn(case.B, case.H, case.Lk, case.D, device=dev, generator=g).half()
            v = torch.randn(case.B, case.H, case.Lk, case.D, device=dev, generator=g).half()
            calls.append((case, (q, k, v, torch.empty_like(q))))
    for case, s in calls[:32]:
        sd.forward(*s, case.scale, stream)
    torch.cuda.synchronize()
    best = None
    for _ in range(3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(20_000_000)
        e0.record(stream)
        for case, s in calls:
            sd.forward(*s, case.scale, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    per_eval_ms = best / steps
    flops_per_eval = sum(c.flops for c, _ in calls[:32])
    bytes_per_eval = sum(c.bytes for c, _ in calls[:32])
    levels = {}
    for level, (L, D) in sorted(wl.LEVELS.items(), reverse=True):
        for kind in ("self", "cross"):
            sel = [(c, s) for c, s in calls if c.Lq == L and c.D == D and c.name.endswith(kind)][:8]
            ms = back_to_back_ms(torch, sd, stream, [s for _, s in sel], sel[0][0].scale, launches=launches)
            c = sel[0][0]
            tf = c.flops / (ms * 1e-3) / 1e12
            gbs = c.bytes / (ms * 1e-3) / 1e9
            levels[f"{level}x{level}_{kind}"] = {
                "us": round(ms * 1e3, 2), "tflops": round(tf, 1), "frac_f16_peak": round(tf / PEAK_F16_TFLOPS, 4),
                "gbs": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                "calls_per_eval": sum(1 for cc, _ in calls[:32] if cc.Lq == L and cc.D == D
                                      and cc.name.endswith(kind)),
                "shape": f"B{c.B} H{c.H} Lq{c.Lq} Lk{c.Lk} D{c.D}"}
    del calls
    return {"ms_per_unet_eval": round(per_eval_ms, 4), "steps": steps, "calls_per_eval": 32,
            "flops_per_eval": flops_per_eval, "bytes_per_eval": bytes_per_eval,
            "tflops": round(flops_per_eval / (per_eval_ms * 1e-3) / 1e12, 1),
            "levels": levels,
            "inputs": "per call N(0,1) fp16 from torch's GPU generator seeded with the call's seed "
                      "(S0 + 1000(t+1) + 10b, +1 for cross)"}


def lk_scaling(torch, sd, wl, dev, stream, case, lks=(256, 512, 1024, 2048, 3072, 4096)):
    """The 64x64-level self-attention kernel (B2 H8 Lq 4096 D40, the same
    256-row workgroups) at several key counts: the least-squares line through
    the average launch times splits the kernel into a fixed part (launch,
    Q load, first tile, the key halves' merge, epilogue) and a cost per
    128-key tile of each key half (two tiles per 256 keys)."""
    pts = []
    for lk in lks:
        q, k, v = wl.make_qkv(case.B, case.H, case.Lq, lk, case.D, case.seed)
        qd, kd, vd = (torch.from_numpy(t).to(dev) for t in (q, k, v))
        ms = back_to_back_ms(torch, sd, stream, [(qd, kd, vd, torch.empty_like(qd))], case.scale,
                             launches=50)
        pts.append((lk, ms * 1e3))
    xs = np.array([p[0] / 256.0 for p in pts])   # 128-key tiles per key half
    ys = np.array([p[1] for p in pts])
    slope, icept = np.polyfit(xs, ys, 1)
    return {"points_us": {str(lk): round(us, 3) for lk, us in pts},
            "fixed_us": round(float(icept), 3), "per_tile_us": round(float(slope), 4),
            "tiles_at_4096": 16,
            "what": "B2 H8 Lq4096 D40 self-attention at Lk = 256..4096, back-to-back launches; "
                    "line through (tiles per key half, us)"}


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
    """The fp64 oracle timed on this host: a bounded row sample of the step
    (median of 3 runs) on every core the process may use, plus configs 1 and
    2 (the 8x8 and 16x16 self-attention) whole on all cores and on one."""
    import oracle
    cores = len(os.sched_getaffinity(0))
    q, k, v = wl.case_inputs(self_case)
    rows = wl.sample_rows(self_case.B, self_case.H, self_case.Lq, rows_per_head, seed=1)
    cq, ck, cv = wl.case_inputs(cross_case)
    crows = wl.sample_rows(cross_case.B, cross_case.H, cross_case.Lq, cross_case.Lq, seed=2)
    runs = []
    for _ in range(3):
        t0 = time.perf_counter()
        oracle.attention(q, k, v, self_case.scale, rows=rows, nthreads=cores)
        oracle.attention(cq, ck, cv, cross_case.scale, rows=crows, nthreads=cores)
        runs.append(time.perf_counter() - t0)
    t = float(np.median(runs))
    flops = 4 * (rows.size * self_case.Lk + crows.size * cross_case.Lk) * self_case.D
    small = {}
    for name in ("mid8_self", "l16_self"):
        case = wl.CASES[name]
        qq, kk, vv = wl.case_inputs(case)
        for n in (cores, 1):
            ts = []
            for _ in range(3):
                t0 = time.perf_counter()
                oracle.attention(qq, kk, vv, case.scale, nthreads=n)
                ts.append(time.perf_counter() - t0)
            small[f"{name}_{'all' if n == cores else 1}_cores"] = {
                "seconds": round(float(np.median(ts)), 4),
                "gflops": round(case.flops / float(np.median(ts)) / 1e9, 3), "threads": n}
    cpu = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"value": round(flops / t / 1e12, 8), "unit": "TFLOP/s",
            "cores": cores, "kind": "oracle", "cpu": cpu,
            "sample": f"{rows.size} self-attention rows and {crows.size} cross-attention rows of the step "
                      f"(fp64 three-pass on {cores} threads, median of 3 runs of {t:.1f} s)",
            "seconds": round(t, 3), "runs_s": [round(x, 3) for x in runs],
            "configs_1_2": small}


if __name__ == "__main__":
    main()
