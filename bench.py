#!/usr/bin/env python3
"""Throughput of the QuaRTZ W4A4 linear hot path on one MI355X.

Workload (default): the four linear layers of a FLUX.1-schnell-like joint
transformer block at 4096 image + 512 text tokens (M = 4608): QKV 3072->9216,
out 3072->3072, MLP fc1 3072->12288 and fc2 12288->3072, seeded synthetic
bf16 activations / weights / bias (workloads.py), LZS subgroup G_s = 16.

One step = one pass of the whole hot path over the block: the weight
pre-pack (RTN int4 + fp16 group scales) of the four layers, then for every
layer the activation quantizer (Stage 1 + LZS) and the W4A4 GEMM (fp8 MFMA,
per-group dequant, bias).  All inputs are resident in HBM before the timed
region.

Prints ONE JSON line (stdout).  value = GEMM tera-ops (2 M N K summed over the
layers) per second of whole steps, from K steps with no event between the
launches.  roofline = the GEMM kernel (the dominant one): algorithmic ops /
its average launch duration, from HIP events recorded on the launch stream
around every launch of K more steps run right after the timed ones (each
event is a barrier in the queue, so those steps are not the ones
ms_per_step is taken from), against the fp8 dense MFMA peak.
cpu_baseline = the CPU oracle on a bounded sample of the same workload (all
weights, the first --cpu-rows rows of every layer), on this host's cores.
roofline.traffic = HBM bytes per GEMM launch from the FETCH_SIZE / WRITE_SIZE
counters of a profiled run, each scaled by what the counter reads for a plain
device copy of known size (--copy-calibration); read from the committed
summary under profiles/ and reported only while the GEMM sources still hash
to the values recorded there (null otherwise).

Secondary sections of the same line (not part of `value`): the other
workloads of the benchmark set (config1, config2, batched_mlp, conv3x3), the
LDM and asymmetric settings, cold-cache and G_s-sweep timings, and
`attention`: LZS attention (quartz_lzs_attention) in the heads x dim and
group settings of Table 8 at the FLUX sequence length, with the stage
pipeline of one head broken down by stage.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP8_TFLOPS = 5000.0      # MI355X dense fp8 MFMA
PEAK_HBM_GBPS = 8000.0        # MI355X HBM3E
SETTLE_S = 0.25               # untimed load before the timed steps (clock settling)
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "w4a4_gemm_hbm_traffic_flux_block_m4608.md")
GEMM_SOURCES = [os.path.join(ROOT, "paper_2509_26436_amd", "csrc", f)
                for f in ("w4a4_linear.hip", "w4a4_linear_kernel.h", "w4a4_gemm_kernel.h", "w4a4_gemm.hip",
                          "w4a4_gemm_plain.hip",
                          "gemm_schedule.h", "quartz_internal.h", "lzs_device.h")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=50,
                    help="untimed steps before the timed ones (the GPU needs a few tens of "
                         "milliseconds of load to reach its steady clock: 5 steps leave the "
                         "timed steps ~10 %% slower)")
    ap.add_argument("--config", type=int, default=3, help="workload config index (workloads.py)")
    ap.add_argument("--lzs-group", type=int, default=16)
    ap.add_argument("--cpu-rows", type=int, default=1536,
                    help="rows per layer in the CPU-oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-attention", action="store_true",
                    help="skip the LZS attention settings of Table 8")
    ap.add_argument("--no-batched-mlp", action="store_true",
                    help="skip the batched FLUX MLP pipeline measurement (M = 18432)")
    ap.add_argument("--no-ldm", action="store_true",
                    help="skip the secondary sections: LDM setting (static activation scale), "
                         "asymmetric mode, implicit-GEMM convolutions, cold cache, the G_s "
                         "sweep and the clocks under load (the profiling runs use this)")
    ap.add_argument("--no-clocks", action="store_true",
                    help="do not start rocm-smi (a child process) for the clock readings")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 5 plain device-to-device copies of MIB MiB (the known-size "
                         "kernel that scales the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


def gemm_sources_sha256() -> str:
    h = hashlib.sha256()
    for p in GEMM_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(workload: str, gs: int):
    """HBM bytes per GEMM launch recorded in the committed counter summary, if
    it covers this workload and the GEMM sources have not changed since."""
    try:
        text = open(TRAFFIC_SUMMARY).read()
    except OSError:
        return None
    fields = dict(re.findall(r"^- (\w+): `([^`]*)`", text, flags=re.M))
    try:
        if (fields.get("gemm_sources_sha256") != gemm_sources_sha256()
                or fields.get("workload") != workload or int(fields.get("lzs_group", -1)) != gs):
            return None
        return float(fields["hbm_bytes_per_gemm_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(mib: int):
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    src.fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}), flush=True)


def layer_bytes(L, gs):
    quant = L.M * L.K * (2 + 0.5 + 1.0 / gs + 2.0 / 64)
    pack = L.N * L.K * (2 + 0.5 + 2.0 / 64 + 2.0 / 64)
    gemm = (L.M * L.K * (0.5 + 1.0 / gs + 2.0 / 64) + L.N * L.K * (0.5 + 2.0 / 64)
            + 2 * L.N + 2 * L.M * L.N)
    return quant, pack, gemm


def batched_mlp(q, W, torch, np, gs, reps=20):
    """The batched FLUX MLP at M = 18432 (4 images x 4608 tokens) as one pipeline:
    quantize x -> fc1 3072->12288 with the GELU epilogue -> quantize -> fc2
    12288->3072.  Per layer: median quantize and GEMM time over `reps` passes
    (timed_chain), and the end-to-end time against the
    sum of the two roofline times (quantize bytes at 8 TB/s + GEMM ops at the
    fp8 dense peak).  Then the same pipeline with fc2's input quantized in
    fc1's epilogue, its time, and whether fc2's output is bit-identical."""
    dev = torch.device("cuda", 0)
    cfg = W.CONFIGS[4]
    L1, L2 = cfg.layers
    to = lambda a: torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
    x1 = to(W.make_x(4, 0))
    w1, b1 = to(W.make_w(4, 0)), to(W.make_bias(4, 0))
    w2, b2 = to(W.make_w(4, 1)), to(W.make_bias(4, 1))
    pw1, pw2 = q.pack_weight(w1), q.pack_weight(w2)
    qa1 = q.quantize_act(x1, lzs_group=gs)
    ws1 = q.gemm_workspace(L1.M, L1.N, L1.K, dev)
    ws2 = q.gemm_workspace(L2.M, L2.N, L2.K, dev)
    y1 = q.w4a4_linear(qa1, pw1, b1, 1, workspace=ws1)
    qa2 = q.quantize_act(y1, lzs_group=gs)
    y2 = q.w4a4_linear(qa2, pw2, b2, 0, workspace=ws2)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    t = timed_chain(torch, np, stream,
                    [lambda: q.quantize_act(x1, lzs_group=gs, out=qa1),
                     lambda: q.w4a4_linear(qa1, pw1, b1, 1, out=y1, workspace=ws1),
                     lambda: q.quantize_act(y1, lzs_group=gs, out=qa2),
                     lambda: q.w4a4_linear(qa2, pw2, b2, 0, out=y2, workspace=ws2)], reps)
    # the same pipeline with fc2's input quantized in fc1's epilogue
    # (quartz_w4a4_linear_quantize): no bf16 fc1 output, no separate quantize
    qa2f = q.w4a4_linear_quantize(qa1, pw1, b1, 1, gs, workspace=ws1)
    y2f = q.w4a4_linear(qa2f, pw2, b2, 0, workspace=ws2)
    torch.cuda.synchronize()
    same = bool(torch.equal(y2f.view(torch.int16), y2.view(torch.int16)))
    tf = timed_chain(torch, np, stream,
                     [lambda: q.quantize_act(x1, lzs_group=gs, out=qa1),
                      lambda: q.w4a4_linear_quantize(qa1, pw1, b1, 1, gs, out=qa2f, workspace=ws1),
                      lambda: q.w4a4_linear(qa2f, pw2, b2, 0, out=y2f, workspace=ws2)], reps)
    fused = {"step": "quantize + fc1 (GELU; its epilogue quantizes the output for fc2) + fc2",
             "quantize_us": round(tf[0], 2), "fc1_quantize_us": round(tf[1], 2),
             "fc2_gemm_us": round(tf[2], 2), "end_to_end_us": round(tf.sum(), 2),
             "unfused_end_to_end_us": round(t.sum(), 2),
             "speedup": round(t.sum() / tf.sum(), 4),
             "fc2_output_identical": same}
    out = []
    for li, L in enumerate((L1, L2)):
        qb, _, _ = layer_bytes(L, gs)
        ops = 2.0 * L.M * L.N * L.K
        tq, tg = t[2 * li], t[2 * li + 1]
        roof = qb / (PEAK_HBM_GBPS * 1e3) + ops / (PEAK_FP8_TFLOPS * 1e6)      # us
        out.append({"layer": L.name, "M": L.M, "K": L.K, "N": L.N,
                    "quantize_us": round(tq, 2), "quantize_gbps": round(qb / (tq * 1e3), 1),
                    "gemm_us": round(tg, 2), "gemm_tflops": round(ops / (tg * 1e6), 1),
                    "end_to_end_us": round(tq + tg, 2), "roofline_us": round(roof, 2),
                    "frac": round(roof / (tq + tg), 4)})
    return {"workload": cfg.name, "lzs_group": gs,
            "step": "quantize + fc1 (GELU) + quantize + fc2", "per_layer": out,
            "fused_quantize": fused}


def timed_chain(torch, np, stream, calls, reps):
    """Median HIP-event time (us) of each launch in `calls` over `reps` passes
    of the whole chain, queued back to back after two untimed passes with one
    synchronization at the end: every launch but the very first follows
    another kernel, as inside a step, so no timed launch starts from an idle
    queue."""
    evs = []
    for _ in range(reps + 2):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
        ev[0].record(stream)
        for k, call in enumerate(calls):
            call()
            ev[k + 1].record(stream)
        evs.append(ev)
    torch.cuda.synchronize()
    t = np.array([[ev[k].elapsed_time(ev[k + 1]) for k in range(len(calls))] for ev in evs[2:]])
    return np.median(t, axis=0) * 1e3


def copy_ceiling_us(torch, np, stream, moved_bytes, reps=20):
    """Median time (us) of a plain device-to-device copy that moves
    `moved_bytes` in all (half read, half written), launched back to back
    (timed_chain), and the bytes it moves: the measured ceiling a streaming
    kernel of that size is compared with."""
    n = max(256, int(moved_bytes // 2) // 256 * 256)
    src = torch.empty(n, dtype=torch.uint8, device=torch.device("cuda", 0))
    src.fill_(1)
    dst = torch.empty_like(src)
    t = timed_chain(torch, np, stream, [lambda: dst.copy_(src)], reps)[0]
    del src, dst
    return float(t), 2 * n


def config_layers(q, W, torch, np, config, gs, reps=20):
    """The other workloads of the benchmark set, layer by layer (the single
    256 x 1152 -> 1152 linear; the PixArt-Sigma 1024px block): per layer the
    quantizer (GB/s, fraction of the HBM peak and of a same-size device copy
    timed in the same run) and the GEMM through the workspace entry point
    (TFLOP/s, fraction of the fp8 peak), medians of `reps` launches
    (timed_chain); config 1 also without bias."""
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream()
    cfg = W.CONFIGS[config]
    to = lambda a: torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
    out = []
    for li, L in enumerate(cfg.layers):
        x, w, b = to(W.make_x(config, li)), to(W.make_w(config, li)), to(W.make_bias(config, li))
        qa = q.quantize_act(x, gs)
        pw = q.pack_weight(w)
        ws = q.gemm_workspace(L.M, L.N, L.K, dev)
        y = q.w4a4_linear(qa, pw, b, L.epilogue, workspace=ws)
        calls = [lambda: q.quantize_act(x, gs, out=qa),
                 lambda: q.w4a4_linear(qa, pw, b, L.epilogue, out=y, workspace=ws)]
        if config == 1:
            calls.append(lambda: q.w4a4_linear(qa, pw, None, L.epilogue, out=y, workspace=ws))
        t = timed_chain(torch, np, stream, calls, reps)
        qb, _, _ = layer_bytes(L, gs)
        tc, moved = copy_ceiling_us(torch, np, stream, qb, reps)
        ops = 2.0 * L.M * L.N * L.K
        r = {"layer": L.name, "M": L.M, "K": L.K, "N": L.N,
             "quantize_us": round(t[0], 2), "quantize_gbps": round(qb / (t[0] * 1e3), 1),
             "quantize_frac": round(qb / (t[0] * 1e3) / PEAK_HBM_GBPS, 4),
             "copy_us": round(tc, 2), "copy_gbps": round(moved / (tc * 1e3), 1),
             "quantize_copy_frac": round(tc / t[0] * qb / moved, 4),
             "gemm_us": round(t[1], 2), "gemm_tflops": round(ops / (t[1] * 1e6), 1),
             "gemm_frac": round(ops / (t[1] * 1e6) / PEAK_FP8_TFLOPS, 4)}
        if config == 1:
            r["gemm_no_bias_us"] = round(t[2], 2)
            r["gemm_no_bias_tflops"] = round(ops / (t[2] * 1e6), 1)
        out.append(r)
        del x, w, b, qa, pw, ws, y
    tot_ops = sum(2.0 * L.M * L.N * L.K for L in cfg.layers)
    tot_us = sum(r["gemm_us"] for r in out)
    return {"workload": cfg.name, "lzs_group": gs,
            "step": "quantize_act + w4a4_linear (workspace entry point) per layer"
                    + ("; the GEMM again without bias" if config == 1 else ""),
            "gemm_tflops": round(tot_ops / (tot_us * 1e6), 1),
            "gemm_frac": round(tot_ops / (tot_us * 1e6) / PEAK_FP8_TFLOPS, 4),
            "per_layer": out}


def ldm_layers(q, W, torch, np, cfg, dev_in, gs, reps=20):
    """The LDM setting (static per-tensor activation scale, per-channel weight
    scales; the K loop is pure integer MFMA) on the same layers: per layer the
    static quantizer and GEMM times (timed_chain).  The static scale is fixed once from
    the synthetic tensor (max |x| / 127, outside the timed region)."""
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream()
    out = []
    for li, ((x, w, b), L) in enumerate(zip(dev_in, cfg.layers)):
        s = float(x.abs().max().float().item()) / 127.0
        qa = q.quantize_act_static(x, s, gs)
        pw = q.pack_weight_per_channel(w)
        ws = q.gemm_workspace(L.M, L.N, L.K, dev)
        y = q.w4a4_linear_static(qa, pw, s, b, L.epilogue, workspace=ws)
        torch.cuda.synchronize()
        t = timed_chain(torch, np, stream,
                        [lambda: q.quantize_act_static(x, s, gs, out=qa),
                         lambda: q.w4a4_linear_static(qa, pw, s, b, L.epilogue, out=y, workspace=ws)],
                        reps)
        ops = 2.0 * L.M * L.N * L.K
        out.append({"layer": L.name, "quantize_us": round(t[0], 2), "gemm_us": round(t[1], 2),
                    "gemm_tflops": round(ops / (t[1] * 1e6), 1),
                    "gemm_frac": round(ops / (t[1] * 1e6) / PEAK_FP8_TFLOPS, 4)})
        del qa, pw, ws, y
    tot_ops = sum(2.0 * L.M * L.N * L.K for L in cfg.layers)
    tot_us = sum(r["gemm_us"] for r in out)
    return {"step": "quantize_act_static + w4a4_linear_static (workspace) per layer",
            "gemm_tflops": round(tot_ops / (tot_us * 1e6), 1),
            "gemm_frac": round(tot_ops / (tot_us * 1e6) / PEAK_FP8_TFLOPS, 4),
            "per_layer": out}


def asym_layers(q, W, torch, np, cfg, dev_in, gs, reps=20):
    """The asymmetric mode (per-group zero points; one extra fp16 correction
    MFMA per tile) on the same layers: per layer the quantizer and GEMM times
    (timed_chain).  The weight group sums are computed once, outside."""
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream()
    out = []
    for (x, w, b), L in zip(dev_in, cfg.layers):
        qa = q.quantize_act(x, gs, mode=q.MODE_ASYMMETRIC)
        pw = q.pack_weight(w)
        sums = q.weight_group_sums(pw)
        ws = q.gemm_workspace(L.M, L.N, L.K, dev)
        y = q.w4a4_linear_asym(qa, pw, sums, b, L.epilogue, workspace=ws)
        torch.cuda.synchronize()
        t = timed_chain(torch, np, stream,
                        [lambda: q.quantize_act(x, gs, out=qa, mode=q.MODE_ASYMMETRIC),
                         lambda: q.w4a4_linear_asym(qa, pw, sums, b, L.epilogue, out=y, workspace=ws)],
                        reps)
        ops = 2.0 * L.M * L.N * L.K
        out.append({"layer": L.name, "quantize_us": round(t[0], 2), "gemm_us": round(t[1], 2),
                    "gemm_tflops": round(ops / (t[1] * 1e6), 1),
                    "gemm_frac": round(ops / (t[1] * 1e6) / PEAK_FP8_TFLOPS, 4)})
        del qa, pw, sums, ws, y
    tot_ops = sum(2.0 * L.M * L.N * L.K for L in cfg.layers)
    tot_us = sum(r["gemm_us"] for r in out)
    return {"step": "quantize_act (asymmetric) + w4a4_linear_asym (workspace) per layer",
            "gemm_tflops": round(tot_ops / (tot_us * 1e6), 1),
            "gemm_frac": round(tot_ops / (tot_us * 1e6) / PEAK_FP8_TFLOPS, 4),
            "per_layer": out}


def conv_layers(q, W, torch, np, gs, reps=20):
    """The SDXL UNet 3 x 3 convolutions (config 5) as implicit GEMMs: per layer
    the feature map's quantizer and the convolution (quartz_w4a4_conv3x3,
    workspace entry point), then the same in the LDM setting (static
    quantizer, quartz_w4a4_conv3x3_static); times by timed_chain.  The
    quantizer reads the H x W x C map once (the im2col matrix would be 9x
    larger and is never formed)."""
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream()
    cfg = W.CONFIGS[5]
    to = lambda a: torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
    out = []
    for li, L in enumerate(cfg.layers):
        C, H = L.K // 9, int(round(L.M ** 0.5))
        fm = to(W.make_feature_map(5, li)).reshape(L.M, C)
        w, b = to(W.make_w(5, li)), to(W.make_bias(5, li))
        ws = q.gemm_workspace(L.M, L.N, L.K, dev)
        pw = q.pack_weight(w)
        qa = q.quantize_act(fm, gs)
        y = q.w4a4_conv3x3(qa, pw, 1, H, H, b, 0, workspace=ws)
        t = timed_chain(torch, np, stream,
                        [lambda: q.quantize_act(fm, gs, out=qa),
                         lambda: q.w4a4_conv3x3(qa, pw, 1, H, H, b, 0, out=y, workspace=ws)], reps)
        s = float(fm.abs().max().float().item()) / 127.0
        pwc = q.pack_weight_per_channel(w)
        qs = q.quantize_act_static(fm, s, gs)
        ts = timed_chain(torch, np, stream,
                         [lambda: q.quantize_act_static(fm, s, gs, out=qs),
                          lambda: q.w4a4_conv3x3_static(qs, pwc, s, 1, H, H, b, 0, out=y, workspace=ws)],
                         reps)
        ops = 2.0 * L.M * L.N * L.K
        qbytes = L.M * C * (2 + 0.5 + 1.0 / gs + 2.0 / 64)
        out.append({"layer": L.name, "M": L.M, "C": C, "N": L.N,
                    "quantize_us": round(t[0], 2), "quantize_gbps": round(qbytes / (t[0] * 1e3), 1),
                    "conv_us": round(t[1], 2), "conv_tflops": round(ops / (t[1] * 1e6), 1),
                    "static_quantize_us": round(ts[0], 2), "static_conv_us": round(ts[1], 2),
                    "static_conv_tflops": round(ops / (ts[1] * 1e6), 1)})
        del fm, w, b, ws, pw, qa, y, pwc, qs
    tot_ops = sum(2.0 * L.M * L.N * L.K for L in cfg.layers)
    return {"workload": cfg.name + " (implicit GEMM)", "lzs_group": gs,
            "step": "quantize_act of the feature map + w4a4_conv3x3 per layer, then the static pair",
            "conv_tflops": round(tot_ops / (sum(r["conv_us"] for r in out) * 1e6), 1),
            "static_conv_tflops": round(tot_ops / (sum(r["static_conv_us"] for r in out) * 1e6), 1),
            "per_layer": out}


def cold_layers(q, torch, np, cfg, dev_in, outs, workspaces, gs, reps=20):
    """Cold-cache variant of each layer's quantizer and GEMM: a 512 MiB write
    (twice the 256 MB Infinity Cache, far beyond L2) before each timed launch,
    so no input is served from a cache that a previous launch warmed; times by
    timed_chain (the flushes are timed too and dropped)."""
    stream = torch.cuda.current_stream()
    scratch = torch.empty((512 << 20,), dtype=torch.uint8, device=torch.device("cuda", 0))
    flush = lambda: scratch.fill_(1)
    res = []
    for (x, w, b), (qa, pw, y), ws, L in zip(dev_in, outs, workspaces, cfg.layers):
        t = timed_chain(torch, np, stream,
                        [flush, lambda: q.quantize_act(x, lzs_group=gs, out=qa),
                         flush, lambda: q.w4a4_linear(qa, pw, b, L.epilogue, out=y, workspace=ws)],
                        reps)
        qb, _, _ = layer_bytes(L, gs)
        ops = 2.0 * L.M * L.N * L.K
        res.append({"layer": L.name, "quantize_us": round(t[1], 2),
                    "quantize_gbps": round(qb / (t[1] * 1e3), 1),
                    "gemm_us": round(t[3], 2), "gemm_tflops": round(ops / (t[3] * 1e6), 1)})
    del scratch
    return {"flush": "512 MiB device write before each timed launch", "per_layer": res}


ATTN_L = 4608                  # FLUX.1 joint sequence: 4096 image + 512 text tokens
ATTN_D = 128
ATTN_SETTINGS = [(h, gs) for h in (32, 40, 64) for gs in (8, 16, 32)]   # Table 8


def attention_bench(q, torch, np, reps=10):
    """LZS attention (quartz_lzs_attention) in the settings of Table 8:
    heads x dim 32 x 128, 40 x 128, 64 x 128 at G_s = 8, 16, 32, each at the
    FLUX sequence length L = 4608 (the table does not give one), seeded
    normal q, k, v.  Per setting the whole call (timed_chain); ops are the two
    products, 4 heads L^2 d.  Then the stages of one setting (32 heads,
    G_s = 16) launched one by one: the Q / K / V^T quantizers over all heads
    and the scores, softmax + quantize and PV of one head, with their
    algorithmic bytes (HBM-bound stages) or ops (products)."""
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream()
    L, d = ATTN_L, ATTN_D
    gen = torch.Generator(device=dev)
    gen.manual_seed(2509)
    hmax = max(h for h, _ in ATTN_SETTINGS)
    qkv = [torch.randn((hmax * L, d), generator=gen, device=dev).to(torch.bfloat16) for _ in range(3)]
    out = torch.empty((L, hmax * d), dtype=torch.bfloat16, device=dev)
    res = []
    for heads, gs in ATTN_SETTINGS:
        qh, kh, vh = (t[: heads * L] for t in qkv)
        ws = q.attention_workspace(heads, L, d, gs, dev)
        o = out[:, : heads * d]
        t = timed_chain(torch, np, stream,
                        [lambda: q.lzs_attention(qh, kh, vh, heads, gs, out=o, workspace=ws)], reps)[0]
        ops = 4.0 * heads * L * L * d
        res.append({"heads": heads, "dim": d, "lzs_group": gs, "L": L, "ms": round(t / 1e3, 4),
                    "tflops": round(ops / (t * 1e6), 1),
                    "frac": round(ops / (t * 1e6) / PEAK_FP8_TFLOPS, 4)})
        del ws
    # stages of the 32-head, G_s = 16 setting
    heads, gs = 32, 16
    qh, kh, vh = (t[: heads * L] for t in qkv)
    qa = q.quantize_act(qh, gs)
    ka = q.quantize_act(kh, gs)
    vt = q.quantize_vt(vh, heads, gs)
    S = torch.empty((L, L), dtype=torch.float32, device=dev)
    pa = q.softmax_quantize(S.zero_(), gs)
    pv_ws = torch.zeros((max(q.quartz_attn_pv_workspace_bytes(L, L, d), 16),), dtype=torch.uint8,
                        device=dev)
    o = out[:, :d]
    scale = float(np.float32(1.0 / np.sqrt(d)))
    calls = [lambda: q.quantize_act(qh, gs, out=qa), lambda: q.quantize_act(kh, gs, out=ka),
             lambda: q.quantize_vt(vh, heads, gs),
             lambda: q.attn_scores(qa, ka, 0, 0, L, L, scale, out=S),
             lambda: q.softmax_quantize(S, gs, out=pa),
             lambda: q.attn_pv(pa, vt, 0, d, out=o, workspace=pv_ws)]
    t = timed_chain(torch, np, stream, calls, reps)
    act = lambda rows, k: rows * k * (0.5 + 1.0 / gs + 2.0 / 64)     # LZS codes + FLAGs + scales
    qbytes = heads * L * d * 2 + act(heads * L, d)
    stages = [
        {"stage": "quantize Q (all heads)", "us": t[0], "bytes": qbytes},
        {"stage": "quantize K (all heads)", "us": t[1], "bytes": qbytes},
        {"stage": "quantize V^T (all heads)", "us": t[2], "bytes": qbytes},
        {"stage": "scores, one head (fp32 out)", "us": t[3], "ops": 2.0 * L * L * d,
         "bytes": 2 * act(L, d) + 4.0 * L * L},
        {"stage": "softmax + quantize, one head", "us": t[4], "bytes": 4.0 * L * L + act(L, L)},
        {"stage": "PV, one head", "us": t[5], "ops": 2.0 * L * L * d,
         "bytes": act(L, L) + act(d, L) + 2.0 * L * d},
    ]
    for r in stages:
        r["gbps"] = round(r["bytes"] / (r["us"] * 1e3), 1)
        if "ops" in r:
            r["tflops"] = round(r["ops"] / (r["us"] * 1e6), 1)
        r["us"] = round(float(r["us"]), 2)
        r["bytes"] = round(r["bytes"])
    del qkv, out, S, pv_ws
    return {"workload": f"LZS attention, L = {L}, dim {d}, seeded normal q, k, v",
            "step": "quartz_lzs_attention: Q, K, V^T quantizers, then per head scores -> "
                    "softmax + quantize -> PV",
            "settings": res,
            "stages_32x128_g16": stages}


def gs_sweep(q, torch, np, cfg, dev_in, outs, workspaces, reps=20):
    """The LZS subgroup sweep of Table 1 on the FLUX qkv layer: quantizer and
    GEMM at G_s = 8, 16, 32 and 64 (timed_chain); the paper's numbers are
    A100 latencies, context only."""
    stream = torch.cuda.current_stream()
    (x, w, b), (qa, pw, y), ws, L = dev_in[0], outs[0], workspaces[0], cfg.layers[0]
    res = []
    for g in (8, 16, 32, 64):
        qg = q.quantize_act(x, lzs_group=g)
        t = timed_chain(torch, np, stream,
                        [lambda: q.quantize_act(x, lzs_group=g, out=qg),
                         lambda: q.w4a4_linear(qg, pw, b, L.epilogue, out=y, workspace=ws)], reps)
        qb = L.M * L.K * (2 + 0.5 + 1.0 / g + 2.0 / 64)
        ops = 2.0 * L.M * L.N * L.K
        res.append({"lzs_group": g, "quantize_us": round(t[0], 2),
                    "quantize_gbps": round(qb / (t[0] * 1e3), 1), "gemm_us": round(t[1], 2),
                    "gemm_tflops": round(ops / (t[1] * 1e6), 1)})
        del qg
    return {"layer": L.name, "M": L.M, "K": L.K, "N": L.N, "per_lzs_group": res}


def gpu_clocks():
    """Current shader and memory clocks as rocm-smi reports them (a child
    process reading the driver's counters; None if unavailable)."""
    import subprocess
    try:
        out = subprocess.run(["rocm-smi", "--showclocks", "--json"], capture_output=True,
                             text=True, timeout=30).stdout
        card = next(iter(json.loads(out).values()))
        return {k: v for k, v in card.items() if "sclk" in k or "mclk" in k or "fclk" in k}
    except Exception:
        return None


def clocks_under_load(torch, launch, launch_us, seconds=3.0):
    """rocm-smi clock readings taken while `launch` (one GEMM) runs back to
    back for about `seconds`: a thread samples while the main thread keeps
    the queue full."""
    import threading
    samples = []

    def sampler():
        for _ in range(3):
            samples.append(gpu_clocks())

    th = threading.Thread(target=sampler)
    th.start()
    for _ in range(max(1, int(seconds * 1e6 / launch_us))):
        launch()
    torch.cuda.synchronize()
    th.join()
    return samples


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(a per-GPU share would be benchmarked as its own shape); use --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2509_26436_amd as q
    import workloads as W

    if not torch.cuda.is_available():
        log("bench.py needs a GPU")
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    dev = torch.device("cuda", 0)
    cfg = W.CONFIGS[args.config]
    gs = args.lzs_group
    layers = list(cfg.layers)
    if any(L.x_kind == "pipeline" for L in layers):
        log("config with a pipelined input is not a bench workload")
        sys.exit(2)

    # ---------------- inputs, resident in HBM
    t0 = time.time()
    host = []
    dev_in = []
    for li, L in enumerate(layers):
        xb = W.make_x(cfg.index, li)
        wb = W.make_w(cfg.index, li)
        bb = W.make_bias(cfg.index, li)
        host.append((xb, wb, bb))
        to = lambda a: torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        dev_in.append((to(xb), to(wb), to(bb)))
        log(f"layer {L.name}: M={L.M} K={L.K} N={L.N} generated")
    log(f"inputs ready in {time.time() - t0:.1f}s")

    # outputs and GEMM workspaces preallocated once (the step allocates nothing new)
    outs = []
    workspaces = []
    for (x, w, b), L in zip(dev_in, layers):
        qa = q.quantize_act(x, lzs_group=gs)
        pw = q.pack_weight(w)
        y = torch.empty((L.M, L.N), dtype=torch.bfloat16, device=dev)
        outs.append((qa, pw, y))
        workspaces.append(q.gemm_workspace(L.M, L.N, L.K, dev))
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    t_warm0 = time.perf_counter()

    def step(events=None):
        # the four weight packs, then quantize + GEMM layer by layer; with
        # `events` (per layer: pack start, pack end, quantize start, quantize
        # end, GEMM end) every launch is bracketed
        items = list(zip(dev_in, outs, workspaces, layers))
        for li, ((x, w, b), (qa, pw, y), ws, L) in enumerate(items):
            ev = events[li] if events is not None else None
            if ev: ev[0].record(stream)
            q.quartz_pack_weight(q._ptr(w), L.N, L.K, 64, q._ptr(pw.data), q._ptr(pw.scales),
                                 q._stream_handle())
            if ev: ev[1].record(stream)
        for li, ((x, w, b), (qa, pw, y), ws, L) in enumerate(items):
            ev = events[li] if events is not None else None
            if ev: ev[2].record(stream)
            q.quantize_act(x, lzs_group=gs, out=qa)
            if ev: ev[3].record(stream)
            q.w4a4_linear(qa, pw, b, L.epilogue, out=y, workspace=ws)
            if ev: ev[4].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Clock settling, part of the protocol: the GPU needs a few tens of
    # milliseconds of sustained load to reach its steady clock, so untimed
    # steps continue until SETTLE_S of work have run since the first warmup
    # step (at least the W warmup steps; reported as "settle").
    settle_steps = 0
    while time.perf_counter() - t_warm0 < SETTLE_S:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
        settle_steps += 10

    # the K timed steps: nothing between the launches but the launches
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for s in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps

    # then K more steps with an event pair around every launch, for the
    # per-kernel durations (each event is a barrier in the queue, so these
    # steps are slower as a whole and do not enter ms_per_step)
    ev_all = [[[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in layers]
              for _ in range(args.steps)]
    for s in range(args.steps):
        step(ev_all[s])
    torch.cuda.synchronize()
    # per launch: [step][layer] durations in ms; the means are what the
    # roofline divides by (the rocprofv3 statistics report averages), the
    # medians are reported beside them
    def durations(a, b):
        return np.array([[ev_all[s][li][a].elapsed_time(ev_all[s][li][b])
                          for li in range(len(layers))] for s in range(args.steps)])
    d_pack, d_quant, d_gemm = durations(0, 1), durations(2, 3), durations(3, 4)
    t_pack, t_quant, t_gemm = d_pack.mean(0), d_quant.mean(0), d_gemm.mean(0)
    m_quant, m_gemm = np.median(d_quant, 0), np.median(d_gemm, 0)

    ops = np.array([2.0 * L.M * L.N * L.K for L in layers])
    qbytes = np.array([layer_bytes(L, gs)[0] for L in layers])
    pbytes = np.array([layer_bytes(L, gs)[1] for L in layers])
    gbytes = np.array([layer_bytes(L, gs)[2] for L in layers])
    value = ops.sum() / (ms_per_step * 1e-3) / 1e12
    gemm_tflops = ops.sum() / (t_gemm.sum() * 1e-3) / 1e12
    gemm_tflops_median = ops.sum() / (m_gemm.sum() * 1e-3) / 1e12
    quant_gbps = qbytes.sum() / (t_quant.sum() * 1e-3) / 1e9
    quant_gbps_median = qbytes.sum() / (m_quant.sum() * 1e-3) / 1e9
    # the same bytes moved by a plain device copy, timed in this run
    copies = [copy_ceiling_us(torch, np, stream, qb) for qb in qbytes]
    pack_gbps = pbytes.sum() / (t_pack.sum() * 1e-3) / 1e9

    per_layer = []
    for li, L in enumerate(layers):
        per_layer.append({
            "layer": L.name, "M": L.M, "K": L.K, "N": L.N,
            "gemm_us": round(t_gemm[li] * 1e3, 2),
            "gemm_us_median": round(m_gemm[li] * 1e3, 2),
            "gemm_tflops": round(ops[li] / (t_gemm[li] * 1e-3) / 1e12, 1),
            "gemm_frac": round(ops[li] / (t_gemm[li] * 1e-3) / 1e12 / PEAK_FP8_TFLOPS, 4),
            "quantize_us": round(t_quant[li] * 1e3, 2),
            "quantize_us_median": round(m_quant[li] * 1e3, 2),
            "quantize_gbps": round(qbytes[li] / (t_quant[li] * 1e-3) / 1e9, 1),
            "copy_us": round(copies[li][0], 2),
            "copy_gbps": round(copies[li][1] / (copies[li][0] * 1e3), 1),
            "quantize_copy_frac": round(copies[li][0] / (m_quant[li] * 1e3)
                                        * qbytes[li] / copies[li][1], 4),
            "pack_us": round(t_pack[li] * 1e3, 2),
            "pack_gbps": round(pbytes[li] / (t_pack[li] * 1e-3) / 1e9, 1),
        })

    traffic = recorded_traffic(cfg.name, gs)

    # Sustained quantizer rate: the four layers' quantize launches back to back,
    # three rounds, under one event pair (per-launch events add a few
    # microseconds to each ~10 us launch).  The inputs and outputs cycled
    # through (~330 MB) exceed the 256 MB Infinity Cache, so the reads are cold.
    qrounds = 3
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(qrounds):
        for (x, w, b), (qa, pw, y) in zip(dev_in, outs):
            q.quantize_act(x, lzs_group=gs, out=qa)
    e1.record(stream)
    torch.cuda.synchronize()
    q_stream_gbps = qrounds * qbytes.sum() / (e0.elapsed_time(e1) * 1e-3) / 1e9

    cold = clocks = load_clocks = sweep = None
    if not args.no_ldm:
        cold = cold_layers(q, torch, np, cfg, dev_in, outs, workspaces, gs)
        sweep = gs_sweep(q, torch, np, cfg, dev_in, outs, workspaces)
        if not args.no_clocks:
            clocks = gpu_clocks()
            (x0, w0, b0), (qa0, pw0, y0) = dev_in[0], outs[0]
            load_clocks = clocks_under_load(
                torch, lambda: q.w4a4_linear(qa0, pw0, b0, layers[0].epilogue, out=y0,
                                             workspace=workspaces[0]),
                per_layer[0]["gemm_us"])

    ldm = None
    if not args.no_ldm:
        t_l = time.time()
        ldm = ldm_layers(q, W, torch, np, cfg, dev_in, gs)
        log(f"LDM-setting layers measured in {time.time() - t_l:.1f}s")

    asym = None
    if not args.no_ldm:
        t_a = time.time()
        asym = asym_layers(q, W, torch, np, cfg, dev_in, gs)
        log(f"asymmetric-mode layers measured in {time.time() - t_a:.1f}s")

    conv = None
    if not args.no_ldm:
        t_c = time.time()
        conv = conv_layers(q, W, torch, np, gs)
        log(f"implicit-GEMM convolutions measured in {time.time() - t_c:.1f}s")

    others = {}
    if not args.no_ldm:
        t_o = time.time()
        for c in (1, 2):
            if c != args.config:
                others[f"config{c}"] = config_layers(q, W, torch, np, c, gs)
        log(f"configs 1 and 2 measured in {time.time() - t_o:.1f}s")

    attn = None
    if not args.no_attention:
        t_at = time.time()
        attn = attention_bench(q, torch, np)
        log(f"LZS attention measured in {time.time() - t_at:.1f}s")

    mlp = None
    if not args.no_batched_mlp:
        del outs, dev_in, workspaces
        torch.cuda.empty_cache()
        t_m = time.time()
        mlp = batched_mlp(q, W, torch, np, gs)
        log(f"batched MLP pipeline measured in {time.time() - t_m:.1f}s")

    # ---------------- CPU oracle on a bounded sample (rank 0, N = 1 only)
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        rows = args.cpu_rows
        t_c = time.perf_counter()
        sample_ops = 0.0
        t_q = 0.0
        q_bytes = 0.0
        for li, L in enumerate(layers):
            xb, wb, bb = host[li]
            wq, sw = oracle.quantize_weight(wb)
            t0 = time.perf_counter()
            a = oracle.quantize_act(xb[:rows], lzs_group=gs)
            t_q += time.perf_counter() - t0
            q_bytes += layer_bytes(L, gs)[0] * rows / L.M
            oracle.linear_f64(a, wq, sw, bb, epilogue=L.epilogue)
            sample_ops += 2.0 * rows * L.N * L.K
        t_c = time.perf_counter() - t_c
        cpu_model = None
        try:
            for line in open("/proc/cpuinfo"):
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
        except OSError:
            pass
        cpu = {"value": round(sample_ops / t_c / 1e12, 6), "unit": "TOPS",
               "cores": oracle.num_threads(), "kind": "oracle",
               "sample": (f"weight pack of all {len(layers)} layers + quantize and linear of the "
                          f"first {rows} of {layers[0].M} rows of every layer; "
                          f"{t_c:.1f}s of CPU time"),
               "quantize_gbps": round(q_bytes / t_q / 1e9, 3),
               "host": {"cpu_model": cpu_model, "nproc": os.cpu_count()}}
        log(f"cpu oracle sample: {t_c:.1f}s")

    result = {
        "metric": "W4A4 linear TOPS + quantize GB/s at FLUX-shaped layers (fraction of roofline)",
        "value": round(value, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle": {"steps": settle_steps, "seconds": SETTLE_S,
                   "why": "untimed steps after the warmup until SETTLE_S of load have run, so "
                          "the timed steps see the GPU's steady clock"},
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8_e4m3",
        "data": "synthetic",
        "config": {
            "workload": cfg.name,
            "layers": [f"{L.name} M={L.M} K={L.K} N={L.N}" for L in layers],
            "group_size": 64, "lzs_group": gs,
            "step": "pack_weight of the 4 layers, then quantize_act + w4a4_linear (workspace "
                    "entry point) per layer",
        },
        "roofline": {
            "bound": "mfma", "achieved": round(gemm_tflops, 1), "peak": PEAK_FP8_TFLOPS,
            "unit": "TFLOP/s", "frac": round(gemm_tflops / PEAK_FP8_TFLOPS, 4),
            "achieved_median": round(gemm_tflops_median, 1),
            "traffic": traffic,
            "algorithmic_bytes": round(float(gbytes.mean())),
            "per": f"GEMM launch, mean over the {len(layers)} layers",
        },
        "quantize_roofline": {
            "bound": "hbm", "achieved": round(quant_gbps, 1), "peak": PEAK_HBM_GBPS,
            "unit": "GB/s", "frac": round(quant_gbps / PEAK_HBM_GBPS, 4),
            "achieved_median": round(quant_gbps_median, 1),
            "copy_frac": round(sum(c[0] for c in copies) / (m_quant.sum() * 1e3)
                               * qbytes.sum() / sum(c[1] for c in copies), 4),
            "per": "launch inside the instrumented steps (HIP events around each launch); "
                   "copy_frac: median quantizer time against a device copy moving the same "
                   "bytes, timed in this run",
        },
        "quantize_sustained": {
            "bound": "hbm", "achieved": round(q_stream_gbps, 1), "peak": PEAK_HBM_GBPS,
            "unit": "GB/s", "frac": round(q_stream_gbps / PEAK_HBM_GBPS, 4),
            "per": f"the four layers' launches back to back, {qrounds} rounds, one event pair",
        },
        "pack_gbps": round(pack_gbps, 1),
        "per_layer": per_layer,
        **others,
        "batched_mlp": mlp,
        "ldm_static": ldm,
        "asymmetric": asym,
        "conv3x3": conv,
        "attention": attn,
        "cold_cache": cold,
        "lzs_group_sweep": sweep,
        "gpu_clocks": {"after_run": clocks, "during_gemm": load_clocks},
        "wall_s_timed": round(wall, 3),
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
