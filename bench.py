"""Benchmark of the NVFP4 W4A4 linear layer on one MI355X.

Workload (the M = 8192 configuration the headline metric is quoted on): the
fused MLP gate/up projection, X 8192 x 5120 bf16 with residual-stream
statistics (seeded synthetic data), W = two separately calibrated segments of
17408 x 5120 (std 0.015 and 0.0195), Y 8192 x 34816 bf16.

A step is one pass of the hot path: dynamic activation quantization of X
(amax pass + quantize pass) followed by the NVFP4 GEMM with the per-segment
scaled epilogue.  The weight prepack is offline and runs once before timing
(its time is reported separately).  Inputs are resident in HBM before the
timed region; the 570 MB output written by every step evicts the 256 MB
MALL, so each step reads X and W from HBM.

value = 2 M N K / (time per step), in TFLOPS.  roofline: the GEMM kernel's
algorithmic FLOPs per launch over its average launch time measured with HIP
events on the launch stream, against the FP16 dense MFMA peak (the GEMM
decodes NVFP4 exactly into FP16 MFMA operands).  cpu_baseline: the CPU oracle
timed on a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--no-cpu-baseline]
"""

import argparse
import dataclasses
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_F16_PEAK_TFLOPS = 2500.0      # MI355X dense FP16/BF16 MFMA
MXFP4_PEAK_TFLOPS = 10100.0        # MI355X dense FP4 MFMA (reported for context)
HBM_PEAK_GBS = 8000.0              # MI355X HBM3E
WORKLOAD = "mlp_gate_up"
# Sources of the headline GEMM kernel (gemm_lds_kernel<LdsSquareSuper>); the
# committed HBM byte counters are used only while their hash matches.
GEMM_SOURCES = ["paper_2609_04098_amd/csrc/gemm.hip", "paper_2609_04098_amd/csrc/gemm_common.h",
                "paper_2609_04098_amd/csrc/gemm_lds.h", "paper_2609_04098_amd/csrc/gemm_lds_super.hip",
                "paper_2609_04098_amd/csrc/packed_layout.h", "paper_2609_04098_amd/csrc/launch.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_mlp_gate_up_traffic.md")
# After host-side set-up the GPU's clock ramps back up over roughly 25 ms of
# back-to-back work (the GEMM's first launches after idle take 2.6-2.8 ms,
# then 2.3, 2.2 and 2.17 ms from about the tenth launch on), so every warmup
# continues past its W calls until this much GPU time has run.
SETTLE_MS = 60.0


def log(msg):
    sys.stderr.write("[bench %s] %s\n" % (time.strftime("%H:%M:%S"), msg))
    sys.stderr.flush()


def gemm_source_hash():
    h = hashlib.sha256()
    for p in GEMM_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def committed_traffic():
    """HBM bytes per GEMM launch from the committed rocprofv3 counter summary,
    if it was taken on the current GEMM source; else None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    text = open(TRAFFIC_FILE).read()
    m_hash = re.search(r"gemm_source_sha256_16:\s*([0-9a-f]+)", text)
    m_bytes = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != gemm_source_hash():
        return None
    return float(m_bytes.group(1))


def cpu_baseline(cfg, x_bits, w_bits, rows=8192, cols_per_seg=17408):
    """The CPU oracle (FP64 numpy, untuned) on a bounded sample of the same
    workload: quantize `rows` rows of X, then the dequantized GEMM of those
    rows against `cols_per_seg` rows of each weight segment (quantized
    beforehand, untimed, like the GPU prepack); timed over two passes (about
    10 s on a 16-thread host), reported per pass."""
    import numpy as np
    from oracle import gemm as OG
    from oracle import quant as OQ
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = os.cpu_count()
    offs = cfg.seg_offsets
    take = [min(cols_per_seg, offs[s + 1] - offs[s]) for s in range(len(offs) - 1)]
    w_rows = np.concatenate([np.arange(offs[s], offs[s] + take[s]) for s in range(len(take))])
    sub_offs = [0] + list(np.cumsum(take))
    rows = min(rows, cfg.m)
    wp, ws, gw = OQ.quantize_segments(w_bits[w_rows], sub_offs)
    passes = 2
    t0 = time.perf_counter()
    for _ in range(passes):
        xp, xs, gx = OQ.quantize_tensor(x_bits[:rows])
        y = OG.gemm_f64(xp, xs, gx, wp, ws, gw, sub_offs)
    dt = (time.perf_counter() - t0) / passes
    flops = 2.0 * rows * len(w_rows) * cfg.k
    assert y.shape == (rows, len(w_rows))
    return {
        "value": round(flops / dt / 1e12, 6), "unit": "TFLOPS", "cores": int(threads), "kind": "oracle",
        "sample": "act-quant of %d x %d rows of X + FP64 dequantized GEMM against %d of %d weight rows "
                  "(up to %d per segment), %d passes, %.1f s each" % (rows, cfg.k, len(w_rows), cfg.n, cols_per_seg,
                                                                       passes, dt),
    }


def warm(fn, warmup, stream, min_ms=SETTLE_MS):
    """Runs fn untimed `warmup` times, then further until at least `min_ms`
    of GPU time has passed since the first call (clock settling); returns
    the number of calls made."""
    import torch
    first = torch.cuda.Event(enable_timing=True)
    last = torch.cuda.Event(enable_timing=True)
    first.record(stream)
    n = 0
    batch = max(1, warmup)
    while True:
        for _ in range(batch):
            fn()
        n += batch
        last.record(stream)
        last.synchronize()
        if first.elapsed_time(last) >= min_ms or n >= 5000:
            return n
        batch = max(1, n)


def measure_workload(name, steps, warmup, dev, log_fn):
    """GEMM and dynamic act-quant of one more workload, timed like the
    headline step (HIP events on the launch stream around each launch);
    not part of `value`."""
    import numpy as np
    import torch
    from paper_2609_04098_amd import linear as L
    from paper_2609_04098_amd import nvfp4 as C
    from paper_2609_04098_amd import synth

    cfg = synth.CONFIGS[name]
    log_fn("drawing inputs for %s" % cfg.description)
    to_dev = lambda b: torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to(dev)
    x = to_dev(synth.make_x(cfg))
    pw = L.pack_weight(to_dev(synth.make_w(cfg)), cfg.seg_offsets)
    aq = L.alloc_act(cfg.m, cfg.k, dev)
    ws = L.act_workspace(cfg.m, cfg.k, dev)
    gws = L.gemm_workspace(cfg.m, cfg.n, cfg.k, dev)
    y = torch.empty((cfg.m, cfg.n), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()
    def step():
        L.quantize_act(x, out=aq, workspace=ws)
        L.gemm(aq, pw, out=y, workspace=gws)

    warm(step, warmup, stream)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for i in range(steps):
        ev[i][0].record(stream)
        L.quantize_act(x, out=aq, workspace=ws)
        ev[i][1].record(stream)
        L.gemm(aq, pw, out=y, workspace=gws)
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    aq_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    gemm_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    aq_bytes = cfg.m * cfg.k * (2 + 0.5 + 1.0 / 16)
    gemm_bytes = (cfg.m + cfg.n) * cfg.k * (0.5 + 1.0 / 16) + 2.0 * cfg.m * cfg.n
    out = {
        "M": cfg.m, "N": cfg.n, "K": cfg.k, "segments": list(cfg.segments),
        "gemm_kernels": L.gemm_kernels(cfg.m, cfg.n, cfg.k),
        "gemm_avg_ms": round(gemm_ms, 4),
        "gemm_tflops": round(cfg.flops / (gemm_ms * 1e-3) / 1e12, 2),
        "gemm_frac_mfma_f16": round(cfg.flops / (gemm_ms * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS, 4),
        "gemm_frac_hbm": round(gemm_bytes / (gemm_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "act_quant_avg_ms": round(aq_ms, 4),
        "act_quant_gbs": round(aq_bytes / (aq_ms * 1e-3) / 1e9, 1),
        "act_quant_frac_hbm": round(aq_bytes / (aq_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "tflops_incl_act_quant": round(cfg.flops / ((aq_ms + gemm_ms) * 1e-3) / 1e12, 2),
    }
    if cfg.n <= 96 and cfg.n % 2 == 0 and cfg.k % 64 == 0 and len(cfg.segments) == 2:
        # The b|a gate projection with the GDN gate transform (Eq. 1) in the
        # GEMM's epilogue, timed like the plain GEMM.
        h = cfg.n // 2
        rng = np.random.default_rng(99)
        a_log = torch.from_numpy(np.log(rng.uniform(1.0, 16.0, h)).astype(np.float32)).to(dev)
        dt_bias = torch.from_numpy(rng.uniform(-4.0, 2.0, h).astype(np.float32)).to(dev)
        warm(lambda: L.gemm_gdn_gates(aq, pw, a_log, dt_bias, out=y), warmup, stream)
        gev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
        for i in range(steps):
            gev[i][0].record(stream)
            L.gemm_gdn_gates(aq, pw, a_log, dt_bias, out=y)
            gev[i][1].record(stream)
        torch.cuda.synchronize()
        out["gemm_gdn_gates_avg_ms"] = round(float(np.mean([a.elapsed_time(b) for a, b in gev])), 4)
    if cfg.n <= 128 and cfg.k % 64 == 0:
        # Narrow output: act-quant fused into the GEMM, calibrated G (one pass
        # over X) and dynamic G (amax pass + one fused launch).
        g_static = aq.g.clone()
        gf = torch.empty(1, dtype=torch.float32, device=dev)
        for mode_name, mode in (("dynamic", C.NVFP4_DYNAMIC), ("static", C.NVFP4_STATIC)):
            gb = gf if mode == C.NVFP4_DYNAMIC else g_static
            wsp = ws if mode == C.NVFP4_DYNAMIC else None
            call = lambda: C.nvfp4_quantize_gemm(x, gb, pw.packed, pw.n, pw.seg_offsets, pw.g_seg, y, mode, wsp,
                                                 stream=stream)
            warm(call, warmup, stream)
            fev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
            for i in range(steps):
                fev[i][0].record(stream)
                call()
                fev[i][1].record(stream)
            torch.cuda.synchronize()
            f_ms = float(np.mean([a.elapsed_time(b) for a, b in fev]))
            out["fused_quantize_gemm_%s_ms" % mode_name] = round(f_ms, 4)
            out["fused_quantize_gemm_%s_tflops" % mode_name] = round(cfg.flops / (f_ms * 1e-3) / 1e12, 2)
    del x, pw, aq, ws, y
    torch.cuda.empty_cache()
    return out


def measure_decode(pws, m, steps, warmup, dev):
    """Decode-shaped calls against the headline's gate/up weight (34816 x
    5120, two segments): m rows of residual-stream X (the 32-token decode
    workload's first rows), dynamic G.  Unfused (quantizer + GEMM, two or
    three launches) and fused (nvfp4_quantize_gemm, one launch).  Before
    every timed call a 640 MB read evicts the weight from the 256 MB MALL;
    HIP events, median.  Sustained: back-to-back calls on 8 copies of the
    packed weight in turn (800 MB, as successive layers of a model would
    read their own weights from HBM), time per call."""
    pw = pws[0]
    import numpy as np
    import torch
    from paper_2609_04098_amd import linear as L
    from paper_2609_04098_amd import synth

    cfg = synth.CONFIGS["decode_m32"]
    xb = synth.make_x(cfg)[:m]
    x = torch.from_numpy(xb.view(np.int16)).view(torch.bfloat16).to(dev)
    stream = torch.cuda.current_stream()
    aq = L.alloc_act(m, cfg.k, dev)
    ws = L.act_workspace(m, cfg.k, dev)
    wsq = L.quantize_gemm_workspace(m, pw.n, cfg.k, dev)
    y = torch.empty((m, pw.n), dtype=torch.bfloat16, device=dev)
    flush = torch.ones(160 << 20, dtype=torch.float32, device=dev)

    def unfused(w=pw):
        L.quantize_act(x, out=aq, workspace=ws)
        L.gemm(aq, w, out=y)

    def fused(w=pw):
        L.quantize_gemm(x, w, out=y, workspace=wsq)

    res = {"M": m, "N": pw.n, "K": cfg.k, "w_bytes": int(pw.packed.numel())}
    for name, fn in (("unfused", unfused), ("fused", fused)):
        warm(fn, warmup, stream)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
        for i in range(steps):
            flush.sum()
            evs[i][0].record(stream)
            fn()
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        ms = float(np.median([a.elapsed_time(b) for a, b in evs]))
        res[name + "_median_ms"] = round(ms, 4)
        res[name + "_w_gbs"] = round(pw.packed.numel() / (ms * 1e-3) / 1e9, 1)
        res[name + "_frac_hbm"] = round(pw.packed.numel() / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        calls = 8 * max(2, steps // 4)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(calls):
            fn(pws[i % len(pws)])
        b.record(stream)
        torch.cuda.synchronize()
        sus = a.elapsed_time(b) / calls
        res[name + "_sustained_ms"] = round(sus, 4)
        res[name + "_sustained_frac_hbm"] = round(pw.packed.numel() / (sus * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
    del flush
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip the secondary per-workload figures (gdn_qkv, mlp_down, ab_gates)")
    ap.add_argument("--workload", default=WORKLOAD, help=argparse.SUPPRESS)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="copy a 1 GiB buffer 3 times with a plain device copy (for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library runs the NVFP4 linear layer on a single "
              "MI355X (no multi-GPU path); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": 1 << 30, "copy_calibration_bytes_written": 1 << 30}))
        return
    from paper_2609_04098_amd import linear as L
    from paper_2609_04098_amd import nvfp4 as C
    from paper_2609_04098_amd import synth

    C.lib()                                      # fail loudly if not built
    cfg = synth.CONFIGS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log("drawing inputs for %s" % cfg.description)
    x_bits = synth.make_x(cfg)
    w_bits = synth.make_w(cfg)
    to_dev = lambda b: torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to(dev)
    x = to_dev(x_bits)
    w = to_dev(w_bits)
    stream = torch.cuda.current_stream()

    # Offline weight prepack (timed separately, not part of a step).
    t_pack0, t_pack1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_pack0.record(stream)
    pw = L.pack_weight(w, cfg.seg_offsets)
    t_pack1.record(stream)
    torch.cuda.synchronize()
    prepack_ms = t_pack0.elapsed_time(t_pack1)
    del w

    aq = L.alloc_act(cfg.m, cfg.k, dev)
    ws = L.act_workspace(cfg.m, cfg.k, dev)
    y = torch.empty((cfg.m, cfg.n), dtype=torch.bfloat16, device=dev)
    gws = L.gemm_workspace(cfg.m, cfg.n, cfg.k, dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        L.quantize_act(x, out=aq, workspace=ws)
        if ev is not None:
            ev[1].record(stream)
        L.gemm(aq, pw, out=y, workspace=gws)
        if ev is not None:
            ev[2].record(stream)

    log("warmup %d steps (continued until %.0f ms of GPU time)" % (args.warmup, SETTLE_MS))
    warmup_run = warm(step, args.warmup, stream)
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    log("timing %d steps" % args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    aq_ms = [e[0].elapsed_time(e[1]) for e in events]
    gemm_ms = [e[1].elapsed_time(e[2]) for e in events]
    step_ms = [e[0].elapsed_time(e[2]) for e in events]
    ms_per_step = wall * 1e3 / args.steps
    flops = cfg.flops
    value = flops / (ms_per_step * 1e-3) / 1e12
    gemm_avg = float(np.mean(gemm_ms))
    aq_avg = float(np.mean(aq_ms))
    gemm_tflops = flops / (gemm_avg * 1e-3) / 1e12
    aq_bytes = cfg.m * cfg.k * (2 + 0.5 + 1.0 / 16)
    aq_gbs = aq_bytes / (aq_avg * 1e-3) / 1e9
    traffic = committed_traffic() if cfg.name == WORKLOAD else None
    gemm_bytes = (cfg.m + cfg.n) * cfg.k * (0.5 + 1.0 / 16) + 2.0 * cfg.m * cfg.n
    gemm_gbs = gemm_bytes / (gemm_avg * 1e-3) / 1e9

    # One-pass quantizers with a given (calibrated) global scale, here the
    # dynamic G just computed: the stand-alone static quantizer and RMSNorm
    # fused with it (gamma ~ U(0.5, 1.5)).  Each launch follows a 640 MB read
    # of another buffer, so X comes from HBM and the MALL holds no dirty lines;
    # HIP events on the launch stream, median over the steps.
    flush = torch.ones(160 << 20, dtype=torch.float32, device=dev)
    gamma = to_dev(synth.f64_to_bf16_bits(np.random.default_rng(77).uniform(0.5, 1.5, cfg.k)))

    def time_one_pass(fn):
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        for i in range(args.steps):
            flush.sum()
            evs[i][0].record(stream)
            fn()
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in evs]))

    aq_static_avg = time_one_pass(
        lambda: C.nvfp4_quantize_act(x, aq.codes, aq.scales, aq.g, C.NVFP4_STATIC, None, stream))
    norm_avg = time_one_pass(
        lambda: C.nvfp4_rmsnorm_quantize_act(x, gamma, 1e-6, aq.codes, aq.scales, aq.g, None, stream))
    del flush

    # The same quantizers called back to back (as the layers of a prefill
    # would) on 8 distinct activations of X's shape (672 MB, more than twice
    # the MALL, visited in turn so that each is read from HBM): HIP events
    # around all the calls, time per call.
    xr = [x] + [torch.roll(x, shifts=17 * i, dims=1) for i in range(1, 8)]

    def time_sustained(fn, calls=32):
        for i in range(8):
            fn(xr[i])
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(calls):
            fn(xr[i % 8])
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / calls

    aq_static_sus = time_sustained(
        lambda xi: C.nvfp4_quantize_act(xi, aq.codes, aq.scales, aq.g, C.NVFP4_STATIC, None, stream))
    norm_sus = time_sustained(
        lambda xi: C.nvfp4_rmsnorm_quantize_act(xi, gamma, 1e-6, aq.codes, aq.scales, aq.g, None, stream))
    del xr

    gates = None
    if cfg.n <= 96 and cfg.n % 2 == 0 and cfg.k % 64 == 0 and len(cfg.segments) == 2:
        # The tall-skinny b|a gate projection with the GDN gate transform
        # (Eq. 1) in its epilogue, timed like the plain GEMM.
        h = cfg.n // 2
        rng = np.random.default_rng(99)
        a_log = torch.from_numpy(np.log(rng.uniform(1.0, 16.0, h)).astype(np.float32)).to(dev)
        dt_bias = torch.from_numpy(rng.uniform(-4.0, 2.0, h).astype(np.float32)).to(dev)
        gev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        for i in range(args.steps):
            L.quantize_act(x, out=aq, workspace=ws)
            gev[i][0].record(stream)
            L.gemm_gdn_gates(aq, pw, a_log, dt_bias, out=y)
            gev[i][1].record(stream)
        torch.cuda.synchronize()
        gates_avg = float(np.mean([a.elapsed_time(b) for a, b in gev]))
        gates = {"avg_ms": round(gates_avg, 4), "plain_gemm_avg_ms": round(gemm_avg, 4),
                 "note": "GEMM with the GDN gate transform (beta | alpha) in the epilogue"}
    fused = None
    if cfg.n <= 128 and cfg.k % 64 == 0:
        # Narrow outputs: act-quant fused into the GEMM (one launch after the
        # amax pass; X read once with a calibrated scale), timed like the step.
        g_static = aq.g.clone()
        gf = torch.empty(1, dtype=torch.float32, device=dev)
        res = {}
        for name, mode in (("dynamic", C.NVFP4_DYNAMIC), ("static", C.NVFP4_STATIC)):
            gb = gf if mode == C.NVFP4_DYNAMIC else g_static
            wsp = ws if mode == C.NVFP4_DYNAMIC else None
            call = lambda: C.nvfp4_quantize_gemm(x, gb, pw.packed, pw.n, pw.seg_offsets, pw.g_seg, y, mode, wsp,
                                                 stream=stream)
            warm(call, args.warmup, stream)
            fev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
            for i in range(args.steps):
                fev[i][0].record(stream)
                call()
                fev[i][1].record(stream)
            torch.cuda.synchronize()
            f_ms = float(np.mean([a.elapsed_time(b) for a, b in fev]))
            res[name] = {"avg_ms": round(f_ms, 4), "tflops_incl_act_quant": round(flops / (f_ms * 1e-3) / 1e12, 2)}
        fused = dict(res, note="nvfp4_quantize_gemm: act-quant fused into the narrow GEMM (dynamic: amax pass + "
                               "one fused launch; static: one launch with the calibrated G); not part of value")
    aq_static_gbs = aq_bytes / (aq_static_avg * 1e-3) / 1e9
    norm_gbs = aq_bytes / (norm_avg * 1e-3) / 1e9
    log("step %.3f ms (events %.3f), act-quant %.3f ms, GEMM %.3f ms" % (
        ms_per_step, float(np.mean(step_ms)), aq_avg, gemm_avg))

    result = {
        "metric": "NVFP4 W4A4 GEMM TFLOPS incl. act-quant (M=8192) and % of MFMA peak",
        "value": round(value, 2),
        "unit": "TFLOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": warmup_run,
        "warmup_note": "untimed steps continue past W until %.0f ms of GPU time have run (clock settling "
                       "after host-side set-up)" % SETTLE_MS,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "nvfp4",
        "compute": "E2M1 x E4M3 decoded exactly to f16, v_mfma_f32_32x32x16_f16, f32 accumulate",
        "data": "synthetic",
        "config": {
            "workload": "%s: %s" % (cfg.name, cfg.description),
            "M": cfg.m, "N": cfg.n, "K": cfg.k, "segments": list(cfg.segments),
            "x": "bf16 N(0,1) with 0.5% channels x U(50,200)", "y": "bf16",
        },
        "pct_of_mfma_peak": round(100.0 * value / MFMA_F16_PEAK_TFLOPS, 2),
        "roofline": {
            "bound": "mfma",
            "kernel": " + ".join(L.gemm_kernels(cfg.m, cfg.n, cfg.k)) + ", bf16 out",
            "achieved": round(gemm_tflops, 2),
            "peak": MFMA_F16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(gemm_tflops / MFMA_F16_PEAK_TFLOPS, 4),
            "traffic": traffic,
            "algorithmic_flops_per_launch": flops,
            "avg_launch_ms": round(gemm_avg, 4),
            "hbm": {"algorithmic_bytes": gemm_bytes, "achieved": round(gemm_gbs, 1), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(gemm_gbs / HBM_PEAK_GBS, 4)},
        },
        "act_quant": {
            "bound": "hbm", "avg_ms": round(aq_avg, 4), "achieved": round(aq_gbs, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(aq_gbs / HBM_PEAK_GBS, 4),
            "algorithmic_bytes": aq_bytes,
        },
        "act_quant_static": {
            "bound": "hbm", "median_ms": round(aq_static_avg, 4), "achieved": round(aq_static_gbs, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(aq_static_gbs / HBM_PEAK_GBS, 4),
            "sustained_ms": round(aq_static_sus, 4),
            "sustained_frac": round(aq_bytes / (aq_static_sus * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "note": "one pass with a given (calibrated) global scale, X from HBM: one call after a 640 MB read "
                    "(median); sustained: back-to-back calls on 8 distinct activations (672 MB); not part of value",
        },
        "rmsnorm_act_quant_static": {
            "bound": "hbm", "median_ms": round(norm_avg, 4), "achieved": round(norm_gbs, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(norm_gbs / HBM_PEAK_GBS, 4),
            "sustained_ms": round(norm_sus, 4),
            "sustained_frac": round(aq_bytes / (norm_sus * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "note": "RMSNorm fused with the static-scale quantizer, one pass, X from HBM (as act_quant_static); "
                    "not part of value",
        },
        "gdn_gates": gates,
        "fused_quantize_gemm": fused,
        "frac_of_mxfp4_peak": round(value / MXFP4_PEAK_TFLOPS, 4),
        "prepack_ms": round(prepack_ms, 3),
        "gemm_source_sha256_16": gemm_source_hash(),
    }
    if not args.no_other_workloads and args.workload == WORKLOAD:
        log("decode shapes against the gate/up weight")
        pws = [pw] + [dataclasses.replace(pw, packed=pw.packed.clone()) for _ in range(7)]
        result["decode"] = {"m%d" % m: measure_decode(pws, m, args.steps, args.warmup, dev) for m in (1, 7, 32)}
        del pws
        result["other_workloads"] = {}
        for name in ("gdn_qkv", "mlp_down", "ab_gates"):
            result["other_workloads"][name] = measure_workload(name, max(5, args.steps // 2), max(2, args.warmup), dev,
                                                               log)
    if not args.no_cpu_baseline:
        log("CPU oracle baseline on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(cfg, x_bits, w_bits)
    print(json.dumps(result))


if __name__ == "__main__":
    main()
