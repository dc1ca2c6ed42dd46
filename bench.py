"""Benchmark: autoregressive WaveNet generation on one MI355X.

A "step" is one wn_generate call over the whole workload (every stream, every
sample) from a reset state, with conditioning and uniforms already resident in
HBM.  Prints ONE JSON line on stdout:
  value      generated samples/s (all streams) over the timed steps
  roofline   the generation kernel's algorithmic FLOP rate (2 x multiply-adds
             per sample of the model) over its average launch duration, from HIP
             events on the stream the kernel runs on, against the chip's peak
  cpu_baseline  the CPU oracle timed on this host on a bounded sample
  batched    (default workload only) a few launches of each batched workload, timed after the
             headline's timed region, with their own roofline records
Default workload: l=20, r=64, s=256, B=1, T=16000 (1 s of 16 kHz audio), fp32.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAKS = {  # MI355X published dense peaks
    "f32_vector_tflops": 157.3,
    "f32_mfma_tflops": 157.3,
    "bf16_mfma_tflops": 2500.0,
    "hbm_gbs": 8000.0,
}
# LDS read bandwidth per CU: one conflict-free ds_read_b128 wave instruction (1 KB) per 4 clocks,
# measured on one MI355X (a read loop over all 256 CUs sustained 148 TB/s, 94 % of 256 B/clk at
# the 2.4 GHz peak engine clock).
LDS_BYTES_PER_CLK_PER_CU = 256
SHADER_CLOCK_GHZ = 2.4
RATE_HZ = 16000
PAPER_RATE_HZ = 16384
HI_RATE_HZ = 48000  # the paper's 48 kHz case: a 20 us per-sample budget (Section 5)


def macs_per_sample(L, r, s, a=256, last_res=False):
    """Multiply-adds one generated sample needs: per layer W_prev and W_cur (2r x r each), W_res
    (r x r, not for the last layer, whose x feeds nothing) and W_skip (s x r); head W_relu (a x s)
    and W_out (a x a)."""
    per_layer = 2 * (2 * r * r) + r * r + s * r
    return L * per_layer - (0 if last_res else r * r) + a * s + a * a


# Source files each kernel family is built from (the digest of a committed counter run must match).
KERNEL_SOURCES = {
    "multi_cu_chain": ["wn_chain.hip", "wn_msg.h", "wn_wave.h", "wn_internal.h"],
    "multi_cu_mfma": ["wn_mchain.hip", "wn_mfma.h", "wn_msg.h", "wn_wave.h", "wn_internal.h"],
    "mfma_group": ["wn_group.hip", "wn_mfma.h", "wn_wave.h", "wn_internal.h"],
    "stream_l2": ["wn_stream.hip", "wn_wave.h", "wn_internal.h"],
    "conditioning": ["wn_cond.hip", "wn_wave.h", "wn_internal.h"],
}


def kernel_source_digest(variant):
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1702_07825_amd", "csrc")
    for f in KERNEL_SOURCES[variant]:
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def traffic_from_profiles(workload, variant):
    """HBM bytes per launch from committed rocprofv3 counter runs, if taken on the current kernels."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        rec = json.load(open(path))[workload]
    except Exception:
        return None
    if rec.get("variant") != variant or rec.get("source_digest") != kernel_source_digest(variant):
        return None
    return rec.get("hbm_bytes_per_launch")


# The oracle computes in double precision (plain sequential C, gcc -O2) and takes each draw in fp32,
# the precision of the paper's inference kernels: as slow as or slower than an fp32 oracle would be.
ORACLE_PRECISION = "fp64 arithmetic, draws compared in fp32"


def host_cores():
    """CPUs this process may run on (the host's nproc) and the machine's total."""
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count()
    return {"nproc": avail, "machine": os.cpu_count()}


def cpu_baseline(wl, w, cond_dev, u_np, min_seconds):
    """The CPU oracle on whole streams of the workload (stream 0, 1, ...; stream 0 again when the
    workload has one), one thread, until at least `min_seconds` of oracle time have passed."""
    import oracle
    m = oracle.Model(w, wl.dilations, bf16_weights=(wl.weight_dtype == "bf16"),
                     int8_weights=(wl.weight_dtype == "i8"))
    steps, secs, runs = 0, 0.0, []
    while secs < min_seconds:
        b = len(runs) % wl.B
        cond = cond_dev[b].cpu().numpy()
        t0 = time.perf_counter()
        oracle.run(m, cond, u=u_np[b], want_logits=False)
        secs += time.perf_counter() - t0
        steps += wl.T
        runs.append(b)
    which = ("stream 0, %d runs" % len(runs)) if wl.B == 1 else \
            ("streams 0..%d" % (len(runs) - 1) if len(runs) <= wl.B else "streams 0..%d, %d runs" % (wl.B - 1, len(runs)))
    return {"value": steps / secs, "unit": "samples/s", "cores": 1, "kind": "oracle",
            "host_cores": host_cores(),
            "precision": ORACLE_PRECISION,
            "sample": "whole streams of %d steps (%s), generation, one thread, fp64 C oracle" % (wl.T, which),
            "seconds": round(secs, 2)}


def algorithmic_hbm_bytes_per_sample(wl):
    """HBM bytes one generated sample needs at least: its conditioning (l x 2r fp32), uniform and
    sample, and the history of every layer read and written once (2 x l x r x 4 B)."""
    return wl.n_layers * 2 * wl.r * 4 + 4 + 4 + 2 * wl.n_layers * wl.r * 4


def _timed_launches(net, cond, u, samples, ws, steps, warmup):
    """`warmup` untimed then `steps` timed wn_generate calls from a reset state; returns the wall
    time of the timed calls and the average launch duration from HIP events on the stream."""
    import torch
    for _ in range(warmup):
        net.generate(cond, u, samples=samples, workspace=ws, reset=True)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(stream)
        net.generate(cond, u, samples=samples, workspace=ws, reset=True)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    assert net.status(ws) == 0
    launch_ms = [a.elapsed_time(b) for a, b in ev]
    return elapsed, sum(launch_ms) / len(launch_ms) / 1e3


def _roofline(name, wl, variant, avg_launch_s, wgs, reps):
    """The dominant kernel's roofline record for one launch of the whole workload."""
    n = wl.B * wl.T
    flop_per_launch = 2.0 * macs_per_sample(wl.n_layers, wl.r, wl.s) * n
    # The MFMA kernels compute their products on bf16 MFMA; the others on the fp32 vector ALUs.
    mfma = variant in ("mfma_group", "multi_cu_mfma")
    bound, peak = ("mfma", PEAKS["bf16_mfma_tflops"]) if mfma else ("alu", PEAKS["f32_vector_tflops"])
    achieved = flop_per_launch / avg_launch_s / 1e12
    hbm_alg = algorithmic_hbm_bytes_per_sample(wl) * n
    onchip = None
    if variant == "multi_cu_chain":
        # Every weight of a replica is read once per step from the LDS/VGPRs of the CUs holding it;
        # the floor is those bytes at the measured LDS rate of the CUs the launch occupies.
        wbytes = 4.0 * macs_per_sample(wl.n_layers, wl.r, wl.s) * reps * wl.T
        lds_gbs = wgs * LDS_BYTES_PER_CLK_PER_CU * SHADER_CLOCK_GHZ
        onchip = {"bound": "lds", "weight_bytes_per_launch": wbytes, "workgroups": wgs, "replicas": reps,
                  "achieved_gbs": round(wbytes / avg_launch_s / 1e9, 2), "peak_gbs": round(lds_gbs, 1),
                  "peak_basis": "%d B/clk/CU x %.1f GHz x workgroups" % (LDS_BYTES_PER_CLK_PER_CU, SHADER_CLOCK_GHZ),
                  "frac": round(wbytes / avg_launch_s / 1e9 / lds_gbs, 6)}
    return {
        "bound": bound,
        "achieved": round(achieved, 4),
        "peak": peak,
        "unit": "TFLOP/s",
        "frac": round(achieved / peak, 6),
        "traffic": traffic_from_profiles(name, variant),
        "algorithmic_flop_per_launch": flop_per_launch,
        "hbm": {"algorithmic_bytes_per_launch": hbm_alg,
                "achieved_gbs": round(hbm_alg / avg_launch_s / 1e9, 2),
                "peak_gbs": PEAKS["hbm_gbs"],
                "frac": round(hbm_alg / avg_launch_s / 1e9 / PEAKS["hbm_gbs"], 6)},
        "onchip": onchip,
        "avg_launch_ms": round(avg_launch_s * 1e3, 4),
    }


def _setup_workload(name, seed):
    import torch
    import synth
    import paper_1702_07825_amd as wn
    wl = synth.WORKLOADS[name]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.make_weights(wl.n_layers, wl.r, wl.s, seed=seed, embed_taps=wl.embed_taps)
    net = wn.WaveNet(w, wl.dilations, weight_dtype=wl.weight_dtype)
    cond = synth.make_cond(wl.n_layers, wl.r, wl.B, wl.T, seed=seed, device="cuda:0")
    u_np = synth.make_uniforms(wl.B, wl.T, seed=seed)
    u = torch.tensor(u_np, device=dev)
    samples = torch.empty((wl.B, wl.T), dtype=torch.int32, device=dev)
    ws = net.new_workspace(wl.B, dev)
    return wl, w, net, cond, u_np, u, samples, ws


# Batched workloads timed beside the headline (outside its timed region), so that their roofline
# fractions appear in the benchmark's own record.
BATCHED = ["l20_r128_b32", "l20_r64_b256_bf16", "l20_r64_b256_i8"]


def batched_record(args):
    """A few launches of each batched workload: per-step time, throughput and roofline fractions."""
    import torch
    rec = {}
    for name in BATCHED:
        wl, w, net, cond, u_np, u, samples, ws = _setup_workload(name, args.seed)
        variant = net.kernel_variant(wl.B)
        wgs, reps = net.launch_info(wl.B)
        print("bench: batched record %s, kernel %s, 1 warmup + %d timed steps" % (wl.description, variant,
              args.batched_steps), file=sys.stderr, flush=True)
        _, avg_s = _timed_launches(net, cond, u, samples, ws, args.batched_steps, 1)
        rf = _roofline(name, wl, variant, avg_s, wgs, reps)
        rec[name] = {"workload": wl.description, "kernel": variant, "workgroups": wgs, "replicas": reps,
                     "source_digest": kernel_source_digest(variant), "launches": args.batched_steps,
                     "samples_per_s": round(wl.B * wl.T / avg_s, 1),
                     "us_per_sample_step": round(avg_s / wl.T * 1e6, 3),
                     "real_time_factor_16khz": round(wl.T / avg_s / RATE_HZ, 3),
                     "roofline": rf}
        net.close()
        del cond, u, samples, ws
        torch.cuda.empty_cache()
    return rec


def run_workload(name, args, batched=False):
    import numpy as np
    import torch

    wl, w, net, cond, u_np, u, samples, ws = _setup_workload(name, args.seed)
    variant = net.kernel_variant(wl.B)
    wgs, reps = net.launch_info(wl.B)
    print("bench: %s, kernel %s, %d warmup + %d timed steps" % (wl.description, variant, args.warmup, args.steps),
          file=sys.stderr, flush=True)
    elapsed, avg_launch_s = _timed_launches(net, cond, u, samples, ws, args.steps, args.warmup)

    n = wl.B * wl.T
    value = n * args.steps / elapsed
    per_stream_rate = wl.T / avg_launch_s
    y = samples.cpu().numpy()
    out = {
        "metric": "generated samples/s (16 kHz mu-law audio, all streams)",
        "value": round(value, 1),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"f32": "f32", "bf16": "bf16-weights/f32", "i8": "i8-weights/f32"}[wl.weight_dtype],
        "data": "synthetic (seeded N(0,1/fan_in) weights, N(0,1) conditioning, U[0,1) uniforms)",
        "config": {"workload": wl.description, "B": wl.B, "T": wl.T, "n_layers": wl.n_layers, "r": wl.r,
                   "s": wl.s, "a": wl.a, "kernel": variant, "workgroups": wgs,
                   "source_digest": kernel_source_digest(variant)},
        "real_time_factor_16khz": round(per_stream_rate / RATE_HZ, 3),
        "real_time_factor_16384hz": round(per_stream_rate / PAPER_RATE_HZ, 3),
        "real_time_factor_48khz": round(per_stream_rate / HI_RATE_HZ, 3),
        "real_time_factor_at_workload_rate": round(per_stream_rate / wl.sample_rate, 3),
        "us_per_sample_step": round(avg_launch_s / wl.T * 1e6, 3),
        "roofline": _roofline(name, wl, variant, avg_launch_s, wgs, reps),
        "sample_histogram_entropy_bits": round(float(-(lambda p: (p[p > 0] * np.log2(p[p > 0])).sum())(
            np.bincount(y.ravel(), minlength=256) / y.size)), 3),
    }
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(wl, w, cond, u_np, args.cpu_seconds)
    else:
        out["cpu_baseline"] = None
    net.close()
    del cond, u, samples, ws
    torch.cuda.empty_cache()
    if batched and args.batched_steps > 0:
        out["batched"] = batched_record(args)
    print(json.dumps(out), flush=True)


def cond_flops(wl):
    """Multiply-adds x 2 of the two layers' gate contractions (both directions): per frame
    2 directions x 3h x 2 inputs-per-tap x cin for each layer."""
    h2 = wl.n_layers * wl.r
    per_frame = 2 * 3 * wl.h1 * 2 * wl.n_features + 2 * 3 * h2 * 2 * (2 * wl.h1)
    return 2.0 * per_frame * wl.B * wl.n_frames


def cond_cpu_baseline(wl, w, x_dev, min_seconds):
    """The CPU oracle's conditioning network on whole utterances of the workload (stream 0, 1, ...),
    one thread, until at least `min_seconds` of oracle time have passed."""
    import oracle
    steps, secs, runs = 0, 0.0, 0
    while secs < min_seconds:
        xb = x_dev[runs % wl.B].cpu().numpy()
        t0 = time.perf_counter()
        oracle.condition(w, xb, wl.T, wl.frame_rate, wl.audio_rate)
        secs += time.perf_counter() - t0
        steps += wl.T
        runs += 1
    return {"value": steps / secs, "unit": "samples/s", "cores": 1, "kind": "oracle",
            "host_cores": host_cores(), "precision": ORACLE_PRECISION,
            "sample": "%d whole utterance(s) of %d frames -> %d audio steps, one thread, fp64 C oracle" %
                      (runs, wl.n_frames, wl.T), "seconds": round(secs, 2)}


def run_cond_workload(name, args):
    """The conditioning network (Appendix A.2) over a batch of utterances: one wn_condition call
    per step, features already in HBM; value = audio steps of conditioning produced per second."""
    import torch
    import synth
    import paper_1702_07825_amd as wn

    wl = synth.COND_WORKLOADS[name]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.make_cond_weights(wl.n_features, wl.h1, wl.n_layers * wl.r, seed=args.seed)
    net = wn.Conditioner(w, wl.n_layers, wl.r, wl.frame_rate, wl.audio_rate)
    x = torch.tensor(synth.make_features(wl.B, wl.n_frames, seed=args.seed), device=dev)
    cond = torch.empty((wl.B, wl.T, wl.n_layers, 2 * wl.r), dtype=torch.float32, device=dev)
    ws = torch.empty(net.workspace_bytes(wl.B, wl.n_frames), dtype=torch.uint8, device=dev)
    print("bench: %s, %d warmup + %d timed steps" % (wl.description, args.warmup, args.steps), file=sys.stderr,
          flush=True)
    for _ in range(args.warmup):
        net(x, wl.T, cond=cond, workspace=ws)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        net(x, wl.T, cond=cond, workspace=ws)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    avg_s = sum(a.elapsed_time(b) for a, b in ev) / args.steps / 1e3
    flop = cond_flops(wl)
    out_bytes = wl.B * wl.T * 2 * wl.n_layers * wl.r * 4
    out = {
        "metric": "conditioned audio steps/s (conditioning network, all streams)",
        "value": round(wl.B * wl.T * args.steps / elapsed, 1),
        "unit": "samples/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded 227-dim phoneme/stress/F0 features, N(0,1/fan_in) weights)",
        "config": {"workload": wl.description, "B": wl.B, "n_frames": wl.n_frames, "T": wl.T, "h1": wl.h1,
                   "h2": wl.n_layers * wl.r, "kernel": "conditioning",
                   "source_digest": kernel_source_digest("conditioning")},
        "real_time_factor_16khz": round(wl.T / avg_s / RATE_HZ, 1),
        "roofline": {
            "bound": "mfma",
            "achieved": round(flop / avg_s / 1e12, 4),
            "peak": PEAKS["f32_mfma_tflops"],
            "unit": "TFLOP/s",
            "frac": round(flop / avg_s / 1e12 / PEAKS["f32_mfma_tflops"], 6),
            "traffic": traffic_from_profiles(name, "conditioning"),
            "note": "whole wn_condition call (gate contractions, pools, upsampling) against the fp32 MFMA peak",
            "algorithmic_flop_per_launch": flop,
            "hbm": {"output_bytes_per_launch": out_bytes, "achieved_gbs": round(out_bytes / avg_s / 1e9, 2),
                    "peak_gbs": PEAKS["hbm_gbs"], "frac": round(out_bytes / avg_s / 1e9 / PEAKS["hbm_gbs"], 6)},
            "avg_launch_ms": round(avg_s * 1e3, 4),
        },
        "cpu_baseline": None,
    }
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cond_cpu_baseline(wl, w, x, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    net.close()
    del x, cond, ws
    torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="l20_r64_b1",
                    help="a generation or conditioning-network workload name, or 'all' (one JSON line each)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="least oracle time for the CPU baseline, in whole streams (0 = skip)")
    ap.add_argument("--cpu-steps", type=int, default=None, choices=[0], help="0: skip the CPU baseline")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--batched-steps", type=int, default=2,
                    help="timed launches of each batched workload recorded beside the default headline "
                         "(after its timed region; 0 = skip)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run one device-to-device copy of BYTES (calibrates HBM byte counters) and exit")
    args = ap.parse_args()
    if args.cpu_steps == 0:
        args.cpu_seconds = 0.0
    if args.copy_probe:
        import torch
        src = torch.ones(args.copy_probe // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": args.copy_probe}))
        return
    if args.gpus != 1:
        print("bench.py: runs on one GPU only; --gpus %d is not supported (streams are independent, so a "
              "batch would shard by stream, each GPU holding a weight replica)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import synth
    names = list(synth.WORKLOADS) + list(synth.COND_WORKLOADS) if args.workload == "all" else [args.workload]
    for name in names:
        if name in synth.COND_WORKLOADS:
            run_cond_workload(name, args)
        else:
            run_workload(name, args, batched=(args.workload == "l20_r64_b1"))


if __name__ == "__main__":
    main()
