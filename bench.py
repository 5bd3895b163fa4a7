#!/usr/bin/env python3
"""Steady-state forward throughput of libgm on one MI355X.

Headline workload: the large rotary decoder -- 32 layers, d_model 4096, 32
heads of 128, SwiGLU FFN 11008, pre-RMSNorm, rotary positions (base 1e4,
table built for 1024 positions and grown on the device to the 2048 the
forward needs), vocab 32000, untied head, bf16, one sequence of 2048 tokens,
synthetic weights N(0, 0.02) and uniform token ids.  It is the largest of the
five synthetic workloads and fits one GPU (13.5 GB of weights).  One step =
one gm_forward: a single hipGraphLaunch of the whole forward, every
data-dependent branch (guards, padding predicate, rotary regrow, effects)
resolved on the device.

Prints one JSON line: throughput, host syncs per forward (library counter),
a roofline entry for the dominant kernel (the MFMA GEMM, timed with HIP
events on its launch stream), the CPU oracle on a bounded sample, and under
``configs`` the same measurement for each of the five workloads (the
single-graph forward next to the graph-broken program the paper starts
from), plus a KV-cache decode and an encoder-decoder leg.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = "decoder_4096"
TABLE = ["tiny_decoder", "causal_lm_768", "encoder_1024", "encoder_clamp_1024", "decoder_4096"]
PEAK_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}   # MI355X dense MFMA / fp32 vector
PEAK_HBM_GBS = 8000.0
WEIGHT_SEED = 1234

DESCR = {
    "tiny_decoder": "1 layer, d_model 64, 2 heads, FFN 256 GELU, LayerNorm, vocab 512, fp32, "
                    "batch 1 x 16, 0..4 trailing pads",
    "causal_lm_768": "12-layer causal LM decoder, d_model 768, 12 heads, FFN 3072 GELU, pre-LN, "
                     "learned positions, vocab 50257, bf16, batch 8 x 512, 0..128 pads",
    "encoder_1024": "24-layer bidirectional encoder, d_model 1024, 16 heads, FFN 4096 GELU, "
                    "post-LN, vocab 30522, bf16, batch 16 x 512, 0..256 pads",
    "encoder_clamp_1024": "24-layer encoder stack with the fp16 overflow clamp, d_model 1024, "
                          "16 heads, GEGLU 2816, RMSNorm, fp16, batch 4 x 1024, weights "
                          "N(0,0.05) with 1% of matrix entries x200",
    "decoder_4096": "32-layer decoder, d_model 4096, 32 heads, SwiGLU FFN 11008, RMSNorm, "
                    "rotary base 1e4 (table 1024 -> regrown to 2048 on the device), vocab 32000, "
                    "untied head, bf16, batch 1 x 2048",
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def time_steps(m, ids_t, mask_t, out, steps, warmup):
    """Wall clock around `steps` forwards, synchronised at both ends (ms per
    forward)."""
    import torch
    for _ in range(warmup):
        m.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        m.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


def cold_call(m, ids_t, mask_t):
    """First forward on a new (batch, sequence, buffers) key: capture +
    instantiate + run of its graph(s)."""
    import torch
    out = m.new_logits(*ids_t.shape)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    m.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3, out


def timed_graph(m, ids_t, mask_t, out, steps, warmup):
    """The timed region: `steps` single-graph forwards between two HIP events
    on the launch stream, with the library's counters read around it."""
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        m.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    s0 = m.stats()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(steps):
        m.forward(ids_t, mask_t, out)
    ev1.record(stream)
    torch.cuda.synchronize()
    s1 = m.stats()
    return {"ms": ev0.elapsed_time(ev1) / steps,
            "syncs": (s1["host_syncs_in_forward"] - s0["host_syncs_in_forward"]) / steps,
            "launches": (s1["graph_launches"] - s0["graph_launches"]) / steps,
            "kernels": s1["kernels_per_forward"]}


def fragmented(m, ids_t, mask_t, steps, warmup):
    """The same forward as the unmended program (one graph per region between
    graph breaks; host sync + read-back + host branch at each break) next to
    the single-graph forward, both timed by wall clock around the loop."""
    cold_g, out = cold_call(m, ids_t, mask_t)
    ms_g = time_steps(m, ids_t, mask_t, out, steps, warmup)
    m.set_exec_mode("fragmented")
    s0 = m.stats()
    cold_f, out = cold_call(m, ids_t, mask_t)
    s1 = m.stats()
    ms_f = time_steps(m, ids_t, mask_t, out, steps, warmup)
    s2 = m.stats()
    m.set_exec_mode("graph")
    runs = steps + warmup
    return {"single_graph": {"ms_per_step": round(ms_g, 4), "cold_ms": round(cold_g, 2)},
            "fragmented": {"ms_per_step": round(ms_f, 4), "cold_ms": round(cold_f, 2),
                           "graphs_per_forward": (s2["graph_launches"] - s1["graph_launches"]) / runs,
                           "host_syncs_per_forward": (s2["host_syncs_in_forward"] - s1["host_syncs_in_forward"]) / runs,
                           "graphs_captured": s1["captures"] - s0["captures"]},
            "steady_speedup": round(ms_f / ms_g, 3), "cold_speedup": round(cold_f / cold_g, 3)}


def kernel_profile(m, ids_t, mask_t, out, reps=3):
    """Per-launch durations of an eager forward (HIP events recorded on the
    launch stream after every kernel), the last of `reps` runs."""
    prof = None
    for _ in range(reps):
        prof = m.profile(ids_t, mask_t, out)
    return prof


def gemm_roofline(prof, dtype, kernel_name):
    """Roofline entry of the GEMM kernel: algorithmic 2*M*N*K per launch over
    the launch durations, overall and per projection."""
    peak = PEAK_TFLOPS[dtype]
    gemm = [p for p in prof if p[0].startswith("gemm")]
    g_ms = sum(p[2] for p in gemm)
    g_flops = sum(p[3] for p in gemm)
    achieved = g_flops / (g_ms * 1e-3) / 1e12
    per = {}
    for kind, layer, kms, flops, nbytes in gemm:
        e = per.setdefault(kind, [0, 0.0, 0.0])
        e[0] += 1
        e[1] += kms
        e[2] += flops
    return {"kernel": kernel_name, "bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
            "unit": "TFLOP/s", "frac": round(achieved / peak, 4), "traffic": None,
            "launches_per_forward": len(gemm), "avg_launch_ms": round(g_ms / len(gemm), 5),
            "flops_per_launch_avg": g_flops / len(gemm),
            "per_projection": {k: {"launches": v[0], "avg_ms": round(v[1] / v[0], 5),
                                   "gflop_per_launch": round(v[2] / v[0] / 1e9, 2),
                                   "tflops": round(v[2] / (v[1] * 1e-3) / 1e12, 1),
                                   "frac": round(v[2] / (v[1] * 1e-3) / 1e12 / peak, 4)}
                               for k, v in per.items()}}


def breakdown(prof):
    by_kind = {}
    for kind, layer, kms, flops, nbytes in prof:
        t = by_kind.setdefault(kind, [0, 0.0, 0.0, 0.0])
        t[0] += 1
        t[1] += kms
        t[2] += flops
        t[3] += nbytes
    return {k: {"launches": v[0], "ms": round(v[1], 4),
                "tflops": round(v[2] / (v[1] * 1e-3) / 1e12, 2) if v[2] else None,
                "gbs": round(v[3] / (v[1] * 1e-3) / 1e9, 1) if v[3] and not v[2] else None}
            for k, v in by_kind.items()}


def measured_traffic(workload):
    """HBM bytes per GEMM launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE record of this workload, if it was taken on the GEMM source as
    it is now."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"gemm_traffic_{workload}.json")
    src = os.path.join(ROOT, "paper_2509_16248_amd", "csrc", "gm_gemm.hip")
    try:
        rec = json.load(open(path))
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    return rec["traffic_bytes_per_launch"] if rec.get("gm_gemm_hip_sha256") == sha else None


def load_model(name, seed=WEIGHT_SEED):
    import torch
    import synth
    from paper_2509_16248_amd.model import GmModel
    cfg = synth.preset(name)
    t0 = time.perf_counter()
    w = synth.make_weights(cfg, seed)
    log(f"[bench] {name}: weights generated in {time.perf_counter() - t0:.1f} s")
    ids, mask = synth.make_inputs(cfg, 0)
    m = GmModel(cfg, w.globals, w.layers, device="cuda:0")
    return cfg, w, m, ids, mask, torch.from_numpy(ids).cuda(), torch.from_numpy(mask).cuda()


def measure(name, args, loaded=None, steps=None, warmup=None, frag=True):
    """One workload: cold call, the timed single-graph region, the per-kernel
    profile and (frag) the graph-broken program on the same inputs."""
    import torch
    steps = steps or args.steps
    warmup = warmup if warmup is not None else args.warmup
    own = loaded is None
    cfg, w, m, ids, mask, ids_t, mask_t = loaded or load_model(name)
    cold_ms, out = cold_call(m, ids_t, mask_t)
    t = timed_graph(m, ids_t, mask_t, out, steps, warmup)
    prof = kernel_profile(m, ids_t, mask_t, out)
    flops = sum(p[3] for p in prof)
    peak = PEAK_TFLOPS[cfg.dtype]
    tokens = int(ids.size)
    r = {"workload": f"{name}: {DESCR[name]}", "dtype": cfg.dtype,
         "tokens_per_forward": tokens, "nonpad_tokens": int(mask.sum()),
         "ms_per_step": round(t["ms"], 4), "tokens_per_s": round(tokens / (t["ms"] * 1e-3), 1),
         "host_syncs_per_forward": t["syncs"], "graph_launches_per_forward": t["launches"],
         "kernels_per_forward": t["kernels"], "cold_ms": round(cold_ms, 2),
         "tflop_per_forward": round(flops / 1e12, 4),
         "forward_frac_of_peak": round(flops / (t["ms"] * 1e-3) / 1e12 / peak, 4)}
    if cfg.dtype != "f32":
        r["gemm"] = gemm_roofline(prof, cfg.dtype, "k_gemm_x")
    if frag:
        r["fragmented_baseline"] = fragmented(m, ids_t, mask_t, max(5, steps // 2), 2)
    log(f"[bench] {name}: {json.dumps({k: r[k] for k in ('ms_per_step', 'tokens_per_s', 'host_syncs_per_forward', 'forward_frac_of_peak')})}")
    if own:
        m.close()
    return r, prof, t, out


def cpu_baseline(cfg, w, ids, mask, depths):
    """The oracle (float64 NumPy) on a bounded sample of the headline
    workload: the whole 2048-position sequence through the embedding, the
    first few layers, the final norm and the head.  Two depths give the
    per-layer and the fixed cost; the full-depth time is the fixed cost plus
    n_layers times the per-layer cost."""
    from oracle import OracleModel
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    times = []
    for nl in depths:
        om = OracleModel(cfg.replace(n_layers=nl), w)
        t0 = time.perf_counter()
        om.forward(ids, mask)
        times.append(time.perf_counter() - t0)
    per_layer = max((times[1] - times[0]) / (depths[1] - depths[0]), 1e-9)
    fixed = max(times[0] - depths[0] * per_layer, 0.0)
    full = fixed + cfg.n_layers * per_layer
    tokens = int(ids.size)
    return {"value": round(tokens / full, 3), "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"all {ids.shape[0]} x {ids.shape[1]} positions through the embedding, the "
                      f"first {depths[0]} and the first {depths[1]} layers, final norm and head "
                      f"({times[0]:.2f} s, {times[1]:.2f} s); the {cfg.n_layers}-layer forward = "
                      f"fixed {fixed:.2f} s + {cfg.n_layers} x {per_layer:.2f} s per layer = "
                      f"{full:.1f} s for {tokens} tokens"}


def seq2seq_bench(args):
    """The encoder-decoder workload (6 + 6 layers, d 768, batch 8, source 512,
    target 128, ragged): single-graph forwards timed with events, then the
    graph-broken program on the same buffers.  Throughput counts source and
    target positions."""
    import torch
    import synth
    from paper_2509_16248_amd.model import GmModel
    cfg = synth.preset("seq2seq_768")
    w = synth.make_weights(cfg, WEIGHT_SEED)
    si, sm = synth.make_inputs(cfg, 0)
    ti, tm = synth.make_target_inputs(cfg, 0)
    m = GmModel(cfg, w.globals, w.layers, dec_layers=w.dec_layers, device="cuda:0")
    del w
    bufs = [torch.from_numpy(a).cuda() for a in (si, sm, ti, tm)]
    out = m.new_logits(cfg.batch, cfg.tgt_seq)
    stream = torch.cuda.current_stream()

    def loop(n):
        for _ in range(n):
            m.forward_seq2seq(*bufs, out)

    def timed(mode):
        m.set_exec_mode(mode)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        loop(1)
        torch.cuda.synchronize()
        cold = (time.perf_counter() - t0) * 1e3
        loop(args.warmup)
        torch.cuda.synchronize()
        s0 = m.stats()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        ev0.record(stream)
        loop(args.steps)
        ev1.record(stream)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3 / args.steps
        s1 = m.stats()
        return {"ms_per_step": round(ev0.elapsed_time(ev1) / args.steps, 4),
                "wall_ms_per_step": round(wall, 4), "cold_ms": round(cold, 2),
                "graph_launches_per_forward": (s1["graph_launches"] - s0["graph_launches"]) / args.steps,
                "host_syncs_per_forward": (s1["host_syncs_in_forward"] - s0["host_syncs_in_forward"]) / args.steps}

    g = timed("graph")
    f = None if args.no_fragmented else timed("fragmented")
    code = m.check_error()
    kernels = m.stats()["kernels_per_forward"]
    m.close()
    tokens = cfg.batch * (cfg.seq + cfg.tgt_seq)
    return {"workload": "seq2seq_768: 6 encoder + 6 decoder layers (cross-attention), d_model 768, "
                        "12 heads, FFN 3072 GELU, pre-LN, vocab 50265, bf16; batch 8, source 512 "
                        "(0..128 pads), target 128 (0..32 pads)",
            "tokens_per_forward": tokens, "kernels_per_forward": kernels,
            "tokens_per_s": round(tokens / (g["ms_per_step"] * 1e-3), 1),
            "single_graph": g, "fragmented": f,
            "steady_speedup": round(f["wall_ms_per_step"] / g["wall_ms_per_step"], 3) if f else None,
            "trap": list(code)}


def decode_bench(name="causal_lm_768", prompt=384, steps=120, warmup=8):
    """Greedy decoding with the KV cache: prefill B x `prompt` positions
    (ragged, 0..128 trailing pads), then `steps` decode steps in which each
    step's greedy tokens (device argmax) are the next step's input, one graph
    launch per step and no host read.  The step is HBM-bound: its algorithmic
    bytes are every weight read once plus the cached keys and values of
    every sequence up to its position."""
    import numpy as np
    import torch
    import synth
    from paper_2509_16248_amd.model import GmModel
    cfg = synth.preset(name)
    w = synth.make_weights(cfg, WEIGHT_SEED)
    B = cfg.batch
    m = GmModel(cfg, w.globals, w.layers, device="cuda:0", kv_cache=True)
    ids, mask = synth.make_inputs(cfg, 3, seq=prompt)
    ids_t = torch.from_numpy(ids).cuda()
    mask_t = torch.from_numpy(mask).cuda()
    out = m.new_logits(B, prompt)
    tok = torch.ones(B, dtype=torch.int32, device="cuda")
    logits = m.new_decode_logits(B)
    stream = torch.cuda.current_stream()
    for _ in range(2):                     # cold captures: prefill and step graphs
        m.forward(ids_t, mask_t, out)
        for _ in range(warmup):
            m.decode(tok, logits, tok)
    torch.cuda.synchronize()
    m.forward(ids_t, mask_t, out)
    tok.fill_(1)
    s0 = m.stats()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(steps):
        m.decode(tok, logits, tok)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    s1 = m.stats()
    code = m.check_error()
    m.close()
    L0 = mask.sum(1).astype(np.int64)            # lengths before the first step
    d, ff, V, nl = cfg.d_model, cfg.d_ff, cfg.vocab, cfg.n_layers
    up = 2 * ff if cfg.gated else ff
    weight_bytes = 2.0 * (nl * (3 * d * d + d * d + up * d + d * ff) + V * d)
    # keys and values read per step, averaged over the timed steps
    kv_bytes = 2.0 * 2 * nl * d * float(np.mean([(L0 + t + 1).sum() for t in range(steps)]))
    gbs = (weight_bytes + kv_bytes) / (ms * 1e-3) / 1e9
    return {"workload": f"{cfg.name}: batch {B}, prompts of {prompt} positions with 0..{cfg.max_pad} "
                        f"trailing pads, {steps} greedy steps (device argmax fed back)",
            "ms_per_step": round(ms, 4), "tokens_per_s": round(B / (ms * 1e-3), 1),
            "graph_launches_per_step": (s1["graph_launches"] - s0["graph_launches"]) / steps,
            "host_syncs_per_step": (s1["host_syncs_in_forward"] - s0["host_syncs_in_forward"]) / steps,
            "trap": list(code),
            "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                         "bytes_per_step": weight_bytes + kv_bytes}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-depths", default="2,6",
                    help="layer counts of the two oracle runs of the CPU sample")
    ap.add_argument("--no-fragmented", action="store_true",
                    help="skip the graph-broken baseline (same kernels, host sync per break)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other four workloads")
    ap.add_argument("--no-decode", action="store_true", help="skip the KV-cache decode measurement")
    ap.add_argument("--no-seq2seq", action="store_true",
                    help="skip the encoder-decoder measurement")
    ap.add_argument("--only", default=None,
                    help="measure one workload only (one JSON object, no headline)")
    ap.add_argument("--seq2seq-only", action="store_true",
                    help="only the encoder-decoder measurement (one JSON object)")
    ap.add_argument("--decode-only", action="store_true",
                    help="only the KV-cache decode measurement (one JSON object)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (got --gpus {args.gpus}); "
              "the multi-GPU layout is a design only, not built", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.seq2seq_only:
        print(json.dumps(seq2seq_bench(args)), flush=True)
        return
    if args.decode_only:
        print(json.dumps(decode_bench()), flush=True)
        return
    if args.only:
        r, _, _, _ = measure(args.only, args, frag=not args.no_fragmented)
        print(json.dumps(r), flush=True)
        return

    loaded = load_model(WORKLOAD)
    cfg, w, m, ids, mask, ids_t, mask_t = loaded
    head, prof, t, out = measure(WORKLOAD, args, loaded, frag=not args.no_fragmented)
    dec = m.decisions()
    m.close()
    del m, loaded, out
    torch.cuda.empty_cache()
    roof = head["gemm"]
    roof["kernel"] = ("k_gemm_big (128x384, 256x256 and 128x256 tiles): every projection GEMM "
                      "and the LM head of the forward")
    roof["traffic"] = measured_traffic(WORKLOAD)
    roof["timing"] = ("HIP events on the launch stream around each kernel of an eager forward "
                      "that runs the same launches as the graph (batch 1: one branch)")
    result = {
        "metric": "steady-state forward tokens/sec + host syncs/forward (must be 0), 1 MI355X",
        "value": head["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": head["workload"], "global_batch": cfg.batch, "seq_len": cfg.seq,
                   "parallelism": "single GPU"},
        "host_syncs_per_forward": head["host_syncs_per_forward"],
        "graph_launches_per_forward": head["graph_launches_per_forward"],
        "kernels_per_forward": head["kernels_per_forward"],
        "cold_ms": head["cold_ms"],
        "forward_frac_of_peak": head["forward_frac_of_peak"],
        "decisions_last_forward": {"regrow": dec["regrow"], "cached_len": dec["cached_len"],
                                   "pad_any": dec["pad_any"]},
        "roofline": roof,
        "kernel_breakdown_eager_ms": breakdown(prof),
    }
    if "fragmented_baseline" in head:
        result["fragmented_baseline"] = head["fragmented_baseline"]
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(cfg, w, ids, mask,
                                              [int(x) for x in args.cpu_depths.split(",")])
        log(f"[bench] cpu_baseline {result['cpu_baseline']}")
    del w
    if not args.no_configs:
        table = {WORKLOAD: {k: v for k, v in head.items() if k != "fragmented_baseline"}}
        if "fragmented_baseline" in head:
            table[WORKLOAD]["graph_broken_steady_speedup"] = head["fragmented_baseline"]["steady_speedup"]
        for name in TABLE:
            if name == WORKLOAD:
                continue
            r, _, _, _ = measure(name, args, frag=not args.no_fragmented)
            if "fragmented_baseline" in r:
                r["graph_broken_steady_speedup"] = r.pop("fragmented_baseline")["steady_speedup"]
            table[name] = r
            torch.cuda.empty_cache()
        result["configs"] = table
    if not args.no_decode:
        result["decode"] = decode_bench()
        log(f"[bench] decode: {result['decode']}")
        torch.cuda.empty_cache()
    if not args.no_seq2seq:
        result["seq2seq"] = seq2seq_bench(args)
        log(f"[bench] seq2seq: {result['seq2seq']}")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
