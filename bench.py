#!/usr/bin/env python3
"""Steady-state forward throughput of libgm on one MI355X.

Workload: the 12-layer causal LM decoder (d_model 768, 12 heads, FFN 3072
GELU, pre-LayerNorm, learned positions, vocab 50257, bf16) over a batch of
8 x 512 tokens with 0..128 trailing pads per sequence (synthetic weights
N(0, 0.02), uniform token ids).  One step = one gm_forward: a single
hipGraphLaunch of the whole forward, every data-dependent branch (padding
mask, guards, effects) resolved on the device.

Prints one JSON line with the throughput, the host syncs per forward (from
the library's counters), a roofline entry for the dominant kernel (the MFMA
GEMM) measured with HIP events on the launch stream, and the CPU oracle
timed on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = "causal_lm_768"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def time_steps(m, ids_t, mask_t, out, steps, warmup):
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
    """First forward on a new (batch, sequence, buffers) key in a warm process:
    capture + instantiate + run of its graph(s)."""
    import torch
    out = m.new_logits(*ids_t.shape)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    m.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3, out


def fragmented(m, ids_t, mask_t, args):
    """The same forward run as the unmended program (one graph per region
    between graph breaks; host sync + read-back + host branch at each break)
    next to the single-graph forward, both measured the same way (wall clock
    around the loop, synchronised at both ends)."""
    cold_g, out = cold_call(m, ids_t, mask_t)
    ms_g = time_steps(m, ids_t, mask_t, out, args.steps, args.warmup)
    m.set_exec_mode("fragmented")
    s0 = m.stats()
    cold_f, out = cold_call(m, ids_t, mask_t)
    s1 = m.stats()
    ms_f = time_steps(m, ids_t, mask_t, out, args.steps, args.warmup)
    s2 = m.stats()
    m.set_exec_mode("graph")
    runs = args.steps + args.warmup
    return {"single_graph": {"ms_per_step": round(ms_g, 4), "cold_ms": round(cold_g, 2)},
            "fragmented": {"ms_per_step": round(ms_f, 4), "cold_ms": round(cold_f, 2),
                           "graphs_per_forward": (s2["graph_launches"] - s1["graph_launches"]) / runs,
                           "host_syncs_per_forward": (s2["host_syncs_in_forward"] - s1["host_syncs_in_forward"]) / runs,
                           "graphs_captured": s1["captures"] - s0["captures"]},
            "steady_speedup": round(ms_f / ms_g, 3), "cold_speedup": round(cold_f / cold_g, 3)}


def break_suite(args):
    """Single graph vs graph-broken forward on every workload (stderr)."""
    import torch
    import synth
    from paper_2509_16248_amd.model import GmModel
    for name in ["tiny_decoder", "causal_lm_768", "encoder_1024", "encoder_clamp_1024",
                 "decoder_4096"]:
        cfg = synth.preset(name)
        w = synth.make_weights(cfg, 5)
        ids, mask = synth.make_inputs(cfg, 0)
        m = GmModel(cfg, w.globals, w.layers, device="cuda:0")
        del w
        ids_t = torch.from_numpy(ids).cuda()
        mask_t = torch.from_numpy(mask).cuda()
        cold_call(m, ids_t, mask_t)           # first capture of the process for this model
        r = fragmented(m, ids_t, mask_t, args)
        r["tokens"] = int(ids.size)
        log("[breaks] " + json.dumps({name: r}))
        m.close()
        torch.cuda.empty_cache()


def seq2seq_bench(args):
    """The encoder-decoder workload (6 + 6 layers, d 768, batch 8, source 512,
    target 128, ragged): single-graph forwards timed with events, then the
    graph-broken program on the same buffers.  Throughput counts source and
    target positions."""
    import torch
    import synth
    from paper_2509_16248_amd.model import GmModel
    cfg = synth.preset("seq2seq_768")
    w = synth.make_weights(cfg, 1234)
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


def decode_bench(cfg, w, prompt=384, steps=120, warmup=8):
    """Greedy decoding with the KV cache on the benchmarked model: prefill
    B x ``prompt`` positions (ragged, 0..128 trailing pads), then ``steps``
    decode steps in which each step's greedy tokens (device argmax) are the
    next step's input, one graph launch per step and no host read.  The
    step is HBM-bound: its algorithmic bytes are every weight read once plus
    the cached keys and values of every sequence up to its position."""
    import numpy as np
    import torch
    import synth
    from paper_2509_16248_amd.model import GmModel
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


def measured_traffic():
    """HBM bytes per GEMM launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary, if it was taken on the GEMM source as it is now."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "gemm_traffic_causal_lm_768.json")
    src = os.path.join(ROOT, "paper_2509_16248_amd", "csrc", "gm_gemm.hip")
    try:
        rec = json.load(open(path))
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    return rec["traffic_bytes_per_launch"] if rec.get("gm_gemm_hip_sha256") == sha else None


def cpu_baseline(cfg, w, ids, mask, rows):
    """The oracle (float64 NumPy) on `rows` sequences of the same batch."""
    import numpy as np
    from oracle import OracleModel
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    m = OracleModel(cfg, w)
    t0 = time.perf_counter()
    m.forward(ids, mask, rows=rows)
    dt = time.perf_counter() - t0
    tokens = len(rows) * ids.shape[1]
    return {"value": tokens / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(rows)} of {ids.shape[0]} sequences x {ids.shape[1]} tokens "
                      f"(full 12-layer forward + LM head), {dt:.2f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=8)
    ap.add_argument("--no-fragmented", action="store_true",
                    help="skip the graph-broken baseline (same kernels, host sync per break)")
    ap.add_argument("--no-decode", action="store_true", help="skip the KV-cache decode measurement")
    ap.add_argument("--no-seq2seq", action="store_true",
                    help="skip the encoder-decoder measurement")
    ap.add_argument("--seq2seq-only", action="store_true",
                    help="only the encoder-decoder measurement (one JSON object)")
    ap.add_argument("--break-suite", action="store_true",
                    help="only compare single-graph and graph-broken forwards on every workload")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (got --gpus {args.gpus}); "
              "the multi-GPU layout is a design only, not built", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2509_16248_amd.model import GmModel

    if args.break_suite:
        break_suite(args)
        return
    if args.seq2seq_only:
        print(json.dumps(seq2seq_bench(args)), flush=True)
        return
    cfg = synth.preset(WORKLOAD)
    B, S = cfg.batch, cfg.seq
    log(f"[bench] generating weights for {WORKLOAD}")
    w = synth.make_weights(cfg, 1234)
    ids, mask = synth.make_inputs(cfg, 0)
    m = GmModel(cfg, w.globals, w.layers, device="cuda:0")
    ids_t = torch.from_numpy(ids).cuda()
    mask_t = torch.from_numpy(mask).cuda()
    out = m.new_logits(B, S)
    stream = torch.cuda.current_stream()

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    m.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    cold_ms = (time.perf_counter() - t0) * 1e3
    log(f"[bench] cold forward (capture + instantiate + run) {cold_ms:.2f} ms")
    for _ in range(args.warmup):
        m.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    s0 = m.stats()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        m.forward(ids_t, mask_t, out)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    s1 = m.stats()
    syncs = (s1["host_syncs_in_forward"] - s0["host_syncs_in_forward"]) / args.steps
    launches = (s1["graph_launches"] - s0["graph_launches"]) / args.steps
    log(f"[bench] {ms:.4f} ms/forward, graph launches/forward {launches}, "
        f"host syncs/forward {syncs}, kernels/forward {s1['kernels_per_forward']}")

    # per-kernel durations: eager forwards with events between the kernels
    prof = None
    for _ in range(3):
        prof = m.profile(ids_t, mask_t, out)
    by_kind = {}
    for kind, layer, kms, flops, nbytes in prof:
        t = by_kind.setdefault(kind, [0, 0.0, 0.0, 0.0])
        t[0] += 1
        t[1] += kms
        t[2] += flops
        t[3] += nbytes
    gemm = [p for p in prof if p[0].startswith("gemm")]
    g_ms = sum(p[2] for p in gemm)
    g_flops = sum(p[3] for p in gemm)
    g_avg_ms = g_ms / len(gemm)
    achieved = g_flops / (g_ms * 1e-3) / 1e12
    roofline = {"kernel": "k_gemm_x<bf16,128,128,2,4,2> (all projection and LM-head GEMMs)",
                "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic(), "launches_per_forward": len(gemm),
                "avg_launch_ms": round(g_avg_ms, 5),
                "flops_per_launch_avg": g_flops / len(gemm)}
    breakdown = {k: {"launches": v[0], "ms": round(v[1], 4),
                     "tflops": round(v[2] / (v[1] * 1e-3) / 1e12, 2) if v[2] else None,
                     "gbs": round(v[3] / (v[1] * 1e-3) / 1e9, 1) if v[3] and not v[2] else None}
                 for k, v in by_kind.items()}
    log(f"[bench] kernel breakdown (eager, ms): " +
        ", ".join(f"{k}={v['ms']}" for k, v in breakdown.items()))

    result = {
        "metric": "steady-state forward tokens/sec + host syncs/forward (must be 0), 1 MI355X",
        "value": round(B * S / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "causal_lm_768: 12-layer causal LM decoder, d_model 768, "
                               "12 heads, FFN 3072 GELU, pre-LayerNorm, learned positions, "
                               "vocab 50257, bf16, weights N(0,0.02)",
                   "global_batch": B, "seq_len": S,
                   "pad_tokens": int((mask == 0).sum()), "parallelism": "single GPU"},
        "host_syncs_per_forward": syncs,
        "graph_launches_per_forward": launches,
        "kernels_per_forward": s1["kernels_per_forward"],
        "cold_ms": round(cold_ms, 2),
        "nonpad_tokens_per_s": round(int(mask.sum()) / (ms * 1e-3), 1),
        "roofline": roofline,
        "kernel_breakdown_eager_ms": breakdown,
    }
    if not args.no_fragmented:
        result["fragmented_baseline"] = fragmented(m, ids_t, mask_t, args)
        log(f"[bench] single graph vs graph-broken: {result['fragmented_baseline']}")
    m.close()
    if not args.no_decode:
        torch.cuda.empty_cache()
        result["decode"] = decode_bench(cfg, w)
        log(f"[bench] decode: {result['decode']}")
    if not args.no_seq2seq:
        torch.cuda.empty_cache()
        result["seq2seq"] = seq2seq_bench(args)
        log(f"[bench] seq2seq: {result['seq2seq']}")
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(cfg, w, ids, mask, list(range(args.cpu_rows)))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
