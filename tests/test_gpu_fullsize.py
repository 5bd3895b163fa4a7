"""GPU parity at the full sizes of the synthetic workloads.

Each model runs at its full shape in one graph launch (as in the benchmark);
the oracle recomputes what it can afford on the host: whole sequences of an
encoder (sequences are independent apart from the batch-wide padding
predicate, which the oracle still takes over the whole batch), a causal
prefix of the long decoder (with a causal mask a prefix does not depend on
later positions), and the whole batch of the fp16 clamp model (its clamp
predicate reads every sequence).

Depth and tolerance.  Two of the workloads amplify rounding-level
differences with depth: evaluating the oracle's own definition with float32
instead of float64 accumulation moves its logits by 0.38 (relative to the
largest logit) on the 24-layer fp16 clamp model (differences grow about
1.3x per layer) and by 0.0435 on the 32-layer rotary decoder.  No
implementation whose summation order differs from the oracle's can meet
2e-2 there.  So each is checked (a) at full width, batch and sequence with
the depth cut to where the same spread is below 2e-2 (8 layers: 0.0066; 2
layers), against 2e-2, and (b) at full depth with every decision and effect
exact and the logits within twice the measured spread.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import OracleModel

from test_gpu_parity import (check_decisions, check_logits, effects_of, f64,
                             gpu_effects, gpu_model, run)

pytestmark = pytest.mark.gpu

# twice the float32-vs-float64 spread of the oracle itself at full depth
FULL_DEPTH_TOL = {"encoder_clamp_1024": 2 * 0.38, "decoder_4096": 2 * 0.0435}


def test_full_encoder_1024_sampled_sequences():
    cfg = synth.preset("encoder_1024")
    w = synth.make_weights(cfg, 77)
    ids, mask = synth.make_inputs(cfg, 1)
    print("pads per sequence", (mask == 0).sum(1).tolist(), flush=True)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    rows = [0, 9]
    res = OracleModel(cfg, w).forward(ids, mask, rows=rows)
    check_logits(f64(out[rows]), res.logits_f64, cfg.dtype, "encoder_1024 rows 0,9")
    check_decisions(m.decisions(), res, cfg)
    assert res.pad_any


def _clamp_case(cfg, wseed, tol):
    w = synth.make_weights(cfg, wseed)
    for seed in range(3):
        ids, mask = synth.make_inputs(cfg, seed)
        res = OracleModel(cfg, w).forward(ids, mask)
        margins = [x for pair in res.clamp_margin for x in pair]
        if min(margins) > 1.0:
            break
        print(f"seed {seed}: a clamp decision lies within 1.0 of its boundary, next seed")
    flat = [t for pair in res.clamp for t in pair]
    print("oracle clamp sites", flat, flush=True)
    assert any(flat) and not all(flat)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    check_decisions(m.decisions(), res, cfg)
    assert gpu_effects(m) == effects_of(res)
    check_logits(f64(out), res.logits_f64, cfg.dtype, f"{cfg.name} {cfg.n_layers} layers", tol)


def test_encoder_clamp_1024_full_width_8_layers():
    _clamp_case(synth.preset("encoder_clamp_1024", n_layers=8), 5, None)


def test_encoder_clamp_1024_full_depth():
    _clamp_case(synth.preset("encoder_clamp_1024"), 5, FULL_DEPTH_TOL["encoder_clamp_1024"])


def _rotary_case(cfg, prefix, tol):
    w = synth.make_weights(cfg, 11)
    ids, mask = synth.make_inputs(cfg, 0)
    m = gpu_model(cfg, w)
    out1 = run(m, ids, mask)
    d1 = m.decisions()
    out2 = run(m, ids, mask)
    d2 = m.decisions()
    print("regrow", d1["regrow"], d2["regrow"], "cached", d1["cached_len"], d2["cached_len"],
          flush=True)
    orc = OracleModel(cfg, w)
    r1 = orc.forward(ids, mask, prefix=prefix)
    r2 = orc.forward(ids, mask, prefix=prefix)
    assert (r1.regrow, r2.regrow) == (True, False)
    check_decisions(d1, r1, cfg)
    check_decisions(d2, r2, cfg)
    check_logits(f64(out1[:, :prefix]), r1.logits_f64, cfg.dtype,
                 f"decoder_4096 {cfg.n_layers} layers prefix {prefix}", tol)
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    assert gpu_effects(m) == effects_of(r1) + effects_of(r2)


def test_decoder_4096_full_width_2_layers():
    _rotary_case(synth.preset("decoder_4096", n_layers=2), 256, None)


def test_decoder_4096_full_depth():
    _rotary_case(synth.preset("decoder_4096"), 96, FULL_DEPTH_TOL["decoder_4096"])
