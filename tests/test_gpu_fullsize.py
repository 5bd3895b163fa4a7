"""GPU parity at the full sizes of the synthetic workloads.

Each model runs at its full shape in one graph launch (as in the benchmark);
the oracle recomputes what it can afford on the host: whole sequences of an
encoder (sequences are independent apart from the batch-wide padding
predicate, which the oracle still takes over the whole batch), all 2048
positions of the long decoder at 2 and at 32 layers, and the whole batch of
the fp16 clamp model (its clamp predicate reads every sequence).  Every
step of every layer of the two deep models is compared at 2e-2 in
test_gpu_stepwise.py.

Depth and tolerance.  Two of the workloads amplify rounding-level
differences with depth.  tests/golden/depth_spread.py measures how far the
oracle's own program moves when it is evaluated with float32 instead of
float64 arithmetic (relative to the largest logit): for the fp16 clamp
model 0.0076 at 2 layers, 0.0165 at 4, 0.056 at 8 and 1.04 at 24 (its q/k
outliers make attention a near-argmax, the overflowing residual stream is
clamped at every site after the first); for the 32-layer rotary decoder over
all 2048 positions the value stored in depth_spread.json.  No implementation whose summation order
differs from the oracle's can be held closer than that.  So the logits are
compared at 2e-2 where the spread is below 1e-2 (2 layers), within twice the
spread where it is larger but informative (8 layers, the 32-layer decoder),
and not at all where it is about 1 (the 24-layer clamp model: its decisions
and effects are still compared exactly, and test_gpu_stepwise.py checks every
step of every layer).
"""
import json
import os

import numpy as np
import pytest
import torch

import synth
from oracle import OracleModel

from test_gpu_parity import (check_decisions, check_logits, effects_of, f64,
                             gpu_effects, gpu_model, run)

pytestmark = pytest.mark.gpu

# the float32-vs-float64 spread of the oracle's own program (depth_spread.py)
SPREAD = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                     "depth_spread.json")))


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
    if tol is not False:
        check_logits(f64(out), res.logits_f64, cfg.dtype, f"{cfg.name} {cfg.n_layers} layers", tol)


def test_encoder_clamp_1024_full_width_2_layers():
    _clamp_case(synth.preset("encoder_clamp_1024", n_layers=2), 5, None)


def test_encoder_clamp_1024_full_width_8_layers():
    _clamp_case(synth.preset("encoder_clamp_1024", n_layers=8), 5,
                2 * SPREAD["encoder_clamp_1024"]["8"])


def test_encoder_clamp_1024_full_depth():
    """Decisions of all 48 sites and the effect records, exactly; the logits
    carry no information at this depth (spread about 1, see above)."""
    assert SPREAD["encoder_clamp_1024"]["24"] > 0.5
    _clamp_case(synth.preset("encoder_clamp_1024"), 5, False)


def _say_layer(l):
    print(f"oracle layer {l} done", flush=True)


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
    r1 = orc.forward(ids, mask, prefix=prefix, progress=_say_layer)
    r2 = orc.forward(ids, mask, prefix=1)   # its decisions and effects; its logits are out1's
    assert (r1.regrow, r2.regrow) == (True, False)
    check_decisions(d1, r1, cfg)
    check_decisions(d2, r2, cfg)
    n = r1.logits_f64.shape[1]
    check_logits(f64(out1[:, :n]), r1.logits_f64, cfg.dtype,
                 f"decoder_4096 {cfg.n_layers} layers, positions [0, {n})", tol)
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    assert gpu_effects(m) == effects_of(r1) + effects_of(r2)


def test_decoder_4096_full_width_2_layers():
    """Every one of the 2048 positions: rows [1024, 2048) of the regrown
    rotary table, rotations at angles up to 2047 rad, and attention over up to
    2048 keys at head size 128."""
    _rotary_case(synth.preset("decoder_4096", n_layers=2), None, None)


def test_decoder_4096_full_depth():
    """All 32 layers over every one of the 2048 positions (the oracle's
    float64 forward of the whole sequence takes minutes on the host)."""
    _rotary_case(synth.preset("decoder_4096"), None, 2 * SPREAD["decoder_4096"]["32_all"])
