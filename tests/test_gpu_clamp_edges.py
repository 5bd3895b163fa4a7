"""GPU parity of the fp16 overflow branch at its edges (rule [Where]: the
branch becomes a select, and the untaken input may hold NaN/Inf that must not
reach the output; Semantics Preservation section).

A one-layer model of the clamp workload's width, with biases, whose layer 0
has Wo = 0 and W1 = b1 = W2 = b2 = 0: the attention site then stores exactly
R(h + bo) and the FFN site exactly the selected stream (plus a zero FFN),
so the bias and the embedding place chosen values at the sites:

* 64480 + 15 = 64495 rounds to 64480: below the threshold, no clamp;
* 64480 + 16 = 64496, the midpoint, rounds (to even) to 64512: clamp;
* 64480 + 24 = 64504 rounds to 64512: clamp;
* +inf in one column and no NaN: clamp, the inf becomes 64512;
* +inf in one column and NaN in another: `max` propagates NaN, the
  comparison is false, no clamp: the inf survives and the NaN spreads.

Decisions, the largest magnitude and the NaN flag of every site, the effect
records and the logits (NaN where the oracle has NaN, the rest within 2e-2)
are compared with the oracle.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import OracleModel

from test_gpu_parity import effects_of, f64, gpu_effects, gpu_model, run

pytestmark = pytest.mark.gpu

C0, C1 = 37, 500          # columns that receive the chosen values
T0 = 11                   # token whose embedding row holds 64480 at C0


def _model(bo_c0, bo_c1=0.0, emb=None):
    cfg = synth.reduced("encoder_clamp_1024").replace(n_layers=1, bias=True)
    w = synth.make_weights(cfg, 3)
    L = w.layers[0]
    for name in ("wo", "w1", "b1", "w2", "b2"):
        L[name][:] = 0
    bo = np.zeros_like(L["bo"])
    bo[C0] = np.float16(bo_c0)
    bo[C1] = np.float16(bo_c1)
    L["bo"] = bo
    if emb is not None:
        w.globals["tok_emb"][T0, C0] = np.float16(emb)
    ids, mask = synth.make_inputs(cfg, 1)
    ids[0, 5] = T0
    ids[1, 100] = T0
    return cfg, w, ids, mask


def _compare_logits(got, ref, tol=2e-2):
    nan_g, nan_r = np.isnan(got), np.isnan(ref)
    assert np.array_equal(nan_g, nan_r), (nan_g.sum(), nan_r.sum())
    fin = ~nan_r
    if fin.any():
        scale = np.abs(ref[fin]).max()
        err = np.abs(got[fin] - ref[fin]).max() / scale
        print(f"finite logits rel={err:.3g}", flush=True)
        assert err <= tol


def _check(cfg, w, ids, mask, want):
    """want: per site (trip, absmax, nan) expected from the construction."""
    res = OracleModel(cfg, w).forward(ids, mask)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    dec = m.decisions()
    flat = [t for pair in res.clamp for t in pair]
    am = [np.float32(v) for pair in res.clamp_absmax for v in pair]
    nans = [bool(v) for pair in res.clamp_nan for v in pair]
    print("oracle", flat, am, nans, "gpu", dec["clamp"], dec["clamp_absmax"], dec["clamp_nan"],
          flush=True)
    assert [(t, a, n) for t, a, n in zip(flat, am, nans)] == want
    assert dec["clamp"] == flat
    assert [np.float32(v) for v in dec["clamp_absmax"]] == am
    assert dec["clamp_nan"] == nans
    assert gpu_effects(m) == effects_of(res)
    _compare_logits(f64(out), res.logits_f64)
    return m, res


@pytest.mark.parametrize("bias,stored,trip", [(15.0, 64480.0, False), (16.0, 64512.0, True),
                                              (24.0, 64512.0, True)])
def test_clamp_rounding_boundary(bias, stored, trip):
    cfg, w, ids, mask = _model(bias, emb=64480.0)
    # the FFN site stores the selected stream: 64504 clamps to 64512 again
    want = [(trip, np.float32(stored), False), (trip, np.float32(stored), False)]
    _check(cfg, w, ids, mask, want)


def test_clamp_inf_without_nan_is_clamped():
    cfg, w, ids, mask = _model(np.inf)
    m, res = _check(cfg, w, ids, mask, [(True, np.float32(np.inf), False),
                                         (True, np.float32(64512.0), False)])
    ids_t = torch.from_numpy(ids).cuda()
    mask_t = torch.from_numpy(mask).cuda()
    dump = m.forward_layers(ids_t, mask_t, m.new_logits(*ids.shape))
    torch.cuda.synchronize()
    assert torch.isinf(dump["h_mid"][0][:, C0]).all()          # before the select
    assert (dump["h_out"][0][:, C0].float() == 64512.0).all()   # after it
    assert torch.isfinite(dump["a2"][0]).all()
    m.close()


def test_clamp_nan_disables_the_branch_and_inf_survives():
    cfg, w, ids, mask = _model(np.inf, np.nan)
    # FFN site: every row read a NaN through the norm, so the stream is NaN
    # everywhere (max |h| over non-NaN elements: none, 0)
    m, res = _check(cfg, w, ids, mask, [(False, np.float32(np.inf), True),
                                         (False, np.float32(0.0), True)])
    ids_t = torch.from_numpy(ids).cuda()
    mask_t = torch.from_numpy(mask).cuda()
    dump = m.forward_layers(ids_t, mask_t, m.new_logits(*ids.shape))
    torch.cuda.synchronize()
    assert torch.isinf(dump["h_mid"][0][:, C0]).all()
    assert torch.isnan(dump["a2"][0]).all()
    m.close()
