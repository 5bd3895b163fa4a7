"""GPU parity of the three remaining rewrite patterns of real models, each
checked against the oracle:

* a `torch.equal(attention_mask, expected)` validation guard lowered by
  rule [Trap] (host metadata check, device (mask == expected).all(), a code
  that maps back to the original exception type and message);
* a tensor-valued log (max |h| of every sequence after every layer)
  deferred by rule [Defer]: the values are taken on the device at the call
  site and replayed in program order after the forward;
* the Phi-4-style long/short rotary frequency select (rule [Where] with the
  memoised initialisations of both sets hoisted to model creation).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import EFFECT_LOG, TRAP_INFO, TRAP_MASK_GUARD, OracleModel, Trap
from paper_2509_16248_amd import gm

from test_gpu_parity import (TOL, check_decisions, check_logits, effects_of, f64, gpu_effects,
                             gpu_model, run)

pytestmark = pytest.mark.gpu


def test_trap_info_matches_the_original_exceptions():
    for code, (typ, msg) in TRAP_INFO.items():
        assert gm.gm_trap_info(code) == (typ, msg)


def test_mask_guard_passes_fails_and_maps_to_the_original_exception():
    cfg = synth.preset("tiny_decoder", batch=2, max_pad=4)
    w = synth.make_weights(cfg, 51)
    ids, mask = synth.make_inputs(cfg, 6)
    m = gpu_model(cfg, w)
    plain = run(m, ids, mask).clone()
    good = torch.from_numpy(mask.copy()).cuda()
    m.set_mask_guard(good)
    out = run(m, ids, mask)
    assert torch.equal(out, plain)
    assert m.check_error() == (0, 0)
    orc = OracleModel(cfg, w)
    bad = mask.copy()
    bad[1, 5] ^= 1
    orc.mask_guard = bad
    with pytest.raises(Trap) as e:
        orc.forward(ids, mask)
    m.set_mask_guard(torch.from_numpy(bad).cuda())
    run(m, ids, mask)
    with pytest.raises(ValueError, match="unsupported attention mask") as err:
        m.raise_on_trap()
    assert (err.value.trap_code, err.value.trap_index) == (e.value.code, e.value.index)
    assert e.value.code == TRAP_MASK_GUARD
    # a guard tensor of another shape never compares equal
    m.set_mask_guard(torch.from_numpy(mask[:, :-1].copy()).cuda())
    run(m, ids, mask)
    assert m.check_error() == (TRAP_MASK_GUARD, 0)
    # the unmended program stops at the guard
    m.set_mask_guard(torch.from_numpy(bad).cuda())
    m.set_exec_mode("fragmented")
    with pytest.raises(gm.GmError) as ge:
        run(m, ids, mask)
    assert ge.value.code == gm.GM_E_TRAP
    m.set_exec_mode("graph")
    m.set_mask_guard(None)
    assert m.check_error() == (TRAP_MASK_GUARD, 5 + cfg.seq)
    assert torch.equal(run(m, ids, mask), plain)


def _log_case(cfg, w, ids, mask):
    orc = OracleModel(cfg, w)
    res = orc.forward(ids, mask)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    check_logits(f64(out), res.logits_f64, cfg.dtype, cfg.name)
    got = gpu_effects(m, with_values=True)
    want = res.effects
    assert [(g[0], g[1], g[2], g[3]) for g in got] == [(e.forward, e.kind, e.layer, e.site)
                                                        for e in want]
    tol = TOL[cfg.dtype]
    for g, e in zip(got, want):
        if e.kind != EFFECT_LOG:
            assert g[4] == np.float32(e.value)
            continue
        ref = np.array(e.values)
        val = np.array(g[5], dtype=np.float64)
        err = np.abs(val - ref).max() / np.abs(ref).max()
        print(f"layer {e.layer} log max|h| per sequence gpu {val} oracle {ref} rel {err:.3g}")
        assert err <= tol
    return m, out


def test_tensor_log_values_and_program_order():
    cfg = synth.reduced("causal_lm_768").replace(log_hidden=True)
    w = synth.make_weights(cfg, 52)
    ids, mask = synth.make_inputs(cfg, 2)
    m, out = _log_case(cfg, w, ids, mask)
    # the unmended program copies each logged tensor to the host at once
    m.set_exec_mode("fragmented")
    s0 = m.stats()
    out2 = run(m, ids, mask)
    s1 = m.stats()
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))
    assert s1["host_syncs_in_forward"] - s0["host_syncs_in_forward"] == 1 + cfg.n_layers


def test_tensor_log_with_clamp_sites():
    cfg = synth.reduced("encoder_clamp_1024").replace(log_hidden=True)
    w = synth.make_weights(cfg, 7)
    ids, mask = synth.make_inputs(cfg, 0)
    _log_case(cfg, w, ids, mask)


@pytest.mark.parametrize("seq", [100, 128, 129, 300])
def test_long_short_rope_select(seq):
    cfg = synth.reduced("decoder_4096_longrope")
    w = synth.make_weights(cfg, 53)
    ids, mask = synth.make_inputs(cfg, 3, seq=seq)
    res = OracleModel(cfg, w).forward(ids, mask)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    d = m.decisions()
    print(f"S={seq}: long {d['rope_long']} (oracle {res.rope_long})")
    assert d["rope_long"] == res.rope_long == (seq > cfg.rope_orig_max)
    check_decisions(d, res, cfg)
    check_logits(f64(out), res.logits_f64, cfg.dtype, f"longrope S={seq}")


def test_full_width_decoder_4096_longrope_2_layers():
    cfg = synth.preset("decoder_4096_longrope", n_layers=2)
    w = synth.make_weights(cfg, 11)
    ids, mask = synth.make_inputs(cfg, 0)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    res = OracleModel(cfg, w).forward(ids, mask, prefix=256)
    assert m.decisions()["rope_long"] and res.rope_long
    check_logits(f64(out[:, :256]), res.logits_f64, cfg.dtype, "decoder_4096_longrope prefix 256")
