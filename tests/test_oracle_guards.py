"""Pins for the oracle's validation guard, tensor-valued log and long/short
rotary select (CPU only).

* scaled rotary table: position 0 is cos = attn, sin = 0 exactly; the
  attention factor is one float32 product on the unscaled entries; a
  constant factor f is a time dilation (the table at position p*f equals the
  unscaled table at p, to float32 rounding); factor 1 agrees with the
  plain table (which rounds the frequency through a power instead of a
  quotient) to float32 rounding;
* long/short select: the decision is max(position) + 1 > original context;
  with equal long and short factors the decision changes nothing (bit for
  bit); with different factors the whole sequence, its earlier positions
  included, follows the set the decision picks;
* guard `if not torch.equal(mask, expected): raise`: equal masks pass and
  change nothing; the first differing element is reported; different
  shapes fail; guard order by code; the exception table names the original
  type and message;
* tensor log: sequences with equal inputs log equal values, a change in one
  sequence changes only its value, and the records sit in program order
  with the clamp sites.
"""
import numpy as np
import pytest

import synth
from oracle import (EFFECT_CLAMP, EFFECT_LOG, TRAP_INFO, TRAP_MASK_GUARD, TRAP_ROPE_CAPACITY,
                    TRAP_TOKEN_RANGE, OracleModel, Trap)
from oracle import numerics as nx


def tiny_longrope(**kw):
    base = synth.preset("decoder_4096", n_layers=2, d_model=64, n_heads=2, d_ff=128,
                        vocab=101, batch=2, seq=24, rope_capacity=32)
    return synth._longrope(base, 12).replace(**kw)


def test_scaled_table_closed_forms():
    hd, n = 16, 40
    f = np.linspace(1.0, 9.0, hd // 2).astype(np.float32)
    c, s = nx.rope_table_scaled(n, hd, 10000.0, f, 1.25)
    assert (c[0] == np.float32(1.25)).all() and (s[0] == 0).all()
    c1, s1 = nx.rope_table_scaled(n, hd, 10000.0, f, 1.0)
    np.testing.assert_array_equal(c, (c1.astype(np.float32) * np.float32(1.25)).astype(np.float32))
    np.testing.assert_array_equal(s, (s1.astype(np.float32) * np.float32(1.25)).astype(np.float32))
    # constant factor 4: position 4p of the scaled table is position p unscaled
    c4, s4 = nx.rope_table_scaled(4 * n, hd, 10000.0, np.full(hd // 2, 4.0, np.float32), 1.0)
    cu, su = nx.rope_table_scaled(n, hd, 10000.0, np.ones(hd // 2, np.float32), 1.0)
    np.testing.assert_allclose(c4[::4], cu, atol=2e-5)
    np.testing.assert_allclose(s4[::4], su, atol=2e-5)
    cp, sp = nx.rope_table(n, hd, 10000.0)
    np.testing.assert_allclose(cu, cp, atol=2e-5)
    np.testing.assert_allclose(su, sp, atol=2e-5)


def test_long_short_decision_and_what_it_selects():
    cfg = tiny_longrope()
    w = synth.make_weights(cfg, 41)
    orc = OracleModel(cfg, w)
    ids, mask = synth.make_inputs(cfg, 1, max_pad=0)
    short = orc.forward(ids[:, :12], mask[:, :12])
    long_ = orc.forward(ids[:, :13], mask[:, :13])
    assert (short.rope_long, long_.rope_long) == (False, True)
    assert short.cached_len == long_.cached_len == cfg.rope_capacity
    # the longer sequence re-rotates its first 12 positions with the long set
    assert not np.allclose(short.logits_f64, long_.logits_f64[:, :12])
    # equal factor sets: the decision makes no difference at all
    w.globals["rope_long_factor"] = w.globals["rope_short_factor"].copy()
    same = OracleModel(cfg, w)
    a = same.forward(ids[:, :12], mask[:, :12]).logits_f64
    b = same.forward(ids[:, :13], mask[:, :13]).logits_f64[:, :12]
    np.testing.assert_array_equal(a, b)


def test_mask_guard():
    cfg = synth.preset("tiny_decoder", batch=2, max_pad=4)
    w = synth.make_weights(cfg, 42)
    ids, mask = synth.make_inputs(cfg, 2)
    plain = OracleModel(cfg, w).forward(ids, mask)
    orc = OracleModel(cfg, w)
    orc.mask_guard = mask.copy()
    np.testing.assert_array_equal(orc.forward(ids, mask).logits_f64, plain.logits_f64)
    bad = mask.copy()
    bad[1, 3] ^= 1
    orc.mask_guard = bad
    with pytest.raises(Trap) as e:
        orc.forward(ids, mask)
    assert (e.value.code, e.value.index) == (TRAP_MASK_GUARD, cfg.seq + 3)
    orc.mask_guard = mask[:, :-1].copy()
    with pytest.raises(Trap) as e:
        orc.forward(ids, mask)
    assert (e.value.code, e.value.index) == (TRAP_MASK_GUARD, 0)
    orc.mask_guard = mask.astype(np.int64)            # same values, another dtype
    with pytest.raises(Trap) as e:
        orc.forward(ids, mask)
    assert e.value.code == TRAP_MASK_GUARD
    ids2 = ids.copy()
    ids2[0, 0] = cfg.vocab
    orc.mask_guard = bad
    with pytest.raises(Trap) as e:
        orc.forward(ids2, mask)
    assert e.value.code == TRAP_TOKEN_RANGE
    assert TRAP_INFO[TRAP_MASK_GUARD] == ("ValueError", "unsupported attention mask")
    rot = synth.preset("decoder_4096", n_layers=1, d_model=64, n_heads=2, d_ff=128, vocab=50,
                       batch=1, seq=10, rope_init_len=4, rope_capacity=8)
    ro = OracleModel(rot, synth.make_weights(rot, 43))
    ids3, mask3 = synth.make_inputs(rot, 3)
    ro.mask_guard = 1 - mask3
    with pytest.raises(Trap) as e:                    # the rotary capacity guard comes first
        ro.forward(ids3, mask3)
    assert e.value.code == TRAP_ROPE_CAPACITY


def test_tensor_log_values_and_order():
    cfg = synth.preset("tiny_decoder", batch=3, max_pad=0, n_layers=2, log_hidden=True)
    w = synth.make_weights(cfg, 44)
    ids, mask = synth.make_inputs(cfg, 4)
    ids[1] = ids[0]
    res = OracleModel(cfg, w).forward(ids, mask)
    logs = [e for e in res.effects if e.kind == EFFECT_LOG]
    assert [e.layer for e in logs] == [0, 1] and all(len(e.values) == 3 for e in logs)
    for e in logs:
        assert e.values[0] == e.values[1] != e.values[2]
    ids2 = ids.copy()
    ids2[2, 0] = (ids2[2, 0] + 1) % cfg.vocab
    res2 = OracleModel(cfg, w).forward(ids2, mask)
    for a, b in zip(logs, [e for e in res2.effects if e.kind == EFFECT_LOG]):
        assert a.values[:2] == b.values[:2] and a.values[2] != b.values[2]
    # with the clamp sites: per layer, site 0, site 1, then the log
    cl = synth.preset("encoder_clamp_1024", n_layers=3, d_model=64, n_heads=4, d_ff=128,
                      vocab=89, batch=2, seq=16, outlier_scale=800.0, log_hidden=True)
    r = OracleModel(cl, synth.make_weights(cl, 5)).forward(*synth.make_inputs(cl, 0))
    order = [(e.layer, e.kind, e.site) for e in r.effects if e.kind in (EFFECT_CLAMP, EFFECT_LOG)]
    assert any(k == EFFECT_CLAMP for _, k, _ in order)
    assert order == sorted(order, key=lambda t: (t[0], t[1] == EFFECT_LOG, t[2]))
