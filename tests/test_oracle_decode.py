"""Pins for the decode oracle (CPU only).

The decode oracle recomputes each step as a forward over the extended
sequences.  What it adds to the pinned forward is bookkeeping (which
positions continue which sequence, the padded batch it builds, the row it
reads, the guards, the rotary decisions and effects of a step, the greedy
choice), so that is what is pinned here:
* greedy: hand-computed indices for ties, NaN and -inf rows;
* batch independence: a sequence decoded inside a padded batch gives the
  same logits (to float64 summation-order level) as the same sequence
  decoded alone with no padding;
* causality: after a few steps, one forward over the final sequence gives,
  at every generated position, the logits the steps produced;
* the rotary decision sequence of a decode loop against its closed form
  (regrow exactly when the new length exceeds every earlier one and the
  initial table), with one REGROW record per regrow;
* guard codes and indices, and a trapped step leaving the state alone.
"""
import numpy as np
import pytest

import synth
from oracle import (EFFECT_REGROW, TRAP_KV_CAPACITY, TRAP_ROPE_CAPACITY, TRAP_TOKEN_RANGE,
                    OracleDecoder, OracleModel, Trap, generate_greedy, greedy)


def tiny_lm():
    return synth.preset("tiny_decoder", seq=32, batch=3, max_pad=5)


def tiny_rotary():
    return synth.preset("decoder_4096", n_layers=2, d_model=64, n_heads=2, d_ff=128,
                        vocab=101, batch=2, seq=40, rope_init_len=12, rope_capacity=40)


def test_greedy_ties_nan_and_inf():
    assert greedy(np.array([1.0, 3.0, 3.0, 2.0])) == 1
    assert greedy(np.array([5.0, np.nan, 7.0, np.nan])) == 1
    assert greedy(np.array([-np.inf, -np.inf])) == 0
    assert greedy(np.array([-1.0, -np.inf, -0.5])) == 2


def test_sequence_in_padded_batch_equals_sequence_alone():
    cfg = tiny_lm()
    w = synth.make_weights(cfg, 21)
    ids, mask = synth.make_inputs(cfg, 4, seq=14)
    mask[0, 10:] = 0            # three different lengths
    mask[1, 13:] = 0
    mask[2, :] = 1
    steps = [[5, 6, 7], [11, 12, 13], [100, 200, 300]]
    dec = OracleDecoder(OracleModel(cfg, w), cfg.seq)
    dec.prefill(ids, mask)
    batched = [dec.step(t).logits_f64 for t in steps]
    for b in range(3):
        L = int(mask[b].sum())
        alone = OracleDecoder(OracleModel(cfg, w), cfg.seq)
        alone.prefill(ids[b:b + 1, :L], np.ones((1, L), dtype=np.int32))
        for k, t in enumerate(steps):
            got = alone.step([t[b]]).logits_f64[0]
            np.testing.assert_allclose(got, batched[k][b], rtol=0, atol=1e-12)


def test_steps_equal_one_forward_over_the_final_sequence():
    cfg = tiny_lm().replace(batch=1)
    w = synth.make_weights(cfg, 22)
    ids, mask = synth.make_inputs(cfg, 5, seq=9, max_pad=0)
    toks, out = generate_greedy(OracleModel(cfg, w), ids, mask, steps=6, max_seq=cfg.seq)
    full = np.concatenate([ids[0], toks[:, 0]])[None].astype(np.int32)
    res = OracleModel(cfg, w).forward(full, np.ones_like(full))
    for k in range(6):
        np.testing.assert_allclose(out[k].logits_f64[0], res.logits_f64[0, 9 + k], rtol=0, atol=1e-12)
    # and the greedy chain follows the step logits
    for k in range(5):
        assert toks[k + 1, 0] == greedy(out[k].logits_f64[0])


def test_rotary_decisions_of_a_decode_loop():
    cfg = tiny_rotary().replace(batch=1)
    w = synth.make_weights(cfg, 23)
    ids, mask = synth.make_inputs(cfg, 6, seq=8, max_pad=0)
    orc = OracleModel(cfg, w)
    dec = OracleDecoder(orc, cfg.seq)
    dec.prefill(ids, mask)
    cached = cfg.rope_init_len
    for k in range(10):
        st = dec.step([k + 1])
        need = 8 + k + 1
        assert st.need == need
        assert st.regrow == (need > cached)
        cached = max(cached, need)
        assert st.cached_len == cached == orc.cached_len
        assert [(e.kind, e.value) for e in st.effects] == ([(EFFECT_REGROW, float(need))]
                                                           if need > 12 else [])


def test_decode_guards_and_state_after_a_trap():
    cfg = tiny_lm()
    w = synth.make_weights(cfg, 24)
    ids, mask = synth.make_inputs(cfg, 7, seq=30, max_pad=0)
    dec = OracleDecoder(OracleModel(cfg, w), 31)
    dec.prefill(ids, mask)
    with pytest.raises(Trap) as e:
        dec.step([1, cfg.vocab, -1])
    assert (e.value.code, e.value.index) == (TRAP_TOKEN_RANGE, 1)
    assert dec.lengths() == [30, 30, 30]
    dec.step([1, 2, 3])                      # position 30: the last one
    with pytest.raises(Trap) as e:
        dec.step([1, 2, 3])
    assert (e.value.code, e.value.index) == (TRAP_KV_CAPACITY, 0)
    assert dec.lengths() == [31, 31, 31]
    rot = tiny_rotary().replace(batch=1, seq=60)
    wr = synth.make_weights(rot, 25)
    ids, mask = synth.make_inputs(rot, 8, seq=rot.rope_capacity, max_pad=0)
    dr = OracleDecoder(OracleModel(rot, wr), 60)
    dr.prefill(ids, mask)
    with pytest.raises(Trap) as e:
        dr.step([3])
    assert (e.value.code, e.value.index) == (TRAP_ROPE_CAPACITY, 0)
