"""GPU parity of the encoder-decoder forward (gm_forward_seq2seq) against
the encoder-decoder oracle.

Logits to the forward's tolerance (1e-4 fp32, 2e-2 bf16, relative to
max |oracle|); the two padding decisions, the trap word and the deferred
PAD records exactly.  Graph replays with new input values must take the
new decisions (the predicates are device values, not captured constants).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import TRAP_MASK_VALUE, TRAP_TOKEN_RANGE, OracleSeq2Seq, Trap

from test_gpu_parity import check_logits, effects_of, f64, gpu_effects

pytestmark = pytest.mark.gpu


def s2s_model(cfg, w, **kw):
    from paper_2509_16248_amd.model import GmModel
    return GmModel(cfg, w.globals, w.layers, dec_layers=w.dec_layers, **kw)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def run_s2s(m, si, sm, ti, tm, out=None):
    if out is None:
        out = m.new_logits(*ti.shape)
    m.forward_seq2seq(dev(si), dev(sm), dev(ti), dev(tm), out)
    torch.cuda.synchronize()
    return out


def tiny_fp32(**kw):
    base = synth.preset("seq2seq_768", n_layers=2, n_dec_layers=2, d_model=64, n_heads=2,
                        d_ff=128, vocab=97, batch=3, seq=37, tgt_seq=19, dtype="f32",
                        max_pad=12, tgt_max_pad=6)
    return base.replace(**kw)


def case(cfg, w, si, sm, ti, tm, what, m=None, orc=None):
    orc = orc or OracleSeq2Seq(cfg, w)
    ref = orc.forward(si, sm, ti, tm)
    m = m or s2s_model(cfg, w)
    out = run_s2s(m, si, sm, ti, tm)
    check_logits(f64(out), ref.logits_f64, cfg.dtype, what)
    d = m.decisions()
    assert (d["pad_any"], d["pad_any_tgt"]) == (ref.pad_any_src, ref.pad_any_tgt)
    assert m.check_error() == (0, 0)
    return m, orc, ref


@pytest.mark.parametrize("pads", ["both", "none", "src", "tgt"])
def test_tiny_fp32_each_padding_outcome(pads):
    cfg = tiny_fp32()
    w = synth.make_weights(cfg, 61)
    si, sm = synth.make_inputs(cfg, 1, max_pad=cfg.max_pad if pads in ("both", "src") else 0)
    ti, tm = synth.make_target_inputs(cfg, 1, max_pad=cfg.tgt_max_pad if pads in ("both", "tgt") else 0)
    sm[0, -3:] = 0 if pads in ("both", "src") else 1
    tm[1, -2:] = 0 if pads in ("both", "tgt") else 1
    m, orc, ref = case(cfg, w, si, sm, ti, tm, f"tiny fp32 pads={pads}")
    assert gpu_effects(m) == effects_of(ref)


def test_reduced_bf16_graph_replays_take_new_decisions():
    """d 768 / 12 heads (MFMA attention path), 2 + 2 layers, ragged source and
    target; the same graph replayed with new values in the same buffers:
    pads, then no pads, then pads again."""
    cfg = synth.reduced("seq2seq_768")
    w = synth.make_weights(cfg, 62)
    orc = OracleSeq2Seq(cfg, w)
    m = s2s_model(cfg, w)
    m.set_exec_mode("graph")
    B, Ss, St = cfg.batch, cfg.seq, cfg.tgt_seq
    bufs = [torch.empty((B, n), dtype=torch.int32, device="cuda") for n in (Ss, Ss, St, St)]
    out = m.new_logits(B, St)
    expect = []
    s0 = m.stats()
    for k, (mp, tp) in enumerate([(cfg.max_pad, cfg.tgt_max_pad), (0, 0), (0, 5), (9, 0)]):
        si, sm = synth.make_inputs(cfg, 10 + k, max_pad=mp)
        ti, tm = synth.make_target_inputs(cfg, 10 + k, max_pad=tp)
        for b, a in zip(bufs, (si, sm, ti, tm)):
            b.copy_(dev(a))
        ref = orc.forward(si, sm, ti, tm)
        m.forward_seq2seq(*bufs, out)
        torch.cuda.synchronize()
        check_logits(f64(out), ref.logits_f64, cfg.dtype, f"reduced bf16 replay {k}")
        d = m.decisions()
        assert (d["pad_any"], d["pad_any_tgt"]) == (ref.pad_any_src, ref.pad_any_tgt)
        expect += effects_of(ref)
    s1 = m.stats()
    assert s1["captures"] - s0["captures"] == 1
    assert s1["graph_launches"] - s0["graph_launches"] == 4
    assert s1["host_syncs_in_forward"] == 0
    assert gpu_effects(m) == expect
    # eager gives the same bits as the graph
    e = s2s_model(cfg, w)
    e.set_exec_mode("eager")
    out_e = e.new_logits(B, St)
    e.forward_seq2seq(*bufs, out_e)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), out_e.view(torch.int16))


def test_traps_concatenated_positions_and_recovery():
    cfg = tiny_fp32()
    w = synth.make_weights(cfg, 63)
    si, sm = synth.make_inputs(cfg, 2)
    ti, tm = synth.make_target_inputs(cfg, 2)
    orc = OracleSeq2Seq(cfg, w)
    m = s2s_model(cfg, w)
    bad_ti = ti.copy()
    bad_ti[2, 4] = cfg.vocab
    bad_sm = sm.copy()
    bad_sm[1, 2] = 7
    bad_tm = tm.copy()
    bad_tm[0, 0] = -1
    for args in ((si, bad_sm, bad_ti, tm), (si, bad_sm, ti, tm), (si, sm, ti, bad_tm)):
        with pytest.raises(Trap) as e:
            orc.forward(*args)
        run_s2s(m, *args)
        got = m.check_error()
        print("trap", got, flush=True)
        assert got == (e.value.code, e.value.index)
    assert m.check_error() == (0, 0)
    # a good forward afterwards: right logits, effects numbered after the traps
    ref = orc.forward(si, sm, ti, tm)
    out = run_s2s(m, si, sm, ti, tm)
    check_logits(f64(out), ref.logits_f64, cfg.dtype, "after traps")
    assert gpu_effects(m) == effects_of(ref)
    assert ref.effects and ref.effects[0].forward == 3


def test_full_size_seq2seq_768_sampled():
    """The full encoder-decoder (6 + 6 layers, d 768, vocab 50265, bf16,
    8 sequences of 512 source / 128 target positions, ragged): the oracle
    computes two of the sequences, with both padding predicates read over
    the whole batch as the program does."""
    cfg = synth.preset("seq2seq_768")
    w = synth.make_weights(cfg, 4321)
    si, sm = synth.make_inputs(cfg, 12)
    ti, tm = synth.make_target_inputs(cfg, 12)
    print("source lengths", sm.sum(1).tolist(), "target lengths", tm.sum(1).tolist(), flush=True)
    m = s2s_model(cfg, w)
    out = run_s2s(m, si, sm, ti, tm)
    d = m.decisions()
    assert (d["pad_any"], d["pad_any_tgt"]) == (bool((sm == 0).any()), bool((tm == 0).any()))
    got = f64(out)
    orc = OracleSeq2Seq(cfg, w)
    force = {"pad_any_src": d["pad_any"], "pad_any_tgt": d["pad_any_tgt"]}
    for b in (0, 5):
        ref = orc.forward(si[b:b + 1], sm[b:b + 1], ti[b:b + 1], tm[b:b + 1], force=force)
        check_logits(got[b:b + 1], ref.logits_f64, cfg.dtype, f"seq2seq_768 full, sequence {b}")
    recs = gpu_effects(m)
    assert [(r[1], r[3], r[4]) for r in recs] == [
        (1, 0, np.float32((sm == 0).sum())), (1, 1, np.float32((tm == 0).sum()))]
    assert m.check_error() == (0, 0)


def test_fragmented_encoder_decoder_equals_single_graph():
    """The unmended encoder-decoder program: a graph break at each input's
    guards and mask.any() (before the encoder, before the decoder), so three
    graphs and two host synchronisations per forward, the same kernels and
    the same bits as the single graph."""
    cfg = synth.reduced("seq2seq_768")
    w = synth.make_weights(cfg, 64)
    si, sm = synth.make_inputs(cfg, 3)
    ti, tm = synth.make_target_inputs(cfg, 3)
    bufs = [dev(a) for a in (si, sm, ti, tm)]
    a = s2s_model(cfg, w)
    b = s2s_model(cfg, w)
    b.set_exec_mode("fragmented")
    out_a = a.new_logits(cfg.batch, cfg.tgt_seq)
    out_b = b.new_logits(cfg.batch, cfg.tgt_seq)
    for k in range(2):
        a.forward_seq2seq(*bufs, out_a)
        s0 = b.stats()
        b.forward_seq2seq(*bufs, out_b)
        torch.cuda.synchronize()
        s1 = b.stats()
        assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16)), f"call {k}"
        assert a.decisions() == b.decisions()
        assert s1["host_syncs_in_forward"] - s0["host_syncs_in_forward"] == 2
        assert s1["graph_launches"] - s0["graph_launches"] == 3
    assert gpu_effects(a) == gpu_effects(b)
    # a failed target guard stops the unmended program at that break
    bad = ti.copy()
    bad[1, 1] = -5
    bufs[2].copy_(dev(bad))
    from paper_2509_16248_amd.gm import GmError
    with pytest.raises(GmError):
        b.forward_seq2seq(*bufs, out_b)
    assert b.check_error() == (TRAP_TOKEN_RANGE, si.size + cfg.tgt_seq + 1)


def test_edge_cases_fully_padded_source_and_length_one():
    """A source sequence that is all padding (its cross-attention sees no
    key: the context is zero), source and target of length 1, one sequence."""
    cfg = tiny_fp32()
    w = synth.make_weights(cfg, 65)
    m = s2s_model(cfg, w)
    orc = OracleSeq2Seq(cfg, w)
    si, sm = synth.make_inputs(cfg, 6)
    ti, tm = synth.make_target_inputs(cfg, 6)
    sm[1, :] = 0
    ref = orc.forward(si, sm, ti, tm)
    check_logits(f64(run_s2s(m, si, sm, ti, tm)), ref.logits_f64, cfg.dtype, "all-pad source")
    expect = effects_of(ref)
    for B, Ss, St in ((3, 1, 1), (1, cfg.seq, 1), (1, 1, cfg.tgt_seq), (2, 5, 3)):
        ids_s, mk_s = si[:B, :Ss].copy(), np.ones((B, Ss), np.int32)
        ids_t, mk_t = ti[:B, :St].copy(), np.ones((B, St), np.int32)
        ref = orc.forward(ids_s, mk_s, ids_t, mk_t)
        got = f64(run_s2s(m, ids_s, mk_s, ids_t, mk_t))
        check_logits(got, ref.logits_f64, cfg.dtype, f"B {B} S_src {Ss} S_tgt {St}")
        expect += effects_of(ref)
    assert gpu_effects(m) == expect
    assert m.check_error() == (0, 0)
