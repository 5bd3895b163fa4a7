"""GPU parity: libgm (through the C ABI) against the CPU oracle.

Logits: max |gpu - oracle| / max |oracle| <= 1e-4 (fp32) or 2e-2 (bf16, fp16).
Decisions (padding branch, rotary regrow, every clamp site), the rotary
state, trap codes/positions and the deferred effect records must match
exactly.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import (TRAP_MASK_VALUE, TRAP_ROPE_CAPACITY, TRAP_TOKEN_RANGE,
                    OracleModel, Trap)

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2, "f16": 2e-2}


def gpu_model(cfg, w, **kw):
    from paper_2509_16248_amd.model import GmModel
    return GmModel(cfg, w.globals, w.layers, **kw)


def run(model, ids, mask):
    ids_t = torch.from_numpy(np.ascontiguousarray(ids)).cuda()
    mask_t = torch.from_numpy(np.ascontiguousarray(mask)).cuda()
    out = model.new_logits(*ids.shape)
    model.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    return out


def f64(t):
    return t.float().cpu().double().numpy()


def check_logits(got, ref, dtype, what="", tol=None):
    tol = TOL[dtype] if tol is None else tol
    scale = np.abs(ref).max()
    diff = np.abs(got - ref)
    err = diff.max() / scale
    print(f"{what} max_abs_diff={diff.max():.4g} max|oracle|={scale:.4g} rel={err:.3g} tol={tol}",
          flush=True)
    assert np.isfinite(got).all() == np.isfinite(ref).all()
    assert err <= tol, f"{what}: relative error {err:.3g} > {tol}"


def effects_of(res):
    return [(e.forward, e.kind, e.layer, e.site, np.float32(e.value)) for e in res.effects]


def gpu_effects(model, with_values=False):
    """Deferred effects as (forward, kind, layer, site, value) tuples; with
    ``with_values`` a sixth entry holds a log record's tensor values."""
    recs, dropped = model.flush_effects()
    assert dropped == 0
    if with_values:
        return [(r[0], r[1], r[2], r[3], np.float32(r[4]), r[5] if len(r) > 5 else None)
                for r in recs]
    return [(r[0], r[1], r[2], r[3], np.float32(r[4])) for r in recs]


def check_decisions(dec, res, cfg):
    assert dec["pad_any"] == res.pad_any
    assert dec["regrow"] == res.regrow
    if cfg.pos == "rotary":
        assert dec["cached_len"] == res.cached_len
        assert dec["need"] == res.need
    if cfg.fp16_clamp:
        flat = [t for pair in res.clamp for t in pair]
        assert dec["clamp"] == flat
        am = [np.float32(v) for pair in res.clamp_absmax for v in pair]
        print("clamp sites", flat, "absmax gpu", dec["clamp_absmax"], "oracle", am)
        # the NaN flag exactly; the largest magnitude of each site's stored
        # stream within the logits tolerance (the two forwards' streams differ
        # by rounding; test_gpu_stepwise compares it exactly on one stream)
        assert dec["clamp_nan"] == [bool(v) for pair in res.clamp_nan for v in pair]
        for g, o in zip(dec["clamp_absmax"], am):
            assert (np.isinf(g) and np.isinf(o)) or abs(g - o) <= TOL[cfg.dtype] * max(abs(o), 1.0)


def inputs(cfg, seed, want_pads):
    if not want_pads:
        return synth.make_inputs(cfg, seed, max_pad=0)
    for s in range(seed, seed + 100):
        ids, mask = synth.make_inputs(cfg, s)
        if (mask == 0).any():
            return ids, mask
    raise AssertionError


# ------------------------------------------------------------ tiny fp32 decoder

@pytest.mark.parametrize("seed", list(range(10)))
def test_tiny_decoder_parity_both_pad_outcomes(seed):
    cfg = synth.preset("tiny_decoder")
    w = synth.make_weights(cfg, 100 + seed)
    ids, mask = synth.make_inputs(cfg, seed)
    res = OracleModel(cfg, w).forward(ids, mask)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    print(f"seed {seed} pads {(mask == 0).sum()}")
    check_logits(f64(out), res.logits_f64, cfg.dtype, f"tiny seed {seed}")
    check_decisions(m.decisions(), res, cfg)
    assert gpu_effects(m) == effects_of(res)
    assert m.check_error() == (0, 0)


def test_tiny_decoder_seeds_cover_both_branch_outcomes():
    cfg = synth.preset("tiny_decoder")
    outcomes = {bool((synth.make_inputs(cfg, s)[1] == 0).any()) for s in range(10)}
    assert outcomes == {True, False}


# ------------------------------------------------------------ reduced shapes

REDUCED = ["causal_lm_768", "encoder_1024", "encoder_clamp_1024", "decoder_4096"]


@pytest.mark.parametrize("name", REDUCED)
def test_reduced_parity(name):
    cfg = synth.reduced(name)
    w = synth.make_weights(cfg, 7)
    for seed in range(5):
        ids, mask = inputs(cfg, seed, cfg.max_pad > 0)
        res = OracleModel(cfg, w).forward(ids, mask)
        margins = [x for pair in res.clamp_margin for x in pair]
        if not margins or min(margins) > 1.0:
            break
        print(f"seed {seed}: clamp decision within 1.0 of its boundary, next seed")
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    check_logits(f64(out), res.logits_f64, cfg.dtype, name)
    check_decisions(m.decisions(), res, cfg)
    assert gpu_effects(m) == effects_of(res)


@pytest.mark.parametrize("name", ["causal_lm_768", "encoder_1024"])
def test_reduced_parity_without_padding(name):
    cfg = synth.reduced(name)
    w = synth.make_weights(cfg, 8)
    ids, mask = inputs(cfg, 3, False)
    res = OracleModel(cfg, w).forward(ids, mask)
    assert not res.pad_any
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    check_logits(f64(out), res.logits_f64, cfg.dtype, name)
    check_decisions(m.decisions(), res, cfg)
    assert gpu_effects(m) == []


@pytest.mark.parametrize("name", ["causal_lm_768", "encoder_1024", "decoder_4096"])
def test_smaller_batch_and_ragged_lengths_in_one_model(name):
    """gm_forward_ex on shapes below the configured maximum: ragged tiles,
    a single token, and back to the full shape, all on one model."""
    cfg = synth.reduced(name)
    w = synth.make_weights(cfg, 12)
    orc = OracleModel(cfg, w)
    m = gpu_model(cfg, w)
    expect = []
    for B, S in [(2, 77), (1, 1), (cfg.batch, cfg.seq), (1, 129)]:
        B = min(B, cfg.batch)
        ids, mask = synth.make_inputs(cfg, B * 1000 + S, batch=B, seq=S,
                                      max_pad=min(cfg.max_pad, max(S - 1, 0)))
        res = orc.forward(ids, mask)
        out = run(m, ids, mask)
        print(f"{name} B={B} S={S}", flush=True)
        check_logits(f64(out), res.logits_f64, cfg.dtype, f"{name} {B}x{S}")
        check_decisions(m.decisions(), res, cfg)
        expect += effects_of(res)
    assert gpu_effects(m) == expect


def test_rotary_regrow_state_persists_across_forwards():
    cfg = synth.reduced("decoder_4096")
    w = synth.make_weights(cfg, 9)
    orc = OracleModel(cfg, w)
    m = gpu_model(cfg, w)
    short_ids, short_mask = synth.make_inputs(cfg, 1, seq=100)
    ids, mask = synth.make_inputs(cfg, 2)
    seq = [(short_ids, short_mask), (ids, mask), (ids, mask), (short_ids, short_mask)]
    for k, (i, mk) in enumerate(seq):
        res = orc.forward(i, mk)
        out = run(m, i, mk)
        dec = m.decisions()
        print(f"call {k}: S={i.shape[1]} regrow gpu {dec['regrow']} oracle {res.regrow} "
              f"cached {dec['cached_len']}/{res.cached_len}")
        check_decisions(dec, res, cfg)
        check_logits(f64(out), res.logits_f64, cfg.dtype, f"rotary call {k}")
    assert [e[1] for e in gpu_effects(m)] == [2]


# ------------------------------------------------------------ traps

def test_traps_reported_at_next_sync_and_model_recovers():
    cfg = synth.preset("tiny_decoder")
    w = synth.make_weights(cfg, 3)
    ids, mask = synth.make_inputs(cfg, 0)
    m = gpu_model(cfg, w)
    orc = OracleModel(cfg, w)
    bad = ids.copy()
    bad[0, 5] = cfg.vocab
    bad[0, 9] = -1
    badm = mask.copy()
    badm[0, 3] = 2
    for i, mk, code, index in [(bad, mask, TRAP_TOKEN_RANGE, 5),
                               (ids, badm, TRAP_MASK_VALUE, 3),
                               (bad, badm, TRAP_TOKEN_RANGE, 5)]:
        with pytest.raises(Trap) as e:
            orc.forward(i, mk)
        assert (e.value.code, e.value.index) == (code, index)
        run(m, i, mk)
        assert m.check_error() == (code, index)
        assert m.check_error() == (0, 0)
    # a trapped forward records no effects; a good forward still matches
    assert gpu_effects(m) == []
    res = orc.forward(ids, mask)
    out = run(m, ids, mask)
    check_logits(f64(out), res.logits_f64, cfg.dtype, "after traps")
    assert gpu_effects(m) == effects_of(res)


def test_trap_rotary_capacity_leaves_cache_untouched():
    cfg = synth.reduced("decoder_4096").replace(seq=600)
    w = synth.make_weights(cfg, 4)
    orc = OracleModel(cfg, w)
    m = gpu_model(cfg, w)
    ids, mask = synth.make_inputs(cfg, 0)
    with pytest.raises(Trap) as e:
        orc.forward(ids, mask)
    assert e.value.code == TRAP_ROPE_CAPACITY
    run(m, ids, mask)
    assert m.check_error() == (TRAP_ROPE_CAPACITY, 0)
    assert m.decisions()["cached_len"] == orc.cached_len == cfg.rope_init_len
    ids2, mask2 = synth.make_inputs(cfg, 1, seq=300)
    res = orc.forward(ids2, mask2)
    out = run(m, ids2, mask2)
    check_decisions(m.decisions(), res, cfg)
    check_logits(f64(out), res.logits_f64, cfg.dtype, "after capacity trap")


# ------------------------------------------------------------ graph / syncs

def test_graph_replay_is_deterministic_and_sync_free():
    cfg = synth.reduced("causal_lm_768")
    w = synth.make_weights(cfg, 5)
    ids, mask = inputs(cfg, 0, True)
    m = gpu_model(cfg, w)
    ids_t = torch.from_numpy(ids).cuda()
    mask_t = torch.from_numpy(mask).cuda()
    out = m.new_logits(*ids.shape)
    m.set_graph_mode(False)
    m.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    eager = out.clone()
    m.set_graph_mode(True)
    outs = []
    for _ in range(4):
        m.forward(ids_t, mask_t, out)
        torch.cuda.synchronize()
        outs.append(out.clone())
    for o in outs:
        assert torch.equal(o.view(torch.int16), eager.view(torch.int16))
    st = m.stats()
    print(st)
    assert st["captures"] == 1 and st["graph_launches"] == 4
    assert st["host_syncs_in_forward"] == 0
    assert st["kernels_per_forward"] > 0


def test_effect_fifo_keeps_forward_order():
    cfg = synth.preset("tiny_decoder")
    w = synth.make_weights(cfg, 6)
    orc = OracleModel(cfg, w)
    m = gpu_model(cfg, w)
    expect = []
    for s in range(6):
        ids, mask = synth.make_inputs(cfg, s)
        expect += effects_of(orc.forward(ids, mask))
        run(m, ids, mask)
    assert gpu_effects(m) == expect


# ------------------------------------------------------------ bench shape

def test_full_size_causal_lm_768_sampled_sequences():
    """The benchmarked workload at full size (12 layers, d=768, vocab 50257,
    batch 8 x 512, bf16), in the same graph launch the benchmark times; the
    oracle recomputes two whole sequences (the padding predicate is taken
    over the whole batch)."""
    cfg = synth.preset("causal_lm_768")
    w = synth.make_weights(cfg, 1234)
    ids, mask = synth.make_inputs(cfg, 0)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    rows = [0, 5]
    res = OracleModel(cfg, w).forward(ids, mask, rows=rows)
    check_logits(f64(out[rows]), res.logits_f64, cfg.dtype, "causal_lm_768 rows 0,5")
    check_decisions(m.decisions(), res, cfg)


def test_attention_workgroup_orders_give_the_same_bits(monkeypatch):
    """The attention kernel's workgroup order (the 3-D grid, or the
    one-dimensional query-block-major order with or without every other run
    of 256 workgroups reversed) only moves (query block, sequence, head)
    items between workgroups, so the logits are the same bits.  8 x 512
    causal with 12 heads in one batch part gives 768 workgroups per launch:
    three runs of 256, the middle one reversed."""
    cfg = synth.preset("causal_lm_768", n_layers=2, vocab=1000)
    w = synth.make_weights(cfg, 61)
    ids, mask = synth.make_inputs(cfg, 9)
    monkeypatch.setenv("GM_SPLIT_PARTS", "1")
    outs = []
    for order in (0, 1, 2):        # 2, the default, last: the setting is process-wide
        monkeypatch.setenv("GM_ATTN_ORDER", str(order))
        outs.append(run(gpu_model(cfg, w), ids, mask))
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))
    res = OracleModel(cfg, w).forward(ids, mask, rows=[3])
    check_logits(f64(outs[2][[3]]), res.logits_f64, cfg.dtype, "row 3")
