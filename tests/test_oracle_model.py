"""Pins for the composed oracle forward (CPU only).

The paper prints no model outputs, so the forward is pinned by
* an independent implementation built from PyTorch CPU functional
  operators (layer_norm, gelu, silu, scaled_dot_product_attention, linear),
* invariants that any correct forward satisfies: causality, masked keys
  have no influence, forcing a branch whose body is a no-op changes nothing,
  rotary-cache persistence, the clamp's fixed points,
* the rule semantics of the paper: guard order and codes ([Trap]), effect
  content and order ([Defer]), NaN never leaking through the clamp select
  ([Where], Semantics Preservation).
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import (EFFECT_CLAMP, EFFECT_PAD, EFFECT_REGROW, TRAP_MASK_VALUE,
                    TRAP_ROPE_CAPACITY, TRAP_TOKEN_RANGE, OracleModel, Trap)


def tiny_encoder():
    return synth.preset("encoder_1024", n_layers=2, d_model=64, n_heads=2,
                        d_ff=128, vocab=97, batch=3, seq=12, max_pad=5)


def tiny_rotary():
    return synth.preset("decoder_4096", n_layers=2, d_model=64, n_heads=2,
                        d_ff=128, vocab=101, batch=2, seq=20, rope_init_len=8,
                        rope_capacity=32)


def tiny_clamp():
    return synth.preset("encoder_clamp_1024", n_layers=3, d_model=64,
                        n_heads=4, d_ff=128, vocab=89, batch=2, seq=16,
                        outlier_scale=800.0)


def tiny_bf16_decoder():
    return synth.preset("causal_lm_768", n_layers=2, d_model=64, n_heads=2,
                        d_ff=256, vocab=120, batch=3, seq=24, max_pad=6)


def inputs_with_pads(cfg, want_pads, start=0):
    if not want_pads and cfg.batch > 1:
        return synth.make_inputs(cfg, start, max_pad=0)
    for seed in range(start, start + 200):
        ids, mask = synth.make_inputs(cfg, seed)
        if bool((mask == 0).any()) == want_pads:
            return ids, mask
    raise AssertionError("no seed found")


# ------------------------------------------------------------ independent forward

def _t_decode(a, dtype):
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).double()
    return torch.from_numpy(np.asarray(a)).double()


def rotate_complex(x, base):
    """Rotary embedding as a complex product: the pair (x_i, x_{i+hd/2}) is
    the complex number x_i + j x_{i+hd/2}, multiplied by exp(j p theta_i)."""
    S, hd = x.shape[-2], x.shape[-1]
    half = hd // 2
    theta = (base ** (-2.0 * torch.arange(half, dtype=torch.float64) / hd)).float().double()
    ang = torch.arange(S, dtype=torch.float64)[:, None] * theta[None, :]
    rot = torch.complex(torch.cos(ang).float().double(), torch.sin(ang).float().double())
    z = torch.complex(x[..., :half], x[..., half:]) * rot
    return torch.cat([z.real, z.imag], -1)


def clamp_guard(cfg, h, R):
    if cfg.fp16_clamp and bool(h.abs().max() > 65504.0 - cfg.clamp_margin):
        lim = 65504.0 - cfg.clamp_margin
        h = R(torch.clamp(h, -lim, lim))
    return h


def torch_forward(cfg, w, ids, mask):
    """The same program written with torch.nn.functional on float64 CPU
    tensors; storage rounding via torch dtype casts."""
    F = torch.nn.functional
    sdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[cfg.dtype]
    R = lambda t: t.to(sdt).double()
    G = {k: _t_decode(v, cfg.dtype) for k, v in w.globals.items()}
    B, S = ids.shape
    d, H = cfg.d_model, cfg.n_heads
    hd = d // H
    pad_any = bool((mask == 0).any())
    am = torch.ones(B, 1, S, S, dtype=torch.bool)
    if cfg.causal:
        am &= torch.ones(S, S, dtype=torch.bool).tril()
    if pad_any:
        am &= torch.from_numpy(mask == 1)[:, None, None, :]
    ids_t = torch.from_numpy(ids.astype(np.int64))
    x = F.embedding(ids_t, G["tok_emb"])
    if cfg.pos == "learned":
        x = x + G["pos_emb"][:S]
    h = R(x)

    def norm(t, g, b):
        if cfg.norm == "rmsnorm":
            return F.rms_norm(t, (d,), g, cfg.norm_eps)
        return F.layer_norm(t, (d,), g, b, cfg.norm_eps)

    if cfg.emb_norm:
        h = R(norm(h, G["emb_ln_g"], G.get("emb_ln_b")))
    for l in range(cfg.n_layers):
        W = {k: _t_decode(v, cfg.dtype) for k, v in w.layers[l].items()}
        a = R(norm(h, W["ln1_g"], W.get("ln1_b"))) if cfg.norm_place == "pre" else h
        qkv = F.linear(a, W["wqkv"], W.get("bqkv"))
        q, k, v = [t.reshape(B, S, H, hd).transpose(1, 2) for t in qkv.split(d, -1)]
        if cfg.pos == "rotary":
            q, k = rotate_complex(q, cfg.rope_base), rotate_complex(k, cfg.rope_base)
        q, k, v = R(q), R(k), R(v)
        ctx = F.scaled_dot_product_attention(q, k, v, attn_mask=am)
        ctx = R(ctx.transpose(1, 2).reshape(B, S, d))
        h = R(h + F.linear(ctx, W["wo"], W.get("bo")))
        if cfg.norm_place == "post":
            h = R(norm(h, W["ln1_g"], W.get("ln1_b")))
        h = clamp_guard(cfg, h, R)
        a = R(norm(h, W["ln2_g"], W.get("ln2_b"))) if cfg.norm_place == "pre" else h
        u = F.linear(a, W["w1"], W.get("b1"))
        if cfg.gated:
            g_, up = u.chunk(2, -1)
            f = R((F.gelu(g_) if cfg.ffn == "geglu" else F.silu(g_)) * up)
        else:
            f = R(F.gelu(u))
        h = R(h + F.linear(f, W["w2"], W.get("b2")))
        if cfg.norm_place == "post":
            h = R(norm(h, W["ln2_g"], W.get("ln2_b")))
        h = clamp_guard(cfg, h, R)
    z = R(norm(h, G["lnf_g"], G.get("lnf_b"))) if cfg.norm_place == "pre" else h
    head = G["tok_emb"] if cfg.tied_head else G["lm_head"]
    return R(F.linear(z, head)).numpy()


@pytest.mark.parametrize("want_pads", [False, True])
def test_tiny_decoder_matches_torch_functional(want_pads):
    cfg = synth.preset("tiny_decoder")
    w = synth.make_weights(cfg, 11)
    ids, mask = inputs_with_pads(cfg, want_pads)
    res = OracleModel(cfg, w).forward(ids, mask)
    assert res.pad_any == want_pads
    ref = torch_forward(cfg, w, ids, mask)
    scale = np.abs(ref).max()
    assert np.abs(res.logits_f64 - ref).max() <= 2e-6 * scale


@pytest.mark.parametrize("mk", [tiny_encoder, tiny_bf16_decoder, tiny_rotary, tiny_clamp])
def test_bf16_models_match_torch_functional(mk):
    cfg = mk()
    w = synth.make_weights(cfg, 5)
    ids, mask = inputs_with_pads(cfg, cfg.max_pad > 0)
    res = OracleModel(cfg, w).forward(ids, mask)
    ref = torch_forward(cfg, w, ids, mask)
    scale = np.abs(ref).max()
    # torch rounds float64 -> bf16 through float32 (double rounding), so a
    # few storage points may differ by one bf16 ulp.
    assert np.abs(res.logits_f64 - ref).max() <= 1e-2 * scale
    assert np.mean(res.logits_f64 == ref) > 0.9


# ------------------------------------------------------------ invariants

def test_causality_future_tokens_do_not_change_past_logits():
    cfg = synth.preset("tiny_decoder")
    w = synth.make_weights(cfg, 3)
    ids, mask = inputs_with_pads(cfg, False)
    a = OracleModel(cfg, w).forward(ids, mask).logits_f64
    ids2 = ids.copy()
    t = 9
    ids2[:, t + 1:] = (ids2[:, t + 1:] + 17) % cfg.vocab
    b = OracleModel(cfg, w).forward(ids2, mask).logits_f64
    np.testing.assert_array_equal(a[:, :t + 1], b[:, :t + 1])
    assert not np.array_equal(a[:, t + 1:], b[:, t + 1:])


@pytest.mark.parametrize("mk", [tiny_encoder, tiny_bf16_decoder])
def test_masked_positions_have_no_influence(mk):
    cfg = mk()
    w = synth.make_weights(cfg, 7)
    ids, mask = inputs_with_pads(cfg, True)
    real = mask == 1
    ids2 = np.where(real, ids, (ids + 31) % cfg.vocab).astype(np.int32)
    a = OracleModel(cfg, w).forward(ids, mask)
    b = OracleModel(cfg, w).forward(ids2, mask)
    assert a.pad_any and b.pad_any
    np.testing.assert_array_equal(a.logits_f64[real], b.logits_f64[real])
    if not cfg.causal:
        # the branch matters: without the key mask the pads leak in
        c = OracleModel(cfg, w).forward(ids2, mask, force={"pad_any": False})
        assert not np.array_equal(a.logits_f64[real], c.logits_f64[real])


@pytest.mark.parametrize("mk", [tiny_encoder, tiny_bf16_decoder,
                                lambda: synth.preset("tiny_decoder")])
def test_forcing_pad_branch_without_pads_is_bit_identical(mk):
    cfg = mk()
    w = synth.make_weights(cfg, 9)
    ids, mask = inputs_with_pads(cfg, False)
    a = OracleModel(cfg, w).forward(ids, mask)
    b = OracleModel(cfg, w).forward(ids, mask, force={"pad_any": True})
    assert not a.pad_any and b.pad_any
    np.testing.assert_array_equal(a.logits, b.logits)


def test_decoder_trailing_pads_hidden_by_causality():
    cfg = tiny_bf16_decoder()
    w = synth.make_weights(cfg, 4)
    ids, mask = inputs_with_pads(cfg, True)
    a = OracleModel(cfg, w).forward(ids, mask)
    b = OracleModel(cfg, w).forward(ids, mask, force={"pad_any": False})
    real = mask == 1
    np.testing.assert_array_equal(a.logits[real], b.logits[real])


def test_row_subset_matches_full_batch():
    cfg = tiny_bf16_decoder()
    w = synth.make_weights(cfg, 4)
    ids, mask = inputs_with_pads(cfg, True)
    full = OracleModel(cfg, w).forward(ids, mask)
    part = OracleModel(cfg, w).forward(ids, mask, rows=[2, 0])
    np.testing.assert_allclose(part.logits_f64, full.logits_f64[[2, 0]], rtol=0,
                               atol=1e-12 * np.abs(full.logits_f64).max())
    assert part.pad_any == full.pad_any


def test_causal_prefix_matches_full_forward():
    for cfg in (tiny_bf16_decoder(), tiny_rotary()):
        w = synth.make_weights(cfg, 4)
        ids, mask = inputs_with_pads(cfg, cfg.max_pad > 0)
        full = OracleModel(cfg, w).forward(ids, mask)
        part = OracleModel(cfg, w).forward(ids, mask, rows=[1], prefix=9)
        assert part.pad_any == full.pad_any and part.regrow == full.regrow
        assert part.cached_len == full.cached_len
        np.testing.assert_allclose(part.logits_f64, full.logits_f64[[1], :9], rtol=0,
                                   atol=1e-12 * np.abs(full.logits_f64).max())
    with pytest.raises(ValueError):
        OracleModel(tiny_encoder(), synth.make_weights(tiny_encoder(), 1)).forward(
            *synth.make_inputs(tiny_encoder(), 0), prefix=4)


# ------------------------------------------------------------ rotary cache

def test_rotary_regrow_decisions_persist_across_calls():
    cfg = tiny_rotary()
    m = OracleModel(cfg, synth.make_weights(cfg, 2))
    ids, mask = synth.make_inputs(cfg, 0)
    assert m.cached_len == 8
    r = [m.forward(ids, mask) for _ in range(3)]
    assert [x.regrow for x in r] == [True, False, False]
    assert [x.cached_len for x in r] == [20, 20, 20]
    np.testing.assert_array_equal(r[0].logits, r[1].logits)
    # regrown table equals a freshly built table of the same length
    fresh = OracleModel(cfg.replace(rope_init_len=20), synth.make_weights(cfg, 2))
    np.testing.assert_array_equal(fresh.rope_cos, m.rope_cos)
    np.testing.assert_array_equal(fresh.rope_sin, m.rope_sin)
    f = fresh.forward(ids, mask)
    assert not f.regrow
    np.testing.assert_array_equal(f.logits, r[0].logits)
    assert [e.kind for e in r[0].effects] == [EFFECT_REGROW]
    assert r[0].effects[0].value == 20.0 and r[1].effects == []


def test_rotary_forced_no_regrow_reads_past_cache():
    cfg = tiny_rotary()
    m = OracleModel(cfg, synth.make_weights(cfg, 2))
    ids, mask = synth.make_inputs(cfg, 0)
    with pytest.raises(IndexError):
        m.forward(ids, mask, force={"regrow": False})


def test_rotary_shorter_sequence_does_not_regrow():
    cfg = tiny_rotary()
    m = OracleModel(cfg, synth.make_weights(cfg, 2))
    ids, mask = synth.make_inputs(cfg, 0, seq=6)
    r = m.forward(ids, mask)
    assert not r.regrow and r.cached_len == 8 and r.need == 6


def test_rotary_position_zero_token_only_sees_itself():
    # with S = 1 attention returns v; rotary at position 0 is the identity,
    # so the result equals the same model without rotary.
    cfg = tiny_rotary()
    w = synth.make_weights(cfg, 2)
    ids, mask = synth.make_inputs(cfg, 0, seq=1)
    a = OracleModel(cfg, w).forward(ids, mask)
    b = OracleModel(cfg.replace(pos="none"), w).forward(ids, mask)
    np.testing.assert_array_equal(a.logits, b.logits)


# ------------------------------------------------------------ fp16 clamp

def test_clamp_trips_and_clamps_to_fp16_limit():
    cfg = tiny_clamp()
    w = synth.make_weights(cfg, 1)
    ids, mask = synth.make_inputs(cfg, 0)
    r = OracleModel(cfg, w).forward(ids, mask)
    flat = [t for pair in r.clamp for t in pair]
    assert any(flat) and not all(flat)
    kinds = [(e.kind, e.layer, e.site) for e in r.effects]
    assert kinds == [(EFFECT_CLAMP, l, s) for l in range(cfg.n_layers)
                     for s in range(2) if r.clamp[l][s]]
    for e in r.effects:
        assert e.value > 64504.0


def test_clamp_forced_below_threshold_is_bit_identical():
    cfg = tiny_clamp()
    w = synth.make_weights(cfg, 1)
    ids, mask = synth.make_inputs(cfg, 0)
    a = OracleModel(cfg, w).forward(ids, mask)
    quiet = [(l, s) for l in range(cfg.n_layers) for s in range(2) if not a.clamp[l][s]]
    assert quiet
    force = {"clamp": {quiet[0]: True}}
    b = OracleModel(cfg, w).forward(ids, mask, force=force)
    np.testing.assert_array_equal(a.logits, b.logits)


def test_clamp_values_saturate_at_64512():
    cfg = tiny_clamp().replace(n_layers=1)
    w = synth.make_weights(cfg, 1)
    ids, mask = synth.make_inputs(cfg, 0)
    m = OracleModel(cfg, w)
    # run the first layer by hand through the forward's clamp site
    h = np.array([[[-np.inf, 70000.0, 64496.0, 64495.0, 1.0, -64512.0]]])
    h = m.R(h)
    out, info = m._clamp_site(h, h, 0, 0, {}, 0, [])
    np.testing.assert_array_equal(out[0, 0], [-64512, 64512, 64512, 64480, 1, -64512])
    assert info[0] is True


def test_clamp_nan_anywhere_disables_clamp():
    cfg = tiny_clamp().replace(n_layers=1)
    m = OracleModel(cfg, synth.make_weights(cfg, 1))
    h = m.R(np.array([[[np.inf, np.nan, 3.0]]]))
    out, info = m._clamp_site(h, h, 0, 0, {}, 0, [])
    assert info[0] is False and info[2] is True
    assert np.isinf(out[0, 0, 0])          # inf survives: the branch is not taken


# ------------------------------------------------------------ traps and effects

def test_trap_codes_indices_and_order():
    cfg = synth.preset("tiny_decoder")
    m = OracleModel(cfg, synth.make_weights(cfg, 1))
    ids, mask = synth.make_inputs(cfg, 0)
    bad = ids.copy()
    bad[0, 5] = cfg.vocab
    bad[0, 9] = -1
    with pytest.raises(Trap) as e:
        m.forward(bad, mask)
    assert (e.value.code, e.value.index) == (TRAP_TOKEN_RANGE, 5)
    badm = mask.copy()
    badm[0, 3] = 2
    with pytest.raises(Trap) as e:
        m.forward(ids, badm)
    assert (e.value.code, e.value.index) == (TRAP_MASK_VALUE, 3)
    # ids are checked before the mask
    with pytest.raises(Trap) as e:
        m.forward(bad, badm)
    assert e.value.code == TRAP_TOKEN_RANGE
    cfg = tiny_rotary()
    m = OracleModel(cfg, synth.make_weights(cfg, 1))
    ids, mask = synth.make_inputs(cfg, 0, seq=40)
    with pytest.raises(Trap) as e:
        m.forward(ids, mask)
    assert (e.value.code, e.value.index) == (TRAP_ROPE_CAPACITY, 0)
    assert m.cached_len == 8


def test_pad_effect_content_and_forward_numbering():
    cfg = synth.preset("tiny_decoder")
    m = OracleModel(cfg, synth.make_weights(cfg, 1))
    ids, mask = inputs_with_pads(cfg, True)
    ids0, mask0 = inputs_with_pads(cfg, False)
    r1 = m.forward(ids, mask)
    r2 = m.forward(ids0, mask0)
    r3 = m.forward(ids, mask)
    assert [(e.forward, e.kind, e.value) for e in r1.effects] == \
        [(0, EFFECT_PAD, float((mask == 0).sum()))]
    assert r2.effects == []
    assert r3.effects[0].forward == 2
