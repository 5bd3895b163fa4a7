"""Pins for the encoder-decoder oracle (CPU only).

* the whole forward against PyTorch's own pre-LN transformer modules
  (torch.nn.TransformerEncoderLayer / TransformerDecoderLayer with
  norm_first, exact GELU, float64, key-padding and causal masks) loaded with
  the same weights: an implementation written by others, so a dropped
  residual, a transposed projection, a swapped k/v half or a cross-attention
  reading the wrong stream fails it;
* causality of the decoder: changing target token t changes no logits at
  positions before t;
* source padding: tokens under the source mask change nothing when the
  branch is taken, and every logit when it is forced off;
* a sequence inside a padded batch equals the same sequence alone, trimmed
  to its real lengths (no padding, both branches untaken);
* guard codes and concatenated indices, the two PAD records and the
  forward counter.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import EFFECT_PAD, TRAP_MASK_VALUE, TRAP_TOKEN_RANGE, OracleSeq2Seq, Trap
from oracle import numerics as nx


def tiny(**kw):
    base = synth.preset("seq2seq_768", n_layers=2, n_dec_layers=2, d_model=64, n_heads=4,
                        d_ff=128, vocab=97, batch=3, seq=20, tgt_seq=12, dtype="f32",
                        max_pad=8, tgt_max_pad=5)
    return base.replace(**kw)


def inputs(cfg, seed):
    src = synth.make_inputs(cfg, seed)
    tgt = synth.make_target_inputs(cfg, seed)
    return src + tgt


def torch_reference(cfg, w, src_ids, src_mask, tgt_ids, tgt_mask):
    """The same model assembled from torch.nn transformer layers (float64)."""
    d, H, ff = cfg.d_model, cfg.n_heads, cfg.d_ff
    dt = torch.float64
    T = lambda a: torch.from_numpy(nx.decode(a, cfg.dtype))

    def load_common(layer, W):
        layer.self_attn.in_proj_weight.data.copy_(T(W["wqkv"]))
        layer.self_attn.in_proj_bias.data.copy_(T(W["bqkv"]))
        layer.self_attn.out_proj.weight.data.copy_(T(W["wo"]))
        layer.self_attn.out_proj.bias.data.copy_(T(W["bo"]))
        layer.linear1.weight.data.copy_(T(W["w1"]))
        layer.linear1.bias.data.copy_(T(W["b1"]))
        layer.linear2.weight.data.copy_(T(W["w2"]))
        layer.linear2.bias.data.copy_(T(W["b2"]))
        layer.norm1.weight.data.copy_(T(W["ln1_g"]))
        layer.norm1.bias.data.copy_(T(W["ln1_b"]))

    kw = dict(d_model=d, nhead=H, dim_feedforward=ff, dropout=0.0, activation="gelu",
              layer_norm_eps=cfg.norm_eps, batch_first=True, norm_first=True, dtype=dt)
    enc = []
    for W in w.layers:
        L = torch.nn.TransformerEncoderLayer(**kw)
        load_common(L, W)
        L.norm2.weight.data.copy_(T(W["ln2_g"]))
        L.norm2.bias.data.copy_(T(W["ln2_b"]))
        enc.append(L.eval())
    dec = []
    for W in w.dec_layers:
        L = torch.nn.TransformerDecoderLayer(**kw)
        load_common(L, W)
        # norm2 precedes the cross-attention, norm3 the feed-forward
        L.norm2.weight.data.copy_(T(W["x_lnc_g"]))
        L.norm2.bias.data.copy_(T(W["x_lnc_b"]))
        L.norm3.weight.data.copy_(T(W["ln2_g"]))
        L.norm3.bias.data.copy_(T(W["ln2_b"]))
        xa = L.multihead_attn
        xa.in_proj_weight.data.copy_(torch.cat([T(W["x_wq"]), T(W["x_wkv"])]))
        xa.in_proj_bias.data.copy_(torch.cat([T(W["x_bq"]), T(W["x_bkv"])]))
        xa.out_proj.weight.data.copy_(T(W["x_wo"]))
        xa.out_proj.bias.data.copy_(T(W["x_bo"]))
        dec.append(L.eval())
    G = {k: T(v) for k, v in w.globals.items()}
    Ss, St = src_ids.shape[1], tgt_ids.shape[1]
    src_pad = torch.from_numpy(src_mask == 0)
    tgt_pad = torch.from_numpy(tgt_mask == 0)
    causal = torch.triu(torch.ones(St, St, dtype=torch.bool), diagonal=1)
    # grad enabled with trainable parameters keeps the modules on their
    # ordinary (non-fused) path
    x = G["tok_emb"][torch.from_numpy(src_ids).long()] + G["enc_pos_emb"][:Ss]
    for L in enc:
        x = L(x, src_key_padding_mask=src_pad)
    mem = torch.nn.functional.layer_norm(x, (d,), G["enc_lnf_g"], G["enc_lnf_b"], cfg.norm_eps)
    y = G["tok_emb"][torch.from_numpy(tgt_ids).long()] + G["pos_emb"][:St]
    for L in dec:
        y = L(y, mem, tgt_mask=causal, tgt_key_padding_mask=tgt_pad,
              memory_key_padding_mask=src_pad)
    z = torch.nn.functional.layer_norm(y, (d,), G["lnf_g"], G["lnf_b"], cfg.norm_eps)
    return (z @ G["tok_emb"].T).detach().numpy()


@pytest.mark.parametrize("pads", [True, False])
def test_matches_torch_transformer_modules(pads):
    cfg = tiny() if pads else tiny(max_pad=0, tgt_max_pad=0)
    w = synth.make_weights(cfg, 51)
    si, sm, ti, tm = inputs(cfg, 1)
    assert (sm == 0).any() == pads and (tm == 0).any() == pads
    res = OracleSeq2Seq(cfg, w).forward(si, sm, ti, tm)
    ref = torch_reference(cfg, w, si, sm, ti, tm)
    scale = np.abs(ref).max()
    assert np.abs(res.logits_f64 - ref).max() <= 2e-6 * scale
    assert (res.pad_any_src, res.pad_any_tgt) == (pads, pads)


def test_bf16_matches_torch_transformer_modules():
    cfg = tiny(dtype="bf16")
    w = synth.make_weights(cfg, 52)
    si, sm, ti, tm = inputs(cfg, 2)
    res = OracleSeq2Seq(cfg, w).forward(si, sm, ti, tm)
    ref = torch_reference(cfg, w, si, sm, ti, tm)
    assert np.abs(res.logits_f64 - ref).max() <= 2e-2 * np.abs(ref).max()


def test_decoder_is_causal_and_source_padding_is_invisible():
    cfg = tiny()
    w = synth.make_weights(cfg, 53)
    si, sm, ti, tm = inputs(cfg, 3)
    orc = OracleSeq2Seq(cfg, w)
    a = orc.forward(si, sm, ti, tm).logits_f64
    t = 7
    ti2 = ti.copy()
    ti2[:, t] = (ti2[:, t] + 1) % cfg.vocab
    b = orc.forward(si, sm, ti2, tm).logits_f64
    np.testing.assert_array_equal(a[:, :t], b[:, :t])
    assert not np.allclose(a[:, t], b[:, t])
    # tokens under the source mask: invisible with the branch taken
    b0 = int(np.argmin(sm.sum(1)))
    assert sm[b0, -1] == 0
    si2 = si.copy()
    si2[sm == 0] = (si2[sm == 0] + 5) % cfg.vocab
    np.testing.assert_array_equal(orc.forward(si2, sm, ti, tm).logits_f64, a)
    f1 = orc.forward(si, sm, ti, tm, force={"pad_any_src": False}).logits_f64
    f2 = orc.forward(si2, sm, ti, tm, force={"pad_any_src": False}).logits_f64
    assert not np.allclose(f1[b0], f2[b0])


def test_sequence_in_padded_batch_equals_sequence_alone():
    cfg = tiny()
    w = synth.make_weights(cfg, 54)
    si, sm, ti, tm = inputs(cfg, 4)
    sm[0, 15:] = 0
    tm[1, 9:] = 0
    full = OracleSeq2Seq(cfg, w).forward(si, sm, ti, tm).logits_f64
    for b in range(cfg.batch):
        Ls, Lt = int(sm[b].sum()), int(tm[b].sum())
        one = OracleSeq2Seq(cfg, w).forward(si[b:b + 1, :Ls], np.ones((1, Ls), np.int32),
                                            ti[b:b + 1, :Lt], np.ones((1, Lt), np.int32))
        assert not one.pad_any_src and not one.pad_any_tgt and not one.effects
        np.testing.assert_allclose(one.logits_f64[0], full[b, :Lt], rtol=0, atol=1e-12)


def test_guards_effects_and_forward_counter():
    cfg = tiny()
    w = synth.make_weights(cfg, 55)
    si, sm, ti, tm = inputs(cfg, 5)
    orc = OracleSeq2Seq(cfg, w)
    r = orc.forward(si, sm, ti, tm)
    assert [(e.forward, e.kind, e.site, e.value) for e in r.effects] == [
        (0, EFFECT_PAD, 0, float((sm == 0).sum())), (0, EFFECT_PAD, 1, float((tm == 0).sum()))]
    nsrc = si.size
    ti2 = ti.copy()
    ti2[2, 3] = -1
    sm2 = sm.copy()
    sm2[1, 0] = 2
    with pytest.raises(Trap) as e:            # token range beats mask value
        orc.forward(si, sm2, ti2, tm)
    assert (e.value.code, e.value.index) == (TRAP_TOKEN_RANGE, nsrc + 2 * cfg.tgt_seq + 3)
    with pytest.raises(Trap) as e:
        orc.forward(si, sm2, ti, tm)
    assert (e.value.code, e.value.index) == (TRAP_MASK_VALUE, cfg.seq)
    tm2 = tm.copy()
    tm2[0, 1] = 3
    with pytest.raises(Trap) as e:
        orc.forward(si, sm, ti, tm2)
    assert (e.value.code, e.value.index) == (TRAP_MASK_VALUE, nsrc + 1)
    sm3 = np.ones_like(sm)
    tm3 = np.ones_like(tm)
    r = orc.forward(si, sm3, ti, tm3)
    assert r.effects == [] and orc.forward_count == 5
    r = orc.forward(si, sm3, ti, tm)
    assert [(e.forward, e.site) for e in r.effects] == [(5, 1)]
