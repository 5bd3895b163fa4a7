"""CPU oracle of the encoder-decoder forward (cross-attention stack).

Test infrastructure only (see the package docstring).

The paper's evaluation includes encoder-decoder text models (Evaluation
section, model list); their forward has the same graph-breaking pattern as
the encoder and decoder models, once per input: a padding branch
``if mask.any()`` on the source mask (it gates the key mask of the
encoder's self-attention and of every cross-attention) and one on the
target mask (it gates the key mask of the decoder's causal
self-attention).  As in :mod:`oracle.model`, the plain definition of the
mended forward is the original one with host-side branches:

* guards (rule [Trap]) run in code order, each over the source and then the
  target: token range (code 1), mask values (code 2); the reported position
  is the row-major index into the concatenation [source (B*S_src), target
  (B*S_tgt)];
* two PAD effect records (rule [Defer]), the source's with site 0 and the
  target's with site 1, each valued at the number of padded positions, in
  that order, each only when its branch is taken;
* pre-LN layers; encoder: ``h += SelfAttn(LN1 h)`` (bidirectional),
  ``h += FFN(LN2 h)``, then a final LayerNorm gives the memory; decoder:
  ``h += SelfAttn(LN1 h)`` (causal), ``h += CrossAttn(LNc h, memory)``,
  ``h += FFN(LN2 h)``, then the final LayerNorm and the tied head;
* learned positions (``enc_pos_emb`` for the source, ``pos_emb`` for the
  target), both from position 0;
* cross-attention: queries from the decoder stream, keys and values
  projected from the memory by the layer's own ``x_wkv`` (k rows, then v
  rows) and stored (rounded) like every k/v.

All arithmetic is float64 with the storage points of :mod:`oracle.model`.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np

from . import numerics as nx
from .model import EFFECT_PAD, TRAP_MASK_VALUE, TRAP_TOKEN_RANGE, Effect, Trap


class Seq2SeqResult:
    def __init__(self, logits_f64, logits, pad_any_src, pad_any_tgt, effects, memory_f64):
        self.logits_f64 = logits_f64      # [B, S_tgt, V]
        self.logits = logits              # storage dtype
        self.pad_any_src = pad_any_src
        self.pad_any_tgt = pad_any_tgt
        self.effects = effects
        self.memory_f64 = memory_f64      # encoder output after its final norm [B, S_src, d]


class OracleSeq2Seq:
    """Float64 reference of the encoder-decoder forward of one synthetic
    model (``cfg.n_layers`` encoder layers, ``cfg.n_dec_layers`` decoder
    layers).  ``forward_count`` counts forwards, trapped ones included."""

    def __init__(self, cfg, weights):
        if cfg.n_dec_layers < 1:
            raise ValueError("not an encoder-decoder configuration")
        if cfg.norm != "layernorm" or cfg.norm_place != "pre" or cfg.pos != "learned":
            raise ValueError("encoder-decoder: pre-LN with learned positions only")
        if cfg.fp16_clamp or cfg.log_hidden or cfg.gated or not cfg.tied_head or not cfg.bias:
            raise ValueError("encoder-decoder: plain GELU FFN, biases, tied head, no clamp or log")
        self.cfg = cfg
        self.w = weights
        self.dt = cfg.dtype
        self.forward_count = 0

    def R(self, x):
        return nx.round_to(x, self.dt)

    def _g(self, name):
        return nx.decode(self.w.globals[name], self.dt)

    def _ln(self, x, g, b):
        return self.R(nx.layer_norm(x, g, b, self.cfg.norm_eps))

    def _attend(self, q_in, kv_rows, Wq, bq, Wk, bk, Wv, bv, allowed):
        """Multi-head attention of the rows ``q_in`` [B, Sq, d] over
        ``kv_rows`` [B, Sk, d]: projections, storage rounding of q/k/v,
        scaled scores, softmax over the allowed keys, context rounding."""
        c = self.cfg
        B, Sq, d = q_in.shape
        Sk = kv_rows.shape[1]
        H, hd = c.n_heads, c.head_dim
        q = self.R(q_in @ Wq.T + bq).reshape(B, Sq, H, hd).transpose(0, 2, 1, 3)
        k = self.R(kv_rows @ Wk.T + bk).reshape(B, Sk, H, hd).transpose(0, 2, 1, 3)
        v = self.R(kv_rows @ Wv.T + bv).reshape(B, Sk, H, hd).transpose(0, 2, 1, 3)
        s = (q @ k.transpose(0, 1, 3, 2)) * (1.0 / np.sqrt(hd))
        p = nx.masked_softmax(s, allowed)
        return self.R(p @ v).transpose(0, 2, 1, 3).reshape(B, Sq, d)

    def _ffn(self, h, W):
        a = self._ln(h, W["ln2_g"], W["ln2_b"])
        f = self.R(nx.gelu(a @ W["w1"].T + W["b1"]))
        return self.R(h + (f @ W["w2"].T + W["b2"]))

    def forward(self, src_ids, src_mask, tgt_ids, tgt_mask,
                force: Optional[Dict] = None) -> Seq2SeqResult:
        """``force`` may override the two padding predicates
        (``pad_any_src``, ``pad_any_tgt``) to exercise each branch."""
        c = self.cfg
        force = force or {}
        fwd = self.forward_count
        self.forward_count += 1
        src_ids, src_mask = np.asarray(src_ids), np.asarray(src_mask)
        tgt_ids, tgt_mask = np.asarray(tgt_ids), np.asarray(tgt_mask)
        B, Ss = src_ids.shape
        St = tgt_ids.shape[1]
        assert src_mask.shape == (B, Ss) and tgt_ids.shape[0] == B and tgt_mask.shape == (B, St)
        d = c.d_model

        # guards in code order, each over the source then the target
        ids_all = np.concatenate([src_ids.reshape(-1), tgt_ids.reshape(-1)])
        mask_all = np.concatenate([src_mask.reshape(-1), tgt_mask.reshape(-1)])
        bad = (ids_all < 0) | (ids_all >= c.vocab)
        if bad.any():
            raise Trap(TRAP_TOKEN_RANGE, int(np.argmax(bad)))
        bad = (mask_all != 0) & (mask_all != 1)
        if bad.any():
            raise Trap(TRAP_MASK_VALUE, int(np.argmax(bad)))

        # the two padding branches (host reads of mask.any())
        effects: List[Effect] = []
        pad_src = bool(force.get("pad_any_src", (src_mask == 0).any()))
        pad_tgt = bool(force.get("pad_any_tgt", (tgt_mask == 0).any()))
        if pad_src:
            effects.append(Effect(fwd, EFFECT_PAD, -1, 0, float((src_mask == 0).sum())))
        if pad_tgt:
            effects.append(Effect(fwd, EFFECT_PAD, -1, 1, float((tgt_mask == 0).sum())))

        enc_allowed = np.ones((B, 1, Ss, Ss), dtype=bool)
        x_allowed = np.ones((B, 1, St, Ss), dtype=bool)
        if pad_src:
            enc_allowed &= (src_mask == 1)[:, None, None, :]
            x_allowed &= (src_mask == 1)[:, None, None, :]
        dec_allowed = np.broadcast_to(np.tril(np.ones((St, St), dtype=bool))[None, None],
                                      (B, 1, St, St)).copy()
        if pad_tgt:
            dec_allowed &= (tgt_mask == 1)[:, None, None, :]

        tok = self._g("tok_emb")
        # ---------------- encoder
        h = self.R(tok[src_ids] + self._g("enc_pos_emb")[:Ss][None])
        for l in range(c.n_layers):
            W = {k: nx.decode(v, self.dt) for k, v in self.w.layers[l].items()}
            wq, wk, wv = W["wqkv"][:d], W["wqkv"][d:2 * d], W["wqkv"][2 * d:]
            bq, bk, bv = W["bqkv"][:d], W["bqkv"][d:2 * d], W["bqkv"][2 * d:]
            a = self._ln(h, W["ln1_g"], W["ln1_b"])
            ctx = self._attend(a, a, wq, bq, wk, bk, wv, bv, enc_allowed)
            h = self.R(h + (ctx @ W["wo"].T + W["bo"]))
            h = self._ffn(h, W)
        memory = self._ln(h, self._g("enc_lnf_g"), self._g("enc_lnf_b"))

        # ---------------- decoder
        h = self.R(tok[tgt_ids] + self._g("pos_emb")[:St][None])
        for l in range(c.n_dec_layers):
            W = {k: nx.decode(v, self.dt) for k, v in self.w.dec_layers[l].items()}
            wq, wk, wv = W["wqkv"][:d], W["wqkv"][d:2 * d], W["wqkv"][2 * d:]
            bq, bk, bv = W["bqkv"][:d], W["bqkv"][d:2 * d], W["bqkv"][2 * d:]
            a = self._ln(h, W["ln1_g"], W["ln1_b"])
            ctx = self._attend(a, a, wq, bq, wk, bk, wv, bv, dec_allowed)
            h = self.R(h + (ctx @ W["wo"].T + W["bo"]))
            a = self._ln(h, W["x_lnc_g"], W["x_lnc_b"])
            xk, xv = W["x_wkv"][:d], W["x_wkv"][d:]
            xbk, xbv = W["x_bkv"][:d], W["x_bkv"][d:]
            ctx = self._attend(a, memory, W["x_wq"], W["x_bq"], xk, xbk, xv, xbv, x_allowed)
            h = self.R(h + (ctx @ W["x_wo"].T + W["x_bo"]))
            h = self._ffn(h, W)
        z = self._ln(h, self._g("lnf_g"), self._g("lnf_b"))
        logits = self.R(z @ tok.T)
        return Seq2SeqResult(logits, nx.to_storage(logits, self.dt), pad_src, pad_tgt,
                             effects, memory)
