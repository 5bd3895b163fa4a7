"""CPU oracle of KV-cache decoding, by full recomputation.

Test infrastructure only (see the package docstring).

A decode step of a causal model appends one token to each sequence and
produces the logits at the new position.  Its plain definition needs no
cache: with a causal mask, the hidden states at position p depend only on
positions 0..p, so the logits at the new position are the last row of an
ordinary forward over the whole extended sequence.  The cache the GPU keeps
is an implementation device; this oracle recomputes every step from the
tokens (the paper's text-generation workloads decode greedily, Evaluation
section, "Experimental Setup" and "Output correctness validation").

Readings taken here (the paper defines no decode program):

* sequence b of a prompt [B, S] continues at position L_b = 1 + its last
  unmasked position; prompt positions the mask hid stay hidden;
* the rotary-cache branch of a step reads need = max_b (L_b + 1) after the
  append, exactly as a forward over the extended batch does;
* a step has no padding branch (its input is one token per sequence, no
  mask), so it records no PAD effect; it records REGROW when the rotary
  branch is taken;
* guards of a step, in order of their codes: token range (code 1, index b),
  rotary capacity (code 3), a sequence already at the capacity ``max_seq``
  (code 4, index b);
* greedy choice = argmax over the logits as stored (the dtype the kernel
  decides in), lowest index among equal values, the first NaN if any.
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np

from .model import (EFFECT_PAD, EFFECT_REGROW, TRAP_KV_CAPACITY, TRAP_ROPE_CAPACITY,
                    TRAP_TOKEN_RANGE, Effect, OracleModel, Trap)


def greedy(logits_row: np.ndarray) -> int:
    """Index of the largest value (first NaN if any; lowest index on ties)."""
    row = np.asarray(logits_row, dtype=np.float64)
    nan = np.isnan(row)
    if nan.any():
        return int(np.argmax(nan))
    return int(np.argmax(row))


class DecodeStep:
    """Result of one oracle decode step."""

    def __init__(self, logits_f64, regrow, need, cached_len, effects):
        self.logits_f64 = logits_f64     # [B, V], values as stored
        self.regrow = regrow
        self.need = need
        self.cached_len = cached_len
        self.effects = effects           # list of Effect

    def greedy(self) -> List[int]:
        return [greedy(r) for r in self.logits_f64]

    def margins(self) -> List[float]:
        """Distance between the largest and the second largest logit of each
        row: a greedy choice is unambiguous when it exceeds the tolerance."""
        out = []
        for r in self.logits_f64:
            top = np.sort(r)[-2:]
            out.append(float(top[1] - top[0]))
        return out


class OracleDecoder:
    """Prefill a prompt, then decode one token per sequence per step.

    ``model`` is an :class:`OracleModel` (its rotary cache and forward
    counter are the program state a decode loop carries); ``max_seq`` is the
    number of positions a sequence may reach.
    """

    def __init__(self, model: OracleModel, max_seq: int):
        if not model.cfg.causal:
            raise ValueError("decoding needs a causal model")
        self.m = model
        self.max_seq = max_seq
        self.seqs: List[List[int]] = []
        self.masks: List[List[int]] = []

    def prefill(self, ids: np.ndarray, mask: np.ndarray):
        """Forward over the prompt; sequence b keeps its first L_b tokens."""
        res = self.m.forward(ids, mask)
        self.seqs, self.masks = [], []
        for b in range(ids.shape[0]):
            on = np.nonzero(mask[b])[0]
            L = int(on[-1]) + 1 if len(on) else 0
            self.seqs.append([int(t) for t in ids[b, :L]])
            self.masks.append([int(v) for v in mask[b, :L]])
        return res

    def lengths(self) -> List[int]:
        return [len(s) for s in self.seqs]

    def step(self, tokens) -> DecodeStep:
        c = self.m.cfg
        tokens = [int(t) for t in tokens]
        B = len(self.seqs)
        assert len(tokens) == B
        # guards, in program order; a failed guard still counts as a forward
        # of the program (its index is taken before the guards run)
        W = max(len(s) for s in self.seqs) + 1
        trap = None
        for b, t in enumerate(tokens):
            if trap is None and (t < 0 or t >= c.vocab):
                trap = Trap(TRAP_TOKEN_RANGE, b)
        if trap is None and c.pos == "rotary" and W > c.rope_capacity:
            trap = Trap(TRAP_ROPE_CAPACITY, 0)
        for b, s in enumerate(self.seqs):
            if trap is None and len(s) >= self.max_seq:
                trap = Trap(TRAP_KV_CAPACITY, b)
        if trap is not None:
            self.m.forward_count += 1
            raise trap
        # the extended batch, trailing padding up to the longest sequence
        ids = np.zeros((B, W), dtype=np.int32)
        mask = np.zeros((B, W), dtype=np.int32)
        for b in range(B):
            seq = self.seqs[b] + [tokens[b]]
            ids[b, :len(seq)] = seq
            mask[b, :len(seq)] = self.masks[b] + [1]
        res = self.m.forward(ids, mask)
        rows = np.stack([res.logits_f64[b, len(self.seqs[b])] for b in range(B)])
        for b in range(B):
            self.seqs[b].append(tokens[b])
            self.masks[b].append(1)
        effects = [Effect(e.forward, e.kind, e.layer, e.site, e.value)
                   for e in res.effects if e.kind != EFFECT_PAD]
        assert all(e.kind == EFFECT_REGROW for e in effects)
        return DecodeStep(rows, res.regrow, res.need, res.cached_len, effects)


def generate_greedy(model: OracleModel, ids: np.ndarray, mask: np.ndarray, steps: int,
                    max_seq: int, first: Optional[List[int]] = None):
    """Greedy generation: the first new token of each sequence is the argmax
    of the prefill logits at its last real position (or ``first``), each
    later one the argmax of the previous step.  Returns (tokens [steps, B],
    list of DecodeStep)."""
    dec = OracleDecoder(model, max_seq)
    pre = dec.prefill(ids, mask)
    if first is None:
        first = [greedy(pre.logits_f64[b, L - 1]) for b, L in enumerate(dec.lengths())]
    toks, out = [list(first)], []
    for t in range(steps):
        st = dec.step(toks[-1])
        out.append(st)
        if t + 1 < steps:
            toks.append(st.greedy())
    return np.array(toks, dtype=np.int32), out
