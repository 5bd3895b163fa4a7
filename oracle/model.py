"""CPU oracle: the *unmended* transformer forward, with host-side branches.

Test infrastructure only.  Only the tests, the smoke check and the CPU
baseline of the benchmark may import this package; the product never does.

GraphMend rewrites a program so that it reaches exactly the result the
original program reaches (Semantics Preservation section; fp32 outputs were
bit-identical in the Output correctness validation paragraph).  The
plain definition of what the mended GPU forward computes is therefore the
original forward, in which every graph-breaking pattern is ordinary host
control flow on a value read back from the tensor:

* a validation guard ``if not C: raise`` on the inputs (Predicated Validation
  Guards paragraph, Figure "guard_example", rule [Trap]);
* a data-dependent ``if`` on the padding mask: ``mask.any()`` gates whether a
  key-padding mask is applied (Data-dependent Control Flow paragraph, Figure
  "dc_example", rule [Where]);
* a data-dependent ``if`` on ``max(position_ids) + 1`` against the size of a
  memoised rotary cache, whose body rebuilds the cache (the Phi-4 example of
  the Motivation section, hoisting of a memoised initialisation in the
  AST Transformation Pass and Semantics Preservation sections);
* a data-dependent ``if`` on ``abs(h).max() > fp16_max - margin`` whose body
  clamps the residual stream (rule [Where]; the untaken path must never leak
  NaN/Inf, Semantics Preservation section);
* print-style side effects at each taken branch, here emitted eagerly in
  program order (rule [Defer]: the mended program replays them after the
  graph, in FIFO order, with the values captured at the call site).

All arithmetic is float64.  ``round_to`` stores a tensor in the workload's
dtype at the storage points of the program: embedding output, norm output,
q/k/v (after rotary), attention context, residual stream after each add,
FFN hidden after the activation, logits.  GEMM results are never rounded
before their epilogue (bias, activation, residual add).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

from . import numerics as nx

# Trap codes, in the order the guards appear in the program.
TRAP_TOKEN_RANGE = 1
TRAP_MASK_VALUE = 2
TRAP_ROPE_CAPACITY = 3
TRAP_KV_CAPACITY = 4
TRAP_MASK_GUARD = 5

# The exception each guard of the original program raises (type, message):
# what a [Trap] failure is reported as once it surfaces on the host.
TRAP_INFO = {
    TRAP_TOKEN_RANGE: ("IndexError", "token id out of range"),
    TRAP_MASK_VALUE: ("ValueError", "attention mask values must be 0 or 1"),
    TRAP_ROPE_CAPACITY: ("ValueError", "rotary position exceeds the table capacity"),
    TRAP_KV_CAPACITY: ("IndexError", "sequence exceeds the KV cache capacity"),
    TRAP_MASK_GUARD: ("ValueError", "unsupported attention mask"),
}

# Kinds of deferred effect records.
EFFECT_PAD = 1
EFFECT_REGROW = 2
EFFECT_CLAMP = 3
EFFECT_LOG = 4

FP16_MAX = 65504.0


class Trap(Exception):
    """A validation guard failed (rule [Trap]); ``index`` is the row-major
    position of the first offending element (0 for the rotary capacity)."""

    def __init__(self, code: int, index: int):
        super().__init__(f"trap code={code} index={index}")
        self.code = code
        self.index = index


@dataclasses.dataclass
class Effect:
    forward: int
    kind: int
    layer: int
    site: int
    value: float
    values: Optional[Tuple[float, ...]] = None   # tensor argument of a log, as cloned


@dataclasses.dataclass
class OracleResult:
    logits: np.ndarray               # storage dtype, [B, S, V]
    logits_f64: np.ndarray           # same values as float64
    pad_any: bool
    regrow: bool
    need: int
    cached_len: int
    clamp: List[Tuple[bool, bool]]   # per layer: (attention site, FFN site)
    clamp_absmax: List[Tuple[float, float]]
    clamp_nan: List[Tuple[bool, bool]]
    clamp_margin: List[Tuple[float, float]]   # distance of max |pre-rounding| from the trip boundary
    effects: List[Effect]
    rope_long: bool = False          # long/short rotary select: long factors used


@dataclasses.dataclass
class _Begin:
    """State of a forward after its prologue (OracleModel.begin)."""
    forward: int
    effects: List[Effect]
    pad_any: bool
    regrow: bool
    need: int
    rope_long: bool
    S: int
    Br: int
    allowed: np.ndarray   # [Br, 1, S, S] keys each query may attend to
    h: np.ndarray         # [Br, S, d] embedding output (stored)


def _cfg_get(cfg, name):
    return getattr(cfg, name)


class OracleModel:
    """Float64 reference of the forward of one synthetic model.

    ``weights`` is a :class:`synth.Weights` (storage-dtype arrays); layers
    are decoded to float64 one at a time.  The rotary cache and the forward
    counter are model state that persists across calls, as in the original
    program (the memoised ``inv_freq``/cos/sin buffers of a rotary module).
    """

    def __init__(self, cfg, weights):
        self.cfg = cfg
        self.w = weights
        self.dt = cfg.dtype
        self.forward_count = 0
        self.cached_len = 0
        self.rope_cos = self.rope_sin = None
        # `if not torch.equal(attention_mask, expected): raise` when set
        self.mask_guard: Optional[np.ndarray] = None
        if cfg.pos == "rotary" and cfg.rope_scaling == "none":
            self._rope_build(cfg.rope_init_len)

    # ---------------------------------------------------------------- helpers
    def _g(self, name):
        return nx.decode(self.w.globals[name], self.dt)

    def _layer(self, l):
        return {k: nx.decode(v, self.dt) for k, v in self.w.layers[l].items()}

    def R(self, x):
        return nx.round_to(x, self.dt)

    def _norm(self, x, g, b):
        c = self.cfg
        if c.norm == "rmsnorm":
            return nx.rms_norm(x, g, c.norm_eps)
        return nx.layer_norm(x, g, b, c.norm_eps)

    def _rope_build(self, n):
        """Body of the rotary-cache branch: (re)build the cos/sin tables for
        positions [0, n) and record the new cache length."""
        self.rope_cos, self.rope_sin = nx.rope_table(
            n, self.cfg.head_dim, self.cfg.rope_base)
        self.cached_len = n

    # ---------------------------------------------------------------- forward
    def forward(self, ids: np.ndarray, mask: np.ndarray,
                force: Optional[Dict] = None,
                rows: Optional[List[int]] = None,
                prefix: Optional[int] = None,
                progress=None) -> OracleResult:
        """Run the original (graph-breaking) forward.

        ``force`` overrides the value a host-side predicate reads
        (``pad_any``, ``regrow`` or ``clamp`` = {(layer, site): bool}) so that
        each branch outcome can be exercised.  ``rows`` restricts the
        computation to a subset of the sequences of the batch; predicates
        that the program evaluates over the whole batch (the padding branch)
        are still evaluated over the whole batch.  It is rejected for the
        fp16 clamp, whose predicate reads the residual of every sequence.
        ``prefix`` (causal models only) computes the first ``prefix``
        positions of each sequence; with a causal mask they depend on no later
        position, so they equal those positions of the full forward.  The
        predicates (padding branch, rotary cache size) still read the full
        inputs, as the original program does.  ``progress``, if given, is
        called with the layer index after each layer (long runs report
        progress through it; it takes no part in the arithmetic).
        """
        c = self.cfg
        st = self.begin(ids, mask, force, rows, prefix)
        force = force or {}
        fwd, effects, h, allowed = st.forward, st.effects, st.h, st.allowed
        pad_any, regrow, need, rope_long, Br = st.pad_any, st.regrow, st.need, st.rope_long, st.Br
        S = st.S

        clamp, absmaxes, nans, margins = [], [], [], []
        for l in range(c.n_layers):
            W = self._layer(l)
            site_out = []
            # ---------------- attention block
            a = self.step_norm(h, W, 1) if c.norm_place == "pre" else h
            q, k, v = self.step_qkv(a, W, S)
            ctx = self.step_attention(q, k, v, allowed)
            h, pre = self.step_residual(h, ctx, W["wo"], W.get("bo"))
            if c.norm_place == "post":
                h = self.step_norm(h, W, 1)
            h, info = self._clamp_site(h, pre, l, 0, force, fwd, effects)
            site_out.append(info)

            # ---------------- feed-forward block
            a = self.step_norm(h, W, 2) if c.norm_place == "pre" else h
            f = self.step_ffn(a, W)
            h, pre = self.step_residual(h, f, W["w2"], W.get("b2"))
            if c.norm_place == "post":
                h = self.step_norm(h, W, 2)
            h, info = self._clamp_site(h, pre, l, 1, force, fwd, effects)
            site_out.append(info)
            if c.log_hidden:
                # logger.info(..., h.abs().amax per sequence): the tensor is
                # taken here; the original prints it at once
                vals = tuple(float(v) for v in np.abs(h).reshape(Br, -1).max(axis=1))
                effects.append(Effect(fwd, EFFECT_LOG, l, 0, float(Br), vals))
            clamp.append((site_out[0][0], site_out[1][0]))
            absmaxes.append((site_out[0][1], site_out[1][1]))
            nans.append((site_out[0][2], site_out[1][2]))
            margins.append((site_out[0][3], site_out[1][3]))
            if progress is not None:
                progress(l)

        # --- head.
        logits = self.step_head(h)
        return OracleResult(
            logits=nx.to_storage(logits, self.dt), logits_f64=logits,
            pad_any=pad_any, regrow=regrow, need=need,
            cached_len=self.cached_len, clamp=clamp, clamp_absmax=absmaxes,
            clamp_nan=nans, clamp_margin=margins, effects=effects, rope_long=rope_long)

    def begin(self, ids, mask, force: Optional[Dict] = None, rows: Optional[List[int]] = None,
              prefix: Optional[int] = None) -> "_Begin":
        """Everything before the first layer: the guards, the padding and
        rotary branches (with their effects and the rotary state update),
        the attention mask and the embedding output.  Counts a forward."""
        c = self.cfg
        force = force or {}
        fwd = self.forward_count
        self.forward_count += 1
        ids = np.asarray(ids)
        mask = np.asarray(mask)
        B, S = ids.shape
        assert mask.shape == (B, S)
        effects: List[Effect] = []

        # --- validation guards on the inputs (rule [Trap]), program order.
        bad = (ids < 0) | (ids >= c.vocab)
        if bad.any():
            raise Trap(TRAP_TOKEN_RANGE, int(np.argmax(bad.reshape(-1))))
        bad = (mask != 0) & (mask != 1)
        if bad.any():
            raise Trap(TRAP_MASK_VALUE, int(np.argmax(bad.reshape(-1))))

        # --- padding branch: a data-dependent if on the mask (host read).
        pad_any = bool((mask == 0).any())
        if "pad_any" in force:
            pad_any = bool(force["pad_any"])
        if pad_any:
            effects.append(Effect(fwd, EFFECT_PAD, -1, -1,
                                  float((mask == 0).sum())))

        # --- rotary cache branch: seq_len read back from max(position_ids).
        positions = np.broadcast_to(np.arange(S), (B, S))
        need = int(positions.max()) + 1
        regrow = False
        rope_long = False
        if c.pos == "rotary" and need > c.rope_capacity:
            raise Trap(TRAP_ROPE_CAPACITY, 0)

        # --- validation guard `if not torch.equal(mask, expected): raise`
        # (shapes and dtypes first: torch.equal is False when they differ).
        if self.mask_guard is not None:
            exp = np.asarray(self.mask_guard)
            if exp.shape != mask.shape or exp.dtype != mask.dtype:
                raise Trap(TRAP_MASK_GUARD, 0)
            diff = (mask != exp).reshape(-1)
            if diff.any():
                raise Trap(TRAP_MASK_GUARD, int(np.argmax(diff)))

        if c.pos == "rotary" and c.rope_scaling == "long_short":
            # Phi-4-style select: the long factors once the sequence exceeds
            # the original context; cos/sin built from the chosen factors
            rope_long = need > c.rope_orig_max
            factor = self.w.globals["rope_long_factor" if rope_long else "rope_short_factor"]
            self.rope_cos, self.rope_sin = nx.rope_table_scaled(
                S, c.head_dim, c.rope_base, factor, c.rope_attn_factor)
            self.cached_len = c.rope_capacity
        elif c.pos == "rotary":
            regrow = need > self.cached_len
            if "regrow" in force:
                regrow = bool(force["regrow"])
            if regrow:
                self._rope_build(need)
                effects.append(Effect(fwd, EFFECT_REGROW, -1, -1, float(need)))
            if need > self.cached_len:
                # The original program indexes the cache past its end.
                raise IndexError(
                    f"rotary cache holds {self.cached_len} positions, {need} needed")

        if rows is None:
            rows = list(range(B))
        if (c.fp16_clamp or c.log_hidden) and len(rows) != B:
            raise ValueError("the clamp predicate and the hidden log read every sequence")
        if prefix is not None:
            if not c.causal or c.fp16_clamp or c.log_hidden:
                raise ValueError("a prefix equals the full forward only for causal models")
            S = min(S, prefix)
        ids_r = ids[rows][:, :S]
        mask_r = mask[rows][:, :S]
        Br = len(rows)

        # --- attention mask: causal and/or key padding (only if pad_any).
        allowed = np.ones((Br, 1, S, S), dtype=bool)
        if c.causal:
            allowed &= np.tril(np.ones((S, S), dtype=bool))[None, None]
        if pad_any:
            allowed &= (mask_r == 1)[:, None, None, :]

        # --- embedding.
        x = self._g("tok_emb")[ids_r]
        if c.pos == "learned":
            x = x + self._g("pos_emb")[:S][None]
        h = self.R(x)
        if c.emb_norm:
            h = self.R(self._norm(h, self._g("emb_ln_g"),
                                  self._g("emb_ln_b") if c.norm == "layernorm" else None))

        return _Begin(forward=fwd, effects=effects, pad_any=pad_any, regrow=regrow, need=need,
                      rope_long=rope_long, S=S, Br=Br, allowed=allowed, h=h)

    # ---------------------------------------------------------------- steps
    # The steps of one layer, each from its stored input to its stored output
    # (the storage points of the module docstring).  ``forward`` composes
    # them; tests may also apply one step to a given input.
    def layer_weights(self, l):
        """Layer l's weights as float64 (nn.Linear layout)."""
        return self._layer(l)

    def step_norm(self, h, W, which):
        """R(Norm(h)) with the layer's first (which=1) or second norm."""
        return self.R(self._norm(h, W[f"ln{which}_g"], W.get(f"ln{which}_b")))

    def step_qkv(self, a, W, S, positions=None):
        """q, k, v = R(a Wqkv^T + b), split per head [B, H, S, hd], with the
        rotary rotation of q and k (rotary models) before the rounding; the
        rows' positions are 0..S-1, or ``positions`` [S]."""
        c = self.cfg
        H, hd, d = c.n_heads, c.head_dim, c.d_model
        B = a.shape[0]
        qkv = a @ W["wqkv"].T
        if c.bias:
            qkv = qkv + W["bqkv"]
        q = qkv[..., :d].reshape(B, S, H, hd).transpose(0, 2, 1, 3)
        k = qkv[..., d:2 * d].reshape(B, S, H, hd).transpose(0, 2, 1, 3)
        v = qkv[..., 2 * d:].reshape(B, S, H, hd).transpose(0, 2, 1, 3)
        if c.pos == "rotary":
            pos = np.arange(S) if positions is None else np.asarray(positions)
            cos = self.rope_cos[pos]
            sin = self.rope_sin[pos]
            q = nx.apply_rope(q, cos, sin)
            k = nx.apply_rope(k, cos, sin)
        return self.R(q), self.R(k), self.R(v)

    def step_attention(self, q, k, v, allowed):
        """ctx = R(softmax over allowed keys of q k^T / sqrt(hd)) v), heads
        concatenated: [B, S, d]; a query with no allowed key gives 0."""
        B, H, S, hd = q.shape
        s = (q @ k.transpose(0, 1, 3, 2)) * (1.0 / np.sqrt(hd))
        p = nx.masked_softmax(s, allowed)
        return self.R(p @ v).transpose(0, 2, 1, 3).reshape(B, S, H * hd)

    def step_residual(self, h, x, Wm, b):
        """The residual add of a block: pre = h + x Wm^T (+ b); returns
        (R(pre), pre)."""
        o = x @ Wm.T
        if b is not None and self.cfg.bias:
            o = o + b
        pre = h + o
        return self.R(pre), pre

    def step_ffn(self, a, W):
        """f = R(gelu(a W1^T + b1)), or for gated FFNs R(act(a Wg^T) * (a Wu^T))
        with the gate rows first in W1."""
        c = self.cfg
        u = a @ W["w1"].T
        if c.bias:
            u = u + W["b1"]
        if c.gated:
            ff = c.d_ff
            g_, up = u[..., :ff], u[..., ff:]
            act = nx.gelu(g_) if c.ffn == "geglu" else nx.silu(g_)
            return self.R(act * up)
        return self.R(nx.gelu(u))

    def step_head(self, h):
        """logits = R(Norm_f(h) W_head^T) (pre-norm; post-norm models read h)."""
        c = self.cfg
        if c.norm_place == "pre":
            z = self.R(self._norm(h, self._g("lnf_g"),
                                  self._g("lnf_b") if c.norm == "layernorm" else None))
        else:
            z = h
        head = self._g("tok_emb") if c.tied_head else self._g("lm_head")
        return self.R(z @ head.T)

    def clamp_decision(self, h):
        """The fp16 overflow branch's predicate on a stored residual stream:
        (trip, max |h| over the non-NaN elements, any NaN).  ``max``
        propagates NaN, so a NaN anywhere makes the comparison false."""
        thr = FP16_MAX - self.cfg.clamp_margin
        has_nan = bool(np.isnan(h).any())
        finite = h[~np.isnan(h)]
        absmax = float(np.abs(finite).max(initial=0.0))
        return (not has_nan) and absmax > thr, absmax, has_nan

    def clamp_apply(self, h):
        """Body of the clamp branch: R(clip(h, -thr, thr))."""
        thr = FP16_MAX - self.cfg.clamp_margin
        return self.R(np.clip(h, -thr, thr))

    def _clamp_site(self, h, pre, l, s, force, fwd, effects):
        """fp16 overflow guard after a residual add: ``if abs(h).max() >
        fp16_max - margin: h = clamp(h)``.  ``max`` propagates NaN, and
        ``NaN > thr`` is False, so a NaN anywhere leaves h unclamped."""
        c = self.cfg
        if not c.fp16_clamp:
            return h, (False, 0.0, False, float("inf"))
        thr = FP16_MAX - c.clamp_margin
        has_nan = bool(np.isnan(h).any())
        m = float(np.abs(h).max()) if not has_nan else float("nan")
        trip = (not has_nan) and m > thr
        # distance of the largest pre-rounding magnitude from the value at
        # which the stored fp16 value first exceeds thr.
        boundary = _fp16_trip_boundary(thr)
        with np.errstate(invalid="ignore"):
            pm = float(np.nanmax(np.abs(pre)))
        margin = abs(pm - boundary)
        if (l, s) in force.get("clamp", {}):
            trip = bool(force["clamp"][(l, s)])
        if trip:
            lim = thr
            h = self.R(np.clip(h, -lim, lim))
            effects.append(Effect(fwd, EFFECT_CLAMP, l, s, m))
        absmax = m if not has_nan else float(np.abs(h[~np.isnan(h)]).max(initial=0.0))
        return h, (trip, absmax, has_nan, margin)


def _fp16_trip_boundary(thr: float) -> float:
    """Smallest magnitude whose fp16 rounding exceeds ``thr``: the midpoint
    between the largest fp16 value <= thr and the next fp16 value."""
    lo = np.float16(thr)
    if float(lo) > thr:
        lo = np.nextafter(lo, np.float16(0))
    hi = np.nextafter(lo, np.float16(np.inf))
    return (float(lo) + float(hi)) / 2.0
