"""Seeded synthetic workloads: model presets, weights and inputs.

This module is shared by the CPU oracle, the GPU tests and the benchmark.
It only draws random numbers and encodes them in the storage dtype of a
workload; it computes nothing of the transformer forward itself.

The paper measures Hugging Face models with their own weights and
unnamed inputs (Evaluation, Experimental Setup and Benchmark Suite).
Those are not available here, so five synthetic model shapes stand in
for them:

* ``tiny_decoder``      1 block, d=64, 2 heads, FFN 256 GELU, LayerNorm,
                        vocab 512, batch 1 x seq 16, fp32 (0..4 trailing pads)
* ``causal_lm_768``     12 layers, d=768, 12 heads, FFN 3072 GELU, pre-LN,
                        learned positions, vocab 50257, batch 8 x seq 512,
                        bf16 (0..128 trailing pads per sequence)
* ``encoder_1024``      24 layers, d=1024, 16 heads, FFN 4096 GELU, post-LN,
                        bidirectional, vocab 30522, batch 16 x seq 512, bf16
                        (0..256 trailing pads per sequence)
* ``encoder_clamp_1024`` 24 layers, d=1024, 16 heads, gated-GELU FFN 2816,
                        RMSNorm, fp16, batch 4 x seq 1024, weights N(0,0.05)
                        with 1% of the entries of every matrix scaled x200
                        (overflow guard)
* ``decoder_4096``      32 layers, d=4096, 32 heads, SwiGLU FFN 11008,
                        RMSNorm, rotary (base 1e4, cache 1024 grown on
                        demand), vocab 32000, batch 1 x seq 2048, bf16
* ``decoder_4096_longrope`` the same shape with a Phi-4-style long/short
                        rotary frequency select (original context 1024:
                        2048 positions take the long factors)
* ``seq2seq_768``       encoder-decoder (BART-base-shaped, pre-LN): 6 encoder
                        + 6 decoder layers with cross-attention, d=768, 12
                        heads, FFN 3072 GELU, learned positions, shared
                        embedding and head, vocab 50265, batch 8, source 512
                        (0..128 pads), target 128 (0..32 pads), bf16

Weights: every tensor is drawn from its own PCG64 stream seeded by
``SeedSequence([seed, tensor_index])``; matrices, embeddings and biases are
N(0, sigma), norm gains are 1 + N(0, sigma), norm shifts N(0, sigma).
Inputs: token ids uniform over the vocabulary; per-sequence trailing pad
counts uniform in [0, max_pad]; mask is 1 for a token and 0 for a pad.
"""
from __future__ import annotations

import copy
import dataclasses
from typing import Dict, List, Optional

import numpy as np

# Storage dtypes of a workload.
F32, BF16, F16 = "f32", "bf16", "f16"
# Norm kinds / placement, FFN kinds and position encodings.
LN, RMS = "layernorm", "rmsnorm"
PRE, POST = "pre", "post"
GELU, GEGLU, SWIGLU = "gelu", "geglu", "swiglu"
POS_NONE, POS_LEARNED, POS_ROTARY = "none", "learned", "rotary"


@dataclasses.dataclass
class ModelConfig:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int
    vocab: int
    batch: int
    seq: int
    dtype: str
    norm: str = LN
    norm_place: str = PRE
    emb_norm: bool = False
    ffn: str = GELU
    pos: str = POS_LEARNED
    causal: bool = True
    bias: bool = True
    tied_head: bool = True
    norm_eps: float = 1e-5
    rope_base: float = 10000.0
    rope_init_len: int = 0
    rope_capacity: int = 0
    fp16_clamp: bool = False
    clamp_margin: float = 1000.0
    sigma: float = 0.02
    outlier_frac: float = 0.0
    outlier_scale: float = 1.0
    max_pad: int = 0
    log_hidden: bool = False          # per-layer tensor-valued log (max |h| per sequence)
    rope_scaling: str = "none"        # "none" or "long_short"
    rope_orig_max: int = 0            # long factors when max(position) + 1 exceeds this
    rope_attn_factor: float = 1.0     # cos/sin scale of the scaled frequencies
    n_dec_layers: int = 0             # > 0: encoder-decoder (n_layers encoder layers)
    tgt_seq: int = 0                  # encoder-decoder: target positions
    tgt_max_pad: int = 0              # encoder-decoder: trailing pads of a target

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    @property
    def gated(self) -> bool:
        return self.ffn in (GEGLU, SWIGLU)

    def replace(self, **kw) -> "ModelConfig":
        c = copy.copy(self)
        for k, v in kw.items():
            if not hasattr(c, k):
                raise AttributeError(k)
            setattr(c, k, v)
        return c


PRESETS: Dict[str, ModelConfig] = {
    "tiny_decoder": ModelConfig(
        name="tiny_decoder", n_layers=1, d_model=64, n_heads=2, d_ff=256,
        vocab=512, batch=1, seq=16, dtype=F32, norm=LN, norm_place=PRE,
        ffn=GELU, pos=POS_LEARNED, causal=True, bias=True, tied_head=True,
        max_pad=4),
    "causal_lm_768": ModelConfig(
        name="causal_lm_768", n_layers=12, d_model=768, n_heads=12, d_ff=3072,
        vocab=50257, batch=8, seq=512, dtype=BF16, norm=LN, norm_place=PRE,
        ffn=GELU, pos=POS_LEARNED, causal=True, bias=True, tied_head=True,
        max_pad=128),
    "encoder_1024": ModelConfig(
        name="encoder_1024", n_layers=24, d_model=1024, n_heads=16, d_ff=4096,
        vocab=30522, batch=16, seq=512, dtype=BF16, norm=LN, norm_place=POST,
        emb_norm=True, ffn=GELU, pos=POS_LEARNED, causal=False, bias=True,
        tied_head=True, max_pad=256),
    "encoder_clamp_1024": ModelConfig(
        name="encoder_clamp_1024", n_layers=24, d_model=1024, n_heads=16,
        d_ff=2816, vocab=32000, batch=4, seq=1024, dtype=F16, norm=RMS,
        norm_place=PRE, ffn=GEGLU, pos=POS_NONE, causal=False, bias=False,
        tied_head=False, norm_eps=1e-6, fp16_clamp=True, sigma=0.05,
        outlier_frac=0.01, outlier_scale=200.0, max_pad=0),
    "decoder_4096": ModelConfig(
        name="decoder_4096", n_layers=32, d_model=4096, n_heads=32, d_ff=11008,
        vocab=32000, batch=1, seq=2048, dtype=BF16, norm=RMS, norm_place=PRE,
        ffn=SWIGLU, pos=POS_ROTARY, causal=True, bias=False, tied_head=False,
        norm_eps=1e-6, rope_base=10000.0, rope_init_len=1024,
        rope_capacity=4096, max_pad=0),
}


PRESETS["seq2seq_768"] = ModelConfig(
    name="seq2seq_768", n_layers=6, n_dec_layers=6, d_model=768, n_heads=12, d_ff=3072,
    vocab=50265, batch=8, seq=512, tgt_seq=128, dtype=BF16, norm=LN, norm_place=PRE,
    ffn=GELU, pos=POS_LEARNED, causal=True, bias=True, tied_head=True, max_pad=128,
    tgt_max_pad=32)


def make_target_inputs(cfg: ModelConfig, seed: int, batch: Optional[int] = None,
                       seq: Optional[int] = None, max_pad: Optional[int] = None):
    """Decoder inputs of an encoder-decoder workload: ids and a trailing-pad
    mask [B, tgt_seq], from a stream of their own."""
    B = cfg.batch if batch is None else batch
    S = cfg.tgt_seq if seq is None else seq
    P = cfg.tgt_max_pad if max_pad is None else max_pad
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7, 1])))
    ids = rng.integers(0, cfg.vocab, size=(B, S), dtype=np.int64).astype(np.int32)
    mask = np.ones((B, S), dtype=np.int32)
    if P > 0:
        pads = rng.integers(0, min(P, S - 1) + 1, size=B)
        for b in range(B):
            if pads[b]:
                mask[b, S - pads[b]:] = 0
    return ids, mask


def _longrope(base: ModelConfig, orig: int) -> ModelConfig:
    """``base`` with the long/short frequency select; the tables hold the
    whole capacity, and cos/sin are scaled by sqrt(1 + ln(c/o)/ln(o))."""
    import math
    cap = base.rope_capacity
    attn = math.sqrt(1.0 + math.log(cap / orig) / math.log(orig)) if cap > orig else 1.0
    return base.replace(rope_scaling="long_short", rope_orig_max=orig,
                        rope_attn_factor=float(np.float32(attn)), rope_init_len=cap)


PRESETS["decoder_4096_longrope"] = _longrope(PRESETS["decoder_4096"], 1024).replace(
    name="decoder_4096_longrope")


def preset(name: str, **overrides) -> ModelConfig:
    return PRESETS[name].replace(**overrides)


# ---------------------------------------------------------------- encoding

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Encode float32 values as bfloat16 bit patterns (round to nearest even)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    # r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16, in place; no uint32 overflow
    # for non-NaN inputs (|u| <= 0xFF800000)
    r = np.right_shift(u, np.uint32(16))
    np.bitwise_and(r, np.uint32(1), out=r)
    np.add(r, np.uint32(0x7FFF), out=r)
    np.add(r, u, out=r)
    np.right_shift(r, np.uint32(16), out=r)
    out = r.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def encode(x: np.ndarray, dtype: str) -> np.ndarray:
    """float32 array -> storage array (float32, uint16 bf16 bits, float16)."""
    if dtype == F32:
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == BF16:
        return f32_to_bf16_bits(x)
    if dtype == F16:
        return np.ascontiguousarray(x.astype(np.float16))
    raise ValueError(dtype)


# ---------------------------------------------------------------- weights

# Fixed tensor indices so that every tensor has its own random stream and a
# layer's weights can be regenerated without drawing the others.
GLOBAL_TENSORS = ["tok_emb", "pos_emb", "emb_ln_g", "emb_ln_b", "lnf_g",
                  "lnf_b", "lm_head", "rope_short_factor", "rope_long_factor",
                  "enc_pos_emb", "enc_lnf_g", "enc_lnf_b"]
# an encoder-decoder's decoder layer: the layer tensors plus its cross-attention
CROSS_TENSORS = ["x_lnc_g", "x_lnc_b", "x_wq", "x_bq", "x_wkv", "x_bkv", "x_wo", "x_bo"]
# rotary frequency factors: float32 whatever the storage dtype
ROPE_FACTORS = {"rope_short_factor", "rope_long_factor"}
LAYER_TENSORS = ["ln1_g", "ln1_b", "wqkv", "bqkv", "wo", "bo", "ln2_g",
                 "ln2_b", "w1", "b1", "w2", "b2"]
MATRICES = {"tok_emb", "pos_emb", "lm_head", "wqkv", "wo", "w1", "w2", "enc_pos_emb", "x_wq",
            "x_wkv", "x_wo"}


def _tensor_index(name: str, layer) -> int:
    if layer is None:
        return GLOBAL_TENSORS.index(name)
    if isinstance(layer, tuple):        # ("dec", l): decoder layer of an encoder-decoder
        return 2000 + 32 * layer[1] + (LAYER_TENSORS + CROSS_TENSORS).index(name)
    return 100 + 16 * layer + LAYER_TENSORS.index(name)


def tensor_shapes(cfg: ModelConfig) -> Dict[str, tuple]:
    """Shapes of the global tensors present in ``cfg`` (PyTorch layout)."""
    d, V = cfg.d_model, cfg.vocab
    s = {"tok_emb": (V, d)}
    if cfg.pos == POS_LEARNED:
        s["pos_emb"] = (cfg.tgt_seq if cfg.n_dec_layers else cfg.seq, d)
    if cfg.n_dec_layers:
        s["enc_pos_emb"] = (cfg.seq, d)
        s["enc_lnf_g"] = (d,)
        if cfg.norm == LN:
            s["enc_lnf_b"] = (d,)
    if cfg.emb_norm:
        s["emb_ln_g"] = (d,)
        if cfg.norm == LN:
            s["emb_ln_b"] = (d,)
    if cfg.norm_place == PRE:
        s["lnf_g"] = (d,)
        if cfg.norm == LN:
            s["lnf_b"] = (d,)
    if not cfg.tied_head:
        s["lm_head"] = (V, d)
    if cfg.rope_scaling == "long_short":
        s["rope_short_factor"] = (cfg.head_dim // 2,)
        s["rope_long_factor"] = (cfg.head_dim // 2,)
    return s


def layer_shapes(cfg: ModelConfig) -> Dict[str, tuple]:
    """Shapes of one layer's tensors. ``w1`` holds the gate rows first and the
    up rows second for gated FFNs; ``wqkv`` holds q, k, v row blocks."""
    d, ff = cfg.d_model, cfg.d_ff
    f1 = 2 * ff if cfg.gated else ff
    s = {"ln1_g": (d,), "wqkv": (3 * d, d), "wo": (d, d), "ln2_g": (d,),
         "w1": (f1, d), "w2": (d, ff)}
    if cfg.norm == LN:
        s["ln1_b"] = (d,)
        s["ln2_b"] = (d,)
    if cfg.bias:
        s.update({"bqkv": (3 * d,), "bo": (d,), "b1": (f1,), "b2": (d,)})
    return s


def cross_shapes(cfg: ModelConfig) -> Dict[str, tuple]:
    """Cross-attention tensors of an encoder-decoder's decoder layer
    (``x_wkv`` holds the k rows, then the v rows)."""
    d = cfg.d_model
    s = {"x_lnc_g": (d,), "x_wq": (d, d), "x_wkv": (2 * d, d), "x_wo": (d, d)}
    if cfg.norm == LN:
        s["x_lnc_b"] = (d,)
    if cfg.bias:
        s.update({"x_bq": (d,), "x_bkv": (2 * d,), "x_bo": (d,)})
    return s


def _draw(cfg: ModelConfig, seed: int, name: str, layer: Optional[int],
          shape: tuple) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([seed, _tensor_index(name, layer)])))
    if name in ROPE_FACTORS:
        # per-frequency factors shaped like a long-context rope: short ones
        # near 1, long ones growing from ~1 (fast frequencies) to ~16 (slow)
        u = np.sort(rng.random(shape, dtype=np.float32))
        if name == "rope_short_factor":
            return np.float32(1.0) + np.float32(0.25) * u
        return np.float32(1.0) + np.float32(15.0) * u * u
    x = rng.standard_normal(shape, dtype=np.float32) * np.float32(cfg.sigma)
    if name.endswith("_g"):
        x += np.float32(1.0)
    elif name in MATRICES and cfg.outlier_frac > 0:
        sel = rng.random(shape, dtype=np.float32) < cfg.outlier_frac
        x[sel] *= np.float32(cfg.outlier_scale)
    return encode(x, cfg.dtype)


def make_global_weights(cfg: ModelConfig, seed: int) -> Dict[str, np.ndarray]:
    return {k: _draw(cfg, seed, k, None, shp)
            for k, shp in tensor_shapes(cfg).items()}


def make_layer_weights(cfg: ModelConfig, seed: int, layer: int) -> Dict[str, np.ndarray]:
    return {k: _draw(cfg, seed, k, layer, shp)
            for k, shp in layer_shapes(cfg).items()}


@dataclasses.dataclass
class Weights:
    """Storage-dtype weights. ``layers`` is a list of per-layer dicts."""
    cfg: ModelConfig
    seed: int
    globals: Dict[str, np.ndarray]
    layers: List[Dict[str, np.ndarray]]
    dec_layers: List[Dict[str, np.ndarray]] = dataclasses.field(default_factory=list)

    def nbytes(self) -> int:
        n = sum(v.nbytes for v in self.globals.values())
        n += sum(v.nbytes for L in self.dec_layers for v in L.values())
        return n + sum(v.nbytes for L in self.layers for v in L.values())


def make_weights(cfg: ModelConfig, seed: int = 1234, threads: Optional[int] = None) -> Weights:
    """All weights; tensors are drawn on a thread pool (each has its own
    generator, so the result does not depend on the thread count)."""
    import concurrent.futures as cf
    import os
    tasks = [(k, None, shp) for k, shp in tensor_shapes(cfg).items()]
    for l in range(cfg.n_layers):
        tasks += [(k, l, shp) for k, shp in layer_shapes(cfg).items()]
    for l in range(cfg.n_dec_layers):
        shapes = dict(layer_shapes(cfg), **cross_shapes(cfg))
        tasks += [(k, ("dec", l), shp) for k, shp in shapes.items()]
    n = threads or min(16, len(os.sched_getaffinity(0)))
    with cf.ThreadPoolExecutor(max_workers=max(1, n)) as ex:
        arrays = list(ex.map(lambda t: _draw(cfg, seed, t[0], t[1], t[2]), tasks))
    glob, layers = {}, [dict() for _ in range(cfg.n_layers)]
    dec = [dict() for _ in range(cfg.n_dec_layers)]
    for (k, l, _), a in zip(tasks, arrays):
        if l is None:
            glob[k] = a
        elif isinstance(l, tuple):
            dec[l[1]][k] = a
        else:
            layers[l][k] = a
    return Weights(cfg, seed, glob, layers, dec)


# ---------------------------------------------------------------- inputs

def make_inputs(cfg: ModelConfig, seed: int, batch: Optional[int] = None,
                seq: Optional[int] = None, max_pad: Optional[int] = None):
    """Token ids int32 [B, S] uniform over the vocabulary, and a key-padding
    mask int32 [B, S] (1 = token, 0 = pad) with a uniform number of trailing
    pads in [0, max_pad] per sequence."""
    B = cfg.batch if batch is None else batch
    S = cfg.seq if seq is None else seq
    P = cfg.max_pad if max_pad is None else max_pad
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7])))
    ids = rng.integers(0, cfg.vocab, size=(B, S), dtype=np.int64).astype(np.int32)
    mask = np.ones((B, S), dtype=np.int32)
    if P > 0:
        pads = rng.integers(0, min(P, S - 1) + 1, size=B)
        for b in range(B):
            if pads[b]:
                mask[b, S - pads[b]:] = 0
    return ids, mask


# Reduced shapes used by parity tests: the same structure as each preset
# with fewer layers, a shorter sequence and a smaller vocabulary, so that the
# oracle finishes in seconds while every kernel still spans several tiles
# and a ragged tail.
def reduced(name: str) -> ModelConfig:
    base = PRESETS[name]
    if name == "tiny_decoder":
        return base
    if name == "causal_lm_768":
        return base.replace(n_layers=2, batch=3, seq=200, vocab=1000, max_pad=40)
    if name == "encoder_1024":
        return base.replace(n_layers=2, batch=3, seq=160, vocab=777, max_pad=60)
    if name == "encoder_clamp_1024":
        return base.replace(n_layers=3, batch=2, seq=192, vocab=900)
    if name == "decoder_4096":
        return base.replace(n_layers=2, d_model=512, n_heads=4, d_ff=1344,
                            batch=1, seq=300, vocab=1100, rope_init_len=128,
                            rope_capacity=512)
    if name == "seq2seq_768":
        return base.replace(n_layers=2, n_dec_layers=2, batch=3, seq=96, tgt_seq=40,
                            vocab=1000, max_pad=30, tgt_max_pad=10)
    if name == "decoder_4096_longrope":
        small = reduced("decoder_4096").replace(name=name)
        return _longrope(small, 128)
    raise KeyError(name)
