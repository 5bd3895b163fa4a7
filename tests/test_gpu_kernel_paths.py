"""GPU parity for the kernel paths the five workloads do not reach, so that
every kernel libgm can launch runs under a test:

* the large-tile GEMM in fp16 (128x384, 128x256 and 256x256 tiles: a
  one-layer fp16 model of the 4096-wide decoder's shape), and a 2048-wide
  model whose products take other tile choices (gate/up: 352 tiles of
  256x256), in bf16 and fp16;
* attention of 16-bit models with head size 32 (the row kernel);
* causal attention with key lengths cut short by long padding, in bf16
  and fp16;
* the GM_DEBUG_SYNC switch (one host synchronisation per forward, same
  results).

Each forward is compared with the oracle over every position at 2e-2, with
decisions exact.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import OracleModel

from test_gpu_parity import check_decisions, check_logits, f64, gpu_model, run

pytestmark = pytest.mark.gpu


def _compare(cfg, seed=3):
    w = synth.make_weights(cfg, seed)
    ids, mask = synth.make_inputs(cfg, 1)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    res = OracleModel(cfg, w).forward(ids, mask)
    check_decisions(m.decisions(), res, cfg)
    check_logits(f64(out), res.logits_f64, cfg.dtype, f"{cfg.name} {cfg.dtype} d {cfg.d_model}")
    m.close()


def test_large_tile_gemm_fp16():
    """QKV 2048x12288x4096 (128x384 tiles, rotary), O and down (128x256),
    gate/up and head (256x256, K step 64 in two stages), in fp16."""
    _compare(synth.preset("decoder_4096", n_layers=1, dtype="f16"))


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_large_tile_gemm_k64_two_stages(dtype):
    """d 2048, SwiGLU 5632: gate/up 2048x11264x2048 gives 352 tiles of
    256x256 (1.375 waves); QKV 2048x6144 takes 128x384; K of 2048."""
    cfg = synth.preset("decoder_4096", n_layers=1, d_model=2048, n_heads=16, d_ff=5632,
                       dtype=dtype)
    _compare(cfg)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_attention_rows_16bit_head_size_32(dtype):
    """24 heads of 32 over d 768: attention of 16-bit models takes the row
    kernel for head sizes the MFMA kernel does not cover; with padding."""
    cfg = synth.reduced("causal_lm_768").replace(n_heads=24, dtype=dtype)
    _compare(cfg)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_causal_attention_with_long_padding(dtype):
    """4 x 512 causal positions with up to 480 trailing pads: key lengths
    from 32 up, so query blocks past a sequence's last key read no key tile
    beyond it, and whole key tiles of other blocks are padding."""
    cfg = synth.reduced("causal_lm_768").replace(seq=512, batch=4, max_pad=480, dtype=dtype)
    w = synth.make_weights(cfg, 5)
    ids, mask = synth.make_inputs(cfg, 2)
    print("pads per sequence", (mask == 0).sum(1).tolist(), flush=True)
    m = gpu_model(cfg, w)
    out = run(m, ids, mask)
    res = OracleModel(cfg, w).forward(ids, mask)
    check_decisions(m.decisions(), res, cfg)
    check_logits(f64(out), res.logits_f64, cfg.dtype, f"causal attention, long padding, {dtype}")
    m.close()


def test_debug_sync_switch(monkeypatch):
    cfg = synth.preset("tiny_decoder")
    w = synth.make_weights(cfg, 4)
    ids, mask = synth.make_inputs(cfg, 2)
    plain = gpu_model(cfg, w)
    ref = run(plain, ids, mask)
    monkeypatch.setenv("GM_DEBUG_SYNC", "1")
    dbg = gpu_model(cfg, w)
    for _ in range(3):
        out = run(dbg, ids, mask)
    assert torch.equal(out, ref)
    s = dbg.stats()
    assert s["host_syncs_in_forward"] == 3 and s["graph_launches"] == 3
    assert plain.stats()["host_syncs_in_forward"] == 0
    plain.close()
    dbg.close()
