"""gm_forward_noalloc (workspace in the library's static device scratch)
against gm_forward_ex through the C ABI: same logits bit for bit, same
decisions and effects, on two calls in a row, the second with a smaller
input, and a workspace beyond the static array is rejected."""
import numpy as np
import pytest
import torch

import synth
from paper_2509_16248_amd import gm

from test_gpu_parity import gpu_effects, gpu_model

pytestmark = pytest.mark.gpu


def _inputs(cfg, seed, B, S):
    ids, mask = synth.make_inputs(cfg, seed, batch=B, seq=S)
    return torch.from_numpy(ids).cuda(), torch.from_numpy(mask).cuda()


@pytest.mark.parametrize("name", ["causal_lm_768", "encoder_1024", "encoder_clamp_1024",
                                  "decoder_4096", "tiny_decoder"])
def test_noalloc_matches_forward_ex(name):
    cfg = synth.preset(name) if name == "tiny_decoder" else synth.reduced(name)
    w = synth.make_weights(cfg, 13)
    a = gpu_model(cfg, w)      # gm_forward_ex (graph)
    b = gpu_model(cfg, w)      # gm_forward_noalloc
    B0, S0 = cfg.batch, cfg.seq
    for k, (B, S) in enumerate([(B0, S0), (max(1, B0 - 1), max(2, S0 // 2 + 3))]):
        ids_t, mask_t = _inputs(cfg, 40 + k, B, S)
        out_a = a.new_logits(B, S)
        out_b = b.new_logits(B, S)
        out_b.fill_(float("nan"))
        a.forward(ids_t, mask_t, out_a)
        b.forward_noalloc(ids_t, mask_t, out_b)
        torch.cuda.synchronize()
        bits = torch.int16 if cfg.dtype != "f32" else torch.int32
        assert torch.equal(out_a.view(bits), out_b.view(bits)), f"{name} call {k} ({B} x {S})"
        da, db = a.decisions(), b.decisions()
        assert da == db, f"{name} call {k}"
        print(f"{name} call {k}: {B} x {S} bit-identical", flush=True)
    assert gpu_effects(a) == gpu_effects(b)
    assert b.check_error() == (0, 0)
    assert b.stats()["graph_launches"] == 0
    a.close()
    b.close()


def test_noalloc_rejects_a_workspace_beyond_the_scratch():
    # 4 x 1024 tokens x (6 * 1024 + 2816) fp16 elements = 73.4 MB > 64 MiB
    cfg = synth.preset("encoder_clamp_1024")
    w = synth.make_weights(cfg, 13)
    m = gpu_model(cfg, w)
    ids_t, mask_t = _inputs(cfg, 1, 4, 1024)
    out = m.new_logits(4, 1024)
    with pytest.raises(gm.GmError) as e:
        m.forward_noalloc(ids_t, mask_t, out)
    assert e.value.code == gm.GM_E_INVAL
    assert "static scratch" in str(e.value)
    m.close()
