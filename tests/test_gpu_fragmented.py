"""The fragmented execution mode: the unmended program, cut into one graph
per region between graph breaks, with a host synchronisation, a read-back
and a host-side branch at every break.  It launches the same kernels, so
its results must equal the single-graph forward bit for bit, while its
counters show the breaks the single-graph forward removes.  Each graph-broken
run is also compared with the oracle on the same inputs: the decisions its
host branches took (padding, rotary regrow, every clamp site) exactly, the
logits within the parity tolerance."""
import numpy as np
import pytest
import torch

import synth
from oracle import TRAP_TOKEN_RANGE, OracleModel

from test_gpu_parity import check_decisions, check_logits, f64, gpu_effects, gpu_model

pytestmark = pytest.mark.gpu


def _forward(m, ids_t, mask_t, out):
    m.forward(ids_t, mask_t, out)
    torch.cuda.synchronize()
    return out.clone()


@pytest.mark.parametrize("name,n_breaks", [
    ("tiny_decoder", 1), ("causal_lm_768", 1), ("encoder_clamp_1024", 1 + 2 * 3),
    ("decoder_4096", 1)])
def test_fragmented_equals_single_graph(name, n_breaks):
    cfg = synth.preset(name) if name == "tiny_decoder" else synth.reduced(name)
    w = synth.make_weights(cfg, 21)
    ids, mask = synth.make_inputs(cfg, 2)
    ids_t = torch.from_numpy(ids).cuda()
    mask_t = torch.from_numpy(mask).cuda()
    a = gpu_model(cfg, w)
    b = gpu_model(cfg, w)
    out_a = a.new_logits(*ids.shape)
    out_b = b.new_logits(*ids.shape)
    b.set_exec_mode("fragmented")
    orc = OracleModel(cfg, w)
    for k in range(2):     # the rotary model regrows in the first call only
        ra = _forward(a, ids_t, mask_t, out_a)
        s0 = b.stats()
        rb = _forward(b, ids_t, mask_t, out_b)
        s1 = b.stats()
        assert torch.equal(ra.view(torch.int16), rb.view(torch.int16)), f"call {k}"
        assert a.decisions() == b.decisions()
        res = orc.forward(ids, mask)
        check_decisions(b.decisions(), res, cfg)
        check_logits(f64(rb), res.logits_f64, cfg.dtype, f"{name} graph-broken call {k}")
        assert s1["host_syncs_in_forward"] - s0["host_syncs_in_forward"] == n_breaks
        assert s1["graph_launches"] - s0["graph_launches"] == n_breaks + 1
        print(f"{name} call {k}: {n_breaks} breaks, {n_breaks + 1} graphs", flush=True)
    assert gpu_effects(a) == gpu_effects(b)
    assert a.stats()["host_syncs_in_forward"] == 0


def test_fragmented_guard_raises_at_the_guard():
    from paper_2509_16248_amd import gm
    cfg = synth.preset("tiny_decoder")
    w = synth.make_weights(cfg, 3)
    ids, mask = synth.make_inputs(cfg, 0)
    ids[0, 4] = cfg.vocab + 7
    m = gpu_model(cfg, w)
    m.set_exec_mode("fragmented")
    out = m.new_logits(*ids.shape)
    with pytest.raises(gm.GmError) as e:
        m.forward(torch.from_numpy(ids).cuda(), torch.from_numpy(mask).cuda(), out)
    assert e.value.code == gm.GM_E_TRAP
    assert m.check_error() == (TRAP_TOKEN_RANGE, 4)
