"""GPU parity of KV-cache decoding (gm_decode_step) against the decode oracle.

Each case prefills a prompt with gm_forward_ex on a model created with
kv_cache, then runs decode steps fed with the oracle's greedy tokens
(teacher forcing, so one ambiguous greedy choice cannot desynchronise the
rest) and checks, every step:
* the logits of the new positions, to the forward's tolerance;
* the rotary decisions (regrow, need, cached length);
* the greedy token the device chose (next_ids) wherever the oracle's top
  two logits differ by more than twice the tolerance (an argmax closer than
  that may legitimately flip under rounding differences);
and at the end the deferred effect records.  A free-running loop (next_ids
fed back as the next step's input, no host read in between) must reproduce
the oracle's greedy sequence on the fp32 model.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import (TRAP_KV_CAPACITY, TRAP_TOKEN_RANGE, OracleDecoder,
                    OracleModel, Trap, generate_greedy, greedy)

from test_gpu_parity import TOL, check_logits, effects_of, f64, gpu_effects, gpu_model, run

pytestmark = pytest.mark.gpu


def decode(m, toks):
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(toks, dtype=np.int32))).cuda()
    out = m.new_decode_logits(len(toks))
    nxt = torch.full((len(toks),), -7, dtype=torch.int32, device="cuda")
    m.decode(t, out, nxt)
    torch.cuda.synchronize()
    return out, nxt.cpu().numpy()


def step_effects(st):
    return [(e.forward, e.kind, e.layer, e.site, np.float32(e.value)) for e in st.effects]


def decode_case(cfg, w, ids, mask, steps, max_seq, what):
    tol = TOL[cfg.dtype]
    orc = OracleModel(cfg, w)
    dec = OracleDecoder(orc, max_seq)
    pre = dec.prefill(ids, mask)
    m = gpu_model(cfg, w, max_seq=max_seq, kv_cache=True)
    out = run(m, ids, mask)
    check_logits(f64(out), pre.logits_f64, cfg.dtype, f"{what} prefill")
    toks = [greedy(pre.logits_f64[b, L - 1]) for b, L in enumerate(dec.lengths())]
    expect_fx = effects_of(pre)
    chosen, oracle_tokens, checked = [], [], 0
    for k in range(steps):
        st = dec.step(toks)
        logits, nxt = decode(m, toks)
        check_logits(f64(logits), st.logits_f64, cfg.dtype, f"{what} step {k}")
        dm = m.decisions()
        assert not dm["pad_any"]
        assert dm["regrow"] == st.regrow
        if cfg.pos == "rotary":
            assert (dm["need"], dm["cached_len"]) == (st.need, st.cached_len)
        scale = np.abs(st.logits_f64).max()
        for b, (g, mg) in enumerate(zip(st.greedy(), st.margins())):
            if mg > 2 * tol * scale:
                assert nxt[b] == g, f"{what} step {k} seq {b}: device chose {nxt[b]}, oracle {g}"
                checked += 1
        expect_fx += step_effects(st)
        chosen.append(nxt)
        toks = st.greedy()
        oracle_tokens.append(toks)
    print(f"{what}: {checked} of {steps * len(toks)} greedy choices unambiguous and equal",
          flush=True)
    assert gpu_effects(m) == expect_fx
    assert m.check_error() == (0, 0)
    return m


def test_decode_tiny_fp32_teacher_forced_and_free_running():
    cfg = synth.preset("tiny_decoder", seq=48, batch=2, max_pad=4)
    w = synth.make_weights(cfg, 31)
    ids, mask = synth.make_inputs(cfg, 3, seq=16)
    decode_case(cfg, w, ids, mask, 24, cfg.seq, "tiny")
    # free-running: next_ids is the next step's input, no host read between steps
    steps = 24
    toks, out = generate_greedy(OracleModel(cfg, w), ids, mask, steps, cfg.seq)
    margins = np.array([st.margins() for st in out])          # [steps, B]
    scale = max(np.abs(st.logits_f64).max() for st in out)
    m = gpu_model(cfg, w, max_seq=cfg.seq, kv_cache=True)
    run(m, ids, mask)
    cur = torch.from_numpy(toks[0].copy()).cuda()
    hist = torch.empty((steps, cfg.batch), dtype=torch.int32, device="cuda")
    logits = m.new_decode_logits(cfg.batch)
    for k in range(steps):
        hist[k].copy_(cur)
        m.decode(cur, logits, cur)
    torch.cuda.synchronize()
    got = hist.cpu().numpy()
    for b in range(cfg.batch):
        assert got[0, b] == toks[0, b]
        for k in range(1, steps):
            # the input of step k is the device's choice from the logits of step k - 1
            if margins[k - 1, b] <= 2 * TOL[cfg.dtype] * scale:
                print(f"seq {b}: ambiguous choice before step {k}, comparison stops", flush=True)
                break
            assert got[k, b] == toks[k, b], f"seq {b} step {k}"
    st = m.stats()
    assert st["decode_steps"] == steps and st["host_syncs_in_forward"] == 0


def test_decode_causal_lm_reduced_bf16_ragged_prompts():
    cfg = synth.reduced("causal_lm_768").replace(seq=96)
    w = synth.make_weights(cfg, 32)
    ids, mask = synth.make_inputs(cfg, 4, seq=72, max_pad=30)
    print("prompt lengths", mask.sum(1).tolist(), flush=True)
    decode_case(cfg, w, ids, mask, 12, cfg.seq, "causal_lm_768 reduced")


def test_decode_rotary_regrow_fires_mid_generation():
    cfg = synth.reduced("decoder_4096")        # rotary table: 128 rows at create
    w = synth.make_weights(cfg, 33)
    ids, mask = synth.make_inputs(cfg, 5, seq=120)
    m = decode_case(cfg, w, ids, mask, 16, cfg.seq, "decoder_4096 reduced")
    # lengths 121 .. 136 after the steps: the table grew at every step past 128
    d = m.decisions()
    assert d["cached_len"] == 136 and d["regrow"]


def test_decode_graph_is_sync_free_and_equals_eager():
    cfg = synth.reduced("causal_lm_768").replace(seq=96)
    w = synth.make_weights(cfg, 34)
    ids, mask = synth.make_inputs(cfg, 6, seq=60, max_pad=10)
    outs = {}
    for mode in ("eager", "graph"):
        m = gpu_model(cfg, w, max_seq=cfg.seq, kv_cache=True)
        m.set_exec_mode(mode)
        run(m, ids, mask)
        # fixed buffers: one graph serves every step
        ids_t = torch.tensor([1, 2, 3], dtype=torch.int32, device="cuda")
        logits = m.new_decode_logits(3)
        nxt = torch.empty(3, dtype=torch.int32, device="cuda")
        s0 = m.stats()
        seq = []
        for k in range(5):
            m.decode(ids_t, logits, nxt)
            seq.append(logits.clone())
            ids_t.copy_(nxt)
        torch.cuda.synchronize()
        s1 = m.stats()
        outs[mode] = seq
        if mode == "graph":
            assert s1["graph_launches"] - s0["graph_launches"] == 5
            assert s1["captures"] - s0["captures"] == 1
            assert s1["host_syncs_in_forward"] == 0
    for a, b in zip(outs["eager"], outs["graph"]):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_prefill_with_cache_equals_forward_without():
    cfg = synth.reduced("causal_lm_768")
    w = synth.make_weights(cfg, 35)
    ids, mask = synth.make_inputs(cfg, 7)
    a = run(gpu_model(cfg, w), ids, mask)
    b = run(gpu_model(cfg, w, kv_cache=True), ids, mask)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_decode_traps_leave_lengths_unchanged():
    cfg = synth.preset("tiny_decoder", seq=20, batch=2, max_pad=0)
    w = synth.make_weights(cfg, 36)
    ids, mask = synth.make_inputs(cfg, 8, seq=18)
    orc = OracleModel(cfg, w)
    dec = OracleDecoder(orc, cfg.seq)
    dec.prefill(ids, mask)
    m = gpu_model(cfg, w, max_seq=cfg.seq, kv_cache=True)
    run(m, ids, mask)
    with pytest.raises(Trap) as e:
        dec.step([3, cfg.vocab])
    decode(m, [3, cfg.vocab])
    assert m.check_error() == (TRAP_TOKEN_RANGE, 1) == (e.value.code, e.value.index)
    for k in range(2):                     # positions 18, 19: the last two
        st = dec.step([4 + k, 5 + k])
        logits, _ = decode(m, [4 + k, 5 + k])
        check_logits(f64(logits), st.logits_f64, cfg.dtype, f"after trap, step {k}")
    with pytest.raises(Trap) as e:
        dec.step([1, 1])
    decode(m, [1, 1])
    assert m.check_error() == (TRAP_KV_CAPACITY, 0) == (e.value.code, e.value.index)
    assert m.check_error() == (0, 0)


def test_full_size_causal_lm_768_decode_sampled():
    """The benchmarked model at full size (12 layers, d 768, vocab 50257,
    bf16): two prompts of 384 positions (ragged), three decode steps."""
    cfg = synth.preset("causal_lm_768", batch=2)
    w = synth.make_weights(cfg, 1234)
    ids, mask = synth.make_inputs(cfg, 9, seq=384, max_pad=100)
    decode_case(cfg, w, ids, mask, 3, cfg.seq, "causal_lm_768 full")


def test_decode_long_cache_several_load_trips():
    """Caches longer than one round trip of the decode attention's loads
    (512 keys at head size 64 in 16-bit; 8 x 12 heads keep one key chunk per
    (sequence, head)): 2 layers of the 768-wide model with a reduced
    vocabulary, prompts of 560-700 positions, three steps."""
    cfg = synth.preset("causal_lm_768", batch=8, n_layers=2, vocab=1000, seq=704, max_pad=140)
    w = synth.make_weights(cfg, 21)
    ids, mask = synth.make_inputs(cfg, 5, seq=700)
    print("prompt lengths", mask.sum(1).tolist(), flush=True)
    assert mask.sum(1).max() > 512
    decode_case(cfg, w, ids, mask, 3, cfg.seq, "causal_lm_768 long cache")


@pytest.mark.parametrize("dtype,batch", [("f16", 1), ("bf16", 3)])
def test_decode_wide_head_on_matrix_cores(dtype, batch):
    """A vocabulary of 9000 (>= 8192) sends the decode step's head to the
    matrix-core few-row kernel: fp16 and bf16, one row and three rows (the
    activation rows padded to 16), a vocabulary that is not a multiple of
    16 columns."""
    cfg = synth.reduced("causal_lm_768").replace(vocab=9001, batch=batch, seq=64, max_pad=8,
                                                 dtype=dtype)
    w = synth.make_weights(cfg, 31)
    ids, mask = synth.make_inputs(cfg, 2, seq=56)       # room for the 4 steps in the cache
    decode_case(cfg, w, ids, mask, 4, cfg.seq, f"causal_lm_768 reduced {dtype} vocab 9001")
