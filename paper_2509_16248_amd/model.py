"""Torch-facing wrapper over the C ABI: uploads host weight arrays with
PyTorch, passes device pointers and the current HIP stream to libgm, and
exposes the synchronising readers.  No compute happens here."""
from __future__ import annotations

import ctypes
from typing import Dict, List, Optional

import numpy as np
import torch

from . import gm

_DTYPES = {"f32": gm.GM_DTYPE_F32, "bf16": gm.GM_DTYPE_BF16, "f16": gm.GM_DTYPE_F16}
_TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
_NORM = {"layernorm": gm.GM_NORM_LAYER, "rmsnorm": gm.GM_NORM_RMS}
_PLACE = {"pre": gm.GM_NORM_PRE, "post": gm.GM_NORM_POST}
_FFN = {"gelu": gm.GM_FFN_GELU, "geglu": gm.GM_FFN_GEGLU, "swiglu": gm.GM_FFN_SWIGLU}
_POS = {"none": gm.GM_POS_NONE, "learned": gm.GM_POS_LEARNED, "rotary": gm.GM_POS_ROTARY}


def make_config(c, max_batch: Optional[int] = None, max_seq: Optional[int] = None,
                kv_cache: bool = False) -> gm.gm_config:
    """gm_config from any object with the workload attributes (n_layers,
    d_model, n_heads, d_ff, vocab, batch, seq, dtype, norm, norm_place,
    emb_norm, ffn, pos, causal, bias, tied_head, norm_eps, rope_*,
    fp16_clamp, clamp_margin)."""
    return gm.gm_config(
        abi_version=gm.GM_ABI_VERSION, n_layers=c.n_layers, d_model=c.d_model,
        n_heads=c.n_heads, d_ff=c.d_ff, vocab=c.vocab,
        max_batch=max_batch or c.batch, max_seq=max_seq or c.seq,
        norm=_NORM[c.norm], norm_place=_PLACE[c.norm_place], emb_norm=int(c.emb_norm),
        ffn=_FFN[c.ffn], pos=_POS[c.pos], causal=int(c.causal), has_bias=int(c.bias),
        tied_head=int(c.tied_head), norm_eps=c.norm_eps, rope_base=c.rope_base,
        rope_init_len=c.rope_init_len, rope_capacity=c.rope_capacity,
        act_dtype=_DTYPES[c.dtype], fp16_clamp=int(c.fp16_clamp),
        clamp_margin=c.clamp_margin, kv_cache=int(kv_cache),
        log_hidden=int(getattr(c, "log_hidden", False)),
        rope_scaling={"none": gm.GM_ROPE_PLAIN, "long_short": gm.GM_ROPE_LONG_SHORT}[
            getattr(c, "rope_scaling", "none")],
        rope_orig_max=int(getattr(c, "rope_orig_max", 0)),
        rope_attn_factor=float(getattr(c, "rope_attn_factor", 1.0)),
        n_dec_layers=int(getattr(c, "n_dec_layers", 0)),
        max_tgt=int(getattr(c, "tgt_seq", 0)))


def to_device(a: np.ndarray, dtype: str, device) -> torch.Tensor:
    """Storage array (float32, bf16 bits as uint16, float16) -> device tensor."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def torch_dtype(dtype: str) -> torch.dtype:
    return _TORCH[dtype]


class GmModel:
    """One libgm model.  ``globals_`` / ``layers`` hold host arrays (or
    device tensors) named as in gm_weights / gm_layer_weights."""

    def __init__(self, cfg, globals_: Dict, layers: List[Dict], device="cuda",
                 max_batch: Optional[int] = None, max_seq: Optional[int] = None,
                 kv_cache: bool = False, dec_layers: Optional[List[Dict]] = None):
        self.cfg = cfg
        self.device = torch.device(device)
        self.c = make_config(cfg, max_batch, max_seq, kv_cache)
        dt = cfg.dtype

        def dev(x):
            if x is None:
                return None
            if isinstance(x, torch.Tensor):
                return x.to(self.device).contiguous()
            return to_device(x, dt, self.device)

        keep = []
        w = gm.gm_weights()
        for name in gm.GLOBAL_FIELDS:
            t = dev(globals_.get(name))
            keep.append(t)
            setattr(w, name, t.data_ptr() if t is not None else None)
        arr = (gm.gm_layer_weights * cfg.n_layers)()
        for l, L in enumerate(layers):
            for name in gm.LAYER_FIELDS:
                t = dev(L.get(name))
                keep.append(t)
                setattr(arr[l], name, t.data_ptr() if t is not None else None)
        w.layers = ctypes.cast(arr, ctypes.POINTER(gm.gm_layer_weights))
        for name in ("enc_pos_emb", "enc_lnf_g", "enc_lnf_b"):
            t = dev(globals_.get(name))
            keep.append(t)
            setattr(w, name, t.data_ptr() if t is not None else None)
        if dec_layers:
            darr = (gm.gm_layer_weights * len(dec_layers))()
            xarr = (gm.gm_cross_weights * len(dec_layers))()
            for l, L in enumerate(dec_layers):
                for name in gm.LAYER_FIELDS:
                    t = dev(L.get(name))
                    keep.append(t)
                    setattr(darr[l], name, t.data_ptr() if t is not None else None)
                for name in gm.CROSS_FIELDS:
                    t = dev(L.get("x_" + name))
                    keep.append(t)
                    setattr(xarr[l], name, t.data_ptr() if t is not None else None)
            keep += [darr, xarr]
            w.dec_layers = ctypes.cast(darr, ctypes.POINTER(gm.gm_layer_weights))
            w.dec_cross = ctypes.cast(xarr, ctypes.POINTER(gm.gm_cross_weights))
        for name in ("rope_short_factor", "rope_long_factor"):
            x = globals_.get(name)
            if x is not None:
                t = torch.as_tensor(np.asarray(x, dtype=np.float32)).to(self.device)
                keep.append(t)
                setattr(w, name, t.data_ptr())
        torch.cuda.synchronize(self.device)
        with torch.cuda.device(self.device):
            self.handle = gm.gm_model_create(self.c, w)
        del keep

    def _stream(self, stream):
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        return s.cuda_stream

    def forward(self, ids: torch.Tensor, mask: torch.Tensor, logits: torch.Tensor,
                stream=None) -> torch.Tensor:
        B, S = ids.shape
        assert ids.dtype == torch.int32 and mask.dtype == torch.int32
        assert mask.shape == ids.shape and ids.is_contiguous() and mask.is_contiguous()
        assert logits.shape == (B, S, self.c.vocab) and logits.is_contiguous()
        assert logits.dtype == _TORCH[self.cfg.dtype]
        gm.gm_forward_ex(self.handle, B, S, ids.data_ptr(), mask.data_ptr(),
                         logits.data_ptr(), self._stream(stream))
        return logits

    def forward_noalloc(self, ids: torch.Tensor, mask: torch.Tensor, logits: torch.Tensor,
                        stream=None) -> torch.Tensor:
        """gm_forward_noalloc: the forward with its workspace in the
        library's static device scratch (no allocation; capturable)."""
        B, S = ids.shape
        assert ids.dtype == torch.int32 and mask.dtype == torch.int32
        assert mask.shape == ids.shape and ids.is_contiguous() and mask.is_contiguous()
        assert logits.shape == (B, S, self.c.vocab) and logits.is_contiguous()
        gm.gm_forward_noalloc(self.handle, B, S, ids.data_ptr(), mask.data_ptr(),
                              logits.data_ptr(), self._stream(stream))
        return logits

    def forward_seq2seq(self, src_ids: torch.Tensor, src_mask: torch.Tensor,
                        tgt_ids: torch.Tensor, tgt_mask: torch.Tensor, logits: torch.Tensor,
                        stream=None) -> torch.Tensor:
        """Encoder-decoder forward (gm_forward_seq2seq): logits [B, S_tgt, V]."""
        B, Ss = src_ids.shape
        St = tgt_ids.shape[1]
        for t in (src_ids, src_mask, tgt_ids, tgt_mask):
            assert t.dtype == torch.int32 and t.is_contiguous()
        assert src_mask.shape == (B, Ss) and tgt_ids.shape == tgt_mask.shape == (B, St)
        assert logits.shape == (B, St, self.c.vocab) and logits.is_contiguous()
        gm.gm_forward_seq2seq(self.handle, B, Ss, src_ids.data_ptr(), src_mask.data_ptr(), St,
                              tgt_ids.data_ptr(), tgt_mask.data_ptr(), logits.data_ptr(),
                              self._stream(stream))
        return logits

    def decode(self, ids: torch.Tensor, logits: torch.Tensor,
               next_ids: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """One gm_decode_step: ids [B] int32 (device), logits [B, vocab];
        next_ids [B] int32 receives the greedy tokens (may be ``ids``)."""
        (B,) = ids.shape
        assert ids.dtype == torch.int32 and ids.is_contiguous()
        assert logits.shape == (B, self.c.vocab) and logits.is_contiguous()
        assert logits.dtype == _TORCH[self.cfg.dtype]
        if next_ids is not None:
            assert next_ids.shape == (B,) and next_ids.dtype == torch.int32
        gm.gm_decode_step(self.handle, B, ids.data_ptr(), logits.data_ptr(),
                          next_ids.data_ptr() if next_ids is not None else None,
                          self._stream(stream))
        return logits

    def new_decode_logits(self, B: int) -> torch.Tensor:
        return torch.empty((B, self.c.vocab), dtype=_TORCH[self.cfg.dtype], device=self.device)

    def profile(self, ids: torch.Tensor, mask: torch.Tensor, logits: torch.Tensor, stream=None):
        """Per-launch timing of one eager forward (see gm_profile_forward)."""
        B, S = ids.shape
        return gm.gm_profile_forward(self.handle, B, S, ids.data_ptr(), mask.data_ptr(),
                                     logits.data_ptr(), self._stream(stream))

    def new_logits(self, B: int, S: int) -> torch.Tensor:
        return torch.empty((B, S, self.c.vocab), dtype=_TORCH[self.cfg.dtype],
                           device=self.device)

    def set_graph_mode(self, enabled: bool):
        gm.gm_set_graph_mode(self.handle, enabled)

    def set_exec_mode(self, mode: str):
        """'graph' (default), 'eager' or 'fragmented' (the unmended program:
        one graph per region, host sync + read-back at every graph break)."""
        gm.gm_set_exec_mode(self.handle, {"graph": gm.GM_EXEC_GRAPH, "eager": gm.GM_EXEC_EAGER,
                                          "fragmented": gm.GM_EXEC_FRAGMENTED}[mode])

    def decisions(self, stream=None) -> dict:
        d = gm.gm_read_decisions(self.handle, self._stream(stream))
        n = d.n_clamp_sites
        return {"pad_any": bool(d.pad_any), "regrow": bool(d.regrow), "need": d.need,
                "cached_len": d.cached_len, "forward_index": d.forward_index,
                "clamp": [bool(d.clamp[i]) for i in range(n)],
                "clamp_absmax": [d.clamp_absmax[i] for i in range(n)],
                "clamp_nan": [bool(d.clamp_nan[i]) for i in range(n)],
                "rope_long": bool(d.rope_long), "pad_any_tgt": bool(d.pad_any_tgt)}

    def check_error(self):
        return gm.gm_check_error(self.handle)

    def raise_on_trap(self):
        """Synchronise, and if a guard failed since the last check raise the
        exception the original guard raises (gm_trap_info)."""
        code, index = gm.gm_check_error(self.handle)
        gm.raise_trap(code, index)

    def set_mask_guard(self, expected: Optional[torch.Tensor]):
        """`if not torch.equal(attention_mask, expected): raise` on every
        later forward (None removes it).  Keeps a reference to ``expected``."""
        if expected is None:
            gm.gm_set_mask_guard(self.handle, None, 0, 0)
            self._guard = None
            return
        assert expected.dtype == torch.int32 and expected.dim() == 2 and expected.is_contiguous()
        self._guard = expected
        gm.gm_set_mask_guard(self.handle, expected.data_ptr(), *expected.shape)

    def flush_effects(self):
        return gm.gm_flush_effects(self.handle)

    def debug_buffer(self, which: int, rows: int, cols: int) -> torch.Tensor:
        """Copy of internal buffer ``which`` (see gm_debug_buffer) as a
        [rows, cols] tensor of the activation dtype; synchronises."""
        ptr, nbytes = gm.gm_debug_buffer(self.handle, which)
        esz = torch.empty((), dtype=_TORCH[self.cfg.dtype]).element_size()
        assert rows * cols * esz <= nbytes
        torch.cuda.synchronize(self.device)
        out = torch.empty((rows, cols), dtype=_TORCH[self.cfg.dtype], device=self.device)
        n = rows * cols * esz
        import ctypes as _ct
        hip = _ct.CDLL("libamdhip64.so")
        rc = hip.hipMemcpy(_ct.c_void_p(out.data_ptr()), _ct.c_void_p(ptr), _ct.c_size_t(n), 3)
        assert rc == 0, rc
        return out

    def forward_layers(self, ids: torch.Tensor, mask: torch.Tensor, logits: torch.Tensor,
                       stream=None) -> dict:
        """Forward (gm_debug_forward_layers) that also returns every layer's
        storage points as device tensors: name -> [n_layers, T, width] with
        names a1, qkv, ctx, h_mid, a2, f, h_out (T = B * S)."""
        B, S = ids.shape
        T, d, ff, L = B * S, self.c.d_model, self.c.d_ff, self.c.n_layers
        widths = [("a1", d), ("qkv", 3 * d), ("ctx", d), ("h_mid", d), ("a2", d), ("f", ff),
                  ("h_out", d)]
        per = T * (8 * d + ff)
        dump = torch.empty((L, per), dtype=_TORCH[self.cfg.dtype], device=self.device)
        gm.gm_debug_forward_layers(self.handle, B, S, ids.data_ptr(), mask.data_ptr(),
                                   logits.data_ptr(), self._stream(stream), dump.data_ptr(),
                                   dump.numel() * dump.element_size())
        out, off = {}, 0
        for name, wdt in widths:
            out[name] = dump[:, off:off + T * wdt].view(L, T, wdt)
            off += T * wdt
        return out

    def stats(self) -> dict:
        s = gm.gm_get_stats(self.handle)
        return {k: getattr(s, k) for k, _ in gm.gm_stats._fields_}

    def close(self):
        if getattr(self, "handle", None):
            gm.gm_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
