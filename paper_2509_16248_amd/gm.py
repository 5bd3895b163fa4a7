"""ctypes binding of libgm (include/gm.h), same names as the C ABI.

Argument marshalling only: every step of the forward runs in the HIP
kernels of libgm.so.  PyTorch provides device memory and streams.  If the
library has not been built, :func:`lib` raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Callable, List, Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgm.so")

GM_ABI_VERSION = 2
GM_MAX_LAYERS = 64
GM_OK, GM_E_INVAL, GM_E_NOMEM, GM_E_HIP, GM_E_CAPTURE, GM_E_TRAP = 0, -1, -2, -3, -4, -5
GM_EXEC_GRAPH, GM_EXEC_EAGER, GM_EXEC_FRAGMENTED = 0, 1, 2
GM_DTYPE_F32, GM_DTYPE_BF16, GM_DTYPE_F16 = 0, 1, 2
GM_NORM_LAYER, GM_NORM_RMS = 0, 1
GM_NORM_PRE, GM_NORM_POST = 0, 1
GM_FFN_GELU, GM_FFN_GEGLU, GM_FFN_SWIGLU = 0, 1, 2
GM_POS_NONE, GM_POS_LEARNED, GM_POS_ROTARY = 0, 1, 2
GM_TRAP_NONE, GM_TRAP_TOKEN_RANGE, GM_TRAP_MASK_VALUE, GM_TRAP_ROPE_CAPACITY = 0, 1, 2, 3
GM_TRAP_KV_CAPACITY, GM_TRAP_MASK_GUARD = 4, 5
GM_EFFECT_PAD, GM_EFFECT_REGROW, GM_EFFECT_CLAMP, GM_EFFECT_LOG = 1, 2, 3, 4
GM_ROPE_PLAIN, GM_ROPE_LONG_SHORT = 0, 1

_i32, _f32, _u64, _vp = ctypes.c_int32, ctypes.c_float, ctypes.c_uint64, ctypes.c_void_p


class gm_config(ctypes.Structure):
    _fields_ = [("abi_version", _i32), ("n_layers", _i32), ("d_model", _i32),
                ("n_heads", _i32), ("d_ff", _i32), ("vocab", _i32),
                ("max_batch", _i32), ("max_seq", _i32), ("norm", _i32),
                ("norm_place", _i32), ("emb_norm", _i32), ("ffn", _i32),
                ("pos", _i32), ("causal", _i32), ("has_bias", _i32),
                ("tied_head", _i32), ("norm_eps", _f32), ("rope_base", _f32),
                ("rope_init_len", _i32), ("rope_capacity", _i32),
                ("act_dtype", _i32), ("fp16_clamp", _i32), ("clamp_margin", _f32),
                ("kv_cache", _i32), ("log_hidden", _i32), ("rope_scaling", _i32),
                ("rope_orig_max", _i32), ("rope_attn_factor", _f32),
                ("n_dec_layers", _i32), ("max_tgt", _i32)]


LAYER_FIELDS = ["ln1_g", "ln1_b", "wqkv", "bqkv", "wo", "bo", "ln2_g", "ln2_b",
                "w1", "b1", "w2", "b2"]
GLOBAL_FIELDS = ["tok_emb", "pos_emb", "emb_ln_g", "emb_ln_b", "lnf_g", "lnf_b", "lm_head"]


class gm_layer_weights(ctypes.Structure):
    _fields_ = [(n, _vp) for n in LAYER_FIELDS]


CROSS_FIELDS = ["lnc_g", "lnc_b", "wq", "bq", "wkv", "bkv", "wo", "bo"]


class gm_cross_weights(ctypes.Structure):
    _fields_ = [(n, _vp) for n in CROSS_FIELDS]


class gm_weights(ctypes.Structure):
    _fields_ = ([(n, _vp) for n in GLOBAL_FIELDS] + [("layers", ctypes.POINTER(gm_layer_weights))]
                + [("rope_short_factor", _vp), ("rope_long_factor", _vp),
                   ("enc_pos_emb", _vp), ("enc_lnf_g", _vp), ("enc_lnf_b", _vp),
                   ("dec_layers", ctypes.POINTER(gm_layer_weights)),
                   ("dec_cross", ctypes.POINTER(gm_cross_weights))])


class gm_decisions(ctypes.Structure):
    _fields_ = [("pad_any", _i32), ("regrow", _i32), ("need", _i32),
                ("cached_len", _i32), ("n_clamp_sites", _i32),
                ("clamp", _i32 * (2 * GM_MAX_LAYERS)),
                ("clamp_absmax", _f32 * (2 * GM_MAX_LAYERS)),
                ("clamp_nan", _i32 * (2 * GM_MAX_LAYERS)),
                ("forward_index", _i32), ("rope_long", _i32), ("pad_any_tgt", _i32)]


class gm_effect(ctypes.Structure):
    _fields_ = [("forward", _i32), ("kind", _i32), ("layer", _i32),
                ("site", _i32), ("value", _f32), ("n_values", _i32),
                ("values", ctypes.POINTER(_f32))]


class gm_stats(ctypes.Structure):
    _fields_ = [("forwards", _u64), ("captures", _u64), ("graph_launches", _u64),
                ("eager_forwards", _u64), ("host_syncs_in_forward", _u64),
                ("kernels_per_forward", _u64), ("decode_steps", _u64)]


class gm_kernel_time(ctypes.Structure):
    _fields_ = [("kind", _i32), ("layer", _i32), ("ms", _f32), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double)]


KERNEL_KINDS = ["prologue", "rope_fill", "embed", "norm", "gemm_qkv", "attention",
                "gemm_o", "gemm_up", "gemm_down", "gemm_head", "effects", "kv_store",
                "argmax", "log", "gemm_xq", "gemm_xkv", "gemm_xo", "xattn"]

gm_effect_cb = ctypes.CFUNCTYPE(None, ctypes.POINTER(gm_effect), ctypes.c_void_p)

EXPORTS = ["gm_model_create", "gm_model_destroy", "gm_forward", "gm_forward_ex",
           "gm_decode_step", "gm_set_mask_guard", "gm_trap_info", "gm_forward_seq2seq",
           "gm_profile_forward", "gm_set_exec_mode", "gm_set_graph_mode", "gm_read_decisions", "gm_decisions_device_ptr",
           "gm_check_error", "gm_flush_effects", "gm_debug_buffer", "gm_debug_forward_layers",
           "gm_get_stats", "gm_forward_noalloc",
           "gm_strerror",
           "gm_last_error"]

_lib = None


def lib(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libgm.so (once).  Raises if it is missing: the forward has no
    other implementation."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2509_16248_amd.build`")
    L = ctypes.CDLL(path)
    L.gm_model_create.argtypes = [ctypes.POINTER(gm_config), ctypes.POINTER(gm_weights),
                                  ctypes.POINTER(_vp)]
    L.gm_model_destroy.argtypes = [_vp]
    L.gm_model_destroy.restype = None
    L.gm_forward.argtypes = [_vp, _vp, _vp, _vp, _vp]
    L.gm_forward_ex.argtypes = [_vp, _i32, _i32, _vp, _vp, _vp, _vp]
    L.gm_forward_noalloc.argtypes = [_vp, _i32, _i32, _vp, _vp, _vp, _vp]
    L.gm_decode_step.argtypes = [_vp, _i32, _vp, _vp, _vp, _vp]
    L.gm_set_mask_guard.argtypes = [_vp, _vp, _i32, _i32]
    L.gm_forward_seq2seq.argtypes = [_vp, _i32, _i32, _vp, _vp, _i32, _vp, _vp, _vp, _vp]
    L.gm_trap_info.argtypes = [_i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_char_p)]
    L.gm_set_graph_mode.argtypes = [_vp, _i32]
    L.gm_set_exec_mode.argtypes = [_vp, _i32]
    L.gm_profile_forward.argtypes = [_vp, _i32, _i32, _vp, _vp, _vp, _vp,
                                     ctypes.POINTER(gm_kernel_time), _i32, ctypes.POINTER(_i32)]
    L.gm_read_decisions.argtypes = [_vp, ctypes.POINTER(gm_decisions), _vp]
    L.gm_decisions_device_ptr.argtypes = [_vp]
    L.gm_decisions_device_ptr.restype = _vp
    L.gm_check_error.argtypes = [_vp, ctypes.POINTER(_i32), ctypes.POINTER(_i32)]
    L.gm_flush_effects.argtypes = [_vp, gm_effect_cb, _vp, ctypes.POINTER(_i32)]
    L.gm_debug_buffer.argtypes = [_vp, _i32, ctypes.POINTER(_vp), ctypes.POINTER(_u64)]
    L.gm_debug_forward_layers.argtypes = [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _u64]
    L.gm_get_stats.argtypes = [_vp, ctypes.POINTER(gm_stats)]
    L.gm_strerror.argtypes = [ctypes.c_int]
    L.gm_strerror.restype = ctypes.c_char_p
    L.gm_last_error.argtypes = []
    L.gm_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name not in ("gm_model_destroy", "gm_decisions_device_ptr", "gm_strerror",
                        "gm_last_error"):
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


class GmError(RuntimeError):
    def __init__(self, code: int, where: str):
        L = lib()
        super().__init__(f"{where}: {L.gm_strerror(code).decode()} ({code}): "
                         f"{L.gm_last_error().decode()}")
        self.code = code


def _check(rc: int, where: str):
    if rc != GM_OK:
        raise GmError(rc, where)


# ------------------------------------------------------------ C-named wrappers

def gm_model_create(cfg: gm_config, w: gm_weights) -> int:
    out = _vp()
    _check(lib().gm_model_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(out)),
           "gm_model_create")
    return out.value


def gm_model_destroy(m: int) -> None:
    lib().gm_model_destroy(m)


def gm_forward(m: int, ids: int, mask: int, logits: int, stream: int) -> None:
    _check(lib().gm_forward(m, ids, mask, logits, stream), "gm_forward")


def gm_forward_ex(m: int, B: int, S: int, ids: int, mask: int, logits: int, stream: int) -> None:
    _check(lib().gm_forward_ex(m, B, S, ids, mask, logits, stream), "gm_forward_ex")


def gm_decode_step(m: int, B: int, ids: int, logits: int, next_ids: Optional[int],
                   stream: int) -> None:
    _check(lib().gm_decode_step(m, B, ids, logits, next_ids, stream), "gm_decode_step")


def gm_forward_seq2seq(m: int, B: int, S_src: int, src_ids: int, src_mask: int, S_tgt: int,
                       tgt_ids: int, tgt_mask: int, logits: int, stream: int) -> None:
    _check(lib().gm_forward_seq2seq(m, B, S_src, src_ids, src_mask, S_tgt, tgt_ids, tgt_mask,
                                    logits, stream), "gm_forward_seq2seq")


def gm_set_mask_guard(m: int, expected: Optional[int], B: int, S: int) -> None:
    _check(lib().gm_set_mask_guard(m, expected, B, S), "gm_set_mask_guard")


def gm_trap_info(code: int):
    """(exception type name, message) of a trap code."""
    t, msg = ctypes.c_char_p(), ctypes.c_char_p()
    _check(lib().gm_trap_info(code, ctypes.byref(t), ctypes.byref(msg)), "gm_trap_info")
    return t.value.decode(), msg.value.decode()


_EXCEPTIONS = {"IndexError": IndexError, "ValueError": ValueError}


def raise_trap(code: int, index: int) -> None:
    """Re-raise a reported trap as the exception the original guard raised
    (rule [Trap]: the uid maps back to the original type and message)."""
    if code == GM_TRAP_NONE:
        return
    typ, msg = gm_trap_info(code)
    err = _EXCEPTIONS[typ](msg)
    err.trap_code, err.trap_index = code, index
    raise err


def gm_profile_forward(m: int, B: int, S: int, ids: int, mask: int, logits: int,
                       stream: int, cap: int = 4096):
    """Per-launch (kind name, layer, ms, flops, bytes) of one eager forward."""
    arr = (gm_kernel_time * cap)()
    n = _i32()
    _check(lib().gm_profile_forward(m, B, S, ids, mask, logits, stream, arr, cap,
                                    ctypes.byref(n)), "gm_profile_forward")
    return [(KERNEL_KINDS[arr[i].kind], arr[i].layer, arr[i].ms, arr[i].flops, arr[i].bytes)
            for i in range(min(n.value, cap))]


def gm_set_exec_mode(m: int, mode: int) -> None:
    _check(lib().gm_set_exec_mode(m, int(mode)), "gm_set_exec_mode")


def gm_set_graph_mode(m: int, enabled: bool) -> None:
    _check(lib().gm_set_graph_mode(m, int(bool(enabled))), "gm_set_graph_mode")


def gm_read_decisions(m: int, stream: int) -> gm_decisions:
    d = gm_decisions()
    _check(lib().gm_read_decisions(m, ctypes.byref(d), stream), "gm_read_decisions")
    return d


def gm_decisions_device_ptr(m: int) -> int:
    return lib().gm_decisions_device_ptr(m)


def gm_check_error(m: int):
    code, index = _i32(), _i32()
    _check(lib().gm_check_error(m, ctypes.byref(code), ctypes.byref(index)), "gm_check_error")
    return code.value, index.value


def gm_flush_effects(m: int, cb: Optional[Callable[[gm_effect], None]] = None):
    """Replay the deferred effects through ``cb`` (FIFO order); returns
    (list of (forward, kind, layer, site, value), dropped)."""
    recs: List[tuple] = []

    def _cb(p, _user):
        e = p.contents
        if e.n_values:
            recs.append((e.forward, e.kind, e.layer, e.site, e.value,
                         tuple(e.values[i] for i in range(e.n_values))))
        else:
            recs.append((e.forward, e.kind, e.layer, e.site, e.value))
        if cb is not None:
            cb(e)

    c_cb = gm_effect_cb(_cb)
    dropped = _i32()
    _check(lib().gm_flush_effects(m, c_cb, None, ctypes.byref(dropped)), "gm_flush_effects")
    return recs, dropped.value


def gm_debug_buffer(m: int, which: int):
    """(device pointer, bytes) of internal buffer ``which`` (see gm.h)."""
    p, n = _vp(), _u64()
    _check(lib().gm_debug_buffer(m, which, ctypes.byref(p), ctypes.byref(n)), "gm_debug_buffer")
    return p.value, n.value


def gm_forward_noalloc(m: int, B: int, S: int, ids: int, mask: int, logits: int,
                       stream: int) -> None:
    _check(lib().gm_forward_noalloc(m, B, S, ids, mask, logits, stream), "gm_forward_noalloc")


def gm_debug_forward_layers(m: int, B: int, S: int, ids: int, mask: int, logits: int,
                            stream: int, dump: int, dump_bytes: int) -> None:
    _check(lib().gm_debug_forward_layers(m, B, S, ids, mask, logits, stream, dump, dump_bytes),
           "gm_debug_forward_layers")


def gm_get_stats(m: int) -> gm_stats:
    s = gm_stats()
    _check(lib().gm_get_stats(m, ctypes.byref(s)), "gm_get_stats")
    return s


def gm_strerror(code: int) -> str:
    return lib().gm_strerror(code).decode()
