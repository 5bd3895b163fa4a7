"""CPU oracle of the graph-break-free transformer forward.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow float64
implementation of the *original* (unmended) forward with host-side
branches.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may import it; the HIP library and its Python binding
never do, and this package imports nothing from them.

Pins: every function is checked in ``tests/test_oracle_*.py`` against
closed forms, invariants, library routines and brute force (see the
docstrings there).  The composed forward as a whole has no value printed in
the paper to compare against; it is pinned by the composition of its pinned
parts and by a cross-check against PyTorch CPU functional operators.
"""
from .model import (EFFECT_CLAMP, EFFECT_LOG, EFFECT_PAD, EFFECT_REGROW, FP16_MAX,
                    TRAP_INFO, TRAP_MASK_GUARD, TRAP_MASK_VALUE, TRAP_ROPE_CAPACITY,
                    TRAP_TOKEN_RANGE, Effect, OracleModel, OracleResult, Trap)
from .decode import DecodeStep, OracleDecoder, generate_greedy, greedy
from .model import TRAP_KV_CAPACITY
from .seq2seq import OracleSeq2Seq, Seq2SeqResult
from . import numerics

__all__ = ["OracleModel", "OracleResult", "Trap", "Effect", "numerics",
           "TRAP_TOKEN_RANGE", "TRAP_MASK_VALUE", "TRAP_ROPE_CAPACITY",
           "EFFECT_PAD", "EFFECT_REGROW", "EFFECT_CLAMP", "FP16_MAX",
           "OracleDecoder", "DecodeStep", "generate_greedy", "greedy", "TRAP_KV_CAPACITY",
           "TRAP_MASK_GUARD", "TRAP_INFO", "EFFECT_LOG", "OracleSeq2Seq", "Seq2SeqResult"]
