"""Conditioning of the end-to-end logits of the deep workloads.

Writes depth_spread.json: for each workload and depth, the relative spread
max |L32 - L64| / max |L64| between the oracle's forward evaluated with
float64 arithmetic (L64, the definition) and the same forward evaluated with
float32 arithmetic (L32: stored values, weights and every product and sum in
float32).  Storage-point rounding turns such arithmetic-level differences
into one-ulp differences of stored activations, and depth amplifies them;
no implementation whose summation order differs from the oracle's can be
expected to agree with it more closely than this.  The end-to-end GPU logits
tests take twice this spread as their tolerance where it exceeds 1e-2, and
the per-step tests (test_gpu_stepwise.py) check every layer at 2e-2.

    python tests/golden/depth_spread.py [workload/key]   (repository root;
    calls only oracle/ and synth/; with an argument, recomputes that entry only)
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import OracleModel, numerics as nx  # noqa: E402


class Float32Oracle(OracleModel):
    """The oracle's program with float32 arithmetic: weights, stored values
    and all intermediate arithmetic in float32 (numpy keeps float32 when
    both operands are float32)."""

    def _g(self, name):
        return super()._g(name).astype(np.float32)

    def _layer(self, l):
        return {k: v.astype(np.float32) for k, v in super()._layer(l).items()}

    def R(self, x):
        return nx.round_to(x, self.dt).astype(np.float32)


def spread(name, n_layers, wseed, iseed):
    cfg = synth.preset(name, n_layers=n_layers)
    w = synth.make_weights(cfg, wseed)
    ids, mask = synth.make_inputs(cfg, iseed)
    ref = OracleModel(cfg, w).forward(ids, mask).logits_f64
    lo = Float32Oracle(cfg, w).forward(ids, mask).logits_f64
    fin = np.isfinite(ref) & np.isfinite(lo)
    return float(np.abs(lo[fin] - ref[fin]).max() / np.abs(ref[fin]).max())


ENTRIES = {
    ("encoder_clamp_1024", "2"): lambda: spread("encoder_clamp_1024", 2, 5, 0),
    ("encoder_clamp_1024", "4"): lambda: spread("encoder_clamp_1024", 4, 5, 0),
    ("encoder_clamp_1024", "8"): lambda: spread("encoder_clamp_1024", 8, 5, 0),
    ("encoder_clamp_1024", "24"): lambda: spread("encoder_clamp_1024", 24, 5, 0),
    # every one of the 2048 positions at full depth
    ("decoder_4096", "32_all"): lambda: spread("decoder_4096", 32, 11, 0),
}


def main(only=None):
    """Recompute every entry, or (only = "workload/key") one of them, and
    write depth_spread.json."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "depth_spread.json")
    out = {"encoder_clamp_1024": {}, "decoder_4096": {}}
    if only and os.path.exists(path):
        with open(path) as fh:
            out.update(json.load(fh))
    for (w, k), fn in ENTRIES.items():
        if only and f"{w}/{k}" != only:
            continue
        out[w][k] = fn()
        print(w, k, out[w][k], flush=True)
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)


if __name__ == "__main__":
    main(sys.argv[1] if len(sys.argv) > 1 else None)
