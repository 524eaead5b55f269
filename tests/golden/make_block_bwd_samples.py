"""Writes block_bwd_B1_T32_S1024_samples.json: expected values of the block
backward at the benchmark's block size (B1 T32 S1024, C 1152, 16 heads, MLP
4608, bf16 weights, pre-LN GELU block), computed by the fp64 oracle
(oracle.st_block_bwd) on the seeded synthetic inputs (synth.block_inputs of
the block workload, dy ~ N(0, 1) from numpy's default_rng(seed + 1)).

The full-size oracle takes many CPU minutes, so its results are sampled and
stored: 8 rows of dx (whole rows of C values) and 128 entries of every weight
gradient, at seeded positions.  Run from the repository root:

    python tests/golden/make_block_bwd_samples.py
"""
import json
import sys
from pathlib import Path

import numpy as np

ROOT = Path(__file__).resolve().parents[2]
sys.path.insert(0, str(ROOT))

import oracle  # noqa: E402
import synth  # noqa: E402

OUT = Path(__file__).resolve().parent / "block_bwd_B1_T32_S1024_samples.json"


def sample_positions(w, n_rows=8, n_entries=128, seed=77):
    """Seeded sample: token rows (b, t, s) of dx and (out, in) entries per weight
    gradient (stored [out][in] layout)."""
    rng = np.random.default_rng(seed)
    C, F = w.C, w.F
    rows = [[int(rng.integers(w.B)), int(rng.integers(w.T)), int(rng.integers(w.S))] for _ in range(n_rows)]
    shapes = {"wqkv_s": (3 * C, C), "wo_s": (C, C), "wqkv_t": (3 * C, C), "wo_t": (C, C), "w1": (F, C),
              "w2": (C, F)}
    entries = {n: [[int(rng.integers(a)), int(rng.integers(b))] for _ in range(n_entries)]
               for n, (a, b) in shapes.items()}
    return rows, entries


def main():
    w = synth.WORKLOADS["block_bf16_B1_T32_S1024"]
    x, p = synth.block_inputs(w)
    po = {n: (None if v is None else (v.T if n.startswith("w") else v)) for n, v in p.items()}
    dy = np.random.default_rng(w.seed + 1).standard_normal((w.B, w.S, w.T, w.C), dtype=np.float32)
    dx, g = oracle.st_block_bwd(x, po, w.H, dy)
    rows, entries = sample_positions(w)
    out = {
        "what": "oracle.st_block_bwd at B1 T32 S1024 C1152 H16 F4608 (bf16 weights, pre-LN GELU), sampled",
        "dy": "numpy default_rng(seed + 1).standard_normal((B, S, T, C), float32), seed of the block workload",
        "dx_rows": rows,
        "dx": [[float(v) for v in dx[b, t, s]] for b, t, s in rows],
        "dx_max_abs": float(np.abs(dx).max()),
        "grads": {},
    }
    for n, pos in entries.items():
        gs = g[n].T  # the oracle's [in, out] -> stored [out][in]
        out["grads"][n] = {"pos": pos, "val": [float(gs[i, j]) for i, j in pos],
                           "max_abs": float(np.abs(gs).max())}
    OUT.write_text(json.dumps(out))
    print(f"wrote {OUT} ({OUT.stat().st_size} bytes)")


if __name__ == "__main__":
    main()
