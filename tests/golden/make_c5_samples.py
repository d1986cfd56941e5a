"""Write tests/golden/c5_oracle_samples.npz: sampled fp64-oracle outputs of
the c5 frame (8 agents x 100,000 points, 512 x 512 BEV, bf16, attention).

Calls only synth/ (seeded inputs) and oracle/ (the fp64 reference).  The
full-size GPU parity test compares the HIP path against these samples; the
cheap parts (pillar lists, canvas) it recomputes with the oracle directly.

Usage: python tests/golden/make_c5_samples.py   (about a minute on 8 cores)
"""

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import synth  # noqa: E402
from oracle import network as N  # noqa: E402
from oracle.bf16 import round_bf16  # noqa: E402

SLOT_CELLS = 128      # sampled cells per agent slot
FUSED_CELLS = 512     # sampled cells of the fused map
HEAD_CELLS = 4096     # sampled cells of the head output


def bf16_bits(x):
    """Exact bfloat16 values (float64) -> uint16 bit patterns."""
    x32 = np.asarray(round_bf16(x), dtype=np.float32)
    return (x32.view(np.uint32) >> 16).astype(np.uint16)


def main():
    cfg = synth.config("c5")
    fr = synth.make_frame(cfg)
    out = N.forward(fr)
    H2, W2 = N.feature_grid(cfg)
    rng = np.random.default_rng(2608)
    res = {}
    for k in range(cfg["K"]):
        cells = rng.choice(H2 * W2, SLOT_CELLS, replace=False)
        slot = out["enc"][k]["slot"].reshape(H2 * W2, -1)
        res["slot_cells_%d" % k] = cells.astype(np.int32)
        res["slot_%d" % k] = bf16_bits(slot[cells])
    cells = rng.choice(H2 * W2, FUSED_CELLS, replace=False)
    res["fused_cells"] = cells.astype(np.int32)
    res["fused"] = bf16_bits(out["fused"].reshape(H2 * W2, -1)[cells])
    res["fused_absmax"] = np.float64(np.max(np.abs(out["fused"])))
    cells = rng.choice(H2 * W2, HEAD_CELLS, replace=False)
    Z = out["head"].reshape(H2 * W2, 16)
    res["head_cells"] = cells.astype(np.int32)
    res["head"] = Z[cells].astype(np.float64)
    res["head_absmax"] = np.float64(np.max(np.abs(Z)))
    det = out["det"]
    res["logits"] = det["logits"].astype(np.float32)
    res["det_anchor_idx"] = det["anchor_idx"].astype(np.int64)
    res["det_boxes"] = det["boxes"]
    res["det_scores"] = det["scores"]
    for k in range(cfg["K"]):
        res["slot_absmax_%d" % k] = np.float64(np.max(np.abs(out["enc"][k]["slot"])))
    path = os.path.join(HERE, "c5_oracle_samples.npz")
    np.savez_compressed(path, **res)
    print("wrote", path, os.path.getsize(path), "bytes;", len(det["anchor_idx"]), "detections")


if __name__ == "__main__":
    main()
