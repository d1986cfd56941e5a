"""Weights checkpoint writer: the weights blob of ``rtcc_create`` with a
manifest (config id, seed, tensor table, SHA-256 of the data), in the layout
``include/rtcc.h`` documents beside ``rtcc_read_checkpoint``.  The library
verifies and loads it (``rtcc_create_from_checkpoint``).

  python -m paper_2608_08330_amd.checkpoint --config c5 --out c5.rtccw
"""

import argparse
import hashlib
import os
import struct
import sys

import numpy as np

MAGIC = b"RTCCWGT\0"
VERSION = 1
HEADER_BYTES = 128
ENTRY_BYTES = 128


def pack(tensors, config_id, seed):
    """Checkpoint bytes of ``tensors``: (name, float32 array) pairs in data
    order."""
    cid = config_id.encode()
    if len(cid) > 31:
        raise ValueError("config id longer than 31 bytes")
    table, data, off = [], [], 0
    for name, arr in tensors:
        a = np.ascontiguousarray(arr, dtype="<f4")
        nm = name.encode()
        if not 0 < len(nm) <= 63 or not 1 <= a.ndim <= 4:
            raise ValueError("tensor %r: name length or rank out of range" % name)
        shape = list(a.shape) + [0] * (4 - a.ndim)
        table.append(nm.ljust(64, b"\0") + struct.pack("<II4qQQ8x", 0, a.ndim, *shape, off, a.nbytes))
        data.append(a.tobytes())
        off += a.nbytes
    body = b"".join(data)
    data_offset = (HEADER_BYTES + ENTRY_BYTES * len(table) + 63) // 64 * 64
    header = (MAGIC + struct.pack("<II", VERSION, len(table)) + cid.ljust(32, b"\0")
              + struct.pack("<QQQ", int(seed), data_offset, len(body)) + hashlib.sha256(body).digest())
    header = header.ljust(HEADER_BYTES, b"\0")
    head = header + b"".join(table)
    return head.ljust(data_offset, b"\0") + body


def for_config(cfg, weights):
    """Checkpoint of a workload's seeded network (the synth draw): config id
    = the workload's name, seed = the root seed of the synthetic inputs."""
    from synth.configs import ROOT_SEED
    from synth.configs import network_layers
    return pack([(name, weights[name]) for name, _shape, _fan in network_layers(cfg)], cfg["name"], ROOT_SEED)


def main(argv=None):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import synth
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", required=True)
    ap.add_argument("--out", required=True)
    a = ap.parse_args(argv)
    cfg = synth.config(a.config)
    with open(a.out, "wb") as f:
        f.write(for_config(cfg, synth.make_weights(cfg)))
    return 0


if __name__ == "__main__":
    sys.exit(main())
