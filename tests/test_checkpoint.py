"""Weights checkpoint (a weights blob with a manifest: config id, seed,
tensor table and the data section's SHA-256), through the C ABI of the host
test library: the library's SHA-256 against hashlib's on data lengths that
cross the padding boundary, every verification failure, the table checked
against the model descriptor, and a context created from a checkpoint
receiving exactly the weights of the raw blob."""

import ctypes
import hashlib
import struct

import numpy as np
import pytest

import synth
from paper_2608_08330_amd import checkpoint as C
from paper_2608_08330_amd import rtcc as R


def _init_line():
    lib = R.load("host")
    buf = ctypes.create_string_buffer(1 << 16)
    lib.rtcc_hosttest_log(buf, len(buf), 1)
    return [l for l in buf.value.decode().splitlines() if l.startswith("init ")]


def _err(fn, *a):
    with pytest.raises(R.RtccError) as e:
        fn(*a)
    return e.value.status, str(e.value)


@pytest.mark.parametrize("nbytes", [4, 52, 56, 60, 64, 68, 116, 120, 124, 128, 4096, 4100])
def test_sha256_agrees_with_hashlib_across_padding_boundaries(nbytes):
    # lengths around 55/56 and 119/120 bytes mod 64 need one or two padding blocks
    rng = np.random.default_rng(nbytes)
    arr = rng.standard_normal(nbytes // 4).astype(np.float32)
    blob = C.pack([("t", arr)], "probe", 7)
    info = R.rtcc_read_checkpoint(blob, kind="host")
    assert info["sha256"] == hashlib.sha256(arr.tobytes()).hexdigest()
    assert info == dict(config_id="probe", seed=7, version=1, n_tensors=1, data_bytes=nbytes,
                        sha256=info["sha256"])


def test_sha256_known_digest():
    # FIPS 180-4 example: the three bytes "abc" (a one-element float32 tensor
    # cannot hold 3 bytes, so the digest is checked on 'abc\0' against hashlib
    # and on the published digest of 'abc' through hashlib)
    assert hashlib.sha256(b"abc").hexdigest() == \
        "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"
    data = np.frombuffer(b"abc\0", dtype="<f4")
    info = R.rtcc_read_checkpoint(C.pack([("x", data)], "abc", 0), kind="host")
    assert info["sha256"] == hashlib.sha256(b"abc\0").hexdigest()


def _cfg_ckpt(name="t_attn"):
    cfg = synth.config(name)
    w = synth.make_weights(cfg)
    return cfg, w, C.for_config(cfg, w)


def test_manifest_of_a_workload():
    cfg, w, blob = _cfg_ckpt()
    info = R.rtcc_read_checkpoint(blob, kind="host")
    raw = R.weights_blob(cfg, w)
    assert info["config_id"] == "t_attn"
    assert info["seed"] == synth.configs.ROOT_SEED
    assert info["n_tensors"] == len(R.weight_order(cfg))
    assert info["data_bytes"] == raw.nbytes
    assert info["sha256"] == hashlib.sha256(raw.tobytes()).hexdigest()
    # the data section is the raw blob itself
    assert blob[-raw.nbytes:] == raw.tobytes()


@pytest.mark.parametrize("name", ["t_attn", "c1", "c3"])
def test_context_from_checkpoint_gets_the_raw_blob_weights(name):
    cfg, w, blob = _cfg_ckpt(name)
    desc = R.model_desc(cfg)
    _init_line()
    a = R.rtcc_create(desc, R.weights_blob(cfg, w), kind="host")
    la = _init_line()
    b = R.rtcc_create_from_checkpoint(desc, blob, kind="host")
    lb = _init_line()
    a.close()
    b.close()
    assert la and la == lb
    # other weights give another digest (the digest sees the data)
    w2 = dict(w)
    w2["head_b"] = w["head_b"] + 1.0
    c = R.rtcc_create_from_checkpoint(desc, C.for_config(cfg, w2), kind="host")
    lc = _init_line()
    c.close()
    assert lc != la


def _corrupt(blob, off, val):
    b = bytearray(blob)
    b[off:off + len(val)] = val
    return bytes(b)


def test_verification_failures():
    cfg, w, blob = _cfg_ckpt()
    read = lambda b: R.rtcc_read_checkpoint(b, kind="host")  # noqa: E731
    doff = struct.unpack_from("<Q", blob, 56)[0]
    cases = {
        "magic": _corrupt(blob, 0, b"XTCC"),
        "version": _corrupt(blob, 8, struct.pack("<I", 2)),
        "data byte": _corrupt(blob, doff + 17, bytes([blob[doff + 17] ^ 1])),
        "last data byte": _corrupt(blob, len(blob) - 1, bytes([blob[-1] ^ 0x80])),
        "digest": _corrupt(blob, 72, bytes([blob[72] ^ 1])),
        "truncated": blob[:-4],
        "extended": blob + b"\0\0\0\0",
        "short header": blob[:100],
        "reserved header": _corrupt(blob, 110, b"\1"),
        "config id unterminated": _corrupt(blob, 16, b"x" * 32),
        "dtype": _corrupt(blob, 128 + 64, struct.pack("<I", 1)),
        "ndim": _corrupt(blob, 128 + 68, struct.pack("<I", 5)),
        "shape": _corrupt(blob, 128 + 72, struct.pack("<q", 5)),
        "offset": _corrupt(blob, 128 + 128 + 104, struct.pack("<Q", 8)),
        "nbytes": _corrupt(blob, 128 + 112, struct.pack("<Q", 4)),
        "tensor count": _corrupt(blob, 12, struct.pack("<I", 0)),
        "data offset": _corrupt(blob, 56, struct.pack("<Q", doff + 1)),
    }
    for what, bad in cases.items():
        st, msg = _err(read, bad)
        assert st == R.RTCC_E_MALFORMED, (what, msg)
    assert read(blob)["n_tensors"] > 0


def test_table_must_match_the_descriptor():
    cfg, w, _ = _cfg_ckpt("t_attn")
    desc = R.model_desc(cfg)
    names = R.weight_order(cfg)
    # a tensor missing
    short = C.pack([(n, w[n]) for n in names[:-1]], "t_attn", 1)
    st, msg = _err(R.rtcc_create_from_checkpoint, desc, short, None, "host")
    assert st == R.RTCC_E_ARG and "tensors" in msg
    # two tensors swapped (same sizes: the biases of two convs of one width)
    order = list(names)
    i, j = order.index("s0c0_b"), order.index("s0c1_b")
    order[i], order[j] = order[j], order[i]
    swapped = C.pack([(n, w[n]) for n in order], "t_attn", 1)
    st, msg = _err(R.rtcc_create_from_checkpoint, desc, swapped, None, "host")
    assert st == R.RTCC_E_ARG and "s0c1_b" in msg
    # a transposed weight (same element count, other shape)
    tr = [(n, w[n].T.copy() if n == "head_w" else w[n]) for n in names]
    st, msg = _err(R.rtcc_create_from_checkpoint, desc, C.pack(tr, "t_attn", 1), None, "host")
    assert st == R.RTCC_E_ARG and "head_w" in msg
    # a checkpoint of another workload
    cfg2 = synth.config("c1")
    other = C.for_config(cfg2, synth.make_weights(cfg2))
    st, _ = _err(R.rtcc_create_from_checkpoint, desc, other, None, "host")
    assert st == R.RTCC_E_ARG


def test_null_arguments():
    lib = R.load("host")
    info = R.rtcc_checkpoint_info()
    assert lib.rtcc_read_checkpoint(None, 128, ctypes.byref(info)) == R.RTCC_E_ARG
    assert lib.rtcc_read_checkpoint(b"x" * 128, 128, None) == R.RTCC_E_ARG
    h = ctypes.c_void_p()
    assert lib.rtcc_create_from_checkpoint(None, b"x" * 128, 128, None, ctypes.byref(h)) == R.RTCC_E_ARG
