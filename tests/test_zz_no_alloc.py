"""The allocation-free NMS entry point against rtcc_rotated_nms: the same
kept records, bit for bit, on two calls in a row (the second with fewer
records, so stale scratch contents of the first would show), on the null
stream and on a stream of the caller; and the size limits."""

import math
import sys

import numpy as np
import pytest

from paper_2608_08330_amd import rtcc as R

pytestmark = pytest.mark.gpu


def _scene(seed, n, spread):
    rng = np.random.default_rng(seed)
    rec = np.zeros((n, 9), dtype=np.float32)
    c = rng.uniform(-spread, spread, (max(1, n // 30), 2))
    rec[:, 0:2] = c[rng.integers(0, len(c), n)] + rng.normal(0, 1.0, (n, 2))
    rec[:, 2] = -1.0
    rec[:, 3] = rng.uniform(1.2, 2.2, n)
    rec[:, 4] = rng.uniform(3.0, 5.0, n)
    rec[:, 5] = 1.5
    rec[:, 6] = rng.uniform(-math.pi, math.pi, n)
    rec[:, 7] = rng.uniform(0.3, 1.0, n)
    rec[:, 8] = np.sort(rng.choice(10 * n, n, replace=False)).astype(np.int32).view(np.float32)
    return rec


def _run(fn, rec, cap, thr, **kw):
    import torch
    d_rec = torch.from_numpy(rec).to("cuda")
    d_out = torch.full((min(len(rec), cap), 9), -7.0, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    kept = fn(d_rec.data_ptr(), len(rec), cap, thr, d_out.data_ptr(), **kw)
    torch.cuda.synchronize()
    return d_out[:kept].cpu().numpy()


@pytest.mark.parametrize("use_stream", [False, True])
def test_noalloc_matches_allocating_entry_point(use_stream):
    import torch
    kw = {}
    if use_stream:
        st = torch.cuda.Stream()
        kw["stream"] = st.cuda_stream
    for seed, n, spread, cap, thr in ((1, 3000, 40.0, 1500, 0.15), (2, 700, 15.0, 4096, 0.15)):
        print("noalloc case seed=%d n=%d cap=%d stream=%s" % (seed, n, cap, use_stream), flush=True)
        sys.stdout.flush()
        rec = _scene(seed, n, spread)
        want = _run(R.rtcc_rotated_nms, rec, cap, thr)
        got = _run(R.rtcc_rotated_nms_noalloc, rec, cap, thr, **kw)
        assert len(want) > 0
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_noalloc_limits_and_empty():
    import torch
    d = torch.zeros((4, 9), dtype=torch.float32, device="cuda")
    for n, cap in ((131073, 16), (4, 4097), (4, 0), (-1, 16)):
        with pytest.raises(R.RtccError) as e:
            R.rtcc_rotated_nms_noalloc(d.data_ptr(), n, cap, 0.15, d.data_ptr())
        assert e.value.status == R.RTCC_E_ARG
    assert R.rtcc_rotated_nms_noalloc(0, 0, 16, 0.15, d.data_ptr()) == 0
