"""A GPU context created from a weights checkpoint gives bit-identical
tensors and detections to one created from the raw weights blob."""

import numpy as np
import pytest

import synth
from paper_2608_08330_amd import checkpoint as C
from paper_2608_08330_amd import rtcc as R
from tests.helpers import make_ctx, run_frame

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["c1", "t_attn"])
def test_checkpoint_context_matches_raw_blob_context(name):
    cfg = synth.config(name)
    fr = synth.make_frame(cfg)
    a = make_ctx(cfg, fr)
    o = R.rtcc_runtime_opts()
    o.exec = R.RTCC_EXEC_PER_BRANCH_STREAMS
    o.premature_tol_s = 1e-6
    desc = R.model_desc(cfg, max(len(p) for p in fr["points"]))
    b = R.rtcc_create_from_checkpoint(desc, C.for_config(cfg, fr["weights"]), o)
    try:
        da = run_frame(a, fr)
        db = run_frame(b, fr)
        assert da["count"] == db["count"]
        assert np.array_equal(da["anchor_idx"], db["anchor_idx"])
        assert np.array_equal(da["boxes"], db["boxes"])
        assert np.array_equal(da["scores"], db["scores"])
        for tid in (R.RTCC_T_HEAD, R.RTCC_T_FUSED):
            ta = R.rtcc_get_tensor(a, tid, 0, np.uint8)
            tb = R.rtcc_get_tensor(b, tid, 0, np.uint8)
            assert np.array_equal(ta, tb), tid
    finally:
        a.close()
        b.close()
