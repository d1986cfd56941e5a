"""Plain, slow CPU oracle of the RTCC fork-join detector path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the HIP path; both consume the seeded inputs of ``synth/``.

Modules
  bf16      round-to-nearest-even to bfloat16, written out from the format
  network   pillarization, point-feature net, backbone, upsampling, pose
            warp, fusion, head and box decode (fp64 unless a storage point
            is bf16)
  schedule  single-stream release-aware execution model, RTCC and barrier
  uplink    slot-level uplink emulation producing branch arrival times,
            with round robin, proportional fair and the five causal
            evaluation schedulers
  ofdma     the evaluation's OFDMA channel (mobility, path loss,
            blockage, fading), DAG upward rank and the paired
            measured-DAG trial in integer nanoseconds
  nms       rotated bird's-eye-view IoU and greedy non-maximum suppression

Parity status: every function is pinned by tests under ``tests/`` against
closed forms, brute force or library routines, except the composition of the
whole network on a real frame, which is "parity unpinned" beyond the
composition of its pinned parts (no trained weights or worked example exist).
"""
