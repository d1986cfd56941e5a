"""Profiled-DAG latency model used to predict the RTCC gain of a trace.

Single non-preemptive compute stream (Sec. III-B): encoders served in (r_k,
k) order start at max(r_k, GPU free) and hold the stream for their profiled
service time (eqs. rtcc_encoder_start, rtcc_encoder_finish,
rtcc_gpu_availability); the post-join subgraph follows.  RTCC: r = a;
Barrier: r = max(a).  The predicted gain T_B - T_R equals the encoder work
RTCC finishes before the last arrival.
"""

import numpy as np


def completion(release, c_enc, c_post):
    r = np.asarray(release, dtype=np.float64)
    c = np.asarray(c_enc, dtype=np.float64)
    free = 0.0
    for k in sorted(range(len(r)), key=lambda k: (r[k], k)):
        free = max(r[k], free) + c[k]
    return free + float(c_post)


def predicted_gain(arrival, c_enc, c_post):
    a = np.asarray(arrival, dtype=np.float64)
    t_rtcc = completion(a, c_enc, c_post)
    t_barrier = completion(np.full(len(a), a.max()), c_enc, c_post)
    return t_barrier - t_rtcc
