"""Profiled-DAG latency model used to predict the RTCC gain of a trace.

Single non-preemptive compute stream (Sec. III-B): encoders served in (r_k,
k) order start at max(r_k, GPU free) and hold the stream for their profiled
service time (eqs. rtcc_encoder_start, rtcc_encoder_finish,
rtcc_gpu_availability); the post-join subgraph follows.  RTCC: r = a;
Barrier: r = max(a).  The predicted gain T_B - T_R equals the encoder work
RTCC finishes before the last arrival.
"""

import numpy as np

from . import rtcc as R


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


def dagrank_weights(c_enc_ns, c_post_ns, kind="gpu"):
    """DAGRank priorities omega_k (Sec. V-A2): the upward rank of every
    encoder in the profiled DAG (encoders E_0..E_{K-1}, each feeding the
    post-join chain P_0 -> P_1 -> ...), from the library's rtcc_upward_rank,
    divided by the largest encoder rank."""
    K, m = len(c_enc_ns), len(c_post_ns)
    cost = [int(c) for c in c_enc_ns] + [int(c) for c in c_post_ns]
    edges = [(k, K) for k in range(K)] + [(K + i, K + i + 1) for i in range(m - 1)]
    rank = R.rtcc_upward_rank(cost, edges, kind=kind)[:K]
    top = float(rank.max())
    return [float(v) / top for v in rank]


def paired_latency_ns(arrival_ns, c_enc_ns, c_post_ns, kind="gpu"):
    """(T_R, T_B, W_pre) in integer nanoseconds from the library's
    single-stream model: RTCC (r = a) and barrier (r = A) on the same
    arrival vector; W_pre is the RTCC encoder work done before A."""
    post = int(sum(int(c) for c in c_post_ns))
    t_r, w_pre, _ = R.rtcc_schedule_model(arrival_ns, c_enc_ns, post, R.RTCC_MODE_RELEASE, kind=kind)
    t_b, _, _ = R.rtcc_schedule_model(arrival_ns, c_enc_ns, post, R.RTCC_MODE_BARRIER, kind=kind)
    return t_r, t_b, w_pre
