"""Release-aware single-stream execution model (test infrastructure only).

The edge GPU is one non-preemptive, work-conserving compute stream
(Sec. III-B).  Encoder E_k may start no earlier than its release r_k
(eq. encoder_release), and a release rule must respect r_k >= a_k
(eq. release_causality).  Released encoders are served in the order of
(r_k, k) (Sec. IV-C ready queue); with g_0 = 0 the j-th served encoder
starts at max(r, g_{j-1}), finishes c later and frees the stream
(eqs. rtcc_encoder_start, rtcc_encoder_finish, rtcc_gpu_availability).  The
post-join subgraph runs after all K encoders, node after node in
topological order (Sec. IV-D), and its last node ends the latency
T = f_o (eq. full_latency).

RTCC releases each encoder at its own arrival (r_k = a_k); the barrier
baseline releases every encoder at the final arrival A = max_k a_k
(Sec. V, compared execution rule).
"""

import numpy as np


def execute(release, c_enc, c_post, h2d=None):
    """Run the single-stream model for a release vector.

    release  r_k per agent
    c_enc    encoder service times c_{E_k}
    c_post   service times of the post-join nodes, in topological order
    h2d      optional host-to-device copy time per agent on a separate
             transfer resource (one copy at a time, in release order); the
             encoder of agent k then also waits for its copy to finish

    Returns dict(order, start, finish, T, g) with start / finish per agent
    and T the finish time of the last post-join node.
    """
    r = np.asarray(release, dtype=np.float64)
    c = np.asarray(c_enc, dtype=np.float64)
    K = len(r)
    order = sorted(range(K), key=lambda k: (r[k], k))
    start = np.zeros(K)
    finish = np.zeros(K)
    ready = r.copy()
    if h2d is not None:
        h = np.asarray(h2d, dtype=np.float64)
        link = 0.0
        for k in order:
            s = max(r[k], link)
            link = s + h[k]
            ready[k] = link
    g = 0.0
    for k in order:
        start[k] = max(ready[k], g)
        finish[k] = start[k] + c[k]
        g = finish[k]
    T = g
    for cv in c_post:
        T = T + float(cv)
    return dict(order=order, start=start, finish=finish, T=T, g=g)


def rtcc(a, c_enc, c_post, h2d=None):
    """RTCC: r_k = a_k."""
    return execute(a, c_enc, c_post, h2d)


def barrier(a, c_enc, c_post, h2d=None):
    """Barrier: every encoder released at A = max_k a_k."""
    A = float(np.max(a))
    return execute(np.full(len(a), A), c_enc, c_post, h2d)


def w_pre(a, c_enc, c_post=()):
    """Encoder work that RTCC performs before the final arrival A: the total
    length of [s_k, f_k) intersected with [0, A) over all encoders."""
    A = float(np.max(a))
    res = rtcc(a, c_enc, c_post)
    s, f = res["start"], res["finish"]
    return float(np.sum(np.clip(np.minimum(f, A) - s, 0.0, None)))


def overlap_window(a):
    """Usable overlap window: time between the first and the last arrival."""
    return float(np.max(a) - np.min(a))


def execute_int(release, c_enc, c_post):
    """The same single-stream model on integer times (e.g. nanoseconds), in
    Python integers, so that every start, finish and latency is exact.
    Returns dict(order, start, finish, T, g) as :func:`execute`."""
    r = [int(v) for v in release]
    c = [int(v) for v in c_enc]
    K = len(r)
    order = sorted(range(K), key=lambda k: (r[k], k))
    start = [0] * K
    finish = [0] * K
    g = 0
    for k in order:
        start[k] = max(r[k], g)
        finish[k] = start[k] + c[k]
        g = finish[k]
    return dict(order=order, start=start, finish=finish, T=g + sum(int(v) for v in c_post), g=g)


def paired_int(a, c_enc, c_post):
    """RTCC and barrier on the same integer arrival vector: returns (T_R,
    T_B, W_pre) with W_pre the RTCC encoder work inside [0, A)."""
    a = [int(v) for v in a]
    A = max(a)
    r = execute_int(a, c_enc, c_post)
    b = execute_int([A] * len(a), c_enc, c_post)
    w = sum(max(0, min(f, A) - s) for s, f in zip(r["start"], r["finish"]))
    return r["T"], b["T"], w
