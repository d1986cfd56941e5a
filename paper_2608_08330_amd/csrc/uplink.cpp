// Host-side models around the release controller: the slot-level uplink
// emulation that turns per-slot RB rates into branch completion slots, the
// single-stream latency model of the profiled DAG, and the DAG upward rank.
//
// Uplink (Sec. III-A, IV-B): Q_k[1] = B_k; in slot t the eligible agents
// have Q_k[t] > 0 and t >= l_k (eq. eligible_set); every RB goes to one
// eligible agent by the causal policy (eqs. rb_orthogonality,
// pluggable_scheduler, evaluation_schedulers, evaluation_scores, ties to
// the smallest index); d_k[t] = Delta * (sum of the rates of the RBs k
// holds, ascending RB order) (eq. slot_payload); Q_k[t+1] = max(0, Q_k[t] -
// d_k[t]) (eq. queue_evolution); the slot in which Q_k reaches zero is the
// completion slot, a_k = slot * Delta (eqs. branch_arrival,
// completion_event).  Every RB of a slot is decided from the slot-start
// state (the causal history of eq. causal_history).
//
// Latency model (Sec. III-B, IV-C, eqs. rtcc_encoder_start,
// rtcc_encoder_finish, rtcc_gpu_availability, full_latency): one
// non-preemptive stream serves the released encoders in (r_k, k) order,
// each from max(r_k, stream free); the post-join subgraph follows.  RTCC
// releases at r_k = a_k, the barrier at r_k = A = max_k a_k.  Integer
// nanoseconds keep every sum exact.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <new>
#include <string>
#include <vector>

#include "../../include/rtcc.h"

namespace rtcc {
void set_thread_error(const std::string &msg);
}

namespace {

constexpr int64_t kTimeLimit = int64_t(1) << 60;  // bound on every time so sums cannot overflow

rtcc_status fail(const std::string &msg) {
    rtcc::set_thread_error(msg);
    return RTCC_E_ARG;
}

template <class F>
rtcc_status guarded(F &&f) {
    try {
        return f();
    } catch (const std::bad_alloc &) {
        rtcc::set_thread_error("host allocation failed");
        return RTCC_E_NOMEM;
    } catch (...) {
        rtcc::set_thread_error("internal error");
        return RTCC_E_INTERNAL;
    }
}

rtcc_status check_uplink(const rtcc_uplink_desc *d, const double *rates, const double *payload,
                         const int32_t *avail, const int32_t *completion) {
    if (!d) return fail("desc is NULL");
    if (d->slots < 1 || d->agents < 1 || d->rbs < 1) return fail("slots, agents and rbs must be >= 1");
    if (double(d->slots) * double(d->agents) * double(d->rbs) > 1e10) return fail("slots * agents * rbs too large");
    if (!(d->slot_s > 0.0) || !std::isfinite(d->slot_s)) return fail("slot_s must be finite and > 0");
    if (d->policy < RTCC_SCHED_MAXRATE || d->policy > RTCC_SCHED_PROPORTIONAL_FAIR) return fail("unknown policy");
    if (!rates || !payload || !completion) return fail("NULL rates, payload or completion_slot");
    const size_t n = size_t(d->slots) * size_t(d->agents) * size_t(d->rbs);
    for (size_t i = 0; i < n; ++i)
        if (!(rates[i] >= 0.0) || !std::isfinite(rates[i])) return fail("rates must be finite and >= 0");
    for (int k = 0; k < d->agents; ++k) {
        if (!(payload[k] > 0.0) || !std::isfinite(payload[k])) return fail("payload_bits must be finite and > 0");
        if (avail && avail[k] < 1) return fail("avail_slot must be >= 1");
    }
    if (d->policy == RTCC_SCHED_WEIGHTED_RATE) {
        if (!d->agent_weight) return fail("agent_weight is NULL");
        for (int k = 0; k < d->agents; ++k)
            if (!std::isfinite(d->agent_weight[k])) return fail("agent_weight must be finite");
    }
    if (d->policy == RTCC_SCHED_PROPORTIONAL_FAIR) {
        if (!(d->pf_window >= 1.0) || !std::isfinite(d->pf_window)) return fail("pf_window must be >= 1");
        if (!(d->pf_init_rate > 0.0) || !std::isfinite(d->pf_init_rate)) return fail("pf_init_rate must be > 0");
    }
    return RTCC_OK;
}

// Priority score of agent k on an RB of rate r (eq. evaluation_scores).
inline double score(const rtcc_uplink_desc &d, int k, double r, double q) {
    switch (d.policy) {
        case RTCC_SCHED_MAXWEIGHT: return q * r;
        case RTCC_SCHED_EARLIEST_RELEASE: {
            const double b = d.slot_s * r;  // payload the RB can deliver in this slot
            return b > 0.0 ? -q / b : -std::numeric_limits<double>::infinity();
        }
        case RTCC_SCHED_WEIGHTED_RATE: return d.agent_weight[k] * r;
        default: return r;  // MaxRate
    }
}

rtcc_status emulate(const rtcc_uplink_desc &d, const double *rates, const double *payload, const int32_t *avail,
                    int32_t *completion, int32_t *rb_agent) {
    const int T = d.slots, K = d.agents, F = d.rbs;
    std::vector<double> Q(payload, payload + K), avg(K, d.pf_init_rate);
    std::vector<int32_t> pick(F);
    std::vector<char> eligible(K);
    std::fill(completion, completion + K, 0);
    if (rb_agent) std::fill(rb_agent, rb_agent + size_t(T) * F, -1);
    int remaining = K, rr_last = -1;
    for (int t = 1; t <= T && remaining > 0; ++t) {
        const double *R = rates + size_t(t - 1) * K * F;  // [K][F] of slot t
        int any = 0;
        for (int k = 0; k < K; ++k) {
            eligible[k] = Q[k] > 0.0 && (!avail || t >= avail[k]);
            any |= eligible[k];
        }
        std::fill(pick.begin(), pick.end(), -1);
        if (any) {
            for (int f = 0; f < F; ++f) {
                int best = -1;
                if (d.policy == RTCC_SCHED_ROUND_ROBIN) {
                    for (int step = 1; step <= K; ++step) {
                        const int k = (rr_last + step) % K;
                        if (eligible[k]) {
                            best = k;
                            break;
                        }
                    }
                    rr_last = best;
                } else {
                    double best_v = 0.0;
                    for (int k = 0; k < K; ++k) {
                        if (!eligible[k]) continue;
                        const double r = R[size_t(k) * F + f];
                        const double v = d.policy == RTCC_SCHED_PROPORTIONAL_FAIR ? r / avg[k] : score(d, k, r, Q[k]);
                        if (best < 0 || v > best_v) {
                            best = k;
                            best_v = v;
                        }
                    }
                }
                pick[f] = best;
            }
        }
        for (int k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int f = 0; f < F; ++f)
                if (pick[f] == k) acc += R[size_t(k) * F + f];
            if (d.policy == RTCC_SCHED_PROPORTIONAL_FAIR)
                avg[k] = (1.0 - 1.0 / d.pf_window) * avg[k] + acc / d.pf_window;
            const double sent = d.slot_s * acc;
            const double next = std::max(0.0, Q[k] - sent);
            if (Q[k] > 0.0 && next == 0.0) {
                completion[k] = t;
                --remaining;
            }
            Q[k] = next;
        }
        if (rb_agent) std::copy(pick.begin(), pick.end(), rb_agent + size_t(t - 1) * F);
    }
    return RTCC_OK;
}

}  // namespace

extern "C" {

rtcc_status rtcc_uplink_emulate(const rtcc_uplink_desc *desc, const double *rates, const double *payload_bits,
                                const int32_t *avail_slot, int32_t *completion_slot, int32_t *rb_agent) {
    return guarded([&] {
        rtcc_status s = check_uplink(desc, rates, payload_bits, avail_slot, completion_slot);
        if (s != RTCC_OK) return s;
        return emulate(*desc, rates, payload_bits, avail_slot, completion_slot, rb_agent);
    });
}

rtcc_status rtcc_schedule_model(int32_t agents, const int64_t *arrival_ns, const int64_t *encoder_ns,
                                int64_t post_ns, int32_t mode, int64_t *latency_ns, int64_t *pre_arrival_ns,
                                int64_t *start_ns) {
    return guarded([&] {
        if (agents < 1) return fail("agents must be >= 1");
        if (!arrival_ns || !encoder_ns || !latency_ns) return fail("NULL arrival_ns, encoder_ns or latency_ns");
        if (mode != RTCC_MODE_RELEASE && mode != RTCC_MODE_BARRIER) return fail("unknown mode");
        if (post_ns < 0 || post_ns >= kTimeLimit) return fail("post_ns out of range");
        int64_t A = 0;
        for (int k = 0; k < agents; ++k) {
            if (arrival_ns[k] < 0 || arrival_ns[k] >= kTimeLimit || encoder_ns[k] < 0 || encoder_ns[k] >= kTimeLimit)
                return fail("arrival and encoder times must be in [0, 2^60)");
            A = std::max(A, arrival_ns[k]);
        }
        std::vector<int64_t> r(agents);
        for (int k = 0; k < agents; ++k) r[k] = mode == RTCC_MODE_RELEASE ? arrival_ns[k] : A;
        std::vector<int32_t> order(agents);
        for (int k = 0; k < agents; ++k) order[k] = k;
        std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return r[a] < r[b]; });
        int64_t g = 0, pre = 0;
        for (int32_t k : order) {
            const int64_t s = std::max(r[k], g);
            g = s + encoder_ns[k];
            pre += std::max<int64_t>(0, std::min(g, A) - s);
            if (start_ns) start_ns[k] = s;
        }
        *latency_ns = g + post_ns;
        if (pre_arrival_ns) *pre_arrival_ns = pre;
        return RTCC_OK;
    });
}

rtcc_status rtcc_upward_rank(int32_t nodes, const int64_t *cost_ns, int32_t edges, const int32_t *edge_list,
                             int64_t *rank_ns) {
    return guarded([&] {
        if (nodes < 1 || edges < 0) return fail("nodes must be >= 1 and edges >= 0");
        if (!cost_ns || !rank_ns || (edges > 0 && !edge_list)) return fail("NULL cost_ns, rank_ns or edge_list");
        int64_t total = 0;
        for (int v = 0; v < nodes; ++v) {
            if (cost_ns[v] < 0 || cost_ns[v] >= kTimeLimit) return fail("node costs must be in [0, 2^60)");
            total += cost_ns[v];
            if (total >= kTimeLimit) return fail("sum of node costs must be < 2^60");
        }
        std::vector<std::vector<int32_t>> succ(nodes);
        std::vector<int32_t> out_deg(nodes, 0);
        std::vector<std::vector<int32_t>> pred(nodes);
        for (int e = 0; e < edges; ++e) {
            const int32_t u = edge_list[2 * e], v = edge_list[2 * e + 1];
            if (u < 0 || u >= nodes || v < 0 || v >= nodes) return fail("edge endpoint out of range");
            if (u == v) return fail("self loop");
            succ[u].push_back(v);
            pred[v].push_back(u);
            ++out_deg[u];
        }
        // Reverse topological order: a node is ranked once all its
        // successors are; nodes left unranked lie on a cycle.
        std::vector<int32_t> ready;
        for (int v = 0; v < nodes; ++v)
            if (out_deg[v] == 0) ready.push_back(v);
        std::vector<int64_t> rank(nodes, 0);
        int done = 0;
        while (!ready.empty()) {
            const int32_t v = ready.back();
            ready.pop_back();
            int64_t best = 0;
            for (int32_t w : succ[v]) best = std::max(best, rank[w]);
            rank[v] = cost_ns[v] + best;
            ++done;
            for (int32_t u : pred[v])
                if (--out_deg[u] == 0) ready.push_back(u);
        }
        if (done != nodes) return fail("the graph has a cycle");
        std::copy(rank.begin(), rank.end(), rank_ns);
        return RTCC_OK;
    });
}

}  // extern "C"
