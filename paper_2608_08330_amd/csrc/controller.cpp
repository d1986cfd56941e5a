// RTCC release controller (Sec. IV-C), executor-agnostic.

#include "controller.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>

namespace rtcc {

rtcc_status Controller::create(const rtcc_model_desc *d, const void *weights, size_t bytes,
                               const rtcc_runtime_opts *opts) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!d) return fail(RTCC_E_ARG, "model descriptor is NULL");
    if (!weights) return fail(RTCC_E_ARG, "weights pointer is NULL");
    if (bytes % 4) return fail(RTCC_E_ARG, "weights_bytes is not a multiple of 4");
    std::string err;
    if (!make_plan(*d, plan_, err)) return fail(RTCC_E_ARG, err);
    rtcc_runtime_opts o{};
    o.exec = RTCC_EXEC_PER_BRANCH_STREAMS;
    o.premature_tol_s = 1e-6;
    if (opts) o = *opts;
    if (o.exec != RTCC_EXEC_PER_BRANCH_STREAMS && o.exec != RTCC_EXEC_SERIAL)
        return fail(RTCC_E_ARG, "bad exec option");
    if (!(o.premature_tol_s >= 0.0) || !std::isfinite(o.premature_tol_s))
        return fail(RTCC_E_ARG, "premature_tol_s must be finite and >= 0");
    if ((o.use_graphs != 0 && o.use_graphs != 1) || (o.node_timing != 0 && o.node_timing != 1))
        return fail(RTCC_E_ARG, "use_graphs and node_timing must be 0 or 1");
    if (o.conv_variant < 0 || o.conv_variant > 12 || o.conv_splits < 0 || o.conv_splits > 64)
        return fail(RTCC_E_ARG, "conv_variant must be in [0, 12] and conv_splits in [0, 64]");
    if ((o.dev_alloc == nullptr) != (o.dev_free == nullptr))
        return fail(RTCC_E_ARG, "dev_alloc and dev_free must be given together");
    opts_ = o;
    HostWeights hw;
    if (!prepare_weights(plan_, static_cast<const float *>(weights), bytes / 4, hw, err))
        return fail(RTCC_E_ARG, err);
    rtcc_status s = ex_->init(plan_, hw, opts_, err);
    if (s != RTCC_OK) return fail(s, err);
    z_.assign(plan_.K, RTCC_WAITING);
    recorded_.assign(plan_.K, 0);
    dispatched_.assign(plan_.K, 0);
    arrival_.assign(plan_.K, 0.0);
    dispatch_.assign(plan_.K, 0.0);
    affine_.assign(plan_.K, std::array<float, 6>{1, 0, 0, 0, 1, 0});
    pose_.assign(plan_.K, std::array<float, 3>{0, 0, 0});
    created_ = true;
    return RTCC_OK;
}

rtcc_status Controller::set_mode(int mode) {
    std::lock_guard<std::mutex> lk(mu_);
    if (mode != RTCC_MODE_RELEASE && mode != RTCC_MODE_BARRIER) return fail(RTCC_E_ARG, "bad mode");
    if (in_frame_) return fail(RTCC_E_STATE, "set_mode inside a frame");
    mode_ = mode;
    return RTCC_OK;
}

rtcc_status Controller::staging(int agent, float **ptr, int64_t *cap) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!ptr || !cap) return fail(RTCC_E_ARG, "NULL output pointer");
    if (agent < 0 || agent >= plan_.K) return fail(RTCC_E_ARG, "agent out of range");
    *ptr = ex_->staging(agent);
    *cap = plan_.n_max;
    return RTCC_OK;
}

rtcc_status Controller::begin_frame(double t0) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!std::isfinite(t0)) return fail(RTCC_E_ARG, "t0 is not finite");
    if (in_frame_) return fail(RTCC_E_STATE, "begin_frame inside a frame");
    std::string err;
    rtcc_status s = ex_->begin_frame(err);
    if (s != RTCC_OK) return fail(s, err);
    t_begin_ = now_s();
    t0_ = t0;
    std::fill(z_.begin(), z_.end(), int(RTCC_WAITING));
    std::fill(recorded_.begin(), recorded_.end(), char(0));
    std::fill(dispatched_.begin(), dispatched_.end(), char(0));
    dispatch_failed_ = false;
    std::fill(arrival_.begin(), arrival_.end(), 0.0);
    std::fill(dispatch_.begin(), dispatch_.end(), 0.0);
    pending_.clear();
    have_output_ = false;
    in_frame_ = true;
    return RTCC_OK;
}

// Release and enqueue the encoders of a group: every z_k becomes RELEASED
// (input received, encoder enqueued); RUNNING and FINISHED follow the device
// (refresh_state).  A failed enqueue leaves the group's branches
// undispatched and marks the frame, whose join then withholds the post-join
// subgraph.
rtcc_status Controller::dispatch_locked(std::vector<Pending> &group) {
    if (group.empty()) return RTCC_OK;
    std::sort(group.begin(), group.end(), [](const Pending &a, const Pending &b) { return a.agent < b.agent; });
    const double now = now_s() - t0_;
    std::vector<DispatchItem> items;
    for (const Pending &pd : group) {
        z_[pd.agent] = RTCC_RELEASED;
        dispatch_[pd.agent] = now;
        items.push_back(DispatchItem{pd.agent, pd.pts, pd.n, pd.device_src, affine_[pd.agent].data()});
    }
    std::string err;
    rtcc_status s = ex_->dispatch(items.data(), int(items.size()), err);
    if (s != RTCC_OK) {
        // not enqueued; the recorded events still make repeats duplicates
        for (const Pending &pd : group) z_[pd.agent] = RTCC_WAITING;
        dispatch_failed_ = true;
        std::string who;
        for (const Pending &pd : group) who += (who.empty() ? "" : ", ") + std::to_string(pd.agent);
        return fail(s, "dispatch of branch " + who + " failed: " + err);
    }
    for (const Pending &pd : group) dispatched_[pd.agent] = 1;
    return RTCC_OK;
}

void Controller::refresh_state(int agent) {
    if (!dispatched_[agent] || z_[agent] == RTCC_FINISHED) return;
    const int st = RTCC_RELEASED + std::min(2, std::max(0, ex_->progress(agent)));
    if (st > z_[agent]) z_[agent] = st;
}

rtcc_status Controller::record_locked(int agent, const float *pts, int64_t n, const float pose[3],
                                      double arrival, bool device_src, Pending *pd) {
    if (!in_frame_) return fail(RTCC_E_STATE, "release outside a frame");
    if (agent < 0 || agent >= plan_.K) return fail(RTCC_E_ARG, "agent out of range");
    if (z_[agent] != RTCC_WAITING || recorded_[agent]) return fail(RTCC_E_DUPLICATE, "duplicate completion event");
    if (n < 0 || n > plan_.n_max) return fail(RTCC_E_MALFORMED, "point count out of range");
    if (!pts && n > 0) return fail(RTCC_E_MALFORMED, "NULL points with n > 0");
    if (!pose || !std::isfinite(pose[0]) || !std::isfinite(pose[1]) || !std::isfinite(pose[2]))
        return fail(RTCC_E_MALFORMED, "non-finite pose");
    if (!std::isfinite(arrival) || arrival < 0.0) return fail(RTCC_E_MALFORMED, "bad arrival time");
    const double now = now_s() - t0_;
    if (now < arrival - opts_.premature_tol_s)
        return fail(RTCC_E_PREMATURE, "completion event precedes its arrival time");

    // Validated: the input is complete.  Inputs given in host memory are
    // staged in pinned memory now, so the caller may reuse its buffer.
    if (!device_src && n > 0) {
        float *stg = ex_->staging(agent);
        if (pts != stg) std::memcpy(stg, pts, size_t(n) * 4 * sizeof(float));
        pts = stg;
    }
    pose_affine(plan_, pose, affine_[agent].data());
    pose_[agent] = {pose[0], pose[1], pose[2]};
    recorded_[agent] = 1;
    arrival_[agent] = arrival;
    *pd = Pending{agent, arrival, pts, n, device_src};
    return RTCC_OK;
}

rtcc_status Controller::release_locked(std::vector<Pending> &accepted) {
    if (accepted.empty()) return RTCC_OK;
    if (mode_ == RTCC_MODE_RELEASE) return dispatch_locked(accepted);
    // Barrier: the branches stay WAITING (their inputs are recorded, their
    // release waits for A); the K-th valid event releases every encoder at
    // A = max_k a_k, as one group in index order.
    pending_.insert(pending_.end(), accepted.begin(), accepted.end());
    if (int(pending_.size()) < plan_.K) return RTCC_OK;
    std::vector<Pending> ready;
    ready.swap(pending_);
    return dispatch_locked(ready);
}

rtcc_status Controller::release(int agent, const float *pts, int64_t n, const float pose[3],
                                double arrival, bool device_src) {
    std::lock_guard<std::mutex> lk(mu_);
    Pending pd{};
    rtcc_status s = record_locked(agent, pts, n, pose, arrival, device_src, &pd);
    if (s != RTCC_OK) return s;
    std::vector<Pending> one{pd};
    return release_locked(one);
}

rtcc_status Controller::release_group(int32_t count, const rtcc_event *events, rtcc_status *status) {
    std::lock_guard<std::mutex> lk(mu_);
    if (count < 0 || count > RTCC_MAX_AGENTS) return fail(RTCC_E_ARG, "event count out of [0, RTCC_MAX_AGENTS]");
    if (count > 0 && !events) return fail(RTCC_E_ARG, "NULL events");
    std::vector<Pending> accepted;
    rtcc_status first = RTCC_OK;
    std::string first_err;
    for (int32_t i = 0; i < count; ++i) {
        const rtcc_event &e = events[i];
        Pending pd{};
        rtcc_status s = e.device != 0 && e.device != 1
                            ? fail(RTCC_E_MALFORMED, "event.device must be 0 or 1")
                            : record_locked(e.agent, e.points, e.n, e.pose, e.arrival_t, e.device == 1, &pd);
        if (status) status[i] = s;
        if (s == RTCC_OK) {
            accepted.push_back(pd);
        } else if (first == RTCC_OK) {
            first = s;
            first_err = "event " + std::to_string(i) + ": " + err_;
        }
    }
    const rtcc_status d = release_locked(accepted);
    if (d != RTCC_OK) return d;  // the frame cannot complete: reported first
    if (first != RTCC_OK) return fail(first, first_err);
    return RTCC_OK;
}

rtcc_status Controller::join(rtcc_detections *out) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!out) return fail(RTCC_E_ARG, "NULL output");
    if (!in_frame_) return fail(RTCC_E_STATE, "join outside a frame");
    for (int k = 0; k < plan_.K; ++k) {
        if (!recorded_[k]) {
            // Communication-infeasible frame: the shared subgraph is withheld.
            in_frame_ = false;
            pending_.clear();
            return fail(RTCC_E_INFEASIBLE, "branch " + std::to_string(k) + " undelivered");
        }
    }
    for (int k = 0; k < plan_.K; ++k) {
        if (!dispatched_[k]) {
            // Every input arrived but an encoder was never enqueued (its
            // dispatch failed): its slot is stale, so no fusion runs.
            in_frame_ = false;
            pending_.clear();
            return fail(RTCC_E_STATE, "branch " + std::to_string(k) +
                                          (dispatch_failed_ ? " was not dispatched (a dispatch failed)"
                                                            : " was not dispatched"));
        }
    }
    std::memset(out, 0, sizeof(*out));
    std::string err;
    rtcc_status s = ex_->join(affine_, pose_, t_begin_ - t0_, out, err);
    in_frame_ = false;
    if (s != RTCC_OK) return fail(s, err);
    // the post-join subgraph ran after every encoder's completion event
    for (int k = 0; k < plan_.K; ++k) z_[k] = RTCC_FINISHED;
    out->t_det_s = now_s() - t0_;
    out->n_agents = plan_.K;
    for (int k = 0; k < plan_.K; ++k) {
        out->arrival_s[k] = arrival_[k];
        out->dispatch_s[k] = dispatch_[k];
    }
    have_output_ = true;
    return RTCC_OK;
}

rtcc_status Controller::branch_state(int agent, int32_t *state) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!state) return fail(RTCC_E_ARG, "NULL output");
    if (agent < 0 || agent >= plan_.K) return fail(RTCC_E_ARG, "agent out of range");
    refresh_state(agent);
    *state = z_[agent];
    return RTCC_OK;
}

rtcc_status Controller::tensor_bytes(int id, int agent, size_t *bytes) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!bytes) return fail(RTCC_E_ARG, "NULL output");
    if (!have_output_) return fail(RTCC_E_STATE, "no completed frame");
    std::string err;
    rtcc_status s = ex_->tensor_bytes(id, agent, bytes, err);
    return s == RTCC_OK ? s : fail(s, err);
}

rtcc_status Controller::get_tensor(int id, int agent, void *dst, size_t bytes) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!dst) return fail(RTCC_E_ARG, "NULL destination");
    if (!have_output_) return fail(RTCC_E_STATE, "no completed frame");
    std::string err;
    rtcc_status s = ex_->get_tensor(id, agent, dst, bytes, err);
    return s == RTCC_OK ? s : fail(s, err);
}

rtcc_status Controller::profile_nodes(int warmup, int reps, float *median_ms, int32_t *n_nodes) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!median_ms || !n_nodes) return fail(RTCC_E_ARG, "NULL output");
    if (warmup < 0 || reps < 1) return fail(RTCC_E_ARG, "warmup < 0 or reps < 1");
    if (!have_output_ || in_frame_) return fail(RTCC_E_STATE, "needs a completed frame and no open frame");
    std::string err;
    int n = 0;
    rtcc_status s = ex_->profile_nodes(warmup, reps, median_ms, &n, err);
    *n_nodes = n;
    return s == RTCC_OK ? s : fail(s, err);
}

rtcc_status Controller::node_times(float *ms, int32_t *n) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!ms || !n) return fail(RTCC_E_ARG, "NULL output");
    if (!opts_.node_timing) return fail(RTCC_E_STATE, "node timing is off");
    if (!have_output_) return fail(RTCC_E_STATE, "no completed frame");
    std::string err;
    int m = 0;
    rtcc_status s = ex_->node_times(ms, &m, err);
    *n = m;
    return s == RTCC_OK ? s : fail(s, err);
}

rtcc_status Controller::node_count(int32_t *n) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!n) return fail(RTCC_E_ARG, "NULL output");
    *n = ex_->node_count();
    return RTCC_OK;
}

rtcc_status Controller::conv_plan(int layer, int32_t out[2]) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!out) return fail(RTCC_E_ARG, "NULL output");
    if (layer < 0 || layer >= int(plan_.convs.size())) return fail(RTCC_E_ARG, "layer out of range");
    if (!ex_->conv_plan(layer, out)) return fail(RTCC_E_STATE, "no kernel plan in this executor");
    return RTCC_OK;
}

rtcc_status Controller::graph_stats(int64_t out[3]) {
    std::lock_guard<std::mutex> lk(mu_);
    if (!out) return fail(RTCC_E_ARG, "NULL output");
    ex_->graph_stats(out);
    return RTCC_OK;
}

}  // namespace rtcc
