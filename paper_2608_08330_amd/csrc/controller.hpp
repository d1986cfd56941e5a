// RTCC release controller (Sec. IV-C) and the executor interface it drives.
//
// The controller owns the per-branch state z_k in {WAITING, RELEASED,
// RUNNING, FINISHED}, validates completion events, applies the release rule
// (RTCC: dispatch at the event; Barrier: dispatch all K at the K-th event in
// (A, k) order) and withholds the post-join subgraph of an infeasible frame.
// It is host-only C++ and is unit-tested against a recording executor.
#pragma once

#include <array>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/rtcc.h"
#include "model.hpp"

namespace rtcc {

// What the controller asks of an executor.  All calls come with the
// controller's mutex held.
struct DispatchItem {
    int agent;
    const float *pts;
    int64_t n;
    bool device_src;
    const float *affine;  // [6]
};

class Executor {
  public:
    virtual ~Executor() = default;
    virtual rtcc_status init(const Plan &p, const HostWeights &w, const rtcc_runtime_opts &o,
                             std::string &err) = 0;
    virtual float *staging(int agent) = 0;
    virtual rtcc_status begin_frame(std::string &err) = 0;
    // Enqueue H2D (unless device_src) and encoder E_k of every item, as one
    // group released together (m >= 1, distinct agents in ascending order).
    // `affine` is the agent's pose warp (index space), used by the branch
    // when the warp is its last node.
    virtual rtcc_status dispatch(const DispatchItem *items, int m, std::string &err) = 0;
    // Progress of a dispatched encoder on the device: 0 enqueued (its input
    // copy or earlier work of its stream still ahead of it), 1 started, 2
    // finished (its slot is stored).  Never blocks.
    virtual int progress(int agent) = 0;
    // Wait for all encoders on the device, run the post-join subgraph with
    // the given per-agent warp affines (feature grid) and poses (for the
    // stage grids of multi-scale fusion), copy detections to the host.  Fills
    // out->count / boxes / scores / anchor_idx / t_head_s (relative to the
    // host time t_begin at which begin_frame was called).
    virtual rtcc_status join(const std::vector<std::array<float, 6>> &affine,
                             const std::vector<std::array<float, 3>> &poses, double t_begin,
                             rtcc_detections *out, std::string &err) = 0;
    virtual rtcc_status tensor_bytes(int id, int agent, size_t *bytes, std::string &err) = 0;
    virtual rtcc_status get_tensor(int id, int agent, void *dst, size_t bytes, std::string &err) = 0;
    virtual rtcc_status profile_nodes(int warmup, int reps, float *median_ms, int *n_nodes,
                                      std::string &err) = 0;
    virtual int node_count() const = 0;
    virtual rtcc_status node_times(float *ms, int *n, std::string &err) = 0;
    // HIP graph instantiations, in-place update attempts and launches so far.
    virtual void graph_stats(int64_t out[3]) const { out[0] = out[1] = out[2] = 0; }
    // Kernel tiling and K split of 3x3 conv layer `layer` (false if out of
    // range).
    virtual bool conv_plan(int layer, int32_t out[2]) const {
        (void)layer;
        out[0] = out[1] = 0;
        return false;
    }
};

// Defined by exactly one executor translation unit of a build.
Executor *make_executor();

struct Pending {
    int agent;
    double arrival;
    const float *pts;
    int64_t n;
    bool device_src;
};

class Controller {
  public:
    explicit Controller(Executor *ex) : ex_(ex) {}
    ~Controller() { delete ex_; }

    rtcc_status create(const rtcc_model_desc *d, const void *weights, size_t bytes,
                       const rtcc_runtime_opts *opts);
    rtcc_status set_mode(int mode);
    rtcc_status staging(int agent, float **ptr, int64_t *cap);
    rtcc_status begin_frame(double t0);
    rtcc_status release(int agent, const float *pts, int64_t n, const float pose[3], double arrival,
                        bool device_src);
    // Events that arrived together: each validated and recorded in order as
    // release() would; the accepted ones are released as one group.
    rtcc_status release_group(int32_t count, const rtcc_event *events, rtcc_status *status);
    rtcc_status join(rtcc_detections *out);
    rtcc_status branch_state(int agent, int32_t *state);
    rtcc_status tensor_bytes(int id, int agent, size_t *bytes);
    rtcc_status get_tensor(int id, int agent, void *dst, size_t bytes);
    rtcc_status profile_nodes(int warmup, int reps, float *median_ms, int32_t *n_nodes);
    rtcc_status node_times(float *ms, int32_t *n);
    rtcc_status node_count(int32_t *n);
    rtcc_status graph_stats(int64_t out[3]);
    rtcc_status conv_plan(int layer, int32_t out[2]);

    const char *last_error() const { return err_.c_str(); }

  private:
    rtcc_status fail(rtcc_status s, const std::string &msg) {
        err_ = msg;
        return s;
    }
    // Validate and record one completion event (Sec. IV-C); on success *pd
    // is the branch's pending release.
    rtcc_status record_locked(int agent, const float *pts, int64_t n, const float pose[3], double arrival,
                              bool device_src, Pending *pd);
    // Release the recorded branches of `group` (ascending agents) together.
    rtcc_status dispatch_locked(std::vector<Pending> &group);
    // RELEASE: dispatch `accepted` now; BARRIER: add it to the pending set
    // and dispatch all K once the K-th event is in.
    rtcc_status release_locked(std::vector<Pending> &accepted);
    // z_k of a dispatched branch follows its encoder on the device.
    void refresh_state(int agent);

    std::mutex mu_;
    Executor *ex_;
    Plan plan_;
    rtcc_runtime_opts opts_{};
    bool created_ = false;
    int mode_ = RTCC_MODE_RELEASE;
    bool in_frame_ = false;
    bool have_output_ = false;
    double t0_ = 0.0, t_begin_ = 0.0;
    std::vector<int> z_;
    std::vector<char> recorded_;    // event validated in this frame (barrier: before A)
    std::vector<char> dispatched_;  // encoder enqueued on the device in this frame
    bool dispatch_failed_ = false;  // an enqueue failed: the frame cannot complete
    std::vector<double> arrival_, dispatch_;
    std::vector<std::array<float, 6>> affine_;
    std::vector<std::array<float, 3>> pose_;
    std::vector<Pending> pending_;
    std::string err_;
};

}  // namespace rtcc
