// extern "C" entry points of include/rtcc.h.  Argument marshalling onto the
// controller (and, for rtcc_conv_tiling, the conv planner).
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "checkpoint.hpp"
#include "controller.hpp"
#include "kernels/conv_plan.hpp"

struct rtcc_ctx {
    rtcc::Controller ctl;
    explicit rtcc_ctx(rtcc::Executor *ex) : ctl(ex) {}
};

namespace {
// Message of the last failed context-free call (rtcc_create,
// rtcc_rotated_nms) on this thread; rtcc_last_error(NULL) returns it.
thread_local std::string t_create_error;

template <class F>
rtcc_status guarded(F &&f) {
    try {
        return f();
    } catch (const std::bad_alloc &) {
        return RTCC_E_NOMEM;
    } catch (...) {
        return RTCC_E_INTERNAL;
    }
}
}  // namespace

namespace rtcc {
void set_thread_error(const std::string &msg) { t_create_error = msg; }
}  // namespace rtcc

extern "C" {

rtcc_status rtcc_create(const rtcc_model_desc *model, const void *weights, size_t weights_bytes,
                        const rtcc_runtime_opts *opts, rtcc_ctx **out) {
    if (!out) return RTCC_E_ARG;
    *out = nullptr;
    rtcc_ctx *ctx = nullptr;
    rtcc_status s = guarded([&] {
        ctx = new rtcc_ctx(rtcc::make_executor());
        return ctx->ctl.create(model, weights, weights_bytes, opts);
    });
    if (s != RTCC_OK) {
        if (ctx) t_create_error = ctx->ctl.last_error();
        delete ctx;
        return s;
    }
    *out = ctx;
    return RTCC_OK;
}

rtcc_status rtcc_read_checkpoint(const void *file, size_t file_bytes, rtcc_checkpoint_info *info) {
    if (!info) {
        t_create_error = "info is NULL";
        return RTCC_E_ARG;
    }
    std::memset(info, 0, sizeof(*info));
    return guarded([&] {
        rtcc::CkptView v;
        std::string err;
        const rtcc_status s = rtcc::parse_checkpoint(file, file_bytes, v, err);
        if (s != RTCC_OK) {
            t_create_error = err;
            return s;
        }
        *info = v.info;
        return RTCC_OK;
    });
}

rtcc_status rtcc_create_from_checkpoint(const rtcc_model_desc *model, const void *file, size_t file_bytes,
                                        const rtcc_runtime_opts *opts, rtcc_ctx **out) {
    if (!out) return RTCC_E_ARG;
    *out = nullptr;
    std::vector<float> blob;
    const rtcc_status s = guarded([&] {
        if (!model) {
            t_create_error = "model descriptor is NULL";
            return RTCC_E_ARG;
        }
        rtcc::CkptView v;
        std::string err;
        rtcc_status st = rtcc::parse_checkpoint(file, file_bytes, v, err);
        if (st != RTCC_OK) {
            t_create_error = err;
            return st;
        }
        rtcc::Plan plan;
        if (!rtcc::make_plan(*model, plan, err)) {
            t_create_error = err;
            return RTCC_E_ARG;
        }
        // the tensor table must list exactly the descriptor's tensors, in
        // blob order, with their shapes
        const std::vector<rtcc::CkptTensor> want = rtcc::expected_tensors(plan);
        if (want.size() != v.tensors.size()) {
            t_create_error = "checkpoint has " + std::to_string(v.tensors.size()) + " tensors, descriptor needs " +
                             std::to_string(want.size());
            return RTCC_E_ARG;
        }
        for (size_t i = 0; i < want.size(); ++i) {
            const rtcc::CkptTensor &a = v.tensors[i], &b = want[i];
            bool same = a.name == b.name && a.ndim == b.ndim;
            for (int d = 0; same && d < 4; ++d) same = a.shape[d] == b.shape[d];
            if (!same) {
                t_create_error = "checkpoint tensor " + std::to_string(i) + " is " + a.name +
                                 " with another shape or name than the descriptor's " + b.name;
                return RTCC_E_ARG;
            }
        }
        // the data section may sit at any alignment in the caller's buffer
        blob.resize(size_t(v.info.data_bytes / 4));
        std::memcpy(blob.data(), v.data, size_t(v.info.data_bytes));
        return RTCC_OK;
    });
    if (s != RTCC_OK) return s;
    return rtcc_create(model, blob.data(), blob.size() * 4, opts, out);
}

void rtcc_destroy(rtcc_ctx *ctx) { delete ctx; }

rtcc_status rtcc_set_mode(rtcc_ctx *ctx, rtcc_mode mode) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.set_mode(int(mode)); });
}

rtcc_status rtcc_staging_buffer(rtcc_ctx *ctx, int32_t agent, float **pinned, int64_t *capacity) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.staging(agent, pinned, capacity); });
}

rtcc_status rtcc_begin_frame(rtcc_ctx *ctx, double t0_monotonic_s) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.begin_frame(t0_monotonic_s); });
}

rtcc_status rtcc_release_branch(rtcc_ctx *ctx, int32_t agent, const float *host_points, int64_t n,
                                const float pose[3], double arrival_t) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.release(agent, host_points, n, pose, arrival_t, false); });
}

rtcc_status rtcc_release_branch_device(rtcc_ctx *ctx, int32_t agent, const float *device_points,
                                       int64_t n, const float pose[3], double arrival_t) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.release(agent, device_points, n, pose, arrival_t, true); });
}

rtcc_status rtcc_release_branches(rtcc_ctx *ctx, int32_t count, const rtcc_event *events, rtcc_status *status) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.release_group(count, events, status); });
}

rtcc_status rtcc_join_and_detect(rtcc_ctx *ctx, rtcc_detections *out) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.join(out); });
}

rtcc_status rtcc_get_branch_state(rtcc_ctx *ctx, int32_t agent, int32_t *state) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.branch_state(agent, state); });
}

rtcc_status rtcc_tensor_bytes(rtcc_ctx *ctx, int32_t id, int32_t agent, size_t *bytes) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.tensor_bytes(id, agent, bytes); });
}

rtcc_status rtcc_get_tensor(rtcc_ctx *ctx, int32_t id, int32_t agent, void *dst, size_t bytes) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.get_tensor(id, agent, dst, bytes); });
}

rtcc_status rtcc_profile_nodes(rtcc_ctx *ctx, int32_t warmup, int32_t reps, float *median_ms,
                               int32_t *n_nodes) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.profile_nodes(warmup, reps, median_ms, n_nodes); });
}

rtcc_status rtcc_node_times(rtcc_ctx *ctx, float *ms, int32_t *n) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.node_times(ms, n); });
}

rtcc_status rtcc_node_count(rtcc_ctx *ctx, int32_t *n) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.node_count(n); });
}

rtcc_status rtcc_conv_plan(rtcc_ctx *ctx, int32_t layer, int32_t *plan) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.conv_plan(layer, plan); });
}

rtcc_status rtcc_conv_tiling(int32_t bf16, const int32_t *shape, int32_t maps, int32_t *out) {
    if (!shape || !out || maps < 1 || maps > 16) return RTCC_E_ARG;
    for (int i = 0; i < 8; ++i)
        if (i != 6 && shape[i] < 1) return RTCC_E_ARG;
    if (shape[6] != 1 && shape[6] != 2) return RTCC_E_ARG;
    const rtcc::kern::ConvPlan p = rtcc::kern::conv_plan(bf16 != 0, shape[0], shape[1], shape[2], shape[3], shape[4],
                                                         shape[5], shape[6], shape[7]);
    out[0] = rtcc::kern::conv_variant_for(p, maps);
    out[1] = p.splits;
    return RTCC_OK;
}

rtcc_status rtcc_graph_stats(rtcc_ctx *ctx, int64_t *counts) {
    if (!ctx) return RTCC_E_ARG;
    return guarded([&] { return ctx->ctl.graph_stats(counts); });
}

const char *rtcc_status_str(rtcc_status s) {
    switch (s) {
        case RTCC_OK: return "RTCC_OK";
        case RTCC_E_ARG: return "RTCC_E_ARG";
        case RTCC_E_STATE: return "RTCC_E_STATE";
        case RTCC_E_DUPLICATE: return "RTCC_E_DUPLICATE";
        case RTCC_E_MALFORMED: return "RTCC_E_MALFORMED";
        case RTCC_E_PREMATURE: return "RTCC_E_PREMATURE";
        case RTCC_E_INFEASIBLE: return "RTCC_E_INFEASIBLE";
        case RTCC_E_NOMEM: return "RTCC_E_NOMEM";
        case RTCC_E_HIP: return "RTCC_E_HIP";
        case RTCC_E_INTERNAL: return "RTCC_E_INTERNAL";
    }
    return "RTCC_E_UNKNOWN";
}

const char *rtcc_last_error(const rtcc_ctx *ctx) {
    if (!ctx) return t_create_error.c_str();
    return ctx->ctl.last_error();
}

}  // extern "C"
