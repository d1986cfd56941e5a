// HIP executor: per-agent device buffers, pinned staging, branch streams and
// events, the post-join subgraph, tensor readback and node timing.
//
// Physical release path (Sec. IV-F): a branch input stays in pinned host
// memory until its completion event; the event triggers an async H2D copy,
// and the encoder kernels are ordered after the copy on the GPU (same
// stream, or in SERIAL mode a copy stream + HIP event + wait on the single
// compute stream).  Each encoder writes only its own agent-indexed buffers
// and slot (Sec. IV-D), so branches never share memory and may overlap.  The
// join waits on every branch's completion event on the GPU (no host wait)
// before the post-join kernels run.
//
// Branches released together (one batch of events, or every branch at the
// barrier's A) share one sequence of launches on the first member's stream:
// every pillar kernel, conv layer and upsampling runs the group's agents side
// by side in one grid, each agent's output bit for bit that of a launch of
// its own.  A single release is a group of one.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "controller.hpp"
#include "kernels/kernels.hpp"

namespace rtcc {

namespace {

#define HIP_TRY(expr)                                                                   \
    do {                                                                                \
        hipError_t e_ = (expr);                                                         \
        if (e_ != hipSuccess) {                                                         \
            err = std::string(#expr) + " failed: " + hipGetErrorString(e_);             \
            return e_ == hipErrorOutOfMemory ? RTCC_E_NOMEM : RTCC_E_HIP;               \
        }                                                                               \
    } while (0)

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

}  // namespace

class HipExecutor : public Executor {
  public:
    ~HipExecutor() override { release_all(); }

    rtcc_status init(const Plan &p, const HostWeights &w, const rtcc_runtime_opts &o,
                     std::string &err) override {
        p_ = p;
        o_ = o;
        dev_ = o.device;
        HIP_TRY(hipSetDevice(dev_));
        // Device arena per agent and for the post-join subgraph.  Nothing is
        // shared between agents.
        const size_t n_max = size_t(p.n_max);
        const size_t n_cells = size_t(p.H) * p.W;
        const size_t n_tiles = (n_cells + kern::kScanTile - 1) / kern::kScanTile;
        const size_t over_cap = n_max / size_t(p.d.max_points_per_pillar + 1) + 1;
        tiles_ = int(n_tiles);
        // Kernel variant and split-K of every conv layer.
        int n_cu = 0;
        HIP_TRY(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev_));
        if (n_cu <= 0) n_cu = 256;
        plans_.clear();
        size_t ws_bytes = 0;
        for (const ConvLayer &c : p.convs) {
            kern::ConvPlan cp = kern::conv_plan(p.bf16, c.Hi, c.Wi, c.Ci, c.Ho, c.Wo, c.Co, c.stride, n_cu);
            if (o.conv_variant > 0)
                cp = kern::conv_plan_forced(p.bf16, cp, o.conv_variant, o.conv_splits, c.Ci, c.Ho, c.Wo, c.Co, c.stride);
            plans_.push_back(cp);
            ws_bytes = std::max(ws_bytes, plans_.back().ws_bytes);
        }
        HIP_TRY(alloc(&d_zero, 256));
        HIP_TRY(hipMemset(d_zero, 0, 256));
        br_.resize(p.K);
        for (int k = 0; k < p.K; ++k) {
            Branch &b = br_[k];
            HIP_TRY(hipHostMalloc(reinterpret_cast<void **>(&b.staging), n_max * 16, hipHostMallocDefault));
            HIP_TRY(alloc(&b.d_pts, n_max * 16));
            HIP_TRY(alloc(&b.d_cell, n_max * 4));
            HIP_TRY(alloc(&b.d_slot, n_max * 4));
            HIP_TRY(alloc(&b.d_member, n_max * 4));
            HIP_TRY(alloc(&b.d_sorted, n_max * 16));
            HIP_TRY(alloc(&b.d_pcells, n_max * 4));
            HIP_TRY(alloc(&b.d_pcounts, n_max * 4));
            HIP_TRY(alloc(&b.d_poffs, n_max * 4));
            HIP_TRY(alloc(&b.d_overfull, over_cap * 4));
            HIP_TRY(alloc(&b.d_ttotal, n_tiles * 4));
            HIP_TRY(hipMemset(b.d_ttotal, 0, n_tiles * 4));  // the pillar kernels leave it zero
            HIP_TRY(alloc(&b.d_tstart, (n_tiles + 1) * 4));
            HIP_TRY(alloc(&b.d_npil, n_tiles * 4));
            HIP_TRY(alloc(&b.d_binned, n_max * 4));
            HIP_TRY(alloc(&b.d_cellb, n_max * 4));
            HIP_TRY(alloc(&b.d_rank, n_max * 4));
            HIP_TRY(alloc(&b.d_tcell, n_cells * 4));
            HIP_TRY(alloc(&b.d_tcount, n_cells * 4));
            HIP_TRY(alloc(&b.d_toff, n_cells * 4));
            HIP_TRY(alloc(&b.d_meta, 64));
            HIP_TRY(hipMemset(b.d_meta, 0, 64));  // no pillars of a previous frame
            HIP_TRY(alloc(&b.d_canvas, n_cells * p.c_pfn * p.elt));
            HIP_TRY(hipMemset(b.d_canvas, 0, n_cells * p.c_pfn * p.elt));  // then nonzero only at pillars
            b.d_act.resize(p.convs.size());
            for (size_t l = 0; l < p.convs.size(); ++l) {
                const ConvLayer &c = p.convs[l];
                HIP_TRY(alloc(&b.d_act[l], size_t(c.Ho) * c.Wo * c.Co * p.elt));
            }
            if (ws_bytes) HIP_TRY(alloc(&b.d_ws, ws_bytes));
            if (p.d.multiscale) b.d_slotbuf = nullptr;  // the branch ends at its stage outputs
            else if (!p.ups.empty()) HIP_TRY(alloc(&b.d_slotbuf, size_t(p.H2) * p.W2 * p.c_slot * p.elt));
            else b.d_slotbuf = b.d_act.back();
            if (p.d.warp_in_branch) HIP_TRY(alloc(&b.d_warped, size_t(p.H2) * p.W2 * p.c_slot * p.elt));
            b.ego_map = b.d_slotbuf;
            HIP_TRY(hipStreamCreateWithFlags(&b.stream, hipStreamNonBlocking));
            HIP_TRY(hipEventCreateWithFlags(&b.done, hipEventDisableTiming));
            HIP_TRY(hipEventCreateWithFlags(&b.h2d_done, hipEventDisableTiming));
            HIP_TRY(hipEventCreateWithFlags(&b.started, hipEventDisableTiming));
            b.ev.resize(5 + p.convs.size() + p.ups.size());
            for (auto &e : b.ev) HIP_TRY(hipEventCreate(&e));
            b.kev.resize(2 * p.convs.size());
            for (auto &e : b.kev) HIP_TRY(hipEventCreate(&e));
            if (p.d.warp_in_branch)
                for (auto &e : b.wev) HIP_TRY(hipEventCreate(&e));
        }
        // every agent's pillar buffers, as the pillar kernels index them
        std::vector<kern::PillarBufs> pb(p.K);
        for (int k = 0; k < p.K; ++k) {
            const Branch &b = br_[k];
            pb[k].cell = static_cast<int32_t *>(b.d_cell);
            pb[k].slot = static_cast<int32_t *>(b.d_slot);
            pb[k].ttotal = static_cast<int32_t *>(b.d_ttotal);
            pb[k].tstart = static_cast<int32_t *>(b.d_tstart);
            pb[k].binned = static_cast<int32_t *>(b.d_binned);
            pb[k].cellb = static_cast<int32_t *>(b.d_cellb);
            pb[k].rank = static_cast<int32_t *>(b.d_rank);
            pb[k].tcell = static_cast<int32_t *>(b.d_tcell);
            pb[k].tcount = static_cast<int32_t *>(b.d_tcount);
            pb[k].toff = static_cast<int32_t *>(b.d_toff);
            pb[k].npil = static_cast<int32_t *>(b.d_npil);
            pb[k].meta = static_cast<int32_t *>(b.d_meta);
            pb[k].pcells = static_cast<int32_t *>(b.d_pcells);
            pb[k].pcounts = static_cast<int32_t *>(b.d_pcounts);
            pb[k].poffs = static_cast<int32_t *>(b.d_poffs);
            pb[k].overfull = static_cast<int32_t *>(b.d_overfull);
            pb[k].member = static_cast<int32_t *>(b.d_member);
            pb[k].sorted = static_cast<float4 *>(b.d_sorted);
            pb[k].canvas = b.d_canvas;
        }
        HIP_TRY(hipEventCreateWithFlags(&ev_clear_, hipEventDisableTiming));
        HIP_TRY(alloc(&d_pbufs_, sizeof(kern::PillarBufs) * p.K));
        HIP_TRY(hipMemcpy(d_pbufs_, pb.data(), sizeof(kern::PillarBufs) * p.K, hipMemcpyHostToDevice));
        HIP_TRY(alloc(&d_fused, size_t(p.H2) * p.W2 * p.c_slot * p.elt));
        d_fused_stage_.assign(p.ups.size(), nullptr);
        if (p.d.multiscale)
            for (const UpLayer &u : p.ups)
                HIP_TRY(alloc(&d_fused_stage_[u.stage], size_t(u.Hi) * u.Wi * u.Ci * p.elt));
        HIP_TRY(alloc(&d_head, size_t(p.H2) * p.W2 * 16 * 4));
        n_anchor_ = size_t(p.H2) * p.W2 * 2;
        HIP_TRY(alloc(&d_head_counts, (size_t(p.H2) * p.W2 + 15) / 16 * 4));
        HIP_TRY(alloc(&d_rec, n_anchor_ * 9 * 4));
        HIP_TRY(alloc(&d_count, 64));
        nms_max_ = p.d.nms_max_candidates;
        if (nms_max_ > 0) {
            const size_t words = size_t(nms_max_ + 63) / 64;
            HIP_TRY(alloc(&d_nms_rank, n_anchor_ * 4));
            HIP_TRY(alloc(&d_nms_flag, n_anchor_ * 4));
            HIP_TRY(alloc(&d_nms_order, size_t(nms_max_) * 4));
            HIP_TRY(alloc(&d_nms_foot, size_t(nms_max_) * kern::kNmsFootDoubles * 8));
            HIP_TRY(alloc(&d_nms_mask, size_t(nms_max_) * words * 8));
            HIP_TRY(alloc(&d_nms_out, size_t(nms_max_) * 9 * 4));
            HIP_TRY(alloc(&d_nms_count, 64));
            HIP_TRY(alloc(&d_nms_mask_t, size_t(nms_max_) * 8));
            HIP_TRY(alloc(&d_nms_partial, size_t(kern::kNmsRankSplits) * n_anchor_ * 4));
            HIP_TRY(alloc(&d_nms_colrows, kern::nms_colrows(nms_max_) * 4));
            HIP_TRY(alloc(&d_nms_colcount, words * 4));
        }
        HIP_TRY(hipHostMalloc(reinterpret_cast<void **>(&h_rec), n_anchor_ * 9 * 4, hipHostMallocDefault));
        HIP_TRY(hipHostMalloc(reinterpret_cast<void **>(&h_small), 64, hipHostMallocDefault));
        // the frame's counts and first records, written by the last kernel
        // of the post-join work (coherent: read by the host once that kernel
        // has set its flag, word 2)
        export_first_ = int(std::min(nms_max_ > 0 ? size_t(nms_max_) : n_anchor_, kFirstRecords));
        HIP_TRY(hipHostMalloc(&h_export, 64 + size_t(export_first_) * 36, hipHostMallocCoherent));
        std::memset(h_export, 0, 64);
        boxes_.resize(n_anchor_ * 7);
        scores_.resize(n_anchor_);
        aidx_.resize(n_anchor_);
        if (o.join_stream) {
            join_stream_ = static_cast<hipStream_t>(o.join_stream);
            own_join_stream_ = false;
        } else {
            HIP_TRY(hipStreamCreateWithFlags(&join_stream_, hipStreamNonBlocking));
        }
        HIP_TRY(hipStreamCreateWithFlags(&copy_stream_, hipStreamNonBlocking));
        HIP_TRY(hipStreamCreateWithFlags(&aux_stream_, hipStreamNonBlocking));
        HIP_TRY(hipStreamCreateWithFlags(&cap_stream_, hipStreamNonBlocking));
        HIP_TRY(hipEventCreate(&ev_frame0_));
        HIP_TRY(hipEventCreate(&ev_head_));
        for (auto &e : post_ev_) HIP_TRY(hipEventCreate(&e));

        // Weights: matrices in the compute dtype, biases and PFN float32.
        const size_t mat_bytes = p.mat_elems * p.elt;
        HIP_TRY(alloc(&d_mat, mat_bytes));
        HIP_TRY(alloc(&d_bias, p.bias_floats * 4));
        const void *mat_src = p.bf16 ? static_cast<const void *>(w.mat_bf16.data())
                                     : static_cast<const void *>(w.mat_f32.data());
        HIP_TRY(hipMemcpy(d_mat, mat_src, mat_bytes, hipMemcpyHostToDevice));
        HIP_TRY(hipMemcpy(d_bias, w.bias.data(), p.bias_floats * 4, hipMemcpyHostToDevice));
        HIP_TRY(hipDeviceSynchronize());
        return RTCC_OK;
    }

    float *staging(int agent) override { return br_[agent].staging; }

    rtcc_status begin_frame(std::string &err) override {
        HIP_TRY(hipSetDevice(dev_));
        // Work of an abandoned (infeasible) frame may still be running and
        // reading the staging buffers that the caller is about to refill.
        // (After a completed join every stream is idle already.)
        if (!idle_) {
            for (Branch &b : br_) HIP_TRY(hipStreamSynchronize(b.stream));
            HIP_TRY(hipStreamSynchronize(copy_stream_));
            HIP_TRY(hipStreamSynchronize(join_stream_));
            idle_ = true;
        }
        HIP_TRY(hipEventRecord(ev_frame0_, compute_stream_for_join()));
        for (Branch &b : br_) b.dispatched = false;
        // canvases the last join did not clear (an abandoned frame)
        HIP_TRY(clear_dirty_canvases(false));
        return RTCC_OK;
    }

    // The last frame's canvas pillars back to zero, in one launch for every
    // branch on the join stream, which the stream of every encoder launch of
    // the next frame then waits for (from its pillar stage's second launch
    // on).  after_join: the branches' canvases stay readable as tensors
    // (rebuilt from their pillar lists).
    // s: the stream of the join's post-join work (default: the join stream).
    hipError_t clear_dirty_canvases(bool after_join, hipStream_t s = nullptr) {
        if (!s) s = join_stream_;
        int dirty[kern::kMaxGroup];
        int nd = 0;
        for (int k = 0; k < p_.K; ++k)
            if (br_[k].canvas_dirty) dirty[nd++] = k;
        if (nd == 0) return hipSuccess;
        hipError_t e = clear_canvases(dirty, nd, s);
        if (e != hipSuccess) return e;
        clear_stream_ = s;
        for (int j = 0; j < nd; ++j) br_[dirty[j]].canvas_consumed = after_join;
        if (o_.exec != RTCC_EXEC_SERIAL) {
            e = hipEventRecord(ev_clear_, s);
            if (e == hipSuccess) clear_pending_ = true;
        }
        return e;
    }

    rtcc_status dispatch(const DispatchItem *items, int m, std::string &err) override {
        HIP_TRY(hipSetDevice(dev_));
        if (m < 1 || m > kern::kMaxGroup) {
            err = "dispatch group of " + std::to_string(m) + " agents";
            return RTCC_E_INTERNAL;
        }
        const bool serial = o_.exec == RTCC_EXEC_SERIAL;
        const bool timing = o_.node_timing != 0;
        Branch &lead = br_[items[0].agent];
        // the group's encoders run on the first member's stream
        hipStream_t ls = serial ? join_stream_ : lead.stream;
        int agents[kern::kMaxGroup];
        for (int j = 0; j < m; ++j) {
            const DispatchItem &it = items[j];
            agents[j] = it.agent;
            Branch &b = br_[it.agent];
            for (int e = 0; e < 6; ++e) b.affine[e] = it.affine[e];
            hipStream_t bs = serial ? join_stream_ : b.stream;
            if (timing) HIP_TRY(hipEventRecord(b.ev[0], bs));
            const float *src = it.pts;
            if (!it.device_src) {
                src = static_cast<const float *>(b.d_pts);
                if (it.n > 0) {
                    // the member's own stream (the lead's is ls), or in
                    // SERIAL mode the transfer stream
                    HIP_TRY(hipMemcpyAsync(b.d_pts, b.staging, size_t(it.n) * 16, hipMemcpyHostToDevice,
                                           serial ? copy_stream_ : bs));
                    if (serial) {
                        HIP_TRY(hipEventRecord(b.h2d_done, copy_stream_));
                        HIP_TRY(hipStreamWaitEvent(ls, b.h2d_done, 0));
                    }
                }
            }
            // ls runs after the member's input copy on the member's stream
            // (the stream holds no other work of the frame)
            if (bs != ls && !it.device_src && it.n > 0) {
                HIP_TRY(hipEventRecord(b.h2d_done, bs));
                HIP_TRY(hipStreamWaitEvent(ls, b.h2d_done, 0));
            }
            b.src = src;
            b.n = int32_t(it.n);
            b.host_input = !it.device_src;
            HIP_TRY(prepare_branch(b, ls));
        }
        // ... and (from its second launch on) after the frame's canvas clear
        // (in stream order when the clear was enqueued on this stream)
        hipEvent_t clear_ev = clear_pending_ && clear_stream_ != ls ? ev_clear_ : nullptr;
        idle_ = false;
        // The group's launches serve every member: the first member's events
        // time them, mark their start and their end for all.
        for (int j = 0; j < m; ++j) {
            br_[agents[j]].ev_src = agents[0];
            br_[agents[j]].group_m = m;
        }
        // reached once every member's input copy and everything queued
        // before the group's encoders have completed: the encoders run
        HIP_TRY(hipEventRecord(lead.started, ls));
        rtcc_status st;
        const bool graphs = o_.use_graphs && !timing;
        // the encoders as one sequence of launches on ls: the pillar stage
        // and then every backbone layer over the whole group
        auto encoders = [&](hipStream_t c, bool t) {
            rtcc_status r = enqueue_pillars(agents, m, c, t, clear_ev, err);
            return r == RTCC_OK ? enqueue_backbone(agents, m, c, t, err) : r;
        };
        if (graphs) {
            // two graphs per branch released alone and for a group: the
            // pillar stage, whose arguments (the members, their inputs and
            // point counts) change from frame to frame, and the backbones,
            // whose buffers are fixed (their graph is updated only for other
            // members or, with branch warps, other poses)
            std::vector<unsigned char> kp, kb;
            for (int j = 0; j < m; ++j) {
                const Branch &b = br_[agents[j]];
                put(kp, agents[j]);
                put(kp, b.src);
                put(kp, b.n);
                put(kb, agents[j]);
                if (p_.d.warp_in_branch)
                    for (int e = 0; e < 6; ++e) put(kb, b.affine[e]);
            }
            // a captured graph cannot wait on the clear inside: it waits
            // before the graph launch
            Graph &pg = m == 1 ? lead.pillar_graph : group_pillar_graph_;
            if (graph_runs(pg, kp)) {
                if (clear_ev) HIP_TRY(hipStreamWaitEvent(ls, clear_ev, 0));
                st = run_graph(pg, kp, ls,
                               [&](hipStream_t c) { return enqueue_pillars(agents, m, c, false, nullptr, err); }, err);
            } else {
                pg.seen = kp;
                st = enqueue_pillars(agents, m, ls, false, clear_ev, err);
            }
            if (st == RTCC_OK)
                st = run_graph(m == 1 ? lead.graph : group_graph_, kb, ls,
                               [&](hipStream_t c) { return enqueue_backbone(agents, m, c, false, err); }, err);
        } else {
            st = encoders(ls, timing);
        }
        if (st != RTCC_OK) return st;
        HIP_TRY(hipEventRecord(lead.done, ls));
        for (int j = 0; j < m; ++j) {
            Branch &b = br_[agents[j]];
            b.canvas_dirty = true;  // the encoder writes this frame's pillars
            b.canvas_consumed = false;
            b.dispatched = true;
        }
        return RTCC_OK;
    }

    int progress(int agent) override {
        const Branch &b = br_[agent];
        if (!b.dispatched) return 0;
        const Branch &g = br_[b.ev_src];  // the launches that serve it
        if (hipEventQuery(g.done) == hipSuccess) return 2;
        return hipEventQuery(g.started) == hipSuccess ? 1 : 0;
    }

    rtcc_status join(const std::vector<std::array<float, 6>> &affine,
                     const std::vector<std::array<float, 3>> &poses, double t_begin, rtcc_detections *out,
                     std::string &err) override {
        HIP_TRY(hipSetDevice(dev_));
        hipStream_t js = compute_stream_for_join();
        const bool timing = o_.node_timing != 0;
        // A frame whose K encoders ran as one group launch: the post-join work
        // follows that launch on its stream (stream order instead of a wait
        // on its completion event from another queue).  Not with the
        // caller's join stream, node timing or the serial executor.
        const int src0 = br_[0].ev_src;
        bool one_launch = own_join_stream_ && !timing && o_.exec != RTCC_EXEC_SERIAL;
        for (int k = 0; k < p_.K && one_launch; ++k) one_launch = br_[k].ev_src == src0;
        if (one_launch) js = br_[src0].stream;
        // every distinct completion event (a group has one)
        for (int k = 0; k < p_.K && !one_launch; ++k)
            if (br_[k].ev_src == k || br_[br_[k].ev_src].ev_src != br_[k].ev_src)
                HIP_TRY(hipStreamWaitEvent(js, br_[br_[k].ev_src].done, 0));
        // one-kernel fusion nodes are timed by events bracketing the kernel
        if (timing && p_.d.multiscale) HIP_TRY(hipEventRecord(post_ev_[0], js));
        rtcc_status s;
        // the export kernel at the end of the post-join work sets this flag;
        // every export enqueued before has completed (joins wait for theirs,
        // node profiling synchronises)
        __atomic_store_n(static_cast<uint32_t *>(h_export) + 2, 0u, __ATOMIC_RELAXED);
        if (o_.use_graphs && !timing) {
            std::vector<unsigned char> key;
            for (int k = 0; k < p_.K; ++k) {
                put(key, br_[k].ego_map);
                for (int e = 0; e < 6; ++e) put(key, affine[k][e]);
                for (int e = 0; e < 3; ++e) put(key, poses[k][e]);
            }
            s = run_graph_or_eager(post_graph_[0], key, js,
                                   [&](hipStream_t c) { return enqueue_post_head(affine, poses, c, false, err); },
                                   err);
            if (s != RTCC_OK) return s;
            HIP_TRY(hipEventRecord(ev_head_, js));
            s = run_graph(post_graph_[1], {}, js, [&](hipStream_t c) { return enqueue_post_detect(c, false, err); },
                          err);
        } else {
            s = enqueue_post(affine, poses, js, timing, err);
        }
        if (s != RTCC_OK) return s;
        // The GPU is idle until the caller's next frame: its canvas pillars go
        // back to zero now, behind the export on the join stream, not at the
        // next frame's start (the canvas tensor is rebuilt when read).
        HIP_TRY(clear_dirty_canvases(true, js));
        // the counts and the first records are in h_export once the export
        // kernel has set the flag (no copy call in the common case; the clear
        // behind it is not waited for); the rest, if any, are copied after
        // them
        s = wait_export(js, err);
        if (s != RTCC_OK) return s;
        const int32_t *hs = static_cast<const int32_t *>(h_export);
        const int64_t decoded = hs[0];
        const int64_t count = nms_max_ > 0 ? hs[1] : decoded;
        if (decoded < 0 || size_t(decoded) > n_anchor_ || count < 0 || count > decoded ||
            (nms_max_ > 0 && count > nms_max_)) {
            err = "decode or NMS produced an out-of-range count";
            return RTCC_E_INTERNAL;
        }
        const size_t first = size_t(export_first_);
        const float *head_recs = reinterpret_cast<const float *>(static_cast<const char *>(h_export) + 64);
        if (size_t(count) > first) {
            const void *recs = nms_max_ > 0 ? d_nms_out : d_rec;
            HIP_TRY(hipMemcpyAsync(h_rec + first * 9, static_cast<const char *>(recs) + first * 36,
                                   (size_t(count) - first) * 36, hipMemcpyDeviceToHost, js));
            HIP_TRY(spin_sync(js));
        }
        idle_ = true;  // the frame's work has completed (the canvas clear may still run)
        for (int64_t i = 0; i < count; ++i) {
            const float *r = size_t(i) < first ? head_recs + i * 9 : h_rec + i * 9;
            std::memcpy(&boxes_[i * 7], r, 7 * sizeof(float));
            scores_[i] = r[7];
            std::memcpy(&aidx_[i], &r[8], 4);
        }
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, ev_frame0_, ev_head_));
        out->count = count;
        out->count_decoded = decoded;
        out->boxes = boxes_.data();
        out->scores = scores_.data();
        out->anchor_idx = aidx_.data();
        out->t_head_s = t_begin + 1e-3 * double(ms);
        last_affine_ = affine;
        last_poses_ = poses;
        return RTCC_OK;
    }

    rtcc_status tensor_bytes(int id, int agent, size_t *bytes, std::string &err) override {
        if (id == RTCC_T_PILLAR_MEMBERS) {
            std::vector<int32_t> m;
            rtcc_status s = used_members(agent, m, err);
            if (s == RTCC_OK) *bytes = m.size() * 4;
            return s;
        }
        void *ptr = nullptr;
        return locate(id, agent, &ptr, bytes, err, false);
    }

    rtcc_status get_tensor(int id, int agent, void *dst, size_t bytes, std::string &err) override {
        if (id == RTCC_T_PILLAR_MEMBERS) {
            std::vector<int32_t> m;
            rtcc_status s = used_members(agent, m, err);
            if (s != RTCC_OK) return s;
            if (bytes != m.size() * 4) {
                err = "destination size " + std::to_string(bytes) + " != tensor size " + std::to_string(m.size() * 4);
                return RTCC_E_ARG;
            }
            if (!m.empty()) std::memcpy(dst, m.data(), bytes);
            return RTCC_OK;
        }
        void *ptr = nullptr;
        size_t need = 0;
        rtcc_status s = locate(id, agent, &ptr, &need, err);
        if (s != RTCC_OK) return s;
        if (bytes != need) {
            err = "destination size " + std::to_string(bytes) + " != tensor size " + std::to_string(need);
            return RTCC_E_ARG;
        }
        if (need == 0) return RTCC_OK;
        HIP_TRY(hipMemcpyAsync(dst, ptr, need, hipMemcpyDeviceToHost, aux_stream_));
        HIP_TRY(hipStreamSynchronize(aux_stream_));
        return RTCC_OK;
    }

    rtcc_status profile_nodes(int warmup, int reps, float *median_ms, int *n_nodes,
                              std::string &err) override {
        HIP_TRY(hipSetDevice(dev_));
        for (const Branch &b : br_)
            if (!b.host_input) {
                err = "profiling replays a frame released from host memory";
                return RTCC_E_STATE;
            }
        hipStream_t s = join_stream_;
        hipEvent_t e0, e1;
        HIP_TRY(hipEventCreate(&e0));
        HIP_TRY(hipEventCreate(&e1));
        std::vector<std::vector<float>> t(p_.K + 1);
        for (int r = 0; r < warmup + reps; ++r) {
            for (int k = 0; k <= p_.K; ++k) {
                if (k < p_.K) HIP_TRY(prepare_branch(br_[k], s));
                HIP_TRY(hipEventRecord(e0, s));
                rtcc_status st;
                if (k < p_.K) {
                    st = enqueue_pillars(&k, 1, s, false, nullptr, err);
                    if (st == RTCC_OK) st = enqueue_backbone(&k, 1, s, false, err);
                } else {
                    st = enqueue_post(last_affine_, last_poses_, s, false, err);
                }
                if (st != RTCC_OK) return st;
                HIP_TRY(hipEventRecord(e1, s));
                if (k < p_.K) {
                    br_[k].canvas_dirty = true;
                    HIP_TRY(clear_canvases(&k, 1, s));  // untimed, as after a frame
                    br_[k].canvas_consumed = true;
                }
                HIP_TRY(hipEventSynchronize(e1));
                float ms = 0.f;
                HIP_TRY(hipEventElapsedTime(&ms, e0, e1));
                if (r >= warmup) t[k].push_back(ms);
            }
        }
        HIP_TRY(hipEventDestroy(e0));
        HIP_TRY(hipEventDestroy(e1));
        for (int k = 0; k <= p_.K; ++k) {
            std::vector<float> &v = t[k];
            std::sort(v.begin(), v.end());
            const size_t h = v.size() / 2;
            median_ms[k] = v.size() % 2 ? v[h] : 0.5f * (v[h - 1] + v[h]);
        }
        *n_nodes = p_.K + 1;
        return RTCC_OK;
    }

    int node_count() const override {
        return p_.K * int(3 + p_.convs.size() + (p_.ups.empty() ? 1 : p_.ups.size()) + 1) + 4;
    }

    // Events of a branch: ev[0] dispatch, ev[1] after the H2D copy, ev[2]
    // after the pillar stage, ev[3] after the PFN canvas, ev[4 + l] after
    // conv l, ev[4 + L + s] after upsampling s, ev[4 + L + S] after the warp.
    rtcc_status node_times(float *ms, int *n, std::string &err) override {
        int q = 0;
        const int L = int(p_.convs.size()), S = int(p_.ups.size());
        for (const Branch &b : br_) {
            float v = 0.f;
            // input copy, then the encoder's launches: shared by a group and
            // timed by the events of its first member, each member takes an
            // equal share (the members' shares add up to the launch)
            const Branch &g = br_[b.ev_src];
            const float share = 1.0f / float(b.group_m);
            HIP_TRY(hipEventElapsedTime(&v, b.ev[0], g.ev[1]));
            ms[q++] = v;
            for (int e = 1; e < 3; ++e) {
                HIP_TRY(hipEventElapsedTime(&v, g.ev[e], g.ev[e + 1]));
                ms[q++] = v * share;
            }
            for (int l = 0; l < L; ++l) {
                HIP_TRY(hipEventElapsedTime(&v, g.kev[2 * l], g.kev[2 * l + 1]));
                ms[q++] = v * share;
            }
            for (int u = 0; u < S; ++u) {
                v = 0.f;
                if (!p_.d.multiscale) HIP_TRY(hipEventElapsedTime(&v, g.ev[3 + L + u], g.ev[4 + L + u]));
                ms[q++] = v * share;
            }
            if (S == 0) ms[q++] = 0.f;
            v = 0.f;
            if (p_.d.warp_in_branch && b.warp_ran) HIP_TRY(hipEventElapsedTime(&v, b.wev[0], b.wev[1]));
            ms[q++] = v;
        }
        for (int e = 0; e < 4; ++e) {
            float v = 0.f;
            HIP_TRY(hipEventElapsedTime(&v, post_ev_[e], post_ev_[e + 1]));
            ms[q++] = v;
        }
        *n = q;
        return RTCC_OK;
    }

    bool conv_plan(int layer, int32_t out[2]) const override {
        if (layer < 0 || layer >= int(plans_.size())) return false;
        out[0] = plans_[layer].variant;
        out[1] = plans_[layer].splits;
        return true;
    }

    void graph_stats(int64_t out[3]) const override {
        for (int i = 0; i < 3; ++i) out[i] = graph_stats_[i];
    }

  private:
    // A captured sequence of kernel launches and the key (the arguments that
    // vary between frames) it was captured with.
    struct Graph {
        hipGraph_t g = nullptr;
        hipGraphExec_t x = nullptr;
        std::vector<unsigned char> key;
        std::vector<unsigned char> seen;  // the last key launched without the graph
    };
    static void drop(Graph &gr) {
        if (gr.x) (void)hipGraphExecDestroy(gr.x);
        if (gr.g) (void)hipGraphDestroy(gr.g);
        gr.x = nullptr;
        gr.g = nullptr;
        gr.key.clear();
        gr.seen.clear();
    }
    template <class T>
    static void put(std::vector<unsigned char> &key, const T &v) {
        const unsigned char *b = reinterpret_cast<const unsigned char *>(&v);
        key.insert(key.end(), b, b + sizeof(T));
    }
    // Launch `gr` on stream s.  If it was captured for another key, capture
    // the launches again on the capture stream and update the executable
    // graph in place (the same kernels with other arguments or grids); a
    // graph of another shape, or the first one, is instantiated.
    // `enqueue(stream)` issues kernel launches only (no memset, copy or wait).
    template <class F>
    rtcc_status run_graph(Graph &gr, const std::vector<unsigned char> &key, hipStream_t s, F &&enqueue,
                          std::string &err) {
        if (!gr.x || gr.key != key) {
            HIP_TRY(hipStreamBeginCapture(cap_stream_, hipStreamCaptureModeRelaxed));
            const rtcc_status st = enqueue(cap_stream_);
            hipGraph_t g = nullptr;
            const hipError_t e = hipStreamEndCapture(cap_stream_, &g);
            if (st != RTCC_OK || e != hipSuccess) {
                if (g) (void)hipGraphDestroy(g);
                drop(gr);
                if (st != RTCC_OK) return st;
                HIP_TRY(e);
            }
            bool updated = false;
            if (gr.x) {
                hipGraphNode_t bad = nullptr;
                hipGraphExecUpdateResult res = hipGraphExecUpdateError;
                updated = hipGraphExecUpdate(gr.x, g, &bad, &res) == hipSuccess && res == hipGraphExecUpdateSuccess;
                (void)hipGetLastError();
                ++graph_stats_[1];
            }
            if (updated) {
                (void)hipGraphDestroy(gr.g);
                gr.g = g;
            } else {
                drop(gr);
                gr.g = g;
                HIP_TRY(hipGraphInstantiate(&gr.x, g, nullptr, nullptr, 0));
                ++graph_stats_[0];
            }
            gr.key = key;
        }
        HIP_TRY(hipGraphLaunch(gr.x, s));
        ++graph_stats_[2];
        return RTCC_OK;
    }

    // For launches whose arguments may change every frame: replay the graph
    // when the key is the one it holds; capture (or update) it when the same
    // new key comes twice in a row; otherwise launch eagerly, which costs
    // less than a capture and an update that a stream of changing frames
    // would pay every frame.
    template <class F>
    rtcc_status run_graph_or_eager(Graph &gr, const std::vector<unsigned char> &key, hipStream_t s, F &&enqueue,
                                   std::string &err) {
        if (graph_runs(gr, key)) return run_graph(gr, key, s, enqueue, err);
        gr.seen = key;
        return enqueue(s);
    }
    // whether run_graph_or_eager runs the graph for this key
    static bool graph_runs(const Graph &gr, const std::vector<unsigned char> &key) {
        return (gr.x && gr.key == key) || gr.seen == key;
    }

    struct Branch {
        float *staging = nullptr;
        void *d_pts = nullptr, *d_cell = nullptr, *d_slot = nullptr, *d_member = nullptr;
        void *d_sorted = nullptr;  // points in segment (pillar) order
        void *d_pcells = nullptr, *d_pcounts = nullptr, *d_poffs = nullptr, *d_overfull = nullptr;
        void *d_ttotal = nullptr, *d_tstart = nullptr, *d_npil = nullptr, *d_meta = nullptr;
        void *d_binned = nullptr, *d_cellb = nullptr, *d_rank = nullptr;
        void *d_tcell = nullptr, *d_tcount = nullptr, *d_toff = nullptr;  // the tiles' pillar lists
        void *d_canvas = nullptr, *d_slotbuf = nullptr, *d_ws = nullptr;
        void *d_warped = nullptr;        // ego-frame map (warp in the branch)
        const void *ego_map = nullptr;   // what the fusion reads when the warp is in the branch
        float affine[6] = {1, 0, 0, 0, 1, 0};
        bool warp_ran = false;           // the last frame ran a branch warp kernel
        bool pillars_clean = true;       // every enqueued K1 was followed by the PFN kernel
        bool canvas_dirty = false;       // the canvas holds pillars not yet cleared (canvas_clear)
        // the last frame's pillars were cleared at the end of its join: the
        // canvas tensor is rebuilt from the pillar lists when read
        bool canvas_consumed = false;
        hipEvent_t wev[2] = {nullptr, nullptr};  // bracket the branch warp kernel
        Graph pillar_graph;              // its pillar stage as a HIP graph (use_graphs, released alone)
        Graph graph;                     // its backbone as a HIP graph (use_graphs, released alone)
        std::vector<void *> d_act;
        hipStream_t stream = nullptr;
        hipEvent_t done = nullptr, h2d_done = nullptr, started = nullptr;
        std::vector<hipEvent_t> ev;
        std::vector<hipEvent_t> kev;  // per conv layer: start / stop of its kernels
        const float *src = nullptr;
        int32_t n = 0;
        bool host_input = true;
        bool dispatched = false;
        int ev_src = 0;   // the branch whose events timed this one's encoder launches
        int group_m = 1;  // branches those launches served
    };

    hipStream_t compute_stream_for_join() const { return join_stream_; }

    // Until the export kernel of this join has set word 2 of h_export to 1
    // (acquire).  A stream error ends the wait with that error; a stream
    // that completes without the store (no export kernel ran) is an
    // internal error.
    rtcc_status wait_export(hipStream_t s, std::string &err) {
        const uint32_t *w = static_cast<const uint32_t *>(h_export) + 2;
        for (;;) {
            if (__atomic_load_n(w, __ATOMIC_ACQUIRE) == 1u) return RTCC_OK;
            const hipError_t e = hipStreamQuery(s);
            if (e == hipErrorNotReady) continue;
            HIP_TRY(e);
            if (__atomic_load_n(w, __ATOMIC_ACQUIRE) == 1u) return RTCC_OK;
            err = "the join stream completed without exporting the frame";
            return RTCC_E_INTERNAL;
        }
    }

    // Wait for a stream by polling: T^det is a latency measurement, and a
    // blocking wait adds the host's wake-up time to it.
    static hipError_t spin_sync(hipStream_t s) {
        for (;;) {
            const hipError_t e = hipStreamQuery(s);
            if (e != hipErrorNotReady) return e;
        }
    }

    hipError_t alloc(void **p, size_t bytes) {
        const size_t b = align256(bytes ? bytes : 1);
        if (o_.dev_alloc) {
            // the caller's allocator (e.g. PyTorch's caching allocator)
            *p = o_.dev_alloc(b, o_.alloc_user);
            if (!*p) return hipErrorOutOfMemory;
            dev_allocs_.push_back(*p);
            return hipSuccess;
        }
        hipError_t e = hipMalloc(p, b);
        if (e == hipSuccess) dev_allocs_.push_back(*p);
        return e;
    }
    template <class T>
    hipError_t alloc(T **p, size_t bytes) {
        return alloc(reinterpret_cast<void **>(p), bytes);
    }

    // Pillar stage of the encoders of `agents` (m of them, side by side in
    // every launch): cell ids, scans, scatter, PFN canvas.  With timing, each
    // member's node times for them are those of the first member's ev[1] /
    // ev[2] / ev[3].
    // With clear_ev, the launches after the first wait for it (the frame's
    // canvas clear reads the members' last pillar lists, which bin_scatter
    // and pillar_lists rewrite; bin_count runs beside it).
    rtcc_status enqueue_pillars(const int *agents, int m, hipStream_t s, bool timing, hipEvent_t clear_ev,
                                std::string &err) {
        const Plan &p = p_;
        const int n_cells = p.H * p.W;
        kern::PillarGroup grp{};
        grp.bufs = static_cast<const kern::PillarBufs *>(d_pbufs_);
        grp.m = m;
        grp.n_max = 0;
        grp.n_cells = n_cells;
        grp.tiles = tiles_;
        for (int j = 0; j < m; ++j) {
            const Branch &b = br_[agents[j]];
            grp.agent[j] = agents[j];
            grp.pts[j] = reinterpret_cast<const float4 *>(b.src);
            grp.n[j] = b.n;
            grp.n_max = std::max(grp.n_max, b.n);
        }
        auto mark = [&](int e) -> hipError_t {
            return timing ? hipEventRecord(br_[agents[0]].ev[e], s) : hipSuccess;
        };
        HIP_TRY(mark(1));
        kern::PillarGeom g{p.d.x_min, p.d.x_max, p.d.y_min, p.d.y_max, p.d.z_min, p.d.z_max,
                           p.d.pillar_size, p.H, p.W};
        // Between frames the canvas is zero outside the last frame's pillars
        // (prepare_branch).
        for (int j = 0; j < m; ++j) br_[agents[j]].pillars_clean = false;
        HIP_TRY(kern::bin_count(grp, g, s));
        if (clear_ev) HIP_TRY(hipStreamWaitEvent(s, clear_ev, 0));
        HIP_TRY(kern::bin_scatter(grp, s));
        HIP_TRY(kern::tile_sort(grp, p.d.max_points_per_pillar, s));
        HIP_TRY(kern::pillar_lists(grp, s));
        HIP_TRY(mark(2));

        HIP_TRY(kern::pfn_canvas(p.bf16, pfn_args(), grp, grp.n_max < n_cells ? grp.n_max : n_cells, s));
        for (int j = 0; j < m; ++j) br_[agents[j]].pillars_clean = true;
        HIP_TRY(mark(3));
        return RTCC_OK;
    }

    // Backbones of the encoders of `agents` (m of them) after their pillar
    // stage: every conv layer and every upsampling as one launch over the m
    // maps (GemmArgs::batch), which gives each map the bits of a launch of
    // its own; then the branch warps when the warp is the branches' last
    // node.  With timing, the first member's events bracket the shared
    // launches.
    rtcc_status enqueue_backbone(const int *agents, int m, hipStream_t s, bool timing, std::string &err) {
        const Plan &p = p_;
        Branch &lead = br_[agents[0]];
        int ev = 4;
        for (size_t l = 0; l < p.convs.size(); ++l) {
            const ConvLayer &c = p.convs[l];
            kern::GemmArgs ga{};
            ga.wt = static_cast<const char *>(d_mat) + c.w_off * p.elt;
            ga.bias = static_cast<const float *>(d_bias) + c.b_off;
            ga.Hi = c.Hi; ga.Wi = c.Wi; ga.Ci = c.Ci;
            ga.Ho = c.Ho; ga.Wo = c.Wo; ga.N = c.Co;
            ga.stride = c.stride;
            ga.u = 1;
            ga.ldo = c.Co;
            ga.c_off = 0;
            ga.splits = plans_[l].splits;
            ga.variant = kern::conv_variant_for(plans_[l], m);
            ga.zero = d_zero;
            ga.batch = m;
            for (int j = 0; j < m; ++j) {
                const Branch &b = br_[agents[j]];
                ga.in_b[j] = l == 0 ? b.d_canvas : b.d_act[l - 1];
                ga.out_b[j] = b.d_act[l];
                ga.ws_b[j] = static_cast<float *>(b.d_ws);
            }
            ga.in = ga.in_b[0];
            ga.out = ga.out_b[0];
            ga.ws = ga.ws_b[0];
            // with timing, conv nodes are timed by events bracketing their
            // kernels' execution (no dispatch gap)
            HIP_TRY(kern::conv3x3(p.bf16, ga, s, timing ? lead.kev[2 * l] : nullptr,
                                  timing ? lead.kev[2 * l + 1] : nullptr));
            if (timing) HIP_TRY(hipEventRecord(lead.ev[ev], s));
            ++ev;
        }
        for (const UpLayer &u : p.ups) {
            if (p.d.multiscale) break;  // upsampling runs once, on the fused maps
            const void *in[kern::kMaxGroup];
            void *out[kern::kMaxGroup];
            for (int j = 0; j < m; ++j) {
                in[j] = br_[agents[j]].d_act[p.stage_last_conv[u.stage]];
                out[j] = br_[agents[j]].d_slotbuf;
            }
            HIP_TRY(upsample(u, in, out, m, s));
            if (timing) HIP_TRY(hipEventRecord(lead.ev[ev], s));
            ++ev;
        }
        if (p.d.warp_in_branch) {
            for (int j = 0; j < m; ++j) {
                Branch &b = br_[agents[j]];
                // The identity pose (the ego agent) samples every cell exactly
                // at itself with weight 1, a copy: the fusion then reads the
                // slot.  (Compared by value: the identity's off-diagonal terms
                // may be -0.)
                static const float kIdentity[6] = {1, 0, 0, 0, 1, 0};
                b.warp_ran = false;
                for (int e = 0; e < 6; ++e) b.warp_ran |= b.affine[e] != kIdentity[e];
                if (!b.warp_ran) {
                    b.ego_map = b.d_slotbuf;
                } else {
                    kern::WarpSlotArgs wa{};
                    wa.slot = b.d_slotbuf;
                    for (int e = 0; e < 6; ++e) wa.affine[e] = b.affine[e];
                    wa.out = b.d_warped;
                    wa.H2 = p.H2;
                    wa.W2 = p.W2;
                    wa.C = p.c_slot;
                    HIP_TRY(kern::warp_slot(p.bf16, wa, s, timing ? b.wev[0] : nullptr,
                                            timing ? b.wev[1] : nullptr));
                    b.ego_map = b.d_warped;
                }
            }
        }
        return RTCC_OK;
    }

    // Before an encoder: the canvas must be zero outside the pillars the
    // encoder writes.  begin_frame clears the last frame's (clear_canvas);
    // should they still be there, they are cleared here.  If an earlier
    // enqueue stopped before the PFN kernel, the tiles' point totals and the
    // whole canvas are reset.  Runs outside any graph: what it enqueues
    // depends on the branch's state, not on the frame's arguments.
    hipError_t prepare_branch(Branch &b, hipStream_t s) {
        const int n_cells = p_.H * p_.W;
        hipError_t e = hipSuccess;
        if (!b.pillars_clean) {
            e = kern::fill_i32(static_cast<int32_t *>(b.d_ttotal), tiles_, 0, s);
            if (e == hipSuccess)
                e = kern::fill_i32(static_cast<int32_t *>(b.d_canvas), int64_t(n_cells) * p_.c_pfn * p_.elt / 4, 0, s);
            if (e != hipSuccess) return e;
            b.pillars_clean = true;
            b.canvas_dirty = false;
        }
        if (!b.canvas_dirty) return hipSuccess;
        const int agent = int(&b - br_.data());
        return clear_canvases(&agent, 1, s);
    }

    // Zero the canvas cells of the last pillars of the given branches (their
    // lists are the pillar stage's output of their last encoders) on stream
    // s, in one launch.
    hipError_t clear_canvases(const int *agents, int m, hipStream_t s) {
        const int n_cells = p_.H * p_.W;
        const int max_p = int(std::min<int64_t>(p_.n_max, n_cells));
        kern::PillarGroup grp{};
        grp.bufs = static_cast<const kern::PillarBufs *>(d_pbufs_);
        grp.m = m;
        for (int j = 0; j < m; ++j) grp.agent[j] = agents[j];
        hipError_t e = kern::canvas_clear(p_.bf16, grp, p_.c_pfn, max_p, s);
        if (e == hipSuccess)
            for (int j = 0; j < m; ++j) br_[agents[j]].canvas_dirty = false;
        return e;
    }

    // Upsampling u of the map `in` into channels [c_off, c_off + Co) of `out`
    // ([H2][W2][c_slot]).
    hipError_t upsample(const UpLayer &u, const void *const *in, void *const *out, int m, hipStream_t s) {
        const Plan &p = p_;
        kern::GemmArgs ga{};
        ga.wt = static_cast<const char *>(d_mat) + u.w_off * p.elt;
        ga.bias = static_cast<const float *>(d_bias) + u.b_off;
        ga.Hi = u.Hi; ga.Wi = u.Wi; ga.Ci = u.Ci;
        ga.Ho = p.H2; ga.Wo = p.W2; ga.N = u.Co;
        ga.stride = 1;
        ga.u = u.u;
        ga.ldo = p.c_slot;
        ga.c_off = u.c_off;
        ga.splits = 1;
        ga.variant = kern::kConvImplicit;
        ga.zero = d_zero;
        ga.ws = nullptr;
        ga.batch = m;
        for (int j = 0; j < m; ++j) {
            ga.in_b[j] = in[j];
            ga.out_b[j] = out[j];
            ga.ws_b[j] = nullptr;
        }
        ga.in = in[0];
        ga.out = out[0];
        return kern::deconv(p.bf16, ga, s);
    }

    // Post-join subgraph: warp + fusion and head, T^head, then decode and NMS.
    rtcc_status enqueue_post(const std::vector<std::array<float, 6>> &affine,
                             const std::vector<std::array<float, 3>> &poses, hipStream_t s, bool timing,
                             std::string &err) {
        rtcc_status st = enqueue_post_head(affine, poses, s, timing, err);
        if (st != RTCC_OK) return st;
        HIP_TRY(hipEventRecord(ev_head_, s));
        return enqueue_post_detect(s, timing, err);
    }

    rtcc_status enqueue_post_head(const std::vector<std::array<float, 6>> &affine,
                                  const std::vector<std::array<float, 3>> &poses, hipStream_t s, bool timing,
                                  std::string &err) {
        const Plan &p = p_;
        if (p.d.multiscale) {
            // every scale: warp the K stage maps onto the stage's ego grid and
            // fuse them, then upsample the fused map into the head's input
            for (const UpLayer &u : p.ups) {
                kern::WarpArgs wa{};
                for (int k = 0; k < p.K; ++k) {
                    wa.slots[k] = br_[k].d_act[p.stage_last_conv[u.stage]];
                    pose_affine_grid(p, poses[k].data(), u.Hi, u.Wi, wa.affine[k]);
                }
                wa.fused = d_fused_stage_[u.stage];
                wa.K = p.K;
                wa.ident = kern::identity_mask(wa.affine, p.K);
                wa.H2 = u.Hi;
                wa.W2 = u.Wi;
                wa.C = u.Ci;
                HIP_TRY(kern::warp_fuse(p.bf16, p.d.fusion == RTCC_FUSE_ATTN, wa, s));
                const void *fin = d_fused_stage_[u.stage];
                void *fout = d_fused;
                HIP_TRY(upsample(u, &fin, &fout, 1, s));
            }
        } else if (p.d.warp_in_branch) {
            kern::FuseArgs fa{};
            for (int k = 0; k < p.K; ++k) fa.maps[k] = br_[k].ego_map;
            fa.fused = d_fused;
            fa.K = p.K;
            fa.cells = p.H2 * p.W2;
            fa.C = p.c_slot;
            HIP_TRY(kern::fuse(p.bf16, p.d.fusion == RTCC_FUSE_ATTN, fa, s, timing ? post_ev_[0] : nullptr,
                               timing ? post_ev_[1] : nullptr));
        } else {
            kern::WarpArgs wa{};
            for (int k = 0; k < p.K; ++k) {
                wa.slots[k] = br_[k].d_slotbuf;
                for (int e = 0; e < 6; ++e) wa.affine[k][e] = affine[k][e];
            }
            wa.fused = d_fused;
            wa.K = p.K;
            wa.ident = kern::identity_mask(wa.affine, p.K);
            wa.H2 = p.H2;
            wa.W2 = p.W2;
            wa.C = p.c_slot;
            HIP_TRY(kern::warp_fuse(p.bf16, p.d.fusion == RTCC_FUSE_ATTN, wa, s, timing ? post_ev_[0] : nullptr,
                                    timing ? post_ev_[1] : nullptr));
        }
        if (timing && p.d.multiscale) HIP_TRY(hipEventRecord(post_ev_[1], s));
        HIP_TRY(kern::head1x1(p.bf16, d_fused, static_cast<const char *>(d_mat) + p.head_w_off * p.elt,
                              static_cast<const float *>(d_bias) + p.head_b_off, static_cast<float *>(d_head),
                              p.H2 * p.W2, p.c_slot, p.d.score_logit_threshold,
                              static_cast<int32_t *>(d_head_counts), s));
        if (timing) HIP_TRY(hipEventRecord(post_ev_[2], s));
        return RTCC_OK;
    }

    rtcc_status enqueue_post_detect(hipStream_t s, bool timing, std::string &err) {
        const Plan &p = p_;
        kern::DecodeArgs da{};
        da.head = static_cast<const float *>(d_head);
        da.H2 = p.H2;
        da.W2 = p.W2;
        da.thr = p.d.score_logit_threshold;
        da.x0 = p.d.x_min;
        da.y0 = p.d.y_min;
        da.dx = float((double(p.d.x_max) - double(p.d.x_min)) / p.W2);
        da.dy = float((double(p.d.y_max) - double(p.d.y_min)) / p.H2);
        da.aw = p.d.anchor_w;
        da.al = p.d.anchor_l;
        da.ah = p.d.anchor_h;
        da.az = p.d.anchor_z;
        da.ayaw0 = p.d.anchor_yaw[0];
        da.ayaw1 = p.d.anchor_yaw[1];
        da.head_counts = static_cast<const int32_t *>(d_head_counts);
        da.rec = static_cast<float *>(d_rec);
        da.count = static_cast<int32_t *>(d_count);
        HIP_TRY(kern::decode(da, s));
        if (timing) HIP_TRY(hipEventRecord(post_ev_[3], s));
        if (nms_max_ > 0) {
            kern::NmsArgs na{};
            na.rec = static_cast<const float *>(d_rec);
            na.count = static_cast<const int32_t *>(d_count);
            na.rank = static_cast<int32_t *>(d_nms_rank);
            na.flag = static_cast<int32_t *>(d_nms_flag);
            na.order = static_cast<int32_t *>(d_nms_order);
            na.foot = static_cast<double *>(d_nms_foot);
            na.mask = static_cast<unsigned long long *>(d_nms_mask);
            na.mask_t = static_cast<unsigned long long *>(d_nms_mask_t);
            na.partial = static_cast<int32_t *>(d_nms_partial);
            na.colrows = static_cast<int32_t *>(d_nms_colrows);
            na.colcount = static_cast<int32_t *>(d_nms_colcount);
            na.out = static_cast<float *>(d_nms_out);
            na.out_count = static_cast<int32_t *>(d_nms_count);
            na.iou_threshold = double(p.d.nms_iou_threshold);
            na.max_candidates = nms_max_;
            HIP_TRY(kern::rotated_nms(na, int64_t(n_anchor_), s));
        }
        if (timing) HIP_TRY(hipEventRecord(post_ev_[4], s));
        HIP_TRY(kern::export_results(static_cast<const int32_t *>(d_count),
                                     nms_max_ > 0 ? static_cast<const int32_t *>(d_nms_count) : nullptr,
                                     static_cast<const float *>(nms_max_ > 0 ? d_nms_out : d_rec), export_first_,
                                     h_export, s));
        return RTCC_OK;
    }

    // The points each pillar of the agent's last frame fed to the PFN: the
    // first min(count, cap) entries of its member segment (the overfull
    // selection moved the lowest indices there), sorted per pillar, pillars
    // in ascending cell order.
    rtcc_status used_members(int agent, std::vector<int32_t> &out, std::string &err) {
        if (agent < 0 || agent >= p_.K) {
            err = "agent out of range";
            return RTCC_E_ARG;
        }
        HIP_TRY(hipSetDevice(dev_));
        const Branch &b = br_[agent];
        int32_t meta[3] = {0, 0, 0};
        HIP_TRY(hipMemcpyAsync(meta, b.d_meta, 12, hipMemcpyDeviceToHost, aux_stream_));
        HIP_TRY(hipStreamSynchronize(aux_stream_));
        const int32_t valid = meta[0], P = meta[1];
        if (valid < 0 || valid > b.n || P < 0 || P > valid) {
            err = "pillar metadata out of range";
            return RTCC_E_INTERNAL;
        }
        std::vector<int32_t> cnt(P), off(P), mem(valid);
        if (P > 0) {
            HIP_TRY(hipMemcpyAsync(cnt.data(), b.d_pcounts, size_t(P) * 4, hipMemcpyDeviceToHost, aux_stream_));
            HIP_TRY(hipMemcpyAsync(off.data(), b.d_poffs, size_t(P) * 4, hipMemcpyDeviceToHost, aux_stream_));
            HIP_TRY(hipMemcpyAsync(mem.data(), b.d_member, size_t(valid) * 4, hipMemcpyDeviceToHost, aux_stream_));
            HIP_TRY(hipStreamSynchronize(aux_stream_));
        }
        const int cap = p_.d.max_points_per_pillar;
        out.clear();
        for (int32_t q = 0; q < P; ++q) {
            const int32_t m = std::min(cnt[q], cap);
            if (m < 1 || off[q] < 0 || int64_t(off[q]) + cnt[q] > valid) {
                err = "pillar segment out of range";
                return RTCC_E_INTERNAL;
            }
            const size_t at = out.size();
            out.insert(out.end(), mem.begin() + off[q], mem.begin() + off[q] + m);
            std::sort(out.begin() + at, out.end());
        }
        return RTCC_OK;
    }

    // The canvas of the agent's last frame, whose pillars were cleared after
    // its join, rebuilt into a buffer of its own: the PFN kernel again over
    // the last pillar lists, the points over the cap as that frame selected
    // them (replay), into a zeroed canvas.  Bit for bit the canvas the first
    // conv layer read.
    rtcc_status rebuild_canvas(int agent, void **ptr, std::string &err) {
        const Plan &p = p_;
        const int n_cells = p.H * p.W;
        const size_t bytes = size_t(n_cells) * p.c_pfn * p.elt;
        HIP_TRY(hipSetDevice(dev_));
        if (!d_canvas_view_) HIP_TRY(alloc(&d_canvas_view_, bytes));
        // after the clear, which reads the same pillar lists
        HIP_TRY(hipStreamSynchronize(clear_stream_ ? clear_stream_ : join_stream_));
        HIP_TRY(kern::fill_i32(static_cast<int32_t *>(d_canvas_view_), int64_t(bytes / 4), 0, aux_stream_));
        const Branch &b = br_[agent];
        kern::PillarGroup grp{};
        grp.bufs = static_cast<const kern::PillarBufs *>(d_pbufs_);
        grp.m = 1;
        grp.agent[0] = agent;
        grp.pts[0] = nullptr;  // not read in replay
        grp.n[0] = b.n;
        grp.n_max = b.n;
        grp.n_cells = n_cells;
        grp.tiles = tiles_;
        kern::PfnArgs pa = pfn_args();
        pa.replay = 1;
        pa.canvas = d_canvas_view_;
        HIP_TRY(kern::pfn_canvas(p.bf16, pa, grp, grp.n_max < n_cells ? grp.n_max : n_cells, aux_stream_));
        HIP_TRY(hipStreamSynchronize(aux_stream_));
        *ptr = d_canvas_view_;
        return RTCC_OK;
    }

    kern::PfnArgs pfn_args() const {
        const Plan &p = p_;
        kern::PfnArgs pa{};
        pa.w = static_cast<const float *>(d_bias) + p.pfn_w_off;
        pa.b = static_cast<const float *>(d_bias) + p.pfn_b_off;
        pa.C = p.c_pfn;
        pa.max_pts = p.d.max_points_per_pillar;
        pa.inv_hx = float(2.0 / (double(p.d.x_max) - double(p.d.x_min)));
        pa.inv_hy = float(2.0 / (double(p.d.y_max) - double(p.d.y_min)));
        pa.z0 = p.d.z_min;
        pa.inv_dz = float(1.0 / (double(p.d.z_max) - double(p.d.z_min)));
        return pa;
    }

    // *ptr, *bytes: where tensor id of the agent is on the device and its size
    // (with data false only the size is needed)
    rtcc_status locate(int id, int agent, void **ptr, size_t *bytes, std::string &err, bool data = true) {
        const Plan &p = p_;
        const bool per_agent = id == RTCC_T_PILLAR_CELLS || id == RTCC_T_PILLAR_COUNTS ||
                               id == RTCC_T_CANVAS || id == RTCC_T_SLOT || id == RTCC_T_WARPED;
        int stage = 0;
        if (id == RTCC_T_CONV_OUT) {
            const int layer = agent >> 8;
            agent &= 255;
            if (layer < 0 || layer >= int(p.convs.size()) || agent < 0 || agent >= p.K) {
                err = "conv layer or agent out of range";
                return RTCC_E_ARG;
            }
            const ConvLayer &c = p.convs[layer];
            *ptr = br_[agent].d_act[layer];
            *bytes = size_t(c.Ho) * c.Wo * c.Co * p.elt;
            return RTCC_OK;
        }
        if (id == RTCC_T_STAGE_OUT) {
            stage = agent >> 8;
            agent &= 255;
            if (stage < 0 || stage >= int(p.stage_last_conv.size())) {
                err = "stage out of range";
                return RTCC_E_ARG;
            }
        }
        if ((per_agent || id == RTCC_T_STAGE_OUT) && (agent < 0 || agent >= p.K)) {
            err = "agent out of range";
            return RTCC_E_ARG;
        }
        switch (id) {
            case RTCC_T_PILLAR_CELLS:
            case RTCC_T_PILLAR_COUNTS: {
                HIP_TRY(hipSetDevice(dev_));
                HIP_TRY(hipMemcpyAsync(h_small, br_[agent].d_meta, 12, hipMemcpyDeviceToHost, aux_stream_));
                HIP_TRY(hipStreamSynchronize(aux_stream_));
                const int32_t P = reinterpret_cast<int32_t *>(h_small)[1];
                *ptr = id == RTCC_T_PILLAR_CELLS ? br_[agent].d_pcells : br_[agent].d_pcounts;
                *bytes = size_t(P) * 4;
                return RTCC_OK;
            }
            case RTCC_T_CANVAS:
                *bytes = size_t(p.H) * p.W * p.c_pfn * p.elt;
                if (!br_[agent].canvas_consumed || !data) {
                    *ptr = br_[agent].d_canvas;
                    return RTCC_OK;
                }
                return rebuild_canvas(agent, ptr, err);
            case RTCC_T_SLOT:
                if (p.d.multiscale) {
                    err = "multi-scale fusion: the branch ends at its stage outputs (no slot)";
                    return RTCC_E_ARG;
                }
                *ptr = br_[agent].d_slotbuf;
                *bytes = size_t(p.H2) * p.W2 * p.c_slot * p.elt;
                return RTCC_OK;
            case RTCC_T_WARPED:
                if (!p.d.warp_in_branch) {
                    err = "no ego-frame maps: the warp is not in the branches";
                    return RTCC_E_ARG;
                }
                *ptr = const_cast<void *>(br_[agent].ego_map);
                *bytes = size_t(p.H2) * p.W2 * p.c_slot * p.elt;
                return RTCC_OK;
            case RTCC_T_FUSED_STAGE: {
                if (!p.d.multiscale || agent < 0 || agent >= int(p.ups.size())) {
                    err = "no fused stage map (needs multiscale = 1 and a stage index)";
                    return RTCC_E_ARG;
                }
                const UpLayer &u = p.ups[agent];
                *ptr = d_fused_stage_[u.stage];
                *bytes = size_t(u.Hi) * u.Wi * u.Ci * p.elt;
                return RTCC_OK;
            }
            case RTCC_T_FUSED:
                *ptr = d_fused;
                *bytes = size_t(p.H2) * p.W2 * p.c_slot * p.elt;
                return RTCC_OK;
            case RTCC_T_HEAD:
                *ptr = d_head;
                *bytes = size_t(p.H2) * p.W2 * 16 * 4;
                return RTCC_OK;
            case RTCC_T_STAGE_OUT: {
                const ConvLayer &c = p.convs[p.stage_last_conv[stage]];
                *ptr = br_[agent].d_act[p.stage_last_conv[stage]];
                *bytes = size_t(c.Ho) * c.Wo * c.Co * p.elt;
                return RTCC_OK;
            }
            case RTCC_T_DECODED: {
                HIP_TRY(hipSetDevice(dev_));
                HIP_TRY(hipMemcpyAsync(h_small, d_count, 4, hipMemcpyDeviceToHost, aux_stream_));
                HIP_TRY(hipStreamSynchronize(aux_stream_));
                const int32_t n = reinterpret_cast<int32_t *>(h_small)[0];
                if (n < 0 || size_t(n) > n_anchor_) {
                    err = "decoded count out of range";
                    return RTCC_E_INTERNAL;
                }
                *ptr = d_rec;
                *bytes = size_t(n) * 9 * 4;
                return RTCC_OK;
            }
        }
        err = "unknown tensor id";
        return RTCC_E_ARG;
    }

    void release_all() {
        if (dev_ < 0) return;
        // Teardown is best effort: errors cannot be reported from a destructor.
        (void)hipSetDevice(dev_);
        (void)hipDeviceSynchronize();
        for (Branch &b : br_) {
            if (b.staging) (void)hipHostFree(b.staging);
            if (b.stream) (void)hipStreamDestroy(b.stream);
            if (b.done) (void)hipEventDestroy(b.done);
            if (b.h2d_done) (void)hipEventDestroy(b.h2d_done);
            if (b.started) (void)hipEventDestroy(b.started);
            for (hipEvent_t e : b.ev)
                if (e) (void)hipEventDestroy(e);
            for (hipEvent_t e : b.kev)
                if (e) (void)hipEventDestroy(e);
            for (hipEvent_t e : b.wev)
                if (e) (void)hipEventDestroy(e);
            drop(b.graph);
            drop(b.pillar_graph);
        }
        drop(group_graph_);
        drop(group_pillar_graph_);
        if (ev_clear_) (void)hipEventDestroy(ev_clear_);
        for (void *ptr : dev_allocs_) {
            if (o_.dev_alloc) o_.dev_free(ptr, o_.alloc_user);
            else (void)hipFree(ptr);
        }
        if (h_rec) (void)hipHostFree(h_rec);
        if (h_small) (void)hipHostFree(h_small);
        if (h_export) (void)hipHostFree(h_export);
        if (join_stream_ && own_join_stream_) (void)hipStreamDestroy(join_stream_);
        if (copy_stream_) (void)hipStreamDestroy(copy_stream_);
        if (aux_stream_) (void)hipStreamDestroy(aux_stream_);
        for (Graph &g : post_graph_) drop(g);
        if (cap_stream_) (void)hipStreamDestroy(cap_stream_);
        if (ev_frame0_) (void)hipEventDestroy(ev_frame0_);
        if (ev_head_) (void)hipEventDestroy(ev_head_);
        for (hipEvent_t e : post_ev_)
            if (e) (void)hipEventDestroy(e);
    }

    Plan p_;
    rtcc_runtime_opts o_{};
    int dev_ = -1;
    std::vector<Branch> br_;
    std::vector<void *> dev_allocs_;
    void *d_mat = nullptr, *d_bias = nullptr, *d_zero = nullptr;
    std::vector<kern::ConvPlan> plans_;
    void *d_fused = nullptr, *d_head = nullptr, *d_head_counts = nullptr, *d_rec = nullptr, *d_count = nullptr;
    int nms_max_ = 0;  // 0: no NMS
    void *d_nms_rank = nullptr, *d_nms_flag = nullptr, *d_nms_order = nullptr, *d_nms_foot = nullptr;
    void *d_nms_mask = nullptr, *d_nms_out = nullptr, *d_nms_count = nullptr;
    void *d_nms_mask_t = nullptr, *d_nms_partial = nullptr, *d_nms_colrows = nullptr, *d_nms_colcount = nullptr;
    float *h_rec = nullptr;
    void *h_small = nullptr;
    void *h_export = nullptr;  // counts + first records of the frame (export_results)
    int export_first_ = 0;
    size_t n_anchor_ = 0;
    std::vector<float> boxes_, scores_;
    std::vector<int32_t> aidx_;
    hipStream_t join_stream_ = nullptr, copy_stream_ = nullptr, aux_stream_ = nullptr;
    bool own_join_stream_ = true;  // false: the caller's stream (opts.join_stream)
    hipStream_t clear_stream_ = nullptr;  // the stream of the last canvas clear
    hipEvent_t ev_frame0_ = nullptr, ev_head_ = nullptr;
    hipEvent_t post_ev_[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
    std::vector<std::array<float, 6>> last_affine_;
    std::vector<std::array<float, 3>> last_poses_;
    std::vector<void *> d_fused_stage_;  // multi-scale: fused map of every stage
    hipStream_t cap_stream_ = nullptr;   // where graphs are captured (use_graphs)
    void *d_canvas_view_ = nullptr;      // a rebuilt canvas (tensor reads)
    Graph post_graph_[2];                // post-join: up to T^head, then decode and NMS
    Graph group_graph_;                  // the backbones of a group of branches
    Graph group_pillar_graph_;           // the pillar stage of a group of branches
    hipEvent_t ev_clear_ = nullptr;      // the frame's canvas clear is done
    bool clear_pending_ = false;         // encoder launches must wait for ev_clear_
    bool idle_ = true;                   // no work queued since the last completed join
    static constexpr size_t kFirstRecords = 1024;  // records read back with the counts
    void *d_pbufs_ = nullptr;            // kern::PillarBufs of every agent
    int tiles_ = 0;                      // tiles of cells of the pillar sort
    int64_t graph_stats_[3] = {0, 0, 0}; // instantiations, update attempts, launches
};

Executor *make_executor() { return new HipExecutor(); }

}  // namespace rtcc
