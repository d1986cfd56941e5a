// Recording executor for host-only tests of the controller and the C ABI.
// It allocates no GPU resources and computes nothing: every call appends a
// line to a log that tests read through rtcc_hosttest_log().  This file is
// linked only into the host test library, never into the GPU library.
#include <cstring>
#include <mutex>
#include <sstream>

#include "controller.hpp"

namespace rtcc {

namespace {
std::mutex g_log_mu;
std::string g_log;
// What the recording executor reports as device progress of each agent's
// encoder (set by tests), and agents whose next dispatch fails.
int g_progress[RTCC_MAX_AGENTS] = {};
bool g_fail_dispatch[RTCC_MAX_AGENTS] = {};
void log_line(const std::string &s) {
    std::lock_guard<std::mutex> lk(g_log_mu);
    g_log += s;
    g_log += '\n';
}
}  // namespace

class FakeExecutor : public Executor {
  public:
    rtcc_status init(const Plan &p, const HostWeights &hw, const rtcc_runtime_opts &o,
                     std::string &) override {
        plan_ = p;
        staging_.assign(p.K, std::vector<float>(size_t(p.n_max) * 4, 0.f));
        std::ostringstream os;
        os << "init K=" << p.K << " H=" << p.H << " W=" << p.W << " H2=" << p.H2 << " W2=" << p.W2
           << " C=" << p.c_slot << " convs=" << p.convs.size() << " ups=" << p.ups.size()
           << " exec=" << o.exec << " weights_fnv=" << std::hex << weights_digest(hw) << std::dec;
        log_line(os.str());
        return RTCC_OK;
    }
    float *staging(int agent) override { return staging_[agent].data(); }
    // FNV-1a (64-bit) over the prepared weight bytes: equal prepared weights
    // give equal digests, so tests can tell which weights a context got
    static uint64_t weights_digest(const HostWeights &hw) {
        uint64_t h = 1469598103934665603ull;
        auto eat = [&](const void *p, size_t n) {
            const unsigned char *b = static_cast<const unsigned char *>(p);
            for (size_t i = 0; i < n; ++i) h = (h ^ b[i]) * 1099511628211ull;
        };
        eat(hw.bias.data(), hw.bias.size() * sizeof(float));
        eat(hw.mat_bf16.data(), hw.mat_bf16.size() * sizeof(uint16_t));
        eat(hw.mat_f32.data(), hw.mat_f32.size() * sizeof(float));
        return h;
    }
    rtcc_status begin_frame(std::string &) override {
        log_line("begin_frame");
        return RTCC_OK;
    }
    rtcc_status dispatch(const DispatchItem *items, int m, std::string &err) override {
        {
            std::lock_guard<std::mutex> lk(g_log_mu);
            for (int j = 0; j < m; ++j) g_progress[items[j].agent] = 0;
            for (int j = 0; j < m; ++j)
                if (g_fail_dispatch[items[j].agent]) {
                    g_fail_dispatch[items[j].agent] = false;
                    err = "injected dispatch failure";
                    return RTCC_E_HIP;
                }
        }
        if (m > 1) {
            std::ostringstream os;
            os << "group";
            for (int j = 0; j < m; ++j) os << " " << items[j].agent;
            log_line(os.str());
        }
        for (int j = 0; j < m; ++j) {
            const DispatchItem &it = items[j];
            const float *affine = it.affine;
            std::ostringstream os;
            os << "dispatch " << it.agent << " n=" << it.n << " src=" << (it.device_src ? "device" : "staging")
               << " staged=" << (it.pts == staging_[it.agent].data() ? 1 : 0) << " affine=[" << affine[0] << ","
               << affine[1] << "," << affine[2] << "," << affine[3] << "," << affine[4] << "," << affine[5] << "]";
            log_line(os.str());
        }
        return RTCC_OK;
    }
    int progress(int agent) override {
        std::lock_guard<std::mutex> lk(g_log_mu);
        return g_progress[agent];
    }
    rtcc_status join(const std::vector<std::array<float, 6>> &affine, const std::vector<std::array<float, 3>> &,
                     double, rtcc_detections *out, std::string &) override {
        std::ostringstream os;
        os << "join";
        for (const auto &m : affine)
            os << " [" << m[0] << "," << m[1] << "," << m[2] << "," << m[3] << "," << m[4] << ","
               << m[5] << "]";
        log_line(os.str());
        out->count = 0;
        out->count_decoded = 0;
        return RTCC_OK;
    }
    rtcc_status tensor_bytes(int, int, size_t *, std::string &err) override {
        err = "no tensors in the recording executor";
        return RTCC_E_STATE;
    }
    rtcc_status get_tensor(int, int, void *, size_t, std::string &err) override {
        err = "no tensors in the recording executor";
        return RTCC_E_STATE;
    }
    rtcc_status profile_nodes(int, int, float *, int *, std::string &err) override {
        err = "no profiling in the recording executor";
        return RTCC_E_STATE;
    }
    int node_count() const override { return 0; }
    rtcc_status node_times(float *, int *n, std::string &) override {
        *n = 0;
        return RTCC_OK;
    }

  private:
    Plan plan_;
    std::vector<std::vector<float>> staging_;
};

Executor *make_executor() { return new FakeExecutor(); }

}  // namespace rtcc

extern "C" __attribute__((visibility("default"))) size_t rtcc_hosttest_log(char *buf, size_t cap, int clear) {
    std::lock_guard<std::mutex> lk(rtcc::g_log_mu);
    size_t n = rtcc::g_log.size();
    if (buf && cap) {
        size_t m = n < cap - 1 ? n : cap - 1;
        std::memcpy(buf, rtcc::g_log.data(), m);
        buf[m] = 0;
    }
    if (clear) rtcc::g_log.clear();
    return n;
}

// Device progress the recording executor reports for `agent` (0 enqueued,
// 1 started, 2 finished) until its next dispatch.
extern "C" __attribute__((visibility("default"))) void rtcc_hosttest_set_progress(int agent, int progress) {
    std::lock_guard<std::mutex> lk(rtcc::g_log_mu);
    if (agent >= 0 && agent < RTCC_MAX_AGENTS) rtcc::g_progress[agent] = progress;
}

// The next dispatch of `agent` fails with RTCC_E_HIP.
extern "C" __attribute__((visibility("default"))) void rtcc_hosttest_fail_dispatch(int agent) {
    std::lock_guard<std::mutex> lk(rtcc::g_log_mu);
    if (agent >= 0 && agent < RTCC_MAX_AGENTS) rtcc::g_fail_dispatch[agent] = true;
}

namespace rtcc {
void set_thread_error(const std::string &msg);
}

// The recording library has no GPU: the context-free NMS entry point only
// reports that.
extern "C" __attribute__((visibility("default"))) rtcc_status rtcc_rotated_nms(const float *, int64_t, int32_t,
                                                                              float, float *, int64_t *kept) {
    if (kept) *kept = 0;
    rtcc::set_thread_error("rtcc_rotated_nms needs the GPU library");
    return RTCC_E_STATE;
}

extern "C" __attribute__((visibility("default"))) rtcc_status rtcc_rotated_nms_noalloc(const float *, int64_t, int32_t,
                                                                                      float, float *, int64_t *kept,
                                                                                      void *) {
    if (kept) *kept = 0;
    rtcc::set_thread_error("rtcc_rotated_nms_noalloc needs the GPU library");
    return RTCC_E_STATE;
}
