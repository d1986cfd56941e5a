// Concurrency and memory stress of the C ABI's release controller, linked
// against the recording executor and built with a sanitizer (thread or
// address) by tests/test_sanitizers.py.  Completion events of different
// agents arrive on different threads (Sec. IV-C requires the controller to
// update z_k atomically), while another thread polls branch states; every
// frame is joined, or found infeasible, and checked.
//
// usage: abi_stress <descriptor.bin> <weights.bin> <frames>
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <ctime>
#include <thread>
#include <vector>

#include "rtcc.h"

extern "C" void rtcc_hosttest_set_progress(int agent, int progress);
extern "C" void rtcc_hosttest_fail_dispatch(int agent);
extern "C" size_t rtcc_hosttest_log(char *buf, size_t cap, int clear);

namespace {

std::vector<char> read_file(const char *path) {
    std::vector<char> v;
    FILE *f = std::fopen(path, "rb");
    if (!f) return v;
    char buf[4096];
    size_t n;
    while ((n = std::fread(buf, 1, sizeof(buf), f)) > 0) v.insert(v.end(), buf, buf + n);
    std::fclose(f);
    return v;
}

double now_s() {
    timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return double(ts.tv_sec) + 1e-9 * double(ts.tv_nsec);
}

int g_failures = 0;
#define CHECK(cond)                                                            \
    do {                                                                       \
        if (!(cond)) {                                                         \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
            ++g_failures;                                                      \
        }                                                                      \
    } while (0)

}  // namespace

int main(int argc, char **argv) {
    if (argc != 4) {
        std::fprintf(stderr, "usage: %s descriptor.bin weights.bin frames\n", argv[0]);
        return 2;
    }
    const std::vector<char> db = read_file(argv[1]), wb = read_file(argv[2]);
    if (db.size() != sizeof(rtcc_model_desc) || wb.empty()) {
        std::fprintf(stderr, "bad inputs (descriptor %zu bytes, expected %zu)\n", db.size(), sizeof(rtcc_model_desc));
        return 2;
    }
    rtcc_model_desc d;
    std::memcpy(&d, db.data(), sizeof(d));
    const int frames = std::atoi(argv[3]);
    const int K = d.n_agents;
    rtcc_ctx *ctx = nullptr;
    if (rtcc_create(&d, wb.data(), wb.size(), nullptr, &ctx) != RTCC_OK) {
        std::fprintf(stderr, "create failed: %s\n", rtcc_last_error(nullptr));
        return 1;
    }
    const int64_t n = 64;
    std::vector<std::vector<float>> pts(K, std::vector<float>(size_t(n) * 4, 0.5f));
    const float pose[3] = {0.25f, 1.0f, -2.0f};

    for (int f = 0; f < frames; ++f) {
        const int mode = f % 2 ? RTCC_MODE_BARRIER : RTCC_MODE_RELEASE;
        CHECK(rtcc_set_mode(ctx, rtcc_mode(mode)) == RTCC_OK);
        CHECK(rtcc_begin_frame(ctx, now_s() - 1.0) == RTCC_OK);
        // every 5th frame leaves one agent undelivered, every 7th injects a
        // failed dispatch
        const int missing = f % 5 == 4 ? f % K : -1;
        const int failing = f % 7 == 6 && missing < 0 ? (f / 7) % K : -1;
        if (failing >= 0) rtcc_hosttest_fail_dispatch(failing);
        std::atomic<bool> stop{false};
        std::thread poller([&] {
            int32_t st = 0;
            while (!stop.load()) {
                for (int k = 0; k < K; ++k) {
                    if (rtcc_get_branch_state(ctx, k, &st) == RTCC_OK) CHECK(st >= RTCC_WAITING && st <= RTCC_FINISHED);
                    rtcc_hosttest_set_progress(k, (f + k) % 3);
                }
            }
        });
        std::vector<std::thread> th;
            for (int k = 0; k < K; ++k) {
            if (k == missing) continue;
            th.emplace_back([&, k] {
                // a duplicate from a second thread races the first event
                std::thread dup([&] {
                    (void)rtcc_release_branch(ctx, k, pts[k].data(), n, pose, 0.0);
                });
                (void)rtcc_release_branch(ctx, k, pts[k].data(), n, pose, 0.0);
                dup.join();
            });
        }
        for (auto &t : th) t.join();
        stop = true;
        poller.join();
        rtcc_detections out;
        const rtcc_status js = rtcc_join_and_detect(ctx, &out);
        if (missing >= 0) {
            CHECK(js == RTCC_E_INFEASIBLE);
        } else if (failing >= 0) {
            // every input arrived, so the failing agent's encoder was
            // dispatched (by its own event, or in barrier mode by whichever
            // event came last) and failed: the join is withheld
            CHECK(js == RTCC_E_STATE);
        } else {
            CHECK(js == RTCC_OK);
            int32_t st = 0;
            for (int k = 0; k < K; ++k) {
                CHECK(rtcc_get_branch_state(ctx, k, &st) == RTCC_OK);
                CHECK(st == RTCC_FINISHED);
            }
        }
        rtcc_hosttest_log(nullptr, 0, 1);
    }
    rtcc_destroy(ctx);
    if (g_failures) {
        std::fprintf(stderr, "%d checks failed\n", g_failures);
        return 1;
    }
    std::printf("abi_stress: %d frames ok\n", frames);
    return 0;
}
