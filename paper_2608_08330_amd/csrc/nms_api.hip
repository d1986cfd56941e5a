// rtcc_rotated_nms: the NMS kernels of the join, on caller-provided records.
// Argument checks, scratch allocation and the launch only; the work is in
// kernels/nms.hip.
#include <hip/hip_runtime.h>

#include <string>

#include "../../include/rtcc.h"
#include "kernels/kernels.hpp"

namespace rtcc {
void set_thread_error(const std::string &msg);
}

namespace {

struct Scratch {
    void *p[10] = {};
    ~Scratch() {
        for (void *q : p)
            if (q) (void)hipFree(q);
    }
};

rtcc_status fail(rtcc_status s, const std::string &msg) {
    rtcc::set_thread_error(msg);
    return s;
}

rtcc_status hip_fail(hipError_t e, const char *what) {
    return fail(e == hipErrorOutOfMemory ? RTCC_E_NOMEM : RTCC_E_HIP,
                std::string(what) + " failed: " + hipGetErrorString(e));
}

}  // namespace

extern "C" RTCC_API rtcc_status rtcc_rotated_nms(const float *device_records, int64_t n, int32_t max_candidates,
                                                 float iou_threshold, float *device_out, int64_t *kept) {
    if (!kept) return fail(RTCC_E_ARG, "kept is NULL");
    *kept = 0;
    if (n < 0 || n > 2147483647) return fail(RTCC_E_ARG, "n out of range");
    if (max_candidates < 1 || max_candidates > rtcc::kern::kNmsMaxCandidates)
        return fail(RTCC_E_ARG, "max_candidates must be in [1, 16384]");
    if (!(iou_threshold >= 0.f && iou_threshold <= 1.f)) return fail(RTCC_E_ARG, "iou_threshold must be in [0, 1]");
    if (n == 0) return RTCC_OK;
    if (!device_records || !device_out) return fail(RTCC_E_ARG, "NULL records or output");

    const size_t m = size_t(max_candidates);
    const size_t words = (m + 63) / 64;
    Scratch sc;
    const size_t sizes[10] = {size_t(n) * 4, size_t(n) * 4, m * 4, m * rtcc::kern::kNmsFootDoubles * 8, m * words * 8, 64,
                              m * 8, size_t(rtcc::kern::kNmsRankSplits) * size_t(n) * 4,
                              rtcc::kern::nms_colrows(max_candidates) * 4, words * 4};
    for (int i = 0; i < 10; ++i) {
        hipError_t e = hipMalloc(&sc.p[i], sizes[i]);
        if (e != hipSuccess) return hip_fail(e, "hipMalloc");
    }
    hipStream_t s = nullptr;
    hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    if (e != hipSuccess) return hip_fail(e, "hipStreamCreateWithFlags");
    // count[0] = n, count[1] = kept, count[2] = NaN-score flag
    const int32_t init[3] = {int32_t(n), 0, 0};
    int32_t *count = static_cast<int32_t *>(sc.p[5]);
    int32_t host_out[2] = {0, 0};
    rtcc::kern::NmsArgs a{};
    a.rec = device_records;
    a.count = count;
    a.rank = static_cast<int32_t *>(sc.p[0]);
    a.flag = static_cast<int32_t *>(sc.p[1]);
    a.order = static_cast<int32_t *>(sc.p[2]);
    a.foot = static_cast<double *>(sc.p[3]);
    a.mask = static_cast<unsigned long long *>(sc.p[4]);
    a.mask_t = static_cast<unsigned long long *>(sc.p[6]);
    a.partial = static_cast<int32_t *>(sc.p[7]);
    a.colrows = static_cast<int32_t *>(sc.p[8]);
    a.colcount = static_cast<int32_t *>(sc.p[9]);
    a.out = device_out;
    a.out_count = count + 1;
    a.bad_score = count + 2;
    a.iou_threshold = double(iou_threshold);
    a.max_candidates = max_candidates;
    e = hipMemcpyAsync(count, init, sizeof(init), hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = rtcc::kern::rotated_nms(a, n, s);
    if (e == hipSuccess) e = hipMemcpyAsync(host_out, count + 1, sizeof(host_out), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    (void)hipStreamDestroy(s);
    if (e != hipSuccess) return hip_fail(e, "rotated NMS");
    if (host_out[1]) return fail(RTCC_E_ARG, "a record's score is NaN (no defined ranking)");
    *kept = host_out[0];
    return RTCC_OK;
}
