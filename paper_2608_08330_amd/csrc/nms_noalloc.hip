// rtcc_rotated_nms_noalloc: the rotated NMS of rtcc_rotated_nms for callers
// that cannot allocate device memory.  Its scratch lives in one file-scope
// device array of fixed size; the call allocates nothing, creates no stream
// and runs the same kernels (kernels/nms.hip) on the caller's stream.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/rtcc.h"
#include "kernels/kernels.hpp"

namespace rtcc {
void set_thread_error(const std::string &msg);
}

namespace {

using rtcc::kern::kNmsFootDoubles;
using rtcc::kern::kNmsRankSplits;

// Limits of one call: records (the anchors of a 256 x 256 head grid) and
// NMS candidates.
constexpr int64_t kMaxRecords = 131072;
constexpr int32_t kMaxCandidates = 4096;
constexpr int64_t kWords = (kMaxCandidates + 63) / 64;

constexpr size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// Byte offsets of the parts of the scratch array (worst-case sizes).
constexpr size_t kOffCount = 0;  // n, kept, NaN-score flag
constexpr size_t kOffRank = kOffCount + 256;
constexpr size_t kOffFlag = kOffRank + align256(size_t(kMaxRecords) * 4);
constexpr size_t kOffPartial = kOffFlag + align256(size_t(kMaxRecords) * 4);
constexpr size_t kOffOrder = kOffPartial + align256(size_t(kNmsRankSplits) * kMaxRecords * 4);
constexpr size_t kOffFoot = kOffOrder + align256(size_t(kMaxCandidates) * 4);
constexpr size_t kOffMask = kOffFoot + align256(size_t(kMaxCandidates) * kNmsFootDoubles * 8);
constexpr size_t kOffMaskT = kOffMask + align256(size_t(kMaxCandidates) * kWords * 8);
constexpr size_t kOffColRows = kOffMaskT + align256(size_t(kMaxCandidates) * 8);
constexpr size_t kOffColCount = kOffColRows + align256((64 * kWords * (kWords - 1) / 2 + 1) * 4);
constexpr size_t kScratchBytes = kOffColCount + align256(size_t(kWords) * 4);  // 11.9 MB

// The scratch.  In host code this name is a host-side stand-in, not a
// device address: host code uses only the per-device address returned by
// hipGetSymbolAddress.
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu[kMaxDevices];      // one call at a time per device (they share its scratch)
void *g_scratch[kMaxDevices] = {}; // device address of `scratch` on each device
std::mutex g_setup_mu;

// n, kept = 0 and the NaN flag = 0, by a kernel (no host-to-device copy)
__global__ void k_noalloc_counts(int32_t *c, int32_t n) {
    if (threadIdx.x == 0) {
        c[0] = n;
        c[1] = 0;
        c[2] = 0;
    }
}

rtcc_status fail(rtcc_status s, const std::string &msg) {
    rtcc::set_thread_error(msg);
    return s;
}

rtcc_status hip_fail(hipError_t e, const char *what) {
    return fail(RTCC_E_HIP, std::string(what) + " failed: " + hipGetErrorString(e));
}

// Address of this device's scratch, looked up once per device with the
// device current.
rtcc_status scratch_of(int dev, void **out) {
    std::lock_guard<std::mutex> lk(g_setup_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return RTCC_OK;
}

}  // namespace

extern "C" RTCC_API rtcc_status rtcc_rotated_nms_noalloc(const float *device_records, int64_t n,
                                                         int32_t max_candidates, float iou_threshold,
                                                         float *device_out, int64_t *kept, void *hip_stream) {
    if (!kept) return fail(RTCC_E_ARG, "kept is NULL");
    *kept = 0;
    if (n < 0) return fail(RTCC_E_ARG, "n < 0");
    if (n > kMaxRecords)
        return fail(RTCC_E_ARG, "n = " + std::to_string(n) + " exceeds the allocation-free limit of " +
                                    std::to_string(kMaxRecords) + " records");
    if (max_candidates < 1 || max_candidates > kMaxCandidates)
        return fail(RTCC_E_ARG, "max_candidates must be in [1, " + std::to_string(kMaxCandidates) +
                                    "] for the allocation-free entry point");
    if (!(iou_threshold >= 0.f && iou_threshold <= 1.f)) return fail(RTCC_E_ARG, "iou_threshold must be in [0, 1]");
    if (n == 0) return RTCC_OK;
    if (!device_records || !device_out) return fail(RTCC_E_ARG, "NULL records or output");

    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(RTCC_E_ARG, "device ordinal out of range");
    std::lock_guard<std::mutex> lk(g_mu[dev]);
    void *base = nullptr;
    rtcc_status st = scratch_of(dev, &base);
    if (st != RTCC_OK) return st;
    unsigned char *p = static_cast<unsigned char *>(base);
    hipStream_t s = static_cast<hipStream_t>(hip_stream);

    int32_t *count = reinterpret_cast<int32_t *>(p + kOffCount);
    rtcc::kern::NmsArgs a{};
    a.rec = device_records;
    a.count = count;
    a.rank = reinterpret_cast<int32_t *>(p + kOffRank);
    a.flag = reinterpret_cast<int32_t *>(p + kOffFlag);
    a.partial = reinterpret_cast<int32_t *>(p + kOffPartial);
    a.order = reinterpret_cast<int32_t *>(p + kOffOrder);
    a.foot = reinterpret_cast<double *>(p + kOffFoot);
    a.mask = reinterpret_cast<unsigned long long *>(p + kOffMask);
    a.mask_t = reinterpret_cast<unsigned long long *>(p + kOffMaskT);
    a.colrows = reinterpret_cast<int32_t *>(p + kOffColRows);
    a.colcount = reinterpret_cast<int32_t *>(p + kOffColCount);
    a.out = device_out;
    a.out_count = count + 1;
    a.bad_score = count + 2;
    a.iou_threshold = double(iou_threshold);
    a.max_candidates = max_candidates;

    int32_t host_out[2] = {0, 0};
    k_noalloc_counts<<<1, 64, 0, s>>>(count, int32_t(n));
    e = hipGetLastError();
    if (e == hipSuccess) e = rtcc::kern::rotated_nms(a, n, s);
    if (e == hipSuccess) e = hipMemcpyAsync(host_out, count + 1, sizeof(host_out), hipMemcpyDeviceToHost, s);
    // the scratch is free for the next call only once this stream is done
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "rotated NMS (allocation-free)");
    if (host_out[1]) return fail(RTCC_E_ARG, "a record's score is NaN (no defined ranking)");
    *kept = host_out[0];
    return RTCC_OK;
}
