// Weights checkpoint: a weights blob with a manifest (config id, seed,
// tensor table, SHA-256 of the data).  The layout is documented beside
// rtcc_read_checkpoint in include/rtcc.h.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/rtcc.h"
#include "model.hpp"

namespace rtcc {

constexpr size_t kCkptHeaderBytes = 128;
constexpr size_t kCkptEntryBytes = 128;
constexpr uint32_t kCkptVersion = 1;

struct CkptTensor {
    std::string name;
    int ndim = 0;
    int64_t shape[4] = {0, 0, 0, 0};
    uint64_t offset = 0;  // within the data section
    uint64_t nbytes = 0;
};

struct CkptView {
    rtcc_checkpoint_info info{};
    std::vector<CkptTensor> tensors;
    const unsigned char *data = nullptr;  // the data section inside the caller's buffer
};

// SHA-256 (FIPS 180-4) of n bytes.
void sha256(const void *data, size_t n, uint8_t out[32]);

// Parse and verify a checkpoint: header, tensor table, exact file size and
// the data section's SHA-256.  Returns RTCC_OK, or RTCC_E_ARG / RTCC_E_MALFORMED
// with a message.
rtcc_status parse_checkpoint(const void *file, size_t bytes, CkptView &v, std::string &err);

// The weight tensors a plan expects, in blob order (names and shapes).
std::vector<CkptTensor> expected_tensors(const Plan &p);

}  // namespace rtcc
