// Network plan derived from the model descriptor, weight-blob parsing and
// host-side weight preparation (bf16 rounding, repacking into the
// K-contiguous layouts the GEMM kernels read).
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/rtcc.h"

namespace rtcc {

struct ConvLayer {
    int stage;
    int Hi, Wi, Ci;   // input grid and channels (NHWC)
    int Ho, Wo, Co;   // output grid and channels
    int stride;
    size_t w_off;     // element offset of Bt[Co][9*Ci] in the matrix buffer
    size_t b_off;     // float offset of the bias in the bias buffer
};

struct UpLayer {
    int stage;
    int Hi, Wi, Ci;   // stage output grid
    int u;            // kernel = stride = u
    int Co;           // up_channels
    int c_off;        // channel offset in the concatenated slot
    size_t w_off;     // element offset of u*u phases of Bt[Co][Ci]
    size_t b_off;
};

struct Plan {
    rtcc_model_desc d{};
    int K = 0;
    int64_t n_max = 0;
    int H = 0, W = 0;     // pillar grid
    int H2 = 0, W2 = 0;   // slot / fused / head grid
    int c_pfn = 0;
    int c_slot = 0;       // channels of the agent slot (= head input)
    bool bf16 = false;
    int elt = 4;          // bytes per stored activation
    std::vector<ConvLayer> convs;
    std::vector<UpLayer> ups;
    std::vector<int> stage_last_conv;      // index into convs
    std::vector<std::pair<int, int>> stage_grid;
    size_t mat_elems = 0;   // total elements of repacked weight matrices
    size_t bias_floats = 0; // pfn_w, pfn_b and all biases (float32)
    size_t pfn_w_off = 0, pfn_b_off = 0;
    size_t head_w_off = 0, head_b_off = 0;
    size_t blob_floats = 0; // expected float count of the weight blob
};

// Validate the descriptor and derive every shape.  Returns false with a
// message on an inconsistent descriptor.
bool make_plan(const rtcc_model_desc &d, Plan &p, std::string &err);

// Host copies of the prepared weights: matrices as raw 16-bit bfloat16
// patterns or float32 (by precision), biases and the PFN as float32.
struct HostWeights {
    std::vector<uint16_t> mat_bf16;
    std::vector<float> mat_f32;
    std::vector<float> bias;
};

bool prepare_weights(const Plan &p, const float *blob, size_t n_floats, HostWeights &hw,
                     std::string &err);

// float32 -> bfloat16 bit pattern, round to nearest even (finite inputs).
uint16_t f32_to_bf16_rne(float x);
float bf16_to_f32(uint16_t h);

// Index-space affine of the pose warp: agent-grid sample position (u, v)
// of ego cell (i, j) is (u, v) = M (j, i) + t.  Output m = {M00, M01, t0,
// M10, M11, t1}.  Identity pose -> exactly {1, 0, 0, 0, 1, 0}.
void pose_affine(const Plan &p, const float pose[3], float m[6]);
// The same for a map of H x W cells covering the BEV region (a stage grid).
void pose_affine_grid(const Plan &p, const float pose[3], int H, int W, float m[6]);

double now_s();

}  // namespace rtcc
