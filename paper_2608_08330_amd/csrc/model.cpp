// Descriptor validation, shape planning and weight preparation.
#include "model.hpp"

#include <cmath>
#include <cstring>
#include <ctime>

namespace rtcc {

double now_s() {
    timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return double(ts.tv_sec) + 1e-9 * double(ts.tv_nsec);
}

uint16_t f32_to_bf16_rne(float x) {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    // add 0x7fff plus the lowest kept bit, then truncate: ties go to the
    // even bfloat16 significand
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

float bf16_to_f32(uint16_t h) {
    uint32_t u = uint32_t(h) << 16;
    float x;
    std::memcpy(&x, &u, 4);
    return x;
}

static bool finite_all(std::initializer_list<float> v) {
    for (float x : v)
        if (!std::isfinite(x)) return false;
    return true;
}

bool make_plan(const rtcc_model_desc &d, Plan &p, std::string &err) {
    p = Plan();
    p.d = d;
    if (d.abi_version != RTCC_ABI_VERSION) { err = "abi_version mismatch"; return false; }
    if (d.n_agents < 1 || d.n_agents > RTCC_MAX_AGENTS) { err = "n_agents out of range"; return false; }
    if (d.max_points < 1 || d.max_points > (int64_t(1) << 26)) { err = "max_points out of range"; return false; }
    if (!finite_all({d.x_min, d.x_max, d.y_min, d.y_max, d.z_min, d.z_max, d.pillar_size})) {
        err = "non-finite geometry"; return false;
    }
    if (!(d.x_min < d.x_max && d.y_min < d.y_max && d.z_min < d.z_max && d.pillar_size > 0.f)) {
        err = "empty region or non-positive pillar size"; return false;
    }
    p.K = d.n_agents;
    p.n_max = d.max_points;
    p.W = int(std::lround((double(d.x_max) - double(d.x_min)) / double(d.pillar_size)));
    p.H = int(std::lround((double(d.y_max) - double(d.y_min)) / double(d.pillar_size)));
    if (p.W < 1 || p.H < 1 || int64_t(p.W) * p.H > (int64_t(1) << 24)) { err = "grid size out of range"; return false; }
    if (d.max_points_per_pillar < 1 || d.max_points_per_pillar > 1024) { err = "max_points_per_pillar out of range"; return false; }
    if (d.precision != RTCC_PREC_FP32 && d.precision != RTCC_PREC_BF16) { err = "bad precision"; return false; }
    p.bf16 = d.precision == RTCC_PREC_BF16;
    p.elt = p.bf16 ? 2 : 4;
    if (d.c_pfn < 32 || d.c_pfn > 512 || d.c_pfn % 32) { err = "c_pfn must be a multiple of 32 in [32, 512]"; return false; }
    p.c_pfn = d.c_pfn;
    if (d.n_stages < 1 || d.n_stages > RTCC_MAX_STAGES) { err = "n_stages out of range"; return false; }
    if (d.fusion != RTCC_FUSE_MAX && d.fusion != RTCC_FUSE_ATTN) { err = "bad fusion"; return false; }
    if (d.n_anchors != 2) { err = "n_anchors must be 2"; return false; }
    if (!finite_all({d.anchor_w, d.anchor_l, d.anchor_h, d.anchor_z, d.anchor_yaw[0], d.anchor_yaw[1],
                     d.score_logit_threshold})) {
        err = "non-finite anchor or threshold"; return false;
    }
    if (d.nms_max_candidates < 0 || d.nms_max_candidates > 16384) {
        err = "nms_max_candidates must be in [0, 16384]"; return false;
    }
    if (d.nms_max_candidates > 0 && !(d.nms_iou_threshold >= 0.f && d.nms_iou_threshold <= 1.f)) {
        err = "nms_iou_threshold must be in [0, 1]"; return false;
    }
    if (d.warp_in_branch != 0 && d.warp_in_branch != 1) { err = "warp_in_branch must be 0 or 1"; return false; }
    if (d.multiscale != 0 && d.multiscale != 1) { err = "multiscale must be 0 or 1"; return false; }
    if (d.multiscale && (d.up_channels == 0 || d.warp_in_branch)) {
        err = "multiscale needs up_channels > 0 and warp_in_branch = 0"; return false;
    }

    size_t blob = 0, mat = 0, bias = 0;
    p.pfn_w_off = bias; bias += size_t(4) * d.c_pfn; blob += size_t(4) * d.c_pfn;
    p.pfn_b_off = bias; bias += d.c_pfn; blob += d.c_pfn;

    int Hc = p.H, Wc = p.W, Cc = d.c_pfn;
    for (int s = 0; s < d.n_stages; ++s) {
        const rtcc_stage &st = d.stages[s];
        if (st.stride != 1 && st.stride != 2) { err = "stage stride must be 1 or 2"; return false; }
        if (st.c_out < 32 || st.c_out > 1024 || st.c_out % 32) { err = "stage c_out must be a multiple of 32 in [32, 1024]"; return false; }
        if (st.n_convs < 1 || st.n_convs > 64) { err = "stage n_convs out of range"; return false; }
        for (int l = 0; l < st.n_convs; ++l) {
            ConvLayer c{};
            c.stage = s;
            c.Hi = Hc; c.Wi = Wc; c.Ci = Cc;
            c.stride = l == 0 ? st.stride : 1;
            c.Ho = (Hc + c.stride - 1) / c.stride;
            c.Wo = (Wc + c.stride - 1) / c.stride;
            c.Co = st.c_out;
            c.w_off = mat; mat += size_t(9) * c.Ci * c.Co; blob += size_t(9) * c.Ci * c.Co;
            c.b_off = bias; bias += c.Co; blob += c.Co;
            p.convs.push_back(c);
            Hc = c.Ho; Wc = c.Wo; Cc = c.Co;
        }
        p.stage_last_conv.push_back(int(p.convs.size()) - 1);
        p.stage_grid.push_back({Hc, Wc});
    }
    p.H2 = p.stage_grid[0].first;
    p.W2 = p.stage_grid[0].second;
    if (d.up_channels) {
        if (d.up_channels < 32 || d.up_channels > 512 || d.up_channels % 32) { err = "up_channels must be 0 or a multiple of 32 in [32, 512]"; return false; }
        int rel = 1;
        for (int s = 0; s < d.n_stages; ++s) {
            if (s > 0) rel *= d.stages[s].stride;
            UpLayer u{};
            u.stage = s;
            u.Hi = p.stage_grid[s].first;
            u.Wi = p.stage_grid[s].second;
            u.Ci = d.stages[s].c_out;
            u.u = rel;
            u.Co = d.up_channels;
            u.c_off = s * d.up_channels;
            if (u.Hi * rel < p.H2 || u.Wi * rel < p.W2) { err = "upsampled stage does not cover the slot grid"; return false; }
            u.w_off = mat; mat += size_t(rel) * rel * u.Ci * u.Co; blob += size_t(rel) * rel * u.Ci * u.Co;
            u.b_off = bias; bias += u.Co; blob += u.Co;
            p.ups.push_back(u);
        }
        p.c_slot = d.up_channels * d.n_stages;
    } else {
        p.c_slot = d.stages[d.n_stages - 1].c_out;
        if (p.stage_grid.back() != p.stage_grid[0]) { err = "without upsampling every stage must keep the grid (stride 1)"; return false; }
    }
    switch (p.c_slot) {
        case 32: case 64: case 128: case 256: case 384: case 512: break;
        default: err = "slot channels must be one of 32, 64, 128, 256, 384, 512"; return false;
    }
    p.head_w_off = mat; mat += size_t(16) * p.c_slot; blob += size_t(16) * p.c_slot;
    p.head_b_off = bias; bias += 16; blob += 16;
    p.mat_elems = mat;
    p.bias_floats = bias;
    p.blob_floats = blob;
    return true;
}

bool prepare_weights(const Plan &p, const float *blob, size_t n_floats, HostWeights &hw,
                     std::string &err) {
    if (n_floats != p.blob_floats) {
        err = "weights blob has " + std::to_string(n_floats) + " floats, descriptor needs " +
              std::to_string(p.blob_floats);
        return false;
    }
    for (size_t i = 0; i < n_floats; ++i)
        if (!std::isfinite(blob[i])) { err = "non-finite weight"; return false; }
    hw.bias.assign(p.bias_floats, 0.f);
    if (p.bf16) hw.mat_bf16.assign(p.mat_elems, 0); else hw.mat_f32.assign(p.mat_elems, 0.f);
    auto put_mat = [&](size_t dst, float v) {
        if (p.bf16) hw.mat_bf16[dst] = f32_to_bf16_rne(v); else hw.mat_f32[dst] = v;
    };
    auto round_w = [&](float v) { return p.bf16 ? bf16_to_f32(f32_to_bf16_rne(v)) : v; };
    const float *src = blob;
    const int C = p.c_pfn;
    for (int i = 0; i < 4 * C; ++i) hw.bias[p.pfn_w_off + i] = round_w(src[i]);
    src += 4 * C;
    for (int i = 0; i < C; ++i) hw.bias[p.pfn_b_off + i] = src[i];
    src += C;
    for (const ConvLayer &c : p.convs) {
        const int Kdim = 9 * c.Ci;
        // source HWIO [3][3][Ci][Co] -> Bt[co][(dy * 3 + dx) * Ci + ci]
        for (int tap = 0; tap < 9; ++tap)
            for (int ci = 0; ci < c.Ci; ++ci)
                for (int co = 0; co < c.Co; ++co)
                    put_mat(c.w_off + size_t(co) * Kdim + size_t(tap) * c.Ci + ci,
                            src[(size_t(tap) * c.Ci + ci) * c.Co + co]);
        src += size_t(9) * c.Ci * c.Co;
        for (int co = 0; co < c.Co; ++co) hw.bias[c.b_off + co] = src[co];
        src += c.Co;
    }
    for (const UpLayer &u : p.ups) {
        // source [u][u][Ci][Co] -> phase (py * u + px): Bt[co][ci]
        for (int ph = 0; ph < u.u * u.u; ++ph)
            for (int ci = 0; ci < u.Ci; ++ci)
                for (int co = 0; co < u.Co; ++co)
                    put_mat(u.w_off + (size_t(ph) * u.Co + co) * u.Ci + ci,
                            src[(size_t(ph) * u.Ci + ci) * u.Co + co]);
        src += size_t(u.u) * u.u * u.Ci * u.Co;
        for (int co = 0; co < u.Co; ++co) hw.bias[u.b_off + co] = src[co];
        src += u.Co;
    }
    // head [C][16] -> Bt[16][C]
    for (int c = 0; c < p.c_slot; ++c)
        for (int o = 0; o < 16; ++o)
            put_mat(p.head_w_off + size_t(o) * p.c_slot + c, src[size_t(c) * 16 + o]);
    src += size_t(16) * p.c_slot;
    for (int o = 0; o < 16; ++o) hw.bias[p.head_b_off + o] = src[o];
    src += 16;
    if (size_t(src - blob) != n_floats) { err = "internal: blob walk mismatch"; return false; }
    return true;
}

void pose_affine(const Plan &p, const float pose[3], float m[6]) { pose_affine_grid(p, pose, p.H2, p.W2, m); }

void pose_affine_grid(const Plan &p, const float pose[3], int H, int W, float m[6]) {
    const double dx = (double(p.d.x_max) - double(p.d.x_min)) / W;
    const double dy = (double(p.d.y_max) - double(p.d.y_min)) / H;
    const double c = std::cos(double(pose[0])), s = std::sin(double(pose[0]));
    const double ox = double(p.d.x_min) + 0.5 * dx, oy = double(p.d.y_min) + 0.5 * dy;
    // ego cell centre o + D (j, i) pulls the agent point R^T (o + D (j, i) - t):
    // in agent-grid index space that is D^-1 R^T D (j, i) + D^-1 (R^T (o - t) - o)
    const double qx = ox - double(pose[1]), qy = oy - double(pose[2]);
    const double rx = c * qx + s * qy, ry = -s * qx + c * qy;
    m[0] = float(c);
    m[1] = float(s * dy / dx);
    m[2] = float((rx - ox) / dx);
    m[3] = float(-s * dx / dy);
    m[4] = float(c);
    m[5] = float((ry - oy) / dy);
}

}  // namespace rtcc
