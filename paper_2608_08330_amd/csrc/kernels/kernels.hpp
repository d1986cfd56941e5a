// Host launchers of the gfx950 kernels.  Every launcher checks nothing but
// enqueues on the given stream and returns hipGetLastError(); the executor
// validates shapes before calling.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "conv_plan.hpp"

namespace rtcc {
namespace kern {

// ------------------------------------------------------------ pillarization
struct PillarGeom {
    float x0, x1, y0, y1, z0, z1, v;
    int H, W;
};

constexpr int kScanTile = 2048;  // cells per block of the cell scans

hipError_t fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s);

// One agent's pillar-stage buffers (device pointers, fixed for a context).
// With tiles = ceil(H*W / kScanTile) tiles of cells, the sizes are: cell,
// slot, binned, cellb, rank, member [n_max]; sorted [n_max] points; ttotal
// [tiles] (zero between frames); tstart [tiles + 1]; npil [tiles]; tcell, tcount, toff
// [H*W]; pcells, pcounts, poffs [min(n_max, H*W)]; overfull
// [n_max / (max_pts + 1) + 1]; meta [3]; canvas [H*W][C].
struct PillarBufs {
    int32_t *cell, *slot, *ttotal, *tstart, *binned, *cellb, *rank;
    int32_t *tcell, *tcount, *toff, *npil;
    int32_t *pcells, *pcounts, *poffs, *overfull, *member, *meta;
    float4 *sorted;
    void *canvas;
};

constexpr int kPtsPerBlock = 512;  // points per block of the per-point kernels

// The agents whose pillar stage one launch chain runs: agent row j is agent
// agent[j] (its buffers bufs[agent[j]], its n[j] points at pts[j]).  One
// agent is a group of one.
constexpr int kMaxGroup = 16;
struct PillarGroup {
    const PillarBufs *bufs;  // device array, indexed by agent
    const float4 *pts[kMaxGroup];
    int32_t n[kMaxGroup];
    int32_t agent[kMaxGroup];
    int32_t m;       // agents in the group, 1..kMaxGroup
    int32_t n_max;   // max over the group of n[j]
    int32_t n_cells; // H * W
    int32_t tiles;   // ceil(n_cells / kScanTile)
};

// The sort of points by cell (counting in LDS):
// K1 bin_count: cell id per point (-1 if dropped); per block of
//    kPtsPerBlock points, its points' count in every tile of cells, one
//    atomic ttotal[tile] += count per non-empty tile (ttotal starts at
//    zero) reserving the block's run in the tile, and each point's
//    position within its tile (slot).
// K2 bin_scatter: tstart[t] = first point of tile t in tile order,
//    tstart[tiles] = meta[0] = valid points, meta[2] (overfull count) = 0;
//    binned / cellb = point index / cell in tile order.
// K3 tile_sort: per tile, LDS counts of its cells: the tile's pillars in
//    ascending cell order at tcell / tcount / toff [tile * kScanTile + q]
//    (npil[tile] of them), the pillars over max_pts listed in overfull
//    (by that index, meta[2] of them), and member / sorted = the points in
//    cell order (rank within a cell: an arbitrary order).
hipError_t bin_count(const PillarGroup &grp, const PillarGeom &g, hipStream_t s);
hipError_t bin_scatter(const PillarGroup &grp, hipStream_t s);
hipError_t tile_sort(const PillarGroup &grp, int32_t max_pts, hipStream_t s);
// K4 pillar_lists: the global pillar lists pcells / pcounts / poffs in
// ascending cell order, meta[1] = P pillars, from the tiles' lists;
// ttotal back to zero.
hipError_t pillar_lists(const PillarGroup &grp, hipStream_t s);
// K5 pfn_canvas: the dense canvas [H*W][C]: per pillar cell, channel max over the first
// min(count, max_pts) members of ReLU(W^T f + b) (for cells over the cap,
// after moving the max_pts lowest point indices to the front of the
// segment).  Writes the pillar cells only: every other cell must already be
// zero (canvas_clear zeroes the previous frame's pillars).
struct PfnArgs {
    const float *w;  // [4][C]
    const float *b;  // [C]
    int32_t C;
    int32_t max_pts;
    float inv_hx, inv_hy, z0, inv_dz;
    int32_t pillar_blocks;  // set by pfn_canvas
    // replay = 1: the pillars over the cap already hold their selected points
    // first (a previous launch on the same lists chose them), so they are
    // not chosen again; the canvas cells come out bit for bit as in that
    // launch.  canvas: where the cells go (nullptr: the agent's canvas).
    int32_t replay;
    void *canvas;
};
// max_pillars bounds every agent's meta[1] (at most min(cells, points)).
hipError_t pfn_canvas(bool bf16, PfnArgs a, const PillarGroup &grp, int32_t max_pillars, hipStream_t s);
// For every agent of the group, the canvas cells of the pillars listed in its
// pcells (meta[1] of them) back to zero; max_pillars bounds meta[1].  Only
// grp.bufs, grp.agent and grp.m are read.
hipError_t canvas_clear(bool bf16, const PillarGroup &grp, int32_t C, int32_t max_pillars, hipStream_t s);

// ------------------------------------------------------------ implicit GEMM
// conv:   out[m][c_off + n] for m = output pixel, 3x3 taps, pad 1, stride.
// deconv: A rows are input pixels, phase = blockIdx.z, output pixel
//         (iy * u + py, ix * u + px), skipped outside Ho x Wo.
struct GemmArgs {
    const void *in;    // NHWC, channel stride Ci
    const void *wt;    // Bt[N][K] (conv) or u*u phases of Bt[N][Ci] (deconv)
    const float *bias; // [N]
    void *out;         // NHWC, channel stride ldo
    int32_t Hi, Wi, Ci;
    int32_t Ho, Wo;
    int32_t N;
    int32_t stride;    // conv only
    int32_t u;         // deconv only
    int32_t ldo, c_off;
    int32_t splits;    // K slices (>= 1); > 1 needs ws and a conv (no deconv)
    int32_t variant;   // conv kernel: kConvImplicit or one of the halo tilings
    const void *zero;  // >= 16 zero bytes in device memory (padding reads)
    float *ws;         // split-K partials [splits][M][N] float32
    // Several agents' maps side by side in one launch (the same layer and
    // weights): batch > 1 takes agent b's input, output and split-K partials
    // from in_b / out_b / ws_b [b] instead of in / out / ws.  Every output
    // element is computed exactly as in a launch of its own.
    int32_t batch;     // 0 or 1: one map
    const void *in_b[16];
    void *out_b[16];
    float *ws_b[16];
};
// With start / stop events, the first kernel of the convolution records
// `start` when it begins executing and the last one `stop` when it ends
// (kernel execution time, without the dispatch gap before it).
hipError_t conv3x3(bool bf16, const GemmArgs &a, hipStream_t s, hipEvent_t start = nullptr,
                   hipEvent_t stop = nullptr);
hipError_t deconv(bool bf16, const GemmArgs &a, hipStream_t s);

// ------------------------------------------------------------ post-join
struct WarpArgs {
    const void *slots[16];  // per agent [H2*W2][C]
    float affine[16][6];    // per agent {M00, M01, t0, M10, M11, t1}
    void *fused;            // [H2*W2][C]
    int32_t K, H2, W2, C;
    uint32_t ident;         // bit k: agent k's affine is exactly the identity
};
// Bit k set iff affine[k] is {1, 0, 0, 0, 1, 0} (by value).
inline uint32_t identity_mask(const float (*affine)[6], int K) {
    uint32_t m = 0;
    for (int k = 0; k < K; ++k)
        if (affine[k][0] == 1.f && affine[k][1] == 0.f && affine[k][2] == 0.f && affine[k][3] == 0.f &&
            affine[k][4] == 1.f && affine[k][5] == 0.f)
            m |= 1u << k;
    return m;
}
// With start / stop events the launch records them around the kernel's own
// execution (hipExtLaunchKernelGGL).
hipError_t warp_fuse(bool bf16, bool attn, const WarpArgs &a, hipStream_t s, hipEvent_t start = nullptr,
                     hipEvent_t stop = nullptr);

// Warp as the last node of a branch: one agent's slot resampled on the ego
// grid (the sampling of warp_fuse) and stored in the activation dtype.
struct WarpSlotArgs {
    const void *slot;  // [H2*W2][C]
    float affine[6];   // {M00, M01, t0, M10, M11, t1}
    void *out;         // [H2*W2][C]
    int32_t H2, W2, C;
};
hipError_t warp_slot(bool bf16, const WarpSlotArgs &a, hipStream_t s, hipEvent_t start = nullptr,
                     hipEvent_t stop = nullptr);

// Fusion (the fold of warp_fuse) of K stored ego-frame maps.
struct FuseArgs {
    const void *maps[16];  // per agent [cells][C]
    void *fused;           // [cells][C]
    int32_t K, cells, C;
};
hipError_t fuse(bool bf16, bool attn, const FuseArgs &a, hipStream_t s, hipEvent_t start = nullptr,
                hipEvent_t stop = nullptr);

// 1x1 head: out[m][16] float32 = bias + Bt[16][C] . in[m][C].  counts[w]
// (w < ceil(M / 16)) = anchors of pixels 16 w .. 16 w + 15 whose class
// logit (output 0 or 8) is > thr: the decode's compaction offsets.
hipError_t head1x1(bool bf16, const void *in, const void *wt, const float *bias, float *out,
                   int32_t M, int32_t C, float thr, int32_t *counts, hipStream_t s);

// Threshold and decode: anchors of [M][16] head outputs (2 anchors x 8).
struct DecodeArgs {
    const float *head;
    int32_t H2, W2;
    float thr;
    float x0, y0, dx, dy;
    float aw, al, ah, az, ayaw0, ayaw1;
    const int32_t *head_counts;  // [ceil(H2 W2 / 16)] from head1x1 with the same thr; 16-byte aligned
    float *rec;            // [n_anchors][9]: box 7, score, index bits
    int32_t *count;        // total kept
};
constexpr int kDecodeTile = 1024;
hipError_t decode(const DecodeArgs &a, hipStream_t s);
// The frame's result into pinned host memory: words 0 and 1 of `host` the
// counts *count0 and *count1 (0 without count1), and from byte 64 the first
// min(*count1 or *count0, first) 36-byte records of `recs`; written with
// vector stores and fenced at system scope; then 1 is stored to word 2 with
// release semantics at system scope, so a host that cleared word 2 before
// enqueuing the kernel and then reads 1 there (acquire) also sees the counts
// and records, without waiting for the stream.
hipError_t export_results(const int32_t *count0, const int32_t *count1, const float *recs, int first, void *host,
                          hipStream_t s);

// Rotated NMS of the decoded records (see nms.hip).
constexpr int kNmsMaxCandidates = 16384;
constexpr int kNmsFootDoubles = 8;
constexpr int kNmsRankSplits = 16;  // per candidate: x, y, w, l, cos yaw, sin yaw, valid, pad
struct NmsArgs {
    const float *rec;             // [n][9] decoded records, ascending anchor index
    const int32_t *count;         // n, on the device
    int32_t *rank;                // [max_records]
    int32_t *flag;                // [max_records]
    int32_t *order;               // [max_candidates]
    double *foot;                 // [max_candidates][kNmsFootDoubles]
    unsigned long long *mask;     // [max_candidates][max_candidates / 64] (rounded up)
    unsigned long long *mask_t;   // [max_candidates]: earlier rows of its own 64-row chunk that suppress it
    int32_t *partial;             // [kNmsRankSplits][max_records] partial rank counts
    int32_t *colrows;             // [64 W (W - 1) / 2], W = words per mask row: listed rows per column chunk
    int32_t *colcount;            // [W] rows listed per column chunk
    float *out;                   // [max_candidates][9] kept records, ascending anchor index
    int32_t *out_count;           // kept, on the device
    double iou_threshold;         // suppress iff IoU > threshold
    int32_t max_candidates;       // 1 .. kNmsMaxCandidates
    int32_t *bad_score = nullptr; // optional: set to 1 if a score is NaN (the caller clears it)
};
// max_records bounds n (the grid of the per-record kernels).
hipError_t rotated_nms(const NmsArgs &a, int64_t max_records, hipStream_t s);
// Elements of NmsArgs::colrows for a candidate cap.
inline size_t nms_colrows(int32_t max_candidates) {
    const size_t w = size_t(max_candidates + 63) / 64;
    return 64 * w * (w > 0 ? w - 1 : 0) / 2 + 1;
}

}  // namespace kern
}  // namespace rtcc
