// Tiling plans of the 3x3 convolutions: which kernel tiling (and K split)
// runs a layer, for a launch over one agent's map and for launches over
// several agents' maps side by side.  Plain C++ (no device code), so the
// host-only build and its tests use the same planner as the GPU library.
#pragma once

#include <cstddef>

namespace rtcc {
namespace kern {

constexpr int kConvImplicit = 0;  // implicit GEMM (any stride)
constexpr int kConvHalo8 = 1;     // stride-1 halo tiles of 8 x 16 pixels, 8 waves
constexpr int kConvHalo4 = 2;     // stride-1 halo tiles of 4 x 16 pixels, 4 waves
constexpr int kConvHalo8S2 = 3;   // stride-2 halo tiles of 8 x 16 output pixels, 8 waves
constexpr int kConvHalo4S2 = 4;   // stride-2 halo tiles of 4 x 16 output pixels, 8 waves
constexpr int kConvHalo4N64K2 = 5;    // stride-1 4 x 16 pixels x 64 channels, 2 groups of 4 waves
constexpr int kConvHalo4S2N64K2 = 6;  // stride-2 4 x 16 pixels x 64 channels, 2 groups of 4 waves
// kConvHalo8 with 64-byte channel chunks also where 128-byte chunks apply
// (C_in * elt >= 512): twice the steps with half the operand bytes each,
// which measured faster in launches over several agents' maps.  (Id 7 is
// the runtime option that forces the implicit GEMM.)
constexpr int kConvHalo8C64 = 8;
// Stride-1 halo tiles of 16 x 16 pixels (8 waves of 64 pixels x 64
// channels): per channel chunk one weight tile serves twice the pixels of
// the 8-row tiles, for batched launches whose 16-row tiles cover the chip.
// kConvHalo16 takes 128-byte chunks where kConvHalo8 does; kConvHalo16C64
// always 64-byte chunks (the accumulation order of kConvHalo8C64).
constexpr int kConvHalo16 = 9;
constexpr int kConvHalo16C64 = 10;
// Stride-2 halo tiles of 8 x 16 output pixels x 256 channels (8 waves of
// 32 pixels x 128 channels): the input patch of a tile is staged once for
// all 256 output channels instead of once per 128.
constexpr int kConvHalo8S2N256 = 11;
// The implicit GEMM with tiles of 256 pixels x 128 channels and a 3-stage
// ring (72 KB of LDS, two blocks per CU).  Odd M tiles run their K steps in
// reverse, another accumulation order than kConvImplicit: a layer's plan
// takes one of the two for every batch size.
constexpr int kConvImplicit256 = 12;
struct ConvPlan {
    int variant;      // tiling of a launch over one map
    int splits;
    size_t ws_bytes;  // split-K workspace needed per map (0 without split)
    // From wide_maps maps per launch on (a batched launch, GemmArgs::batch),
    // tiling variant_wide, whose every output element is accumulated in the
    // same order as with `variant` (the same K chunks, taps and MFMA
    // sequence; only the output tile differs), so batching never changes a
    // bit of the result.
    int variant_wide;
    int wide_maps;
    // From wider_maps maps on, tiling variant_wider (the same order again).
    // wider_maps >= wide_maps.
    int variant_wider;
    int wider_maps;
};
// Kernel variant and K split of one 3x3 conv layer on a GPU with n_cu CUs.
// Only tilings with one wave group per tile are planned (a second group
// would sum half of the K chunks apart, another accumulation order).
ConvPlan conv_plan(bool bf16, int Hi, int Wi, int Ci, int Ho, int Wo, int Co, int stride, int n_cu);
// The plan with tiling `variant` (1..6, 8..12, or 7 = the implicit GEMM) and K split
// `splits` forced where the layer's stride and channels allow it; `planned`
// elsewhere.  A forced tiling is used for batched launches too.
ConvPlan conv_plan_forced(bool bf16, const ConvPlan &planned, int variant, int splits, int Ci, int Ho, int Wo,
                          int Co, int stride);
// The tiling of a launch over `maps` maps.
inline int conv_variant_for(const ConvPlan &p, int maps) {
    return maps >= p.wider_maps ? p.variant_wider : maps >= p.wide_maps ? p.variant_wide : p.variant;
}
// Output tiles of the implicit GEMM.
int gemm_tiles(int M, int N);

}  // namespace kern
}  // namespace rtcc
