// The conv planner (conv_plan.hpp).  Every rule below was chosen by timing
// the c5 layers on one MI355X, alone and in 8-agent launches; the comments
// give the measurements.
#include "conv_plan.hpp"

namespace rtcc {
namespace kern {

ConvPlan conv_plan(bool bf16, int Hi, int Wi, int Ci, int Ho, int Wo, int Co, int stride, int n_cu) {
    (void)Hi;
    (void)Wi;
    const int bk = bf16 ? 32 : 16;  // implicit GEMM K step (64 bytes)
    ConvPlan p{kConvImplicit, 1, 0, kConvImplicit, 1, kConvImplicit, 1 << 30};
    const int elt = bf16 ? 2 : 4;
    if (stride == 1 && Co % 128 == 0) {
        // 8 x 16-pixel tiles with 8 wavefronts where the grid fills the
        // chip; otherwise 4 x 16-pixel tiles with 4 wavefronts, split over
        // channel chunks until half the CUs hold a tile (an f32 partial
        // round trip costs more than idle CUs beyond that, measured on
        // 64 x 64 grids).  Batched maps take the 8 x 16 tiles once their
        // tiles fill the chip.
        const int tx = (Wo + 15) / 16, nt = Co / 128;
        const int t8 = tx * ((Ho + 7) / 8) * nt, t4 = tx * ((Ho + 3) / 4) * nt;
        const int chunk_bytes = ((Ci * elt) % 128 == 0 && Ci * elt >= 512) ? 128 : 64;
        const int chunks = Ci * elt / chunk_bytes;
        // 16 x 16 tiles for batches whose 16-row tiles cover the CUs, on maps
        // whose 8-row tiles give at most one block per CU (c5, 8 agents per
        // launch: 128 x 128 x 256 -> 256 4-7%, 64 x 64 x 256 -> 256 8% faster
        // than 8-row tiles; 256 x 256 x 128 -> 128, two 8-row blocks per CU
        // per map, 2-4% slower)
        const int t16 = ((Wo + 15) / 16) * ((Ho + 15) / 16) * nt;
        if (t8 <= n_cu) p.wider_maps = (n_cu + t16 - 1) / t16;
        p.variant_wide = kConvHalo8;
        p.variant_wider = kConvHalo16;
        if (t8 >= n_cu && chunk_bytes == 128) {
            // a map whose 8 x 16 tiles fill the chip by themselves: 64-byte
            // chunks (at 128 x 128 x 256 -> 256, 8 maps per launch: 7%
            // faster per map than 128-byte chunks, one map alone 10%
            // slower; the batched frame decides, and all launches of a
            // layer must accumulate alike)
            p.variant = p.variant_wide = kConvHalo8C64;
            p.variant_wider = kConvHalo16C64;
        } else if (t8 >= n_cu) {
            p.variant = kConvHalo8;
        } else {
            p.variant = kConvHalo4;
            p.wide_maps = (n_cu + t8 - 1) / t8;
            if (t4 < n_cu / 2)
                for (int sp = 2; sp <= chunks && t4 * p.splits < n_cu / 2; ++sp)
                    if (chunks % sp == 0) p.splits = sp;
        }
    } else if (stride == 2 && Co % 128 == 0 && Ci * elt >= 256) {
        // stride-2 patches (2 TH + 1 rows of 33 pixels, column-split); at
        // 64 input channels (two chunks) the implicit GEMM is faster, alone
        // and in the 8-agent launch of the c5 frame (19.4-19.8 us per agent
        // against 20.2-20.6 with 4-row and 22.3 with 8-row stride-2 tiles)
        const int tx = (Wo + 15) / 16, nt = Co / 128;
        const int t8 = tx * ((Ho + 7) / 8) * nt;
        p.variant_wide = kConvHalo8S2;
        if (Co % 256 == 0) {
            // 256-channel tiles once a batch's tiles cover the CUs (c5, 8
            // agents per launch: 256 x 256 x 128 -> 128 x 128 x 256 17% and
            // 128 x 128 x 256 -> 64 x 64 x 256 14% faster than 128-channel
            // tiles)
            p.variant_wider = kConvHalo8S2N256;
            p.wider_maps = (n_cu + t8 / 2 - 1) / (t8 / 2);
        }
        if (t8 >= n_cu) {
            p.variant = kConvHalo8S2;
        } else {
            p.variant = kConvHalo4S2;
            p.wide_maps = (n_cu + t8 - 1) / t8;
        }
    } else if (stride == 2 && Co % 128 == 0 && ((Ho * Wo + 255) / 256) * (Co / 128) >= n_cu) {
        // the 64-channel stride-2 first layer: 256-pixel tiles, two blocks
        // per CU (512 x 512 x 64 -> 256 x 256 x 128: 21% faster than 128 x
        // 128 tiles with 8 maps per launch, 13% with 2, as fast alone)
        p.variant = p.variant_wide = p.variant_wider = kConvImplicit256;
    } else {
        const int tiles = gemm_tiles(Ho * Wo, Co);
        const int kt = 9 * Ci / bk;
        if (tiles < n_cu)
            for (int sp = 2; sp <= 16 && tiles * p.splits < 2 * n_cu; ++sp)
                if (kt % sp == 0 && kt / sp >= 8) p.splits = sp;
    }
    if (p.splits > 1) p.ws_bytes = size_t(p.splits) * Ho * Wo * Co * 4;
    return p;
}

ConvPlan conv_plan_forced(bool bf16, const ConvPlan &planned, int variant, int splits, int Ci, int Ho, int Wo,
                          int Co, int stride) {
    (void)Ho;
    (void)Wo;
    const int elt = bf16 ? 2 : 4;
    const int row_bytes = Ci * elt;
    const bool rb128 = row_bytes % 128 == 0 && row_bytes >= 512;
    // K steps of the kernel the forced tiling launches: input-channel chunks
    // (halo tilings, split further over the wave groups) or 64-byte K steps
    int steps = 0, groups = 1;
    bool fits = false;
    switch (variant) {
        case 7:  // the implicit GEMM everywhere
            variant = kConvImplicit;
            steps = 9 * Ci / (bf16 ? 32 : 16);
            fits = true;
            break;
        case kConvHalo8:
        case kConvHalo4:
            fits = stride == 1 && Co % 128 == 0;
            steps = row_bytes / (rb128 ? 128 : 64);
            break;
        case kConvHalo8C64:
        case kConvHalo16C64:
            fits = stride == 1 && Co % 128 == 0 && row_bytes % 64 == 0;
            steps = row_bytes / 64;
            break;
        case kConvHalo16:
            fits = stride == 1 && Co % 128 == 0;
            steps = row_bytes / (rb128 ? 128 : 64);
            break;
        case kConvHalo8S2N256:
            fits = stride == 2 && Co % 256 == 0 && row_bytes % 64 == 0;
            steps = row_bytes / 64;
            break;
        case kConvImplicit256:
            fits = Co % 128 == 0;
            steps = 9 * Ci / (bf16 ? 32 : 16);
            break;
        case kConvHalo8S2:
        case kConvHalo4S2:
            fits = stride == 2 && Co % 128 == 0 && row_bytes % 64 == 0;
            steps = row_bytes / 64;
            break;
        case kConvHalo4N64K2:
            fits = stride == 1 && Co % 64 == 0;
            steps = row_bytes / (rb128 ? 128 : 64);
            groups = 2;
            break;
        case kConvHalo4S2N64K2:
            fits = stride == 2 && Co % 64 == 0 && row_bytes % 64 == 0;
            steps = row_bytes / 64;
            groups = 2;
            break;
        default: break;
    }
    if (!fits || steps % groups != 0 || steps / groups < 1) return planned;
    ConvPlan p{variant, 1, 0, variant, 1, variant, 1 << 30};
    // a split-K slice holds whole chunks of one wave group's share; the
    // two-group tilings run unsplit
    if (splits > 1 && groups == 1 && steps % splits == 0) p.splits = splits;
    if (p.splits > 1) p.ws_bytes = size_t(p.splits) * Ho * Wo * Co * 4;
    return p;
}

int gemm_tiles(int M, int N) { return ((M + 127) / 128) * (N % 128 == 0 ? N / 128 : (N + 63) / 64); }

}  // namespace kern
}  // namespace rtcc
