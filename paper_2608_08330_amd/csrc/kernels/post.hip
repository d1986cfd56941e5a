// Post-join subgraph on gfx950: pose warp + cross-agent fusion, 1x1 head,
// threshold + box decode.
//
// warp_fuse: 32 lanes (half a wavefront) per ego cell, VEC = C / 32
//   channels per lane.  For every agent the lane computes the agent-grid
//   sample position from the index-space affine, reads the four bilinear
//   corners of its channel slice (zero outside the grid) and folds the
//   sample into a running channel max, or into an online softmax over
//   agents whose scores <X_0, X_k> / sqrt(C) are reduced across the 32 lanes
//   with butterfly shuffles (fixed order, so deterministic).  Bandwidth
//   bound: every slot is read about once through L2, the fused map written
//   once.
// warp_slot + fuse: the same two steps split at the join when the warp is
//   the last node of each branch: warp_slot resamples one agent's slot on
//   the ego grid and stores it; fuse folds the K stored maps (sequential
//   reads) with the same arithmetic.
// head1x1: one wavefront per 16 pixels; the 16 outputs of a pixel are one
//   16 x 16 MFMA tile per 32 (bf16) or 16 (fp32) input channels.
// decode: the head counts the kept anchors of each of its wavefronts;
//   every decode tile adds up the counts before it, rescans its own flags
//   and writes its kept anchors in ascending anchor order (stable
//   compaction, deterministic).
#include <hip/hip_ext.h>

#include <cmath>

#include "kernels.hpp"

namespace rtcc {
namespace kern {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ inline float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ inline float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }
__device__ inline uint32_t rne_bits(float x) {
    uint32_t u = __float_as_uint(x);
    return u + 0x7fffu + ((u >> 16) & 1u);
}

template <int VEC>
__device__ inline void load_vec_bf16(const uint16_t *p, float *v) {
    if constexpr (VEC % 4 == 0) {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            const uint2 u = reinterpret_cast<const uint2 *>(p)[q];
            v[4 * q + 0] = bf16_lo(u.x);
            v[4 * q + 1] = bf16_hi(u.x);
            v[4 * q + 2] = bf16_lo(u.y);
            v[4 * q + 3] = bf16_hi(u.y);
        }
    } else if constexpr (VEC == 2) {
        const uint32_t u = *reinterpret_cast<const uint32_t *>(p);
        v[0] = bf16_lo(u);
        v[1] = bf16_hi(u);
    } else {
        v[0] = __uint_as_float(uint32_t(p[0]) << 16);
    }
}
// Load VEC consecutive elements as float.
template <typename T, int VEC>
__device__ inline void load_vec(const T *p, float *v) {
    if constexpr (sizeof(T) == 2) {
        load_vec_bf16<VEC>(reinterpret_cast<const uint16_t *>(p), v);
    } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) v[e] = reinterpret_cast<const float *>(p)[e];
    }
}
template <int VEC>
__device__ inline void store_vec_bf16(uint16_t *p, const float *v) {
    if constexpr (VEC % 4 == 0) {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            uint2 u;
            u.x = (rne_bits(v[4 * q]) >> 16) | (rne_bits(v[4 * q + 1]) & 0xffff0000u);
            u.y = (rne_bits(v[4 * q + 2]) >> 16) | (rne_bits(v[4 * q + 3]) & 0xffff0000u);
            reinterpret_cast<uint2 *>(p)[q] = u;
        }
    } else if constexpr (VEC == 2) {
        *reinterpret_cast<uint32_t *>(p) = (rne_bits(v[0]) >> 16) | (rne_bits(v[1]) & 0xffff0000u);
    } else {
        p[0] = uint16_t(rne_bits(v[0]) >> 16);
    }
}

template <typename T, int VEC>
__device__ inline void store_vec(T *p, const float *v) {
    if constexpr (sizeof(T) == 2) {
        store_vec_bf16<VEC>(reinterpret_cast<uint16_t *>(p), v);
    } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) reinterpret_cast<float *>(p)[e] = v[e];
    }
}

// Channel slice of lane l (0 .. 31) of a cell.  Contiguous: channels
// [VEC l, VEC l + VEC).  Split (bf16, 384 channels): [8 l, 8 l + 8) and
// [256 + 4 l, 256 + 4 l + 4), so that the 32 lanes read one 512-byte and one
// 256-byte run with 16- and 8-byte loads instead of three 8-byte loads at a
// 24-byte stride.  The arithmetic of a channel does not depend on the lane
// that holds it.
template <typename T, int VEC>
constexpr bool kSplitSlice = sizeof(T) == 2 && VEC == 12;

template <typename T, int VEC, bool SPLIT>
__device__ inline void load_slice(const T *cell, int l, float *v) {
    if constexpr (SPLIT) {
        const uint4 a = reinterpret_cast<const uint4 *>(cell)[l];
        const uint2 b = reinterpret_cast<const uint2 *>(cell + 256)[l];
        const uint32_t w[6] = {a.x, a.y, a.z, a.w, b.x, b.y};
#pragma unroll
        for (int q = 0; q < 6; ++q) {
            v[2 * q] = bf16_lo(w[q]);
            v[2 * q + 1] = bf16_hi(w[q]);
        }
    } else {
        load_vec<T, VEC>(cell + l * VEC, v);
    }
}

template <typename T, int VEC, bool SPLIT>
__device__ inline void store_slice(T *cell, int l, const float *v) {
    if constexpr (SPLIT) {
        uint32_t w[6];
#pragma unroll
        for (int q = 0; q < 6; ++q) w[q] = (rne_bits(v[2 * q]) >> 16) | (rne_bits(v[2 * q + 1]) & 0xffff0000u);
        reinterpret_cast<uint4 *>(cell)[l] = make_uint4(w[0], w[1], w[2], w[3]);
        reinterpret_cast<uint2 *>(cell + 256)[l] = make_uint2(w[4], w[5]);
    } else {
        store_vec<T, VEC>(cell + l * VEC, v);
    }
}

// Bilinear sample of one agent's slot (affine m = {M00, M01, t0, M10, M11,
// t1}) at the ego cell (i, j): VEC channels starting at c0, zero outside the
// grid.  Branch-free: a corner outside the grid loads cell (0, 0) instead and
// its value is replaced by 0, so the four corner loads of this agent (and of
// the agent sampled next to it) are all in flight before the first is
// consumed.  No contraction into FMAs: the sample is the same sequence of
// IEEE operations in every kernel it is inlined into (warp + fusion, branch
// warp), so both placements of the warp sample identical values.
template <typename T, int VEC, bool SPLIT>
__device__ inline void warp_sample(const T *slot, const float *m, int H2, int W2, int C, float fi, float fj,
                                   int l, float *x) {
#pragma clang fp contract(off)
    const float u = m[0] * fj + m[1] * fi + m[2];
    const float v = m[3] * fj + m[4] * fi + m[5];
    const float fx0 = floorf(u), fy0 = floorf(v);
    const float fx = u - fx0, fy = v - fy0;
    const int x0 = int(fx0), y0 = int(fy0);
    float val[4][VEC];
    bool in[4];
#pragma unroll
    for (int cnr = 0; cnr < 4; ++cnr) {
        const int yy = y0 + (cnr >> 1), xx = x0 + (cnr & 1);
        in[cnr] = unsigned(yy) < unsigned(H2) && unsigned(xx) < unsigned(W2);
        const size_t cell = in[cnr] ? size_t(yy) * W2 + xx : 0;
        load_slice<T, VEC, SPLIT>(slot + cell * C, l, val[cnr]);
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) x[e] = 0.f;
#pragma unroll
    for (int cnr = 0; cnr < 4; ++cnr) {
        const float wy = (cnr >> 1) ? fy : 1.f - fy;
        const float wx = (cnr & 1) ? fx : 1.f - fx;
        const float wgt = wx * wy;
#pragma unroll
        for (int e = 0; e < VEC; ++e) x[e] += in[cnr] ? wgt * val[cnr][e] : 0.f;
    }
}

// Sum over the 32 lanes of a half wavefront, bitwise the same in every lane:
// within each 16-lane row, DPP quad permutes (lane ^ 1, lane ^ 2) and the
// row's half mirror and mirror (every lane of an 8- or 16-lane group meets a
// lane of the other half, which holds the other half's sum), then a swizzle
// that swaps the two rows (lane ^ 16).  Each step adds a pair of partial
// sums that are the same in both lanes, so the tree, and the rounding, is
// the same everywhere.  DPP moves are register-to-register; only the last
// step goes through the LDS crossbar.
template <int CTRL>
__device__ inline float dpp_move(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}
__device__ inline float half_wave_sum(float d) {
    d += dpp_move<0xb1>(d);   // quad_perm [1, 0, 3, 2]
    d += dpp_move<0x4e>(d);   // quad_perm [2, 3, 0, 1]
    d += dpp_move<0x141>(d);  // row_half_mirror
    d += dpp_move<0x140>(d);  // row_mirror
    // bit-mask swizzle within 32 lanes: and 0x1f, or 0, xor 0x10
    d += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, d), 0x401f));
    return d;
}

// Cross-agent fusion of one cell's VEC-channel slice, agents folded in index
// order: a running channel max, or an online softmax whose scores
// <X_0, X_k> / sqrt(C) are reduced over the 32 lanes of the cell
// (half_wave_sum: a fixed tree, so deterministic).
template <int VEC, bool ATTN>
struct Fold {
    float q[VEC], acc[VEC];
    float run_max = -INFINITY, run_sum = 0.f, inv_sqrt_c;
    __device__ explicit Fold(int C) : inv_sqrt_c(1.0f / sqrtf(float(C))) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
    }
    __device__ void add(int k, const float *x) {
        if constexpr (!ATTN) {
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[e] = k == 0 ? x[e] : fmaxf(acc[e], x[e]);
        } else {
            if (k == 0) {
#pragma unroll
                for (int e = 0; e < VEC; ++e) q[e] = x[e];
            }
            float d = 0.f;
#pragma unroll
            for (int e = 0; e < VEC; ++e) d += q[e] * x[e];
            d = half_wave_sum(d);
            const float sc = d * inv_sqrt_c;
            const float nm = fmaxf(run_max, sc);
            const float scale = __expf(run_max - nm);
            const float p = __expf(sc - nm);
            run_sum = run_sum * scale + p;
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[e] = acc[e] * scale + p * x[e];
            run_max = nm;
        }
    }
    __device__ void finish() {
        if constexpr (ATTN) {
            const float inv = 1.0f / run_sum;
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[e] *= inv;
        }
    }
};

// Cell of this half wavefront.  XCD-aware order: block ids go to the 8 XCDs
// round-robin; give each XCD a contiguous band of cells, so bilinear corners
// shared by neighbouring cells are reused from that XCD's L2 (and the fused
// maps are read in long runs).
__device__ inline int cell_of_thread() {
    int bid = blockIdx.x;
    const int nb = gridDim.x;
    if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
    return (bid * 256 + int(threadIdx.x)) >> 5;
}

template <typename T, int VEC, bool ATTN>
__global__ __launch_bounds__(256) void k_warp_fuse(WarpArgs a) {
    const int cell = cell_of_thread();
    if (cell >= a.H2 * a.W2) return;  // uniform over the 32 lanes of a cell
    const int i = cell / a.W2, j = cell - (cell / a.W2) * a.W2;
    const int l = threadIdx.x & 31;
    const float fj = float(j), fi = float(i);
    Fold<VEC, ATTN> f(a.C);
    // with branch-free sampling one agent at a time already keeps 8 loads
    // per lane in flight; that measured fastest at the 8-agent size.  An
    // agent whose affine is the identity (the ego) samples every cell at
    // itself with weight 1: one load of the cell's slice gives the same value
    // as the four corners.
    for (int k = 0; k < a.K; ++k) {
        float x[VEC];
        if ((a.ident >> k) & 1u)
            load_slice<T, VEC, false>(static_cast<const T *>(a.slots[k]) + size_t(cell) * a.C, l, x);
        else
            warp_sample<T, VEC, false>(static_cast<const T *>(a.slots[k]), a.affine[k], a.H2, a.W2, a.C, fi, fj, l, x);
        f.add(k, x);
    }
    f.finish();
    store_slice<T, VEC, false>(static_cast<T *>(a.fused) + size_t(cell) * a.C, l, f.acc);
}

// Branch-side warp: agent k's slot resampled on the ego grid and stored in
// the activation dtype.
template <typename T, int VEC>
__global__ __launch_bounds__(256) void k_warp_slot(WarpSlotArgs a) {
    const int cell = cell_of_thread();
    if (cell >= a.H2 * a.W2) return;
    const int i = cell / a.W2, j = cell - (cell / a.W2) * a.W2;
    constexpr bool SPLIT = kSplitSlice<T, VEC>;
    const int l = threadIdx.x & 31;
    float x[VEC];
    warp_sample<T, VEC, SPLIT>(static_cast<const T *>(a.slot), a.affine, a.H2, a.W2, a.C, float(i), float(j), l, x);
    store_slice<T, VEC, SPLIT>(static_cast<T *>(a.out) + size_t(cell) * a.C, l, x);
}

// Fusion of K ego-frame maps: the same fold as k_warp_fuse over stored
// maps, read as K sequential streams; the next agent's slice is loaded
// before the current one is folded.
template <typename T, int VEC, bool ATTN>
__global__ __launch_bounds__(256) void k_fuse(FuseArgs a) {
    const int cell = cell_of_thread();
    if (cell >= a.cells) return;
    constexpr bool SPLIT = kSplitSlice<T, VEC>;
    const size_t off = size_t(cell) * a.C;
    const int l = threadIdx.x & 31;
    Fold<VEC, ATTN> f(a.C);
    float x[2][VEC];
    load_slice<T, VEC, SPLIT>(static_cast<const T *>(a.maps[0]) + off, l, x[0]);
    for (int k = 0; k < a.K; ++k) {
        if (k + 1 < a.K) load_slice<T, VEC, SPLIT>(static_cast<const T *>(a.maps[k + 1]) + off, l, x[(k + 1) & 1]);
        f.add(k, x[k & 1]);
    }
    f.finish();
    store_slice<T, VEC, SPLIT>(static_cast<T *>(a.fused) + off, l, f.acc);
}

// Launch on stream s; with events, through hipExtLaunchKernelGGL so that they
// bracket the kernel's own execution.
template <typename F, typename A>
void launch_timed(F kernel, unsigned g, hipStream_t s, hipEvent_t e0, hipEvent_t e1, const A &a) {
    if (e0 || e1) hipExtLaunchKernelGGL(kernel, dim3(g), dim3(256), 0, s, e0, e1, 0, a);
    else kernel<<<g, 256, 0, s>>>(a);
}

template <typename T, int VEC>
hipError_t launch_warp(int kind, bool attn, const void *args, int64_t cells, hipStream_t s, hipEvent_t e0,
                       hipEvent_t e1) {
    const unsigned g = unsigned((cells * 32 + 255) / 256);
    if (kind == 0) {
        const WarpArgs &a = *static_cast<const WarpArgs *>(args);
        if (attn) launch_timed(k_warp_fuse<T, VEC, true>, g, s, e0, e1, a);
        else launch_timed(k_warp_fuse<T, VEC, false>, g, s, e0, e1, a);
    } else if (kind == 1) {
        launch_timed(k_warp_slot<T, VEC>, g, s, e0, e1, *static_cast<const WarpSlotArgs *>(args));
    } else {
        const FuseArgs &a = *static_cast<const FuseArgs *>(args);
        if (attn) launch_timed(k_fuse<T, VEC, true>, g, s, e0, e1, a);
        else launch_timed(k_fuse<T, VEC, false>, g, s, e0, e1, a);
    }
    return hipGetLastError();
}

// kind 0: warp + fusion, 1: branch warp, 2: fusion of stored maps
template <typename T>
hipError_t warp_dispatch(int kind, bool attn, const void *args, int C, int64_t cells, hipStream_t s,
                         hipEvent_t e0, hipEvent_t e1) {
    switch (C) {
        case 32: return launch_warp<T, 1>(kind, attn, args, cells, s, e0, e1);
        case 64: return launch_warp<T, 2>(kind, attn, args, cells, s, e0, e1);
        case 128: return launch_warp<T, 4>(kind, attn, args, cells, s, e0, e1);
        case 256: return launch_warp<T, 8>(kind, attn, args, cells, s, e0, e1);
        case 384: return launch_warp<T, 12>(kind, attn, args, cells, s, e0, e1);
        case 512: return launch_warp<T, 16>(kind, attn, args, cells, s, e0, e1);
    }
    return hipErrorInvalidValue;
}

// ------------------------------------------------------------------ head

template <typename T>
__device__ inline f32x4_t head_mma(uint4 w, uint4 x, f32x4_t c);
template <>
__device__ inline f32x4_t head_mma<uint16_t>(uint4 w, uint4 x, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, w),
                                                   __builtin_bit_cast(bf16x8_t, x), c, 0, 0, 0);
}
template <>
__device__ inline f32x4_t head_mma<float>(uint4 w, uint4 x, f32x4_t c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.x), __uint_as_float(x.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.y), __uint_as_float(x.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.z), __uint_as_float(x.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.w), __uint_as_float(x.w), c, 0, 0, 0);
    return c;
}

template <typename T>
__global__ __launch_bounds__(256) void k_head(const T *__restrict__ in, const T *__restrict__ wt,
                                              const float *__restrict__ bias, float *__restrict__ out,
                                              int32_t M, int32_t C, float thr, int32_t *__restrict__ counts) {
    constexpr int EPV = 16 / sizeof(T);
    constexpr int BK = 4 * EPV;
    const int lane = threadIdx.x & 63;
    const int m0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * 16;
    if (m0 >= M) return;
    const int fr = lane & 15, fk = lane >> 4;
    const int m = m0 + fr;
    const bool ok = m < M;
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < C; k0 += BK) {
        const uint4 w = *reinterpret_cast<const uint4 *>(wt + size_t(fr) * C + k0 + fk * EPV);
        uint4 x = make_uint4(0, 0, 0, 0);
        if (ok) x = *reinterpret_cast<const uint4 *>(in + size_t(m) * C + k0 + fk * EPV);
        acc = head_mma<T>(w, x, acc);
    }
    const int n = fk * 4;
    const float v0 = acc[0] + bias[n];
    if (ok) {
        *reinterpret_cast<float4 *>(out + size_t(m) * 16 + n) =
            make_float4(v0, acc[1] + bias[n + 1], acc[2] + bias[n + 2], acc[3] + bias[n + 3]);
    }
    // anchors of these 16 pixels above the class-logit threshold (output 0
    // of anchor 0 in the lanes fk = 0, output 8 of anchor 1 in fk = 2), the
    // same comparison of the same stored value that the decode makes
    const unsigned long long kept = __ballot(ok && (fk == 0 || fk == 2) && v0 > thr);
    if (lane == 0) counts[m0 >> 4] = __popcll(kept);
}

// ------------------------------------------------------------------ decode

__device__ inline int block_excl_scan256(int v, int *total) {
    __shared__ int wsum[4];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int t = __shfl_up(inc, d, 64);
        if (lane >= d) inc += t;
    }
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    int base = 0, tot = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (q < w) base += wsum[q];
        tot += wsum[q];
    }
    __syncthreads();
    *total = tot;
    return base + inc - v;
}

constexpr int kPerThread = kDecodeTile / 256;
static_assert(kDecodeTile % 256 == 0 && kDecodeTile % 32 == 0, "a decode tile is whole head wavefronts");

__global__ __launch_bounds__(256) void k_decode_write(DecodeArgs a) {
    const int n_anchor = a.H2 * a.W2 * 2;
    const int base = blockIdx.x * kDecodeTile + threadIdx.x * kPerThread;
    bool keep[kPerThread];
    int c = 0;
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
        const int ai = base + q;
        keep[q] = ai < n_anchor && a.head[size_t(ai >> 1) * 16 + (ai & 1) * 8] > a.thr;
        c += keep[q];
    }
    // this tile's first record: the kept anchors before it, summed by the
    // block itself from the head's per-wavefront counts (a head wavefront
    // covers 16 pixels, 32 anchors; a tile 32 wavefronts, read as 16-byte
    // vectors, several in flight per lane); the last tile also writes the total
    constexpr int kHeadWavesPerTile = kDecodeTile / 32;
    const int4 *hc = reinterpret_cast<const int4 *>(a.head_counts);
    const int nv = int(blockIdx.x) * (kHeadWavesPerTile / 4);
    int before = 0;
#pragma unroll 4
    for (int t = threadIdx.x; t < nv; t += 256) {
        const int4 v = hc[t];
        before += (v.x + v.y) + (v.z + v.w);
    }
    int prefix, tot;
    block_excl_scan256(before, &prefix);
    int pos = prefix + block_excl_scan256(c, &tot);
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *a.count = prefix + tot;
    const float diag = sqrtf(a.aw * a.aw + a.al * a.al);
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
        if (!keep[q]) continue;
        const int ai = base + q;
        const int cell = ai >> 1, an = ai & 1;
        const int i = cell / a.W2, j = cell - (cell / a.W2) * a.W2;
        const float *r = a.head + size_t(cell) * 16 + an * 8;
        const float xa = a.x0 + (float(j) + 0.5f) * a.dx;
        const float ya = a.y0 + (float(i) + 0.5f) * a.dy;
        float *o = a.rec + size_t(pos) * 9;
        o[0] = xa + r[1] * diag;
        o[1] = ya + r[2] * diag;
        o[2] = a.az + r[3] * a.ah;
        o[3] = a.aw * expf(r[4]);
        o[4] = a.al * expf(r[5]);
        o[5] = a.ah * expf(r[6]);
        o[6] = (an ? a.ayaw1 : a.ayaw0) + r[7];
        o[7] = 1.0f / (1.0f + expf(-r[0]));
        o[8] = __int_as_float(ai);
        ++pos;
    }
}

}  // namespace

hipError_t warp_fuse(bool bf16, bool attn, const WarpArgs &a, hipStream_t s, hipEvent_t start, hipEvent_t stop) {
    const int64_t cells = int64_t(a.H2) * a.W2;
    return bf16 ? warp_dispatch<uint16_t>(0, attn, &a, a.C, cells, s, start, stop)
                : warp_dispatch<float>(0, attn, &a, a.C, cells, s, start, stop);
}

hipError_t warp_slot(bool bf16, const WarpSlotArgs &a, hipStream_t s, hipEvent_t start, hipEvent_t stop) {
    const int64_t cells = int64_t(a.H2) * a.W2;
    return bf16 ? warp_dispatch<uint16_t>(1, false, &a, a.C, cells, s, start, stop)
                : warp_dispatch<float>(1, false, &a, a.C, cells, s, start, stop);
}

hipError_t fuse(bool bf16, bool attn, const FuseArgs &a, hipStream_t s, hipEvent_t start, hipEvent_t stop) {
    return bf16 ? warp_dispatch<uint16_t>(2, attn, &a, a.C, a.cells, s, start, stop)
                : warp_dispatch<float>(2, attn, &a, a.C, a.cells, s, start, stop);
}

hipError_t head1x1(bool bf16, const void *in, const void *wt, const float *bias, float *out,
                   int32_t M, int32_t C, float thr, int32_t *counts, hipStream_t s) {
    const unsigned g = unsigned((M + 63) / 64);
    if (bf16)
        k_head<uint16_t><<<g, 256, 0, s>>>(static_cast<const uint16_t *>(in),
                                           static_cast<const uint16_t *>(wt), bias, out, M, C, thr, counts);
    else
        k_head<float><<<g, 256, 0, s>>>(static_cast<const float *>(in), static_cast<const float *>(wt),
                                        bias, out, M, C, thr, counts);
    return hipGetLastError();
}

hipError_t decode(const DecodeArgs &a, hipStream_t s) {
    const int n_anchor = a.H2 * a.W2 * 2;
    const int n_tiles = (n_anchor + kDecodeTile - 1) / kDecodeTile;
    k_decode_write<<<n_tiles, 256, 0, s>>>(a);
    return hipGetLastError();
}

// One block: the counts, then the records as 4-byte words.
__global__ __launch_bounds__(256) void k_export(const int32_t *count0, const int32_t *count1, const uint32_t *recs,
                                                int first, uint32_t *host) {
    const int32_t c0 = *count0, c1 = count1 ? *count1 : 0;
    const int32_t n = count1 ? c1 : c0;
    const int words = (n < 0 ? 0 : n < first ? n : first) * 9;
    // 16-byte stores across the bus (host + 64 and recs are 16-byte aligned),
    // then the last words
    const int quads = words >> 2;
    for (int i = int(threadIdx.x); i < quads; i += 256)
        reinterpret_cast<uint4 *>(host + 16)[i] = reinterpret_cast<const uint4 *>(recs)[i];
    for (int i = 4 * quads + int(threadIdx.x); i < words; i += 256) host[16 + i] = recs[i];
    if (threadIdx.x == 0) {
        host[0] = uint32_t(c0);
        host[1] = uint32_t(c1);
    }
    __threadfence_system();
    __syncthreads();  // every thread's stores are fenced before the flag
    if (threadIdx.x == 0) __hip_atomic_store(&host[2], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

hipError_t export_results(const int32_t *count0, const int32_t *count1, const float *recs, int first, void *host,
                          hipStream_t s) {
    k_export<<<1, 256, 0, s>>>(count0, count1, reinterpret_cast<const uint32_t *>(recs), first,
                               static_cast<uint32_t *>(host));
    return hipGetLastError();
}

}  // namespace kern
}  // namespace rtcc
