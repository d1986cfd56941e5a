// Pillarization and point-feature canvas for gfx950.
//
// Deterministic counting sort by cell (no float atomics, no order-dependent
// result), five dependent launches:
//   cell_ids        one thread per point: float32 cell index, atomic count
//                   per cell (the counts start at zero); the returned old
//                   count is the point's rank of arrival in its cell
//   scan_reduce /   exclusive prefix over all H*W cells -> segment offsets,
//   scan_down       ascending list of non-empty cells (pillars) and their
//                   counts, list of cells over the per-pillar point cap (each
//                   block of the second pass adds up the tile sums before it)
//   scatter         member[offset[cell] + rank] = point index
//   pfn_canvas      one lane per (pillar, 8 channels): linear 4 -> C, ReLU,
//                   max over the pillar's points into its cell; the pillar's
//                   count is returned to zero for the next frame.  Extra
//                   blocks take the few cells over the cap: one wavefront
//                   moves the cap lowest point indices (found by bisection on
//                   the index value) to the front of the segment and writes
//                   that pillar's features
// The canvas is zero outside the pillars: canvas_clear zeroes the last
// frame's pillar cells again (off the encoder's path: the executor runs it
// when the next frame begins, before any branch input has arrived).
// The only order-dependent intermediate is the order of members inside a
// segment, and every consumer of it is order-independent (max, set
// selection), so every output is bitwise reproducible.
#include <climits>

#include "kernels.hpp"

namespace rtcc {
namespace kern {

namespace {

__device__ inline int2 add2(int2 a, int2 b) { return make_int2(a.x + b.x, a.y + b.y); }

// Inclusive scan across the 64 lanes of a wavefront.
__device__ inline int2 wave_incl_scan(int2 v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int ax = __shfl_up(v.x, d, 64);
        int ay = __shfl_up(v.y, d, 64);
        if (lane >= d) {
            v.x += ax;
            v.y += ay;
        }
    }
    return v;
}

// Exclusive scan of one int2 per thread over a 256-thread block.
__device__ inline int2 block_excl_scan256(int2 v, int2 *total) {
    __shared__ int2 wsum[4];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int2 inc = wave_incl_scan(v);
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    int2 base = make_int2(0, 0), tot = make_int2(0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if (i < w) base = add2(base, wsum[i]);
        tot = add2(tot, wsum[i]);
    }
    __syncthreads();
    *total = tot;
    return make_int2(base.x + inc.x - v.x, base.y + inc.y - v.y);
}

__global__ __launch_bounds__(256) void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256)
        p[i] = v;
}

// 16 bytes with the non-temporal hint: the canvas is read by the backbone,
// not by the pillar kernels.
__device__ inline void nt_store16(void *p, uint4 v) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, static_cast<u32x4 *>(p));
}

__global__ __launch_bounds__(256) void k_cell_ids(const float4 *__restrict__ pts, int32_t n, PillarGeom g,
                                                  int32_t *__restrict__ cell, int32_t *__restrict__ slot,
                                                  int32_t *__restrict__ counts) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const float4 p = pts[i];
    int c = -1;
    if (__builtin_isfinite(p.x) && __builtin_isfinite(p.y) && __builtin_isfinite(p.z) &&
        __builtin_isfinite(p.w) && p.x >= g.x0 && p.x < g.x1 && p.y >= g.y0 && p.y < g.y1 &&
        p.z >= g.z0 && p.z < g.z1) {
        // float32, round-to-nearest subtract and divide, then floor
        const float fx = floorf(__fdiv_rn(__fsub_rn(p.x, g.x0), g.v));
        const float fy = floorf(__fdiv_rn(__fsub_rn(p.y, g.y0), g.v));
        if (fx >= 0.f && fx < float(g.W) && fy >= 0.f && fy < float(g.H)) c = int(fy) * g.W + int(fx);
    }
    cell[i] = c;
    if (c >= 0) slot[i] = atomicAdd(&counts[c], 1);
}

__global__ __launch_bounds__(256) void k_scan_reduce(const int32_t *__restrict__ counts,
                                                     int32_t n_cells, int32_t *__restrict__ tile_sums,
                                                     int32_t *__restrict__ meta) {
    if (blockIdx.x == 0 && threadIdx.x == 0) meta[2] = 0;  // overfull count, appended to by the scan
    const int base = blockIdx.x * kScanTile + threadIdx.x * 8;
    int s = 0, f = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int c = base + i;
        if (c < n_cells) {
            const int v = counts[c];
            s += v;
            f += v > 0;
        }
    }
    int2 tot;
    block_excl_scan256(make_int2(s, f), &tot);
    if (threadIdx.x == 0) {
        tile_sums[2 * blockIdx.x] = tot.x;
        tile_sums[2 * blockIdx.x + 1] = tot.y;
    }
}

__global__ __launch_bounds__(256) void k_scan_down(const int32_t *__restrict__ counts, int32_t n_cells,
                                                   const int32_t *__restrict__ ts, int32_t max_pts,
                                                   int32_t *__restrict__ offsets,
                                                   int32_t *__restrict__ pcells,
                                                   int32_t *__restrict__ pcounts,
                                                   int32_t *__restrict__ poffs,
                                                   int32_t *__restrict__ overfull,
                                                   int32_t *__restrict__ meta) {
    const int base = blockIdx.x * kScanTile + threadIdx.x * 8;
    int v[8];
    int s = 0, f = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int c = base + i;
        v[i] = c < n_cells ? counts[c] : 0;
        s += v[i];
        f += v[i] > 0;
    }
    // the sums of the tiles before this one, added up by the block itself
    // (no separate scan of the tile sums); the last tile writes the totals
    int2 before = make_int2(0, 0);
    for (int t = threadIdx.x; t < int(blockIdx.x); t += 256) before = add2(before, make_int2(ts[2 * t], ts[2 * t + 1]));
    int2 prefix, tot;
    block_excl_scan256(before, &prefix);
    const int2 ex = block_excl_scan256(make_int2(s, f), &tot);
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) {
        meta[0] = prefix.x + tot.x;
        meta[1] = prefix.y + tot.y;
    }
    int off = prefix.x + ex.x;
    int p = prefix.y + ex.y;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int c = base + i;
        if (c < n_cells) {
            offsets[c] = off;
            if (v[i] > 0) {
                pcells[p] = c;
                pcounts[p] = v[i];
                poffs[p] = off;
                ++p;
                if (v[i] > max_pts) overfull[atomicAdd(&meta[2], 1)] = c;
            }
            off += v[i];
        }
    }
}

__global__ __launch_bounds__(256) void k_scatter(const int32_t *__restrict__ cell,
                                                 const int32_t *__restrict__ slot,
                                                 const int32_t *__restrict__ offsets, int32_t n,
                                                 const float4 *__restrict__ pts,
                                                 int32_t *__restrict__ member, float4 *__restrict__ sorted) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const int c = cell[i];
    if (c >= 0) {
        const int d = offsets[c] + slot[i];
        member[d] = i;
        sorted[d] = pts[i];
    }
}

__device__ inline uint32_t pack_bf16x2(float a, float b) {
    uint32_t ua = __float_as_uint(a), ub = __float_as_uint(b);
    ua += 0x7fffu + ((ua >> 16) & 1u);
    ub += 0x7fffu + ((ub >> 16) & 1u);
    return (ua >> 16) | (ub & 0xffff0000u);
}

// One point's contribution to 8 channels of its pillar: ReLU(b + W^T f),
// f = (x / hx, y / hy, (z - z0) / dz, r), maxed into mx.  The same code for
// pillars under and over the cap.
__device__ inline void pfn_point(const PfnArgs &a, const float4 pt, const float (&w0)[8], const float (&w1)[8],
                                 const float (&w2)[8], const float (&w3)[8], const float (&bb)[8], float (&mx)[8]) {
    const float f0 = pt.x * a.inv_hx;
    const float f1 = pt.y * a.inv_hy;
    const float f2 = (pt.z - a.z0) * a.inv_dz;
    const float f3 = pt.w;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        float h = bb[i] + w0[i] * f0 + w1[i] * f1 + w2[i] * f2 + w3[i] * f3;
        h = h > 0.f ? h : 0.f;  // +0 for every non-positive value
        mx[i] = fmaxf(mx[i], h);
    }
}

template <bool BF16>
__device__ inline void store_canvas8(const PfnArgs &a, int cell, int ch, const float (&mx)[8]) {
    if (BF16) {
        uint4 o;
        o.x = pack_bf16x2(mx[0], mx[1]);
        o.y = pack_bf16x2(mx[2], mx[3]);
        o.z = pack_bf16x2(mx[4], mx[5]);
        o.w = pack_bf16x2(mx[6], mx[7]);
        nt_store16(static_cast<uint16_t *>(a.canvas) + size_t(cell) * a.C + ch, o);
    } else {
        float *dst = static_cast<float *>(a.canvas) + size_t(cell) * a.C + ch;
        nt_store16(dst, make_uint4(__float_as_uint(mx[0]), __float_as_uint(mx[1]), __float_as_uint(mx[2]),
                                   __float_as_uint(mx[3])));
        nt_store16(dst + 4, make_uint4(__float_as_uint(mx[4]), __float_as_uint(mx[5]), __float_as_uint(mx[6]),
                                       __float_as_uint(mx[7])));
    }
}

// Blocks [0, a.pillar_blocks): a lane per (pillar, 8 channels) over the
// ascending pillar list from the scan: ReLU(W^T f + b) maxed over the
// pillar's points, read in segment order from `sorted`, into the pillar's
// cell; pillars over the cap are left to the other blocks.  Blocks from
// a.pillar_blocks on: one wavefront per cell over the cap moves the cap
// lowest point indices to the front of its segment (member indices and
// points) and writes the features of those points.  The lanes read the
// cell, count and segment offset together; the other cells of the canvas
// already hold zeros.  Counts go back to zero for the next frame.
template <bool BF16>
__global__ __launch_bounds__(256) void k_pfn_canvas(PfnArgs a) {
    // PFN weights and bias, read once per block into LDS (C <= 512)
    __shared__ float sw[5 * 512];
    for (int q = threadIdx.x; q < 5 * a.C; q += 256) sw[q] = q < 4 * a.C ? a.w[q] : a.b[q - 4 * a.C];
    __syncthreads();
    if (int(blockIdx.x) >= a.pillar_blocks) {
        // cells over the cap, one wavefront each
        const int lane = threadIdx.x & 63;
        const int wave = ((int(blockIdx.x) - a.pillar_blocks) * 256 + int(threadIdx.x)) >> 6;
        const int n_waves = ((int(gridDim.x) - a.pillar_blocks) * 256) >> 6;
        const int n_over = a.meta[2];
        for (int w = wave; w < n_over; w += n_waves) {
            const int c = a.overfull[w];
            const int cnt = a.counts[c];
            int32_t *seg = a.member + a.offsets[c];
            float4 *sseg = a.sorted + a.offsets[c];
            // Smallest T with #{members < T} >= max_pts.  Members are
            // distinct point indices in [0, n), so exactly max_pts members
            // lie below T.
            int lo = 1, hi = a.n;
            while (lo < hi) {
                const int mid = lo + (hi - lo) / 2;
                int below = 0;
                for (int j = lane; j < cnt; j += 64) below += seg[j] < mid;
#pragma unroll
                for (int d = 32; d >= 1; d >>= 1) below += __shfl_xor(below, d, 64);
                if (below >= a.max_pts) hi = mid;
                else lo = mid + 1;
            }
            const int T = lo;
            // Stable in-place compaction of the selected members to the
            // front: a chunk is read completely before any of it is
            // overwritten, and writes never pass the chunk being read.
            int pos = 0;
            for (int base = 0; base < cnt && pos < a.max_pts; base += 64) {
                const int j = base + lane;
                const int e = j < cnt ? seg[j] : INT_MAX;
                const bool sel = j < cnt && e < T;
                const unsigned long long m = __ballot(sel);
                const int my = pos + __popcll(m & ((1ull << lane) - 1ull));
                if (sel) {
                    seg[my] = e;
                    sseg[my] = a.pts[e];
                }
                pos += __popcll(m);
            }
            // the wave's own writes above are read back by other lanes
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            for (int ch = lane * 8; ch < a.C; ch += 64 * 8) {
                float w0[8], w1[8], w2[8], w3[8], bb[8], mx[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    w0[i] = sw[0 * a.C + ch + i];
                    w1[i] = sw[1 * a.C + ch + i];
                    w2[i] = sw[2 * a.C + ch + i];
                    w3[i] = sw[3 * a.C + ch + i];
                    bb[i] = sw[4 * a.C + ch + i];
                    mx[i] = 0.f;
                }
                for (int t = 0; t < a.max_pts; ++t) pfn_point(a, sseg[t], w0, w1, w2, w3, bb, mx);
                store_canvas8<BF16>(a, c, ch, mx);
            }
            if (lane == 0) a.counts[c] = 0;
        }
        return;
    }
    const int lanes_per_cell = a.C >> 3;
    const int gid = int(blockIdx.x) * 256 + int(threadIdx.x);
    const int p = gid / lanes_per_cell;
    const int ch = (gid - p * lanes_per_cell) * 8;
    if (p >= a.meta[1]) return;
    const int cell = a.pcells[p];
    const int cnt = a.pcounts[p];
    const int off = a.poffs[p];
    if (cnt > a.max_pts) return;  // over the cap: the blocks above
    // the cell's count back to zero, the state the next frame's K1 starts from
    if (ch == 0) a.counts[cell] = 0;
    float w0[8], w1[8], w2[8], w3[8], bb[8], mx[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        w0[i] = sw[0 * a.C + ch + i];
        w1[i] = sw[1 * a.C + ch + i];
        w2[i] = sw[2 * a.C + ch + i];
        w3[i] = sw[3 * a.C + ch + i];
        bb[i] = sw[4 * a.C + ch + i];
        mx[i] = 0.f;
    }
    // two points per step, both loads in flight (max is order-free)
    for (int t = 0; t < cnt; t += 2) {
        const float4 p0 = a.sorted[off + t];
        const bool two = t + 1 < cnt;
        const float4 p1 = a.sorted[off + (two ? t + 1 : t)];
        pfn_point(a, p0, w0, w1, w2, w3, bb, mx);
        if (two) pfn_point(a, p1, w0, w1, w2, w3, bb, mx);
    }
    store_canvas8<BF16>(a, cell, ch, mx);
}

// The canvas cells of the last frame's pillars back to zero, one lane per
// (pillar, 8 channels); the rest of the canvas holds zeros already.
template <bool BF16>
__global__ __launch_bounds__(256) void k_canvas_clear(void *canvas, const int32_t *__restrict__ pcells,
                                                      const int32_t *__restrict__ meta, int32_t C) {
    const int lanes = C >> 3;
    const int gid = int(blockIdx.x) * 256 + int(threadIdx.x);
    const int p = gid / lanes;
    if (p >= meta[1]) return;
    const size_t off = size_t(pcells[p]) * C + (gid - p * lanes) * 8;
    if (BF16) {
        nt_store16(static_cast<uint16_t *>(canvas) + off, make_uint4(0u, 0u, 0u, 0u));
    } else {
        nt_store16(static_cast<float *>(canvas) + off, make_uint4(0u, 0u, 0u, 0u));
        nt_store16(static_cast<float *>(canvas) + off + 4, make_uint4(0u, 0u, 0u, 0u));
    }
}

inline unsigned blocks_for(int64_t n, int per) { return unsigned((n + per - 1) / per); }

}  // namespace

hipError_t fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    unsigned g = blocks_for(n, 256);
    if (g > 4096) g = 4096;
    k_fill_i32<<<g, 256, 0, s>>>(p, n, v);
    return hipGetLastError();
}

hipError_t cell_ids(const float *pts, int32_t n, const PillarGeom &g, int32_t *cell, int32_t *slot,
                    int32_t *counts, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    k_cell_ids<<<blocks_for(n, 256), 256, 0, s>>>(reinterpret_cast<const float4 *>(pts), n, g, cell, slot, counts);
    return hipGetLastError();
}

hipError_t scan_reduce(const int32_t *counts, int32_t n_cells, int32_t *tile_sums, int32_t *meta, hipStream_t s) {
    k_scan_reduce<<<blocks_for(n_cells, kScanTile), 256, 0, s>>>(counts, n_cells, tile_sums, meta);
    return hipGetLastError();
}

hipError_t scan_down(const int32_t *counts, int32_t n_cells, const int32_t *tile_sums,
                     int32_t max_pts, int32_t *offsets, int32_t *pcells, int32_t *pcounts, int32_t *poffs,
                     int32_t *overfull, int32_t *meta, hipStream_t s) {
    k_scan_down<<<blocks_for(n_cells, kScanTile), 256, 0, s>>>(counts, n_cells, tile_sums, max_pts,
                                                                offsets, pcells, pcounts, poffs, overfull, meta);
    return hipGetLastError();
}

hipError_t scatter(const int32_t *cell, const int32_t *slot, const int32_t *offsets, int32_t n,
                   const float *pts, int32_t *member, float *sorted, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    k_scatter<<<blocks_for(n, 256), 256, 0, s>>>(cell, slot, offsets, n, reinterpret_cast<const float4 *>(pts),
                                                 member, reinterpret_cast<float4 *>(sorted));
    return hipGetLastError();
}

hipError_t pfn_canvas(bool bf16, PfnArgs a, int32_t max_pillars, hipStream_t s) {
    // pillar blocks, then 64 blocks for the cells over the cap when any
    // cell can exceed it
    a.pillar_blocks = int32_t(blocks_for(int64_t(max_pillars) * (a.C / 8), 256));
    const unsigned blocks = unsigned(a.pillar_blocks) + (a.n > a.max_pts ? 64u : 0u);
    if (blocks == 0) return hipSuccess;
    if (bf16) k_pfn_canvas<true><<<blocks, 256, 0, s>>>(a);
    else k_pfn_canvas<false><<<blocks, 256, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t canvas_clear(bool bf16, void *canvas, const int32_t *pcells, const int32_t *meta, int32_t C,
                        int32_t max_pillars, hipStream_t s) {
    const unsigned blocks = blocks_for(int64_t(max_pillars) * (C / 8), 256);
    if (blocks == 0) return hipSuccess;
    if (bf16) k_canvas_clear<true><<<blocks, 256, 0, s>>>(canvas, pcells, meta, C);
    else k_canvas_clear<false><<<blocks, 256, 0, s>>>(canvas, pcells, meta, C);
    return hipGetLastError();
}

}  // namespace kern
}  // namespace rtcc
