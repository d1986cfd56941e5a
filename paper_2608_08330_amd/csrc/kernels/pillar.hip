// Pillarization and point-feature canvas for gfx950.
//
// Deterministic sort of points by cell (LDS, one global atomic per non-empty (point block, tile) bin, no
// order-dependent result), five dependent launches, each
// over a group of agents released together (the blocks of the group's
// agents are interleaved, see group_block; a single release is a group of
// one).  Cells are cut into tiles of kScanTile cells, points into blocks of
// kPtsPerBlock:
//   bin_count    cell id per point; per point block, an LDS histogram of its
//                points over the tiles, the point's rank in its (block,
//                tile) bin from the LDS atomic; every non-empty bin
//                reserves its run in its tile (the only global atomics: one
//                per non-empty bin, not one per point)
//   bin_scatter  the tiles' first points (each block scans the tiles'
//                totals itself), point indices and cells in tile order
//   tile_sort    one block per tile: LDS counts of the tile's cells, their
//                scan -> the tile's pillars in ascending cell order and
//                each point's place in cell order (member, sorted)
//   pillar_lists one block per tile: its pillar list moved to its place in
//                the global lists (the block adds up the earlier tiles'
//                pillar counts itself)
//   pfn_canvas   one lane per (two pillars, 8 channels): linear 4 -> C,
//                ReLU, max over the pillar's points into its cell.  Extra
//                blocks take the few pillars over the cap: one wavefront
//                moves the cap lowest point indices (found by bisection on
//                the index value) to the front of the segment and writes
//                that pillar's features
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

// Block -> (agent row j of the group, block index b within that agent's
// grid): the agents' blocks are interleaved.  The dispatcher hands
// consecutive blocks to the XCDs in turn, so in a group of 8 every agent's
// blocks run on one XCD, and the random accesses of its pillar stage (cell
// counts, offsets, member lists) stay in that XCD's L2.
struct GroupBlock {
    int j, b, nb;  // agent row, block within the agent, blocks per agent
};
__device__ inline GroupBlock group_block(const PillarGroup &grp) {
    const int m = grp.m;
    return GroupBlock{int(blockIdx.x) % m, int(blockIdx.x) / m, int(gridDim.x) / m};
}
__device__ inline PillarBufs group_bufs(const PillarGroup &grp, int j) { return grp.bufs[grp.agent[j]]; }

__device__ inline int cell_of(const float4 p, const PillarGeom &g) {
    int c = -1;
    if (__builtin_isfinite(p.x) && __builtin_isfinite(p.y) && __builtin_isfinite(p.z) &&
        __builtin_isfinite(p.w) && p.x >= g.x0 && p.x < g.x1 && p.y >= g.y0 && p.y < g.y1 &&
        p.z >= g.z0 && p.z < g.z1) {
        // float32, round-to-nearest subtract and divide, then floor
        const float fx = floorf(__fdiv_rn(__fsub_rn(p.x, g.x0), g.v));
        const float fy = floorf(__fdiv_rn(__fsub_rn(p.y, g.y0), g.v));
        if (fx >= 0.f && fx < float(g.W) && fy >= 0.f && fy < float(g.H)) c = int(fy) * g.W + int(fx);
    }
    return c;
}

inline __device__ int blocks_of(int n) { return (n + kPtsPerBlock - 1) / kPtsPerBlock; }

// K1: cell ids, per-(block, tile) counts and the block's run in every
// tile; two points per thread.
__global__ __launch_bounds__(256) void k_bin_count(const PillarGroup grp, const PillarGeom g) {
    extern __shared__ int lds[];  // [grp.tiles] counts, then [grp.tiles] bases
    int *hist = lds, *base = lds + grp.tiles;
    const GroupBlock gb = group_block(grp);
    const int j = gb.j;
    const int n = grp.n[j];
    if (gb.b >= blocks_of(n)) return;  // the whole block: past this agent's points
    const PillarBufs B = group_bufs(grp, j);
    const float4 *pts = grp.pts[j];
    for (int t = threadIdx.x; t < grp.tiles; t += 256) hist[t] = 0;
    __syncthreads();
    int tile[2], rank[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int i = gb.b * kPtsPerBlock + u * 256 + int(threadIdx.x);
        tile[u] = -1;
        if (i < n) {
            const int c = cell_of(pts[i], g);
            B.cell[i] = c;
            if (c >= 0) {
                tile[u] = c / kScanTile;
                rank[u] = atomicAdd(&hist[tile[u]], 1);
            }
        }
    }
    __syncthreads();
    // the block's run in every tile it touches: one global atomic per
    // non-empty (block, tile) bin
    for (int t = threadIdx.x; t < grp.tiles; t += 256) {
        const int h = hist[t];
        if (h > 0) base[t] = atomicAdd(&B.ttotal[t], h);
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 2; ++u)
        if (tile[u] >= 0) B.slot[gb.b * kPtsPerBlock + u * 256 + int(threadIdx.x)] = base[tile[u]] + rank[u];
}

// K2: every point to its place in tile order.  Each block scans the tiles'
// totals in LDS into the tiles' first points; the agent's first block also
// stores them (tstart) and the point count.
__global__ __launch_bounds__(256) void k_bin_scatter(const PillarGroup grp) {
    extern __shared__ int ts[];  // [grp.tiles + 1]
    const GroupBlock gb = group_block(grp);
    const int j = gb.j;
    const int n = grp.n[j];
    const PillarBufs B = group_bufs(grp, j);
    const int T = grp.tiles;
    const int per = (T + 255) / 256;
    int s = 0;
    for (int r = 0; r < per; ++r) {
        const int t = int(threadIdx.x) * per + r;
        if (t < T) s += B.ttotal[t];
    }
    int2 tot;
    int acc = block_excl_scan256(make_int2(s, 0), &tot).x;
    for (int r = 0; r < per; ++r) {
        const int t = int(threadIdx.x) * per + r;
        if (t < T) {
            ts[t] = acc;
            acc += B.ttotal[t];
        }
    }
    if (threadIdx.x == 0) ts[T] = tot.x;
    __syncthreads();
    if (gb.b == 0) {
        for (int t = threadIdx.x; t <= T; t += 256) B.tstart[t] = ts[t];
        if (threadIdx.x == 0) {
            B.meta[0] = tot.x;
            B.meta[1] = 0;  // the pillar lists' kernel writes the pillar count
            B.meta[2] = 0;  // pillars over the cap, appended to by the tile sort
        }
    }
    if (gb.b >= blocks_of(n)) return;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int i = gb.b * kPtsPerBlock + u * 256 + int(threadIdx.x);
        if (i < n) {
            const int c = B.cell[i];
            if (c >= 0) {
                const int d = ts[c / kScanTile] + B.slot[i];
                B.binned[d] = i;
                B.cellb[d] = c;
            }
        }
    }
}

// K4: one block per tile of cells.
constexpr int kSortCache = 8;
__global__ __launch_bounds__(256) void k_tile_sort(const PillarGroup grp, int32_t max_pts) {
    __shared__ int cnt[kScanTile];
    __shared__ int loff[kScanTile];
    const GroupBlock gb = group_block(grp);
    const int j = gb.j, t = gb.b;
    const PillarBufs B = group_bufs(grp, j);
    const float4 *pts = grp.pts[j];
    const int lo = B.tstart[t], hi = B.tstart[t + 1];
    const int c0 = t * kScanTile;
    for (int q = threadIdx.x; q < kScanTile; q += 256) cnt[q] = 0;
    __syncthreads();
    // the tile's first kSortCache * 256 points keep their cell and rank in
    // registers between the passes; any further ones go through `rank`
    int lcell[kSortCache], rk[kSortCache];
#pragma unroll
    for (int u = 0; u < kSortCache; ++u) {
        const int e = lo + int(threadIdx.x) + u * 256;
        lcell[u] = e < hi ? B.cellb[e] - c0 : 0;
    }
#pragma unroll
    for (int u = 0; u < kSortCache; ++u)
        if (lo + int(threadIdx.x) + u * 256 < hi) rk[u] = atomicAdd(&cnt[lcell[u]], 1);
    for (int e = lo + int(threadIdx.x) + kSortCache * 256; e < hi; e += 256)
        B.rank[e] = atomicAdd(&cnt[B.cellb[e] - c0], 1);
    __syncthreads();
    int v[8];
    int s = 0, f = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        v[i] = cnt[threadIdx.x * 8 + i];
        s += v[i];
        f += v[i] > 0;
    }
    int2 tot;
    const int2 ex = block_excl_scan256(make_int2(s, f), &tot);
    int off = ex.x, q = ex.y;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int lc = int(threadIdx.x) * 8 + i;
        loff[lc] = off;
        if (v[i] > 0) {
            const int sidx = c0 + q;
            B.tcell[sidx] = c0 + lc;
            B.tcount[sidx] = v[i];
            B.toff[sidx] = lo + off;
            if (v[i] > max_pts) B.overfull[atomicAdd(&B.meta[2], 1)] = sidx;
            ++q;
        }
        off += v[i];
    }
    if (threadIdx.x == 0) B.npil[t] = tot.y;
    __syncthreads();
    int idx[kSortCache];
#pragma unroll
    for (int u = 0; u < kSortCache; ++u) {
        const int e = lo + int(threadIdx.x) + u * 256;
        idx[u] = e < hi ? B.binned[e] : 0;
    }
#pragma unroll
    for (int u = 0; u < kSortCache; ++u) {
        const int e = lo + int(threadIdx.x) + u * 256;
        if (e < hi) {
            const int d = lo + loff[lcell[u]] + rk[u];
            B.member[d] = idx[u];
            B.sorted[d] = pts[idx[u]];
        }
    }
    for (int e = lo + int(threadIdx.x) + kSortCache * 256; e < hi; e += 256) {
        const int d = lo + loff[B.cellb[e] - c0] + B.rank[e];
        const int i = B.binned[e];
        B.member[d] = i;
        B.sorted[d] = pts[i];
    }
}

// K5: the tiles' pillar lists concatenated into the global ones, one block
// per tile: its first global pillar is the sum of the earlier tiles'
// pillar counts.  The last tile's block writes the pillar count.
__global__ __launch_bounds__(256) void k_pillar_lists(const PillarGroup grp) {
    const GroupBlock gb = group_block(grp);
    const int t = gb.b;
    const PillarBufs B = group_bufs(grp, gb.j);
    int s = 0;
    for (int q = threadIdx.x; q < t; q += 256) s += B.npil[q];
    int2 tot;
    block_excl_scan256(make_int2(s, 0), &tot);
    const int first = tot.x, np = B.npil[t];
    const int c0 = t * kScanTile;
    for (int q = threadIdx.x; q < np; q += 256) {
        B.pcells[first + q] = B.tcell[c0 + q];
        B.pcounts[first + q] = B.tcount[c0 + q];
        B.poffs[first + q] = B.toff[c0 + q];
    }
    if (t == grp.tiles - 1 && threadIdx.x == 0) B.meta[1] = first + np;
    // the tile's point total back to zero, the state the next frame's bin
    // count starts from (every reader of it has finished)
    if (threadIdx.x == 0) B.ttotal[t] = 0;
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
__device__ inline void store_canvas8(const PfnArgs &a, void *canvas, int cell, int ch, const float (&mx)[8]) {
    if (BF16) {
        uint4 o;
        o.x = pack_bf16x2(mx[0], mx[1]);
        o.y = pack_bf16x2(mx[2], mx[3]);
        o.z = pack_bf16x2(mx[4], mx[5]);
        o.w = pack_bf16x2(mx[6], mx[7]);
        nt_store16(static_cast<uint16_t *>(canvas) + size_t(cell) * a.C + ch, o);
    } else {
        float *dst = static_cast<float *>(canvas) + size_t(cell) * a.C + ch;
        nt_store16(dst, make_uint4(__float_as_uint(mx[0]), __float_as_uint(mx[1]), __float_as_uint(mx[2]),
                                   __float_as_uint(mx[3])));
        nt_store16(dst + 4, make_uint4(__float_as_uint(mx[4]), __float_as_uint(mx[5]), __float_as_uint(mx[6]),
                                       __float_as_uint(mx[7])));
    }
}

// Blocks [0, a.pillar_blocks): a lane per (two pillars, 8 channels) of the
// global pillar list takes ReLU(W^T f + b) maxed over the pillar's points,
// read in segment order from `sorted`, into the pillar's cell.  Pillars
// over the cap are left to the other blocks.  Blocks from
// a.pillar_blocks on: one wavefront per pillar over the cap moves the cap
// lowest point indices to the front of its segment (member indices and
// points) and writes the features of those points.  The other cells of the
// canvas already hold zeros.
template <bool BF16>
__global__ __launch_bounds__(256) void k_pfn_canvas(const PfnArgs a, const PillarGroup grp) {
    // PFN weights and bias, read once per block into LDS (C <= 512)
    __shared__ float sw[5 * 512];
    for (int q = threadIdx.x; q < 5 * a.C; q += 256) sw[q] = q < 4 * a.C ? a.w[q] : a.b[q - 4 * a.C];
    __syncthreads();
    const GroupBlock gb = group_block(grp);
    const int j = gb.j;
    const PillarBufs B = group_bufs(grp, j);
    void *const canvas = a.canvas ? a.canvas : B.canvas;
    if (gb.b >= a.pillar_blocks) {
        // pillars over the cap, one wavefront each
        const int lane = threadIdx.x & 63;
        const int wave = ((gb.b - a.pillar_blocks) * 256 + int(threadIdx.x)) >> 6;
        const int n_waves = ((gb.nb - a.pillar_blocks) * 256) >> 6;
        const int n_over = B.meta[2];
        const float4 *pts = grp.pts[j];
        for (int w = wave; w < n_over; w += n_waves) {
            const int sidx = B.overfull[w];  // in the tiles' pillar lists
            const int c = B.tcell[sidx];
            const int cnt = B.tcount[sidx];
            int32_t *seg = B.member + B.toff[sidx];
            float4 *sseg = B.sorted + B.toff[sidx];
            if (!a.replay) {
                // Smallest T with #{members < T} >= max_pts.  Members are
                // distinct point indices in [0, n), so exactly max_pts members
                // lie below T.
                int lo = 1, hi = grp.n[j];
                while (lo < hi) {
                    const int mid = lo + (hi - lo) / 2;
                    int below = 0;
                    for (int q = lane; q < cnt; q += 64) below += seg[q] < mid;
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
                    const int q = base + lane;
                    const int e = q < cnt ? seg[q] : INT_MAX;
                    const bool sel = q < cnt && e < T;
                    const unsigned long long m = __ballot(sel);
                    const int my = pos + __popcll(m & ((1ull << lane) - 1ull));
                    if (sel) {
                        seg[my] = e;
                        sseg[my] = pts[e];
                    }
                    pos += __popcll(m);
                }
                // the wave's own writes above are read back by other lanes
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            }
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
                store_canvas8<BF16>(a, canvas, c, ch, mx);
            }
        }
        return;
    }
    // two pillars per lane (8 channels of each): their loads are in flight
    // together
    const int lanes_per_cell = a.C >> 3;
    const int gid = gb.b * 256 + int(threadIdx.x);
    const int pp = gid / lanes_per_cell;
    const int ch = (gid - pp * lanes_per_cell) * 8;
    const int P = B.meta[1];
    const int p0 = 2 * pp;
    if (p0 >= P) return;
    const bool has1 = p0 + 1 < P;
    const int cell0 = B.pcells[p0], cnt0 = B.pcounts[p0], off0 = B.poffs[p0];
    const int cell1 = has1 ? B.pcells[p0 + 1] : 0;
    const int cnt1 = has1 ? B.pcounts[p0 + 1] : 0;
    const int off1 = has1 ? B.poffs[p0 + 1] : off0;
    // pillars over the cap are left to the blocks above
    const int n0 = cnt0 <= a.max_pts ? cnt0 : 0;
    const int n1 = cnt1 <= a.max_pts ? cnt1 : 0;
    float w0[8], w1[8], w2[8], w3[8], bb[8], m0[8], m1[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        w0[i] = sw[0 * a.C + ch + i];
        w1[i] = sw[1 * a.C + ch + i];
        w2[i] = sw[2 * a.C + ch + i];
        w3[i] = sw[3 * a.C + ch + i];
        bb[i] = sw[4 * a.C + ch + i];
        m0[i] = 0.f;
        m1[i] = 0.f;
    }
    // the last point of a pillar stands in for the points past its end (the
    // max is unchanged by a repeat); every index stays inside its segment
    const int l0 = n0 > 0 ? n0 - 1 : 0, l1 = n1 > 0 ? n1 - 1 : 0;
    const int tmax = n0 > n1 ? n0 : n1;
    for (int t = 0; t < tmax; ++t) {
        const float4 q0 = B.sorted[off0 + (t < l0 ? t : l0)];
        const float4 q1 = B.sorted[off1 + (t < l1 ? t : l1)];
        if (n0 > 0) pfn_point(a, q0, w0, w1, w2, w3, bb, m0);
        if (n1 > 0) pfn_point(a, q1, w0, w1, w2, w3, bb, m1);
    }
    if (n0 > 0) store_canvas8<BF16>(a, canvas, cell0, ch, m0);
    if (n1 > 0) store_canvas8<BF16>(a, canvas, cell1, ch, m1);
}

// The canvas cells of the last frame's pillars back to zero, one lane per
// (pillar, 8 channels), for every agent of the group (its pillar list and
// count are those of its last encoder); the rest of each canvas holds zeros
// already.
template <bool BF16>
__global__ __launch_bounds__(256) void k_canvas_clear(const PillarGroup grp, int32_t C) {
    const GroupBlock gb = group_block(grp);
    const PillarBufs B = group_bufs(grp, gb.j);
    const int lanes = C >> 3;
    const int gid = gb.b * 256 + int(threadIdx.x);
    const int p = gid / lanes;
    if (p >= B.meta[1]) return;
    const size_t off = size_t(B.pcells[p]) * C + (gid - p * lanes) * 8;
    if (BF16) {
        nt_store16(static_cast<uint16_t *>(B.canvas) + off, make_uint4(0u, 0u, 0u, 0u));
    } else {
        nt_store16(static_cast<float *>(B.canvas) + off, make_uint4(0u, 0u, 0u, 0u));
        nt_store16(static_cast<float *>(B.canvas) + off + 4, make_uint4(0u, 0u, 0u, 0u));
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

hipError_t bin_count(const PillarGroup &grp, const PillarGeom &g, hipStream_t s) {
    if (grp.n_max <= 0) return hipSuccess;
    k_bin_count<<<blocks_for(grp.n_max, kPtsPerBlock) * unsigned(grp.m), 256, size_t(grp.tiles) * 8, s>>>(grp, g);
    return hipGetLastError();
}

hipError_t bin_scatter(const PillarGroup &grp, hipStream_t s) {
    // at least one block per agent: the first one stores the tile starts
    const unsigned nb = grp.n_max > 0 ? blocks_for(grp.n_max, kPtsPerBlock) : 1u;
    k_bin_scatter<<<nb * unsigned(grp.m), 256, size_t(grp.tiles + 1) * 4, s>>>(grp);
    return hipGetLastError();
}

hipError_t tile_sort(const PillarGroup &grp, int32_t max_pts, hipStream_t s) {
    k_tile_sort<<<unsigned(grp.tiles) * unsigned(grp.m), 256, 0, s>>>(grp, max_pts);
    return hipGetLastError();
}

hipError_t pillar_lists(const PillarGroup &grp, hipStream_t s) {
    k_pillar_lists<<<unsigned(grp.tiles) * unsigned(grp.m), 256, 0, s>>>(grp);
    return hipGetLastError();
}

hipError_t pfn_canvas(bool bf16, PfnArgs a, const PillarGroup &grp, int32_t max_pillars, hipStream_t s) {
    // pillar blocks, then 64 blocks for the cells over the cap when any
    // agent's cell can exceed it
    a.pillar_blocks = int32_t(blocks_for(int64_t((max_pillars + 1) / 2) * (a.C / 8), 256));
    const unsigned blocks = unsigned(a.pillar_blocks) + (grp.n_max > a.max_pts ? 64u : 0u);
    if (blocks == 0) return hipSuccess;
    const unsigned grid = blocks * unsigned(grp.m);
    if (bf16) k_pfn_canvas<true><<<grid, 256, 0, s>>>(a, grp);
    else k_pfn_canvas<false><<<grid, 256, 0, s>>>(a, grp);
    return hipGetLastError();
}

hipError_t canvas_clear(bool bf16, const PillarGroup &grp, int32_t C, int32_t max_pillars, hipStream_t s) {
    const unsigned blocks = blocks_for(int64_t(max_pillars) * (C / 8), 256);
    if (blocks == 0) return hipSuccess;
    const unsigned grid = blocks * unsigned(grp.m);
    if (bf16) k_canvas_clear<true><<<grid, 256, 0, s>>>(grp, C);
    else k_canvas_clear<false><<<grid, 256, 0, s>>>(grp, C);
    return hipGetLastError();
}

}  // namespace kern
}  // namespace rtcc
