// Rotated non-maximum suppression on bird's-eye-view boxes, after decoding
// (part of the detection post-processing that ends T^det, Sec. V-A3).
//
// Input: the decoded records rec[n][9] (x, y, z, w, l, h, yaw, score,
// anchor index bits) in ascending anchor index, n = *count on the device.
//   k_nms_rank     rank of every record: records with a higher score, plus
//                  records with the same score and a lower anchor index
//                  (= a lower record index, the records being in anchor
//                  order), as one 64-bit key compare (score bits, then the
//                  complemented index).  O(n^2) compares over tiles of 256
//                  keys in LDS, split over up to kNmsRankSplits blocks per
//                  record tile (partial counts, summed by the gather); the
//                  ranks are a permutation, so the order is unique.
//   k_nms_gather   the first m = min(n, max_candidates) records by rank:
//                  order[rank] = record, footprint (x, y, w, l, cos yaw,
//                  sin yaw, valid) as f64.
//   k_nms_mask     bit b of word (a, b / 64) is set iff b > a and the BEV
//                  IoU of candidates a and b exceeds the threshold; one
//                  block per 64 x 64 tile, which lists the pairs whose
//                  circumcircles meet in LDS and then evaluates that list
//                  densely; the rows with a nonzero word in a later chunk
//                  are listed per column chunk.  IoU in float64: the intersection area is the
//                  shoelace sum over the edge pieces of each rectangle
//                  inside the other (Cyrus-Beck clipped, crossing points
//                  shared by the two pieces that meet there); pairs whose
//                  centres are farther apart than the sum of their
//                  circumradii are disjoint and skip the clipping.  A box
//                  with a non-finite parameter or w <= 0 or l <= 0 overlaps
//                  nothing.
//   k_nms_select   one wavefront walks the ranking 64 rows at a time: the
//                  rows removed by earlier chunks are the OR of the listed
//                  words of the kept rows (copied into LDS first), then the
//                  chunk resolves itself from its in-chunk suppressors.  The
//                  kept records are then compacted in ascending record
//                  (anchor) order.
// Everything is integer or float64 except the scores, which are compared as
// stored: the decisions do not depend on the grid or the timing.
#include "kernels.hpp"

#include <cmath>

namespace rtcc {
namespace kern {

namespace {

constexpr int kRecFloats = 9;
constexpr int kFoot = kNmsFootDoubles;  // x, y, w, l, cos, sin, valid, circumradius

// Ranking key of record i: an order-preserving image of the score above the
// complement of i, so key_j > key_i iff record j precedes record i (higher
// score, or equal score and lower index).  The image flips the sign bit of
// a non-negative float and every bit of a negative one, which orders all
// finite and infinite values like the numbers (-0 is taken as +0); a NaN
// maps to 0 and ranks after every number (callers reject NaN scores).
__device__ inline unsigned long long rank_key(const NmsArgs &a, int i) {
    const float sc = a.rec[size_t(i) * kRecFloats + 7];
    uint32_t bits = sc == 0.f ? 0u : __float_as_uint(sc);
    uint32_t ord = (bits >> 31) ? ~bits : (bits | 0x80000000u);
    if (sc != sc) ord = 0u;
    return (static_cast<unsigned long long>(ord) << 32) | (0xffffffffu - uint32_t(i));
}

// Blocks (tile I of 256 records, split v of the key tiles): each thread
// counts the records of the key tiles J = v, v + S, ... that precede its own
// record and writes that partial count; the gather sums the S partials.
// No atomics: every partial is written once.  Grid-stride over (I, v).
__global__ __launch_bounds__(256) void k_nms_rank(NmsArgs a) {
    __shared__ unsigned long long tk[256];
    const int n = *a.count;
    const int T = (n + 255) / 256;
    const int S = T < kNmsRankSplits ? T : kNmsRankSplits;
    for (int item = blockIdx.x; item < T * S; item += gridDim.x) {  // uniform over the block
        const int I = item / S, v = item - (item / S) * S;
        const int i = I * 256 + int(threadIdx.x);
        const unsigned long long ki = i < n ? rank_key(a, i) : ~0ull;
        if (a.bad_score && v == 0 && i < n) {
            const float sc = a.rec[size_t(i) * kRecFloats + 7];
            if (sc != sc) *a.bad_score = 1;
        }
        int r = 0;
        for (int J = v; J < T; J += S) {
            const int j0 = J * 256;
            const int jn = n - j0 < 256 ? n - j0 : 256;
            __syncthreads();  // the previous tile has been read
            tk[threadIdx.x] = int(threadIdx.x) < jn ? rank_key(a, j0 + int(threadIdx.x)) : 0ull;
            __syncthreads();
#pragma unroll 8
            for (int q = 0; q < 256; ++q) r += tk[q] > ki;  // padding keys 0 never count
        }
        if (i < n) a.partial[size_t(v) * n + i] = r;
        __syncthreads();
    }
}

__device__ inline void gather_one(const NmsArgs &a, int i, int r) {
    a.order[r] = i;
    const float *p = a.rec + size_t(i) * kRecFloats;
    const double x = p[0], y = p[1], w = p[3], l = p[4], yaw = p[6];
    const bool ok = isfinite(x) && isfinite(y) && isfinite(w) && isfinite(l) && isfinite(yaw) && w > 0.0 && l > 0.0;
    double *f = a.foot + size_t(r) * kFoot;
    f[0] = x;
    f[1] = y;
    f[2] = w;
    f[3] = l;
    f[4] = ok ? cos(yaw) : 1.0;
    f[5] = ok ? sin(yaw) : 0.0;
    f[6] = ok ? 1.0 : 0.0;
    f[7] = ok ? 0.5 * sqrt(w * w + l * l) : 0.0;  // circumradius
}

__global__ __launch_bounds__(256) void k_nms_gather(NmsArgs a) {
    if (blockIdx.x == 0)  // the mask kernel counts the listed rows per column chunk from zero
        for (int c = threadIdx.x; c < (a.max_candidates + 63) / 64; c += 256) a.colcount[c] = 0;
    const int n = *a.count;
    const int T = (n + 255) / 256;
    const int S = T < kNmsRankSplits ? T : kNmsRankSplits;
    for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) {
        int r = 0;
        for (int v = 0; v < S; ++v) r += a.partial[size_t(v) * n + i];
        a.rank[i] = r;
        if (r < a.max_candidates) gather_one(a, i, r);
    }
}

template <typename R>
struct Foot {
    R x, y, w, l, c, s, rad;
    bool ok;
};

template <typename R>
__device__ inline Foot<R> load_foot(const double *f) {
    Foot<R> b;
    b.x = R(f[0]);
    b.y = R(f[1]);
    b.w = R(f[2]);
    b.l = R(f[3]);
    b.c = R(f[4]);
    b.s = R(f[5]);
    b.ok = f[6] != 0.0;
    b.rad = R(f[7]);
    return b;
}

// corners counter-clockwise: (+l/2, +w/2), (-l/2, +w/2), (-l/2, -w/2),
// (+l/2, -w/2) in the box frame (l along the heading), relative to (ox, oy)
template <typename R>
__device__ inline void foot_corners(const Foot<R> &b, R ox, R oy, R *px, R *py) {
#pragma clang fp contract(off)
    const R hl = R(0.5) * b.l, hw = R(0.5) * b.w;
    const R sa[4] = {hl, -hl, -hl, hl}, sb[4] = {hw, hw, -hw, -hw};
    const R cx = b.x - ox, cy = b.y - oy;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        px[k] = cx + (sa[k] * b.c - sb[k] * b.s);
        py[k] = cy + (sa[k] * b.s + sb[k] * b.c);
    }
}

// Twice the area of the intersection of two counter-clockwise rectangles P
// and Q.  The boundary of the intersection consists of the pieces of P's
// edges inside Q and of Q's edges inside P; its shoelace sum (Green's
// theorem) is twice the area.  Each piece is the part of an edge inside the
// other rectangle's four half-planes cross(e_j, p - q_j) >= 0 (Cyrus-Beck
// clipping; the bounds are kept as fractions and compared crosswise, one
// division per end).  Where a piece of P ends on an edge of Q, the piece of
// Q begins at the same point: both take it from P's parametrisation, so the
// boundary closes even for nearly parallel edges.  An edge of P lying on an
// edge of Q counts once, for P, if both run the same way; an edge of Q on
// an edge of P never counts.  No fused multiply-add: these collinearity
// tests need exact zeros.  Fixed trip counts: registers only.
template <typename R>
__device__ __forceinline__ R inter_twice(const R *px, const R *py, const R *qx, const R *qy) {
#pragma clang fp contract(off)
    R pdx[4], pdy[4], qdx[4], qdy[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        pdx[k] = px[(k + 1) & 3] - px[k];
        pdy[k] = py[(k + 1) & 3] - py[k];
        qdx[k] = qx[(k + 1) & 3] - qx[k];
        qdy[k] = qy[(k + 1) & 3] - qy[k];
    }
    R AL[4][4], BE[4][4];  // P edge i against Q's edge line j
    R twice = R(0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        R n0 = R(0), d0 = R(1), n1 = R(1), d1 = R(1);
        bool empty = false;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const R al = qdx[j] * (py[i] - qy[j]) - qdy[j] * (px[i] - qx[j]);
            const R be = qdx[j] * pdy[i] - qdy[j] * pdx[i];
            AL[i][j] = al;
            BE[i][j] = be;
            if (be > R(0)) {
                if (-al * d0 > n0 * be) {
                    n0 = -al;
                    d0 = be;
                }
            } else if (be < R(0)) {
                if (al * d1 < n1 * -be) {
                    n1 = al;
                    d1 = -be;
                }
            } else if (al < R(0) || (al == R(0) && !(qdx[j] * pdx[i] + qdy[j] * pdy[i] > R(0)))) {
                empty = true;
            }
        }
        const R t0 = n0 / d0, t1 = n1 / d1;
        if (!empty && t0 < t1) {
            const R x0 = px[i] + t0 * pdx[i], y0 = py[i] + t0 * pdy[i];
            const R x1 = px[i] + t1 * pdx[i], y1 = py[i] + t1 * pdy[i];
            twice += x0 * y1 - x1 * y0;
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        R n0 = R(0), d0 = R(1), n1 = R(1), d1 = R(1);
        bool empty = false;
        // the chosen bounds as (P edge: corner, direction, AL, BE)
        R ax0 = qx[j], ay0 = qy[j], ax1 = qx[(j + 1) & 3], ay1 = qy[(j + 1) & 3];
        R cx0 = R(0), cy0 = R(0), cal0 = R(0), cbe0 = R(1), cx1 = R(0), cy1 = R(0), cal1 = R(0), cbe1 = R(1);
        R ex0 = R(0), ey0 = R(0), ex1 = R(0), ey1 = R(0);
        bool b0 = false, b1 = false;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const R al = pdx[i] * (qy[j] - py[i]) - pdy[i] * (qx[j] - px[i]);
            const R be = pdx[i] * qdy[j] - pdy[i] * qdx[j];
            if (be > R(0)) {
                if (-al * d0 > n0 * be) {
                    n0 = -al;
                    d0 = be;
                    b0 = true;
                    cx0 = px[i];
                    cy0 = py[i];
                    ex0 = pdx[i];
                    ey0 = pdy[i];
                    cal0 = AL[i][j];
                    cbe0 = BE[i][j];
                }
            } else if (be < R(0)) {
                if (al * d1 < n1 * -be) {
                    n1 = al;
                    d1 = -be;
                    b1 = true;
                    cx1 = px[i];
                    cy1 = py[i];
                    ex1 = pdx[i];
                    ey1 = pdy[i];
                    cal1 = AL[i][j];
                    cbe1 = BE[i][j];
                }
            } else if (al <= R(0)) {
                empty = true;
            }
        }
        if (empty || !(n0 / d0 < n1 / d1)) continue;
        if (b0) {
            const R t = -cal0 / cbe0;
            ax0 = cx0 + t * ex0;
            ay0 = cy0 + t * ey0;
        }
        if (b1) {
            const R t = -cal1 / cbe1;
            ax1 = cx1 + t * ex1;
            ay1 = cy1 + t * ey1;
        }
        twice += ax0 * ay1 - ax1 * ay0;
    }
    return twice;
}

// BEV IoU of two footprints (0 if either is invalid or they are farther
// apart than the sum of their circumradii), coordinates relative to A's
// centre, in the arithmetic R.
template <typename R>
__device__ __forceinline__ R foot_iou(const Foot<R> &A, const Foot<R> &B) {
#pragma clang fp contract(off)
    if (!A.ok || !B.ok) return R(0);
    const R dx = A.x - B.x, dy = A.y - B.y;
    if (dx * dx + dy * dy > (A.rad + B.rad) * (A.rad + B.rad)) return R(0);
    R px[4], py[4], qx[4], qy[4];
    foot_corners(A, A.x, A.y, px, py);
    foot_corners(B, A.x, A.y, qx, qy);
    const R twice = inter_twice(px, py, qx, qy);
    const R inter = twice > R(0) ? R(0.5) * twice : R(0);
    const R uni = A.w * A.l + B.w * B.l - inter;
    return uni > R(0) ? inter / uni : R(0);
}

// Whether the footprints' circumcircles meet in float32 or in float64, the
// same comparisons foot_iou makes before clipping: a pair for which both
// fail has IoU 0 in both precisions.
__device__ __forceinline__ bool circles_meet(const double *A, const double *B) {
#pragma clang fp contract(off)
    const float dxf = float(A[0]) - float(B[0]), dyf = float(A[1]) - float(B[1]);
    const float rf = float(A[7]) + float(B[7]);
    const double dx = A[0] - B[0], dy = A[1] - B[1], rd = A[7] + B[7];
    return !(dxf * dxf + dyf * dyf > rf * rf) || !(dx * dx + dy * dy > rd * rd);
}

// The decision IoU > threshold, taken in float64.  The float32 evaluation
// of the same formula decides first whenever it lies more than kFilter from
// the threshold: its rounding error, for footprints whose coordinates
// relative to A's centre are bounded by their circumradii, is orders of
// magnitude below that margin, so it agrees with the float64 decision.
constexpr float kFilter = 1e-3f;

__device__ __forceinline__ bool suppresses(const double *fa, const double *fb, double thr) {
    const float v = foot_iou(load_foot<float>(fa), load_foot<float>(fb));
    if (v > float(thr) + kFilter) return true;
    if (v < float(thr) - kFilter) return false;
    return foot_iou(load_foot<double>(fa), load_foot<double>(fb)) > thr;
}

// Column chunk c of the mask: the rows of earlier chunks that have a
// nonzero word there are listed from colrows[col_base(c)], at most 64 c.
__host__ __device__ inline int64_t col_base(int c) { return int64_t(64) * c * (c - 1) / 2; }

// One 64 x 64 tile (row chunk rb, column chunk cb >= rb) of the suppression
// matrix.  The pairs whose footprints' circumcircles meet (in float32 or
// float64: the two tests that can let `suppresses` return true) are first
// compacted into an LDS list, then the block evaluates that list, so the
// clipping runs on dense lanes instead of the few close pairs scattered
// over the tile.  Writes every word (row, cb) of the tile (no zeroing
// needed), lists the rows with a nonzero off-diagonal word, and on the
// diagonal tile the transposed words: for every column, the earlier rows
// of its own chunk that suppress it.
__global__ __launch_bounds__(256) void k_nms_mask(NmsArgs a) {
    __shared__ double fr[64 * kFoot], fc[64 * kFoot];
    __shared__ unsigned short list[64 * 64];
    __shared__ unsigned long long rowbits[64], tq[64];
    __shared__ int nlist;
    const int n = *a.count;
    const int m = n < a.max_candidates ? n : a.max_candidates;
    const int T = (m + 63) / 64;
    const int words = (a.max_candidates + 63) / 64;
    const int tid = threadIdx.x;
    for (int item = blockIdx.x; item < T * (T + 1) / 2; item += gridDim.x) {  // uniform over the block
        int tri = item, rb = 0;
        while (tri >= T - rb) {
            tri -= T - rb;
            ++rb;
        }
        const int cb = rb + tri;
        const int r0 = rb * 64, c0 = cb * 64;
        for (int q = tid; q < 64 * kFoot; q += 256) {
            const int k = q / kFoot;
            fr[q] = r0 + k < m ? a.foot[size_t(r0) * kFoot + q] : 0.0;
            fc[q] = c0 + k < m ? a.foot[size_t(c0) * kFoot + q] : 0.0;
        }
        if (tid < 64) {
            rowbits[tid] = 0ull;
            tq[tid] = 0ull;
        }
        if (tid == 0) nlist = 0;
        __syncthreads();
        // close pairs (row i, column j), j > i on the diagonal tile
        const int i = tid >> 2;
        for (int k = 0; k < 16; ++k) {
            const int j = (tid & 3) * 16 + k;
            bool close = false;
            if (r0 + i < m && c0 + j < m && (cb > rb || j > i)) {
                const double *A = fr + i * kFoot, *B = fc + j * kFoot;
                if (A[6] != 0.0 && B[6] != 0.0) close = circles_meet(A, B);
            }
            if (close) list[atomicAdd(&nlist, 1)] = static_cast<unsigned short>((i << 6) | j);
        }
        __syncthreads();
        const int nl = nlist;
        for (int q = tid; q < nl; q += 256) {
            const int ii = list[q] >> 6, jj = list[q] & 63;
            if (suppresses(fr + ii * kFoot, fc + jj * kFoot, a.iou_threshold)) {
                atomicOr(&rowbits[ii], 1ull << jj);
                if (cb == rb) atomicOr(&tq[jj], 1ull << ii);
            }
        }
        __syncthreads();
        if (tid < 64 && r0 + tid < m) {
            const unsigned long long w = rowbits[tid];
            a.mask[size_t(r0 + tid) * words + cb] = w;
            if (cb != rb && w) a.colrows[col_base(cb) + atomicAdd(&a.colcount[cb], 1)] = r0 + tid;
        }
        if (cb == rb && tid < 64 && c0 + tid < m) a.mask_t[c0 + tid] = tq[tid];
        __syncthreads();  // the tile's LDS is reused by the next item
    }
}

__device__ inline unsigned long long uniform64(unsigned long long v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(v >> 32));
    return (static_cast<unsigned long long>(hi) << 32) | lo;
}

// OR over the 64 lanes of a wavefront (DPP row shifts, then row
// broadcasts; lane 63 holds the total), returned to every lane.
__device__ inline uint32_t wave_or32(uint32_t v) {
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x111, 0xf, 0xf, false);  // row_shr:1
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x112, 0xf, 0xf, false);  // row_shr:2
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x114, 0xf, 0xf, false);  // row_shr:4
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x118, 0xf, 0xf, false);  // row_shr:8
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x142, 0xa, 0xf, false);  // row_bcast:15
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x143, 0xc, 0xf, false);  // row_bcast:31
    return __builtin_amdgcn_readlane(v, 63);
}
__device__ inline unsigned long long wave_or64(unsigned long long v) {
    return (static_cast<unsigned long long>(wave_or32(uint32_t(v >> 32))) << 32) | wave_or32(uint32_t(v));
}

// The same resolution in parallel: lane r holds `sup`, the earlier rows of
// the chunk that suppress row r.  kept = standing rows none of whose kept
// suppressors exist, iterated from kept = standing: after t rounds rows
// 0 .. t-1 are final, so the iteration stops at the unique fixed point
// within 65 rounds (usually a few).
__device__ inline unsigned long long resolve_chunk_parallel(unsigned long long rem, unsigned long long sup, int rows) {
    const unsigned long long rowmask = rows >= 64 ? ~0ull : (1ull << rows) - 1ull;
    const int lane = threadIdx.x & 63;
    const unsigned long long standing = ~uniform64(rem) & rowmask;
    unsigned long long kept = standing;
    for (int it = 0; it <= 64; ++it) {
        const bool mine = ((standing >> lane) & 1ull) && !(kept & sup);
        const unsigned long long next = __ballot(mine);
        if (next == kept) break;
        kept = next;
    }
    return kept;
}

constexpr int kSelectThreads = 1024;
constexpr int kMaxWords = kNmsMaxCandidates / 64;

// Kept candidates (bit q of keep[q / 64] for ranking position q) -> flags
// by record (an LDS bitmap up to kFlagBits records, else a.flag, cleared at
// the start of the select kernels), then the kept records in ascending
// record (anchor) order.  Called by every thread of a kSelectThreads block.
constexpr int kFlagBits = 131072;

__device__ void compact_kept(const NmsArgs &a, const unsigned long long *keep, int m, int n) {
    __shared__ uint32_t fbits[kFlagBits / 32];
    __shared__ int wsum[kSelectThreads / 64];
    __shared__ int base_sh;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const bool lds = n <= kFlagBits;
    if (lds) {
        for (int w = tid; w < (n + 31) / 32; w += kSelectThreads) fbits[w] = 0u;
        __syncthreads();
    }
    for (int q = tid; q < m; q += kSelectThreads) {
        if (!((keep[q >> 6] >> (q & 63)) & 1ull)) continue;
        const int i = a.order[q];
        if (lds) atomicOr(&fbits[i >> 5], 1u << (i & 31));
        else a.flag[i] = 1;
    }
    if (tid == 0) base_sh = 0;
    __syncthreads();
    for (int t0 = 0; t0 < n; t0 += kSelectThreads) {
        const int i = t0 + tid;
        const bool f = i < n && (lds ? ((fbits[i >> 5] >> (i & 31)) & 1u) != 0u : a.flag[i] != 0);
        const unsigned long long bal = __ballot(f);
        const int in_wave = __popcll(bal & ((1ull << lane) - 1ull));
        if (lane == 0) wsum[wave] = __popcll(bal);
        __syncthreads();
        int before = base_sh;
        for (int v = 0; v < wave; ++v) before += wsum[v];
        if (f) {
            const float *src = a.rec + size_t(i) * kRecFloats;
            float *dst = a.out + size_t(before + in_wave) * kRecFloats;
#pragma unroll
            for (int e = 0; e < kRecFloats; ++e) dst[e] = src[e];
        }
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int v = 0; v < kSelectThreads / 64; ++v) tot += wsum[v];
            base_sh += tot;
        }
        __syncthreads();
    }
    if (tid == 0) *a.out_count = base_sh;
}

// The greedy walk over the ranking, 64 rows (one chunk) at a time, by one
// wavefront: the rows of chunk c removed by earlier chunks are the OR of
// the words (r, c) of the kept rows r listed for column chunk c; the rows
// of the chunk then resolve among themselves from their in-chunk
// suppressors (resolve_chunk_parallel).  The listed rows and their words
// are first copied into LDS by the whole block when they fit (the lists
// are short: suppression is local), else the walk reads them from global
// memory.  The kept records are then compacted in ascending record order.
constexpr int kSelCap = 5120;   // listed words held in LDS
constexpr int kSupLds = 4096;   // candidates whose in-chunk suppressors are held in LDS

__global__ __launch_bounds__(kSelectThreads) void k_nms_select(NmsArgs a) {
    __shared__ unsigned long long keep[kMaxWords];
    __shared__ unsigned long long eword[kSelCap];
    __shared__ unsigned short erow[kSelCap];
    __shared__ int coff[kMaxWords + 1];
    __shared__ unsigned long long supl[kSupLds];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = *a.count;
    const int m = n < a.max_candidates ? n : a.max_candidates;
    const int T = (m + 63) / 64;
    const int words = (a.max_candidates + 63) / 64;
    if (n > kFlagBits)
        for (int i = tid; i < n; i += kSelectThreads) a.flag[i] = 0;
    // exclusive prefix of the per-chunk list lengths: read in parallel, then
    // summed from LDS (one global load latency, not T)
    for (int c = tid; c < T; c += kSelectThreads) coff[c + 1] = a.colcount[c];
    __syncthreads();
    if (tid == 0) {
        int o = 0;
        for (int c = 0; c < T; ++c) {
            const int k = coff[c + 1];
            coff[c] = o;
            o += k;
        }
        coff[T] = o;
    }
    __syncthreads();
    const bool fits = coff[T] <= kSelCap;
    const bool sup_lds = m <= kSupLds;
    if (sup_lds)
        for (int q = tid; q < m; q += kSelectThreads) supl[q] = a.mask_t[q];
    if (fits) {
        for (int e = tid; e < coff[T]; e += kSelectThreads) {
            int lo = 0, hi = T - 1;  // the chunk c with coff[c] <= e < coff[c + 1]
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (coff[mid] <= e) lo = mid;
                else hi = mid - 1;
            }
            const int r = a.colrows[col_base(lo) + (e - coff[lo])];
            erow[e] = static_cast<unsigned short>(r);
            eword[e] = a.mask[size_t(r) * words + lo];
        }
    }
    __syncthreads();
    if (wave == 0) {
        // in-chunk suppressors from LDS, or prefetched a chunk ahead
        unsigned long long sup_next = !sup_lds && lane < m ? a.mask_t[lane] : 0ull;
        for (int c = 0; c < T; ++c) {
            const int row = c * 64 + lane, nxt = row + 64;
            unsigned long long sup;
            if (sup_lds) {
                sup = row < m ? supl[row] : 0ull;
            } else {
                sup = sup_next;
                sup_next = nxt < m ? a.mask_t[nxt] : 0ull;
            }
            unsigned long long rem = 0ull;
            for (int k = coff[c] + lane; k < coff[c + 1]; k += 64) {
                const int r = fits ? int(erow[k]) : a.colrows[col_base(c) + (k - coff[c])];
                const unsigned long long w = fits ? eword[k] : a.mask[size_t(r) * words + c];
                if ((keep[r >> 6] >> (r & 63)) & 1ull) rem |= w;
            }
            rem = wave_or64(rem);
            const int rows = m - c * 64 < 64 ? m - c * 64 : 64;
            const unsigned long long kb = resolve_chunk_parallel(rem, lane < rows ? sup : 0ull, rows);
            if (lane == 0) keep[c] = kb;
        }
    }
    __syncthreads();
    compact_kept(a, keep, m, n);
}

}  // namespace

hipError_t rotated_nms(const NmsArgs &a, int64_t max_records, hipStream_t s) {
    if (a.max_candidates < 1 || a.max_candidates > kNmsMaxCandidates || max_records < 1)
        return hipErrorInvalidValue;
    // grids are bounded by the worst case and loop over the work of the
    // actual count read on the device
    const unsigned blocks = unsigned((max_records + 255) / 256);
    const unsigned small = blocks < 64u ? blocks : 64u;
    k_nms_rank<<<blocks < 1024u ? blocks : 1024u, 256, 0, s>>>(a);
    k_nms_gather<<<small, 256, 0, s>>>(a);
    const unsigned chunks = unsigned((a.max_candidates + 63) / 64);
    const unsigned tiles = chunks * (chunks + 1u) / 2u;
    k_nms_mask<<<tiles < 2048u ? tiles : 2048u, 256, 0, s>>>(a);
    k_nms_select<<<1, kSelectThreads, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace kern
}  // namespace rtcc
