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
//                  IoU of candidates a and b exceeds the threshold; four
//                  lanes per (row a, 16 columns), storing a 16-bit part of
//                  the word.  IoU in float64: the intersection area is the
//                  shoelace sum over the edge pieces of each rectangle
//                  inside the other (Cyrus-Beck clipped, crossing points
//                  shared by the two pieces that meet there); pairs whose
//                  centres are farther apart than the sum of their
//                  circumradii are disjoint and skip the clipping.  A box
//                  with a non-finite parameter or w <= 0 or l <= 0 overlaps
//                  nothing.
//   k_nms_select   one block: the greedy walk over the ranking, 64 rows at a
//                  time: wave 0 resolves the rows of a chunk against each
//                  other with the chunk's diagonal mask words (scalar loop;
//                  the words were prefetched during the previous chunk),
//                  then every thread takes (kept row, later word) pairs and
//                  ORs the mask word into the LDS removed set (one load per
//                  pair, all in flight together).  The kept records are then
//                  compacted in ascending record (anchor) order.
// Everything is integer or float64 except the scores, which are compared as
// stored: the decisions do not depend on the grid or the timing.
#include "kernels.hpp"

#include <cmath>

namespace rtcc {
namespace kern {

namespace {

constexpr int kRecFloats = 9;
constexpr int kFoot = kNmsFootDoubles;  // x, y, w, l, cos, sin, valid, circumradius

// Ranking key of record i: the score's bit pattern above the complement of
// i.  Scores are sigmoids (>= +0), whose bit patterns order like the
// values, so key_j > key_i iff record j precedes record i (higher score, or
// equal score and lower index).
__device__ inline unsigned long long rank_key(const NmsArgs &a, int i) {
    const uint32_t bits = __float_as_uint(a.rec[size_t(i) * kRecFloats + 7]);
    return (static_cast<unsigned long long>(bits) << 32) | (0xffffffffu - uint32_t(i));
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

__device__ __forceinline__ void mask_piece(const NmsArgs &a, int m, int rb, int cb, int piece, double *cf) {
    const int c0 = cb * 64 + piece * 16;
    if (c0 >= m) return;  // uniform over the block
    for (int q = threadIdx.x; q < 16 * kFoot; q += 256) {
        const int b = c0 + q / kFoot;
        cf[q] = b < m ? a.foot[size_t(c0) * kFoot + q] : 0.0;
    }
    __syncthreads();
    const int row = rb * 64 + int(threadIdx.x >> 2);
    const int sub = threadIdx.x & 3;  // columns c0 + 4 sub .. c0 + 4 sub + 3
    unsigned bits = 0u;
    if (row < m) {
        const double *fa = a.foot + size_t(row) * kFoot;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int q = 4 * sub + k, col = c0 + q;
            if (col >= m || col <= row) continue;
            if (suppresses(fa, cf + q * kFoot, a.iou_threshold)) bits |= 1u << q;
        }
    }
    if (cb == rb) {
        // diagonal block: also the transposed words, column q of this piece
        // <- the rows of the chunk that suppress it
        __shared__ unsigned long long tq[16];
        if (threadIdx.x < 16) tq[threadIdx.x] = 0ull;
        __syncthreads();
        if (bits) {
            unsigned rest = bits;
            while (rest) {
                const int q = __builtin_ctz(rest);
                rest &= rest - 1u;
                atomicOr(&tq[q], 1ull << (row & 63));
            }
        }
        __syncthreads();
        if (threadIdx.x < 16 && c0 + int(threadIdx.x) < m) a.mask_t[c0 + threadIdx.x] = tq[threadIdx.x];
    }
    bits |= __shfl_xor(bits, 1, 64);
    bits |= __shfl_xor(bits, 2, 64);
    if (row < m && sub == 0) {
        const int words = (a.max_candidates + 63) / 64;
        reinterpret_cast<unsigned short *>(a.mask + size_t(row) * words + cb)[piece] =
            static_cast<unsigned short>(bits);
    }
}

__global__ __launch_bounds__(256) void k_nms_mask(NmsArgs a) {
    const int n = *a.count;
    const int m = n < a.max_candidates ? n : a.max_candidates;
    const int T = (m + 63) / 64;
    const int items = 4 * (T * (T + 1) / 2);
    __shared__ double cf[16 * kFoot];
    for (int item = blockIdx.x; item < items; item += gridDim.x) {
        // item -> (row chunk rb, column chunk cb >= rb, 16-column piece)
        int tri = item >> 2, rb = 0;
        while (tri >= T - rb) {
            tri -= T - rb;
            ++rb;
        }
        mask_piece(a, m, rb, rb + tri, item & 3, cf);
        __syncthreads();
    }
}

__device__ inline unsigned long long uniform64(unsigned long long v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(v >> 32));
    return (static_cast<unsigned long long>(hi) << 32) | lo;
}

// Greedy resolution of one chunk of 64 ranked rows (one wavefront): `rem`
// are the rows already removed by earlier chunks, lane r holds the
// diagonal word of row r (bits of later rows of the chunk it suppresses).
// Visits only the rows still standing, in rank order; all loop state is
// wave-uniform (scalar registers).  Returns the kept rows.
__device__ inline unsigned long long resolve_chunk(unsigned long long rem, unsigned long long diag, int rows);

__device__ inline unsigned long long readlane64(unsigned long long v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane(uint32_t(v), lane);
    const uint32_t hi = __builtin_amdgcn_readlane(uint32_t(v >> 32), lane);
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

__device__ inline unsigned long long resolve_chunk(unsigned long long rem, unsigned long long diag, int rows) {
    const unsigned long long rowmask = rows >= 64 ? ~0ull : (1ull << rows) - 1ull;
    rem = uniform64(rem);
    unsigned long long kb = 0ull, done = 0ull;
    for (;;) {
        const unsigned long long avail = ~rem & rowmask & ~done;
        if (!avail) break;
        const int r = __builtin_ctzll(avail);
        kb |= 1ull << r;
        rem |= readlane64(diag, r);
        done = r == 63 ? ~0ull : (2ull << r) - 1ull;
    }
    return kb;
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

__global__ __launch_bounds__(kSelectThreads) void k_nms_select(NmsArgs a) {
    __shared__ unsigned long long removed[kMaxWords];
    __shared__ unsigned long long keep[kMaxWords];
    __shared__ int klist[64];
    __shared__ int kcnt;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = *a.count;
    const int m = n < a.max_candidates ? n : a.max_candidates;
    const int nw = (m + 63) / 64;
    const int words = (a.max_candidates + 63) / 64;
    for (int w = tid; w < nw; w += kSelectThreads) removed[w] = 0ull;
    if (n > kFlagBits)
        for (int i = tid; i < n; i += kSelectThreads) a.flag[i] = 0;
    unsigned long long diag_next = 0ull;
    if (wave == 0 && lane < m) diag_next = a.mask[size_t(lane) * words];
    __syncthreads();

    for (int c = 0; c < nw; ++c) {
        if (wave == 0) {
            const unsigned long long diag = diag_next;
            const unsigned long long kb = resolve_chunk(removed[c], diag, m - c * 64);
            if ((kb >> lane) & 1ull) klist[__popcll(kb & ((1ull << lane) - 1ull))] = lane;
            if (lane == 0) {
                keep[c] = kb;
                kcnt = __popcll(kb);
            }
        }
        __syncthreads();
        // (kept row, later word) pairs: every load of this chunk in flight at once
        const int kc = kcnt;
        const int total = kc * (nw - c - 1);
        for (int q = tid; q < total; q += kSelectThreads) {
            const int r = klist[q % kc], w = c + 1 + q / kc;
            const unsigned long long v = a.mask[size_t(c * 64 + r) * words + w];
            if (v) atomicOr(&removed[w], v);
        }
        if (wave == 0 && c + 1 < nw) {
            const int row = (c + 1) * 64 + lane;
            diag_next = row < m ? a.mask[size_t(row) * words + c + 1] : 0ull;
        }
        __syncthreads();
    }

    compact_kept(a, keep, m, n);
}


// Pull form of the greedy walk for max_candidates <= kPullMax: the removed
// bits of chunk c are the OR, over the kept rows of the earlier chunks, of
// their word c (column c of the mask).  Columns are read two chunks ahead
// (registers, then LDS), so the walk itself only touches LDS.
constexpr int kPullMax = 4096;

__global__ __launch_bounds__(kSelectThreads) void k_nms_select_pull(NmsArgs a) {
    __shared__ unsigned long long col[2][kPullMax];
    __shared__ unsigned long long keep[kPullMax / 64];
    __shared__ unsigned long long part[kSelectThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = *a.count;
    const int m = n < a.max_candidates ? n : a.max_candidates;
    const int nw = (m + 63) / 64;
    const int words = (a.max_candidates + 63) / 64;
    constexpr int PER = kPullMax / kSelectThreads;
    // column w of the rows that have a word there: rows < min(64 (w + 1), m)
    auto load_col = [&](int w, unsigned long long *dst) {
        const int rows = (w + 1) * 64 < m ? (w + 1) * 64 : m;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int r = tid + k * kSelectThreads;
            dst[k] = (w < nw && r < rows) ? a.mask[size_t(r) * words + w] : 0ull;
        }
    };
    if (n > kFlagBits)
        for (int i = tid; i < n; i += kSelectThreads) a.flag[i] = 0;
    for (int r = tid; r < 64 && r < m; r += kSelectThreads) col[0][r] = a.mask[size_t(r) * words];
    // two columns ahead in registers: column c + 1 was issued during chunk
    // c - 1 and lands in LDS at the end of chunk c
    unsigned long long pre1[PER], pre2[PER];
    load_col(1, pre1);
    // wave 0 lane r: the in-chunk suppressors of row r of the current chunk
    // (read one chunk ahead)
    unsigned long long sup_cur = (wave == 0 && lane < m) ? a.mask_t[lane] : 0ull;
    __syncthreads();
    for (int c = 0; c < nw; ++c) {
        const int buf = c & 1;
        load_col(c + 2, pre2);
        const int next_row = (c + 1) * 64 + lane;
        const unsigned long long sup_next = (wave == 0 && next_row < m) ? a.mask_t[next_row] : 0ull;
        const int rows_next = (c + 2) * 64 < m ? (c + 2) * 64 : m;
        // removed bits of chunk c: word c of every kept row before the chunk
        unsigned long long acc = 0ull;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int r = tid + k * kSelectThreads;
            if (r < c * 64 && ((keep[r >> 6] >> (r & 63)) & 1ull)) acc |= col[buf][r];
        }
        acc = wave_or64(acc);
        if (lane == 0) part[wave] = acc;
        __syncthreads();
        if (wave == 0) {
            const int rows = m - c * 64 < 64 ? m - c * 64 : 64;
            unsigned long long rem = lane < kSelectThreads / 64 ? part[lane] : 0ull;
            rem = wave_or64(rem);
            const unsigned long long sup = lane < rows ? sup_cur : 0ull;
            const unsigned long long kb = resolve_chunk_parallel(rem, sup, rows);
            if (lane == 0) keep[c] = kb;
        }
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int r = tid + k * kSelectThreads;
            if (r < rows_next) col[buf ^ 1][r] = pre1[k];
            pre1[k] = pre2[k];
        }
        sup_cur = sup_next;
        __syncthreads();
    }
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
    const unsigned items = 4u * chunks * (chunks + 1u) / 2u;
    k_nms_mask<<<items < 2048u ? items : 2048u, 256, 0, s>>>(a);
    if (a.max_candidates <= kPullMax) k_nms_select_pull<<<1, kSelectThreads, 0, s>>>(a);
    else k_nms_select<<<1, kSelectThreads, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace kern
}  // namespace rtcc
