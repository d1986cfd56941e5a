// Implicit-GEMM 3x3 convolution and kernel=stride transposed convolution on
// gfx950 matrix cores.
//
// GEMM view, NHWC activations, K contiguous on both operands:
//   conv    M = Ho*Wo output pixels, N = C_out, K = 9 * C_in with
//           k = (dy * 3 + dx) * C_in + c; the A row of pixel (oy, ox) at k
//           reads in[oy*s + dy - 1][ox*s + dx - 1][c] (zero outside).
//   deconv  one GEMM per phase (py, px) of the u x u kernel: M = input
//           pixels, N = up channels, K = C_in; row (iy, ix) lands on output
//           pixel (iy*u + py, ix*u + px) of the concatenated slot, at a
//           channel offset, and is skipped outside the cropped grid.
// Epilogue: + bias, ReLU, round to the stored dtype; or, with split-K, a
// float32 partial tile per K slice that k_splitk_reduce sums in slice order.
//
// Pipeline (per block of WGM x WGN wavefronts, BM x BN tile):
//   * every K step stages 64 bytes of each of the BM activation rows and BN
//     weight rows in LDS, straight from global memory with
//     global_load_lds_dwordx4 (no register staging): one wave instruction
//     fills 1 KB = 16 rows, lane i writing bytes [16 i, 16 i + 16);
//   * STAGES LDS buffers form a ring; loads run STAGES - 1 steps ahead of
//     the MFMAs, and a step waits only for its own loads (vmcnt);
//   * 16-byte vectors of a row are XOR-swizzled by bits 1..2 of the row
//     index: ds_read_b128 serves 8 lanes (128 bytes, 32 banks) per cycle,
//     and any 8 consecutive rows then cover the 32 banks exactly once;
//   * padding and rows past M / N read a zero line in global memory;
//   * per step one v_mfma_f32_16x16x32_bf16 per 16 x 16 tile (bf16), or four
//     v_mfma_f32_16x16x4_f32 (fp32); the weight fragment is the MFMA A
//     operand, so each lane's four accumulators are four consecutive
//     output channels of one pixel.
// Blocks are ordered so that every XCD (block id mod 8) receives contiguous
// M tiles, which share halo rows in that XCD's L2.  The K loop order and the
// split-K reduction order are fixed: results do not depend on M, the grid or
// the stream.
#include "kernels.hpp"

#include <hip/hip_ext.h>

#include <type_traits>

namespace rtcc {
namespace kern {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kRowBytes = 64;  // bytes of one row per K step

// s_waitcnt immediate for gfx9: vmcnt = n, expcnt and lgkmcnt unconstrained.
template <int N>
struct VmWait {
    static constexpr int imm = (N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8);
};
// Before a barrier after which another wave may refill an LDS buffer that
// this wave read in the previous step: wait until this wave's LDS reads
// have returned.  The compiler places its own lgkmcnt waits just before the
// MFMAs that use the data and may sink those MFMAs (and the waits) below the
// barrier, leaving reads in flight while the refill lands.  Inline assembly
// with a memory clobber: no LDS access moves across it.
__device__ inline void lds_reads_done() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// s_waitcnt vmcnt(n) for n <= NMAX; n must fold to a constant after
// unrolling, so that the chain collapses to the one instruction.
template <int NMAX>
__device__ inline void vm_wait(int n) {
    if (n == NMAX) __builtin_amdgcn_s_waitcnt(VmWait<NMAX>::imm);
    else if constexpr (NMAX > 0) vm_wait<NMAX - 1>(n);
}

template <typename T>
struct Traits;
template <>
struct Traits<uint16_t> {
    static constexpr int EPV = 8;    // elements per 16-byte vector
    static constexpr int MFMAS = 1;  // MFMA instructions per mma()
    __device__ static inline f32x4_t mma(uint4 a, uint4 b, f32x4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                       __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
    }
    __device__ static inline void store4(uint16_t *p, float v0, float v1, float v2, float v3) {
        uint32_t u0 = __float_as_uint(v0), u1 = __float_as_uint(v1);
        uint32_t u2 = __float_as_uint(v2), u3 = __float_as_uint(v3);
        u0 += 0x7fffu + ((u0 >> 16) & 1u);
        u1 += 0x7fffu + ((u1 >> 16) & 1u);
        u2 += 0x7fffu + ((u2 >> 16) & 1u);
        u3 += 0x7fffu + ((u3 >> 16) & 1u);
        uint2 o;
        o.x = (u0 >> 16) | (u1 & 0xffff0000u);
        o.y = (u2 >> 16) | (u3 & 0xffff0000u);
        *reinterpret_cast<uint2 *>(p) = o;
    }
};
template <>
struct Traits<float> {
    static constexpr int EPV = 4;
    static constexpr int MFMAS = 4;
    __device__ static inline f32x4_t mma(uint4 a, uint4 b, f32x4_t c) {
        // lane group g holds k = 4g .. 4g+3 of both operands; the four
        // MFMAs sum k = e, 4 + e, 8 + e, 12 + e for e = 0..3
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
        return c;
    }
    __device__ static inline void store4(float *p, float v0, float v1, float v2, float v3) {
        *reinterpret_cast<float4 *>(p) = make_float4(v0, v1, v2, v3);
    }
};

// 16 bytes per lane from global memory into LDS at m0 + 16 * lane.  Issued
// as inline assembly so that the compiler does not treat the DMA as an
// unknown LDS write that every later LDS read must wait for; the kernel
// waits for these loads itself with s_waitcnt vmcnt (they retire in issue
// order, and all of them are drained before the epilogue).
__device__ inline void load_lds16(const void *g, uint32_t lds_addr) {
    // the address is wave-uniform (wave index and stage only)
    const uint32_t a = __builtin_amdgcn_readfirstlane(lds_addr);
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(a)
                 : "memory", "m0");
}

// Scheduling hint for the scheduler of the step that follows: NR LDS reads
// spread evenly between NM MFMAs (MFMAs first), so that neither the LDS
// queue nor the matrix pipe idles behind the other in issue order.
template <int NR, int NM, int I = 0>
__device__ inline void interleave_reads() {
    if constexpr (I < NR) {
        constexpr int q = (NM * (I + 1)) / NR - (NM * I) / NR;
        if constexpr (q > 0) __builtin_amdgcn_sched_group_barrier(0x008, q, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);                        // LDS read
        interleave_reads<NR, NM, I + 1>();
    }
}

// 16 bytes to global memory with the non-temporal hint: outputs are read
// by the next kernel, not by this one, and stream past the L2.
__device__ inline void store16_nt(void *p, uint4 v) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, static_cast<u32x4 *>(p));
}

// Epilogue through LDS.  Every lane first writes its ReLU(acc + bias)
// values (four consecutive channels of one pixel) into a [pixels][BN] tile
// in `stage` (rows padded by 16 bytes), then the block writes the tile out
// as whole 16-byte vectors of each pixel's BN-channel row: every pixel's
// row is one contiguous run of BN * elt bytes in global memory.  `pix(p)`
// gives the global element offset of tile pixel p's channel n0, or -1 to
// skip it.  Called by every thread of the block (it holds two barriers);
// `holds` is false for threads that hold no accumulators.
template <typename T, int NPIX, int BN, int NT, int FM, int FN, typename PixF, typename RowF, typename ChF>
__device__ inline void staged_store(unsigned char *stage, const f32x4_t (&acc)[FM][FN], bool holds, const float *bias,
                                    int n0, T *out, PixF pix, RowF row_of, ChF ch_of, int tid) {
    constexpr int RS = BN * int(sizeof(T)) + 16;
    __syncthreads();  // every wave is done with the LDS it staged operands in
    if (holds) {
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int p = row_of(i), ch = ch_of(j);
                const int n = n0 + ch;
                Traits<T>::store4(reinterpret_cast<T *>(stage + p * RS) + ch, fmaxf(acc[i][j][0] + bias[n + 0], 0.f),
                                  fmaxf(acc[i][j][1] + bias[n + 1], 0.f), fmaxf(acc[i][j][2] + bias[n + 2], 0.f),
                                  fmaxf(acc[i][j][3] + bias[n + 3], 0.f));
            }
        }
    }
    __syncthreads();
    constexpr int VPP = BN * int(sizeof(T)) / 16;  // 16-byte vectors per pixel row
    constexpr int NV = NPIX * VPP;
#pragma unroll
    for (int q = 0; q < (NV + NT - 1) / NT; ++q) {
        const int v = tid + q * NT;
        if (v >= NV) break;
        const int p = v / VPP, part = v - (v / VPP) * VPP;
        const int64_t off = pix(p);
        if (off < 0) continue;
        store16_nt(reinterpret_cast<uint4 *>(out + off) + part,
                   *reinterpret_cast<const uint4 *>(stage + p * RS + part * 16));
    }
}

// The arguments of map bt of a batched launch (see GemmArgs::batch).
__device__ inline GemmArgs batch_args(const GemmArgs &a0, int bt) {
    GemmArgs a = a0;
    if (a0.batch > 1) {
        a.in = a0.in_b[bt];
        a.out = a0.out_b[bt];
        a.ws = a0.ws_b[bt];
    }
    return a;
}
__device__ inline int batch_of(const GemmArgs &a0) { return a0.batch > 1 ? a0.batch : 1; }

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, bool DECONV>
__global__ __launch_bounds__(64 * WGM * WGN) void k_igemm(GemmArgs a0) {
    constexpr int NW = WGM * WGN;                    // wavefronts per block
    constexpr int EPV = Traits<T>::EPV;
    constexpr int BK = kRowBytes / int(sizeof(T));  // elements per row per K step
    constexpr int IA = BM / 16, IB = BN / 16;        // 1-KB load instructions per step
    static_assert((IA + IB) % NW == 0, "load instructions must split evenly over waves");
    constexpr int LPS = (IA + IB) / NW;              // loads per wave per step
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int FM = WM / 16, FN = WN / 16;
    static_assert(FM >= 1 && FN >= 1, "wave tile below one MFMA tile");
    constexpr int A_BYTES = BM * kRowBytes, B_BYTES = BN * kRowBytes;
    constexpr int STAGE_BYTES = A_BYTES + B_BYTES;

    __shared__ __attribute__((aligned(1024))) unsigned char smem[STAGES * STAGE_BYTES];
    const uint32_t lds_base = __builtin_amdgcn_readfirstlane(
        uint32_t(reinterpret_cast<uintptr_t>((lds_void *)smem)));

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WGM, wn = wave / WGM;

    // XCD-aware tile order: block ids are dealt to the 8 XCDs round-robin;
    // give each XCD a contiguous run of tiles.  Batched, map bt's blocks are
    // one contiguous run (with 8 maps, one XCD's).
    int bid = blockIdx.x;
    const int nbx = gridDim.x;
    if ((nbx & 7) == 0) bid = (bid & 7) * (nbx >> 3) + (bid >> 3);
    const int per_map = nbx / batch_of(a0);
    const int bt = bid / per_map;
    bid -= bt * per_map;
    const GemmArgs a = batch_args(a0, bt);
    // upsampling: the u x u output phases of one input tile are neighbours
    // (same XCD: the input tile is read from its L2, and the phases' writes
    // fill whole output rows together)
    int phase = 0;
    if (DECONV) {
        const int uu = a.u * a.u;
        phase = bid % uu;
        bid /= uu;
    }

    const int Ci = a.Ci;
    const int M = DECONV ? a.Hi * a.Wi : a.Ho * a.Wo;
    const int N = a.N;
    const int K = DECONV ? Ci : 9 * Ci;
    const int KT_all = K / BK;
    const int KT = KT_all / a.splits;

    const int mt = (M + BM - 1) / BM;
    const int nt = (N + BN - 1) / BN;
    const int m_tile = bid % mt;
    const int rest = bid / mt;  // n tile, then split
    const int n_tile = rest % nt;
    const int split = rest / nt;
    const int m0 = m_tile * BM;
    const int n0 = n_tile * BN;
    const int kt0 = split * KT;

    const T *in = static_cast<const T *>(a.in);
    const T *wt = static_cast<const T *>(a.wt) + (DECONV ? size_t(phase) * N * Ci : 0);
    const char *zero = static_cast<const char *>(a.zero);

    // Load instruction c of a step covers 16 rows: A rows 16 c .. (c < IA)
    // or B rows 16 (c - IA) ..; wave w issues c = w, w + NW, ...  Lane i
    // takes row + (i >> 2) and logical vector (i & 3) ^ ((row >> 1) & 3).
    int l_iy[LPS], l_ix[LPS], l_vec[LPS], l_row[LPS];
    bool l_ok[LPS], l_isa[LPS];
#pragma unroll
    for (int j = 0; j < LPS; ++j) {
        const int c = wave + j * NW;
        const bool isa = c < IA;
        const int row = 16 * (isa ? c : c - IA) + (lane >> 2);
        l_isa[j] = isa;
        l_row[j] = row;
        l_vec[j] = (lane & 3) ^ ((row >> 1) & 3);
        if (isa) {
            const int m = m0 + row;
            l_ok[j] = m < M;
            if (DECONV) {
                l_iy[j] = m;
                l_ix[j] = 0;
            } else {
                const int oy = m / a.Wo, ox = m - (m / a.Wo) * a.Wo;
                l_iy[j] = oy * a.stride - 1;
                l_ix[j] = ox * a.stride - 1;
            }
        } else {
            l_ok[j] = n0 + row < N;
            l_iy[j] = 0;
            l_ix[j] = 0;
        }
    }

    // 256-pixel conv tiles (one output row of a stride-2 layer each): every
    // other tile runs its K steps backwards, so that the input row two
    // neighbouring tiles share (the last tap row of one, the first of the
    // other) is read by both in the same steps, while it is in the L2
    const bool rev = !DECONV && BM == 256 && (m_tile & 1);
    auto issue = [&](int kt, int buf) {
        const int k0 = (kt0 + (rev ? KT - 1 - kt : kt)) * BK;
        int tap = 0, c0 = k0;
        if (!DECONV) {
            tap = k0 / Ci;
            c0 = k0 - tap * Ci;
        }
        const int dy = tap / 3, dx = tap - (tap / 3) * 3;
        const uint32_t st = lds_base + buf * STAGE_BYTES;
#pragma unroll
        for (int j = 0; j < LPS; ++j) {
            const int c = wave + j * NW;
            const void *g = zero;
            if (l_isa[j]) {
                if (DECONV) {
                    if (l_ok[j]) g = in + size_t(l_iy[j]) * Ci + c0 + l_vec[j] * EPV;
                } else {
                    const int iy = l_iy[j] + dy, ix = l_ix[j] + dx;
                    if (l_ok[j] && iy >= 0 && iy < a.Hi && ix >= 0 && ix < a.Wi)
                        g = in + (size_t(iy) * a.Wi + ix) * Ci + c0 + l_vec[j] * EPV;
                }
            } else if (l_ok[j]) {
                g = wt + size_t(n0 + l_row[j]) * K + k0 + l_vec[j] * EPV;
            }
            load_lds16(g, st + c * 1024);
        }
    };

    f32x4_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < KT) issue(s, s);

    // fragment addresses (bytes within a stage): row r, logical vector fk
    const int fr = lane & 15, fk = lane >> 4;
    int a_off[FM], b_off[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int r = wm * WM + i * 16 + fr;
        a_off[i] = r * kRowBytes + ((fk ^ ((r >> 1) & 3)) << 4);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int r = wn * WN + j * 16 + fr;
        b_off[j] = A_BYTES + r * kRowBytes + ((fk ^ ((r >> 1) & 3)) << 4);
    }

    for (int kt = 0; kt < KT; ++kt) {
        // Loads of steps kt+1 .. kt+STAGES-2 may stay in flight.
        if (kt + STAGES - 2 < KT) __builtin_amdgcn_s_waitcnt(VmWait<(STAGES - 2) * LPS>::imm);
        else __builtin_amdgcn_s_waitcnt(VmWait<0>::imm);
        lds_reads_done();  // step kt-1's buffer is refilled right after the barrier
        // No fence: only this step's loads are awaited above, later steps
        // stay in flight across the barrier.
        __builtin_amdgcn_s_barrier();  // step kt visible to all waves; step kt-1 consumed
        asm volatile("" ::: "memory");  // keep LDS reads below the barrier
        if (kt + STAGES - 1 < KT) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
        const unsigned char *st = smem + (kt % STAGES) * STAGE_BYTES;
        uint4 af[FM], bfr[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) af[i] = *reinterpret_cast<const uint4 *>(st + a_off[i]);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[j] = *reinterpret_cast<const uint4 *>(st + b_off[j]);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = Traits<T>::mma(bfr[j], af[i], acc[i][j]);
    }

    // Epilogue: lane holds channels n .. n+3 of pixel m for every tile.
    if (a.splits > 1) {
        float *ws = a.ws + size_t(split) * M * N;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int m = m0 + wm * WM + i * 16 + fr;
            if (m >= M) continue;
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int n = n0 + wn * WN + j * 16 + fk * 4;
                if (n >= N) continue;
                *reinterpret_cast<float4 *>(ws + size_t(m) * N + n) =
                    make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            }
        }
        return;
    }
    T *out = static_cast<T *>(a.out);
    const int py = DECONV ? phase / a.u : 0, px = DECONV ? phase - py * a.u : 0;
    // global element offset of tile row p (channel n0), -1 outside the output
    auto pix = [&](int p) -> int64_t {
        const int m = m0 + p;
        if (m >= M) return -1;
        size_t q;
        if (DECONV) {
            const int iy = m / a.Wi, ix = m - (m / a.Wi) * a.Wi;
            const int oy = iy * a.u + py, ox = ix * a.u + px;
            if (oy >= a.Ho || ox >= a.Wo) return -1;
            q = size_t(oy) * a.Wo + ox;
        } else {
            q = size_t(m);
        }
        return int64_t(q * a.ldo + a.c_off + n0);
    };
    constexpr int RS = BN * int(sizeof(T)) + 16;
    if constexpr (BM * RS <= STAGES * STAGE_BYTES) {
        if (n0 + BN <= N) {
            staged_store<T, BM, BN, 64 * NW, FM, FN>(
                smem, acc, true, a.bias, n0, out, pix, [&](int i) { return wm * WM + i * 16 + fr; },
                [&](int j) { return wn * WN + j * 16 + fk * 4; }, tid);
            return;
        }
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int64_t off = pix(wm * WM + i * 16 + fr);
        if (off < 0) continue;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int ch = wn * WN + j * 16 + fk * 4, n = n0 + ch;
            if (n >= N) continue;
            const float v0 = fmaxf(acc[i][j][0] + a.bias[n + 0], 0.f);
            const float v1 = fmaxf(acc[i][j][1] + a.bias[n + 1], 0.f);
            const float v2 = fmaxf(acc[i][j][2] + a.bias[n + 2], 0.f);
            const float v3 = fmaxf(acc[i][j][3] + a.bias[n + 3], 0.f);
            Traits<T>::store4(out + off + ch, v0, v1, v2, v3);
        }
    }
}

// Stride-1 3x3 convolution as a halo-tiled direct convolution.
//
// A block owns TH x 16 output pixels and BN output channels.  The K loop runs
// over input-channel chunks of 64 bytes; per chunk the block stages the
// (TH + 2) x 18 input patch (halo included, zero outside the grid) in LDS
// once, and the 9 taps then read their shifted 16-pixel rows from it, so an
// input element is fetched from L2 once per chunk instead of once per tap.
// Only the per-tap weight tile (BN rows x RB bytes) streams through an
// R-buffer ring, R - 1 taps ahead.  WGM x WGN wavefronts: WGM along output rows,
// WGN along channels; every wave holds (TH / WGM) x (BN / WGN / 16) MFMA tiles.
// With KG > 1 the block holds KG such groups of wavefronts over the same
// output tile: group g takes the channel chunks g, g + KG, ... with its own
// patch and weight buffers, and at the end groups 1 .. KG-1 hand their
// accumulators to group 0 through LDS, which adds them in group order
// (fixed, so the result does not depend on timing).  The tap
// loop is unrolled, so every s_waitcnt vmcnt bound is a constant:
// once step s's weights have landed, the loads still allowed in flight are
// the weights of the next R - 2 steps plus, at taps 1 .. R - 1, the next
// chunk's patch (issued at tap 0 after the weights of step s + R - 1).
template <typename T, int TH, int BN, int WGM, int WGN, int RB, int STRIDE, int KG, int R, bool ILV>
__global__ __launch_bounds__(64 * WGM * WGN * KG) void k_conv3s1(GemmArgs a0) {
    constexpr int NW = WGM * WGN;  // wavefronts per group
    constexpr int EPV = Traits<T>::EPV;
    constexpr int VPR = RB / 16;                 // 16-byte vectors per row and step
    constexpr int RPI = 1024 / RB;               // rows per 1-KB load instruction
    constexpr int KS = RB / 64;                  // MFMA k-substeps per step
    constexpr int BK = RB / int(sizeof(T));      // channels per step
    // input patch of a TH x TW output tile: (STRIDE (TH - 1) + 3) rows of
    // (STRIDE (TW - 1) + 3) pixels; with stride 2 the even patch columns
    // are stored first and the odd ones after them, so the 16 pixels a
    // fragment reads (columns 2 x + dx) are consecutive rows in LDS
    constexpr int TW = 16;
    constexpr int HW = STRIDE * (TW - 1) + 3, HH = STRIDE * (TH - 1) + 3;
    constexpr int EVEN = (HW + 1) / 2;
    constexpr int HALO = HH * HW;
    constexpr int IA = ((HALO + RPI - 1) / RPI + NW - 1) / NW * NW;  // patch loads, multiple of NW
    constexpr int LA = IA / NW;
    constexpr int IB = BN / RPI;
    static_assert(IB % NW == 0, "weight loads must split over the waves");
    constexpr int LB = IB / NW;
    constexpr int A_BYTES = IA * 1024, B_BYTES = BN * RB;
    constexpr int FM = TH / WGM, FN = BN / WGN / 16;
    static_assert(FM * WGM == TH && FN >= 1, "wave layout must tile the block");

    static_assert(R >= 3 && R <= 9, "weight ring depth");
    constexpr int G_BYTES = 2 * A_BYTES + R * B_BYTES;  // LDS of one group
    static_assert((KG - 1) * NW * 64 * FM * FN * 16 <= KG * G_BYTES, "group reduction must fit in LDS");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[KG * G_BYTES];

    // 16-byte vector v of row r sits at position v ^ swz(r); any 8
    // consecutive rows then cover the 32 banks once per ds_read_b128 cycle.
    auto swz = [](int r) { return VPR == 4 ? ((r >> 1) & 3) : (r & 7); };

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int grp = (tid >> 6) / NW;   // wave group: channel chunks grp, grp + KG, ...
    const int wave = (tid >> 6) % NW;  // wavefront within its group
    const int wm = wave % WGM, wn = wave / WGM;
    unsigned char *gsmem = smem + grp * G_BYTES;
    const uint32_t lds_base = __builtin_amdgcn_readfirstlane(
        uint32_t(reinterpret_cast<uintptr_t>((lds_void *)gsmem)));
    const uint32_t lds_b = lds_base + 2 * A_BYTES;

    int bid = blockIdx.x;
    const int nbx = gridDim.x;
    if ((nbx & 7) == 0) bid = (bid & 7) * (nbx >> 3) + (bid >> 3);
    // batched: map bt's blocks are one contiguous run (with 8 maps, one XCD's)
    const int per_map = nbx / batch_of(a0);
    const int bt = bid / per_map;
    bid -= bt * per_map;
    const GemmArgs a = batch_args(a0, bt);

    const int Ci = a.Ci, N = a.N, Ho = a.Ho, Wo = a.Wo;
    const int K = 9 * Ci;
    const int CH = (Ci / BK) / a.splits / KG;  // chunks of this split and group

    const int tx = (Wo + TW - 1) / TW, ty = (Ho + TH - 1) / TH;
    const int nt = N / BN;
    // channel tile fastest: the nt blocks that read the same input patch
    // are neighbours in the remapped order and so run on the same XCD,
    // where the patch is fetched from HBM once and then hits in L2
    const int n_tile = bid % nt;
    const int rest = bid / nt;
    const int sp_tile = rest % (tx * ty);
    const int split = rest / (tx * ty);
    const int oy0 = (sp_tile / tx) * TH, ox0 = (sp_tile % tx) * TW;
    const int n0 = n_tile * BN;
    const int c_begin = split * CH;

    const T *in = static_cast<const T *>(a.in);
    const T *wt = static_cast<const T *>(a.wt);
    const char *zero = static_cast<const char *>(a.zero);

    int p_off[LA], p_vec[LA];
    bool p_ok[LA];
#pragma unroll
    for (int j = 0; j < LA; ++j) {
        const int row = RPI * (wave + j * NW) + lane / VPR;
        p_vec[j] = (lane % VPR) ^ swz(row);
        const int hy = row / HW, lc = row - (row / HW) * HW;
        const int hx = STRIDE == 1 ? lc : (lc < EVEN ? 2 * lc : 2 * (lc - EVEN) + 1);
        const int iy = STRIDE * oy0 - 1 + hy, ix = STRIDE * ox0 - 1 + hx;
        p_ok[j] = row < HALO && iy >= 0 && iy < a.Hi && ix >= 0 && ix < a.Wi;
        p_off[j] = p_ok[j] ? (iy * a.Wi + ix) : 0;
    }
    int w_row[LB], w_vec[LB];
#pragma unroll
    for (int j = 0; j < LB; ++j) {
        const int row = RPI * (wave + j * NW) + lane / VPR;
        w_row[j] = row;
        w_vec[j] = (lane % VPR) ^ swz(row);
    }

    // local chunk i of this group is chunk c_begin + grp + KG i of the layer
    auto issue_patch = [&](int chunk) {
        const int c0 = (c_begin + grp + KG * chunk) * BK;
        const uint32_t dst = lds_base + (chunk & 1) * A_BYTES;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            const void *g = zero;
            if (p_ok[j]) g = in + size_t(p_off[j]) * Ci + c0 + p_vec[j] * EPV;
            load_lds16(g, dst + (wave + j * NW) * 1024);
        }
    };
    // step s = chunk * 9 + tap: weight columns k = tap * Ci + chunk channels
    auto issue_w = [&](int s) {
        const int chunk = s / 9, tap = s - (s / 9) * 9;
        const int k0 = tap * Ci + (c_begin + grp + KG * chunk) * BK;
        const uint32_t dst = lds_b + (s % R) * B_BYTES;
#pragma unroll
        for (int j = 0; j < LB; ++j)
            load_lds16(wt + size_t(n0 + w_row[j]) * K + k0 + w_vec[j] * EPV, dst + (wave + j * NW) * 1024);
    };

    f32x4_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int fr = lane & 15, fk = lane >> 4;
    int b_row[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) b_row[j] = wn * (BN / WGN) + j * 16 + fr;

    // MFMA operands of one step, read from LDS a step ahead of their use
    struct Frag {
        uint4 a[KS][FM], b[KS][FN];
    };
    // step (chunk c, tap t): patch buffer c & 1, weight buffer s % R
    auto read_frags = [&](Frag &f, int c, int t, int s) {
        const unsigned char *pa = gsmem + (c & 1) * A_BYTES;
        const unsigned char *pb = gsmem + 2 * A_BYTES + (s % R) * B_BYTES;
        const int dy = t / 3, dx = t % 3;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int v = fk + 4 * ks;
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int col = STRIDE == 1 ? dx + fr : ((dx & 1) ? EVEN : dx >> 1) + fr;
                const int r = (STRIDE * (wm * FM + i) + dy) * HW + col;
                f.a[ks][i] = *reinterpret_cast<const uint4 *>(pa + r * RB + ((v ^ swz(r)) << 4));
            }
#pragma unroll
            for (int j = 0; j < FN; ++j)
                f.b[ks][j] = *reinterpret_cast<const uint4 *>(pb + b_row[j] * RB + ((v ^ swz(b_row[j])) << 4));
        }
    };

    // Prologue: the first patch and the weights of steps 0 .. R-1; once the
    // patch and step 0's weights have landed, step 0's operands are read.
    const int S = CH * 9;
    issue_patch(0);
#pragma unroll
    for (int q = 0; q < R; ++q)
        if (q < S) issue_w(q);
    vm_wait<(R - 1) * LB>((S - 1 < R - 1 ? S - 1 : R - 1) * LB);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    Frag cur, nxt;
    read_frags(cur, 0, 0, 0);
    // Step s = 9 c + t (chunk c, tap t; LAST: c is the group's last chunk):
    // wait for step s + 1's operands to land, barrier, refill the weight
    // buffer of step s (whose operands every wave has read) with step
    // s + R, at tap 0 also the other patch buffer with chunk c + 1, read
    // step s + 1's operands and run step s's MFMAs on the operands read
    // during the previous step.
    auto step = [&](auto tc, auto lastc, int c) {
        constexpr int t = decltype(tc)::value;
        constexpr bool last = decltype(lastc)::value;
        constexpr bool more = !(last && t == 8);
        const int s = c * 9 + t;
        if constexpr (more) {
            // still in flight once step s + 1's weights (and at tap 8 the
            // next patch, issued before them) have landed: the weights of
            // steps s + 2 .. s + R - 1 (fewer near the end) and, at taps
            // 1 .. R - 2, the next chunk's patch
            if constexpr (!last) vm_wait<(R - 2) * LB + LA>((R - 2) * LB + (t >= 1 && t <= R - 2 ? LA : 0));
            else vm_wait<(R - 2) * LB>((7 - t < R - 2 ? 7 - t : R - 2) * LB);
            lds_reads_done();
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            if constexpr (!last || t + R < 9) issue_w(s + R);
            if constexpr (t == 0 && !last) issue_patch(c + 1);
            if constexpr (t < 8) read_frags(nxt, c, t + 1, s + 1);
            else read_frags(nxt, c + 1, 0, s + 1);
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = Traits<T>::mma(cur.b[ks][j], cur.a[ks][i], acc[i][j]);
        if constexpr (more && ILV) interleave_reads<KS * (FM + FN), KS * FM * FN * Traits<T>::MFMAS>();
        cur = nxt;
    };
    auto chunk = [&](auto lastc, int c) {
        step(std::integral_constant<int, 0>{}, lastc, c);
        step(std::integral_constant<int, 1>{}, lastc, c);
        step(std::integral_constant<int, 2>{}, lastc, c);
        step(std::integral_constant<int, 3>{}, lastc, c);
        step(std::integral_constant<int, 4>{}, lastc, c);
        step(std::integral_constant<int, 5>{}, lastc, c);
        step(std::integral_constant<int, 6>{}, lastc, c);
        step(std::integral_constant<int, 7>{}, lastc, c);
        step(std::integral_constant<int, 8>{}, lastc, c);
    };
    for (int c = 0; c + 1 < CH; ++c) chunk(std::false_type{}, c);
    chunk(std::true_type{}, CH - 1);

    if constexpr (KG > 1) {
        // every wave has read its last LDS operands and every DMA load has
        // landed (vmcnt(0) at the last step) before the buffers are reused
        __syncthreads();
        float *red = reinterpret_cast<float *>(smem);
        constexpr int E = FM * FN * 4;  // accumulators per lane
        if (grp > 0) {
            float *dst = red + ((grp - 1) * NW + wave) * 64 * E;
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) dst[((i * FN + j) * 4 + q) * 64 + lane] = acc[i][j][q];
        }
        __syncthreads();
        if (grp == 0) {
            for (int g = 1; g < KG; ++g) {
                const float *src = red + ((g - 1) * NW + wave) * 64 * E;
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q) acc[i][j][q] += src[((i * FN + j) * 4 + q) * 64 + lane];
            }
        }
    }

    // Group 0 holds the block's accumulators.
    constexpr int RS = BN * int(sizeof(T)) + 16;
    if constexpr (TH * TW * RS <= KG * G_BYTES) {
        if (a.splits == 1) {
            // the staging tile overwrites the reduction area: staged_store
            // starts with a barrier, after group 0 has read it
            staged_store<T, TH * TW, BN, 64 * NW * KG, FM, FN>(
                smem, acc, grp == 0, a.bias, n0, static_cast<T *>(a.out),
                [&](int p) -> int64_t {
                    const int oy = oy0 + p / TW, ox = ox0 + p % TW;
                    if (oy >= Ho || ox >= Wo) return -1;
                    return int64_t((size_t(oy) * Wo + ox) * a.ldo + a.c_off + n0);
                },
                [&](int i) { return (wm * FM + i) * TW + fr; },
                [&](int j) { return wn * (BN / WGN) + j * 16 + fk * 4; }, tid);
            return;
        }
    }
    if (grp > 0) return;
    const int ox = ox0 + fr;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int oy = oy0 + wm * FM + i;
        if (oy >= Ho || ox >= Wo) continue;
        const size_t m = size_t(oy) * Wo + ox;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * (BN / WGN) + j * 16 + fk * 4;
            if (a.splits > 1) {
                *reinterpret_cast<float4 *>(a.ws + (size_t(split) * Ho * Wo + m) * N + n) =
                    make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            } else {
                Traits<T>::store4(static_cast<T *>(a.out) + m * a.ldo + a.c_off + n,
                                  fmaxf(acc[i][j][0] + a.bias[n + 0], 0.f), fmaxf(acc[i][j][1] + a.bias[n + 1], 0.f),
                                  fmaxf(acc[i][j][2] + a.bias[n + 2], 0.f), fmaxf(acc[i][j][3] + a.bias[n + 3], 0.f));
            }
        }
    }
}

// out[m][n] = ReLU(bias[n] + sum over slices s = 0 .. S-1 of ws[s][m][n]),
// summed in slice order.  Four channels per thread.
template <typename T>
__global__ __launch_bounds__(256) void k_splitk_reduce(GemmArgs a0) {
    const GemmArgs a = batch_args(a0, blockIdx.y);
    const int M = a.Ho * a.Wo;
    const int N = a.N;
    const int64_t q = int64_t(blockIdx.x) * 256 + threadIdx.x;
    const int64_t total = int64_t(M) * (N / 4);
    if (q >= total) return;
    const int m = int(q / (N / 4));
    const int n = int(q - int64_t(m) * (N / 4)) * 4;
    float4 s = *reinterpret_cast<const float4 *>(a.ws + size_t(m) * N + n);
    for (int sp = 1; sp < a.splits; ++sp) {
        const float4 t = *reinterpret_cast<const float4 *>(a.ws + (size_t(sp) * M + m) * N + n);
        s.x += t.x;
        s.y += t.y;
        s.z += t.z;
        s.w += t.w;
    }
    Traits<T>::store4(static_cast<T *>(a.out) + size_t(m) * a.ldo + a.c_off + n,
                      fmaxf(s.x + a.bias[n], 0.f), fmaxf(s.y + a.bias[n + 1], 0.f),
                      fmaxf(s.z + a.bias[n + 2], 0.f), fmaxf(s.w + a.bias[n + 3], 0.f));
}

// Launch on stream s; with events, through hipExtLaunchKernelGGL so that they
// bracket the kernel's own execution.
template <typename F>
hipError_t launch_kernel(F kernel, dim3 grid, dim3 block, hipStream_t s, hipEvent_t e0, hipEvent_t e1,
                         const GemmArgs &a) {
    if (e0 || e1) hipExtLaunchKernelGGL(kernel, grid, block, 0, s, e0, e1, 0, a);
    else kernel<<<grid, block, 0, s>>>(a);
    return hipGetLastError();
}

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, bool DECONV>
hipError_t launch_cfg(const GemmArgs &a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr) {
    const int M = DECONV ? a.Hi * a.Wi : a.Ho * a.Wo;
    const unsigned phases = DECONV ? unsigned(a.u * a.u) : 1u;
    const unsigned nb = unsigned(a.batch > 1 ? a.batch : 1);
    const unsigned nx =
        unsigned((M + BM - 1) / BM) * unsigned((a.N + BN - 1) / BN) * unsigned(a.splits) * phases * nb;
    hipError_t e = launch_kernel(k_igemm<T, BM, BN, WGM, WGN, STAGES, DECONV>, dim3(nx),
                                 dim3(64 * WGM * WGN), s, e0, a.splits == 1 ? e1 : nullptr, a);
    if (e != hipSuccess || a.splits == 1) return e;
    const int64_t total = int64_t(M) * (a.N / 4);
    return launch_kernel(k_splitk_reduce<T>, dim3(unsigned((total + 255) / 256), nb), dim3(256), s, nullptr, e1, a);
}

template <typename T, int TH, int BN, int WGM, int WGN, int RB, int STRIDE, int KG, int R, bool ILV>
hipError_t launch_halo(const GemmArgs &a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr) {
    const unsigned nb = unsigned(a.batch > 1 ? a.batch : 1);
    const unsigned tiles = unsigned((a.Wo + 15) / 16) * unsigned((a.Ho + TH - 1) / TH);
    const unsigned nx = tiles * unsigned(a.N / BN) * unsigned(a.splits) * nb;
    hipError_t e = launch_kernel(k_conv3s1<T, TH, BN, WGM, WGN, RB, STRIDE, KG, R, ILV>, dim3(nx),
                                 dim3(64 * WGM * WGN * KG), s, e0, a.splits == 1 ? e1 : nullptr, a);
    if (e != hipSuccess || a.splits == 1) return e;
    const int64_t total = int64_t(a.Ho) * a.Wo * (a.N / 4);
    return launch_kernel(k_splitk_reduce<T>, dim3(unsigned((total + 255) / 256), nb), dim3(256), s, nullptr, e1, a);
}

template <typename T, bool DECONV>
hipError_t launch(const GemmArgs &a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr) {
    if (!DECONV) {
        // 128-byte K steps pay off from 256 input channels (bf16) on, where
        // one block holds a CU (kConvHalo8C64 keeps 64-byte steps)
        const bool rb128 = (a.Ci * int(sizeof(T))) % 128 == 0 && a.Ci * int(sizeof(T)) >= 512;
        // template arguments: TH, BN, WGM, WGN, RB, STRIDE, KG, weight ring
        // depth R, interleaved LDS reads; R and the interleaving as they
        // measured fastest at the c5 shapes
        switch (a.variant) {
            case kConvHalo8:
                return rb128 ? launch_halo<T, 8, 128, 4, 2, 128, 1, 1, 4, true>(a, s, e0, e1)
                             : launch_halo<T, 8, 128, 4, 2, 64, 1, 1, 4, false>(a, s, e0, e1);
            case kConvHalo8C64: return launch_halo<T, 8, 128, 4, 2, 64, 1, 1, 4, false>(a, s, e0, e1);
            case kConvHalo16:
                // with 128-byte chunks the interleaving hints spill registers
                // (256 VGPRs + 72 bytes): 6% slower than without
                return rb128 ? launch_halo<T, 16, 128, 4, 2, 128, 1, 1, 4, false>(a, s, e0, e1)
                             : launch_halo<T, 16, 128, 4, 2, 64, 1, 1, 4, true>(a, s, e0, e1);
            case kConvHalo16C64: return launch_halo<T, 16, 128, 4, 2, 64, 1, 1, 4, true>(a, s, e0, e1);
            case kConvHalo4:
                return rb128 ? launch_halo<T, 4, 128, 2, 2, 128, 1, 1, 3, true>(a, s, e0, e1)
                             : launch_halo<T, 4, 128, 2, 2, 64, 1, 1, 3, true>(a, s, e0, e1);
            case kConvHalo8S2: return launch_halo<T, 8, 128, 4, 2, 64, 2, 1, 4, true>(a, s, e0, e1);
            case kConvHalo4S2: return launch_halo<T, 4, 128, 4, 2, 64, 2, 1, 4, true>(a, s, e0, e1);
            case kConvHalo8S2N256: return launch_halo<T, 8, 256, 4, 2, 64, 2, 1, 4, true>(a, s, e0, e1);
            case kConvHalo4N64K2:
                return rb128 ? launch_halo<T, 4, 64, 2, 2, 128, 1, 2, 4, true>(a, s, e0, e1)
                             : launch_halo<T, 4, 64, 2, 2, 64, 1, 2, 3, true>(a, s, e0, e1);
            case kConvHalo4S2N64K2: return launch_halo<T, 4, 64, 2, 2, 64, 2, 2, 4, false>(a, s, e0, e1);
            default: break;
        }
    }
    if (!DECONV && a.variant == kConvImplicit256 && a.N % 128 == 0)
        return launch_cfg<T, 256, 128, 4, 2, 3, DECONV>(a, s, e0, e1);
    // the upsamplings' short K loops (4 or 8 steps) run as fast with a
    // 3-stage ring, whose 48 KB let more blocks share a CU
    if (a.N % 128 == 0)
        return DECONV ? launch_cfg<T, 128, 128, 4, 2, 3, DECONV>(a, s, e0, e1)
                      : launch_cfg<T, 128, 128, 4, 2, 4, DECONV>(a, s, e0, e1);
    return launch_cfg<T, 128, 64, 4, 1, 4, DECONV>(a, s, e0, e1);
}

}  // namespace

hipError_t conv3x3(bool bf16, const GemmArgs &a, hipStream_t s, hipEvent_t start, hipEvent_t stop) {
    return bf16 ? launch<uint16_t, false>(a, s, start, stop) : launch<float, false>(a, s, start, stop);
}

hipError_t deconv(bool bf16, const GemmArgs &a, hipStream_t s) {
    return bf16 ? launch<uint16_t, true>(a, s) : launch<float, true>(a, s);
}

}  // namespace kern
}  // namespace rtcc
