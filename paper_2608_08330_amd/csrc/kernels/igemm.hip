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
// Epilogue: + bias, ReLU, round to the stored dtype.
//
// Tiling: a 256-thread block (4 wavefronts of 64, 2 x 2) computes a BM x BN
// tile; every wavefront owns (BM/2) x (BN/2) made of 16 x 16 MFMA tiles.
// Per K step the block stages 64 bytes of every A row and every weight row
// in LDS (double buffered, rows padded to 80 bytes so the 16 lanes that
// read one 16-byte column hit 64 distinct banks).  One K step is one
// v_mfma_f32_16x16x32_bf16 per tile (bf16), or four v_mfma_f32_16x16x4_f32
// (fp32).  The weight fragment is the MFMA A operand, so each lane's four
// accumulators are four consecutive output channels of one pixel and the
// epilogue stores 8 (bf16) or 16 (fp32) contiguous bytes.  The K loop order
// is fixed, so results do not depend on M, the grid or the stream.
#include "kernels.hpp"

namespace rtcc {
namespace kern {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kRowPitch = 5;  // uint4 per LDS row: 64 data bytes + 16 pad

template <typename T>
struct Traits;
template <>
struct Traits<uint16_t> {
    static constexpr int EPV = 8;  // elements per 16-byte vector
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

template <typename T, int BM, int BN, bool DECONV>
__global__ __launch_bounds__(256) void k_igemm(GemmArgs a) {
    constexpr int EPV = Traits<T>::EPV;
    constexpr int BK = 4 * EPV;          // elements per row per K step (64 bytes)
    constexpr int AV = BM / 64;          // A vectors per thread per step
    constexpr int BV = BN / 64;          // B vectors per thread per step
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 16, FN = WN / 16;

    __shared__ uint4 As[2][BM * kRowPitch];
    __shared__ uint4 Bs[2][BN * kRowPitch];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;

    const int Ci = a.Ci;
    const int M = DECONV ? a.Hi * a.Wi : a.Ho * a.Wo;
    const int N = a.N;
    const int K = DECONV ? Ci : 9 * Ci;
    const int KT = K / BK;
    const int m0 = blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int phase = DECONV ? int(blockIdx.z) : 0;

    const T *in = static_cast<const T *>(a.in);
    const T *wt = static_cast<const T *>(a.wt) + (DECONV ? size_t(phase) * N * Ci : 0);

    // Per-thread A rows: pixel coordinates fixed for the whole K loop.
    int a_row[AV], a_kv[AV], a_iy[AV], a_ix[AV];
    bool a_ok[AV];
#pragma unroll
    for (int r = 0; r < AV; ++r) {
        const int v = tid + 256 * r;
        a_row[r] = v >> 2;
        a_kv[r] = v & 3;
        const int m = m0 + a_row[r];
        a_ok[r] = m < M;
        if (DECONV) {
            a_iy[r] = m;  // flat input pixel
            a_ix[r] = 0;
        } else {
            const int oy = m / a.Wo, ox = m - (m / a.Wo) * a.Wo;
            a_iy[r] = oy * a.stride - 1;
            a_ix[r] = ox * a.stride - 1;
        }
    }
    int b_row[BV], b_kv[BV];
    bool b_ok[BV];
#pragma unroll
    for (int r = 0; r < BV; ++r) {
        const int v = tid + 256 * r;
        b_row[r] = v >> 2;
        b_kv[r] = v & 3;
        b_ok[r] = n0 + b_row[r] < N;
    }

    uint4 ra[AV], rb[BV];
    auto load_global = [&](int kt) {
        const int k0 = kt * BK;
        int tap = 0, c0 = k0;
        if (!DECONV) {
            tap = k0 / Ci;
            c0 = k0 - tap * Ci;
        }
        const int dy = tap / 3, dx = tap - (tap / 3) * 3;
#pragma unroll
        for (int r = 0; r < AV; ++r) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (DECONV) {
                if (a_ok[r]) v = *reinterpret_cast<const uint4 *>(in + size_t(a_iy[r]) * Ci + c0 + a_kv[r] * EPV);
            } else {
                const int iy = a_iy[r] + dy, ix = a_ix[r] + dx;
                if (a_ok[r] && iy >= 0 && iy < a.Hi && ix >= 0 && ix < a.Wi)
                    v = *reinterpret_cast<const uint4 *>(in + (size_t(iy) * a.Wi + ix) * Ci + c0 + a_kv[r] * EPV);
            }
            ra[r] = v;
        }
#pragma unroll
        for (int r = 0; r < BV; ++r) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (b_ok[r]) v = *reinterpret_cast<const uint4 *>(wt + size_t(n0 + b_row[r]) * K + k0 + b_kv[r] * EPV);
            rb[r] = v;
        }
    };
    auto store_lds = [&](int buf) {
#pragma unroll
        for (int r = 0; r < AV; ++r) As[buf][a_row[r] * kRowPitch + a_kv[r]] = ra[r];
#pragma unroll
        for (int r = 0; r < BV; ++r) Bs[buf][b_row[r] * kRowPitch + b_kv[r]] = rb[r];
    };

    f32x4_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    load_global(0);
    store_lds(0);
    __syncthreads();

    const int fr = lane & 15, fk = lane >> 4;
    for (int kt = 0; kt < KT; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < KT) load_global(kt + 1);
        uint4 af[FM], bfr[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) af[i] = As[buf][(wm * WM + i * 16 + fr) * kRowPitch + fk];
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[j] = Bs[buf][(wn * WN + j * 16 + fr) * kRowPitch + fk];
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = Traits<T>::mma(bfr[j], af[i], acc[i][j]);
        if (kt + 1 < KT) store_lds(buf ^ 1);
        __syncthreads();
    }

    // Epilogue: lane holds channels n .. n+3 of pixel m for every tile.
    T *out = static_cast<T *>(a.out);
    const int py = DECONV ? phase / a.u : 0, px = DECONV ? phase - py * a.u : 0;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int m = m0 + wm * WM + i * 16 + fr;
        if (m >= M) continue;
        size_t pix;
        if (DECONV) {
            const int iy = m / a.Wi, ix = m - (m / a.Wi) * a.Wi;
            const int oy = iy * a.u + py, ox = ix * a.u + px;
            if (oy >= a.Ho || ox >= a.Wo) continue;
            pix = size_t(oy) * a.Wo + ox;
        } else {
            pix = size_t(m);
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * WN + j * 16 + fk * 4;
            if (n >= N) continue;
            const float v0 = fmaxf(acc[i][j][0] + a.bias[n + 0], 0.f);
            const float v1 = fmaxf(acc[i][j][1] + a.bias[n + 1], 0.f);
            const float v2 = fmaxf(acc[i][j][2] + a.bias[n + 2], 0.f);
            const float v3 = fmaxf(acc[i][j][3] + a.bias[n + 3], 0.f);
            Traits<T>::store4(out + pix * a.ldo + a.c_off + n, v0, v1, v2, v3);
        }
    }
}

template <typename T, bool DECONV>
hipError_t launch(const GemmArgs &a, hipStream_t s) {
    const int M = DECONV ? a.Hi * a.Wi : a.Ho * a.Wo;
    const unsigned gz = DECONV ? unsigned(a.u * a.u) : 1u;
    if (a.N % 128 == 0) {
        dim3 g((M + 127) / 128, a.N / 128, gz);
        k_igemm<T, 128, 128, DECONV><<<g, 256, 0, s>>>(a);
    } else {
        dim3 g((M + 127) / 128, (a.N + 63) / 64, gz);
        k_igemm<T, 128, 64, DECONV><<<g, 256, 0, s>>>(a);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t conv3x3(bool bf16, const GemmArgs &a, hipStream_t s) {
    return bf16 ? launch<uint16_t, false>(a, s) : launch<float, false>(a, s);
}

hipError_t deconv(bool bf16, const GemmArgs &a, hipStream_t s) {
    return bf16 ? launch<uint16_t, true>(a, s) : launch<float, true>(a, s);
}

}  // namespace kern
}  // namespace rtcc
