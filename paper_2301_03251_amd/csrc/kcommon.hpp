// kcommon.hpp -- device helpers shared by the kernel sources (tile.hip,
// kernels.hip): complex types, wavefront reductions by DPP and readlane,
// angle sources of rotation and Pauli-channel slots, and the per-sample op
// record of the tile ops.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>

#include "launch.hpp"

namespace qlayer {
namespace {

template <typename Real> struct Cx;
template <> struct Cx<float> { using T = float2; };
template <> struct Cx<double> { using T = double2; };

template <typename T2, typename Real>
__device__ __forceinline__ T2 mk(Real x, Real y) {
    T2 r;
    r.x = x;
    r.y = y;
    return r;
}

// Sum over the 64 lanes of a wavefront (every lane gets the total). The
// butterfly order is fixed, so the result is reproducible.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// DPP lane moves (gfx9 encodings): quad_perm [1,0,3,2], quad_perm [2,3,0,1],
// row_half_mirror, row_mirror. Each is a VALU operand modifier, so a row-local
// butterfly costs one instruction per step instead of an LDS-pipe permute.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const long long u = __builtin_bit_cast(long long, v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(u & 0xffffffff), CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(u >> 32), CTRL, 0xF, 0xF, false);
    return __builtin_bit_cast(double, ((long long)hi << 32) | (unsigned int)lo);
}

// Wavefront sum: butterfly inside each 16-lane row (4 DPP adds), then the four
// row sums combined from readlanes. Returns the (uniform) total in fp64; the
// adds run in Real, which for fp32 is a 64-term sum of per-thread partials.
__device__ __forceinline__ double wave_total(float v) {
    v += dpp_f32<0xB1>(v);
    v += dpp_f32<0x4E>(v);
    v += dpp_f32<0x141>(v);
    v += dpp_f32<0x140>(v);
    const float a = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
    const float b = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
    const float c = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
    const float d = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
    return ((double)a + (double)b) + ((double)c + (double)d);
}
__device__ __forceinline__ double wave_total(double v) {
    v += dpp_f64<0xB1>(v);
    v += dpp_f64<0x4E>(v);
    v += dpp_f64<0x141>(v);
    v += dpp_f64<0x140>(v);
    auto lane = [&](int l) {
        const long long u = __builtin_bit_cast(long long, v);
        const int lo = __builtin_amdgcn_readlane((int)(u & 0xffffffff), l);
        const int hi = __builtin_amdgcn_readlane((int)(u >> 32), l);
        return __builtin_bit_cast(double, ((long long)hi << 32) | (unsigned int)lo);
    };
    return (lane(0) + lane(16)) + (lane(32) + lane(48));
}

// Complex products of float2 / double2.
template <typename T2>
__device__ __forceinline__ T2 cxmul(T2 a, T2 b) {
    T2 r;
    r.x = a.x * b.x - a.y * b.y;
    r.y = a.x * b.y + a.y * b.x;
    return r;
}
// conj(a) * b
template <typename T2>
__device__ __forceinline__ T2 cxmulc(T2 a, T2 b) {
    T2 r;
    r.x = a.x * b.x + a.y * b.y;
    r.y = a.x * b.y - a.y * b.x;
    return r;
}
template <typename T2, typename Real>
__device__ __forceinline__ T2 to_real(double2 v) {
    return mk<T2>((Real)v.x, (Real)v.y);
}

// Leave-one-out contractions of a thread's registers with per-bit factors:
// for every register bit m, S[m][u] = sum over registers i with bit m = u of
// conj(prod_{m' != m} f_{m'}(bit m' of i)) v[i]. The bits [LO, HI) of v's
// index are split in halves: contracting the upper half away gives a tensor
// over the lower half (and the other way round), and each half recurses, so
// every partial contraction is shared by the bits that need it.
template <int LO, int HI, typename T2>
__device__ __forceinline__ void loo_contract(const T2* v, const T2* f0, const T2* f1, T2 (*S)[2]) {
    if constexpr (HI - LO == 1) {
        S[LO][0] = v[0];
        S[LO][1] = v[1];
    } else {
        constexpr int MID = (LO + HI) / 2;
        constexpr int H0 = 1 << (HI - LO - 1);
        {
            // contract bits HI-1 .. MID (highest first): a tensor over LO..MID-1
            T2 w[H0];
#pragma unroll
            for (int i = 0; i < H0; ++i) {
                const T2 x = cxmulc(f0[HI - 1], v[i]), y = cxmulc(f1[HI - 1], v[i + H0]);
                w[i].x = x.x + y.x;
                w[i].y = x.y + y.y;
            }
#pragma unroll
            for (int m = HI - 2; m >= MID; --m) {
#pragma unroll
                for (int i = 0; i < H0; ++i)
                    if (i < (1 << (m - LO))) {
                        const T2 x = cxmulc(f0[m], w[i]), y = cxmulc(f1[m], w[i + (1 << (m - LO))]);
                        w[i].x = x.x + y.x;
                        w[i].y = x.y + y.y;
                    }
            }
            loo_contract<LO, MID, T2>(w, f0, f1, S);
        }
        {
            // contract bits LO .. MID-1 (lowest first): a tensor over MID..HI-1
            T2 w[H0];
#pragma unroll
            for (int i = 0; i < H0; ++i) {
                const T2 x = cxmulc(f0[LO], v[2 * i]), y = cxmulc(f1[LO], v[2 * i + 1]);
                w[i].x = x.x + y.x;
                w[i].y = x.y + y.y;
            }
#pragma unroll
            for (int m = LO + 1; m < MID; ++m) {
#pragma unroll
                for (int i = 0; i < H0; ++i)
                    if (i < (1 << (HI - m - 1))) {
                        const T2 x = cxmulc(f0[m], w[2 * i]), y = cxmulc(f1[m], w[2 * i + 1]);
                        w[i].x = x.x + y.x;
                        w[i].y = x.y + y.y;
                    }
            }
            loo_contract<MID, HI, T2>(w, f0, f1, S);
        }
    }
}

// ---------------------------------------------------------------------------
// angle sources (shared by the binding kernels)

// The angle (fp64) of a rotation slot for circuit b: scale * the bound input
// or weight (scale 1, or +-1/2 for the halves of a controlled rotation). In a
// parameter-shift chunk (vper > 0) circuit b is virtual circuit v = v0 + b of
// sample v / vper.
template <typename Real>
__device__ __forceinline__ double angle_of(const void* inputs, const void* weights, int F, const SlotSrc& src,
                                           int64_t b, int64_t v0, int32_t vper, int64_t& bs) {
    bs = vper > 0 ? (v0 + b) / vper : b;
    if (src.src == S_WEIGHT) return src.scale * (double)((const Real*)weights)[src.index];
    return src.scale * (double)((const Real*)inputs)[bs * F + src.index];
}

// The Pauli a channel slot applies in circuit b: 1 X, 2 Y, 3 Z, 0 none, from
// fp64 comparisons of the trajectory uniform with the cumulative
// probabilities formed on the host.
template <typename Real>
__device__ __forceinline__ int pauli_of(const void* inputs, int F, const SlotSrc& src, int64_t b, int64_t v0,
                                        int32_t vper) {
    const int64_t bs = vper > 0 ? (v0 + b) / vper : b;
    const double u = (double)((const Real*)inputs)[bs * F + src.index];
    return u < src.c1 ? 1 : u < src.c2 ? 2 : u < src.c3 ? 3 : 0;
}

// Parameter-shift offset of slot s in circuit b: v % vper = 2s+1 adds pi/2,
// 2s+2 subtracts it (the two-term rule of exp(-i t P / 2) gates).
__device__ __forceinline__ double shift_of(int64_t b, int64_t v0, int32_t vper, int s) {
    if (vper <= 0) return 0.0;
    const int64_t v = v0 + b;
    const int j = (int)(v - (v / vper) * vper);
    const double half_pi = 1.570796326794896619231;
    if (j == 2 * s + 1) return half_pi;
    if (j == 2 * s + 2) return -half_pi;
    return 0.0;
}


template <typename Real> struct XOp;
template <> struct XOp<float> {
    uint32_t h, arg;
    float a, b;
};
template <> struct XOp<double> {
    uint32_t h, arg;
    double a, b;
    uint64_t pad;
};

// DPP row broadcast (row_bcast:15 into rows 1 and 3, row_bcast:31 into rows 2
// and 3); lanes of the other rows read 0.
template <int CTRL, int ROWS>
__device__ __forceinline__ float bcast_f32(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                 ROWS, 0xF, false));
}
template <int CTRL, int ROWS>
__device__ __forceinline__ double bcast_f64(double v) {
    const long long u = __builtin_bit_cast(long long, v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(u & 0xffffffff), CTRL, ROWS, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(u >> 32), CTRL, ROWS, 0xF, false);
    return __builtin_bit_cast(double, ((long long)hi << 32) | (unsigned int)lo);
}

// Wavefront sum left in lane 63 (other lanes hold partial sums): the row
// butterfly, then rows 0+1 and 2+3, then all four. Fixed order.
__device__ __forceinline__ float wave_to_last(float v) {
    v += dpp_f32<0xB1>(v);
    v += dpp_f32<0x4E>(v);
    v += dpp_f32<0x141>(v);
    v += dpp_f32<0x140>(v);
    v += bcast_f32<0x142, 0xA>(v);
    v += bcast_f32<0x143, 0xC>(v);
    return v;
}
__device__ __forceinline__ double wave_to_last(double v) {
    v += dpp_f64<0xB1>(v);
    v += dpp_f64<0x4E>(v);
    v += dpp_f64<0x141>(v);
    v += dpp_f64<0x140>(v);
    v += bcast_f64<0x142, 0xA>(v);
    v += bcast_f64<0x143, 0xC>(v);
    return v;
}

// Sum over each 16-lane row, left in every lane of the row (the first four
// steps of wave_to_last).
__device__ __forceinline__ float row_sum(float v) {
    v += dpp_f32<0xB1>(v);
    v += dpp_f32<0x4E>(v);
    v += dpp_f32<0x141>(v);
    v += dpp_f32<0x140>(v);
    return v;
}
__device__ __forceinline__ double row_sum(double v) {
    v += dpp_f64<0xB1>(v);
    v += dpp_f64<0x4E>(v);
    v += dpp_f64<0x141>(v);
    v += dpp_f64<0x140>(v);
    return v;
}


}  // namespace
}  // namespace qlayer
