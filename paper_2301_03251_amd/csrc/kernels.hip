// kernels.hip -- HIP kernels of the batched quantum layer, written for gfx950.
//
// State vectors are sample-major: psi[b][j], j = amplitude index, qubit q is
// bit q of j. Complex numbers are interleaved (re, im): float2 for complex64,
// double2 for complex128. Gates follow exp(-i t P / 2) for RX/RY/RZ.
//
// Kernels:
//   k_bind   -- angle -> (cos(t/2), sin(t/2)) per (sample, rotation slot), in fp64
//   k_whole  -- small states: one workgroup per sample keeps psi and lambda in
//               LDS and runs the forward pass, <Z_q>, the lambda seed and the
//               adjoint sweep in one launch (no HBM state traffic)
//   k_tile   -- one tile pass over every sample: each workgroup streams 2^k
//               amplitudes (a tile) from HBM into registers, applies the pass's
//               gates there (LDS only to change which tile bits sit in
//               registers), and streams them back; the backward variant carries
//               psi and lambda and accumulates Im<lambda|P|psi> per rotation
//   k_reduce -- deterministic fp64 sums of the per-workgroup partials into
//               <Z_q>, input gradients and (batch-summed) weight gradients
//   k_wave   -- states of n <= 8 qubits: one wavefront per sample holds psi and
//               lambda in registers (same job as k_whole, no LDS, no barriers)
//   k_bind_tile -- per-sample op records of the tile ops (handler, argument,
//               shear coefficients; the Pauli of a channel trajectory)
//   k_embed_* -- basis / amplitude embedding of the initial state, and the
//               amplitude embedding's VJP from lambda_0
//   k_shift_dot, k_shift_grad -- parameter-shift VJP from batched shifted circuits
//   k_state_phase, k_phase_fix -- the global phase of the tile path's final states
//   k_block_sums, k_block_scan, k_shots, k_shot_z -- shot sampling by inverse CDF
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

// ---------------------------------------------------------------------------
// k_bind

template <typename Real>
__global__ void k_bind(const BindArgs a) {
    using T2 = typename Cx<Real>::T;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= a.B * a.n_slots) return;
    const int64_t b = t / a.n_slots;
    const int s = (int)(t - b * a.n_slots);
    const SlotSrc src = a.slots[s];
    if (src.src == S_PAULI) {
        ((T2*)a.coef)[t] = mk<T2>((Real)pauli_of<Real>(a.inputs, a.F, src, b, a.v0, a.vper), (Real)0);
        return;
    }
    int64_t bs = b;
    const double th = angle_of<Real>(a.inputs, a.weights, a.F, src, b, a.v0, a.vper, bs) +
                      shift_of(b, a.v0, a.vper, s);
    double sn, cs;
    sincos(0.5 * th, &sn, &cs);
    ((T2*)a.coef)[t] = mk<T2>((Real)cs, (Real)sn);
}

// ---------------------------------------------------------------------------
// k_whole: the whole state of one sample in LDS

// Insert a zero bit at position q of p.
__device__ __forceinline__ int insert0(int p, int q) {
    return ((p >> q) << (q + 1)) | (p & ((1 << q) - 1));
}

template <typename T2, typename Real>
__device__ __forceinline__ void lds_gate(T2* st, const DevGate g, Real c, Real s, int n, int tid,
                                         int nt) {
    const int dim = 1 << n, half = dim >> 1;
    switch (g.kind) {
        case K_H:
        case K_RX:
        case K_RY: {
            const int M = 1 << g.q0;
            const Real r = (Real)0.70710678118654752440;
            for (int p = tid; p < half; p += nt) {
                const int i = insert0(p, g.q0);
                const T2 u = st[i], v = st[i | M];
                if (g.kind == K_H) {
                    st[i] = mk<T2>((u.x + v.x) * r, (u.y + v.y) * r);
                    st[i | M] = mk<T2>((u.x - v.x) * r, (u.y - v.y) * r);
                } else if (g.kind == K_RX) {
                    st[i] = mk<T2>(c * u.x + s * v.y, c * u.y - s * v.x);
                    st[i | M] = mk<T2>(c * v.x + s * u.y, c * v.y - s * u.x);
                } else {
                    st[i] = mk<T2>(c * u.x - s * v.x, c * u.y - s * v.y);
                    st[i | M] = mk<T2>(s * u.x + c * v.x, s * u.y + c * v.y);
                }
            }
        } break;
        case K_RZ:
            for (int i = tid; i < dim; i += nt) {
                const T2 u = st[i];
                if (i >> g.q0 & 1) st[i] = mk<T2>(c * u.x - s * u.y, c * u.y + s * u.x);
                else st[i] = mk<T2>(c * u.x + s * u.y, c * u.y - s * u.x);
            }
            break;
        case K_CNOT: {
            const int M = 1 << g.q1;
            for (int p = tid; p < half; p += nt) {
                const int i = insert0(p, g.q1);
                if (i >> g.q0 & 1) {
                    const T2 t = st[i];
                    st[i] = st[i | M];
                    st[i | M] = t;
                }
            }
        } break;
        default: {  // CZ
            const int m = (1 << g.q0) | (1 << g.q1);
            for (int i = tid; i < dim; i += nt)
                if ((i & m) == m) st[i] = mk<T2>(-st[i].x, -st[i].y);
        } break;
    }
}

// Pauli X (1), Y (2) or Z (3) on qubit q of a state in LDS; 0 leaves it.
template <typename T2>
__device__ __forceinline__ void lds_pauli(T2* st, int q, int which, int n, int tid, int nt) {
    if (which == 0) return;
    const int half = 1 << (n - 1), M = 1 << q;
    for (int p = tid; p < half; p += nt) {
        const int i = insert0(p, q);
        const T2 u = st[i], v = st[i | M];
        if (which == 1) {
            st[i] = v;
            st[i | M] = u;
        } else if (which == 2) {
            st[i] = mk<T2>(v.y, -v.x);
            st[i | M] = mk<T2>(-u.y, u.x);
        } else {
            st[i | M] = mk<T2>(-v.x, -v.y);
        }
    }
}

template <typename T2, typename Real>
__device__ __forceinline__ Real lds_grad(const T2* p, const T2* l, const DevGate g, int n, int tid,
                                         int nt) {
    const int dim = 1 << n, half = dim >> 1;
    Real acc = 0;
    if (g.kind == K_RZ) {
        for (int i = tid; i < dim; i += nt) {
            const Real t = l[i].x * p[i].y - l[i].y * p[i].x;
            acc += (i >> g.q0 & 1) ? -t : t;
        }
    } else {
        const int M = 1 << g.q0;
        for (int q = tid; q < half; q += nt) {
            const int i = insert0(q, g.q0), v = i | M;
            if (g.kind == K_RX)
                acc += (l[i].x * p[v].y - l[i].y * p[v].x) + (l[v].x * p[i].y - l[v].y * p[i].x);
            else
                acc += (l[v].x * p[i].x + l[v].y * p[i].y) - (l[i].x * p[v].x + l[i].y * p[v].y);
        }
    }
    return acc;
}

template <typename Real>
__global__ void __launch_bounds__(256) k_whole(const WholeArgs a) {
    using T2 = typename Cx<Real>::T;
    extern __shared__ __align__(16) unsigned char smem[];
    const int n = a.n, dim = 1 << n;
    const int tid = threadIdx.x, nt = blockDim.x, NW = nt >> 6;
    const int wave = tid >> 6, lane = tid & 63;
    const int64_t b = blockIdx.x;
    T2* psi = (T2*)smem;
    T2* lam = psi + dim;
    double* red = (double*)(lam + dim);  // [n][NW]
    const T2* coef = (const T2*)a.coef + b * a.n_slots;

    if (a.psi_in)
        for (int j = tid; j < dim; j += nt) psi[j] = ((const T2*)a.psi_in)[b * dim + j];
    else
        for (int j = tid; j < dim; j += nt) psi[j] = mk<T2>((Real)(j == 0), (Real)0);
    __syncthreads();
    for (int gi = 0; gi < a.n_gates; ++gi) {
        const DevGate g = a.gates[gi];
        if (g.kind == K_PAULI) {
            lds_pauli(psi, g.q0, (int)coef[g.slot].x, n, tid, nt);
            __syncthreads();
            continue;
        }
        Real c = 1, s = 0;
        if (g.slot >= 0) {
            const T2 cs = coef[g.slot];
            c = cs.x;
            s = cs.y;
        }
        lds_gate(psi, g, c, s, n, tid, nt);
        __syncthreads();
    }
    if (a.psi_out)
        for (int j = tid; j < dim; j += nt) ((T2*)a.psi_out)[b * dim + j] = psi[j];
    for (int q = 0; q < n; ++q) {
        Real acc = 0;
        for (int j = tid; j < dim; j += nt) {
            const Real p = psi[j].x * psi[j].x + psi[j].y * psi[j].y;
            acc += (j >> q & 1) ? -p : p;
        }
        const double d = wave_sum((double)acc);
        if (lane == 0) red[q * NW + wave] = d;
    }
    __syncthreads();
    if (tid < n) {
        double t = 0;
        for (int w = 0; w < NW; ++w) t += red[tid * NW + w];
        a.zpart[b * n + tid] = t;
    }
    if (!a.bwd) return;
    __syncthreads();
    const Real* go = (const Real*)a.grad_out + b * n;
    for (int j = tid; j < dim; j += nt) {
        Real d = 0;
        for (int q = 0; q < n; ++q) d += (j >> q & 1) ? -go[q] : go[q];
        lam[j] = mk<T2>(d * psi[j].x, d * psi[j].y);
    }
    __syncthreads();
    for (int gi = a.n_gates - 1; gi >= 0; --gi) {
        const DevGate g = a.gates[gi];
        if (g.kind == K_PAULI) {  // its own inverse, no gradient
            const int which = (int)coef[g.slot].x;
            lds_pauli(psi, g.q0, which, n, tid, nt);
            lds_pauli(lam, g.q0, which, n, tid, nt);
            __syncthreads();
            continue;
        }
        Real c = 1, s = 0;
        if (g.slot >= 0) {
            const T2 cs = coef[g.slot];
            c = cs.x;
            s = cs.y;
            const double d = wave_sum((double)lds_grad<T2, Real>(psi, lam, g, n, tid, nt));
            if (lane == 0) red[wave] = d;
            __syncthreads();
            if (tid == 0) {
                double t = 0;
                for (int w = 0; w < NW; ++w) t += red[w];
                a.gpart[(size_t)g.slot * a.B + b] = t;
            }
        }
        lds_gate(psi, g, c, -s, n, tid, nt);
        lds_gate(lam, g, c, -s, n, tid, nt);
        __syncthreads();
    }
    if (a.lam_out)
        for (int j = tid; j < dim; j += nt) ((T2*)a.lam_out)[b * dim + j] = lam[j];
}

// ---------------------------------------------------------------------------
// k_tile: one tile pass
//
// Each workgroup streams tiles of 2^k amplitudes between HBM and registers and
// applies the pass's ops there. Every op is a per-sample record (handler id,
// argument, two coefficients) written by k_bind_tile; the op loop prefetches
// the next record and dispatches on the handler id into a handler whose
// register indices are compile-time constants.
//
// Every gate updates registers in place, so the state keeps its registers
// through the dispatch (the library is built with uniform regions left
// unstructurised). Rotations are exact three-shear products: a plane rotation
// by phi of (x, y) is  x -= a y;  y += b x;  x -= a y  with a = tan(phi/2),
// b = sin(phi). RY(theta) rotates (re u, re v) and (im u, im v) by theta/2; RX
// rotates (re u, im v) by -theta/2 and (im u, re v) by theta/2. Angles are
// reduced to [-pi, pi] first (a sign common to psi and lambda, which cancels in
// <Z> and in Im<lambda|P|psi>), so |a| <= 1.
//
// RZ(theta) = exp(-i theta/2) diag(1, exp(i theta)). On a register bit the
// kernel applies diag(1, exp(i theta)) only: the dropped factor is a global
// phase applied identically to psi and lambda (lambda is seeded from psi and
// both are un-applied by the same inverses), so it cancels in <Z> and in every
// Im<lambda|P|psi>. Only the bit-1 amplitudes are rotated, by theta reduced to
// [-pi/2, pi/2]; when the reduction moved theta by pi the rotated amplitudes
// are also negated (handler H_RZN, chosen per sample by k_bind_tile).

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

// Plane rotation of (x, y) by phi, in place: a = tan(phi/2), b = sin(phi).
template <typename Real>
__device__ __forceinline__ void shear(Real& x, Real& y, Real a, Real b) {
    x = fma(-a, y, x);
    y = fma(b, x, y);
    x = fma(-a, y, x);
}

// -(rotation by phi) of (x, y), in place; the negations are operand modifiers.
template <typename Real>
__device__ __forceinline__ void shear_neg(Real& x, Real& y, Real a, Real b) {
    x = fma(-a, y, x);
    y = fma(-b, x, -y);
    x = fma(-a, y, -x);
}

// One-qubit gate (KIND: 0 H, 1 RX, 2 RY, 3 RZ) on register bit J, in place.
// RZ applies diag(1, exp(i phi)) (a, b from phi; NEG: diag(1, -exp(i phi))).
template <int LOG_R, int KIND, int J, typename T2, typename Real, bool NEG = false>
__device__ __forceinline__ void g1(T2* s, Real a, Real b) {
    constexpr int R = 1 << LOG_R, M = 1 << J;
#pragma unroll
    for (int i = 0; i < R; ++i) {
        if (KIND == 3) {  // RZ: phase on the bit-1 amplitudes only
            if (i & M) {
                if (NEG) shear_neg(s[i].x, s[i].y, a, b);
                else shear(s[i].x, s[i].y, a, b);
            }
            continue;
        }
        if (i & M) continue;
        T2& u = s[i];
        T2& v = s[i | M];
        if (KIND == 0) {  // H: (u + v, u - v) / sqrt2
            const Real r = (Real)0.70710678118654752440;
            u.x += v.x;
            u.y += v.y;
            v.x = fma((Real)-2, v.x, u.x);
            v.y = fma((Real)-2, v.y, u.y);
            u.x *= r;
            u.y *= r;
            v.x *= r;
            v.y *= r;
        } else if (KIND == 1) {  // RX
            shear(u.x, v.y, -a, -b);
            shear(u.y, v.x, a, b);
        } else {  // RY
            shear(u.x, v.x, a, b);
            shear(u.y, v.y, a, b);
        }
    }
}

// Thread partial of Im<l | P_J | p> for the generator P of rotation KIND, as
// two interleaved FMA chains.
template <int LOG_R, int KIND, int J, typename T2, typename Real>
__device__ __forceinline__ Real gpart(const T2* p, const T2* l) {
    constexpr int R = 1 << LOG_R, M = 1 << J;
    Real acc[2] = {0, 0};
#pragma unroll
    for (int i = 0; i < R; ++i) {
        if (KIND == 3) {  // Z: (l.x p.y - l.y p.x), negated where bit J is set
            Real& c = acc[i & 1];
            if (i & M) {
                c = fma(-l[i].x, p[i].y, c);
                c = fma(l[i].y, p[i].x, c);
            } else {
                c = fma(l[i].x, p[i].y, c);
                c = fma(-l[i].y, p[i].x, c);
            }
            continue;
        }
        if (i & M) continue;
        const int v = i | M;
        Real& c = acc[(i >> (J == 0 ? 1 : 0)) & 1];
        if (KIND == 1) {  // X
            c = fma(l[i].x, p[v].y, c);
            c = fma(-l[i].y, p[v].x, c);
            c = fma(l[v].x, p[i].y, c);
            c = fma(-l[v].y, p[i].x, c);
        } else {  // Y
            c = fma(l[v].x, p[i].x, c);
            c = fma(l[v].y, p[i].y, c);
            c = fma(-l[i].x, p[v].x, c);
            c = fma(-l[i].y, p[v].y, c);
        }
    }
    return acc[0] + acc[1];
}

// Sum over this thread's registers of Im(conj(l) p) = l.x p.y - l.y p.x, over
// all registers (ALL) or those with register bit J set. The full sum is
// invariant under every op inside one register layout: each acts unitarily on
// the thread's registers, or multiplies psi and lambda by the same phase.
template <int LOG_R, int J, typename T2, typename Real>
__device__ __forceinline__ Real im_sum(const T2* p, const T2* l) {
    constexpr int R = 1 << LOG_R;
    Real acc[2] = {0, 0};
#pragma unroll
    for (int i = 0; i < R; ++i) {
        if (J >= 0 && !(i >> (J < 0 ? 0 : J) & 1)) continue;
        Real& c = acc[i & 1];
        c = fma(l[i].x, p[i].y, c);
        c = fma(-l[i].y, p[i].x, c);
    }
    return acc[0] + acc[1];
}

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

// Add the wavefront's gradient partial to its LDS accumulators gacc[g][wave]
// [2]: a row butterfly and one row broadcast leave each half-wavefront's sum
// in lanes 31 and 63, which add it to their own word (two words instead of
// one save the last broadcast step). Every word has one writer lane, so its
// sum is in program order (deterministic); the add has no return value.
constexpr int GRAD_WORDS = TILE_GRAD_WORDS;
template <typename Real>
__device__ __forceinline__ void grad_add(Real* gacc, uint32_t g, Real part, int lane, int wave, int nw) {
    Real v = row_sum(part);
    if constexpr (sizeof(Real) == 4) v += bcast_f32<0x142, 0xA>(v);
    else v += bcast_f64<0x142, 0xA>(v);
    if ((lane & 31) == 31)
        __hip_atomic_fetch_add(gacc + (g * (uint32_t)nw + (uint32_t)wave) * GRAD_WORDS + (lane >> 5), v,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Exchange two values in place (their registers keep their roles, so the
// state's register assignment is the same before and after the op).
__device__ __forceinline__ void xswap(float& x, float& y) {
    asm("v_swap_b32 %0, %1" : "+v"(x), "+v"(y));
}
__device__ __forceinline__ void xswap(double& x, double& y) {
    uint2 a = __builtin_bit_cast(uint2, x), b = __builtin_bit_cast(uint2, y);
    asm("v_swap_b32 %0, %1" : "+v"(a.x), "+v"(b.x));
    asm("v_swap_b32 %0, %1" : "+v"(a.y), "+v"(b.y));
    x = __builtin_bit_cast(double, a);
    y = __builtin_bit_cast(double, b);
}
template <typename T2>
__device__ __forceinline__ void xswap2(T2& u, T2& v) {
    xswap(u.x, v.x);
    xswap(u.y, v.y);
}

template <int LOG_R, int J, int MC, typename T2>
__device__ __forceinline__ void cnot_rr(T2* a) {
    constexpr int R = 1 << LOG_R, M = 1 << J, C = 1 << MC;
#pragma unroll
    for (int i = 0; i < R; ++i)
        if (!(i & M) && (i & C)) xswap2(a[i], a[i | M]);
}

// swap every pair across register bit J (X on that bit)
template <int LOG_R, int J, typename T2>
__device__ __forceinline__ void swap_all(T2* a) {
    constexpr int R = 1 << LOG_R, M = 1 << J;
#pragma unroll
    for (int i = 0; i < R; ++i)
        if (!(i & M)) xswap2(a[i], a[i | M]);
}

// Pauli P (0 X, 1 Y, 2 Z) on register bit J, exactly. Y maps (u, v) to
// (-i v, i u): swap u.x with v.y and u.y with v.x, then negate u.y and v.x.
template <int LOG_R, int P, int J, typename T2>
__device__ __forceinline__ void pauli(T2* a) {
    constexpr int R = 1 << LOG_R, M = 1 << J;
    if constexpr (P == 0) {
        swap_all<LOG_R, J>(a);
    } else {
#pragma unroll
        for (int i = 0; i < R; ++i)
            if (!(i & M)) {
                if constexpr (P == 1) {
                    xswap(a[i].x, a[i | M].y);
                    xswap(a[i].y, a[i | M].x);
                    a[i].y = -a[i].y;
                    a[i | M].x = -a[i | M].x;
                } else {
                    a[i | M].x = -a[i | M].x;
                    a[i | M].y = -a[i | M].y;
                }
            }
    }
}

// swap_all in the lanes where `on` holds
template <int LOG_R, int J, typename T2>
__device__ __forceinline__ void cnot_sel(T2* a, bool on) {
    if (on) swap_all<LOG_R, J>(a);
}

template <int LOG_R, int A, int B, typename T2>
__device__ __forceinline__ void cz_rr(T2* a) {
    constexpr int R = 1 << LOG_R, MA = 1 << A, MB = 1 << B;
#pragma unroll
    for (int i = 0; i < R; ++i)
        if ((i & MA) && (i & MB)) {
            a[i].x = -a[i].x;
            a[i].y = -a[i].y;
        }
}

// negate the amplitudes with register bit A set (all when A < 0) where on
template <int LOG_R, int A, typename T2>
__device__ __forceinline__ void cz_sel(T2* a, bool on) {
    constexpr int R = 1 << LOG_R;
#pragma unroll
    for (int i = 0; i < R; ++i)
        if (A < 0 || (i >> A & 1)) {
            a[i].x = on ? -a[i].x : a[i].x;
            a[i].y = on ? -a[i].y : a[i].y;
        }
}

// RZ on a thread bit or fixed qubit `bit`.
template <int LOG_R, typename T2, typename Real>
__device__ __forceinline__ void rz_u(T2* s, Real a, Real b, bool bit) {
    const Real sa = bit ? a : -a, sb = bit ? b : -b;
#pragma unroll
    for (int i = 0; i < (1 << LOG_R); ++i) shear(s[i].x, s[i].y, sa, sb);
}

// Tile bits `tb` and LDS byte offset `ts` of thread `tid` in phase F: every
// thread-index bit contributes its tile bit and its (precomputed) slot offset.
// Thread-index bits at or above log2(threads) are zero.
template <int LOG_T>
__device__ __forceinline__ void thread_layout(uint32_t tid, const DevPhase& F, uint32_t& tb, uint32_t& ts) {
    tb = 0;
    ts = 0;
#pragma unroll
    for (int b = 0; b < LOG_T; ++b) {
        const uint32_t on = (tid >> b) & 1u;
        tb |= on << F.thr_bit[b];
        ts ^= on ? F.thr_slot[b] : 0u;
    }
}

// Exchange the tile through LDS from layout `from` to layout `to`. The slot map
// is linear over GF(2) and thread and register bits are disjoint, so the byte
// offset of (thread, register i) is the thread's offset XOR the register's, and
// the register's is the XOR of its bits' columns reg_slot[1 << m]. Registers
// are visited in Gray-code order, so each access costs one XOR.
template <int LOG_R, typename T2>
__device__ __forceinline__ void lds_exchange(T2* a, unsigned char* lds, const DevPhase& from,
                                             const DevPhase& to, uint32_t ts_from, uint32_t ts_to) {
    constexpr int R = 1 << LOG_R;
    uint32_t cf[LOG_R], ct[LOG_R];
#pragma unroll
    for (int m = 0; m < LOG_R; ++m) {
        cf[m] = from.reg_slot[1 << m];
        ct[m] = to.reg_slot[1 << m];
    }
    uint32_t ad = ts_from;
#pragma unroll
    for (int g = 0; g < R; ++g) {
        *(T2*)(lds + ad) = a[g ^ (g >> 1)];
        if (g + 1 < R) ad ^= cf[__builtin_ctz(g + 1)];
    }
    __syncthreads();
    ad = ts_to;
#pragma unroll
    for (int g = 0; g < R; ++g) {
        a[g ^ (g >> 1)] = *(const T2*)(lds + ad);
        if (g + 1 < R) ad ^= ct[__builtin_ctz(g + 1)];
    }
    __syncthreads();
}

// Exchange register bit M with lane bit B (4 or 5) of a register tile: the
// amplitude at (lane L, register i) moves to (lane L with bit B := bit M of
// i, register i with bit M := bit B of L). For each register pair (lo: bit M
// = 0, hi: bit M = 1) the lanes with bit B = 1 of lo trade places with the
// lanes with bit B = 0 of hi, which is what the gfx950 permlane swaps do in
// one instruction per 32-bit register pair.
template <int B>
__device__ __forceinline__ void lane_swap_u32(uint32_t& lo, uint32_t& hi) {
    static_assert(B == 4 || B == 5, "lane swaps exist for lane bits 4 and 5");
    if constexpr (B == 5) {
        const auto r = __builtin_amdgcn_permlane32_swap(lo, hi, false, false);
        lo = r[0];
        hi = r[1];
    } else {
        const auto r = __builtin_amdgcn_permlane16_swap(lo, hi, false, false);
        lo = r[0];
        hi = r[1];
    }
}
template <int B>
__device__ __forceinline__ void lane_swap_real(float& lo, float& hi) {
    uint32_t l = __builtin_bit_cast(uint32_t, lo), h = __builtin_bit_cast(uint32_t, hi);
    lane_swap_u32<B>(l, h);
    lo = __builtin_bit_cast(float, l);
    hi = __builtin_bit_cast(float, h);
}
template <int B>
__device__ __forceinline__ void lane_swap_real(double& lo, double& hi) {
    uint2 l = __builtin_bit_cast(uint2, lo), h = __builtin_bit_cast(uint2, hi);
    lane_swap_u32<B>(l.x, h.x);
    lane_swap_u32<B>(l.y, h.y);
    lo = __builtin_bit_cast(double, l);
    hi = __builtin_bit_cast(double, h);
}
template <int LOG_R, int M, int B, typename T2>
__device__ __forceinline__ void lane_swap(T2* a) {
#pragma unroll
    for (int i = 0; i < (1 << LOG_R); ++i)
        if (!(i >> M & 1)) {
            lane_swap_real<B>(a[i].x, a[i | (1 << M)].x);
            lane_swap_real<B>(a[i].y, a[i | (1 << M)].y);
        }
}

// bit of an operand location word (thread bit or fixed qubit)
__device__ __forceinline__ bool loc_bit(uint32_t w, uint32_t tb, uint32_t gb) {
    const uint32_t pos = w & 0xff;
    return (((w >> 8) & 3) == LOC_THR ? (tb >> pos) : (gb >> pos)) & 1u;
}

// Per-thread tile state shared by the handlers.
struct TileCtx {
    uint32_t tb;   // tile-index bits of this thread (current phase)
    uint32_t ts;   // LDS byte offset of this thread's slots (current phase)
    uint32_t gb;   // amplitude-index bits of the qubits outside the tile (ps)
    uint32_t gb2;  // the same for the tile in lm (equal to gb unless two tiles)
    int ph;        // current phase
};

// An empty asm that uses an op record in scalar registers: the first record
// of an op loop is waited for before the loop, so the loop header (reached
// from the preheader and from the back edge) has no pending scalar load and
// each iteration's load of the next record overlaps the current op. (Without
// it the header waits on every iteration, since scalar loads return out of
// order and the wait must cover the record just issued.)
__device__ __forceinline__ void op_ready(const XOp<float>& o) {
    asm volatile("" ::"s"(o.h), "s"(o.arg), "s"(o.a), "s"(o.b));
}
__device__ __forceinline__ void op_ready(const XOp<double>& o) {
    asm volatile("" ::"s"(o.h), "s"(o.arg), "s"(o.a), "s"(o.b));
}

// An empty asm that reads every amplitude of a register tile: the compiler
// waits for the tile's pending loads here, once, instead of before the first
// use of each register inside every op handler.
template <int R>
__device__ __forceinline__ void tile_ready(const float2* t) {
#pragma unroll
    for (int i = 0; i < R; i += 4)
        asm volatile("" ::"v"(t[i].x), "v"(t[i].y), "v"(t[i + 1].x), "v"(t[i + 1].y), "v"(t[i + 2].x),
                     "v"(t[i + 2].y), "v"(t[i + 3].x), "v"(t[i + 3].y));
}
template <int R>
__device__ __forceinline__ void tile_ready(const double2* t) {
#pragma unroll
    for (int i = 0; i < R; i += 4)
        asm volatile("" ::"v"(t[i].x), "v"(t[i].y), "v"(t[i + 1].x), "v"(t[i + 1].y), "v"(t[i + 2].x),
                     "v"(t[i + 2].y), "v"(t[i + 3].x), "v"(t[i + 3].y));
}

// RZ group (H_DZ): register i of the tile gets the phase exp(i phi_i), phi_i
// the sum of the group's angles over the set bits of i (each RZ as
// diag(1, exp(i theta)), as on a single register bit); tab[i] = (cos phi_i,
// sin phi_i) from the binding kernel, INV: the inverse phase. A phase of any
// size is exact this way (four operations per register).
template <int LOG_R, bool INV, bool BOTH, typename T2>
__device__ __forceinline__ void dz_apply(T2* a, T2* b, const T2* __restrict__ tab) {
#pragma unroll
    for (int i = 1; i < (1 << LOG_R); ++i) {
        const T2 cs = tab[i];
        const auto c = cs.x, sn = INV ? -cs.y : cs.y;
        const auto x = a[i].x, y = a[i].y;
        a[i].x = fma(c, x, -sn * y);
        a[i].y = fma(c, y, sn * x);
        if constexpr (BOTH) {
            const auto u = b[i].x, v = b[i].y;
            b[i].x = fma(c, u, -sn * v);
            b[i].y = fma(c, v, sn * u);
        }
    }
}

// Gradient slot of the group's RZ on register bit J (NO_GSLOT: none), from
// the record's two coefficient words.
__device__ __forceinline__ uint32_t dz_gslot(float a, float b, int j) {
    const uint32_t w = __builtin_bit_cast(uint32_t, j < 2 ? a : b);
    return (w >> ((j & 1) * 16)) & 0xffffu;
}
__device__ __forceinline__ uint32_t dz_gslot(double a, double, int j) {
    return (uint32_t)(__builtin_bit_cast(uint64_t, a) >> (j * 16)) & 0xffffu;
}

// Z-generator terms of the group's RZs (each as for a single RZ on its bit;
// a diagonal op leaves every register's Im(conj(lambda) psi) unchanged, so
// the terms are the same before and after the group's phase).
template <int LOG_R, int J, typename T2, typename Real>
__device__ __forceinline__ void dz_grads(const T2* ps, const T2* lm, Real ca, Real cb, Real ival, Real* gacc,
                                         int lane, int wave, int nw) {
    if constexpr (J < LOG_R) {
        const uint32_t g = dz_gslot(ca, cb, J);
        if (g != NO_GSLOT)
            grad_add(gacc, g, fma((Real)-2, im_sum<LOG_R, J, T2, Real>(ps, lm), ival), lane, wave, nw);
        dz_grads<LOG_R, J + 1>(ps, lm, ca, cb, ival, gacc, lane, wave, nw);
    }
}

// Apply one op. OPM selects the register arrays it acts on:
//   OP_ONE  -- ps only (one forward tile);
//   OP_PAIR -- ps and lm, two forward tiles that differ in their fixed bits
//              (cx.gb for ps, cx.gb2 for lm);
//   OP_BWD  -- the gradient term Im<lambda|P|psi> of a rotation into the
//              wavefront's accumulator, then the op (its inverse, from the
//              binding) on psi (ps) and lambda (lm) of one tile.
enum { OP_ONE = 0, OP_PAIR = 1, OP_BWD = 2 };
//
// In OP_BWD, `ival` holds the thread's full Im(conj(lambda) psi) sum of the
// current layout (refreshed after each exchange), so the Z-generator term of
// an RZ is ival - 2 * (the bit-1 half), and of an RZ on a thread or fixed bit
// +-ival.
template <int LOG_R, int LOG_T, int OPM, typename T2, typename Real>
__device__ __forceinline__ void run_op(uint32_t h, uint32_t arg, Real ca, Real cb, T2* ps, T2* lm,
                                       TileCtx& cx, Real& ival, unsigned char* lds,
                                       const DevPhase* phases, Real* gacc, int lane, int wave, int nw,
                                       int tid, const T2* __restrict__ dz, const T2* __restrict__ fz) {
#define QL_G1_CASE(KIND, J)                                                                 \
    case H_G1 + KIND * 5 + J:                                                               \
        if constexpr (J < LOG_R) {                                                          \
            if constexpr (OPM == OP_BWD && KIND == 3)                                       \
                grad_add(gacc, arg, fma((Real)-2, im_sum<LOG_R, J, T2, Real>(ps, lm), ival),  \
                         lane, wave, nw);                                                   \
            else if constexpr (OPM == OP_BWD && KIND != 0)                                  \
                grad_add(gacc, arg, gpart<LOG_R, KIND, J, T2, Real>(ps, lm), lane, wave, nw); \
            if constexpr (OPM != OP_ONE) g1<LOG_R, KIND, J, T2, Real>(lm, ca, cb);            \
            g1<LOG_R, KIND, J, T2, Real>(ps, ca, cb);                                       \
        }                                                                                   \
        break;
#define QL_RZN_CASE(J)                                                                      \
    case H_RZN + J:                                                                         \
        if constexpr (J < LOG_R) {                                                          \
            if constexpr (OPM == OP_BWD)                                                    \
                grad_add(gacc, arg, fma((Real)-2, im_sum<LOG_R, J, T2, Real>(ps, lm), ival),  \
                         lane, wave, nw);                                                   \
            if constexpr (OPM != OP_ONE) g1<LOG_R, 3, J, T2, Real, true>(lm, ca, cb);         \
            g1<LOG_R, 3, J, T2, Real, true>(ps, ca, cb);                                    \
        }                                                                                   \
        break;
#define QL_G1_J(J) QL_G1_CASE(0, J) QL_G1_CASE(1, J) QL_G1_CASE(2, J) QL_G1_CASE(3, J)
#define QL_CNOT_RR(J, M)                                                                    \
    case H_CNOT_RR + J * 5 + M:                                                             \
        if constexpr (J < LOG_R && M < LOG_R && J != M) {                                   \
            cnot_rr<LOG_R, J, M>(ps);                                                       \
            if constexpr (OPM != OP_ONE) cnot_rr<LOG_R, J, M>(lm);                          \
        }                                                                                   \
        break;
#define QL_CNOT_RR_J(J) QL_CNOT_RR(J, 0) QL_CNOT_RR(J, 1) QL_CNOT_RR(J, 2) QL_CNOT_RR(J, 3) QL_CNOT_RR(J, 4)
#define QL_CNOT_X(J)                                                                        \
    case H_CNOT_T + J:                                                                      \
        if constexpr (J < LOG_R) {                                                          \
            const bool on = (cx.tb >> arg) & 1u;                                            \
            cnot_sel<LOG_R, J>(ps, on);                                                     \
            if constexpr (OPM != OP_ONE) cnot_sel<LOG_R, J>(lm, on);                        \
        }                                                                                   \
        break;                                                                              \
    case H_CNOT_F + J:                                                                      \
        if constexpr (J < LOG_R) {                                                          \
            if ((cx.gb >> arg) & 1u) swap_all<LOG_R, J>(ps);                                \
            if constexpr (OPM != OP_ONE)                                                    \
                if ((cx.gb2 >> arg) & 1u) swap_all<LOG_R, J>(lm);                           \
        }                                                                                   \
        break;
#define QL_CZ_RR(A, B)                                                                      \
    case H_CZ_RR + A * 5 + B:                                                               \
        if constexpr (A < LOG_R && B < LOG_R && A != B) {                                   \
            cz_rr<LOG_R, A, B>(ps);                                                         \
            if constexpr (OPM != OP_ONE) cz_rr<LOG_R, A, B>(lm);                            \
        }                                                                                   \
        break;
#define QL_CZ_RR_A(A) QL_CZ_RR(A, 0) QL_CZ_RR(A, 1) QL_CZ_RR(A, 2) QL_CZ_RR(A, 3) QL_CZ_RR(A, 4)
// A lane swap moves one tile bit x off lane bit B and tile bit y onto it: the
// threads with lane bit B set trade x for y in their tile bits and in their
// LDS offset (linear in the tile bits).
#define QL_LSWAP(M, B)                                                                      \
    case H_LSWAP + M * 6 + B:                                                               \
        if constexpr (M < LOG_R && B < LOG_T) {                                             \
            lane_swap<LOG_R, M, B>(ps);                                                     \
            if constexpr (OPM != OP_ONE) lane_swap<LOG_R, M, B>(lm);                        \
            cx.ph = (int)(arg & 0xfffff);                                                   \
            const uint32_t dtb = (1u << ((arg >> 20) & 31)) | (1u << (arg >> 25));         \
            if ((lane >> B) & 1) {                                                          \
                cx.tb ^= dtb;                                                               \
                cx.ts ^= lds_slot(dtb) * (uint32_t)sizeof(T2);                              \
            }                                                                               \
            if constexpr (OPM == OP_BWD) ival = im_sum<LOG_R, -1, T2, Real>(ps, lm);        \
        }                                                                                   \
        break;
#define QL_LSWAP_M(M) QL_LSWAP(M, 4) QL_LSWAP(M, 5)
// A Pauli is its own inverse and maps each thread's register set onto itself,
// so the backward sweep applies it as is and the per-thread Im<lambda|psi>
// stays valid.
#define QL_PAULI_CASE(P, J)                                                                 \
    case H_PX + P * 5 + J:                                                                  \
        if constexpr (J < LOG_R) {                                                          \
            pauli<LOG_R, P, J>(ps);                                                         \
            if constexpr (OPM != OP_ONE) pauli<LOG_R, P, J>(lm);                            \
        }                                                                                   \
        break;
#define QL_PAULI_J(J) QL_PAULI_CASE(0, J) QL_PAULI_CASE(1, J) QL_PAULI_CASE(2, J)
// RY then RZ on register bit J (the RZ's shear coefficients, forward, from
// the pair table; the backward form inverts both and runs them in reverse
// order, each with its gradient term first, as the two separate ops would).
#define QL_RYZ_CASE(J, NEG)                                                                 \
    case (NEG ? H_RYZN : H_RYZ) + J:                                                        \
        if constexpr (J < LOG_R) {                                                          \
            const T2 zc = fz[arg >> 16];                                                    \
            if constexpr (OPM == OP_BWD) {                                                  \
                grad_add(gacc, (arg >> 8) & 0xffu,                                          \
                         fma((Real)-2, im_sum<LOG_R, J, T2, Real>(ps, lm), ival), lane, wave, nw); \
                g1<LOG_R, 3, J, T2, Real, NEG>(lm, -zc.x, -zc.y);                           \
                g1<LOG_R, 3, J, T2, Real, NEG>(ps, -zc.x, -zc.y);                           \
                grad_add(gacc, arg & 0xffu, gpart<LOG_R, 2, J, T2, Real>(ps, lm), lane, wave, nw); \
                g1<LOG_R, 2, J, T2, Real>(lm, ca, cb);                                      \
                g1<LOG_R, 2, J, T2, Real>(ps, ca, cb);                                      \
            } else {                                                                        \
                g1<LOG_R, 2, J, T2, Real>(ps, ca, cb);                                      \
                if constexpr (OPM == OP_PAIR) g1<LOG_R, 2, J, T2, Real>(lm, ca, cb);        \
                g1<LOG_R, 3, J, T2, Real, NEG>(ps, zc.x, zc.y);                             \
                if constexpr (OPM == OP_PAIR) g1<LOG_R, 3, J, T2, Real, NEG>(lm, zc.x, zc.y); \
            }                                                                               \
        }                                                                                   \
        break;
#define QL_RYZ_J(J) QL_RYZ_CASE(J, false) QL_RYZ_CASE(J, true)
#define QL_CZ_RX(A)                                                                         \
    case H_CZ_RX + A:                                                                       \
        if constexpr (A < LOG_R) {                                                          \
            cz_sel<LOG_R, A>(ps, loc_bit(arg, cx.tb, cx.gb));                               \
            if constexpr (OPM != OP_ONE) cz_sel<LOG_R, A>(lm, loc_bit(arg, cx.tb, cx.gb2));   \
        }                                                                                   \
        break;
    switch (h) {
        QL_G1_J(0) QL_G1_J(1) QL_G1_J(2) QL_G1_J(3) QL_G1_J(4)
        QL_CNOT_RR_J(0) QL_CNOT_RR_J(1) QL_CNOT_RR_J(2) QL_CNOT_RR_J(3) QL_CNOT_RR_J(4)
        QL_CNOT_X(0) QL_CNOT_X(1) QL_CNOT_X(2) QL_CNOT_X(3) QL_CNOT_X(4)
        QL_CZ_RR_A(0) QL_CZ_RR_A(1) QL_CZ_RR_A(2) QL_CZ_RR_A(3) QL_CZ_RR_A(4)
        QL_CZ_RX(0) QL_CZ_RX(1) QL_CZ_RX(2) QL_CZ_RX(3) QL_CZ_RX(4)
        QL_RZN_CASE(0) QL_RZN_CASE(1) QL_RZN_CASE(2) QL_RZN_CASE(3) QL_RZN_CASE(4)
        QL_LSWAP_M(0) QL_LSWAP_M(1) QL_LSWAP_M(2) QL_LSWAP_M(3) QL_LSWAP_M(4)
        QL_PAULI_J(0) QL_PAULI_J(1) QL_PAULI_J(2) QL_PAULI_J(3) QL_PAULI_J(4)
        QL_RYZ_J(0) QL_RYZ_J(1) QL_RYZ_J(2) QL_RYZ_J(3) QL_RYZ_J(4)
        case H_NOP:
            break;
        case H_DZ:
            if constexpr (LOG_R <= MAX_DZ_BITS) {
                if constexpr (OPM == OP_BWD) dz_grads<LOG_R, 0>(ps, lm, ca, cb, ival, gacc, lane, wave, nw);
                dz_apply<LOG_R, OPM == OP_BWD, OPM != OP_ONE>(ps, lm, dz + (size_t)arg * DZ_REGS);
            }
            break;
        case H_RZU: {
            const bool bit = loc_bit(arg, cx.tb, cx.gb);
            if constexpr (OPM == OP_BWD) {
                grad_add(gacc, arg >> 16, bit ? -ival : ival, lane, wave, nw);
                rz_u<LOG_R>(lm, ca, cb, bit);
            } else if constexpr (OPM == OP_PAIR) {
                rz_u<LOG_R>(lm, ca, cb, loc_bit(arg, cx.tb, cx.gb2));
            }
            rz_u<LOG_R>(ps, ca, cb, bit);
        } break;
        case H_CZ_XX: {
            const bool on = loc_bit(arg & 0xffff, cx.tb, cx.gb) && loc_bit(arg >> 16, cx.tb, cx.gb);
            cz_sel<LOG_R, -1>(ps, on);
            if constexpr (OPM != OP_ONE)
                cz_sel<LOG_R, -1>(lm, loc_bit(arg & 0xffff, cx.tb, cx.gb2) && loc_bit(arg >> 16, cx.tb, cx.gb2));
        } break;
        case H_TRANSPOSE: {
            const DevPhase& to = phases[arg];
            uint32_t tb_to, ts_to;
            thread_layout<LOG_T>((uint32_t)tid, to, tb_to, ts_to);
            lds_exchange<LOG_R>(ps, lds, phases[cx.ph], to, cx.ts, ts_to);
            if constexpr (OPM != OP_ONE) lds_exchange<LOG_R>(lm, lds, phases[cx.ph], to, cx.ts, ts_to);
            if constexpr (OPM == OP_BWD) ival = im_sum<LOG_R, -1, T2, Real>(ps, lm);
            cx.tb = tb_to;
            cx.ts = ts_to;
            cx.ph = (int)arg;
        } break;
        default:
            __builtin_unreachable();
    }
#undef QL_G1_CASE
#undef QL_RZN_CASE
#undef QL_G1_J
#undef QL_CNOT_RR
#undef QL_CNOT_RR_J
#undef QL_CNOT_X
#undef QL_CZ_RR
#undef QL_CZ_RR_A
#undef QL_CZ_RX
#undef QL_LSWAP
#undef QL_LSWAP_M
#undef QL_PAULI_CASE
#undef QL_PAULI_J
#undef QL_RYZ_CASE
#undef QL_RYZ_J
}

// <Z_q> partials of one tile held in registers t: register bits from the
// signed register sums, lane bits from lane-signed wavefront sums, wavefront
// bits and fixed bits (tbit: this lane's fixed-qubit bit of the tile) from the
// tile total with a uniform sign. Lane q of accz collects tile qubit q; lane i
// of accf collects fixed qubit i.
template <int LOG_R, int LOG_T, typename Real, typename T2>
__device__ __forceinline__ void zpart_tile(const T2* t, uint32_t tbit, const uint32_t* qreg,
                                           const uint32_t* qthr, int lane, int wave, double& accz,
                                           double& accf) {
    Real pt = 0, dm[LOG_R];
#pragma unroll
    for (int m = 0; m < LOG_R; ++m) dm[m] = 0;
#pragma unroll
    for (int i = 0; i < (1 << LOG_R); ++i) {
        const Real p = t[i].x * t[i].x + t[i].y * t[i].y;
        pt += p;
#pragma unroll
        for (int m = 0; m < LOG_R; ++m) dm[m] += (i >> m & 1) ? -p : p;
    }
#pragma unroll
    for (int m = 0; m < LOG_R; ++m) {
        const double d = wave_total(dm[m]);
        accz += (lane == (int)qreg[m]) ? d : 0.0;
    }
#pragma unroll
    for (int b = 0; b < 6; ++b) {
        const double d = wave_total((lane >> b & 1) ? -pt : pt);
        accz += (lane == (int)qthr[b]) ? d : 0.0;
    }
    const double wp = wave_total(pt);
#pragma unroll
    for (int b = 6; b < LOG_T; ++b) accz += (lane == (int)qthr[b]) ? ((wave >> (b - 6) & 1) ? -wp : wp) : 0.0;
    accf += tbit ? -wp : wp;
}

// Bits of t deposited, lowest first, on the set bits of mask (both uniform:
// scalar arithmetic).
__device__ __forceinline__ uint32_t deposit_bits(uint32_t t, uint32_t mask) {
    uint32_t r = 0;
    while (mask) {
        const uint32_t low = mask & (0u - mask);
        if (t & 1u) r |= low;
        t >>= 1;
        mask ^= low;
    }
    return r;
}

// Kernel modes: one forward tile per iteration, two forward tiles per
// iteration (the tile index and the same index with its top bit set), or the
// backward sweep (psi and lambda of one tile).
enum { KM_FWD1 = 0, KM_FWD2 = 1, KM_BWD = 2 };

template <typename Real, int LOG_R, int KM, int MAXT>
__global__ void __launch_bounds__(MAXT) __attribute__((amdgpu_waves_per_eu(2)))
k_tile(const TileArgs a, const DevPass* __restrict__ pass, const DevPhase* __restrict__ phases,
       const XOp<Real>* __restrict__ xops_all, const Real* __restrict__ gout_all,
       const int32_t* __restrict__ gslots, const typename Cx<Real>::T* __restrict__ dz_all,
       const typename Cx<Real>::T* __restrict__ fz_all) {
    using T2 = typename Cx<Real>::T;
    constexpr bool BWD = KM == KM_BWD, PAIR = KM == KM_FWD2;
    constexpr int R = 1 << LOG_R;
    constexpr int LOG_T = MAXT == 512 ? 9 : 8;
    // The tile exchange buffer is static (its LDS address is a compile-time
    // constant, so exchange addresses need no base add); the reduction
    // scratch is dynamic and follows it.
    __shared__ __align__(16) unsigned char tile_lds[tile_lds_bytes<Real, LOG_R, MAXT>()];
    extern __shared__ __align__(16) unsigned char smem[];
    const DevPass& P = *pass;
    const int tid = threadIdx.x, nt = blockDim.x, NW = nt >> 6;
    const int wave = tid >> 6, lane = tid & 63;
    const int flags = a.flags;
    const int64_t b = blockIdx.x / a.n_wg;
    const int w = (int)(blockIdx.x - b * a.n_wg);
    const int n = a.n, k = P.k, n_fixed = P.n_fixed;
    const int fwd_begin = P.fwd_begin, fwd_end = P.fwd_end;
    const int bwd_begin = P.bwd_begin, bwd_end = P.bwd_end;
    unsigned char* lds = tile_lds;
    double* red = (double*)smem;                       // [n][NW]
    constexpr int GW = GRAD_WORDS;
    Real* gacc = (Real*)(red + (size_t)n * NW);        // [n_gslots][NW][GW]

    const size_t dim = (size_t)1 << n;
    const T2* psi_s = (const T2*)a.psi + b * dim;
    T2* psi_o = (T2*)a.psi_out + b * dim;
    T2* lam_s = (T2*)a.lam + b * dim;
    const XOp<Real>* xops = xops_all + b * (a.n_ops + 1);
    const T2* dz = dz_all + b * a.n_diags * DZ_REGS;
    const T2* fz = fz_all + b * a.n_fuses;
    const Real* gout = gout_all + b * n;

    if (BWD && (flags & PF_BWD)) {
        for (int i = tid; i < a.n_gslots * NW * GW; i += nt) gacc[i] = (Real)0;
        __syncthreads();
    }

    // Phases are the same for every tile: the pass loads in ph0, stores in
    // ph_st (the backward ops walk the forward layouts back to the first one),
    // and takes <Z> and the lambda seed in the last forward layout. Only the
    // fixed (out-of-tile) qubit bits change from tile to tile.
    auto amp_offset = [&](uint32_t tb) {  // amplitude-index bits of tile bits tb
        uint32_t g = 0;
        for (int j = 0; j < k; ++j) g |= ((tb >> j) & 1u) << P.tile_qubit[j];
        return g;
    };
    const int ph0 = (flags & PF_FWD) ? P.load_phase : P.bwd_phase;
    const int ph_st = (BWD && (flags & PF_BWD)) ? P.load_phase : P.bwd_phase;
    uint32_t tb0, ts0, tb_st, ts_st;
    thread_layout<LOG_T>((uint32_t)tid, phases[ph0], tb0, ts0);
    thread_layout<LOG_T>((uint32_t)tid, phases[ph_st], tb_st, ts_st);
    const uint32_t toff0 = amp_offset(tb0), toff_st = amp_offset(tb_st);
    // lane i < n_fixed holds fixed qubit i (for the per-qubit sums)
    const uint32_t fq_lane = lane < n_fixed ? (uint32_t)P.fixed_qubit[lane] : 0u;
    // a tile's fixed (out-of-tile) amplitude-index bits: the bits of the tile
    // index deposited on the fixed qubits, lowest first. Uniform arithmetic:
    // no lane-dependent value is needed where the tile loop begins, so its
    // first wait is not a wait for every memory operation in flight.
    uint32_t fixed_mask = 0;
    for (int j = 0; j < n_fixed; ++j) fixed_mask |= 1u << P.fixed_qubit[j];

    // <Z> and seed constants of the last forward layout: the qubit of each
    // register bit and of each thread-index bit
    uint32_t tbz = 0, qreg[LOG_R], qthr[LOG_T];
    Real seed_base = 0, gm[LOG_R], gfix = 0;
    double accz = 0.0, accf = 0.0;  // lane q: <Z_q> of tile qubit q; lane i: of fixed qubit i
#pragma unroll
    for (int m = 0; m < LOG_R; ++m) {
        gm[m] = 0;
        qreg[m] = 0;
    }
#pragma unroll
    for (int t = 0; t < LOG_T; ++t) qthr[t] = 0;
    if (flags & (PF_ZPART | PF_SEED)) {
        const DevPhase& F = phases[P.bwd_phase];
        uint32_t tsz;
        thread_layout<LOG_T>((uint32_t)tid, F, tbz, tsz);
#pragma unroll
        for (int m = 0; m < LOG_R; ++m) qreg[m] = (uint32_t)P.tile_qubit[F.reg_bit[m]];
#pragma unroll
        for (int t = 0; t < LOG_T; ++t)  // 64 (no lane) for thread bits this launch does not have
            qthr[t] = t < P.log_t ? (uint32_t)P.tile_qubit[F.thr_bit[t]] : 64u;
        if (BWD && (flags & PF_SEED)) {
            Real gs = 0, sthr = 0;
            for (int q = 0; q < n; ++q) gs += gout[q];
            for (int j = 0; j < k; ++j)
                if ((F.thr_mask >> j & 1u) && (tbz >> j & 1u)) sthr += gout[P.tile_qubit[j]];
            seed_base = gs - (Real)2 * sthr;
#pragma unroll
            for (int m = 0; m < LOG_R; ++m) gm[m] = gout[P.tile_qubit[F.reg_bit[m]]];
            gfix = lane < n_fixed ? gout[fq_lane] : (Real)0;
        }
    }

    const bool load = !(flags & PF_INIT);
    const bool load_lam = BWD && (flags & PF_LOAD_LAM);
    auto load_tile = [&](T2* dst, const T2* state, uint32_t gb) {
        const DevPhase& F = phases[ph0];
        const T2* src = state + (gb | toff0);
#pragma unroll
        for (int i = 0; i < R; ++i) dst[i] = src[F.reg_qoff[i]];
    };

    // two-tile mode: the second tile has the top tile-index bit set, i.e. the
    // highest fixed qubit
    const int64_t tiles = PAIR ? a.tiles >> 1 : a.tiles;
    const uint32_t top_fixed = (PAIR && n_fixed > 0) ? 1u << P.fixed_qubit[n_fixed - 1] : 0u;
    auto fixed_bits = [&](int64_t t) { return deposit_bits((uint32_t)t, fixed_mask); };
    T2 ps[R], lm[R];
    // one-tile forward mode: the next tile's loads are issued before this
    // tile's ops run (nothing in the ops reads nx, so they stay in flight
    // through the exchanges)
    constexpr bool PREF = KM == KM_FWD1;
    T2 nx[PREF ? R : 1];
    if (PREF && load && w < tiles) load_tile(nx, psi_s, fixed_bits(w));
    Real ival = 0;  // see run_op
    for (int64_t tile = w; tile < tiles; tile += a.n_wg) {
        const uint32_t tbit = lane < n_fixed ? (((uint32_t)tile >> lane) & 1u) : 0u;
        TileCtx cx;
        cx.gb = fixed_bits(tile);
        cx.gb2 = cx.gb | top_fixed;
        cx.ph = ph0;
        cx.tb = tb0;
        cx.ts = ts0;

        if (!load) {
#pragma unroll
            for (int i = 0; i < R; ++i) ps[i] = mk<T2>((Real)0, (Real)0);
            if (cx.gb == 0 && cx.tb == 0) ps[0] = mk<T2>((Real)1, (Real)0);
            if constexpr (PAIR) {  // the second tile never holds amplitude 0
#pragma unroll
                for (int i = 0; i < R; ++i) lm[i] = mk<T2>((Real)0, (Real)0);
            }
        } else if constexpr (PREF) {
#pragma unroll
            for (int i = 0; i < R; ++i) ps[i] = nx[i];
            if (tile + a.n_wg < tiles) load_tile(nx, psi_s, fixed_bits(tile + a.n_wg));
        } else {
            load_tile(ps, psi_s, cx.gb);
            if (PAIR) load_tile(lm, psi_s, cx.gb2);
            else if (load_lam) load_tile(lm, lam_s, cx.gb);
            tile_ready<R>(ps);
            if (PAIR || load_lam) tile_ready<R>(lm);
        }

        // ---- forward ops
        if (flags & PF_FWD) {
            XOp<Real> cur = xops[fwd_begin];
            op_ready(cur);
            for (int o = fwd_begin; o < fwd_end; ++o) {
                const XOp<Real> nxt = xops[o + 1];
                run_op<LOG_R, LOG_T, PAIR ? OP_PAIR : OP_ONE>(cur.h, cur.arg, cur.a, cur.b, ps, lm, cx,
                                                              ival, lds, phases, gacc, lane, wave, NW,
                                                              tid, dz, fz);
                cur = nxt;
            }
        }

        // ---- <Z_q> partials over this tile: register bits from the signed
        // register sums, lane bits from lane-signed wavefront sums, wavefront
        // bits and fixed bits from the tile total with a uniform sign
        if (flags & PF_ZPART) {
            zpart_tile<LOG_R, LOG_T, Real>(ps, tbit, qreg, qthr, lane, wave, accz, accf);
            if constexpr (PAIR)
                zpart_tile<LOG_R, LOG_T, Real>(lm, tbit | (uint32_t)(lane == n_fixed - 1), qreg, qthr, lane,
                                               wave, accz, accf);
        }

        if constexpr (BWD) {
            // ---- lambda = (sum_q g_q Z_q) psi
            if (flags & PF_SEED) {
                const Real sfix = (Real)wave_total(tbit ? gfix : (Real)0);
                const Real base = seed_base - (Real)2 * sfix;
#pragma unroll
                for (int i = 0; i < R; ++i) {
                    Real sr = 0;
#pragma unroll
                    for (int m = 0; m < LOG_R; ++m)
                        if (i >> m & 1) sr += gm[m];
                    const Real d = base - (Real)2 * sr;
                    lm[i] = mk<T2>(d * ps[i].x, d * ps[i].y);
                }
            }

            // ---- backward ops
            if (flags & PF_BWD) {
                ival = im_sum<LOG_R, -1, T2, Real>(ps, lm);
                XOp<Real> cur = xops[bwd_begin];
                op_ready(cur);
                for (int o = bwd_begin; o < bwd_end; ++o) {
                    const XOp<Real> nxt = xops[o + 1];
                    run_op<LOG_R, LOG_T, OP_BWD>(cur.h, cur.arg, cur.a, cur.b, ps, lm, cx, ival, lds,
                                                 phases, gacc, lane, wave, NW, tid, dz, fz);
                    cur = nxt;
                }
            }
        }

        if (flags & (PF_STORE_PSI | PF_STORE_LAM)) {
            const DevPhase& F = phases[ph_st];
            const uint32_t base = cx.gb | toff_st;
            if (flags & PF_STORE_PSI) {
                T2* dst = psi_o + base;
#pragma unroll
                for (int i = 0; i < R; ++i) dst[F.reg_qoff[i]] = ps[i];
                if constexpr (PAIR) {
                    T2* dst2 = psi_o + (cx.gb2 | toff_st);
#pragma unroll
                    for (int i = 0; i < R; ++i) dst2[F.reg_qoff[i]] = lm[i];
                }
            }
            if (BWD && (flags & PF_STORE_LAM)) {
                T2* dst = lam_s + base;
#pragma unroll
                for (int i = 0; i < R; ++i) dst[F.reg_qoff[i]] = lm[i];
            }
        }
    }

    // combine the wavefronts' accumulators (fixed order) and write the partials
    if (flags & PF_ZPART) {
        // two stores from one wavefront land in order: a fixed qubit's slot
        // first gets 0 from accz, then its own sum
        if (lane < n) red[lane * NW + wave] = accz;
        if (lane < n_fixed) red[fq_lane * NW + wave] = accf;
    }
    __syncthreads();
    if (flags & PF_ZPART)
        for (int q = tid; q < n; q += nt) {
            double t = 0;
            for (int v = 0; v < NW; ++v) t += red[q * NW + v];
            a.zpart[((size_t)b * a.n_wg + w) * n + q] = t;
        }
    if (BWD && (flags & PF_BWD))
        for (int g = tid; g < a.n_gslots; g += nt) {
            double t = 0;
            for (int v = 0; v < NW * GW; ++v) t += (double)gacc[g * NW * GW + v];
            a.gpart[((size_t)gslots[g] * a.B + b) * a.n_wg + w] = t;
        }
}

// ---------------------------------------------------------------------------
// k_wave: the whole state of one sample in one wavefront's registers (n <= 8)
//
// Amplitude j = lane + 64 i sits in register i of lane j mod 64: 2^(n-6)
// registers per lane, one for n <= 6 (lanes >= 2^n then hold zeros and never
// mix with the others). A gate on qubit q < 6 pairs each lane with lane ^ 2^q
// through a cross-lane shuffle; on qubit q >= 6, register i with register
// i ^ 2^(q-6) of the same lane. Every lane computes its own new amplitude from
// its old one and its partner's, so there is no LDS traffic and no barrier:
// each gate is wavefront-synchronous. Same arguments, coefficient table and
// partial layouts as k_whole.

// bit q of amplitude lane + 64 r
__device__ __forceinline__ int amp_bit(int q, int lane, int r) {
    return q < 6 ? (lane >> q) & 1 : (r >> (q - 6)) & 1;
}

// The value of lane ^ 2^B, without the LDS pipe: quad permutes (B = 0, 1),
// two row shifts under bank masks (B = 2, 3: lanes with bit B clear read from
// +2^B, the others from -2^B), a permlane swap of two copies and a select
// (B = 4, 5).
template <int B>
__device__ __forceinline__ uint32_t xor_lane_u32(uint32_t v, int lane) {
    if constexpr (B == 0) {
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
    } else if constexpr (B == 1) {
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
    } else if constexpr (B <= 3) {
        constexpr int SHL = 0x100 + (1 << B), SHR = 0x110 + (1 << B);
        constexpr int LOW = B == 2 ? 0x5 : 0x3, HIGH = B == 2 ? 0xA : 0xC;  // banks by lane bit B
        const int lo = __builtin_amdgcn_update_dpp(0, (int)v, SHL, 0xF, LOW, false);
        return (uint32_t)__builtin_amdgcn_update_dpp(lo, (int)v, SHR, 0xF, HIGH, false);
    } else {
        const auto r = B == 4 ? __builtin_amdgcn_permlane16_swap(v, v, false, false)
                              : __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return ((lane >> B) & 1) ? r[0] : r[1];
    }
}
template <int B>
__device__ __forceinline__ float xor_lane(float v, int lane) {
    return __builtin_bit_cast(float, xor_lane_u32<B>(__builtin_bit_cast(uint32_t, v), lane));
}
template <int B>
__device__ __forceinline__ double xor_lane(double v, int lane) {
    uint2 u = __builtin_bit_cast(uint2, v);
    u.x = xor_lane_u32<B>(u.x, lane);
    u.y = xor_lane_u32<B>(u.y, lane);
    return __builtin_bit_cast(double, u);
}
template <typename T2>
__device__ __forceinline__ T2 xlane(T2 v, int q, int lane) {
    switch (q) {
        case 0: return mk<T2>(xor_lane<0>(v.x, lane), xor_lane<0>(v.y, lane));
        case 1: return mk<T2>(xor_lane<1>(v.x, lane), xor_lane<1>(v.y, lane));
        case 2: return mk<T2>(xor_lane<2>(v.x, lane), xor_lane<2>(v.y, lane));
        case 3: return mk<T2>(xor_lane<3>(v.x, lane), xor_lane<3>(v.y, lane));
        case 4: return mk<T2>(xor_lane<4>(v.x, lane), xor_lane<4>(v.y, lane));
        default: return mk<T2>(xor_lane<5>(v.x, lane), xor_lane<5>(v.y, lane));
    }
}

// New value of one amplitude (bit `bit` of the gate's qubit) from its old value
// and its partner's: H, RX (both bits alike), RY; Pauli X (1), Y (2), Z (3) by
// `which` for K_PAULI. (c, s) = (cos t/2, sin t/2); the inverse passes -s.
template <typename T2, typename Real>
__device__ __forceinline__ T2 mix_el(int kind, T2 own, T2 par, int bit, Real c, Real s, int which) {
    const Real sg = bit ? (Real)1 : (Real)-1;
    switch (kind) {
        case K_H: {
            const Real r = (Real)0.70710678118654752440;
            return mk<T2>((par.x - sg * own.x) * r, (par.y - sg * own.y) * r);
        }
        case K_RX:
            return mk<T2>(c * own.x + s * par.y, c * own.y - s * par.x);
        case K_RY:
            return mk<T2>(c * own.x + sg * s * par.x, c * own.y + sg * s * par.y);
        default:  // K_PAULI
            if (which == 1) return par;
            if (which == 2) return mk<T2>(-sg * par.y, sg * par.x);
            return bit ? mk<T2>(-own.x, -own.y) : own;
    }
}

// This element's term of Im<l | P | p> for the rotation's generator P.
template <typename T2, typename Real>
__device__ __forceinline__ Real grad_el(int kind, T2 l, T2 own, T2 par, int bit) {
    if (kind == K_RX) return l.x * par.y - l.y * par.x;
    if (kind == K_RY) return (bit ? (Real)1 : (Real)-1) * (l.x * par.x + l.y * par.y);
    const Real t = l.x * own.y - l.y * own.x;  // K_RZ
    return bit ? -t : t;
}

// Apply gate g to st (and, when GRAD, return this lane's gradient term taken
// before the gate with l = lambda). Uniform branches only.
template <int R, typename T2, typename Real>
__device__ __forceinline__ void wave_gate(T2* st, const DevGate g, Real c, Real s, int which, int lane) {
    const int q = g.kind == K_CNOT ? g.q1 : g.q0;
    if (g.kind == K_RZ) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const Real sg = amp_bit(q, lane, r) ? (Real)1 : (Real)-1;
            const T2 u = st[r];
            st[r] = mk<T2>(c * u.x - sg * s * u.y, c * u.y + sg * s * u.x);
        }
        return;
    }
    if (g.kind == K_CZ) {
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (amp_bit(g.q0, lane, r) & amp_bit(g.q1, lane, r)) st[r] = mk<T2>(-st[r].x, -st[r].y);
        return;
    }
    if (g.kind == K_PAULI && which == 0) return;
    T2 old[R];
#pragma unroll
    for (int r = 0; r < R; ++r) old[r] = st[r];
    if (q < 6) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const T2 par = xlane(old[r], q, lane);
            if (g.kind == K_CNOT) st[r] = amp_bit(g.q0, lane, r) ? par : old[r];
            else st[r] = mix_el<T2, Real>(g.kind, old[r], par, amp_bit(q, lane, r), c, s, which);
        }
    } else {
        const int m = 1 << (q - 6);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            T2 par = old[r];
            // registers are compile-time indices: pick the partner by a
            // uniform comparison instead of a runtime array index
#pragma unroll
            for (int u = 0; u < R; ++u)
                if (u == (r ^ m)) par = old[u];
            if (g.kind == K_CNOT) st[r] = amp_bit(g.q0, lane, r) ? par : old[r];
            else st[r] = mix_el<T2, Real>(g.kind, old[r], par, (r & m) ? 1 : 0, c, s, which);
        }
    }
}

template <int R, typename T2, typename Real>
__device__ __forceinline__ Real wave_grad(const T2* p, const T2* l, const DevGate g, int lane) {
    const int q = g.q0;
    Real acc = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        T2 par = p[r];
        if (g.kind != K_RZ) {
            if (q < 6) {
                par = xlane(p[r], q, lane);
            } else {
#pragma unroll
                for (int u = 0; u < R; ++u)
                    if (u == (r ^ (1 << (q - 6)))) par = p[u];
            }
        }
        acc += grad_el<T2, Real>(g.kind, l[r], p[r], par, amp_bit(q, lane, r));
    }
    return acc;
}

// Coefficients of gate g for this sample: (c, s) = (cos t/2, sin t/2), or the
// Pauli index of a channel in c.
template <typename T2>
__device__ __forceinline__ T2 gate_coef(const DevGate& g, const T2* coef) {
    return g.slot >= 0 ? coef[g.slot] : mk<T2>((decltype(T2::x))1, (decltype(T2::x))0);
}

// One wavefront (one sample) per workgroup: the sample index is uniform, so
// the gate table and the sample's coefficients are scalar loads, issued one
// gate ahead of their use.
// The gate table and coefficients come in as restrict parameters: the kernel
// writes only outputs, so they stay scalar loads even next to those stores.
template <typename Real, int R>
__global__ void __launch_bounds__(64) k_wave(const WholeArgs a, const DevGate* __restrict__ gates,
                                             const typename Cx<Real>::T* __restrict__ coef_all) {
    using T2 = typename Cx<Real>::T;
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int n = a.n, dim = 1 << n, G = a.n_gates;
    const T2* coef = coef_all + b * a.n_slots;
    T2 ps[R], lm[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int j = lane + 64 * r;
        if (j >= dim) ps[r] = mk<T2>((Real)0, (Real)0);
        else if (a.psi_in) ps[r] = ((const T2*)a.psi_in)[b * dim + j];
        else ps[r] = mk<T2>((Real)(j == 0), (Real)0);
    }
    // gate records two gates ahead, coefficients one ahead: each iteration
    // waits only for loads issued during the previous gate
    auto gate_at = [&](int i) { return gates[__builtin_amdgcn_readfirstlane(i < 0 ? 0 : i < G ? i : G - 1)]; };
    if (G > 0) {
        DevGate g0 = gate_at(0), g1 = gate_at(1);
        T2 c0 = gate_coef(g0, coef);
        for (int gi = 0; gi < G; ++gi) {
            const T2 c1 = gate_coef(g1, coef);
            const DevGate g2 = gate_at(gi + 2);
            wave_gate<R, T2, Real>(ps, g0, c0.x, c0.y, (int)c0.x, lane);
            g0 = g1;
            g1 = g2;
            c0 = c1;
        }
    }
    if (a.psi_out)
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (lane + 64 * r < dim) ((T2*)a.psi_out)[b * dim + lane + 64 * r] = ps[r];
    for (int q = 0; q < n; ++q) {
        Real acc = 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const Real p = ps[r].x * ps[r].x + ps[r].y * ps[r].y;
            acc += amp_bit(q, lane, r) ? -p : p;
        }
        const Real t = wave_to_last(acc);
        if (lane == 63) a.zpart[b * n + q] = (double)t;
    }
    if (!a.bwd) return;
    const Real* go = (const Real*)a.grad_out + b * n;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        Real d = 0;
        for (int q = 0; q < n; ++q) d += amp_bit(q, lane, r) ? -go[q] : go[q];
        lm[r] = mk<T2>(d * ps[r].x, d * ps[r].y);
    }
    if (G > 0) {
        DevGate g0 = gate_at(G - 1), g1 = gate_at(G - 2);
        T2 c0 = gate_coef(g0, coef);
        for (int gi = G - 1; gi >= 0; --gi) {
            const T2 c1 = gate_coef(g1, coef);
            const DevGate g2 = gate_at(gi - 2);
            if (g0.slot >= 0 && g0.kind != K_PAULI) {
                const Real t = wave_to_last(wave_grad<R, T2, Real>(ps, lm, g0, lane));
                if (lane == 63) a.gpart[(size_t)g0.slot * a.B + b] = (double)t;
            }
            wave_gate<R, T2, Real>(ps, g0, c0.x, -c0.y, (int)c0.x, lane);
            wave_gate<R, T2, Real>(lm, g0, c0.x, -c0.y, (int)c0.x, lane);
            g0 = g1;
            g1 = g2;
            c0 = c1;
        }
    }
    if (a.lam_out)
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (lane + 64 * r < dim) ((T2*)a.lam_out)[b * dim + lane + 64 * r] = lm[r];
}

// ---------------------------------------------------------------------------
// k_bind_tile: per-sample op records of every tile op (one thread per
// (sample, op)); shear coefficients in fp64, rounded once. The inverse of a
// rotation (backward ops) negates both coefficients.

template <typename Real>
__global__ void k_bind_tile(const BindTileArgs a) {
    using T2 = typename Cx<Real>::T;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t per = (int64_t)a.n_ops + 1;
    if (t >= a.B * per) return;
    const int64_t b = t / per;
    const int o = (int)(t - b * per);
    XOp<Real> e{};
    if (o == a.n_ops) {  // the record after the last op (read by the op-loop prefetch)
        e.h = H_END;
        ((XOp<Real>*)a.opc)[t] = e;
        return;
    }
    const DevOp op = a.ops[o];
    e.h = op.h;
    e.arg = op.arg;
    if (op.h == H_DZ) {
        // RZ group: the members' gradient slots in the two coefficient words;
        // the forward record also writes the sample's phase table (the
        // backward record reads the same table and applies its inverse)
        const DevDiag d = a.diags[op.arg];
        uint64_t w = 0;
        for (int j = 0; j < MAX_DZ_BITS; ++j) w |= (uint64_t)(d.gslot[j] & 0xffffu) << (16 * j);
        if constexpr (sizeof(Real) == 4) {
            e.a = __builtin_bit_cast(float, (uint32_t)w);
            e.b = __builtin_bit_cast(float, (uint32_t)(w >> 32));
        } else {
            e.a = __builtin_bit_cast(double, w);
        }
        if (o < a.bwd_first) {
            double th[MAX_DZ_BITS];
            for (int j = 0; j < MAX_DZ_BITS; ++j) {
                th[j] = 0.0;
                if (d.slot[j] < 0) continue;
                int64_t bs;
                th[j] = angle_of<Real>(a.inputs, a.weights, a.F, a.slots[d.slot[j]], b, a.v0, a.vper, bs) +
                        shift_of(b, a.v0, a.vper, d.slot[j]);
            }
            T2* tab = (T2*)a.dzc + ((size_t)b * a.n_diags + op.arg) * DZ_REGS;
            for (int i = 0; i < DZ_REGS; ++i) {
                double phi = 0.0;
                for (int j = 0; j < MAX_DZ_BITS; ++j)
                    if (i >> j & 1) phi += th[j];
                double sn, cs;
                sincos(phi, &sn, &cs);
                tab[i] = mk<T2>((Real)cs, (Real)sn);
            }
        }
    } else if (op.kind == K_PAULI) {
        // the Pauli this sample's trajectory draws, on the op's register bit
        const int which = pauli_of<Real>(a.inputs, a.F, a.slots[op.slot], b, a.v0, a.vper);
        e.h = which == 0 ? (uint32_t)H_NOP : op.h + 5u * (uint32_t)(which - 1);
    } else if (op.slot >= 0) {
        const SlotSrc src = a.slots[op.slot];
        int64_t bs;
        double th = angle_of<Real>(a.inputs, a.weights, a.F, src, b, a.v0, a.vper, bs) +
                    shift_of(b, a.v0, a.vper, op.slot);
        const double two_pi = 6.283185307179586476925;
        th -= two_pi * rint(th / two_pi);  // [-pi, pi]; the dropped sign is common to psi and lambda
        if (o >= a.bwd_first) th = -th;     // backward ops apply the inverse
        if (op.h >= H_G1 + 15 && op.h < H_G1 + 20) {
            // RZ on a register bit: phase exp(i phi) on the bit-1 amplitudes,
            // phi = theta moved into [-pi/2, pi/2] (a move by pi negates them)
            const double half_pi = 1.570796326794896619231;
            double phi = th;
            if (phi > half_pi) phi -= 2.0 * half_pi;
            else if (phi < -half_pi) phi += 2.0 * half_pi;
            if (phi != th) e.h = H_RZN + (op.h - (H_G1 + 15));
            e.a = (Real)tan(0.5 * phi);
            e.b = (Real)sin(phi);
        } else {
            // plane rotation by phi = theta/2: a = tan(phi/2), b = sin(phi)
            e.a = (Real)tan(0.25 * th);
            e.b = (Real)sin(0.5 * th);
        }
        if (op.h >= H_RYZ && op.h < H_RYZ + 5) {
            // RY-RZ pair: the RZ's phase, reduced as for a single RZ, from the
            // forward angle in both records (the backward form inverts it);
            // the forward record writes the sample's coefficients
            const uint32_t fi = op.arg >> 16;
            int64_t bz;
            double tz = angle_of<Real>(a.inputs, a.weights, a.F, a.slots[a.fuses[fi].slot], b, a.v0, a.vper, bz) +
                        shift_of(b, a.v0, a.vper, a.fuses[fi].slot);
            tz -= two_pi * rint(tz / two_pi);
            const double half_pi = 1.570796326794896619231;
            double phi = tz;
            if (phi > half_pi) phi -= 2.0 * half_pi;
            else if (phi < -half_pi) phi += 2.0 * half_pi;
            if (phi != tz) e.h = H_RYZN + (op.h - H_RYZ);
            if (o < a.bwd_first)
                ((T2*)a.fzc)[(size_t)b * a.n_fuses + fi] = mk<T2>((Real)tan(0.5 * phi), (Real)sin(phi));
        }
    }
    ((XOp<Real>*)a.opc)[t] = e;
}

// ---------------------------------------------------------------------------
// k_reduce: one wavefront per output element, lanes stride over the partials

template <typename Real>
__global__ void __launch_bounds__(256) k_reduce(const ReduceArgs a) {
    const int64_t e = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    const int64_t nz = a.B * a.n;
    const int64_t nx = (a.grads && a.grad_inputs) ? a.B * a.F : 0;
    const int64_t nw = (a.grads && a.grad_weights) ? a.P : 0;
    double acc = 0;
    if (e < nz) {
        const int64_t b = e / a.n;
        const int q = (int)(e - b * a.n);
        for (int w = lane; w < a.n_wg; w += 64) acc += a.zpart[((size_t)b * a.n_wg + w) * a.n + q];
        acc = wave_sum(acc);
        if (lane == 0) ((Real*)a.expz)[e] = (Real)acc;
    } else if (e < nz + nx) {
        const int64_t u = e - nz;
        const int64_t b = u / a.F;
        const int f = (int)(u - b * a.F);
        for (int i = a.x_ptr[f]; i < a.x_ptr[f + 1]; ++i) {
            const int s = a.x_slot[i];
            const double sc = a.slots[s].scale;
            for (int w = lane; w < a.n_wg; w += 64) acc += sc * a.gpart[((size_t)s * a.B + b) * a.n_wg + w];
        }
        acc = wave_sum(acc);
        if (lane == 0) ((Real*)a.grad_inputs)[u] = (Real)acc;
    } else if (e < nz + nx + nw) {
        const int p = (int)(e - nz - nx);
        const int64_t per = a.B * a.n_wg;
        for (int i = a.w_ptr[p]; i < a.w_ptr[p + 1]; ++i) {
            const double* src = a.gpart + (size_t)a.w_slot[i] * per;
            const double sc = a.slots[a.w_slot[i]].scale;
            for (int64_t j = lane; j < per; j += 64) acc += sc * src[j];
        }
        acc = wave_sum(acc);
        if (lane == 0) ((Real*)a.grad_weights)[p] = (Real)acc;
    }
}

// ---------------------------------------------------------------------------
// parameter shift: per-circuit VJP, then the two-term differences

template <typename Real>
__global__ void __launch_bounds__(256) k_shift_dot(const ShiftDotArgs a) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= a.count) return;
    const int64_t v = a.v0 + i;
    const int64_t b = v / a.vper;
    const Real* e = (const Real*)a.ev + i * a.n;
    const Real* g = (const Real*)a.grad_out + b * a.n;
    double d = 0;
    for (int q = 0; q < a.n; ++q) d += (double)g[q] * (double)e[q];
    a.dv[v] = d;
    if (v - b * a.vper == 0)
        for (int q = 0; q < a.n; ++q) ((Real*)a.expz)[b * a.n + q] = e[q];
}

// One wavefront per output element: input gradient (b, f) or weight p.
template <typename Real>
__global__ void __launch_bounds__(256) k_shift_grad(const ShiftGradArgs a) {
    const int64_t e = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    const int64_t nx = a.grad_inputs ? a.B * a.F : 0;
    const int64_t nw = a.grad_weights ? a.P : 0;
    double acc = 0;
    if (e < nx) {
        const int64_t b = e / a.F;
        const int f = (int)(e - b * a.F);
        const int cnt = a.x_ptr[f + 1] - a.x_ptr[f];
        for (int i = lane; i < cnt; i += 64) {
            const int s = a.x_slot[a.x_ptr[f] + i];
            const double* d = a.dv + b * a.vper;
            acc += a.slots[s].scale * 0.5 * (d[2 * s + 1] - d[2 * s + 2]);
        }
        acc = wave_sum(acc);
        if (lane == 0) ((Real*)a.grad_inputs)[e] = (Real)acc;
    } else if (e < nx + nw) {
        const int p = (int)(e - nx);
        const int cnt = a.w_ptr[p + 1] - a.w_ptr[p];
        const int64_t per = (int64_t)cnt * a.B;
        for (int64_t j = lane; j < per; j += 64) {
            const int64_t b = j / cnt;
            const int s = a.w_slot[a.w_ptr[p] + (int)(j - b * cnt)];
            const double* d = a.dv + b * a.vper;
            acc += a.slots[s].scale * 0.5 * (d[2 * s + 1] - d[2 * s + 2]);
        }
        acc = wave_sum(acc);
        if (lane == 0) ((Real*)a.grad_weights)[p] = (Real)acc;
    }
}

// ---------------------------------------------------------------------------
// exact final states of the tile path
//
// The tile kernel applies each rotation with its angle reduced to [-pi, pi]
// (a factor (-1)^k per rotation whose angle moved by 2 pi k) and an RZ on a
// register bit as diag(1, exp(i t)) (dropping exp(-i t / 2)); both are global
// phases per sample. k_state_phase sums them over the forward ops, from the
// same angle sources and reduction as k_bind_tile and stores the inverse
// phase factor (cos, sin) per sample; k_phase_fix multiplies the state by it.

template <typename Real>
__global__ void k_state_phase(const BindTileArgs a, double* phase) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= a.B) return;
    const double pi = 3.141592653589793238463, two_pi = 2.0 * pi;
    double ph = 0.0;
    int64_t bs;
    for (int o = 0; o < a.bwd_first; ++o) {
        const DevOp op = a.ops[o];
        if (op.h == H_DZ) {  // an RZ group drops exp(-i theta / 2) per member, unreduced
            const DevDiag d = a.diags[op.arg];
            for (int j = 0; j < MAX_DZ_BITS; ++j)
                if (d.slot[j] >= 0)
                    ph += 0.5 * angle_of<Real>(a.inputs, a.weights, a.F, a.slots[d.slot[j]], b, 0, 0, bs);
            continue;
        }
        if (op.slot < 0 || op.kind == K_PAULI) continue;  // Paulis are applied exactly
        const double th = angle_of<Real>(a.inputs, a.weights, a.F, a.slots[op.slot], b, 0, 0, bs);
        const double k = rint(th / two_pi);
        ph += pi * k;
        if (op.h >= H_G1 + 15 && op.h < H_G1 + 20) ph += 0.5 * (th - two_pi * k);
        if (op.h >= H_RYZ && op.h < H_RYZ + 5)  // the pair's RZ, as a single RZ on a register bit
            ph += 0.5 * angle_of<Real>(a.inputs, a.weights, a.F, a.slots[a.fuses[op.arg >> 16].slot], b, 0, 0, bs);
    }
    double sn, cs;  // the inverse phase factor, once per sample
    sincos(-ph, &sn, &cs);
    phase[2 * b] = cs;
    phase[2 * b + 1] = sn;
}

template <typename T2>
__global__ void k_phase_fix(void* psi, const double* phase, int64_t B, int n) {
    const int64_t total = B << n;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const double cs = phase[2 * (i >> n)], sn = phase[2 * (i >> n) + 1];
        T2 v = ((T2*)psi)[i];
        const double x = (double)v.x, y = (double)v.y;
        v.x = (decltype(v.x))(x * cs - y * sn);
        v.y = (decltype(v.y))(x * sn + y * cs);
        ((T2*)psi)[i] = v;
    }
}

// ---------------------------------------------------------------------------
// initial-state embeddings

// Sum of 256 per-thread fp64 values in a fixed tree order (thread 0 returns it).
__device__ __forceinline__ double block_sum256(double v, double* red) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    return red[0];
}

// Per circuit (one 256-thread workgroup each): amplitude embedding |x| of the
// 2^n features, basis embedding the basis index (exact in fp64).
template <typename Real>
__global__ void __launch_bounds__(256) k_embed_norm(const EmbedArgs a) {
    __shared__ double red[256];
    const int64_t i = blockIdx.x;
    const int64_t bs = a.vper > 0 ? (a.v0 + i) / a.vper : i;
    const Real* x = (const Real*)a.inputs + bs * a.F + a.first;
    if (a.kind == E_BASIS) {
        if (threadIdx.x == 0) {
            int64_t idx = 0;
            for (int q = 0; q < a.n; ++q)
                if ((double)x[q] >= 0.5) idx |= (int64_t)1 << q;
            a.norm[i] = (double)idx;
        }
        return;
    }
    const int64_t dim = (int64_t)1 << a.n;
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < dim; j += 256) {
        const double v = (double)x[j];
        acc = fma(v, v, acc);
    }
    const double t = block_sum256(acc, red);
    if (threadIdx.x == 0) a.norm[i] = sqrt(t);
}

// psi_0 of every circuit, grid-stride over count * 2^n amplitudes.
template <typename Real>
__global__ void __launch_bounds__(256) k_embed_write(const EmbedArgs a) {
    using T2 = typename Cx<Real>::T;
    const int64_t dim = (int64_t)1 << a.n, total = a.count << a.n;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = t >> a.n, j = t & (dim - 1);
        const double r = a.norm[i];
        Real re;
        if (a.kind == E_BASIS) {
            re = (Real)(j == (int64_t)r);
        } else {
            const int64_t bs = a.vper > 0 ? (a.v0 + i) / a.vper : i;
            const Real v = ((const Real*)a.inputs)[bs * a.F + a.first + j];
            re = r > 0 ? (Real)((double)v / r) : (Real)0;
        }
        ((T2*)a.psi)[t] = mk<T2>(re, (Real)0);
    }
}

// L_b = sum_j x_j Re lam_j / |x| (one 256-thread workgroup per sample).
template <typename Real>
__global__ void __launch_bounds__(256) k_embed_dot(const EmbedGradArgs a) {
    using T2 = typename Cx<Real>::T;
    __shared__ double red[256];
    const int64_t b = blockIdx.x;
    const int64_t dim = (int64_t)1 << a.n;
    const Real* x = (const Real*)a.inputs + b * a.F + a.first;
    const T2* lam = (const T2*)a.lam + b * dim;
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < dim; j += 256) acc = fma((double)x[j], (double)lam[j].x, acc);
    const double t = block_sum256(acc, red);
    if (threadIdx.x == 0) a.dot[b] = a.norm[b] > 0 ? t / a.norm[b] : 0.0;
}

// grad_inputs[b][first + j] += (2 / |x|) (Re lam_j - (x_j / |x|) L_b).
template <typename Real>
__global__ void __launch_bounds__(256) k_embed_grad(const EmbedGradArgs a) {
    using T2 = typename Cx<Real>::T;
    const int64_t dim = (int64_t)1 << a.n, total = a.B << a.n;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = t >> a.n, j = t & (dim - 1);
        const double r = a.norm[b];
        if (!(r > 0)) continue;
        const double x = (double)((const Real*)a.inputs)[b * a.F + a.first + j];
        const double g = 2.0 / r * ((double)((const T2*)a.lam)[t].x - x / r * a.dot[b]);
        Real* out = (Real*)a.grad_inputs + b * a.F + a.first + j;
        *out = (Real)((double)*out + g);
    }
}

// ---------------------------------------------------------------------------
// shot sampling (inverse CDF). A block of 2^bb amplitudes is 64 lane chunks
// of consecutive amplitudes. The chunk sums are computed once and stored; the
// block totals and the in-block search both lane-scan those stored sums, so
// they see bitwise the same numbers.

// Inclusive scan over the 64 lanes, Hillis-Steele, fixed order.
__device__ __forceinline__ double lane_scan(double v, int lane) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const double t = __shfl_up(v, off, 64);
        if (lane >= off) v += t;
    }
    return v;
}

// Chunk geometry of a block: lane l covers [l * csz, l * csz + cnt_l).
__device__ __forceinline__ void chunk_of(int bb, int lane, int64_t& lo, int64_t& cnt) {
    const int64_t bs = (int64_t)1 << bb;
    const int64_t csz = bs >= 64 ? bs / 64 : 1;
    lo = (int64_t)lane * csz;
    cnt = lo < bs ? csz : 0;
}

// One wavefront per (sample, block): the 64 chunk sums into csum and the
// block total into bsum. The block is read in coalesced rows of 64
// amplitudes; a row holds 64 / csz whole chunks, summed by a butterfly over
// each group of csz lanes (fixed order), and lane c keeps chunk c's sum.
template <typename T2>
__global__ void __launch_bounds__(256) k_block_sums(const SampleArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t stride = (int64_t)gridDim.x * (blockDim.x >> 6);
    for (int64_t wv = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6; wv < a.B * a.nblk; wv += stride) {
        const int64_t b = wv / a.nblk, blk = wv - b * a.nblk;
        const int64_t bs = (int64_t)1 << a.bb;
        const int csz = bs >= 64 ? (int)(bs / 64) : 1, per = 64 / csz;
        const int rows = bs >= 64 ? 64 / per : 1;
        const T2* p = (const T2*)a.psi + (b << a.n) + (blk << a.bb);
        double mine = 0.0;
        for (int k = 0; k < rows; ++k) {
            const int64_t i = lane + 64 * (int64_t)k;
            double q = 0.0;
            if (i < bs) {
                const T2 v = p[i];
                q = (double)v.x * (double)v.x + (double)v.y * (double)v.y;
            }
            for (int off = 1; off < csz; off <<= 1) q += __shfl_xor(q, off, 64);
            const double g = __shfl(q, (lane % per) * csz, 64);
            if (lane / per == k) mine = g;
        }
        a.csum[wv * 64 + lane] = mine;
        const double s = lane_scan(mine, lane);
        if (lane == 63) a.bsum[wv] = s;
    }
}

// One workgroup per sample: inclusive prefix of the block totals, in place,
// fixed order (contiguous thread ranges, then the range offsets in order).
__global__ void __launch_bounds__(256) k_block_scan(const SampleArgs a) {
    __shared__ double off[256];
    const int64_t b = blockIdx.x;
    const int t = threadIdx.x, nt = blockDim.x;
    double* s = a.bsum + b * a.nblk;
    const int64_t per = (a.nblk + nt - 1) / nt;
    const int64_t lo = t * per, hi = lo + per < a.nblk ? lo + per : a.nblk;
    double acc = 0.0;
    for (int64_t i = lo; i < hi; ++i) acc += s[i];
    off[t] = acc;
    __syncthreads();
    if (t == 0) {
        double run = 0.0;
        for (int i = 0; i < nt; ++i) {
            const double v = off[i];
            off[i] = run;
            run += v;
        }
    }
    __syncthreads();
    double run = off[t];
    for (int64_t i = lo; i < hi; ++i) {
        run += s[i];
        s[i] = run;
    }
}

// One wavefront per shot: the block (binary search over the prefix), the lane
// chunk (the block's stored chunk sums, the same lane scan, a ballot), then
// the amplitude (a lane scan of the chunk's probabilities, a ballot). The
// index is the first one whose running total exceeds u * total.
template <typename T2>
__global__ void __launch_bounds__(256) k_shots(const SampleArgs a, const double* __restrict__ pre_all,
                                               const double* __restrict__ cs_all,
                                               const double* __restrict__ uni) {
    // the wavefront's shots, uniform by construction (scalar loads below)
    const int lane = threadIdx.x & 63;
    const int64_t stride = (int64_t)gridDim.x * (blockDim.x >> 6);
    for (int64_t wv = (int64_t)blockIdx.x * (blockDim.x >> 6) +
                      __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
         wv < a.B * a.shots; wv += stride) {
        const int64_t b = wv / a.shots;
        const double* pre = pre_all + b * a.nblk;
        const double total = pre[a.nblk - 1];
        const double r = uni[wv] * total;
        int64_t lo = 0, hi = a.nblk - 1;  // first block with pre > r (pre[nblk-1] = total > r)
        while (lo < hi) {
            const int64_t mid = lo + (hi - lo) / 2;
            if (pre[mid] > r) hi = mid;
            else lo = mid + 1;
        }
        const int64_t blk = lo;
        const double before = blk > 0 ? pre[blk - 1] : 0.0;
        int64_t clo, ccnt;
        chunk_of(a.bb, lane, clo, ccnt);
        const int64_t base = (b << a.n) + (blk << a.bb);
        const T2* p = (const T2*)a.psi;
        const double mine = cs_all[(b * a.nblk + blk) * 64 + lane];  // this lane's chunk sum
        const double incl = lane_scan(mine, lane);
        // shuffle with every lane active, then select (a shuffle inside the
        // conditional would read lane 0 while it is switched off)
        const double up = __shfl_up(incl, 1, 64);
        const double prev = lane > 0 ? up : 0.0;
        const uint64_t hit = __ballot(before + incl > r && ccnt > 0 && mine > 0.0);
        int L = hit ? (int)__builtin_ctzll(hit) : -1;
        if (L < 0) {  // rounding left r above the block: the last chunk of nonzero probability
            const uint64_t has = __ballot(ccnt > 0 && mine > 0.0);
            L = has ? 63 - (int)__builtin_clzll(has) : 63 - (int)__builtin_clzll(__ballot(ccnt > 0));
        }
        const double start = before + __shfl(prev, L, 64);
        int64_t lL, cL;
        chunk_of(a.bb, L, lL, cL);  // cL <= 64: one amplitude per lane
        double q = 0.0;
        if (lane < cL) {
            const T2 v = p[base + lL + lane];
            q = (double)v.x * (double)v.x + (double)v.y * (double)v.y;
        }
        const double run = start + lane_scan(q, lane);
        const uint64_t in = __ballot(lane < cL && run > r && q > 0.0);
        int64_t idx;
        if (in) {
            idx = lL + (int64_t)__builtin_ctzll(in);
        } else {  // rounding: the chunk's last amplitude of nonzero probability
            const uint64_t nz = __ballot(lane < cL && q > 0.0);
            idx = nz ? lL + 63 - (int64_t)__builtin_clzll(nz) : lL;
        }
        if (lane == 0) a.samples[wv] = (blk << a.bb) + idx;
    }
}

// <Z_q> from the shots: one thread per (sample, qubit), exact integer counts.
template <typename Real>
__global__ void __launch_bounds__(256) k_shot_z(const SampleArgs a) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < a.B * a.n; t += stride) {
        const int64_t b = t / a.n;
        const int q = (int)(t - b * a.n);
        int64_t ones = 0;
        for (int64_t s = 0; s < a.shots; ++s) ones += (a.samples[b * a.shots + s] >> q) & 1;
        ((Real*)a.zhat)[t] = a.shots > 0 ? (Real)((double)(a.shots - 2 * ones) / (double)a.shots) : (Real)0;
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers

hipError_t launch_bind(int dtype, const BindArgs& a, hipStream_t s) {
    const int64_t total = a.B * a.n_slots;
    if (total == 0) return hipSuccess;
    const unsigned grid = (unsigned)((total + 255) / 256);
    if (dtype == 0) hipLaunchKernelGGL(k_bind<float>, dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_bind<double>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

// Circuits per launch from which a forward-only whole-state launch of n <= 8
// qubits takes the LDS kernel: with that many wavefronts in flight its LDS
// partner exchanges outrun k_wave's DPP and permlane ones (parameter-shift
// chunks of the 7-qubit autoencoder: 0.53 against 0.72 ms at 49408 circuits,
// 1.56 against 1.78 ms at 2048, even at 512).
constexpr int64_t WAVE_MAX_FWD_CIRCUITS = 2048;

hipError_t launch_whole(int dtype, const WholeArgs& a, int threads, size_t lds, hipStream_t s) {
    if (a.n <= 8 && (a.bwd || a.B < WAVE_MAX_FWD_CIRCUITS)) {  // one wavefront per sample
        const dim3 grid((unsigned)a.B), block(64);
#define QL_WAVE(REAL)                                                                     \
    {                                                                                     \
        const auto* cf = (const typename Cx<REAL>::T*)a.coef;                             \
        if (a.n <= 6) hipLaunchKernelGGL((k_wave<REAL, 1>), grid, block, 0, s, a, a.gates, cf);      \
        else if (a.n == 7) hipLaunchKernelGGL((k_wave<REAL, 2>), grid, block, 0, s, a, a.gates, cf); \
        else hipLaunchKernelGGL((k_wave<REAL, 4>), grid, block, 0, s, a, a.gates, cf);               \
    }
        if (dtype == 0) {
            QL_WAVE(float)
        } else {
            QL_WAVE(double)
        }
#undef QL_WAVE
        return hipGetLastError();
    }
    if (dtype == 0) hipLaunchKernelGGL(k_whole<float>, dim3((unsigned)a.B), dim3(threads), lds, s, a);
    else hipLaunchKernelGGL(k_whole<double>, dim3((unsigned)a.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

template <typename Real, int LOG_R, int MAXT>
static hipError_t launch_tile_t(bool bwd, const TileArgs& a, int threads, size_t lds, hipStream_t s) {
    const dim3 grid((unsigned)(a.B * a.n_wg));
    const XOp<Real>* xo = (const XOp<Real>*)a.opc;
    const Real* gout = (const Real*)a.grad_out;
    const typename Cx<Real>::T* dzt = (const typename Cx<Real>::T*)a.dzc;
    const typename Cx<Real>::T* fzt = (const typename Cx<Real>::T*)a.fzc;
    if (bwd)
        hipLaunchKernelGGL((k_tile<Real, LOG_R, KM_BWD, MAXT>), grid, dim3(threads), lds, s, a, a.pass,
                           a.phases, xo, gout, a.gslots, dzt, fzt);
    else if (a.tiles >= 2)  // forward passes carry two tiles per iteration when there are two
        hipLaunchKernelGGL((k_tile<Real, LOG_R, KM_FWD2, MAXT>), grid, dim3(threads), lds, s, a, a.pass,
                           a.phases, xo, gout, a.gslots, dzt, fzt);
    else
        hipLaunchKernelGGL((k_tile<Real, LOG_R, KM_FWD1, MAXT>), grid, dim3(threads), lds, s, a, a.pass,
                           a.phases, xo, gout, a.gslots, dzt, fzt);
    return hipGetLastError();
}

hipError_t launch_bind_tile(int dtype, const BindTileArgs& a, hipStream_t s) {
    const int64_t total = a.B * ((int64_t)a.n_ops + 1);
    const unsigned grid = (unsigned)((total + 255) / 256);
    if (dtype == 0) hipLaunchKernelGGL(k_bind_tile<float>, dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_bind_tile<double>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_tile(int dtype, int log_r, bool bwd, const TileArgs& a, int threads, size_t lds,
                       hipStream_t s) {
    const bool big = threads > 256;
#define QL_LT(REAL, LR)                                                                   \
    return big ? launch_tile_t<REAL, LR, 512>(bwd, a, threads, lds, s)                    \
               : launch_tile_t<REAL, LR, 256>(bwd, a, threads, lds, s);
    if (dtype == 0) {
        switch (log_r) {
            case 2: QL_LT(float, 2)
            case 3: QL_LT(float, 3)
            case 4: QL_LT(float, 4)
            case 5: QL_LT(float, 5)
        }
    } else {
        switch (log_r) {
            case 2: QL_LT(double, 2)
            case 3: QL_LT(double, 3)
            case 4: QL_LT(double, 4)
        }
    }
#undef QL_LT
    return hipErrorInvalidValue;
}

hipError_t launch_reduce(int dtype, const ReduceArgs& a, hipStream_t s) {
    const int64_t nz = a.B * a.n;
    const int64_t nx = (a.grads && a.grad_inputs) ? a.B * a.F : 0;
    const int64_t nw = (a.grads && a.grad_weights) ? a.P : 0;
    const int64_t waves = nz + nx + nw;
    if (waves == 0) return hipSuccess;
    const unsigned grid = (unsigned)((waves + 3) / 4);
    if (dtype == 0) hipLaunchKernelGGL(k_reduce<float>, dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_reduce<double>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

size_t tile_static_lds(int dtype, int log_r, int threads) {
    const size_t maxt = threads > 256 ? 512 : 256;
    return maxt * ((size_t)1 << log_r) * 2 * (dtype == 0 ? sizeof(float) : sizeof(double));
}

hipError_t launch_shift_dot(int dtype, const ShiftDotArgs& a, hipStream_t s) {
    if (a.count == 0) return hipSuccess;
    const unsigned grid = (unsigned)((a.count + 255) / 256);
    if (dtype == 0) hipLaunchKernelGGL(k_shift_dot<float>, dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_shift_dot<double>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_embed(int dtype, const EmbedArgs& a, hipStream_t s) {
    if (a.count <= 0) return hipSuccess;
    const int64_t total = a.count << a.n;
    const int grid = (int)std::min<int64_t>((total + 255) / 256, 65536);
    if (dtype == 0) {
        hipLaunchKernelGGL(k_embed_norm<float>, dim3((unsigned)a.count), dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_embed_write<float>, dim3(grid), dim3(256), 0, s, a);
    } else {
        hipLaunchKernelGGL(k_embed_norm<double>, dim3((unsigned)a.count), dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_embed_write<double>, dim3(grid), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_embed_grad(int dtype, const EmbedGradArgs& a, hipStream_t s) {
    if (a.B <= 0) return hipSuccess;
    const int64_t total = a.B << a.n;
    const int grid = (int)std::min<int64_t>((total + 255) / 256, 65536);
    if (dtype == 0) {
        hipLaunchKernelGGL(k_embed_dot<float>, dim3((unsigned)a.B), dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_embed_grad<float>, dim3(grid), dim3(256), 0, s, a);
    } else {
        hipLaunchKernelGGL(k_embed_dot<double>, dim3((unsigned)a.B), dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_embed_grad<double>, dim3(grid), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_shift_grad(int dtype, const ShiftGradArgs& a, hipStream_t s) {
    const int64_t waves = (a.grad_inputs ? a.B * a.F : 0) + (a.grad_weights ? a.P : 0);
    if (waves == 0) return hipSuccess;
    const unsigned grid = (unsigned)((waves + 3) / 4);
    if (dtype == 0) hipLaunchKernelGGL(k_shift_grad<float>, dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_shift_grad<double>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_state_phase(int dtype, const BindTileArgs& a, double* phase, void* psi, int n,
                              hipStream_t s) {
    const unsigned g1 = (unsigned)((a.B + 255) / 256);
    const int64_t total = a.B << n;
    const unsigned g2 = (unsigned)std::min<int64_t>((total + 255) / 256, 65536);
    if (dtype == 0) {
        hipLaunchKernelGGL(k_state_phase<float>, dim3(g1), dim3(256), 0, s, a, phase);
        hipLaunchKernelGGL(k_phase_fix<float2>, dim3(g2), dim3(256), 0, s, psi, (const double*)phase, a.B, n);
    } else {
        hipLaunchKernelGGL(k_state_phase<double>, dim3(g1), dim3(256), 0, s, a, phase);
        hipLaunchKernelGGL(k_phase_fix<double2>, dim3(g2), dim3(256), 0, s, psi, (const double*)phase, a.B, n);
    }
    return hipGetLastError();
}

// Workgroups of 256 threads for `items` work items of `per_block` per
// workgroup, capped (the sampling kernels stride over the rest).
static unsigned sample_grid(int64_t items, int64_t per_block) {
    const int64_t g = (items + per_block - 1) / per_block;
    return (unsigned)std::max<int64_t>(1, std::min<int64_t>(g, (int64_t)1 << 20));
}

hipError_t launch_sample(int dtype, const SampleArgs& a, hipStream_t s) {
    const int64_t wb = a.B * a.nblk, ws = a.B * a.shots;
    hipError_t e;
    if (dtype == 0) hipLaunchKernelGGL(k_block_sums<float2>, dim3(sample_grid(wb, 4)), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_block_sums<double2>, dim3(sample_grid(wb, 4)), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_block_scan, dim3((unsigned)a.B), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ws > 0) {
        if (dtype == 0)
            hipLaunchKernelGGL(k_shots<float2>, dim3(sample_grid(ws, 4)), dim3(256), 0, s, a, a.bsum, a.csum,
                               a.uniforms);
        else
            hipLaunchKernelGGL(k_shots<double2>, dim3(sample_grid(ws, 4)), dim3(256), 0, s, a, a.bsum, a.csum,
                               a.uniforms);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (a.zhat) {
        const int64_t t = a.B * a.n;
        if (dtype == 0) hipLaunchKernelGGL(k_shot_z<float>, dim3(sample_grid(t, 256)), dim3(256), 0, s, a);
        else hipLaunchKernelGGL(k_shot_z<double>, dim3(sample_grid(t, 256)), dim3(256), 0, s, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t configure_kernels(size_t max_lds) {
    hipError_t e = hipSuccess;
#define QL_ATTR_V(fn, v)                                                                 \
    if (e == hipSuccess)                                                                 \
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),                       \
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)(v));
#define QL_ATTR(fn) QL_ATTR_V(fn, max_lds)
    QL_ATTR((k_whole<float>))
    QL_ATTR((k_whole<double>))
    // tile kernels: what the static exchange buffer leaves
#define QL_ATTR_TK(REAL, LR, BW, MT)                                                      \
    {                                                                                     \
        const size_t st = tile_lds_bytes<REAL, LR, MT>();                                 \
        if (st < max_lds) QL_ATTR_V((k_tile<REAL, LR, BW, MT>), max_lds - st)             \
    }
#define QL_ATTR_T(REAL, LR)                                                               \
    QL_ATTR_TK(REAL, LR, KM_FWD1, 256) QL_ATTR_TK(REAL, LR, KM_FWD2, 256)                  \
    QL_ATTR_TK(REAL, LR, KM_BWD, 256) QL_ATTR_TK(REAL, LR, KM_FWD1, 512)                   \
    QL_ATTR_TK(REAL, LR, KM_FWD2, 512) QL_ATTR_TK(REAL, LR, KM_BWD, 512)
    QL_ATTR_T(float, 2)
    QL_ATTR_T(float, 3)
    QL_ATTR_T(float, 4)
    QL_ATTR_T(float, 5)
    QL_ATTR_T(double, 2)
    QL_ATTR_T(double, 3)
    QL_ATTR_T(double, 4)
#undef QL_ATTR_T
#undef QL_ATTR_TK
#undef QL_ATTR
#undef QL_ATTR_V
    return e;
}

}  // namespace qlayer
