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
//   k_tile   -- (tile.hip) one tile pass over every sample: each workgroup
//               streams 2^k amplitudes (a tile) from HBM into registers,
//               applies the pass's gates there (LDS only to change which tile
//               bits sit in registers), and streams them back; the backward
//               variant carries psi and lambda and accumulates Im<lambda|P|psi>
//               per rotation
//   k_reduce -- deterministic fp64 sums of the per-workgroup partials into
//               <Z_q>, input gradients and (batch-summed) weight gradients
//   k_wave   -- states of n <= 8 qubits: one wavefront per sample holds psi and
//               lambda in registers (same job as k_whole, no LDS, no barriers)
//   k_bind_tile -- per-sample op records of the tile ops (handler, argument,
//               shear coefficients; the Pauli of a channel trajectory)
//   k_embed_* -- basis / amplitude embedding of the initial state, and the
//               amplitude embedding's VJP from lambda_0
//   k_shift_dot, k_shift_grad -- parameter-shift VJP from batched shifted circuits
//   k_bind_prefix, k_env, k_env_grad -- the product-state prefix: per-sample
//               factors of the first pass's initial state, the environment sums
//               of lambda at the end of the backward sweep, and the prefix
//               gates' gradient terms
//   k_state_phase, k_phase_fix -- the global phase of the tile path's final states
//   k_block_sums, k_block_scan, k_shots, k_shot_z -- shot sampling by inverse CDF
#include "kcommon.hpp"

namespace qlayer {
namespace {

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

// Handler id of a gate for the one-wavefront kernel: one-qubit kinds (H, RX,
// RY, RZ, Pauli) 8 * kind + q, CNOT 40 + 8 c + t, CZ 104 + 8 a + b (a < b).
// Each id is a case of wave_op whose gate is a compile-time constant, so the
// lane and register choices of wave_gate and wave_grad fold away.
__device__ __forceinline__ int wave_handler(const DevGate& g) {
    if (g.kind == K_CNOT) return 40 + 8 * g.q0 + g.q1;
    if (g.kind == K_CZ) return 104 + 8 * min(g.q0, g.q1) + max(g.q0, g.q1);
    return 8 * (g.kind == K_PAULI ? 4 : g.kind) + g.q0;
}

// BWD = false: the gate on ps. BWD = true: when `want`, this lane's term of
// the gradient (before the gate) into *grad, then the inverse on ps and lm.
template <int R, bool BWD, typename T2, typename Real>
__device__ __forceinline__ void wave_op(int h, T2* ps, T2* lm, Real c, Real s, int which, int lane, Real* grad,
                                        bool want) {
    constexpr int NQ = R == 1 ? 6 : R == 2 ? 7 : 8;  // qubits a sample's registers hold
#define QL_W(H, KIND, Q0, Q1)                                                             \
    case H:                                                                               \
        if constexpr (Q0 < NQ && Q1 < NQ && Q0 != Q1) {                                   \
            constexpr DevGate g{KIND, Q0, Q1, 0};                                         \
            if constexpr (BWD) {                                                          \
                if (want) *grad = wave_grad<R, T2, Real>(ps, lm, g, lane);                \
                wave_gate<R, T2, Real>(ps, g, c, -s, which, lane);                        \
                wave_gate<R, T2, Real>(lm, g, c, -s, which, lane);                        \
            } else {                                                                      \
                wave_gate<R, T2, Real>(ps, g, c, s, which, lane);                         \
            }                                                                             \
        }                                                                                 \
        break;
#define QL_W1(Q)                                                                          \
    QL_W(Q, K_H, Q, -1) QL_W(8 + Q, K_RX, Q, -1) QL_W(16 + Q, K_RY, Q, -1)                 \
    QL_W(24 + Q, K_RZ, Q, -1) QL_W(32 + Q, K_PAULI, Q, -1)
#define QL_W2(BASE, KIND, A)                                                              \
    QL_W(BASE + 8 * A + 0, KIND, A, 0) QL_W(BASE + 8 * A + 1, KIND, A, 1)                 \
    QL_W(BASE + 8 * A + 2, KIND, A, 2) QL_W(BASE + 8 * A + 3, KIND, A, 3)                 \
    QL_W(BASE + 8 * A + 4, KIND, A, 4) QL_W(BASE + 8 * A + 5, KIND, A, 5)                 \
    QL_W(BASE + 8 * A + 6, KIND, A, 6) QL_W(BASE + 8 * A + 7, KIND, A, 7)
    switch (h) {
        QL_W1(0) QL_W1(1) QL_W1(2) QL_W1(3) QL_W1(4) QL_W1(5) QL_W1(6) QL_W1(7)
        QL_W2(40, K_CNOT, 0) QL_W2(40, K_CNOT, 1) QL_W2(40, K_CNOT, 2) QL_W2(40, K_CNOT, 3)
        QL_W2(40, K_CNOT, 4) QL_W2(40, K_CNOT, 5) QL_W2(40, K_CNOT, 6) QL_W2(40, K_CNOT, 7)
        QL_W2(104, K_CZ, 0) QL_W2(104, K_CZ, 1) QL_W2(104, K_CZ, 2) QL_W2(104, K_CZ, 3)
        QL_W2(104, K_CZ, 4) QL_W2(104, K_CZ, 5) QL_W2(104, K_CZ, 6) QL_W2(104, K_CZ, 7)
        default:
            break;
    }
#undef QL_W
#undef QL_W1
#undef QL_W2
}

// Up to 64 consecutive gates held by the lanes of a wavefront: lane i holds
// gate base + i (its handler id, slot and kind) and this sample's (cos t/2,
// sin t/2) of its angle (a Pauli channel: the Pauli's index in c), bound in
// fp64 as k_bind does. The gate loop then reads them with readlane: no
// memory access per gate.
template <typename Real>
struct WaveChunk {
    int h, slot, kind;
    Real c, s;
};

template <typename Real>
__device__ __forceinline__ WaveChunk<Real> wave_chunk(const WholeArgs& a, const DevGate* __restrict__ gates,
                                                      int base, int lane, int64_t b) {
    WaveChunk<Real> w{0, -1, K_H, (Real)1, (Real)0};
    const int i = base + lane;
    if (i >= a.n_gates) return w;
    const DevGate g = gates[i];
    w.h = wave_handler(g);
    w.slot = g.slot;
    w.kind = g.kind;
    if (g.slot < 0) return w;
    const SlotSrc src = a.slots[g.slot];
    if (src.src == S_PAULI) {
        w.c = (Real)pauli_of<Real>(a.inputs, a.F, src, b, a.v0, a.vper);
        return w;
    }
    int64_t bs = b;
    const double th = angle_of<Real>(a.inputs, a.weights, a.F, src, b, a.v0, a.vper, bs) +
                      shift_of(b, a.v0, a.vper, g.slot);
    double sn, cs;
    sincos(0.5 * th, &sn, &cs);
    w.c = (Real)cs;
    w.s = (Real)sn;
    return w;
}

__device__ __forceinline__ int rl(int v, int i) { return __builtin_amdgcn_readlane(v, i); }
__device__ __forceinline__ float rl(float v, int i) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), i));
}
__device__ __forceinline__ double rl(double v, int i) {
    const long long u = __builtin_bit_cast(long long, v);
    const int lo = __builtin_amdgcn_readlane((int)(u & 0xffffffff), i);
    const int hi = __builtin_amdgcn_readlane((int)(u >> 32), i);
    return __builtin_bit_cast(double, ((long long)hi << 32) | (unsigned int)lo);
}

// One wavefront (one sample) per workgroup. The gates stream through the
// lanes 64 at a time (wave_chunk): the forward walks the chunks in order, the
// backward in reverse (a circuit of at most 64 gates keeps its one chunk).
template <typename Real, int R>
__global__ void __launch_bounds__(64) k_wave(const WholeArgs a, const DevGate* __restrict__ gates) {
    using T2 = typename Cx<Real>::T;
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int n = a.n, dim = 1 << n, G = a.n_gates;
    T2 ps[R], lm[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int j = lane + 64 * r;
        if (j >= dim) ps[r] = mk<T2>((Real)0, (Real)0);
        else if (a.psi_in) ps[r] = ((const T2*)a.psi_in)[b * dim + j];
        else ps[r] = mk<T2>((Real)(j == 0), (Real)0);
    }
    WaveChunk<Real> ch{};
    int loaded = -1;  // base of the chunk in `ch`
    for (int base = 0; base < G; base += 64) {
        ch = wave_chunk<Real>(a, gates, base, lane, b);
        loaded = base;
        const int cnt = min(64, G - base);
        for (int i = 0; i < cnt; ++i) {
            const Real c = rl(ch.c, i);
            wave_op<R, false, T2, Real>(rl(ch.h, i), ps, lm, c, rl(ch.s, i), (int)c, lane, nullptr, false);
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
    for (int base = G > 0 ? ((G - 1) / 64) * 64 : -64; base >= 0; base -= 64) {
        if (base != loaded) {
            ch = wave_chunk<Real>(a, gates, base, lane, b);
            loaded = base;
        }
        for (int i = min(64, G - base) - 1; i >= 0; --i) {
            const int slot = rl(ch.slot, i);
            const bool want = slot >= 0 && rl(ch.kind, i) != K_PAULI;
            const Real c = rl(ch.c, i);
            Real part = 0;
            wave_op<R, true, T2, Real>(rl(ch.h, i), ps, lm, c, rl(ch.s, i), (int)c, lane, &part, want);
            if (want) {
                const Real t = wave_to_last(part);
                if (lane == 63) a.gpart[(size_t)slot * a.B + b] = (double)t;
            }
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
// product-state prefix
//
// The one-qubit gates a qubit meets before anything entangles it (its prefix)
// act on |0> independently per qubit, so the circuit's first pass starts from
// the product of the per-qubit states phi_q = G_m ... G_1 |0> (k_bind_prefix,
// fp64). Their gradients need no pass either: with lambda_P the adjoint state
// at the end of the prefix and rest the product of the other qubits' factors,
// the term of gate j of qubit q is Im <lambda_j| P_j |psi_j> = Im <r_q|
// A_j P_j B_j |0>, where B_j = G_j ... G_1, A_j = G_m ... G_{j+1} and r_q(v) =
// sum over amplitudes i with bit q = v of lambda_P(i) conj(rest(i)). The last
// backward pass stores lambda_P; k_env forms every workgroup's share of all
// r_q in one read of it, and k_env_grad sums the shares and evaluates the
// terms.

__device__ __forceinline__ double2 zmul(double2 a, double2 b) {
    return make_double2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}

// v <- G v for prefix gate kind k with angle t (G = exp(-i t P / 2) for RX,
// RY, RZ; the Hadamard for H); inv applies G^dagger.
__device__ __forceinline__ void apply_gate1(int kind, double t, bool inv, double2& v0, double2& v1) {
    if (kind == K_H) {
        const double r = 0.70710678118654752440;
        const double2 a = v0, b = v1;
        v0 = make_double2(r * (a.x + b.x), r * (a.y + b.y));
        v1 = make_double2(r * (a.x - b.x), r * (a.y - b.y));
        return;
    }
    if (inv) t = -t;
    double s, c;
    sincos(0.5 * t, &s, &c);
    const double2 a = v0, b = v1;
    if (kind == K_RX) {  // [[c, -i s], [-i s, c]]
        v0 = make_double2(c * a.x + s * b.y, c * a.y - s * b.x);
        v1 = make_double2(s * a.y + c * b.x, -s * a.x + c * b.y);
    } else if (kind == K_RY) {  // [[c, -s], [s, c]]
        v0 = make_double2(c * a.x - s * b.x, c * a.y - s * b.y);
        v1 = make_double2(s * a.x + c * b.x, s * a.y + c * b.y);
    } else {  // RZ: diag(exp(-i t/2), exp(i t/2))
        v0 = zmul(a, make_double2(c, -s));
        v1 = zmul(b, make_double2(c, s));
    }
}

// One thread per (circuit, qubit): the qubit's prefix factor.
template <typename Real>
__global__ void __launch_bounds__(256) k_bind_prefix(const PrefixArgs a) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= a.B * a.n) return;
    const int64_t b = t / a.n;
    const int q = (int)(t - b * a.n);
    double2 v0 = make_double2(1.0, 0.0), v1 = make_double2(0.0, 0.0);
    for (int i = a.pre_ptr[q]; i < a.pre_ptr[q + 1]; ++i) {
        const DevPrefix g = a.pre_ops[i];
        double th = 0.0;
        if (g.slot >= 0) {
            int64_t bs;
            th = angle_of<Real>(a.inputs, a.weights, a.F, a.slots[g.slot], b, a.v0, a.vper, bs) +
                 shift_of(b, a.v0, a.vper, g.slot);
        }
        apply_gate1(g.kind, th, false, v0, v1);
    }
    double2* out = (double2*)a.phi + 2 * t;
    out[0] = v0;
    out[1] = v1;
}

// Environment sums of the prefix: 256 threads (4 wavefronts) per workgroup;
// a wavefront takes blocks of 64 * 2^LR consecutive amplitudes of lambda_P,
// so register bit m is qubit m, lane bit t qubit LR + t, and the block index
// holds the other (fixed) qubits. A wavefront's blocks are blk0 + k * stride
// (stride a power of two): their fixed bits below lo = log2(stride) are
// blk0's, the h = nfix - lo bits above are k's (at most ENV_HIGH_BITS, by the
// launch). Per block and thread the register bits are contracted (Real, leave-
// one-out); the shares of the register and lane qubits are sums over the
// blocks of conj(the block's fixed factors) times the contractions (Real, in
// registers), with each lane's constant factors applied once at the end. The
// fixed qubits need the block's wavefront sum U(k) of the lane-weighted
// contraction (fp64), kept in an LDS table, whose leave-one-out contractions
// over k's bits give them at the end. The wavefront sums (fp64) go to LDS and
// the four wavefronts are combined in a fixed order.
constexpr int ENV_HIGH_BITS = 8;
template <typename Real, int LR>
__global__ void __launch_bounds__(256) k_env(const PrefixArgs a) {
    using T2 = typename Cx<Real>::T;
    constexpr int R = 1 << LR, KMAX = 1 << ENV_HIGH_BITS;
    __shared__ double acc[4][32][4];
    __shared__ double2 ut[4][KMAX];  // per wavefront: U(k) of its blocks
    __shared__ double2 tab[4][32];   // per wavefront: products of the high fixed factors of
                                     // k's low four bits [0, 16) and of its other bits [16, 32)
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int n = a.n;
    const int64_t b = blockIdx.x / a.env_wg;
    const int w = (int)(blockIdx.x - b * a.env_wg);
    for (int i = tid; i < 4 * 32 * 4; i += 256) (&acc[0][0][0])[i] = 0.0;
    for (int i = tid; i < 4 * KMAX; i += 256) (&ut[0][0])[i] = make_double2(0.0, 0.0);
    const double2* fac = (const double2*)a.phi + b * 2 * n;
    const T2* lam = (const T2*)a.lam + (b << n);
    const int nfix = n - LR - 6;
    const int64_t nblk = (int64_t)1 << nfix;
    const int64_t blk0 = (int64_t)w * 4 + wave, stride = (int64_t)a.env_wg * 4;
    const int lo = std::min(nfix, (int)__builtin_ctzll((unsigned long long)stride));
    const int h = nfix - lo, ha = std::min(h, 4), hb = h - ha;
    auto ffac = [&](int i, int64_t bit) { return fac[2 * (LR + 6 + i) + (int)bit]; };  // fixed qubit i
    if (lane < 32) {
        const int e = lane & 15, base = lane < 16 ? 0 : ha, cnt = lane < 16 ? ha : hb;
        double2 p = make_double2(1.0, 0.0);
        for (int j = 0; j < cnt; ++j) p = cxmul(p, ffac(lo + base + j, (e >> j) & 1));
        tab[wave][lane] = p;
    }
    __syncthreads();
    T2 f0[LR], f1[LR];
#pragma unroll
    for (int m = 0; m < LR; ++m) {
        f0[m] = to_real<T2, Real>(fac[2 * m]);
        f1[m] = to_real<T2, Real>(fac[2 * m + 1]);
    }
    // the lane's factors: all six (cl) and all but lane bit t (lf[t])
    double2 cl = make_double2(1.0, 0.0);
    T2 lf[6];
#pragma unroll
    for (int t = 0; t < 6; ++t) {
        double2 p = make_double2(1.0, 0.0);
#pragma unroll
        for (int t2 = 0; t2 < 6; ++t2)
            if (t2 != t) p = cxmul(p, fac[2 * (LR + t2) + ((lane >> t2) & 1)]);
        lf[t] = to_real<T2, Real>(p);
        cl = t == 0 ? fac[2 * LR + (lane & 1)] : cxmul(cl, fac[2 * (LR + t) + ((lane >> t) & 1)]);
    }
    const T2 clr = to_real<T2, Real>(cl);
    // the low fixed factors: all (clo) and all but this lane's (glo, lane < lo)
    double2 clo = make_double2(1.0, 0.0), glo = make_double2(1.0, 0.0);
    for (int i = 0; i < lo; ++i) {
        const double2 f = ffac(i, (blk0 >> i) & 1);
        clo = cxmul(clo, f);
        if (i != lane) glo = cxmul(glo, f);
    }
    Real sr[LR][4], wx = 0, wy = 0;  // sums over the blocks: conj(cf) S[m][u]; conj(cf) T
#pragma unroll
    for (int m = 0; m < LR; ++m)
#pragma unroll
        for (int c = 0; c < 4; ++c) sr[m][c] = 0;
    for (int64_t blk = blk0; blk < nblk; blk += stride) {
        T2 v[R];
        const T2* src = lam + (blk << (LR + 6)) + ((int64_t)lane << LR);
#pragma unroll
        for (int i = 0; i < R; ++i) v[i] = src[i];
        T2 S[LR][2];
        loo_contract<0, LR, T2>(v, f0, f1, S);
        const T2 T = [&] {
            const T2 x = cxmulc(f0[0], S[0][0]), y = cxmulc(f1[0], S[0][1]);
            return mk<T2>(x.x + y.x, x.y + y.y);
        }();
        const int k = (int)(blk >> lo);
        const T2 cf = to_real<T2, Real>(cxmul(clo, cxmul(tab[wave][k & 15], tab[wave][16 + (k >> 4)])));
#pragma unroll
        for (int m = 0; m < LR; ++m) {
            const T2 s0 = cxmulc(cf, S[m][0]), s1 = cxmulc(cf, S[m][1]);
            sr[m][0] += s0.x;
            sr[m][1] += s0.y;
            sr[m][2] += s1.x;
            sr[m][3] += s1.y;
        }
        const T2 x = cxmulc(cf, T);
        wx += x.x;
        wy += x.y;
        const T2 uu = cxmulc(clr, T);
        const double ux = wave_total(uu.x), uy = wave_total(uu.y);
        if (lane == 0) ut[wave][k] = make_double2(ux, uy);
    }
    // register qubits: conj(cl) times the sums
#pragma unroll
    for (int m = 0; m < LR; ++m) {
        const T2 s0 = cxmulc(clr, mk<T2>(sr[m][0], sr[m][1])), s1 = cxmulc(clr, mk<T2>(sr[m][2], sr[m][3]));
        const Real q[4] = {s0.x, s0.y, s1.x, s1.y};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const double t = wave_total(q[c]);
            if (lane == 0) acc[wave][m][c] = t;
        }
    }
    // lane qubits: conj(every lane factor but t's) times the sum, in the bin of
    // the lane's bit t
#pragma unroll
    for (int t = 0; t < 6; ++t) {
        const T2 x = cxmulc(lf[t], mk<T2>(wx, wy));
        const bool one = (lane >> t) & 1;
        const Real q[4] = {one ? (Real)0 : x.x, one ? (Real)0 : x.y, one ? x.x : (Real)0, one ? x.y : (Real)0};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const double s = wave_total(q[c]);
            if (lane == 0) acc[wave][LR + t][c] = s;
        }
    }
    __syncthreads();  // the U table of each wavefront is complete
    // fixed qubits above lo (bit j of k): U contracted with conj(the low and
    // the other high factors), in the bin of bit j
    const int K = 1 << h;
    for (int j = 0; j < h; ++j) {
        double r[4] = {0.0, 0.0, 0.0, 0.0};
        for (int k = lane; k < K; k += 64) {
            double2 p = clo;
            for (int j2 = 0; j2 < h; ++j2)
                if (j2 != j) p = cxmul(p, ffac(lo + j2, (k >> j2) & 1));
            const double2 x = cxmulc(p, ut[wave][k]);
            const bool one = (k >> j) & 1;
            r[0] += one ? 0.0 : x.x;
            r[1] += one ? 0.0 : x.y;
            r[2] += one ? x.x : 0.0;
            r[3] += one ? x.y : 0.0;
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const double t = wave_total(r[c]);
            if (lane == 0) acc[wave][LR + 6 + lo + j][c] = t;
        }
    }
    // fixed qubits below lo (bit i of blk0 in every block): the whole table
    // contracted with conj(the high factors), times conj(the other low factors)
    if (lo > 0) {
        double fx = 0.0, fy = 0.0;
        for (int k = lane; k < K; k += 64) {
            double2 p = make_double2(1.0, 0.0);
            for (int j2 = 0; j2 < h; ++j2) p = cxmul(p, ffac(lo + j2, (k >> j2) & 1));
            const double2 x = cxmulc(p, ut[wave][k]);
            fx += x.x;
            fy += x.y;
        }
        const double2 F = make_double2(wave_total(fx), wave_total(fy));
        if (lane < lo) {
            const double2 r = cxmulc(glo, F);
            const bool one = (blk0 >> lane) & 1;
            acc[wave][LR + 6 + lane][0] = one ? 0.0 : r.x;
            acc[wave][LR + 6 + lane][1] = one ? 0.0 : r.y;
            acc[wave][LR + 6 + lane][2] = one ? r.x : 0.0;
            acc[wave][LR + 6 + lane][3] = one ? r.y : 0.0;
        }
    }
    __syncthreads();
    double* dst = a.envpart + ((size_t)b * a.env_wg + w) * n * 4;
    for (int i = tid; i < n * 4; i += 256) {
        const double* p = &acc[0][0][0] + i;
        dst[i] = ((p[0] + p[32 * 4]) + p[2 * 32 * 4]) + p[3 * 32 * 4];
    }
}

// One wavefront per (sample, qubit): r_q from the workgroups' environment
// sums in a fixed order, then the gradient term of every prefix rotation of q.
template <typename Real>
__global__ void __launch_bounds__(256) k_env_grad(const PrefixArgs a) {
    const int64_t e = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    if (e >= a.B * a.n) return;
    const int64_t b = e / a.n;
    const int q = (int)(e - b * a.n);
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int64_t t = lane; t < a.env_wg; t += 64) {
        const double* src = a.envpart + ((b * a.env_wg + t) * a.n + q) * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] += src[c];
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = wave_sum(acc[c]);
    const int beg = a.pre_ptr[q], end = a.pre_ptr[q + 1];
    // zero columns w >= 1 of every prefix rotation's gradient row
    for (int i = beg; i < end; ++i) {
        const int s = a.pre_ops[i].slot;
        if (s < 0) continue;
        double* row = a.gpart + ((size_t)s * a.B + b) * a.n_wg;
        for (int w = 1 + lane; w < a.n_wg; w += 64) row[w] = 0.0;
    }
    if (lane != 0) return;
    auto angle = [&](const DevPrefix& gt) {
        int64_t bs;
        return gt.slot >= 0 ? angle_of<Real>(a.inputs, a.weights, a.F, a.slots[gt.slot], b, 0, 0, bs) : 0.0;
    };
    // f: the factor after all prefix gates; g: r_q
    double2 f0 = make_double2(1.0, 0.0), f1 = make_double2(0.0, 0.0);
    for (int i = beg; i < end; ++i) apply_gate1(a.pre_ops[i].kind, angle(a.pre_ops[i]), false, f0, f1);
    double2 g0 = make_double2(acc[0], acc[1]), g1 = make_double2(acc[2], acc[3]);
    // walk back: at gate j, f = B_j |0> and g = A_j^dagger r_q
    for (int i = end - 1; i >= beg; --i) {
        const DevPrefix gt = a.pre_ops[i];
        const double t = angle(gt);
        if (gt.slot >= 0) {
            // P f for P = X, Y, Z, then Im <g| P f>
            double2 p0, p1;
            if (gt.kind == K_RX) {
                p0 = f1;
                p1 = f0;
            } else if (gt.kind == K_RY) {  // Y = [[0, -i], [i, 0]]
                p0 = make_double2(f1.y, -f1.x);
                p1 = make_double2(-f0.y, f0.x);
            } else {
                p0 = f0;
                p1 = make_double2(-f1.x, -f1.y);
            }
            const double im = (g0.x * p0.y - g0.y * p0.x) + (g1.x * p1.y - g1.y * p1.x);
            a.gpart[((size_t)gt.slot * a.B + b) * a.n_wg] = im;
        }
        apply_gate1(gt.kind, t, true, f0, f1);
        apply_gate1(gt.kind, t, true, g0, g1);
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

bool whole_uses_wave(int n, bool bwd, int64_t B) { return n <= 8 && (bwd || B < WAVE_MAX_FWD_CIRCUITS); }

hipError_t launch_whole(int dtype, const WholeArgs& a, int threads, size_t lds, hipStream_t s) {
    if (whole_uses_wave(a.n, a.bwd != 0, a.B)) {  // one wavefront per sample
        const dim3 grid((unsigned)a.B), block(64);
#define QL_WAVE(REAL)                                                                     \
    {                                                                                     \
        if (a.n <= 6) hipLaunchKernelGGL((k_wave<REAL, 1>), grid, block, 0, s, a, a.gates);      \
        else if (a.n == 7) hipLaunchKernelGGL((k_wave<REAL, 2>), grid, block, 0, s, a, a.gates); \
        else hipLaunchKernelGGL((k_wave<REAL, 4>), grid, block, 0, s, a, a.gates);               \
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

hipError_t launch_bind_tile(int dtype, const BindTileArgs& a, hipStream_t s) {
    const int64_t total = a.B * ((int64_t)a.n_ops + 1);
    const unsigned grid = (unsigned)((total + 255) / 256);
    if (dtype == 0) hipLaunchKernelGGL(k_bind_tile<float>, dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_bind_tile<double>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
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

hipError_t launch_bind_prefix(int dtype, const PrefixArgs& a, hipStream_t s) {
    const int64_t items = a.B * a.n;
    if (items == 0) return hipSuccess;
    const unsigned grid = (unsigned)((items + 255) / 256);
    if (dtype == 0) hipLaunchKernelGGL(k_bind_prefix<float>, dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_bind_prefix<double>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

// Register bits per lane of the environment kernel: 8 (complex64) or 4
// (complex128) amplitudes per lane keep it at 128 VGPRs or fewer.
int env_log_regs(int dtype, int n) { return std::min(dtype == 0 ? 3 : 2, n - 6); }

int env_workgroups(int dtype, int n, int64_t B) {
    const int lr = env_log_regs(dtype, n);
    const int64_t nblk = (int64_t)1 << (n - lr - 6);
    // a power of two, so that a wavefront's blocks share their low index bits
    int64_t want = 1;
    while (want * 2 * std::max<int64_t>(B, 1) <= 2048) want *= 2;
    int64_t cap = 1;
    while (cap * 4 < nblk) cap *= 2;
    // at most 2^ENV_HIGH_BITS blocks per wavefront (its LDS table of U)
    int64_t floor = 1;
    while (floor * 4 * ((int64_t)1 << ENV_HIGH_BITS) < nblk) floor *= 2;
    return (int)std::max(std::min(want, cap), floor);
}

hipError_t launch_env(int dtype, const PrefixArgs& a, hipStream_t s) {
    if (a.n < 8 || a.n > 32) return hipErrorInvalidValue;
    const dim3 grid((unsigned)(a.B * a.env_wg));
    const int lr = env_log_regs(dtype, a.n);
    // a wavefront's blocks fit its LDS table: nblk / (4 env_wg) <= 2^ENV_HIGH_BITS
    if (a.env_wg < 1 || (a.env_wg & (a.env_wg - 1)) != 0 ||
        ((int64_t)1 << (a.n - lr - 6)) > (int64_t)a.env_wg * 4 * ((int64_t)1 << ENV_HIGH_BITS))
        return hipErrorInvalidValue;
    if (dtype == 0) {
        if (lr == 2) hipLaunchKernelGGL((k_env<float, 2>), grid, dim3(256), 0, s, a);
        else hipLaunchKernelGGL((k_env<float, 3>), grid, dim3(256), 0, s, a);
    } else {
        hipLaunchKernelGGL((k_env<double, 2>), grid, dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_env_grad(int dtype, const PrefixArgs& a, hipStream_t s) {
    const int64_t waves = a.B * a.n;
    if (waves == 0) return hipSuccess;
    const unsigned grid = (unsigned)((waves + 3) / 4);
    if (dtype == 0) hipLaunchKernelGGL(k_env_grad<float>, dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_env_grad<double>, dim3(grid), dim3(256), 0, s, a);
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
    for (const void* fn : {reinterpret_cast<const void*>(k_whole<float>),
                           reinterpret_cast<const void*>(k_whole<double>)})
        if (e == hipSuccess) e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)max_lds);
    return e == hipSuccess ? configure_tile_kernels(max_lds) : e;
}

}  // namespace qlayer
