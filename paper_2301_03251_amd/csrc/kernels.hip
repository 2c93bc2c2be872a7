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
#include <hip/hip_runtime.h>

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

// Scatter the low bits of x into the set bits of mask (ascending).
__device__ __forceinline__ uint32_t deposit(uint32_t x, uint32_t mask) {
    uint32_t r = 0;
    for (int j = 0; j < MAX_TILE_BITS; ++j) {
        if (mask >> j & 1u) {
            r |= (x & 1u) << j;
            x >>= 1;
        }
    }
    return r;
}

// ---------------------------------------------------------------------------
// one-qubit gates on the register bit J of a thread's 2^LOG_R amplitudes.
// s carries the sign of the rotation: the inverse gate passes -s.

template <int LOG_R, int J, typename T2, typename Real>
__device__ __forceinline__ void reg_g1(int kind, T2* a, Real c, Real s) {
    constexpr int R = 1 << LOG_R, M = 1 << J;
    if (kind == K_H) {
        const Real r = (Real)0.70710678118654752440;
#pragma unroll
        for (int i = 0; i < R; ++i)
            if (!(i & M)) {
                const T2 u = a[i], v = a[i | M];
                a[i] = mk<T2>((u.x + v.x) * r, (u.y + v.y) * r);
                a[i | M] = mk<T2>((u.x - v.x) * r, (u.y - v.y) * r);
            }
    } else if (kind == K_RX) {  // [[c, -is], [-is, c]]
#pragma unroll
        for (int i = 0; i < R; ++i)
            if (!(i & M)) {
                const T2 u = a[i], v = a[i | M];
                a[i] = mk<T2>(c * u.x + s * v.y, c * u.y - s * v.x);
                a[i | M] = mk<T2>(c * v.x + s * u.y, c * v.y - s * u.x);
            }
    } else if (kind == K_RY) {  // [[c, -s], [s, c]]
#pragma unroll
        for (int i = 0; i < R; ++i)
            if (!(i & M)) {
                const T2 u = a[i], v = a[i | M];
                a[i] = mk<T2>(c * u.x - s * v.x, c * u.y - s * v.y);
                a[i | M] = mk<T2>(s * u.x + c * v.x, s * u.y + c * v.y);
            }
    } else {  // RZ: diag(c - is, c + is)
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const T2 u = a[i];
            if (i & M) a[i] = mk<T2>(c * u.x - s * u.y, c * u.y + s * u.x);
            else a[i] = mk<T2>(c * u.x + s * u.y, c * u.y - s * u.x);
        }
    }
}

template <int LOG_R, typename T2, typename Real>
__device__ __forceinline__ void reg_g1_at(int j, int kind, T2* a, Real c, Real s) {
    switch (j) {
        case 0: if constexpr (LOG_R > 0) reg_g1<LOG_R, 0>(kind, a, c, s); break;
        case 1: if constexpr (LOG_R > 1) reg_g1<LOG_R, 1>(kind, a, c, s); break;
        case 2: if constexpr (LOG_R > 2) reg_g1<LOG_R, 2>(kind, a, c, s); break;
        case 3: if constexpr (LOG_R > 3) reg_g1<LOG_R, 3>(kind, a, c, s); break;
        case 4: if constexpr (LOG_R > 4) reg_g1<LOG_R, 4>(kind, a, c, s); break;
        default: break;
    }
}

// Thread partial of Im<l | P_J | p> for the rotation generator P of `kind`.
template <int LOG_R, int J, typename T2, typename Real>
__device__ __forceinline__ Real reg_grad(int kind, const T2* p, const T2* l) {
    constexpr int R = 1 << LOG_R, M = 1 << J;
    Real acc = 0;
    if (kind == K_RZ) {
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const Real t = l[i].x * p[i].y - l[i].y * p[i].x;
            acc += (i & M) ? -t : t;
        }
    } else if (kind == K_RX) {
#pragma unroll
        for (int i = 0; i < R; ++i)
            if (!(i & M)) {
                const int v = i | M;
                acc += (l[i].x * p[v].y - l[i].y * p[v].x) + (l[v].x * p[i].y - l[v].y * p[i].x);
            }
    } else {  // RY
#pragma unroll
        for (int i = 0; i < R; ++i)
            if (!(i & M)) {
                const int v = i | M;
                acc += (l[v].x * p[i].x + l[v].y * p[i].y) - (l[i].x * p[v].x + l[i].y * p[v].y);
            }
    }
    return acc;
}

template <int LOG_R, typename T2, typename Real>
__device__ __forceinline__ Real reg_grad_at(int j, int kind, const T2* p, const T2* l) {
    switch (j) {
        case 0: if constexpr (LOG_R > 0) return reg_grad<LOG_R, 0, T2, Real>(kind, p, l); break;
        case 1: if constexpr (LOG_R > 1) return reg_grad<LOG_R, 1, T2, Real>(kind, p, l); break;
        case 2: if constexpr (LOG_R > 2) return reg_grad<LOG_R, 2, T2, Real>(kind, p, l); break;
        case 3: if constexpr (LOG_R > 3) return reg_grad<LOG_R, 3, T2, Real>(kind, p, l); break;
        case 4: if constexpr (LOG_R > 4) return reg_grad<LOG_R, 4, T2, Real>(kind, p, l); break;
        default: break;
    }
    return 0;
}

// CNOT with target register bit J and control register bit m (runtime).
template <int LOG_R, int J, typename T2>
__device__ __forceinline__ void reg_cnot_rr(int m, T2* a) {
    constexpr int R = 1 << LOG_R, M = 1 << J;
#pragma unroll
    for (int i = 0; i < R; ++i)
        if (!(i & M) && (i >> m & 1)) {
            const T2 t = a[i];
            a[i] = a[i | M];
            a[i | M] = t;
        }
}

// CNOT with target register bit J and a per-thread control bit.
template <int LOG_R, int J, typename T2>
__device__ __forceinline__ void reg_cnot_sel(bool on, T2* a) {
    constexpr int R = 1 << LOG_R, M = 1 << J;
#pragma unroll
    for (int i = 0; i < R; ++i)
        if (!(i & M)) {
            const T2 u = a[i], v = a[i | M];
            a[i] = on ? v : u;
            a[i | M] = on ? u : v;
        }
}

template <int LOG_R, typename T2>
__device__ __forceinline__ void reg_cnot_at(int j, bool reg_ctrl, int m, bool on, T2* a) {
#define QL_CNOT_CASE(J)                                                            \
    case J:                                                                       \
        if constexpr (LOG_R > J) {                                                \
            if (reg_ctrl) reg_cnot_rr<LOG_R, J>(m, a);                            \
            else reg_cnot_sel<LOG_R, J>(on, a);                                   \
        }                                                                         \
        break;
    switch (j) {
        QL_CNOT_CASE(0)
        QL_CNOT_CASE(1)
        QL_CNOT_CASE(2)
        QL_CNOT_CASE(3)
        QL_CNOT_CASE(4)
        default: break;
    }
#undef QL_CNOT_CASE
}

// Bank-spreading permutation of LDS slots: folds the upper nibbles of the tile
// index into the lowest one (an involution on each aligned 2^16 block).
__device__ __forceinline__ uint32_t lds_slot(uint32_t t) {
    return t ^ (((t >> 4) ^ (t >> 8) ^ (t >> 12)) & 15u);
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
    const double th = src.src == S_INPUT
                          ? (double)((const Real*)a.inputs)[b * a.F + src.index]
                          : (double)((const Real*)a.weights)[src.index];
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

    for (int j = tid; j < dim; j += nt) psi[j] = mk<T2>((Real)(j == 0), (Real)0);
    __syncthreads();
    for (int gi = 0; gi < a.n_gates; ++gi) {
        const DevGate g = a.gates[gi];
        Real c = 1, s = 0;
        if (g.slot >= 0) {
            const T2 cs = coef[g.slot];
            c = cs.x;
            s = cs.y;
        }
        lds_gate(psi, g, c, s, n, tid, nt);
        __syncthreads();
    }
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
}

// ---------------------------------------------------------------------------
// k_tile: one tile pass

template <int LOG_R, typename T2>
__device__ __forceinline__ void lds_exchange(T2* a, T2* lds, const DevPhase& from,
                                             const DevPhase& to, uint32_t& tb, int tid) {
    constexpr int R = 1 << LOG_R;
#pragma unroll
    for (int i = 0; i < R; ++i) lds[lds_slot(tb | from.reg_off[i])] = a[i];
    __syncthreads();
    tb = deposit((uint32_t)tid, to.thr_mask);
#pragma unroll
    for (int i = 0; i < R; ++i) a[i] = lds[lds_slot(tb | to.reg_off[i])];
    __syncthreads();
}

template <typename Real, int LOG_R, bool BWD>
__global__ void __launch_bounds__(256) k_tile(const TileArgs a) {
    using T2 = typename Cx<Real>::T;
    constexpr int R = 1 << LOG_R;
    extern __shared__ __align__(16) unsigned char smem[];
    const DevPass& P = *a.pass;
    const DevPhase* phases = a.phases;
    const int tid = threadIdx.x, nt = blockDim.x, NW = nt >> 6;
    const int wave = tid >> 6, lane = tid & 63;
    const int flags = a.flags;
    const int64_t b = blockIdx.x / a.n_wg;
    const int w = (int)(blockIdx.x - b * a.n_wg);
    const int n = a.n, k = P.k;
    T2* lds = (T2*)smem;
    double* accz = (double*)(smem + a.lds_tile_bytes);  // [n][NW]
    double* accg = accz + n * NW;                       // [n_gslots][NW]
    for (int i = tid; i < (n + a.n_gslots) * NW; i += nt) accz[i] = 0.0;
    __syncthreads();

    const size_t dim = (size_t)1 << n;
    T2* psi_s = (T2*)a.psi + b * dim;
    T2* lam_s = (T2*)a.lam + b * dim;
    const T2* coef = (const T2*)a.coef + b * a.n_slots;
    const Real* gout = (const Real*)a.grad_out + b * n;

    T2 ps[R], lm[R];
    for (int64_t tile = w; tile < a.tiles; tile += a.n_wg) {
        uint32_t gb = 0;  // amplitude index bits of the qubits outside the tile
        for (int i = 0; i < P.n_fixed; ++i) gb |= (uint32_t)((tile >> i) & 1) << P.fixed_qubit[i];
        int ph = (flags & PF_FWD) ? P.load_phase : P.bwd_phase;
        uint32_t tb = deposit((uint32_t)tid, phases[ph].thr_mask);

        auto gaddr_thr = [&](uint32_t tbits) {
            uint32_t g = 0;
            for (int j = 0; j < k; ++j) g |= ((tbits >> j) & 1u) << P.tile_qubit[j];
            return gb | g;
        };

        if (flags & PF_INIT) {
#pragma unroll
            for (int i = 0; i < R; ++i) ps[i] = mk<T2>((Real)0, (Real)0);
            if (gb == 0 && tb == 0) ps[0] = mk<T2>((Real)1, (Real)0);
        } else {
            const uint32_t base = gaddr_thr(tb);
#pragma unroll
            for (int i = 0; i < R; ++i) ps[i] = psi_s[base + phases[ph].greg_off[i]];
            if (BWD && (flags & PF_LOAD_LAM)) {
#pragma unroll
                for (int i = 0; i < R; ++i) lm[i] = lam_s[base + phases[ph].greg_off[i]];
            }
        }

        // ---- forward ops
        if (flags & PF_FWD) {
            for (int o = P.fwd_begin; o < P.fwd_end; ++o) {
                const DevOp op = a.ops[o];
                Real c = 1, s = 0;
                if (op.slot >= 0) {
                    const T2 cs = coef[op.slot];
                    c = cs.x;
                    s = cs.y;
                }
                switch (op.code) {
                    case OP_G1:
                        reg_g1_at<LOG_R>(op.a_pos, op.kind, ps, c, s);
                        break;
                    case OP_RZ_U: {
                        const uint32_t bit = op.a_type == LOC_THR ? (tb >> op.a_pos) & 1u
                                                                  : (gb >> op.a_pos) & 1u;
                        const Real ss = bit ? s : -s;
#pragma unroll
                        for (int i = 0; i < R; ++i)
                            ps[i] = mk<T2>(c * ps[i].x - ss * ps[i].y, c * ps[i].y + ss * ps[i].x);
                    } break;
                    case OP_CNOT: {
                        const bool rc = op.b_type == LOC_REG;
                        const bool on = op.b_type == LOC_THR ? ((tb >> op.b_pos) & 1u)
                                                             : ((gb >> op.b_pos) & 1u);
                        reg_cnot_at<LOG_R>(op.a_pos, rc, op.b_pos, on, ps);
                    } break;
                    case OP_CZ: {
                        uint32_t rm = 0;
                        bool on = true;
                        if (op.a_type == LOC_REG) rm |= 1u << op.a_pos;
                        else on = on && ((op.a_type == LOC_THR ? tb : gb) >> op.a_pos & 1u);
                        if (op.b_type == LOC_REG) rm |= 1u << op.b_pos;
                        else on = on && ((op.b_type == LOC_THR ? tb : gb) >> op.b_pos & 1u);
                        const Real sg = on ? (Real)-1 : (Real)1;
#pragma unroll
                        for (int i = 0; i < R; ++i)
                            if ((i & rm) == rm) ps[i] = mk<T2>(sg * ps[i].x, sg * ps[i].y);
                    } break;
                    default: {  // OP_TRANSPOSE
                        lds_exchange<LOG_R>(ps, lds, phases[ph], phases[op.arg], tb, tid);
                        ph = op.arg;
                    } break;
                }
            }
        }

        // ---- <Z_q> partials over this tile
        if (flags & PF_ZPART) {
            const DevPhase& F = phases[ph];
            Real pt = 0, dm[LOG_R];
#pragma unroll
            for (int m = 0; m < LOG_R; ++m) dm[m] = 0;
#pragma unroll
            for (int i = 0; i < R; ++i) {
                const Real p = ps[i].x * ps[i].x + ps[i].y * ps[i].y;
                pt += p;
#pragma unroll
                for (int m = 0; m < LOG_R; ++m) dm[m] += (i >> m & 1) ? -p : p;
            }
            const double wp = wave_sum((double)pt);
            for (int j = 0; j < k; ++j) {
                Real v = (tb >> j & 1u) ? -pt : pt;
#pragma unroll
                for (int m = 0; m < LOG_R; ++m)
                    if ((int)F.reg_bit[m] == j) v = dm[m];
                const double d = wave_sum((double)v);
                if (lane == 0) accz[P.tile_qubit[j] * NW + wave] += d;
            }
            if (lane == 0)
                for (int i = 0; i < P.n_fixed; ++i) {
                    const int q = P.fixed_qubit[i];
                    accz[q * NW + wave] += (gb >> q & 1u) ? -wp : wp;
                }
        }

        if constexpr (BWD) {
            // ---- lambda = (sum_q g_q Z_q) psi
            if (flags & PF_SEED) {
                const DevPhase& F = phases[ph];
                Real gs = 0, sfix = 0, sthr = 0, gm[LOG_R];
                for (int q = 0; q < n; ++q) gs += gout[q];
                for (int i = 0; i < P.n_fixed; ++i) {
                    const int q = P.fixed_qubit[i];
                    if (gb >> q & 1u) sfix += gout[q];
                }
                for (int j = 0; j < k; ++j)
                    if ((F.thr_mask >> j & 1u) && (tb >> j & 1u)) sthr += gout[P.tile_qubit[j]];
#pragma unroll
                for (int m = 0; m < LOG_R; ++m) gm[m] = gout[P.tile_qubit[F.reg_bit[m]]];
#pragma unroll
                for (int i = 0; i < R; ++i) {
                    Real sr = 0;
#pragma unroll
                    for (int m = 0; m < LOG_R; ++m)
                        if (i >> m & 1) sr += gm[m];
                    const Real d = gs - (Real)2 * (sfix + sthr + sr);
                    lm[i] = mk<T2>(d * ps[i].x, d * ps[i].y);
                }
            }

            // ---- backward ops: gradient, then un-apply on psi and lambda
            if (flags & PF_BWD) {
                for (int o = P.bwd_begin; o < P.bwd_end; ++o) {
                    const DevOp op = a.ops[o];
                    Real c = 1, s = 0;
                    if (op.slot >= 0) {
                        const T2 cs = coef[op.slot];
                        c = cs.x;
                        s = -cs.y;  // inverse rotation
                    }
                    switch (op.code) {
                        case OP_G1:
                            if (op.gslot >= 0) {
                                const double d = wave_sum(
                                    (double)reg_grad_at<LOG_R, T2, Real>(op.a_pos, op.kind, ps, lm));
                                if (lane == 0) accg[op.gslot * NW + wave] += d;
                            }
                            reg_g1_at<LOG_R>(op.a_pos, op.kind, ps, c, s);
                            reg_g1_at<LOG_R>(op.a_pos, op.kind, lm, c, s);
                            break;
                        case OP_RZ_U: {
                            const uint32_t bit = op.a_type == LOC_THR ? (tb >> op.a_pos) & 1u
                                                                      : (gb >> op.a_pos) & 1u;
                            Real acc = 0;
#pragma unroll
                            for (int i = 0; i < R; ++i) acc += lm[i].x * ps[i].y - lm[i].y * ps[i].x;
                            const double d = wave_sum((double)(bit ? -acc : acc));
                            if (lane == 0) accg[op.gslot * NW + wave] += d;
                            const Real ss = bit ? s : -s;
#pragma unroll
                            for (int i = 0; i < R; ++i) {
                                ps[i] = mk<T2>(c * ps[i].x - ss * ps[i].y, c * ps[i].y + ss * ps[i].x);
                                lm[i] = mk<T2>(c * lm[i].x - ss * lm[i].y, c * lm[i].y + ss * lm[i].x);
                            }
                        } break;
                        case OP_CNOT: {
                            const bool rc = op.b_type == LOC_REG;
                            const bool on = op.b_type == LOC_THR ? ((tb >> op.b_pos) & 1u)
                                                                 : ((gb >> op.b_pos) & 1u);
                            reg_cnot_at<LOG_R>(op.a_pos, rc, op.b_pos, on, ps);
                            reg_cnot_at<LOG_R>(op.a_pos, rc, op.b_pos, on, lm);
                        } break;
                        case OP_CZ: {
                            uint32_t rm = 0;
                            bool on = true;
                            if (op.a_type == LOC_REG) rm |= 1u << op.a_pos;
                            else on = on && ((op.a_type == LOC_THR ? tb : gb) >> op.a_pos & 1u);
                            if (op.b_type == LOC_REG) rm |= 1u << op.b_pos;
                            else on = on && ((op.b_type == LOC_THR ? tb : gb) >> op.b_pos & 1u);
                            const Real sg = on ? (Real)-1 : (Real)1;
#pragma unroll
                            for (int i = 0; i < R; ++i)
                                if ((i & rm) == rm) {
                                    ps[i] = mk<T2>(sg * ps[i].x, sg * ps[i].y);
                                    lm[i] = mk<T2>(sg * lm[i].x, sg * lm[i].y);
                                }
                        } break;
                        default: {  // OP_TRANSPOSE
                            uint32_t tb0 = tb;
                            lds_exchange<LOG_R>(ps, lds, phases[ph], phases[op.arg], tb, tid);
                            lds_exchange<LOG_R>(lm, lds, phases[ph], phases[op.arg], tb0, tid);
                            ph = op.arg;
                        } break;
                    }
                }
            }
        }

        if (flags & (PF_STORE_PSI | PF_STORE_LAM)) {
            const uint32_t base = gaddr_thr(tb);
            if (flags & PF_STORE_PSI) {
#pragma unroll
                for (int i = 0; i < R; ++i) psi_s[base + phases[ph].greg_off[i]] = ps[i];
            }
            if (BWD && (flags & PF_STORE_LAM)) {
#pragma unroll
                for (int i = 0; i < R; ++i) lam_s[base + phases[ph].greg_off[i]] = lm[i];
            }
        }
    }

    __syncthreads();
    if (flags & PF_ZPART)
        for (int q = tid; q < n; q += nt) {
            double t = 0;
            for (int v = 0; v < NW; ++v) t += accz[q * NW + v];
            a.zpart[((size_t)b * a.n_wg + w) * n + q] = t;
        }
    if (BWD && (flags & PF_BWD))
        for (int g = tid; g < a.n_gslots; g += nt) {
            double t = 0;
            for (int v = 0; v < NW; ++v) t += accg[g * NW + v];
            a.gpart[((size_t)a.gslots[g] * a.B + b) * a.n_wg + w] = t;
        }
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
            for (int w = lane; w < a.n_wg; w += 64) acc += a.gpart[((size_t)s * a.B + b) * a.n_wg + w];
        }
        acc = wave_sum(acc);
        if (lane == 0) ((Real*)a.grad_inputs)[u] = (Real)acc;
    } else if (e < nz + nx + nw) {
        const int p = (int)(e - nz - nx);
        const int64_t per = a.B * a.n_wg;
        for (int i = a.w_ptr[p]; i < a.w_ptr[p + 1]; ++i) {
            const double* src = a.gpart + (size_t)a.w_slot[i] * per;
            for (int64_t j = lane; j < per; j += 64) acc += src[j];
        }
        acc = wave_sum(acc);
        if (lane == 0) ((Real*)a.grad_weights)[p] = (Real)acc;
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

hipError_t launch_whole(int dtype, const WholeArgs& a, int threads, size_t lds, hipStream_t s) {
    if (dtype == 0) hipLaunchKernelGGL(k_whole<float>, dim3((unsigned)a.B), dim3(threads), lds, s, a);
    else hipLaunchKernelGGL(k_whole<double>, dim3((unsigned)a.B), dim3(threads), lds, s, a);
    return hipGetLastError();
}

template <typename Real, int LOG_R>
static hipError_t launch_tile_t(bool bwd, const TileArgs& a, int threads, size_t lds, hipStream_t s) {
    const dim3 grid((unsigned)(a.B * a.n_wg));
    if (bwd) hipLaunchKernelGGL((k_tile<Real, LOG_R, true>), grid, dim3(threads), lds, s, a);
    else hipLaunchKernelGGL((k_tile<Real, LOG_R, false>), grid, dim3(threads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_tile(int dtype, int log_r, bool bwd, const TileArgs& a, int threads, size_t lds,
                       hipStream_t s) {
    if (dtype == 0) {
        switch (log_r) {
            case 2: return launch_tile_t<float, 2>(bwd, a, threads, lds, s);
            case 3: return launch_tile_t<float, 3>(bwd, a, threads, lds, s);
            case 4: return launch_tile_t<float, 4>(bwd, a, threads, lds, s);
            case 5: return launch_tile_t<float, 5>(bwd, a, threads, lds, s);
        }
    } else {
        switch (log_r) {
            case 2: return launch_tile_t<double, 2>(bwd, a, threads, lds, s);
            case 3: return launch_tile_t<double, 3>(bwd, a, threads, lds, s);
            case 4: return launch_tile_t<double, 4>(bwd, a, threads, lds, s);
        }
    }
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

hipError_t configure_kernels(size_t max_lds) {
    const int v = (int)max_lds;
    hipError_t e = hipSuccess;
#define QL_ATTR(fn)                                                                      \
    if (e == hipSuccess)                                                                 \
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),                       \
                                hipFuncAttributeMaxDynamicSharedMemorySize, v);
    QL_ATTR((k_whole<float>))
    QL_ATTR((k_whole<double>))
    QL_ATTR((k_tile<float, 2, false>))
    QL_ATTR((k_tile<float, 2, true>))
    QL_ATTR((k_tile<float, 3, false>))
    QL_ATTR((k_tile<float, 3, true>))
    QL_ATTR((k_tile<float, 4, false>))
    QL_ATTR((k_tile<float, 4, true>))
    QL_ATTR((k_tile<float, 5, false>))
    QL_ATTR((k_tile<float, 5, true>))
    QL_ATTR((k_tile<double, 2, false>))
    QL_ATTR((k_tile<double, 2, true>))
    QL_ATTR((k_tile<double, 3, false>))
    QL_ATTR((k_tile<double, 3, true>))
    QL_ATTR((k_tile<double, 4, false>))
    QL_ATTR((k_tile<double, 4, true>))
#undef QL_ATTR
    return e;
}

}  // namespace qlayer
