// tile.hip -- the register-tile pass kernel k_tile (gfx950) and its launcher.
//
// One launch is one tile pass over every sample; see the comment below for
// the layout of a tile in registers and LDS, the op interpreter and the
// gate arithmetic.
#include "kcommon.hpp"

namespace qlayer {
namespace {

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

// Add the wavefront's gradient partial to its LDS accumulators gacc[g][wave]
// [2]: a row butterfly and one row broadcast leave each half-wavefront's sum
// in lanes 31 and 63, which add it to their own word (two words instead of
// one save the last broadcast step). Every word has one writer lane, so its
// sum is in program order (deterministic); the add has no return value.
// `gthr` is this thread's word of accumulator 0, gacc + wave * GRAD_WORDS +
// (lane >> 5), and `stride` the uniform distance between accumulators: the
// address then costs one vector add.
constexpr int GRAD_WORDS = TILE_GRAD_WORDS;
template <typename Real>
__device__ __forceinline__ void grad_add(Real* gthr, uint32_t g, Real part, int lane, int /*wave*/,
                                         int stride) {
    Real v = row_sum(part);
    if constexpr (sizeof(Real) == 4) v += bcast_f32<0x142, 0xA>(v);
    else v += bcast_f64<0x142, 0xA>(v);
    if ((lane & 31) == 31)
        __hip_atomic_fetch_add(gthr + g * (uint32_t)stride, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
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

// ---- product-state prefix (see k_bind_prefix)

// The product state on one tile in layout F: register i of the thread gets
// C * prod_m phi_{q_m}(bit m of i), with C (fp64) the product of the factors
// of the thread's tile bits tb and of the tile's fixed amplitude-index bits gb.
// fac[2q + v] = phi_q(v) of this sample.
template <int LOG_R, int LOG_T, typename T2, typename Real>
__device__ __forceinline__ void product_tile(T2* dst, const double2* __restrict__ fac, const DevPass& P,
                                             const DevPhase& F, uint32_t tb, uint32_t gb) {
    double2 c = make_double2(1.0, 0.0);
#pragma unroll
    for (int t = 0; t < LOG_T; ++t)
        if (t < P.log_t) {
            const uint32_t j = F.thr_bit[t];
            c = cxmul(c, fac[2 * P.tile_qubit[j] + ((tb >> j) & 1u)]);
        }
    for (int i = 0; i < P.n_fixed; ++i) {
        const int q = P.fixed_qubit[i];
        c = cxmul(c, fac[2 * q + ((gb >> q) & 1u)]);
    }
    dst[0] = to_real<T2, Real>(c);
#pragma unroll
    for (int m = 0; m < LOG_R; ++m) {
        const int q = P.tile_qubit[F.reg_bit[m]];
        const T2 f0 = to_real<T2, Real>(fac[2 * q]), f1 = to_real<T2, Real>(fac[2 * q + 1]);
#pragma unroll
        for (int i = 0; i < (1 << m); ++i) {
            dst[i | (1 << m)] = cxmul(dst[i], f1);
            dst[i] = cxmul(dst[i], f0);
        }
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

// Negate x where bit 31 of s is set (the sign bit of a float; of the high word
// of a double).
__device__ __forceinline__ float xor_sign(float x, uint32_t s) {
    return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, x) ^ s);
}
__device__ __forceinline__ double xor_sign(double x, uint32_t s) {
    return __builtin_bit_cast(double, __builtin_bit_cast(uint64_t, x) ^ ((uint64_t)s << 32));
}

// CZ group g on a register tile (and on lm too when BOTH: the same tile's
// second state). Register i of a lane is negated when bit i of the lane's mask
//   M = (s ? all : 0) ^ sum over register bits a with c_a = 1 of (registers with bit a set)
//       ^ g.reg_mask
// is set, with s the parity of the pairs without a register operand (thread-
// thread pairs from the lane's tile bits tb, thread-fixed pairs linear in tb
// with coefficients from the tile's fixed bits gb, fixed-fixed pairs uniform)
// and c_a the parity of register bit a's thread and fixed partners.
template <int LOG_R, bool BOTH, typename T2>
__device__ __forceinline__ void czg_apply(T2* ps, T2* lm, const DevCzg* __restrict__ g, uint32_t tb,
                                          uint32_t gb) {
    constexpr int R = 1 << LOG_R;
    const uint32_t n_tt = g->n_tt, n_pairs = g->n_pairs;
    uint32_t s = 0, lin = 0, u = 0;
    for (uint32_t p = 0; p < n_tt; ++p) {
        const uint32_t w = g->pair[p];
        s ^= (tb >> (w & 0xffu)) & (tb >> ((w >> 8) & 0xffu));
    }
    for (uint32_t p = n_tt; p < n_pairs; ++p) {  // second operand: a fixed qubit
        const uint32_t w = g->pair[p], wa = w & 0xffffu;
        const uint32_t fb = (gb >> ((w >> 16) & 0xffu)) & 1u;
        if (((wa >> 8) & 3u) == LOC_THR) lin ^= fb << (wa & 0xffu);
        else u ^= fb & (gb >> (wa & 0xffu));
    }
    // the registers with bit a set, as a mask over the R registers
    constexpr uint32_t half[5] = {0xaaaaaaaau, 0xccccccccu, 0xf0f0f0f0u, 0xff00ff00u, 0xffff0000u};
    constexpr uint32_t all = R == 32 ? 0xffffffffu : (1u << R) - 1u;
    uint32_t m = g->reg_mask ^ (((s ^ u ^ (uint32_t)__builtin_popcount(tb & lin)) & 1u) ? all : 0u);
#pragma unroll
    for (int a = 0; a < LOG_R; ++a)
        if ((__builtin_popcount(tb & g->thr[a]) ^ __builtin_popcount(gb & g->fix[a])) & 1) m ^= half[a] & all;
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const uint32_t t = (m << (31 - i)) & 0x80000000u;
        ps[i].x = xor_sign(ps[i].x, t);
        ps[i].y = xor_sign(ps[i].y, t);
        if constexpr (BOTH) {
            lm[i].x = xor_sign(lm[i].x, t);
            lm[i].y = xor_sign(lm[i].y, t);
        }
    }
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
// current layout (refreshed after a layout change whose argument carries
// ARG_IVAL: one that an RZ-type term follows), so the Z-generator term of an
// RZ is ival - 2 * (the bit-1 half), and of an RZ on a thread or fixed bit
// +-ival. `gacc` is the thread's word of gradient accumulator 0 and `nw` the
// stride between accumulators (see grad_add).
template <int LOG_R, int LOG_T, int OPM, typename T2, typename Real>
__device__ __forceinline__ void run_op(uint32_t h, uint32_t arg, Real ca, Real cb, T2* ps, T2* lm,
                                       TileCtx& cx, Real& ival, unsigned char* lds,
                                       const DevPhase* phases, Real* gacc, int lane, int wave, int nw,
                                       int tid, const T2* __restrict__ dz, const T2* __restrict__ fz,
                                       const DevCzg* __restrict__ czg, const uint32_t* __restrict__ pthr) {
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
            const uint32_t dtb = (1u << ((arg >> 20) & 31)) | (1u << ((arg >> 25) & 31));  \
            if ((lane >> B) & 1) {                                                          \
                cx.tb ^= dtb;                                                               \
                cx.ts ^= lds_slot(dtb) * (uint32_t)sizeof(T2);                              \
            }                                                                               \
            if constexpr (OPM == OP_BWD)                                                    \
                if (arg & ARG_IVAL) ival = im_sum<LOG_R, -1, T2, Real>(ps, lm);             \
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
        case H_CZG:
            if constexpr (LOG_R <= CZG_REG_BITS) {
                if constexpr (OPM == OP_PAIR) {
                    czg_apply<LOG_R, false>(ps, lm, czg + arg, cx.tb, cx.gb);
                    czg_apply<LOG_R, false>(lm, ps, czg + arg, cx.tb, cx.gb2);
                } else {
                    czg_apply<LOG_R, OPM == OP_BWD>(ps, lm, czg + arg, cx.tb, cx.gb);
                }
            }
            break;
        case H_CZ_XX: {
            const bool on = loc_bit(arg & 0xffff, cx.tb, cx.gb) && loc_bit(arg >> 16, cx.tb, cx.gb);
            cz_sel<LOG_R, -1>(ps, on);
            if constexpr (OPM != OP_ONE)
                cz_sel<LOG_R, -1>(lm, loc_bit(arg & 0xffff, cx.tb, cx.gb2) && loc_bit(arg >> 16, cx.tb, cx.gb2));
        } break;
        case H_TRANSPOSE: {
            const uint32_t ph_to = arg & 0xfffffu;
            const DevPhase& to = phases[ph_to];
            // the thread's layout in the new phase, from its lane's and its
            // wavefront's table words
            const uint32_t* pt = pthr + (size_t)ph_to * PTHR_WORDS;
            const uint32_t tw = pt[lane] ^ pt[64 + wave];
            const uint32_t tb_to = tw & ((1u << PTHR_TB_BITS) - 1u), ts_to = tw >> PTHR_TB_BITS;
            lds_exchange<LOG_R>(ps, lds, phases[cx.ph], to, cx.ts, ts_to);
            if constexpr (OPM != OP_ONE) lds_exchange<LOG_R>(lm, lds, phases[cx.ph], to, cx.ts, ts_to);
            if constexpr (OPM == OP_BWD)
                if (arg & ARG_IVAL) ival = im_sum<LOG_R, -1, T2, Real>(ps, lm);
            cx.tb = tb_to;
            cx.ts = ts_to;
            cx.ph = (int)ph_to;
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
    Real* gthr = gacc + wave * GW + (lane >> 5);       // this thread's word of accumulator 0

    const size_t dim = (size_t)1 << n;
    const T2* psi_s = (const T2*)a.psi + b * dim;
    T2* psi_o = (T2*)a.psi_out + b * dim;
    T2* lam_s = (T2*)a.lam + b * dim;
    const XOp<Real>* xops = xops_all + b * (a.n_ops + 1);
    // this sample's product-prefix factors, fac[2q + v] = phi_q(v)
    const double2* fac = (const double2*)a.phi + (a.phi ? b * 2 * n : 0);
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

    const bool load = !(flags & (PF_INIT | PF_PRODUCT));
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

        if (!load && (flags & PF_PRODUCT)) {
            const double2* ft = fac;  // opaque: the factor loads stay in the loop
            asm volatile("" : "+s"(ft));
            product_tile<LOG_R, LOG_T, T2, Real>(ps, ft, P, phases[ph0], tb0, cx.gb);
            if constexpr (PAIR) product_tile<LOG_R, LOG_T, T2, Real>(lm, ft, P, phases[ph0], tb0, cx.gb2);
        } else if (!load) {
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
                                                              ival, lds, phases, gthr, lane, wave, NW * GW,
                                                              tid, dz, fz, a.czg, a.pthr);
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
                                                 phases, gthr, lane, wave, NW * GW, tid, dz, fz, a.czg,
                                                 a.pthr);
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

}  // namespace

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

size_t tile_static_lds(int dtype, int log_r, int threads) {
    const size_t maxt = threads > 256 ? 512 : 256;
    return maxt * ((size_t)1 << log_r) * 2 * (dtype == 0 ? sizeof(float) : sizeof(double));
}

hipError_t configure_tile_kernels(size_t max_lds) {
    hipError_t e = hipSuccess;
    // dynamic LDS of the tile kernels: what the static exchange buffer leaves
#define QL_ATTR_TK(REAL, LR, BW, MT)                                                      \
    if (e == hipSuccess) {                                                                \
        const size_t st = tile_lds_bytes<REAL, LR, MT>();                                 \
        if (st < max_lds)                                                                 \
            e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_tile<REAL, LR, BW, MT>), \
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)(max_lds - st)); \
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
    return e;
}

}  // namespace qlayer
