/*
 * oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, gate-by-gate complex128 state-vector simulator of the
 * paper's quantum node (Sec. "Quantum Node": a parameterised circuit is
 * simulated and its measurement turned into classical data), with the
 * vector-Jacobian product the hybrid optimisation feeds back to the classical
 * optimiser (Sec. "Optimization"; the quantum node's backward hands back the
 * gradient multiplied by the upstream gradient, appendix "Hybrid
 * Quantum-Classical Neural Networks", class Hybrid).
 *
 * Only tests/, the smoke check and the benchmark's CPU-baseline leg may load
 * this library. The HIP product path never links or calls it, and the two
 * share no code.
 *
 * Definitions (readings of the paper where it is silent are listed in the
 * design notes):
 *   - qubit q is bit q of the amplitude index (little-endian);
 *   - initial state |0...0>;
 *   - H = [[1,1],[1,-1]]/sqrt2, RX(t) = exp(-i t X/2), RY(t) = exp(-i t Y/2),
 *     RZ(t) = exp(-i t Z/2); CNOT(c,t) flips bit t where bit c is 1;
 *     CZ(a,b) negates amplitudes where bits a and b are both 1;
 *   - the measured output is the exact <Z_i> (the shots -> infinity limit of
 *     the paper's Monte Carlo measurement), no renormalisation;
 *   - gradients are the VJP sum_i g[b,i] d<Z_i>_b/d(theta), summed over the
 *     batch for weights, per sample for inputs, and over every occurrence of
 *     a shared parameter.
 *   - the adjoint sweep is the published adjoint-differentiation method
 *     (Jones & Gacon 2020, Algorithm 1): lambda = O psi, then for each gate
 *     from last to first, take Im<lambda|P|psi> for a rotation exp(-i t P/2)
 *     and un-apply the gate on both psi and lambda.
 *   - parameter shift is the standard two-term rule
 *     d f / d t = (f(t + pi/2) - f(t - pi/2)) / 2 for exp(-i t P/2) gates
 *     (the paper's Hybrid class takes the same shifted difference).
 *
 * Every reduction over amplitudes is a pairwise (tree) sum in fp64.
 */
#include <complex.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef double complex cplx;

enum { G_H = 0, G_RX = 1, G_RY = 2, G_RZ = 3, G_CNOT = 4, G_CZ = 5 };
enum { SRC_NONE = 0, SRC_INPUT = 1, SRC_WEIGHT = 2 };

#define PAR_MIN (1 << 14) /* run amplitude loops in parallel above this size */

typedef struct { int32_t kind, q0, q1, src, index; } gate_t;

/* ------------------------------------------------------------------ */
/* validation                                                          */

static int check_circuit(int n, const gate_t* g, int G, int F, int P)
{
    if (n < 1 || n > 34 || G < 0) return -1;
    for (int k = 0; k < G; k++) {
        const gate_t* x = &g[k];
        if (x->q0 < 0 || x->q0 >= n) return -1;
        switch (x->kind) {
        case G_H:
            if (x->src != SRC_NONE) return -1;
            break;
        case G_RX: case G_RY: case G_RZ:
            if (x->src == SRC_INPUT) { if (x->index < 0 || x->index >= F) return -1; }
            else if (x->src == SRC_WEIGHT) { if (x->index < 0 || x->index >= P) return -1; }
            else return -1;
            break;
        case G_CNOT: case G_CZ:
            if (x->src != SRC_NONE || x->q1 < 0 || x->q1 >= n || x->q1 == x->q0) return -1;
            break;
        default:
            return -1;
        }
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* gates                                                               */

/* 2x2 matrix of a one-qubit gate: m[0] m[1] / m[2] m[3]. */
static void gate_matrix(int kind, double theta, cplx m[4])
{
    double c = cos(0.5 * theta), s = sin(0.5 * theta);
    switch (kind) {
    case G_H: {
        double r = 1.0 / sqrt(2.0);
        m[0] = r; m[1] = r; m[2] = r; m[3] = -r;
        break;
    }
    case G_RX: m[0] = c; m[1] = -I * s; m[2] = -I * s; m[3] = c; break;
    case G_RY: m[0] = c; m[1] = -s; m[2] = s; m[3] = c; break;
    case G_RZ: m[0] = c - I * s; m[1] = 0; m[2] = 0; m[3] = c + I * s; break;
    default: m[0] = 1; m[1] = 0; m[2] = 0; m[3] = 1; break;
    }
}

static void adjoint2(const cplx m[4], cplx a[4])
{
    a[0] = conj(m[0]); a[1] = conj(m[2]);
    a[2] = conj(m[1]); a[3] = conj(m[3]);
}

static void apply_matrix(cplx* psi, int64_t dim, int q, const cplx m[4])
{
    const int64_t bit = (int64_t)1 << q;
#pragma omp parallel for schedule(static) if (dim >= PAR_MIN)
    for (int64_t j = 0; j < dim; j++) {
        if (j & bit) continue;
        cplx a = psi[j], b = psi[j | bit];
        psi[j] = m[0] * a + m[1] * b;
        psi[j | bit] = m[2] * a + m[3] * b;
    }
}

static void apply_cnot(cplx* psi, int64_t dim, int c, int t)
{
    const int64_t cb = (int64_t)1 << c, tb = (int64_t)1 << t;
#pragma omp parallel for schedule(static) if (dim >= PAR_MIN)
    for (int64_t j = 0; j < dim; j++) {
        if ((j & cb) && !(j & tb)) {
            cplx tmp = psi[j];
            psi[j] = psi[j | tb];
            psi[j | tb] = tmp;
        }
    }
}

static void apply_cz(cplx* psi, int64_t dim, int a, int b)
{
    const int64_t ab = ((int64_t)1 << a) | ((int64_t)1 << b);
#pragma omp parallel for schedule(static) if (dim >= PAR_MIN)
    for (int64_t j = 0; j < dim; j++)
        if ((j & ab) == ab) psi[j] = -psi[j];
}

static double angle_of(const gate_t* g, const double* x_b, const double* w)
{
    if (g->src == SRC_INPUT) return x_b[g->index];
    if (g->src == SRC_WEIGHT) return w[g->index];
    return 0.0;
}

/* Apply gate g (dagger=1: its inverse) with the given angle. */
static void apply_gate(cplx* psi, int64_t dim, const gate_t* g, double theta, int dagger)
{
    if (g->kind == G_CNOT) { apply_cnot(psi, dim, g->q0, g->q1); return; }
    if (g->kind == G_CZ) { apply_cz(psi, dim, g->q0, g->q1); return; }
    cplx m[4], a[4];
    gate_matrix(g->kind, theta, m);
    if (dagger) { adjoint2(m, a); apply_matrix(psi, dim, g->q0, a); }
    else apply_matrix(psi, dim, g->q0, m);
}

/* ------------------------------------------------------------------ */
/* pairwise sums                                                       */

/* Term functions evaluated on the fly so no term array is materialised. */
typedef struct {
    const cplx* psi;
    const cplx* lam;
    int64_t bit;     /* 1 << q */
    int kind;        /* generator for inner products: X, Y or Z */
} term_ctx;

/* Pairwise sum of f(j) for j in [lo, hi). */
static double psum_real(const term_ctx* c, double (*f)(const term_ctx*, int64_t),
                        int64_t lo, int64_t hi)
{
    if (hi - lo <= 32) {
        double s = 0.0;
        for (int64_t j = lo; j < hi; j++) s += f(c, j);
        return s;
    }
    int64_t mid = lo + (hi - lo) / 2;
    return psum_real(c, f, lo, mid) + psum_real(c, f, mid, hi);
}

/* Pairwise over [0, dim): top levels split into 2^L equal chunks summed in
 * parallel, then combined as a binary tree (still a pairwise sum). */
static double pairwise(const term_ctx* c, double (*f)(const term_ctx*, int64_t), int64_t dim)
{
    int L = 0;
    while (L < 8 && (dim >> (L + 1)) >= PAR_MIN) L++;
    int nch = 1 << L;
    double part[256];
    int64_t len = dim / nch;
#pragma omp parallel for schedule(static) if (nch > 1)
    for (int i = 0; i < nch; i++) part[i] = psum_real(c, f, (int64_t)i * len, (int64_t)(i + 1) * len);
    for (int w = 1; w < nch; w <<= 1)
        for (int i = 0; i + w < nch; i += 2 * w) part[i] += part[i + w];
    return part[0];
}

static double term_zsign_prob(const term_ctx* c, int64_t j)
{
    double p = creal(c->psi[j]) * creal(c->psi[j]) + cimag(c->psi[j]) * cimag(c->psi[j]);
    return (j & c->bit) ? -p : p;
}

/* Im of the j-th term of <lam | P_q | psi>. */
static double term_im_inner(const term_ctx* c, int64_t j)
{
    const int64_t b = c->bit;
    cplx pj; /* (P_q psi)_j */
    switch (c->kind) {
    case G_RX: pj = c->psi[j ^ b]; break;
    case G_RY: pj = (j & b) ? I * c->psi[j ^ b] : -I * c->psi[j ^ b]; break;
    default:   pj = (j & b) ? -c->psi[j] : c->psi[j]; break;
    }
    return cimag(conj(c->lam[j]) * pj);
}

/* <Z_q> of psi. */
static double expect_z(const cplx* psi, int64_t dim, int q)
{
    term_ctx c = { psi, NULL, (int64_t)1 << q, 0 };
    return pairwise(&c, term_zsign_prob, dim);
}

/* Im <lam | P_q | psi>, P from the rotation kind. */
static double im_inner(const cplx* lam, const cplx* psi, int64_t dim, int q, int kind)
{
    term_ctx c = { psi, lam, (int64_t)1 << q, kind };
    return pairwise(&c, term_im_inner, dim);
}

/* ------------------------------------------------------------------ */
/* one sample                                                          */

static void run_forward(cplx* psi, int n, const gate_t* g, int G,
                        const double* x_b, const double* w, int shift_gate, double shift)
{
    const int64_t dim = (int64_t)1 << n;
    memset(psi, 0, sizeof(cplx) * (size_t)dim);
    psi[0] = 1.0;
    for (int k = 0; k < G; k++) {
        double th = angle_of(&g[k], x_b, w);
        if (k == shift_gate) th += shift;
        apply_gate(psi, dim, &g[k], th, 0);
    }
}

/*
 * Forward + adjoint VJP over a batch.
 *
 *   gates      [G][5] int32 rows (kind, q0, q1, src, index)
 *   inputs     [B][F] angles bound to features (fp64)
 *   weights    [P]    angles bound to trainable weights (fp64)
 *   grad_out   [B][n] upstream gradient g (NULL: forward only)
 *   expz       [B][n] out: <Z_i>
 *   grad_in    [B][F] out (may be NULL): sum_i g[b,i] d<Z_i>_b / d x[b,f]
 *   grad_w     [P]    out (may be NULL): sum_b sum_i g[b,i] d<Z_i>_b / d w[p]
 *   state_out  [B][2^n] complex out (may be NULL): final psi per sample
 *   back_psi   [B][2^n] complex out (may be NULL): psi after un-applying all gates
 *   back_lam0  [B] complex out (may be NULL): lambda[0] after un-applying all gates
 *
 * Returns 0, -1 on invalid arguments, -2 when out of memory.
 */
int oracle_run(int n, const int32_t* gates, int G, int B, int F, int P,
               const double* inputs, const double* weights, const double* grad_out,
               double* expz, double* grad_in, double* grad_w,
               double* state_out, double* back_psi, double* back_lam0)
{
    const gate_t* g = (const gate_t*)gates;
    if (B < 0 || F < 0 || P < 0 || check_circuit(n, g, G, F, P) != 0) return -1;
    if (!expz) return -1;
    const int64_t dim = (int64_t)1 << n;
    cplx* psi = (cplx*)malloc(sizeof(cplx) * (size_t)dim);
    cplx* lam = grad_out ? (cplx*)malloc(sizeof(cplx) * (size_t)dim) : NULL;
    if (!psi || (grad_out && !lam)) { free(psi); free(lam); return -2; }
    if (grad_w) memset(grad_w, 0, sizeof(double) * (size_t)P);
    if (grad_in) memset(grad_in, 0, sizeof(double) * (size_t)B * (size_t)F);

    for (int b = 0; b < B; b++) {
        const double* x_b = inputs + (size_t)b * (size_t)F;
        run_forward(psi, n, g, G, x_b, weights, -1, 0.0);
        for (int q = 0; q < n; q++) expz[(size_t)b * n + q] = expect_z(psi, dim, q);
        if (state_out) memcpy(state_out + (size_t)b * 2 * (size_t)dim, psi, sizeof(cplx) * (size_t)dim);
        if (!grad_out) continue;

        /* lambda = (sum_i g_i Z_i) psi; the observable is diagonal. */
        const double* g_b = grad_out + (size_t)b * n;
#pragma omp parallel for schedule(static) if (dim >= PAR_MIN)
        for (int64_t j = 0; j < dim; j++) {
            double d = 0.0;
            for (int q = 0; q < n; q++) d += ((j >> q) & 1) ? -g_b[q] : g_b[q];
            lam[j] = d * psi[j];
        }
        /* reverse sweep */
        for (int k = G - 1; k >= 0; k--) {
            const gate_t* gk = &g[k];
            double th = angle_of(gk, x_b, weights);
            if (gk->kind == G_RX || gk->kind == G_RY || gk->kind == G_RZ) {
                double v = im_inner(lam, psi, dim, gk->q0, gk->kind);
                if (gk->src == SRC_WEIGHT) { if (grad_w) grad_w[gk->index] += v; }
                else if (grad_in) grad_in[(size_t)b * F + gk->index] += v;
            }
            apply_gate(psi, dim, gk, th, 1);
            apply_gate(lam, dim, gk, th, 1);
        }
        if (back_psi) memcpy(back_psi + (size_t)b * 2 * (size_t)dim, psi, sizeof(cplx) * (size_t)dim);
        if (back_lam0) { back_lam0[2 * b] = creal(lam[0]); back_lam0[2 * b + 1] = cimag(lam[0]); }
    }
    free(psi);
    free(lam);
    return 0;
}

/*
 * Parameter-shift VJP (cross-check of the adjoint sweep): for every rotation
 * occurrence k, d f / d theta_k = (f(theta_k + pi/2) - f(theta_k - pi/2)) / 2
 * with f = sum_i g[b,i] <Z_i>, accumulated into the bound input or weight.
 */
int oracle_param_shift(int n, const int32_t* gates, int G, int B, int F, int P,
                       const double* inputs, const double* weights, const double* grad_out,
                       double* grad_in, double* grad_w)
{
    const gate_t* g = (const gate_t*)gates;
    if (B < 0 || F < 0 || P < 0 || !grad_out || check_circuit(n, g, G, F, P) != 0) return -1;
    const int64_t dim = (int64_t)1 << n;
    cplx* psi = (cplx*)malloc(sizeof(cplx) * (size_t)dim);
    if (!psi) return -2;
    if (grad_w) memset(grad_w, 0, sizeof(double) * (size_t)P);
    if (grad_in) memset(grad_in, 0, sizeof(double) * (size_t)B * (size_t)F);
    const double half_pi = acos(-1.0) / 2.0;
    for (int b = 0; b < B; b++) {
        const double* x_b = inputs + (size_t)b * (size_t)F;
        const double* g_b = grad_out + (size_t)b * n;
        for (int k = 0; k < G; k++) {
            if (g[k].kind != G_RX && g[k].kind != G_RY && g[k].kind != G_RZ) continue;
            double fp = 0.0, fm = 0.0;
            run_forward(psi, n, g, G, x_b, weights, k, +half_pi);
            for (int q = 0; q < n; q++) fp += g_b[q] * expect_z(psi, dim, q);
            run_forward(psi, n, g, G, x_b, weights, k, -half_pi);
            for (int q = 0; q < n; q++) fm += g_b[q] * expect_z(psi, dim, q);
            double d = 0.5 * (fp - fm);
            if (g[k].src == SRC_WEIGHT) { if (grad_w) grad_w[g[k].index] += d; }
            else if (grad_in) grad_in[(size_t)b * F + g[k].index] += d;
        }
    }
    free(psi);
    return 0;
}

/*
 * Shot sampling: the paper's measurement is Monte Carlo (a finite number of
 * shots turned into probabilities, Sec. "Quantum Node" and the appendix
 * examples). A shot draws one basis state j with probability |psi_j|^2.
 * Definition by the inverse CDF: with C(j) = sum_{i <= j} |psi_i|^2 the
 * running sum in index order (fp64) and u in [0, 1) passed in, the shot
 * returns the smallest j with C(j) > u * C(2^n - 1). A zero-probability
 * index is never returned. States: psi[B][2^n]; uniforms u[B][shots];
 * out[B][shots] (amplitude index = bitstring, qubit q = bit q). Returns -1 on
 * bad arguments or a state with zero norm.
 */
int oracle_sample(int n, int B, const double* psi_ri, int64_t shots, const double* u, int64_t* out)
{
    if (n < 0 || n > 34 || B < 0 || shots < 0 || (B > 0 && shots > 0 && (!psi_ri || !u || !out))) return -1;
    const int64_t dim = (int64_t)1 << n;
    double* cdf = (double*)malloc(sizeof(double) * (size_t)dim);
    if (!cdf) return -2;
    for (int b = 0; b < B; b++) {
        const double* p = psi_ri + (size_t)b * (size_t)dim * 2;
        double acc = 0.0;
        for (int64_t j = 0; j < dim; j++) {
            acc += p[2 * j] * p[2 * j] + p[2 * j + 1] * p[2 * j + 1];
            cdf[j] = acc;
        }
        if (!(acc > 0.0)) { free(cdf); return -1; }
        for (int64_t s = 0; s < shots; s++) {
            const double r = u[(size_t)b * (size_t)shots + (size_t)s] * acc;
            int64_t lo = 0, hi = dim - 1;  /* smallest j with cdf[j] > r; cdf[dim-1] = acc > r */
            while (lo < hi) {
                const int64_t mid = lo + (hi - lo) / 2;
                if (cdf[mid] > r) hi = mid;
                else lo = mid + 1;
            }
            out[(size_t)b * (size_t)shots + (size_t)s] = lo;
        }
    }
    free(cdf);
    return 0;
}

/* Number of OpenMP threads the parallel loops use (1 without OpenMP). */
int oracle_num_threads(void)
{
    int t = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            t = omp_get_num_threads();
#endif
        }
    }
    return t;
}
