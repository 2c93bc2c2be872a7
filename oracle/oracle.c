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
 *     (the paper's Hybrid class takes the same shifted difference);
 *   - controlled rotations CRX/CRY/CRZ(c, t) apply RX/RY/RZ to qubit t on the
 *     amplitudes whose bit c is 1 (the controlled gates of the paper's quantum
 *     autoencoder, appendix "Quantum Autoencoder"); their generator is
 *     |1><1|_c (x) P_t, so the adjoint takes Im<lambda|P_t|psi> over the
 *     control-1 amplitudes, and parameter shift takes the four-term rule for
 *     generators with eigenvalues {0, +-1/2} (Anselmetti et al. 2021):
 *     f' = d1 (f(t + pi/2) - f(t - pi/2)) - d2 (f(t + 3pi/2) - f(t - 3pi/2)),
 *     d1 = (sqrt2 + 1) / (4 sqrt2), d2 = (sqrt2 - 1) / (4 sqrt2);
 *   - initial-state embeddings (Sec. "Quantum Data"): basis embedding sets
 *     qubit q to 1 where feature first + q is >= 0.5; amplitude embedding
 *     takes psi_0 = x / |x| for the 2^n real features first .. first + 2^n - 1
 *     (a zero vector gives the zero state). The VJP with respect to those
 *     features is (2 / |x|) (Re lambda_0 - psi_0 Re<psi_0|lambda_0>), from
 *     lambda_0 = U^dagger O psi and d psi_0 / d x = (I - psi_0 psi_0^T) / |x|;
 *   - noise (Sec. "Unification of Classical and Quantum Machine", the
 *     noise-inclusive simulator) as quantum trajectories of Pauli channels:
 *     a channel on qubit q with probabilities (p_x, p_y, p_z) applies, for a
 *     uniform u in [0, 1) read from an input feature, X if u < p_x, else Y if
 *     u < p_x + p_y, else Z if u < p_x + p_y + p_z, else nothing (sums in
 *     fp64 in that order). Averaging <Z> over trajectories estimates the
 *     channel's expectation; gradients of one trajectory are those of its
 *     unitary circuit.
 *
 * Every reduction over amplitudes is a pairwise (tree) sum in fp64.
 */
#include <complex.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef double complex cplx;

enum { G_H = 0, G_RX = 1, G_RY = 2, G_RZ = 3, G_CNOT = 4, G_CZ = 5,
       G_CRX = 6, G_CRY = 7, G_CRZ = 8, G_PAULI = 9 };
enum { SRC_NONE = 0, SRC_INPUT = 1, SRC_WEIGHT = 2 };
enum { EMB_NONE = 0, EMB_BASIS = 1, EMB_AMPLITUDE = 2 };

#define PAR_MIN (1 << 14) /* run amplitude loops in parallel above this size */

typedef struct { int32_t kind, q0, q1, src, index; } gate_t;

/* ------------------------------------------------------------------ */
/* validation                                                          */

static int is_rot(int kind) { return kind == G_RX || kind == G_RY || kind == G_RZ; }
static int is_crot(int kind) { return kind == G_CRX || kind == G_CRY || kind == G_CRZ; }

static int check_source(const gate_t* x, int F, int P)
{
    if (x->src == SRC_INPUT) return (x->index < 0 || x->index >= F) ? -1 : 0;
    if (x->src == SRC_WEIGHT) return (x->index < 0 || x->index >= P) ? -1 : 0;
    return -1;
}

/* pauli_p[c][3] holds the probabilities of the c-th Pauli channel of the list. */
static int check_circuit(int n, const gate_t* g, int G, int F, int P, const double* pauli_p)
{
    if (n < 1 || n > 34 || G < 0) return -1;
    int nch = 0;
    for (int k = 0; k < G; k++) {
        const gate_t* x = &g[k];
        if (x->q0 < 0 || x->q0 >= n) return -1;
        switch (x->kind) {
        case G_H:
            if (x->src != SRC_NONE || x->q1 != -1) return -1;
            break;
        case G_RX: case G_RY: case G_RZ:
            if (x->q1 != -1 || check_source(x, F, P)) return -1;
            break;
        case G_CNOT: case G_CZ:
            if (x->src != SRC_NONE || x->q1 < 0 || x->q1 >= n || x->q1 == x->q0) return -1;
            break;
        case G_CRX: case G_CRY: case G_CRZ:
            if (x->q1 < 0 || x->q1 >= n || x->q1 == x->q0 || check_source(x, F, P)) return -1;
            break;
        case G_PAULI: {
            if (x->q1 != -1 || x->src != SRC_INPUT || x->index < 0 || x->index >= F || !pauli_p) return -1;
            const double* p = pauli_p + 3 * nch++;
            if (!(p[0] >= 0 && p[1] >= 0 && p[2] >= 0 && p[0] + p[1] + p[2] <= 1.0)) return -1;
            break;
        }
        default:
            return -1;
        }
    }
    return 0;
}

static int check_embedding(int n, int F, int embed, int first)
{
    if (embed == EMB_NONE) return 0;
    if (first < 0) return -1;
    if (embed == EMB_BASIS) return first + n <= F ? 0 : -1;
    if (embed == EMB_AMPLITUDE) return (n <= 30 && (int64_t)first + ((int64_t)1 << n) <= F) ? 0 : -1;
    return -1;
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

/* m on qubit q of the amplitudes whose bits in cmask are all 1 (cmask = 0:
 * every amplitude; a controlled rotation passes its control bit). */
static void apply_matrix(cplx* psi, int64_t dim, int64_t cmask, int q, const cplx m[4])
{
    const int64_t bit = (int64_t)1 << q;
#pragma omp parallel for schedule(static) if (dim >= PAR_MIN)
    for (int64_t j = 0; j < dim; j++) {
        if ((j & bit) || (j & cmask) != cmask) continue;
        cplx a = psi[j], b = psi[j | bit];
        psi[j] = m[0] * a + m[1] * b;
        psi[j | bit] = m[2] * a + m[3] * b;
    }
}

/* Pauli X (1), Y (2) or Z (3) on qubit q; 0 leaves psi alone. */
static void apply_pauli(cplx* psi, int64_t dim, int q, int which)
{
    const int64_t bit = (int64_t)1 << q;
    if (which == 0) return;
#pragma omp parallel for schedule(static) if (dim >= PAR_MIN)
    for (int64_t j = 0; j < dim; j++) {
        if (j & bit) continue;
        cplx a = psi[j], b = psi[j | bit];
        if (which == 1) { psi[j] = b; psi[j | bit] = a; }
        else if (which == 2) { psi[j] = -I * b; psi[j | bit] = I * a; }
        else psi[j | bit] = -b;
    }
}

/* Trajectory choice of a Pauli channel for the uniform u. */
static int pauli_outcome(double u, const double p[3])
{
    const double c1 = p[0], c2 = c1 + p[1], c3 = c2 + p[2];
    if (u < c1) return 1;
    if (u < c2) return 2;
    if (u < c3) return 3;
    return 0;
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

/* Apply gate g (dagger=1: its inverse) with the given angle; a Pauli channel
 * applies the Pauli `which` (its own inverse). */
static void apply_gate(cplx* psi, int64_t dim, const gate_t* g, double theta, int which, int dagger)
{
    if (g->kind == G_CNOT) { apply_cnot(psi, dim, g->q0, g->q1); return; }
    if (g->kind == G_CZ) { apply_cz(psi, dim, g->q0, g->q1); return; }
    if (g->kind == G_PAULI) { apply_pauli(psi, dim, g->q0, which); return; }
    cplx m[4], a[4];
    const int crot = is_crot(g->kind);
    gate_matrix(crot ? g->kind - (G_CRX - G_RX) : g->kind, theta, m);
    if (dagger) { adjoint2(m, a); memcpy(m, a, sizeof(m)); }
    if (crot) apply_matrix(psi, dim, (int64_t)1 << g->q0, g->q1, m);
    else apply_matrix(psi, dim, 0, g->q0, m);
}

/* ------------------------------------------------------------------ */
/* pairwise sums                                                       */

/* Term functions evaluated on the fly so no term array is materialised. */
typedef struct {
    const cplx* psi;
    const cplx* lam;
    int64_t bit;     /* 1 << q */
    int kind;        /* generator for inner products: X, Y or Z */
    int64_t cbit;    /* control: only amplitudes with this bit set count (0: all) */
    const double* x; /* real vector for term_dot */
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
    if (c->cbit && !(j & c->cbit)) return 0.0;
    cplx pj; /* (P_q psi)_j */
    switch (c->kind) {
    case G_RX: pj = c->psi[j ^ b]; break;
    case G_RY: pj = (j & b) ? I * c->psi[j ^ b] : -I * c->psi[j ^ b]; break;
    default:   pj = (j & b) ? -c->psi[j] : c->psi[j]; break;
    }
    return cimag(conj(c->lam[j]) * pj);
}

static double term_sq(const term_ctx* c, int64_t j) { return c->x[j] * c->x[j]; }

/* x_j * Re lam_j */
static double term_dot(const term_ctx* c, int64_t j) { return c->x[j] * creal(c->lam[j]); }

/* <Z_q> of psi. */
static double expect_z(const cplx* psi, int64_t dim, int q)
{
    term_ctx c = { psi, NULL, (int64_t)1 << q, 0, 0, NULL };
    return pairwise(&c, term_zsign_prob, dim);
}

/* Im <lam | P_t | psi> for rotation gate g (over the control-1 amplitudes of a
 * controlled rotation). */
static double im_inner(const cplx* lam, const cplx* psi, int64_t dim, const gate_t* g)
{
    const int crot = is_crot(g->kind);
    term_ctx c = { psi, lam, (int64_t)1 << (crot ? g->q1 : g->q0),
                   crot ? g->kind - (G_CRX - G_RX) : g->kind, crot ? (int64_t)1 << g->q0 : 0, NULL };
    return pairwise(&c, term_im_inner, dim);
}

/* Initial state of sample b (x_b: its features). For amplitude embedding,
 * returns |x| and writes psi_0 = x / |x|. */
static double init_state(cplx* psi, int n, int embed, int first, const double* x_b)
{
    const int64_t dim = (int64_t)1 << n;
    memset(psi, 0, sizeof(cplx) * (size_t)dim);
    if (embed == EMB_AMPLITUDE) {
        term_ctx c = { NULL, NULL, 0, 0, 0, x_b + first };
        const double r = sqrt(pairwise(&c, term_sq, dim));
        if (r > 0)
            for (int64_t j = 0; j < dim; j++) psi[j] = x_b[first + j] / r;
        return r;
    }
    int64_t idx = 0;
    if (embed == EMB_BASIS)
        for (int q = 0; q < n; q++)
            if (x_b[first + q] >= 0.5) idx |= (int64_t)1 << q;
    psi[idx] = 1.0;
    return 1.0;
}

/* Pauli outcome of gate k (a channel) for sample b; 0 for other gates. */
static int outcome_of(const gate_t* g, int G, int k, const double* x_b, const double* pauli_p)
{
    if (g[k].kind != G_PAULI) return 0;
    int c = 0;
    for (int i = 0; i < k; i++) c += g[i].kind == G_PAULI;
    return pauli_outcome(x_b[g[k].index], pauli_p + 3 * c);
}

/* ------------------------------------------------------------------ */
/* one sample                                                          */

typedef struct {
    int embed, first;       /* initial-state embedding */
    const double* pauli_p;  /* [channels][3] */
} ext_t;

static void run_forward(cplx* psi, int n, const gate_t* g, int G, const ext_t* e,
                        const double* x_b, const double* w, int shift_gate, double shift)
{
    const int64_t dim = (int64_t)1 << n;
    init_state(psi, n, e->embed, e->first, x_b);
    for (int k = 0; k < G; k++) {
        double th = angle_of(&g[k], x_b, w);
        if (k == shift_gate) th += shift;
        apply_gate(psi, dim, &g[k], th, outcome_of(g, G, k, x_b, e->pauli_p), 0);
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
int oracle_run_ext(int n, const int32_t* gates, int G, int B, int F, int P,
                   int embed, int embed_first, const double* pauli_p,
                   const double* inputs, const double* weights, const double* grad_out,
                   double* expz, double* grad_in, double* grad_w,
                   double* state_out, double* back_psi, double* back_lam0)
{
    const gate_t* g = (const gate_t*)gates;
    if (B < 0 || F < 0 || P < 0 || check_circuit(n, g, G, F, P, pauli_p) != 0) return -1;
    if (check_embedding(n, F, embed, embed_first) != 0) return -1;
    if (!expz) return -1;
    const ext_t ext = { embed, embed_first, pauli_p };
    const int64_t dim = (int64_t)1 << n;
    cplx* psi = (cplx*)malloc(sizeof(cplx) * (size_t)dim);
    cplx* lam = grad_out ? (cplx*)malloc(sizeof(cplx) * (size_t)dim) : NULL;
    if (!psi || (grad_out && !lam)) { free(psi); free(lam); return -2; }
    if (grad_w) memset(grad_w, 0, sizeof(double) * (size_t)P);
    if (grad_in) memset(grad_in, 0, sizeof(double) * (size_t)B * (size_t)F);

    for (int b = 0; b < B; b++) {
        const double* x_b = inputs + (size_t)b * (size_t)F;
        run_forward(psi, n, g, G, &ext, x_b, weights, -1, 0.0);
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
            if (is_rot(gk->kind) || is_crot(gk->kind)) {
                double v = im_inner(lam, psi, dim, gk);
                if (gk->src == SRC_WEIGHT) { if (grad_w) grad_w[gk->index] += v; }
                else if (grad_in) grad_in[(size_t)b * F + gk->index] += v;
            }
            const int which = outcome_of(g, G, k, x_b, pauli_p);
            apply_gate(psi, dim, gk, th, which, 1);
            apply_gate(lam, dim, gk, th, which, 1);
        }
        if (embed == EMB_AMPLITUDE && grad_in) {
            /* lam is now lambda_0; psi_0 = x / |x| rebuilt exactly */
            const double r = init_state(psi, n, embed, embed_first, x_b);
            if (r > 0) {
                term_ctx c = { NULL, lam, 0, 0, 0, x_b + embed_first };
                const double L = pairwise(&c, term_dot, dim) / r;
                for (int64_t j = 0; j < dim; j++)
                    grad_in[(size_t)b * F + embed_first + j] +=
                        2.0 / r * (creal(lam[j]) - creal(psi[j]) * L);
            }
        }
        if (back_psi) memcpy(back_psi + (size_t)b * 2 * (size_t)dim, psi, sizeof(cplx) * (size_t)dim);
        if (back_lam0) { back_lam0[2 * b] = creal(lam[0]); back_lam0[2 * b + 1] = cimag(lam[0]); }
    }
    free(psi);
    free(lam);
    return 0;
}

/* oracle_run_ext with the |0...0> initial state and no Pauli channels. */
int oracle_run(int n, const int32_t* gates, int G, int B, int F, int P,
               const double* inputs, const double* weights, const double* grad_out,
               double* expz, double* grad_in, double* grad_w,
               double* state_out, double* back_psi, double* back_lam0)
{
    return oracle_run_ext(n, gates, G, B, F, P, EMB_NONE, 0, NULL, inputs, weights, grad_out,
                          expz, grad_in, grad_w, state_out, back_psi, back_lam0);
}

/*
 * Parameter-shift VJP (cross-check of the adjoint sweep): for every rotation
 * occurrence k, d f / d theta_k = (f(theta_k + pi/2) - f(theta_k - pi/2)) / 2
 * (four-term rule for controlled rotations) with f = sum_i g[b,i] <Z_i>,
 * accumulated into the bound input or weight. Amplitude-embedding features get
 * no gradient here.
 */
int oracle_param_shift_ext(int n, const int32_t* gates, int G, int B, int F, int P,
                           int embed, int embed_first, const double* pauli_p,
                           const double* inputs, const double* weights, const double* grad_out,
                           double* grad_in, double* grad_w)
{
    const gate_t* g = (const gate_t*)gates;
    if (B < 0 || F < 0 || P < 0 || !grad_out || check_circuit(n, g, G, F, P, pauli_p) != 0) return -1;
    if (check_embedding(n, F, embed, embed_first) != 0) return -1;
    const ext_t ext = { embed, embed_first, pauli_p };
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
            if (!is_rot(g[k].kind) && !is_crot(g[k].kind)) continue;
            double f[4];
            const double sh[4] = { half_pi, -half_pi, 3 * half_pi, -3 * half_pi };
            const int ns = is_crot(g[k].kind) ? 4 : 2;
            for (int i = 0; i < ns; i++) {
                run_forward(psi, n, g, G, &ext, x_b, weights, k, sh[i]);
                f[i] = 0.0;
                for (int q = 0; q < n; q++) f[i] += g_b[q] * expect_z(psi, dim, q);
            }
            double d;
            if (ns == 2) {
                d = 0.5 * (f[0] - f[1]);
            } else {
                const double r2 = sqrt(2.0);
                d = (r2 + 1) / (4 * r2) * (f[0] - f[1]) - (r2 - 1) / (4 * r2) * (f[2] - f[3]);
            }
            if (g[k].src == SRC_WEIGHT) { if (grad_w) grad_w[g[k].index] += d; }
            else if (grad_in) grad_in[(size_t)b * F + g[k].index] += d;
        }
    }
    free(psi);
    return 0;
}

int oracle_param_shift(int n, const int32_t* gates, int G, int B, int F, int P,
                       const double* inputs, const double* weights, const double* grad_out,
                       double* grad_in, double* grad_w)
{
    return oracle_param_shift_ext(n, gates, G, B, F, P, EMB_NONE, 0, NULL, inputs, weights,
                                  grad_out, grad_in, grad_w);
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
