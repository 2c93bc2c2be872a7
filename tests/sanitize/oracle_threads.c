/* Driver of the CPU oracle for the ThreadSanitizer run of
 * tests/test_sanitizers.py: a 16-qubit random circuit (parallel amplitude
 * loops, chunked pairwise sums), forward + adjoint + parameter shift, in the
 * thread count OpenMP is given. Prints the results as hex words, so that runs
 * with different thread counts can be compared bit for bit. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

int oracle_run_ext(int n, const int32_t* gates, int G, int B, int F, int P, int embed, int first,
                   const double* pauli_p, const double* x, const double* w, const double* g, double* expz,
                   double* grad_x, double* grad_w, double* state, double* back_psi, double* back_lam0);
int oracle_param_shift_ext(int n, const int32_t* gates, int G, int B, int F, int P, int embed, int first,
                           const double* pauli_p, const double* x, const double* w, const double* g,
                           double* grad_x, double* grad_w);

static uint64_t rng = 0x9e3779b97f4a7c15ull;
static uint64_t next(void) {
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return rng;
}
static double unif(void) { return (double)(next() >> 11) / 9007199254740992.0; }

int main(void) {
    enum { N = 16, G = 40, F = 3, P = 5, NCH = 1 };
    int32_t gates[G * 5];
    for (int k = 0; k < G; k++) {
        int32_t* q = gates + 5 * k;
        const int kind = k == G - 1 ? 9 : (int)(next() % 9);
        q[0] = kind;
        q[1] = (int)(next() % N);
        q[2] = -1;
        q[3] = 0;
        q[4] = 0;
        if (kind == 4 || kind == 5 || kind >= 6) {
            if (kind != 9) {
                q[2] = (q[1] + 1 + (int)(next() % (N - 1))) % N;
            }
        }
        if (kind == 1 || kind == 2 || kind == 3 || (kind >= 6 && kind <= 8)) {
            q[3] = (next() & 1) ? 1 : 2;
            q[4] = q[3] == 1 ? (int)(next() % F) : (int)(next() % P);
        }
        if (kind == 9) {
            q[3] = 1;
            q[4] = F - 1;
        }
    }
    double x[F], w[P], g[N], expz[N], gx[F], gw[P], sx[F], sw[P];
    const double pp[3 * NCH] = {0.1, 0.2, 0.3};
    for (int i = 0; i < F; i++) x[i] = 3.0 * unif();
    for (int i = 0; i < P; i++) w[i] = 6.0 * unif() - 3.0;
    for (int i = 0; i < N; i++) g[i] = 2.0 * unif() - 1.0;
    memset(gx, 0, sizeof gx);
    memset(gw, 0, sizeof gw);
    memset(sx, 0, sizeof sx);
    memset(sw, 0, sizeof sw);
    int rc = oracle_run_ext(N, gates, G, 1, F, P, 0, 0, pp, x, w, g, expz, gx, gw, NULL, NULL, NULL);
    if (rc) return 10 + rc;
    rc = oracle_param_shift_ext(N, gates, G, 1, F, P, 0, 0, pp, x, w, g, sx, sw);
    if (rc) return 20 + rc;
    const double* all[] = {expz, gx, gw, sx, sw};
    const int len[] = {N, F, P, F, P};
    for (int a = 0; a < 5; a++)
        for (int i = 0; i < len[a]; i++) {
            uint64_t u;
            memcpy(&u, &all[a][i], 8);
            printf("%016llx\n", (unsigned long long)u);
        }
    return 0;
}
