/*
 * CyFA CPU oracle -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * Only the test suite, the package smoke check and the benchmark's CPU
 * baseline may load this library.  The GPU operator never calls it, and it
 * shares no code, header or table with the GPU operator.
 *
 * It evaluates Cyclic Flow Attention in its defining relative-time-slot form,
 * token by token, in double precision:
 *
 *   real Fourier basis Phi (m odd)                 App. A.1, Eq. (app-real-fourier)
 *   U(tau) = 1 (+) Rot(2 pi j tau / m), j=1..(m-1)/2   Sec. 3.1, Eqs. (cyfa-rotation-block),
 *   P(tau) = Phi U(tau) Phi^T                                   (cyfa-fractional-shift)
 *   K_t = a_t P(delta_t) K_{t-1} + b_t e_0 k_t^T   Sec. 3.1, Eq. (cyfa-physical-recurrence)
 *   V_t = a_t P(delta_t) V_{t-1} + b_t e_0 v_t^T
 *   o_t = (R V_t)^T softmax(scale * R K_t q_t)    Sec. 3.1, Eq. (cyfa-physical-readout)
 *
 * where a_t = exp(log_alpha_t) is the scalar forget gate and b_t the write
 * strength.  The readout uses the state after token t has been written.  The
 * dot-product scale the paper leaves out of its notation is an explicit
 * argument that multiplies the slot logits.  P(delta_t) is rebuilt densely at
 * every token; nothing is blocked, fused or reordered.
 *
 * Also provided: the maps between relative-time states and absolute-clock
 * states, Kbar = U(-lambda) Phi^T K and back (App. A.4, Eq. (app-three-K)),
 * used by the tests to compare final states with the GPU operator.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

static const double kPi = 3.14159265358979323846264338327950288;

/* Phi[r*m + c]: column 0 = DC, column 2j-1 = cos_j, column 2j = sin_j. */
void cyfa_oracle_phi(int m, double *phi)
{
    const double dc = 1.0 / sqrt((double)m);
    const double ac = sqrt(2.0 / (double)m);
    for (int r = 0; r < m; ++r) {
        phi[r * m + 0] = dc;
        for (int j = 1; j <= (m - 1) / 2; ++j) {
            const double ang = 2.0 * kPi * (double)j * (double)r / (double)m;
            phi[r * m + 2 * j - 1] = ac * cos(ang);
            phi[r * m + 2 * j] = ac * sin(ang);
        }
    }
}

/* U(tau): identity on the DC coordinate, Rot(2 pi j tau / m) on pair (2j-1, 2j). */
void cyfa_oracle_rotation(int m, double tau, double *U)
{
    memset(U, 0, sizeof(double) * (size_t)m * (size_t)m);
    U[0] = 1.0;
    for (int j = 1; j <= (m - 1) / 2; ++j) {
        const double th = 2.0 * kPi * (double)j * tau / (double)m;
        const double c = cos(th), s = sin(th);
        const int a = 2 * j - 1, b = 2 * j;
        U[a * m + a] = c;
        U[a * m + b] = -s;
        U[b * m + a] = s;
        U[b * m + b] = c;
    }
}

/* C = A * B for dense row-major n x n (A, B) -- plain triple loop. */
static void matmul_sq(int n, const double *A, const double *B, double *C)
{
    for (int i = 0; i < n; ++i) {
        double *ci = C + (size_t)i * n;
        for (int j = 0; j < n; ++j) ci[j] = 0.0;
        for (int k = 0; k < n; ++k) {
            const double aik = A[(size_t)i * n + k];
            const double *bk = B + (size_t)k * n;
            for (int j = 0; j < n; ++j) ci[j] += aik * bk[j];
        }
    }
}

/* P(tau) = Phi U(tau) Phi^T, built densely.  phiT is Phi transposed;
 * work: 2*m*m doubles. */
static void shift_with(int m, double tau, const double *phi, const double *phiT,
                       double *P, double *work)
{
    double *U = work, *PU = work + (size_t)m * m;
    cyfa_oracle_rotation(m, tau, U);
    matmul_sq(m, phi, U, PU);                       /* Phi U */
    matmul_sq(m, PU, phiT, P);                      /* (Phi U) Phi^T */
}

static void transpose_sq(int n, const double *A, double *AT)
{
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) AT[(size_t)j * n + i] = A[(size_t)i * n + j];
}

void cyfa_oracle_shift(int m, double tau, double *P)
{
    double *phi = (double *)malloc(sizeof(double) * (size_t)m * m * 4);
    double *phiT = phi + (size_t)m * m;
    cyfa_oracle_phi(m, phi);
    transpose_sq(m, phi, phiT);
    shift_with(m, tau, phi, phiT, P, phiT + (size_t)m * m);
    free(phi);
}

/*
 * Run one (b, h) sequence.
 *   q: T rows of dk with row stride sq; k likewise; v: T rows of dv (stride sv).
 *   delta, la, be: T scalars with stride ss (la/be may be NULL: alpha=1 / beta=1).
 *   R: m x m (NULL: identity).  K, V: m x dk / m x dv relative-time state, in/out.
 *   o: T x dv, z: T x m (may be NULL).  lam: in/out cumulative clock.
 */
static void run_sequence(int T, int dk, int dv, int m, double scale,
                         const float *q, const float *k, const float *v, size_t sq, size_t sv,
                         const float *delta, const float *la, const float *be, size_t ss,
                         const double *R, const double *phi, const double *phiT,
                         double *K, double *V, double *o, double *z, double *lam,
                         double *work)
{
    const int dmax = dk > dv ? dk : dv;
    double *P = work;
    double *scratch = P + (size_t)m * m;            /* 2 m^2 for shift_with */
    double *tmp = scratch + 2 * (size_t)m * m;      /* m * dmax */
    double *y = tmp + (size_t)m * dmax;             /* K q           (m) */
    double *zl = y + m;                             /* logits        (m) */
    double *w = zl + m;                             /* softmax       (m) */
    double *u = w + m;                              /* R^T w         (m) */
    double *qt = u + m;                             /* query row     (dk) */

    for (int t = 0; t < T; ++t) {
        const double dlt = (double)delta[(size_t)t * ss];
        const double alpha = la ? exp((double)la[(size_t)t * ss]) : 1.0;
        const double beta = be ? (double)be[(size_t)t * ss] : 1.0;

        /* relative-time transport and insertion */
        shift_with(m, dlt, phi, phiT, P, scratch);
        for (int pass = 0; pass < 2; ++pass) {
            double *S = pass ? V : K;
            const int d = pass ? dv : dk;
            const float *x = pass ? v + (size_t)t * sv : k + (size_t)t * sq;
            for (int r = 0; r < m; ++r) {
                double *tr = tmp + (size_t)r * d;
                for (int c = 0; c < d; ++c) tr[c] = 0.0;
                for (int s = 0; s < m; ++s) {
                    const double prs = P[(size_t)r * m + s];
                    const double *srow = S + (size_t)s * d;
                    for (int c = 0; c < d; ++c) tr[c] += prs * srow[c];
                }
            }
            for (size_t i = 0; i < (size_t)m * d; ++i) S[i] = alpha * tmp[i];
            for (int c = 0; c < d; ++c) S[c] += beta * (double)x[c];
        }

        /* softmax readout through R on the updated states */
        for (int c = 0; c < dk; ++c) qt[c] = (double)q[(size_t)t * sq + c];
        for (int r = 0; r < m; ++r) {
            double acc = 0.0;
            for (int c = 0; c < dk; ++c) acc += K[(size_t)r * dk + c] * qt[c];
            y[r] = acc;
        }
        double zmax = -INFINITY;
        for (int i = 0; i < m; ++i) {
            double acc = 0.0;
            if (R) {
                for (int r = 0; r < m; ++r) acc += R[(size_t)i * m + r] * y[r];
            } else {
                acc = y[i];
            }
            zl[i] = scale * acc;
            if (zl[i] > zmax) zmax = zl[i];
        }
        double den = 0.0;
        for (int i = 0; i < m; ++i) { w[i] = exp(zl[i] - zmax); den += w[i]; }
        for (int i = 0; i < m; ++i) w[i] /= den;
        for (int r = 0; r < m; ++r) {
            double acc = 0.0;
            if (R) {
                for (int i = 0; i < m; ++i) acc += R[(size_t)i * m + r] * w[i];
            } else {
                acc = w[r];
            }
            u[r] = acc;
        }
        for (int c = 0; c < dv; ++c) {
            double acc = 0.0;
            for (int r = 0; r < m; ++r) acc += V[(size_t)r * dv + c] * u[r];
            o[(size_t)t * dv + c] = acc;
        }
        if (z) for (int i = 0; i < m; ++i) z[(size_t)t * m + i] = zl[i];
        *lam += dlt;
    }
}

/*
 * Batched entry point over [B, T, H, ...] inputs.
 *   pairs: npairs flattened indices b*H + h (NULL: all B*H in order).
 *   T_run: tokens processed per pair (<= T).
 *   K0, V0: [npairs, m, dk] / [npairs, m, dv] relative-time initial states (NULL: zero).
 *   lam0: [npairs] initial clock (NULL: 0).
 *   o: [npairs, T_run, dv]; z: [npairs, T_run, m] or NULL;
 *   K_out, V_out: [npairs, m, d] or NULL; lam_out: [npairs] or NULL.
 *   nthreads <= 0: OpenMP default.
 * Returns the number of threads used, or -1 on bad arguments.
 */
int cyfa_oracle_forward(int B, int T, int H, int dk, int dv, int m, double scale,
                        const float *q, const float *k, const float *v,
                        const float *delta, const float *log_alpha, const float *beta,
                        const float *R,
                        const double *K0, const double *V0, const double *lam0,
                        int npairs, const int32_t *pairs, int T_run,
                        double *o, double *z, double *K_out, double *V_out, double *lam_out,
                        int nthreads)
{
    if (B < 0 || T < 0 || H <= 0 || dk <= 0 || dv <= 0 || m < 3 || (m % 2) == 0) return -1;
    if (T_run < 0 || T_run > T) return -1;
    if (!pairs) npairs = B * H;
    if (npairs < 0) return -1;
    for (int p = 0; p < npairs && pairs; ++p)
        if (pairs[p] < 0 || pairs[p] >= B * H) return -1;

    const size_t mm = (size_t)m * m;
    double *phi = (double *)malloc(sizeof(double) * mm * 2);
    double *phiT = phi + mm;
    double *Rd = R ? (double *)malloc(sizeof(double) * mm * (size_t)H) : NULL;
    cyfa_oracle_phi(m, phi);
    transpose_sq(m, phi, phiT);
    if (Rd) for (size_t i = 0; i < mm * (size_t)H; ++i) Rd[i] = (double)R[i];

    int used = 1;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
    const int dmax = dk > dv ? dk : dv;
    const size_t wsz = 3 * mm + (size_t)m * dmax + 4 * (size_t)m + (size_t)dk;

#pragma omp parallel
    {
#ifdef _OPENMP
#pragma omp single
        used = omp_get_num_threads();
#endif
        double *work = (double *)malloc(sizeof(double) * wsz);
        double *K = (double *)malloc(sizeof(double) * (size_t)m * dk);
        double *V = (double *)malloc(sizeof(double) * (size_t)m * dv);
#pragma omp for schedule(dynamic, 1)
        for (int p = 0; p < npairs; ++p) {
            const int bh = pairs ? pairs[p] : p;
            const int b = bh / H, h = bh % H;
            if (K0) memcpy(K, K0 + (size_t)p * m * dk, sizeof(double) * (size_t)m * dk);
            else memset(K, 0, sizeof(double) * (size_t)m * dk);
            if (V0) memcpy(V, V0 + (size_t)p * m * dv, sizeof(double) * (size_t)m * dv);
            else memset(V, 0, sizeof(double) * (size_t)m * dv);
            double lam = lam0 ? lam0[p] : 0.0;
            const size_t base = (size_t)b * T * H + h;          /* scalar index at t=0 */
            run_sequence(T_run, dk, dv, m, scale,
                         q + base * dk, k + base * dk, v + base * dv,
                         (size_t)H * dk, (size_t)H * dv,
                         delta + base, log_alpha ? log_alpha + base : NULL,
                         beta ? beta + base : NULL, (size_t)H,
                         Rd ? Rd + (size_t)h * mm : NULL, phi, phiT, K, V,
                         o + (size_t)p * T_run * dv, z ? z + (size_t)p * T_run * m : NULL,
                         &lam, work);
            if (K_out) memcpy(K_out + (size_t)p * m * dk, K, sizeof(double) * (size_t)m * dk);
            if (V_out) memcpy(V_out + (size_t)p * m * dv, V, sizeof(double) * (size_t)m * dv);
            if (lam_out) lam_out[p] = lam;
        }
        free(work);
        free(K);
        free(V);
    }
    free(phi);
    free(Rd);
    return used;
}

/* Relative-time state (m x d) -> absolute-clock state: Kbar = U(-lam) Phi^T K. */
void cyfa_oracle_to_absolute(int m, int d, double lam, const double *K, double *Kbar)
{
    double *phi = (double *)malloc(sizeof(double) * (size_t)m * m * 2);
    double *U = phi + (size_t)m * m;
    double *hat = (double *)malloc(sizeof(double) * (size_t)m * d);
    cyfa_oracle_phi(m, phi);
    cyfa_oracle_rotation(m, -lam, U);
    for (int i = 0; i < m; ++i)
        for (int c = 0; c < d; ++c) {
            double acc = 0.0;
            for (int r = 0; r < m; ++r) acc += phi[(size_t)r * m + i] * K[(size_t)r * d + c];
            hat[(size_t)i * d + c] = acc;
        }
    for (int i = 0; i < m; ++i)
        for (int c = 0; c < d; ++c) {
            double acc = 0.0;
            for (int j = 0; j < m; ++j) acc += U[(size_t)i * m + j] * hat[(size_t)j * d + c];
            Kbar[(size_t)i * d + c] = acc;
        }
    free(hat);
    free(phi);
}

/* Absolute-clock state -> relative-time state: K = Phi U(lam) Kbar. */
void cyfa_oracle_to_relative(int m, int d, double lam, const double *Kbar, double *K)
{
    double *phi = (double *)malloc(sizeof(double) * (size_t)m * m * 2);
    double *U = phi + (size_t)m * m;
    double *hat = (double *)malloc(sizeof(double) * (size_t)m * d);
    cyfa_oracle_phi(m, phi);
    cyfa_oracle_rotation(m, lam, U);
    for (int i = 0; i < m; ++i)
        for (int c = 0; c < d; ++c) {
            double acc = 0.0;
            for (int j = 0; j < m; ++j) acc += U[(size_t)i * m + j] * Kbar[(size_t)j * d + c];
            hat[(size_t)i * d + c] = acc;
        }
    for (int r = 0; r < m; ++r)
        for (int c = 0; c < d; ++c) {
            double acc = 0.0;
            for (int i = 0; i < m; ++i) acc += phi[(size_t)r * m + i] * hat[(size_t)i * d + c];
            K[(size_t)r * d + c] = acc;
        }
    free(hat);
    free(phi);
}
