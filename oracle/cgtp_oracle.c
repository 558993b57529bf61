/*
 * cgtp oracle: plain, slow, fp64 CPU definition of the contracted Clebsch-Gordan
 * products computed by the GPU library.
 *
 * TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load this code. The product path never does.
 * It shares no code, header, table or constant with the HIP library: it is built
 * from this file alone by gcc.
 *
 * What it computes (Bochkarev, Lysogorskiy, Drautz, "Fast contracted
 * Clebsch-Gordan tensor products for equivariant graph neural networks"):
 *
 *   on-site   (Eq. phi-cg with the CP form Eq. cp-decomp):
 *     H1[r][k1] = sum_n U_A[l1][n][r] A[n][k1],  H2 likewise with U_B, B
 *     Ta[r][k]  = sum_{k1,k2} GR[k1][k2][k] H1[r][k1] H2[r][k2]   (Category alpha)
 *     Tb[r][k]  = sum_{k1,k2} QR[k1][k2][k] H1[r][k1] H2[r][k2]   (Category beta)
 *     out_even[n][k] = sum_r U_oe[l][n][r] Ta[r][k],  out_odd likewise with Tb
 *
 *   message passing (Eq. msgpass-parity-start; edge factor R*Y as in
 *   Eq. msgpass-tildeR), natural-parity node slot:
 *     E_e[r][k1] = (sum_n U_E[l1][n][r] Rad_e[n][l1]) * Y_k1(rhat_e)
 *     H_j[r][k2] = sum_n U_I[l2][n][r] I_j[n][k2]
 *     Ta_i[r][k] = sum_{e=(j->i)} sum GR E_e H_j,  Tb_i likewise with QR
 *
 *   General parity (Eqs. msgpass-cp-alpha / msgpass-cp-beta, Table 1, Cases A-D):
 *   the Gaunt and curl couplings may carry their own input factors (U_*_curl
 *   for the curl one; NULL means the Gaunt factor), and an operand may carry a
 *   parity-flipped slot (parity -(-1)^l) beside its natural one. Parity is
 *   multiplicative: a pair of slots of equal relative parity sends its Gaunt
 *   coupling to out_even (parity (-1)^l) and its curl coupling to out_odd, a
 *   mixed pair the other way round. The edge factor has natural parity.
 *
 * GR and QR are the real-basis triple integrals
 *     GR[k1][k2][k] = int Y_k1 Y_k2 Y_k dOmega                 (Eq. gaunt)
 *     QR[k1][k2][k] = int {Y_k1, Y_k2} Y_k dOmega              (Eq. Q-def)
 * with {A,B} the spherical Poisson bracket (Eq. poisson-S2), first operand A.
 * They are formed from the complex tables of Eq. cg-integral and Eq. Q-CG
 * (kappa^-1 from Eq. kappa-inv-closed, kept on the parity-odd support only)
 * by the unitary map of App. C, Eq. realY.
 *
 * Real basis (App. C, Eq. realY), no Condon-Shortley phase in Ptilde:
 *     Y_{l,m>0} = sqrt2 Pt_l^m(cos th) cos(m ph),  Y_{l,0} = Pt_l^0,
 *     Y_{l,m<0} = sqrt2 Pt_l^|m| sin(|m| ph),  Pt_l^m = N_lm P_l^m,
 *     N_lm = sqrt((2l+1)/(4 pi) (l-m)!/(l+m)!);  flattened index k = l*l + l + m.
 *
 * Parity pins (tests under -m "not gpu"): 3j against exact sympy values and the
 * closed form Eq. cg-explicit/triangle; CG orthogonality; kappa^-1 against the
 * values printed in App. A and App. B; GR/QR against brute-force dense-grid
 * quadrature with finite-difference surface gradients; the {x,y}=z bracket;
 * symmetry/antisymmetry and parity supports; Jacobi identity; end-to-end
 * rotation/inversion equivariance; self-coupled vanishing; dense-grid brute force
 * of the on-site and message-passing sums at tiny sizes.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <complex.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_MAXJ 64
#define ORC_FOURPI (4.0L * 3.14159265358979323846264338327950288L)

static long double g_fact[4 * ORC_MAXJ + 8];
static int g_fact_ready = 0;

static void init_fact(void)
{
    if (g_fact_ready) return;
    g_fact[0] = 1.0L;
    for (int i = 1; i < (int)(sizeof(g_fact) / sizeof(g_fact[0])); ++i)
        g_fact[i] = g_fact[i - 1] * (long double)i;
    g_fact_ready = 1;
}

static int imax(int a, int b) { return a > b ? a : b; }
static int imin(int a, int b) { return a < b ? a : b; }
static long double parity_sign(int n) { return (n % 2 == 0) ? 1.0L : -1.0L; }

/* Wigner 3j symbol (j1 j2 j3; m1 m2 m3) by the Racah formula, long double. */
static long double w3j_ld(int j1, int j2, int j3, int m1, int m2, int m3)
{
    init_fact();
    if (m1 + m2 + m3 != 0) return 0.0L;
    if (j1 < 0 || j2 < 0 || j3 < 0) return 0.0L;
    if (j3 < abs(j1 - j2) || j3 > j1 + j2) return 0.0L;
    if (abs(m1) > j1 || abs(m2) > j2 || abs(m3) > j3) return 0.0L;
    if (j1 + j2 + j3 + 1 >= (int)(sizeof(g_fact) / sizeof(g_fact[0]))) return NAN;
    long double tri = g_fact[j1 + j2 - j3] * g_fact[j1 - j2 + j3] * g_fact[-j1 + j2 + j3]
                      / g_fact[j1 + j2 + j3 + 1];
    long double pre = sqrtl(tri) * sqrtl(g_fact[j1 + m1] * g_fact[j1 - m1] * g_fact[j2 + m2]
                                         * g_fact[j2 - m2] * g_fact[j3 + m3] * g_fact[j3 - m3]);
    int kmin = imax(0, imax(j2 - j3 - m1, j1 - j3 + m2));
    int kmax = imin(j1 + j2 - j3, imin(j1 - m1, j2 + m2));
    long double s = 0.0L;
    for (int k = kmin; k <= kmax; ++k) {
        long double den = g_fact[k] * g_fact[j3 - j2 + k + m1] * g_fact[j3 - j1 + k - m2]
                          * g_fact[j1 + j2 - j3 - k] * g_fact[j1 - k - m1] * g_fact[j2 - k + m2];
        s += parity_sign(k) / den;
    }
    return parity_sign(j1 - j2 - m3) * pre * s;
}

double cgo_wigner3j(int j1, int j2, int j3, int m1, int m2, int m3)
{
    return (double)w3j_ld(j1, j2, j3, m1, m2, m3);
}

/* Clebsch-Gordan coefficient G^{lm}_{l1m1 l2m2} = <l1 m1 l2 m2 | l m>, via the
 * standard 3j relation (Condon-Shortley convention). */
static long double cg_ld(int l1, int m1, int l2, int m2, int l, int m)
{
    if (m1 + m2 != m) return 0.0L;
    return parity_sign(l1 - l2 + m) * sqrtl((long double)(2 * l + 1))
           * w3j_ld(l1, l2, l, m1, m2, -m);
}

double cgo_cg(int l1, int m1, int l2, int m2, int l, int m)
{
    return (double)cg_ld(l1, m1, l2, m2, l, m);
}

/* Eq. cg-integral: int Y_{l1m1} Y_{l2m2} Y*_{lm} dOmega (complex, CS phase). */
static long double gaunt_conj_ld(int l1, int m1, int l2, int m2, int l, int m)
{
    long double pref = sqrtl((long double)((2 * l1 + 1) * (2 * l2 + 1))
                             / (ORC_FOURPI * (long double)(2 * l + 1)));
    return pref * cg_ld(l1, 0, l2, 0, l, 0) * cg_ld(l1, m1, l2, m2, l, m);
}

double cgo_gaunt_conj(int l1, int m1, int l2, int m2, int l, int m)
{
    return (double)gaunt_conj_ld(l1, m1, l2, m2, l, m);
}

/* Eq. kappa-inv-closed, imaginary part. The closed form is used only on the
 * parity-odd support l1+l2+l odd with l1, l2 >= 1 (App. A, step 3 fixes
 * kappa^-1 = 0 on the even support; the 3j with bottom row (-1 1 0) itself is
 * not zero there, so the support is imposed explicitly). */
static long double kappa_inv_im_ld(int l1, int l2, int l)
{
    if (((l1 + l2 + l) & 1) == 0) return 0.0L;
    if (l1 < 1 || l2 < 1) return 0.0L;
    if (l < abs(l1 - l2) || l > l1 + l2) return 0.0L;
    long double r = sqrtl((long double)(2 * l1 + 1) * (2 * l2 + 1) * l1 * (l1 + 1) * l2 * (l2 + 1)
                          / ORC_FOURPI);
    return -parity_sign(l1 - l2) * r * w3j_ld(l1, l2, l, -1, 1, 0);
}

double cgo_kappa_inv_im(int l1, int l2, int l)
{
    return (double)kappa_inv_im_ld(l1, l2, l);
}

/* Eq. Q-CG: int Y*_{lm} {Y_{l1m1}, Y_{l2m2}} dOmega = kappa^-1 G^{lm}_{l1m1 l2m2};
 * purely imaginary, the imaginary part is returned. */
static long double curl_conj_im_ld(int l1, int m1, int l2, int m2, int l, int m)
{
    return kappa_inv_im_ld(l1, l2, l) * cg_ld(l1, m1, l2, m2, l, m);
}

double cgo_curl_conj_im(int l1, int m1, int l2, int m2, int l, int m)
{
    return (double)curl_conj_im_ld(l1, m1, l2, m2, l, m);
}

/* Unitary map of App. C: Y^R_{l,m} = sum_mu U[m][mu] Y_{l,mu} (CS complex Y).
 *   m > 0:  ((-1)^m Y_m + Y_{-m}) / sqrt2
 *   m = 0:  Y_0
 *   m < 0:  -i ((-1)^|m| Y_|m| - Y_-|m|) / sqrt2
 * Returns the coefficient of Y_mu in Y^R_m. */
static long double complex real_from_complex(int m, int mu)
{
    const long double s = 1.0L / sqrtl(2.0L);
    if (m == 0) return (mu == 0) ? 1.0L : 0.0L;
    if (m > 0) {
        if (mu == m) return parity_sign(m) * s;
        if (mu == -m) return s;
        return 0.0L;
    }
    int k = -m;
    if (mu == k) return -I * parity_sign(k) * s;
    if (mu == -k) return I * s;
    return 0.0L;
}

/* Unconjugated complex triple integrals of the CS basis, from the conjugated
 * ones via Y_{l,mu} = (-1)^mu conj(Y_{l,-mu}). */
static long double complex gaunt_c(int l1, int m1, int l2, int m2, int l3, int m3)
{
    return parity_sign(m3) * gaunt_conj_ld(l1, m1, l2, m2, l3, -m3);
}

static long double complex curl_c(int l1, int m1, int l2, int m2, int l3, int m3)
{
    return parity_sign(m3) * I * curl_conj_im_ld(l1, m1, l2, m2, l3, -m3);
}

/* Real-basis table entry int Y^R_{k1} (op) Y^R_{k2} Y^R_{k3}: the full unitary
 * sum over (mu1, mu2, mu3), where each Y^R is a combination of Y_{+-|m|}.
 * kind 0: Gaunt (product), kind 1: Poisson bracket. Imaginary residue is
 * reported through *im. */
static long double real_entry(int kind, int l1, int m1, int l2, int m2, int l3, int m3,
                              long double *im)
{
    long double complex acc = 0.0L;
    int mus1[2] = {abs(m1), -abs(m1)};
    int mus2[2] = {abs(m2), -abs(m2)};
    int mus3[2] = {abs(m3), -abs(m3)};
    for (int a = 0; a < (m1 == 0 ? 1 : 2); ++a)
        for (int b = 0; b < (m2 == 0 ? 1 : 2); ++b)
            for (int c = 0; c < (m3 == 0 ? 1 : 2); ++c) {
                int mu1 = mus1[a], mu2 = mus2[b], mu3 = mus3[c];
                if (mu1 + mu2 + mu3 != 0) continue;
                long double complex u = real_from_complex(m1, mu1) * real_from_complex(m2, mu2)
                                        * real_from_complex(m3, mu3);
                long double complex t = (kind == 0) ? gaunt_c(l1, mu1, l2, mu2, l3, mu3)
                                                    : curl_c(l1, mu1, l2, mu2, l3, mu3);
                acc += u * t;
            }
    if (im) *im = cimagl(acc);
    return creall(acc);
}

double cgo_real_entry(int kind, int l1, int m1, int l2, int m2, int l3, int m3, double *im)
{
    long double imv = 0.0L;
    long double v = real_entry(kind, l1, m1, l2, m2, l3, m3, &imv);
    if (im) *im = (double)imv;
    return (double)v;
}

/* Entries of one l1 block, appended at arrays + n (count only when val is NULL). */
static long real_table_block(int kind, int l1, int l2max, int lmax_out, int32_t *k1,
                             int32_t *k2, int32_t *k3, double *val, long n, long double *worst_im)
{
    for (int m1 = -l1; m1 <= l1; ++m1)
        for (int l2 = 0; l2 <= l2max; ++l2)
            for (int m2 = -l2; m2 <= l2; ++m2)
                for (int l3 = abs(l1 - l2); l3 <= imin(l1 + l2, lmax_out); ++l3)
                    for (int m3 = -l3; m3 <= l3; ++m3) {
                        int am = abs(m3);
                        /* only |m3| = |m1|+|m2| or ||m1|-|m2|| can pair with mu1+mu2+mu3=0 */
                        if (am != abs(m1) + abs(m2) && am != abs(abs(m1) - abs(m2))) continue;
                        long double im = 0.0L;
                        long double v = real_entry(kind, l1, m1, l2, m2, l3, m3, &im);
                        if (fabsl(im) > *worst_im) *worst_im = fabsl(im);
                        if (fabsl(v) <= 1e-12L) continue;
                        if (val) {
                            k1[n] = l1 * l1 + l1 + m1;
                            k2[n] = l2 * l2 + l2 + m2;
                            k3[n] = l3 * l3 + l3 + m3;
                            val[n] = (double)v;
                        }
                        ++n;
                    }
    return n;
}

/* Sparse real table over all k1, k2 <= lmax_in and k3 <= lmax_out:
 * entries (k1, k2, k3, value) with |value| > 1e-12. Entries that vanish exactly
 * (e.g. an odd number of sine factors under the phi integral) come out of the
 * unitary sum as cancellation residue of at most ~1e-15, while every genuine
 * entry up to lmax = 20 is above 9e-7, so the cut only removes residue. When
 * arrays are NULL (or cap is short) only the count is returned. max_imag receives the largest
 * |Im| seen (must be ~0: the real-basis tables are real). */
/* Entries with l1 <= l1max, l2 <= l2max and l3 <= lmax_out (see cgo_real_table). */
static long real_table(int kind, int l1max, int l2max, int lmax_out, int32_t *k1, int32_t *k2,
                       int32_t *k3, double *val, long cap, double *max_imag)
{
    init_fact();
    long counts[ORC_MAXJ + 1];
    long double worst[ORC_MAXJ + 1];
    if (l1max > ORC_MAXJ || l2max > ORC_MAXJ || lmax_out > ORC_MAXJ) return -1;
    /* pass 1: entries per l1 block (blocks are independent) */
#pragma omp parallel for schedule(dynamic, 1)
    for (int l1 = 0; l1 <= l1max; ++l1) {
        worst[l1] = 0.0L;
        counts[l1] = real_table_block(kind, l1, l2max, lmax_out, NULL, NULL, NULL, NULL, 0,
                                      &worst[l1]);
    }
    long total = 0;
    long start[ORC_MAXJ + 1];
    long double worst_im = 0.0L;
    for (int l1 = 0; l1 <= l1max; ++l1) {
        start[l1] = total;
        total += counts[l1];
        if (worst[l1] > worst_im) worst_im = worst[l1];
    }
    /* pass 2: fill each block at its offset, in the same (l1, m1, l2, m2, l3, m3) order */
    if (val && cap >= total) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int l1 = 0; l1 <= l1max; ++l1) {
            long double w = 0.0L;
            real_table_block(kind, l1, l2max, lmax_out, k1, k2, k3, val, start[l1], &w);
        }
    }
    if (max_imag) *max_imag = (double)worst_im;
    return total;
}

/* Sparse real table over all k1, k2 <= lmax_in and k3 <= lmax_out:
 * entries (k1, k2, k3, value) with |value| > 1e-12. Entries that vanish exactly
 * (e.g. an odd number of sine factors under the phi integral) come out of the
 * unitary sum as cancellation residue of at most ~1e-15, while every genuine
 * entry up to lmax = 20 is above 9e-7, so the cut only removes residue. When
 * arrays are NULL (or cap is short) only the count is returned. max_imag receives the largest
 * |Im| seen (must be ~0: the real-basis tables are real). */
long cgo_real_table(int kind, int lmax_in, int lmax_out, int32_t *k1, int32_t *k2, int32_t *k3,
                    double *val, long cap, double *max_imag)
{
    return real_table(kind, lmax_in, lmax_in, lmax_out, k1, k2, k3, val, cap, max_imag);
}

/* Real spherical harmonics of App. C, Eq. realY, in the direction of (x, y, z):
 * out[l*l + l + m] for l <= lmax. Associated Legendre P_l^m (no CS phase) by the
 * textbook recurrences in long double:
 *   P_m^m = (2m-1)!! (1-t^2)^{m/2},  P_{m+1}^m = (2m+1) t P_m^m,
 *   (l-m) P_l^m = (2l-1) t P_{l-1}^m - (l+m-1) P_{l-2}^m. */
void cgo_real_sh(int lmax, double x, double y, double z, double *out)
{
    init_fact();
    /* only the direction matters: fp32-rounded unit vectors are renormalized */
    long double nrm = sqrtl((long double)x * x + (long double)y * y + (long double)z * z);
    long double t = (nrm > 0.0L) ? (long double)z / nrm : 1.0L;
    long double st = sqrtl(fmaxl(0.0L, 1.0L - t * t));
    long double phi = atan2l((long double)y, (long double)x);
    for (int m = 0; m <= lmax; ++m) {
        long double pmm = 1.0L;
        for (int i = 1; i <= m; ++i) pmm *= (long double)(2 * i - 1) * st;
        long double p_lm2 = 0.0L, p_lm1 = pmm;
        for (int l = m; l <= lmax; ++l) {
            long double p;
            if (l == m) p = pmm;
            else if (l == m + 1) p = (long double)(2 * m + 1) * t * pmm;
            else p = ((long double)(2 * l - 1) * t * p_lm1 - (long double)(l + m - 1) * p_lm2)
                     / (long double)(l - m);
            if (l > m) { p_lm2 = p_lm1; p_lm1 = p; }
            long double nlm = sqrtl((long double)(2 * l + 1) / ORC_FOURPI * g_fact[l - m]
                                    / g_fact[l + m]);
            long double pt = nlm * p;
            if (m == 0) {
                out[l * l + l] = (double)pt;
            } else {
                out[l * l + l + m] = (double)(sqrtl(2.0L) * pt * cosl((long double)m * phi));
                out[l * l + l - m] = (double)(sqrtl(2.0L) * pt * sinl((long double)m * phi));
            }
        }
    }
}

/* ---------------------------------------------------------------------------
 * Contracted products. Tables are built per call (plain and slow by design).
 * ------------------------------------------------------------------------- */

typedef struct {
    long n;
    int32_t *k1, *k2, *k3;
    double *v;
} sparse_tab;

static int build_tab3(int kind, int l1max, int l2max, int lomax, sparse_tab *t)
{
    t->n = real_table(kind, l1max, l2max, lomax, NULL, NULL, NULL, NULL, 0, NULL);
    if (t->n < 0) return -1;
    long n = t->n > 0 ? t->n : 1;
    t->k1 = (int32_t *)malloc(sizeof(int32_t) * n);
    t->k2 = (int32_t *)malloc(sizeof(int32_t) * n);
    t->k3 = (int32_t *)malloc(sizeof(int32_t) * n);
    t->v = (double *)malloc(sizeof(double) * n);
    if (!t->k1 || !t->k2 || !t->k3 || !t->v) return -1;
    real_table(kind, l1max, l2max, lomax, t->k1, t->k2, t->k3, t->v, t->n, NULL);
    return 0;
}

static int build_tab(int kind, int lmax, sparse_tab *t)
{
    return build_tab3(kind, lmax, lmax, lmax, t);
}

static void free_tab(sparse_tab *t)
{
    free(t->k1); free(t->k2); free(t->k3); free(t->v);
}

static int degree_of(int k)
{
    int l = 0;
    while ((l + 1) * (l + 1) <= k) ++l;
    return l;
}

/* One CP rank r of Eq. struct-H: H[k] = sum_n U[l(k)][n][r] X[n][k], X is [C][L^2]. */
static void channel_contract_r(int lmax, int C, int R, int r, const double *U, const double *X,
                               double *H)
{
    int L2 = (lmax + 1) * (lmax + 1);
    for (int k = 0; k < L2; ++k) {
        int l = degree_of(k);
        double s = 0.0;
        for (int n = 0; n < C; ++n) s += U[((size_t)l * C + n) * R + r] * X[(size_t)n * L2 + k];
        H[k] = s;
    }
}

/* out[n][k] = sum_r U[l(k)][n][r] T[r][k]  (structured pipeline, Eq. struct-phi). */
static void project_out(int lmax, int C, int R, const double *U, const double *T, double *out)
{
    int L2 = (lmax + 1) * (lmax + 1);
    for (int n = 0; n < C; ++n)
        for (int k = 0; k < L2; ++k) {
            int l = degree_of(k);
            double s = 0.0;
            for (int r = 0; r < R; ++r) s += U[((size_t)l * C + n) * R + r] * T[(size_t)r * L2 + k];
            out[(size_t)n * L2 + k] = s;
        }
}

/* T[k3] += sum_entries v * X1[k1] * X2[k2]  (the explicit sparse sum, one rank). */
static void sparse_couple(const sparse_tab *t, const double *X1, const double *X2, double *T)
{
    for (long e = 0; e < t->n; ++e) T[t->k3[e]] += t->v[e] * X1[t->k1[e]] * X2[t->k2[e]];
}

static int set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
    return omp_get_max_threads();
#else
    (void)nthreads;
    return 1;
#endif
}

/* Projection of Ta/Tb [n][R][L^2] to out_even/out_odd [n][C][L^2]. */
/* Factor blocks (Eqs. msgpass-cp-alpha and msgpass-cp-beta): the model parameterizes the
 * couplings of each category (0: Gaunt, Category alpha; 1: surface curl, Category beta) and
 * each output parity sector (0: out_even, parity (-1)^l; 1: out_odd, parity -(-1)^l) with
 * their own input factors and output weights. Block b = 2 * category + sector. */
#define CGO_NB 4

/* out_s[n][k] = sum_{cat} sum_r Uo[2 cat + s][l(k)][n][r] T[2 cat + s][r][k]; a block with
 * no coupling routed to it (live[b] == 0) holds zeros and is skipped. */
static void project_blocks(int lmax, int C, int R, long n, const double *const *Uo,
                           double *const *T, const int *live, double *out_even, double *out_odd)
{
    int L2 = (lmax + 1) * (lmax + 1);
    double *outs[2] = {out_even, out_odd};
#pragma omp parallel
    {
        double *tmp = (double *)malloc(sizeof(double) * (size_t)C * L2);
#pragma omp for schedule(static)
        for (long i = 0; i < n; ++i)
            for (int sec = 0; sec < 2; ++sec) {
                if (!outs[sec]) continue;
                double *o = outs[sec] + (size_t)i * C * L2;
                memset(o, 0, sizeof(double) * (size_t)C * L2);
                for (int cat = 0; cat < 2; ++cat) {
                    int b = 2 * cat + sec;
                    if (!live[b] || !tmp) continue;
                    project_out(lmax, C, R, Uo[b], T[b] + (size_t)i * R * L2, tmp);
                    for (size_t q = 0; q < (size_t)C * L2; ++q) o[q] += tmp[q];
                }
            }
        free(tmp);
    }
}

/* Block receiving the coupling of category cat for a slot pair of relative parity rel
 * (0: equal slots, 1: mixed): by p = p1 p2 with the Gaunt coupling keeping the
 * parity-of-degree rule and the curl coupling reversing it (Table 1), Gaunt sends equal
 * pairs to the natural sector and mixed pairs to the opposite one; curl the other way. */
static int block_of(int cat, int rel)
{
    int sec = cat ? !rel : rel;
    return 2 * cat + sec;
}

/* On-site contraction for nodes [0, n_nodes). Arrays (fp64, row-major):
 *   A, B: [N][C][L^2] natural-parity slots of the two operands;
 *   A_flip, B_flip: NULL, or the parity-flipped slots [N][C][L^2];
 *   U_A[b], U_B[b]: [L][C][R] input factors of block b (the four may alias);
 *   U_out[b]: [L][C][R] output weights of block b;
 *   out_even, out_odd: [N][C][L^2] (either may be NULL).
 * Every slot pair (s1, s2) of the operands contributes its Gaunt and its curl coupling, each
 * computed with the factors of the block it is routed to (block_of).
 * Every (node, rank) pair is independent; they are spread over the threads. */
int cgo_onsite(int lmax, int C, int R, long n_nodes, const double *A, const double *A_flip,
               const double *B, const double *B_flip, const double *const *U_A,
               const double *const *U_B, const double *const *U_out, double *out_even,
               double *out_odd, int nthreads)
{
    if (lmax < 0 || C < 1 || R < 1 || n_nodes < 0) return -1;
    set_threads(nthreads);
    int L2 = (lmax + 1) * (lmax + 1);
    const double *X1[2] = {A, A_flip}, *X2[2] = {B, B_flip};
    int live[CGO_NB] = {0, 0, 0, 0};
    for (int s1 = 0; s1 < 2; ++s1)
        for (int s2 = 0; s2 < 2; ++s2)
            if (X1[s1] && X2[s2])
                for (int cat = 0; cat < 2; ++cat) {
                    int b = block_of(cat, s1 != s2);
                    if ((b & 1) ? out_odd != NULL : out_even != NULL) live[b] = 1;
                }
    sparse_tab G, Q;
    if (build_tab(0, lmax, &G) || build_tab(1, lmax, &Q)) return -2;
    double *T[CGO_NB];
    int err = 0;
    for (int b = 0; b < CGO_NB; ++b) {
        T[b] = (double *)calloc(live[b] ? (size_t)n_nodes * R * L2 + 1 : 1, sizeof(double));
        if (!T[b]) err = -2;
    }
    if (!err) {
#pragma omp parallel
        {
            double *h1 = (double *)malloc(sizeof(double) * 2 * L2), *h2 = h1 ? h1 + L2 : NULL;
            if (!h1) {
#pragma omp atomic write
                err = -2;
            } else {
#pragma omp for schedule(dynamic, 4)
                for (long ir = 0; ir < n_nodes * R; ++ir) {
                    long i = ir / R;
                    int r = (int)(ir % R);
                    for (int s1 = 0; s1 < 2; ++s1)
                        for (int s2 = 0; s2 < 2; ++s2) {
                            if (!X1[s1] || !X2[s2]) continue;
                            for (int cat = 0; cat < 2; ++cat) {
                                int b = block_of(cat, s1 != s2);
                                if (!live[b]) continue;
                                channel_contract_r(lmax, C, R, r, U_A[b], X1[s1] + (size_t)i * C * L2, h1);
                                channel_contract_r(lmax, C, R, r, U_B[b], X2[s2] + (size_t)i * C * L2, h2);
                                sparse_couple(cat ? &Q : &G, h1, h2, T[b] + (size_t)ir * L2);
                            }
                        }
                }
            }
            free(h1);
        }
    }
    if (!err) project_blocks(lmax, C, R, n_nodes, U_out, T, live, out_even, out_odd);
    for (int b = 0; b < CGO_NB; ++b) free(T[b]);
    free_tab(&G); free_tab(&Q);
    return err;
}

/* Message passing for the receivers listed in recv[0..n_recv) (CSR by receiver):
 *   row_ptr: [N+1], col: [E] (sender of edge e), edge_unit: [E][3],
 *   edge_radial: [E][C][L] (R_{n l1}(r_ji)), node_feat: [N][C][L^2],
 *   node_flip: NULL, or the parity-flipped node slot [N][C][L^2],
 *   U_E[b], U_I[b]: [L][C][R] edge / node input factors of block b (the four may alias);
 *   U_out[b]: [L][C][R] output weights of block b;
 *   out_even, out_odd: [n_recv][C][L^2] (row q is receiver recv[q]).
 * The edge feature R Y has natural parity, so the natural node slot pairs with it as an
 * equal pair and the flipped slot as a mixed one: by Table 1 (Cases A-D) out_even collects
 * the Gaunt coupling with the natural slot and the curl coupling with the flipped slot,
 * out_odd the curl coupling with the natural slot and the Gaunt coupling with the flipped.
 * Every (receiver, rank) pair is independent; they are spread over the threads. */
int cgo_message_pass(int lmax, int C, int R, long n_nodes, long n_edges, const int32_t *row_ptr,
                     const int32_t *col, const double *edge_unit, const double *edge_radial,
                     const double *node_feat, const double *node_flip,
                     const double *const *U_E, const double *const *U_I,
                     const double *const *U_out, const int64_t *recv, long n_recv,
                     double *out_even, double *out_odd, int nthreads)
{
    if (lmax < 0 || C < 1 || R < 1 || n_nodes < 0 || n_edges < 0 || n_recv < 0) return -1;
    for (long q = 0; q < n_recv; ++q)
        if (recv[q] < 0 || recv[q] >= n_nodes) return -1;
    set_threads(nthreads);
    int L = lmax + 1, L2 = L * L;
    const double *X2[2] = {node_feat, node_flip};
    int live[CGO_NB] = {0, 0, 0, 0};
    for (int s2 = 0; s2 < 2; ++s2)
        if (X2[s2])
            for (int cat = 0; cat < 2; ++cat) {
                int b = block_of(cat, s2);
                if ((b & 1) ? out_odd != NULL : out_even != NULL) live[b] = 1;
            }
    sparse_tab G, Q;
    if (build_tab(0, lmax, &G) || build_tab(1, lmax, &Q)) return -2;
    double *T[CGO_NB];
    int err = 0;
    for (int b = 0; b < CGO_NB; ++b) {
        T[b] = (double *)calloc(live[b] ? (size_t)n_recv * R * L2 + 1 : 1, sizeof(double));
        if (!T[b]) err = -2;
    }
    if (!err) {
#pragma omp parallel
        {
            double *E = (double *)malloc(sizeof(double) * 3 * L2), *H = E ? E + L2 : NULL;
            double *Y = H ? H + L2 : NULL;
            if (!E) {
#pragma omp atomic write
                err = -2;
            } else {
#pragma omp for schedule(dynamic, 1)
                for (long qr = 0; qr < n_recv * R; ++qr) {
                    long i = (long)recv[qr / R];
                    int r = (int)(qr % R);
                    for (long e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                        long j = col[e];
                        const double *u = edge_unit + 3 * (size_t)e;
                        cgo_real_sh(lmax, u[0], u[1], u[2], Y);
                        const double *rad = edge_radial + (size_t)e * C * L;
                        for (int s2 = 0; s2 < 2; ++s2) {
                            if (!X2[s2]) continue;
                            for (int cat = 0; cat < 2; ++cat) {
                                int b = block_of(cat, s2);
                                if (!live[b]) continue;
                                /* Eq. msgpass-tildeR, then multiply by Y_{l1 m1}(rhat) */
                                for (int l1 = 0; l1 < L; ++l1) {
                                    double s = 0.0;
                                    for (int n = 0; n < C; ++n)
                                        s += U_E[b][((size_t)l1 * C + n) * R + r] * rad[(size_t)n * L + l1];
                                    for (int m1 = -l1; m1 <= l1; ++m1)
                                        E[l1 * l1 + l1 + m1] = s * Y[l1 * l1 + l1 + m1];
                                }
                                /* Eq. msgpass-HI */
                                channel_contract_r(lmax, C, R, r, U_I[b], X2[s2] + (size_t)j * C * L2, H);
                                sparse_couple(cat ? &Q : &G, E, H, T[b] + (size_t)qr * L2);
                            }
                        }
                    }
                }
            }
            free(E);
        }
    }
    if (!err) project_blocks(lmax, C, R, n_recv, U_out, T, live, out_even, out_odd);
    for (int b = 0; b < CGO_NB; ++b) free(T[b]);
    free_tab(&G); free_tab(&Q);
    return err;
}

/* Message passing with two parity-bearing fields (Eq. twoparity-phi): the edge operand is a
 * general per-edge feature with its own parity slots instead of R Y, so its channel
 * contraction runs per edge like the node side (Eq. msgpass-HI applied to the edge field).
 *   edge_feat: [E][C][L^2] natural-parity slot of the edge field I^(E);
 *   edge_flip: NULL, or its parity-flipped slot [E][C][L^2];
 *   node_feat, node_flip: the node field I^(N) as in cgo_message_pass;
 *   U_E[b], U_I[b], U_out[b]: per-block factors as in cgo_onsite;
 *   out_even, out_odd: [n_recv][C][L^2] (row q is receiver recv[q]).
 * For every edge e = (j -> i) every slot pair (s1 of the edge field, s2 of the node field of
 * sender j) contributes its Gaunt and curl couplings, routed to blocks by p = p1 p2 exactly as
 * the on-site pairs; the sum over the edges of a receiver replaces the on-site product.
 * Every (receiver, rank) pair is independent; they are spread over the threads. */
int cgo_message_pass_fields(int lmax, int C, int R, long n_nodes, long n_edges,
                            const int32_t *row_ptr, const int32_t *col, const double *edge_feat,
                            const double *edge_flip, const double *node_feat,
                            const double *node_flip, const double *const *U_E,
                            const double *const *U_I, const double *const *U_out,
                            const int64_t *recv, long n_recv, double *out_even, double *out_odd,
                            int nthreads)
{
    if (lmax < 0 || C < 1 || R < 1 || n_nodes < 0 || n_edges < 0 || n_recv < 0) return -1;
    for (long q = 0; q < n_recv; ++q)
        if (recv[q] < 0 || recv[q] >= n_nodes) return -1;
    set_threads(nthreads);
    int L2 = (lmax + 1) * (lmax + 1);
    const double *X1[2] = {edge_feat, edge_flip}, *X2[2] = {node_feat, node_flip};
    int live[CGO_NB] = {0, 0, 0, 0};
    for (int s1 = 0; s1 < 2; ++s1)
        for (int s2 = 0; s2 < 2; ++s2)
            if (X1[s1] && X2[s2])
                for (int cat = 0; cat < 2; ++cat) {
                    int b = block_of(cat, s1 != s2);
                    if ((b & 1) ? out_odd != NULL : out_even != NULL) live[b] = 1;
                }
    sparse_tab G, Q;
    if (build_tab(0, lmax, &G) || build_tab(1, lmax, &Q)) return -2;
    double *T[CGO_NB];
    int err = 0;
    for (int b = 0; b < CGO_NB; ++b) {
        T[b] = (double *)calloc(live[b] ? (size_t)n_recv * R * L2 + 1 : 1, sizeof(double));
        if (!T[b]) err = -2;
    }
    if (!err) {
#pragma omp parallel
        {
            double *h1 = (double *)malloc(sizeof(double) * 2 * L2), *h2 = h1 ? h1 + L2 : NULL;
            if (!h1) {
#pragma omp atomic write
                err = -2;
            } else {
#pragma omp for schedule(dynamic, 1)
                for (long qr = 0; qr < n_recv * R; ++qr) {
                    long i = (long)recv[qr / R];
                    int r = (int)(qr % R);
                    for (long e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                        long j = col[e];
                        for (int s1 = 0; s1 < 2; ++s1)
                            for (int s2 = 0; s2 < 2; ++s2) {
                                if (!X1[s1] || !X2[s2]) continue;
                                for (int cat = 0; cat < 2; ++cat) {
                                    int b = block_of(cat, s1 != s2);
                                    if (!live[b]) continue;
                                    channel_contract_r(lmax, C, R, r, U_E[b], X1[s1] + (size_t)e * C * L2, h1);
                                    channel_contract_r(lmax, C, R, r, U_I[b], X2[s2] + (size_t)j * C * L2, h2);
                                    sparse_couple(cat ? &Q : &G, h1, h2, T[b] + (size_t)qr * L2);
                                }
                            }
                    }
                }
            }
            free(h1);
        }
    }
    if (!err) project_blocks(lmax, C, R, n_recv, U_out, T, live, out_even, out_odd);
    for (int b = 0; b < CGO_NB; ++b) free(T[b]);
    free_tab(&G); free_tab(&Q);
    return err;
}

/* nu-body on-site product: the grid pointwise product extended to nu operands (the
 * ACE-style extension in the discussion of other algorithms; Eq. phi-cg is nu = 2):
 *   H_t[r][k] = sum_n U_t[l][n][r] X_t[n][k],                    t = 1 .. nu
 *   T[r][k]   = int Y_k prod_t (sum_{k'} H_t[r][k'] Y_{k'}) dOmega,
 *   out[n][k] = sum_r U_out[l][n][r] T[r][k].
 * The integral is written out as the exact chain of real Gaunt couplings: P_1 = H_1 and
 * P_t[k] = sum GR[k1][k2][k] P_{t-1}[k1] H_t[k2], where P_t keeps every degree up to t lmax
 * (a product of fields of degrees a and b has degree a + b) and the last step only the
 * output degrees up to lmax. Only Gaunt couplings enter: with natural-parity inputs the
 * product has natural parity. Arrays: X[t] [N][C][L^2], U[t] [L][C][R], U_out [L][C][R],
 * out [N][C][L^2]; operands may alias. */
int cgo_nbody(int lmax, int C, int R, int nu, long n_nodes, const double *const *X,
              const double *const *U, const double *U_out, double *out, int nthreads)
{
    if (lmax < 0 || C < 1 || R < 1 || nu < 1 || n_nodes < 0) return -1;
    if ((long)nu * lmax > ORC_MAXJ) return -1;
    set_threads(nthreads);
    const int L2 = (lmax + 1) * (lmax + 1);
    /* intermediate products: degrees up to (nu - 1) lmax, and at least the input's */
    const int Lp = (nu > 1 ? nu - 1 : 1) * lmax + 1, P2 = Lp * Lp;
    sparse_tab *G = (sparse_tab *)calloc((size_t)nu + 1, sizeof(sparse_tab));
    if (!G) return -2;
    for (int t = 2; t <= nu; ++t)
        if (build_tab3(0, (t - 1) * lmax, lmax, t == nu ? lmax : t * lmax, &G[t])) return -2;
    double *T = (double *)calloc((size_t)n_nodes * R * L2 + 1, sizeof(double));
    if (!T) return -2;
    int err = 0;
#pragma omp parallel
    {
        double *buf = (double *)malloc(sizeof(double) * ((size_t)L2 + 2 * (size_t)P2));
        if (!buf) {
#pragma omp atomic write
            err = -2;
        } else {
            double *h = buf, *p = buf + L2, *q = p + P2;
#pragma omp for schedule(dynamic, 4)
            for (long ir = 0; ir < n_nodes * R; ++ir) {
                long i = ir / R;
                int r = (int)(ir % R);
                channel_contract_r(lmax, C, R, r, U[0], X[0] + (size_t)i * C * L2, h);
                memset(p, 0, sizeof(double) * P2);
                memcpy(p, h, sizeof(double) * L2);
                for (int t = 2; t <= nu; ++t) {
                    channel_contract_r(lmax, C, R, r, U[t - 1], X[t - 1] + (size_t)i * C * L2, h);
                    memset(q, 0, sizeof(double) * P2);
                    sparse_couple(&G[t], p, h, q);
                    double *sw = p; p = q; q = sw;
                }
                memcpy(T + (size_t)ir * L2, p, sizeof(double) * L2);
            }
        }
        free(buf);
    }
    if (!err) {
#pragma omp parallel for schedule(static)
        for (long i = 0; i < n_nodes; ++i)
            project_out(lmax, C, R, U_out, T + (size_t)i * R * L2, out + (size_t)i * C * L2);
    }
    free(T);
    for (int t = 2; t <= nu; ++t) free_tab(&G[t]);
    free(G);
    return err;
}

int cgo_max_threads(void)
{
    return set_threads(0);
}
