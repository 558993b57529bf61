// Host-side grid tables in fp64: Gauss-Legendre nodes and weights, normalised
// associated Legendre functions and their x-derivatives at the nodes, real
// Fourier factors, and the small recurrence tables the kernels use.
//
// Grid (Sec. "Representation using Structured Tensor-Product Grids"): U
// Gauss-Legendre nodes x_u = cos(theta_u) with weights w_u and V equispaced
// azimuths phi_v = 2 pi v / V; exact for the degree-3 lmax integrands when
// U >= (3 lmax + 1)/2 and V >= 3 lmax + 1. Basis: App. C, Eqs. realY and realq.
#include <cmath>
#include <cstring>
#include <vector>

#include "internal.h"

namespace cgtp {

static const double kPi = 3.14159265358979323846;

bool resolve_grid(int lmax, int n_theta, int n_phi, int *U, int *V)
{
    if (lmax < 0 || lmax > CGTP_MAX_LMAX) return false;
    int u_min = (3 * lmax + 2) / 2;           // ceil((3 lmax + 1) / 2)
    int u_def = (3 * lmax + 3) / 2;           // ceil((3 lmax + 2) / 2)
    int v_min = 3 * lmax + 1;
    if (u_min < 1) u_min = 1;
    if (u_def < 1) u_def = 1;
    int u = n_theta == 0 ? u_def : n_theta;
    int v = n_phi == 0 ? v_min : n_phi;
    if (u < u_min || v < v_min || u > 4 * CGTP_MAX_LMAX + 8 || v > 8 * CGTP_MAX_LMAX + 8)
        return false;
    *U = u;
    *V = v;
    return true;
}

Dims make_dims(int lmax, int U, int V)
{
    Dims d;
    d.lmax = lmax;
    d.L = lmax + 1;
    d.K = (lmax + 1) * (lmax + 1);
    d.M = 2 * lmax + 1;
    d.P = (lmax + 1) * (lmax + 2) / 2;
    d.U = U;
    d.V = V;
    d.UV = U * V;
    d.UVs = (d.UV + 31) / 32 * 32;
    d.lds_max = 65536;
    d.lds_cu = 65536;
    return d;
}

// Newton iteration on P_n from the asymptotic guess cos(pi (i - 1/4) / (n + 1/2)).
void gauss_legendre(int n, double *x, double *w)
{
    for (int i = 0; i < n; ++i) {
        double z = std::cos(kPi * (i + 0.75) / (n + 0.5));
        double dp = 1.0;
        for (int it = 0; it < 100; ++it) {
            double p0 = 1.0, p1 = z;
            for (int k = 2; k <= n; ++k) {
                double p2 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p0) / k;
                p0 = p1;
                p1 = p2;
            }
            double pn = n == 0 ? 1.0 : (n == 1 ? z : p1);
            double pn1 = n == 1 ? 1.0 : p0;
            dp = n * (z * pn - pn1) / (z * z - 1.0);
            double dz = pn / dp;
            z -= dz;
            if (std::fabs(dz) < 1e-16) break;
        }
        // recompute the derivative at the converged node for the weight
        double p0 = 1.0, p1 = z;
        for (int k = 2; k <= n; ++k) {
            double p2 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p0) / k;
            p0 = p1;
            p1 = p2;
        }
        double pn = n == 1 ? z : p1;
        double pn1 = n == 1 ? 1.0 : p0;
        dp = n * (z * pn - pn1) / (z * z - 1.0);
        x[i] = z;
        w[i] = 2.0 / ((1.0 - z * z) * dp * dp);
    }
}

// Normalised Pt_l^m (no Condon-Shortley phase) by the standard stable recurrences
//   Pt_0^0 = 1/sqrt(4 pi),  Pt_m^m = sqrt((2m+1)/(2m)) s Pt_{m-1}^{m-1},
//   Pt_{m+1}^m = sqrt(2m+3) x Pt_m^m,
//   Pt_l^m = a_lm (x Pt_{l-1}^m - b_lm Pt_{l-2}^m),
//   a_lm = sqrt((4l^2-1)/(l^2-m^2)),  b_lm = sqrt(((l-1)^2-m^2)/(4(l-1)^2-1)),
// and (1-x^2) dPt_l^m/dx = sqrt((2l+1)(l^2-m^2)/(2l-1)) Pt_{l-1}^m - l x Pt_l^m.
void legendre_tables(int lmax, int U, const double *x, double *p, double *dp)
{
    const int P = (lmax + 1) * (lmax + 2) / 2;
    for (int u = 0; u < U; ++u) {
        double z = x[u], s = std::sqrt(std::fmax(0.0, 1.0 - z * z));
        double *pu = p + (size_t)u * P, *dpu = dp + (size_t)u * P;
        double pmm = 1.0 / std::sqrt(4.0 * kPi);
        for (int m = 0; m <= lmax; ++m) {
            if (m > 0) pmm *= std::sqrt((2.0 * m + 1.0) / (2.0 * m)) * s;
            double pl2 = 0.0, pl1 = pmm;
            for (int l = m; l <= lmax; ++l) {
                double v;
                if (l == m) {
                    v = pmm;
                } else if (l == m + 1) {
                    v = std::sqrt(2.0 * m + 3.0) * z * pmm;
                } else {
                    double a = std::sqrt((4.0 * l * l - 1.0) / ((double)l * l - (double)m * m));
                    double b = std::sqrt(((l - 1.0) * (l - 1.0) - (double)m * m)
                                         / (4.0 * (l - 1.0) * (l - 1.0) - 1.0));
                    v = a * (z * pl1 - b * pl2);
                }
                if (l > m) {
                    pl2 = pl1;
                    pl1 = v;
                }
                int idx = l * (l + 1) / 2 + m;
                pu[idx] = v;
                double prev = (l > m) ? pl2 : 0.0;  // Pt_{l-1}^m
                double c = (l > m) ? std::sqrt((2.0 * l + 1.0) * ((double)l * l - (double)m * m)
                                               / (2.0 * l - 1.0))
                                   : 0.0;
                dpu[idx] = (c * prev - l * z * v) / (1.0 - z * z);
            }
        }
    }
}

void fourier_table(int lmax, int V, double *q)
{
    const int M = 2 * lmax + 1;
    for (int v = 0; v < V; ++v) {
        double ph = 2.0 * kPi * v / V;
        for (int m = -lmax; m <= lmax; ++m) {
            double val;
            if (m > 0) val = std::sqrt(2.0) * std::cos(m * ph);
            else if (m == 0) val = 1.0;
            else val = std::sqrt(2.0) * std::sin(-m * ph);
            q[(size_t)v * M + m + lmax] = val;
        }
    }
}

// Region sizes, in the member order of Tabs<T>.
static void region_sizes(const Dims &d, size_t *n)
{
    n[0] = d.U;                 // x
    n[1] = d.U;                 // sx
    n[2] = d.U;                 // xsx
    n[3] = d.U;                 // wq
    n[4] = (size_t)d.U * d.P;   // p
    n[5] = (size_t)d.U * d.P;   // dp
    n[6] = (size_t)d.V * d.M;   // q
    n[7] = d.V;                 // cphi
    n[8] = d.V;                 // sphi
    n[9] = d.L;                 // cl
    n[10] = d.L;                // rc1
    n[11] = d.L;                // rc2
    n[12] = d.P;                // ya
    n[13] = d.P;                // yb
    n[14] = d.L;                // ymm
    const size_t ut = (size_t)(d.U + 3) / 4 * 4;
    n[15] = (size_t)d.P * ut;   // pt
    n[16] = (size_t)d.P * ut;   // dpt
    n[17] = (size_t)d.P * ut;   // wpt
    n[18] = d.P;                // yc
    n[19] = d.lmax <= kDenseSynthMaxL ? (size_t)(d.K + 3) / 4 * 4 * 3 * d.UVs : 0;  // ysyn
    n[20] = (size_t)d.V * d.M;  // qd
    n[21] = (size_t)d.P * ut;   // wdpt
}

static const int kRegions = 22;

static size_t round_up(size_t n) { return (n + 63) & ~(size_t)63; }  // 512 B for fp64

size_t table_elems(const Dims &d)
{
    size_t n[kRegions], t = 0;
    region_sizes(d, n);
    for (int i = 0; i < kRegions; ++i) t += round_up(n[i]);
    return t;
}

void fill_tables(const Dims &d, double *h)
{
    size_t n[kRegions], off[kRegions], t = 0;
    region_sizes(d, n);
    for (int i = 0; i < kRegions; ++i) {
        off[i] = t;
        t += round_up(n[i]);
    }
    std::memset(h, 0, sizeof(double) * t);
    std::vector<double> w(d.U);
    gauss_legendre(d.U, h + off[0], w.data());
    for (int u = 0; u < d.U; ++u) {
        double x = h[off[0] + u];
        double s = std::sqrt(std::fmax(0.0, 1.0 - x * x));
        h[off[1] + u] = s;
        h[off[2] + u] = x / s;
        h[off[3] + u] = w[u] * 2.0 * kPi / d.V;
    }
    legendre_tables(d.lmax, d.U, h + off[0], h + off[4], h + off[5]);
    fourier_table(d.lmax, d.V, h + off[6]);
    for (int v = 0; v < d.V; ++v) {
        h[off[7] + v] = std::cos(2.0 * kPi * v / d.V);
        h[off[8] + v] = std::sin(2.0 * kPi * v / d.V);
    }
    for (int l = 0; l <= d.lmax; ++l) {
        h[off[9] + l] = (2.0 * l + 1.0) / (4.0 * kPi);
        h[off[10] + l] = l > 0 ? (2.0 * l - 1.0) / l : 0.0;
        h[off[11] + l] = l > 0 ? (l - 1.0) / l : 0.0;
        h[off[14] + l] = l == 0 ? 1.0 / std::sqrt(4.0 * kPi) : std::sqrt((2.0 * l + 1.0) / (2.0 * l));
    }
    // transposed copies [P][Ut] (u fastest, rows zero padded to a multiple of 4)
    const int ut = (d.U + 3) / 4 * 4;
    for (int u = 0; u < d.U; ++u)
        for (int i = 0; i < d.P; ++i) {
            const double pv = h[off[4] + (size_t)u * d.P + i];
            h[off[15] + (size_t)i * ut + u] = pv;
            h[off[16] + (size_t)i * ut + u] = h[off[5] + (size_t)u * d.P + i];
            h[off[17] + (size_t)i * ut + u] = h[off[3] + u] * pv;
            h[off[21] + (size_t)i * ut + u] = h[off[3] + u] * h[off[5] + (size_t)u * d.P + i];
        }
    for (int l = 0; l <= d.lmax; ++l)
        for (int m = 0; m <= l; ++m) {
            int idx = l * (l + 1) / 2 + m;
            if (l > m)
                h[off[18] + idx] = std::sqrt((2.0 * l + 1.0) * ((double)l * l - (double)m * m)
                                             / (2.0 * l - 1.0));
            if (l >= m + 2) {
                h[off[12] + idx] = std::sqrt((4.0 * l * l - 1.0) / ((double)l * l - (double)m * m));
                h[off[13] + idx] = std::sqrt(((l - 1.0) * (l - 1.0) - (double)m * m)
                                             / (4.0 * (l - 1.0) * (l - 1.0) - 1.0));
            } else if (l == m + 1) {
                h[off[12] + idx] = std::sqrt(2.0 * m + 3.0);
                h[off[13] + idx] = 0.0;
            }
        }
    // phi-derivative weights of the Fourier factors (real basis: d/dphi maps cos(k phi) to
    // -k sin(k phi) and sin(k phi) to k cos(k phi))
    for (int v = 0; v < d.V; ++v)
        for (int k = 1; k <= d.lmax; ++k) {
            h[off[20] + (size_t)v * d.M + d.lmax + k] = k * h[off[6] + (size_t)v * d.M + d.lmax + k];
            h[off[20] + (size_t)v * d.M + d.lmax - k] = -k * h[off[6] + (size_t)v * d.M + d.lmax - k];
        }
    // Dense synthesis table: with k = l^2 + l + m and the real basis Y_k = Pt_l^|m|(x) q_m(phi),
    // d/dphi maps q_m to -m q_{-m} (cos(m phi) -> -m sin(m phi), sin(|m| phi) -> |m| cos(|m| phi)).
    if (n[19]) {
        const size_t ld = 3 * (size_t)d.UVs;
        for (int l = 0; l <= d.lmax; ++l)
            for (int m = -l; m <= l; ++m) {
                const int k = l * l + l + m, am = m < 0 ? -m : m;
                const int pi = l * (l + 1) / 2 + am;
                double *row = h + off[19] + (size_t)k * ld;
                for (int u = 0; u < d.U; ++u) {
                    const double pv = h[off[4] + (size_t)u * d.P + pi];
                    const double dv = h[off[5] + (size_t)u * d.P + pi];
                    for (int v = 0; v < d.V; ++v) {
                        const double qm = h[off[6] + (size_t)v * d.M + m + d.lmax];
                        const double qn = h[off[6] + (size_t)v * d.M - m + d.lmax];
                        const size_t pnt = (size_t)u * d.V + v;
                        row[pnt] = pv * qm;
                        row[d.UVs + pnt] = dv * qm;
                        row[2 * (size_t)d.UVs + pnt] = -m * pv * qn;
                    }
                }
            }
    }
}

template <typename T>
Tabs<T> bind_tables(const Dims &d, const void *dev)
{
    size_t n[kRegions];
    region_sizes(d, n);
    const T *ptr[kRegions];
    const T *b = static_cast<const T *>(dev);
    size_t t = 0;
    for (int i = 0; i < kRegions; ++i) {
        ptr[i] = b + t;
        t += round_up(n[i]);
    }
    Tabs<T> tb;
    tb.x = ptr[0];
    tb.sx = ptr[1];
    tb.xsx = ptr[2];
    tb.wq = ptr[3];
    tb.p = ptr[4];
    tb.dp = ptr[5];
    tb.q = ptr[6];
    tb.cphi = ptr[7];
    tb.sphi = ptr[8];
    tb.cl = ptr[9];
    tb.rc1 = ptr[10];
    tb.rc2 = ptr[11];
    tb.ya = ptr[12];
    tb.yb = ptr[13];
    tb.ymm = ptr[14];
    tb.pt = ptr[15];
    tb.dpt = ptr[16];
    tb.wpt = ptr[17];
    tb.yc = ptr[18];
    tb.ysyn = ptr[19];
    tb.qd = ptr[20];
    tb.wdpt = ptr[21];
    tb.d = d;
    return tb;
}

template Tabs<float> bind_tables<float>(const Dims &, const void *);
template Tabs<double> bind_tables<double>(const Dims &, const void *);

}  // namespace cgtp
