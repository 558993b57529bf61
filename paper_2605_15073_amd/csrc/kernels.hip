// HIP kernels for gfx950 (wave64): channel contractions, grid synthesis, the
// on-site grid product / surface curl, the message-passing receiver pass and
// the quadrature analysis. Templated on the scalar type (fp32, fp64).
//
// Layouts (row-major): coefficients [b][c][K]; grid fields [b][r][f][UV] with
// UV = u * V + v; azimuthal index mi = m + lmax.
#include "internal.h"

namespace cgtp {

static constexpr int kThreads = 256;

__device__ __forceinline__ int degree_of(int k)
{
    int l = (int)sqrtf((float)k);
    while (l * l > k) --l;
    while ((l + 1) * (l + 1) <= k) ++l;
    return l;
}

// ---------------------------------------------------------------------------
// Per-degree channel contraction (Eqs. struct-H, msgpass-HI, msgpass-tildeR,
// struct-phi): Y[b][o][k] = scale[l] * sum_i W[l*w_sl + i*w_si + o*w_so] X[b][i][k].
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void k_contract(int64_t B, int Cin, int Cout, int K,
                                                       int kdeg, const T *__restrict__ W,
                                                       int64_t w_sl, int64_t w_si, int64_t w_so,
                                                       const T *__restrict__ X, T *__restrict__ Y,
                                                       const T *__restrict__ scale)
{
    const int64_t total = B * (int64_t)Cout * K;
    for (int64_t idx = blockIdx.x * (int64_t)kThreads + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * kThreads) {
        int k = (int)(idx % K);
        int64_t rest = idx / K;
        int o = (int)(rest % Cout);
        int64_t b = rest / Cout;
        int l = kdeg ? k : degree_of(k);
        const T *w = W + l * w_sl + o * w_so;
        const T *x = X + b * (int64_t)Cin * K + k;
        T acc = 0;
        for (int i = 0; i < Cin; ++i) acc += w[i * w_si] * x[(int64_t)i * K];
        if (scale) acc *= scale[l];
        Y[idx] = acc;
    }
}

template <typename T>
hipError_t launch_contract(int64_t B, int Cin, int Cout, int K, bool kdeg, const T *W,
                           int64_t w_sl, int64_t w_si, int64_t w_so, const T *X, T *Y,
                           const T *scale, hipStream_t s)
{
    int64_t total = B * (int64_t)Cout * K;
    if (total == 0) return hipSuccess;
    int64_t blocks = (total + kThreads - 1) / kThreads;
    if (blocks > (1 << 20)) blocks = 1 << 20;
    hipLaunchKernelGGL(k_contract<T>, dim3((unsigned)blocks), dim3(kThreads), 0, s, B, Cin, Cout,
                       K, kdeg ? 1 : 0, W, w_sl, w_si, w_so, X, Y, scale);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Shared device pieces of the structured transforms.
// ---------------------------------------------------------------------------

// Legendre synthesis (Eq. struct-F) and its x-derivative pass:
//   F[mi][u] = sum_{l>=|m|} Pt_l^|m|(x_u) H[l,m],  Fx likewise with dPt/dx.
template <typename T>
__device__ void legendre_synth(const Tabs<T> &tb, const T *H, T *F, T *Fx)
{
    const Dims &d = tb.d;
    for (int idx = threadIdx.x; idx < d.M * d.U; idx += blockDim.x) {
        int mi = idx / d.U, u = idx - mi * d.U;
        int m = mi - d.lmax, am = m < 0 ? -m : m;
        const T *pu = tb.p + (size_t)u * d.P;
        const T *dpu = tb.dp + (size_t)u * d.P;
        T f = 0, fx = 0;
        for (int l = am; l <= d.lmax; ++l) {
            T h = H[l * l + l + m];
            int pi = l * (l + 1) / 2 + am;
            f += pu[pi] * h;
            fx += dpu[pi] * h;
        }
        F[idx] = f;
        Fx[idx] = fx;
    }
}

// Fourier synthesis at one grid point (Eq. struct-tildeA) of the field, its
// x-derivative, and its phi-derivative. In the real basis d/dphi maps the cosine
// slot +k to -k * (sine slot) and the sine slot -k to +k * (cosine slot).
template <typename T>
__device__ __forceinline__ void fourier_point(const Tabs<T> &tb, const T *F, const T *Fx, int u,
                                              int v, T &a, T &ax, T &ap)
{
    const Dims &d = tb.d;
    const T *qv = tb.q + (size_t)v * d.M;
    const int lm = d.lmax, U = d.U;
    a = qv[lm] * F[lm * U + u];
    ax = qv[lm] * Fx[lm * U + u];
    ap = 0;
    for (int k = 1; k <= lm; ++k) {
        T qc = qv[lm + k], qs = qv[lm - k];
        T fc = F[(lm + k) * U + u], fs = F[(lm - k) * U + u];
        a += qc * fc + qs * fs;
        ax += qc * Fx[(lm + k) * U + u] + qs * Fx[(lm - k) * U + u];
        ap += (T)k * (fs * qc - fc * qs);
    }
}

// Quadrature analysis (Eqs. struct-Tmu, struct-Tlm) of two grid fields S1, S2
// [UV] held on chip, through Tm scratch [2][M][U]; writes out1/out2 [K].
template <typename T>
__device__ void analysis2(const Tabs<T> &tb, const T *S1, const T *S2, T *Tm, T *out1, T *out2)
{
    const Dims &d = tb.d;
    const int MU = d.M * d.U;
    for (int idx = threadIdx.x; idx < 2 * MU; idx += blockDim.x) {
        int which = idx >= MU;
        int rem = idx - which * MU;
        int mi = rem / d.U, u = rem - mi * d.U;
        const T *S = (which ? S2 : S1) + u * d.V;
        T s = 0;
        for (int v = 0; v < d.V; ++v) s += tb.q[(size_t)v * d.M + mi] * S[v];
        Tm[idx] = s;
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < 2 * d.K; idx += blockDim.x) {
        int which = idx >= d.K;
        int k = idx - which * d.K;
        int l = degree_of(k), m = k - l * l - l, am = m < 0 ? -m : m;
        const T *tm = Tm + which * MU + (m + d.lmax) * d.U;
        int pi = l * (l + 1) / 2 + am;
        T s = 0;
        for (int u = 0; u < d.U; ++u) s += tb.wq[u] * tb.p[(size_t)u * d.P + pi] * tm[u];
        (which ? out2 : out1)[k] = s;
    }
}

// ---------------------------------------------------------------------------
// Sender (node-side) grid fields: SF[b][r][0..2][UV] = (A, dA/dx, dA/dphi).
// One block per (node, rank).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void k_sender_fields(Tabs<T> tb, int R,
                                                            const T *__restrict__ H,
                                                            T *__restrict__ SF)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    const int64_t br = blockIdx.x;  // b * R + r
    T *Hs = smem;
    T *F = Hs + d.K;
    T *Fx = F + d.M * d.U;
    for (int k = threadIdx.x; k < d.K; k += blockDim.x) Hs[k] = H[br * d.K + k];
    __syncthreads();
    legendre_synth(tb, Hs, F, Fx);
    __syncthreads();
    T *out = SF + br * 3 * (int64_t)d.UV;
    for (int uv = threadIdx.x; uv < d.UV; uv += blockDim.x) {
        int u = uv / d.V, v = uv - u * d.V;
        T a, ax, ap;
        fourier_point(tb, F, Fx, u, v, a, ax, ap);
        out[uv] = a;
        out[d.UV + uv] = ax;
        out[2 * d.UV + uv] = ap;
    }
}

template <typename T>
hipError_t launch_sender_fields(const Tabs<T> &tb, int64_t B, int R, const T *H, T *SF,
                                hipStream_t s)
{
    int64_t blocks = B * R;
    if (blocks == 0) return hipSuccess;
    size_t sh = sizeof(T) * (tb.d.K + 2 * tb.d.M * tb.d.U);
    hipLaunchKernelGGL(k_sender_fields<T>, dim3((unsigned)blocks), dim3(kThreads), sh, s, tb, R,
                       H, SF);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// On-site: per (node, rank) synthesise both operands, form
//   S_alpha = A1 A2 (Eq. struct-S)  and
//   S_beta  = dA1/dphi dA2/dx - dA1/dx dA2/dphi (Eq. poisson-S2-x),
// then analyse both back to (l, m).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void k_onsite_grid(Tabs<T> tb, int R,
                                                          const T *__restrict__ HA,
                                                          const T *__restrict__ HB,
                                                          T *__restrict__ Ta, T *__restrict__ Tb)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    const int64_t br = blockIdx.x;
    const int MU = d.M * d.U;
    T *H1 = smem;
    T *H2 = H1 + d.K;
    T *F1 = H2 + d.K;
    T *F1x = F1 + MU;
    T *F2 = F1x + MU;
    T *F2x = F2 + MU;
    T *Sa = F2x + MU;
    T *Sb = Sa + d.UV;
    for (int k = threadIdx.x; k < d.K; k += blockDim.x) {
        H1[k] = HA[br * d.K + k];
        H2[k] = HB[br * d.K + k];
    }
    __syncthreads();
    legendre_synth(tb, H1, F1, F1x);
    legendre_synth(tb, H2, F2, F2x);
    __syncthreads();
    for (int uv = threadIdx.x; uv < d.UV; uv += blockDim.x) {
        int u = uv / d.V, v = uv - u * d.V;
        T a1, a1x, a1p, a2, a2x, a2p;
        fourier_point(tb, F1, F1x, u, v, a1, a1x, a1p);
        fourier_point(tb, F2, F2x, u, v, a2, a2x, a2p);
        Sa[uv] = a1 * a2;
        Sb[uv] = a1p * a2x - a1x * a2p;
    }
    __syncthreads();
    analysis2(tb, Sa, Sb, F1 /* reused as Tm scratch [2][M][U] */, Ta + br * d.K, Tb + br * d.K);
}

template <typename T>
hipError_t launch_onsite_grid(const Tabs<T> &tb, int64_t B, int R, const T *HA, const T *HB,
                              T *Ta, T *Tb, hipStream_t s)
{
    int64_t blocks = B * R;
    if (blocks == 0) return hipSuccess;
    size_t sh = sizeof(T) * (2 * tb.d.K + 4 * tb.d.M * tb.d.U + 2 * tb.d.UV);
    hipLaunchKernelGGL(k_onsite_grid<T>, dim3((unsigned)blocks), dim3(kThreads), sh, s, tb, R, HA,
                       HB, Ta, Tb);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Message passing, receiver side. One block per (receiver, rank); each thread
// owns NPT grid points and accumulates over the CSR row in registers
// (Eqs. msgpass-S, cat-beta-curl; no atomics). Edge field by the addition
// theorem: sum_m Y_lm(rhat) Y_lm(Omega) = (2l+1)/(4 pi) P_l(rhat . Omega), so with
// Rt already scaled by (2l+1)/(4 pi):
//   A_E = sum_l Rt_l P_l(t), g = sum_l Rt_l P_l'(t), t = rhat . Omega(x, phi),
//   dA_E/dx = g dt/dx, dA_E/dphi = g dt/dphi.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void load_unit(const T *unit, int64_t e, T &ux, T &uy, T &uz)
{
    ux = unit[3 * e];
    uy = unit[3 * e + 1];
    uz = unit[3 * e + 2];
    T inv = (T)1 / sqrt(ux * ux + uy * uy + uz * uz);
    ux *= inv;
    uy *= inv;
    uz *= inv;
}

template <typename T, int NPT>
__global__ __launch_bounds__(kThreads) void k_receiver_zonal(Tabs<T> tb, int R,
                                                             const int32_t *__restrict__ row_ptr,
                                                             const int32_t *__restrict__ col,
                                                             const T *__restrict__ unit,
                                                             const T *__restrict__ Rt,
                                                             const T *__restrict__ SF,
                                                             T *__restrict__ Ta,
                                                             T *__restrict__ Tb)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    const int64_t br = blockIdx.x;
    const int64_t i = br / R;
    const int r = (int)(br - i * R);
    T sa[NPT], sb[NPT];
#pragma unroll
    for (int s = 0; s < NPT; ++s) sa[s] = sb[s] = 0;
    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    for (int e = e0; e < e1; ++e) {
        const int64_t j = col[e];
        T ux, uy, uz;
        load_unit(unit, e, ux, uy, uz);
        const T *rt = Rt + ((int64_t)e * R + r) * d.L;
        const T *sf = SF + (j * R + r) * 3 * (int64_t)d.UV;
#pragma unroll
        for (int s = 0; s < NPT; ++s) {
            int uv = threadIdx.x + s * kThreads;
            if (uv < d.UV) {
                int u = uv / d.V, v = uv - u * d.V;
                T x = tb.x[u], sx = tb.sx[u], cp = tb.cphi[v], sp = tb.sphi[v];
                T h = ux * cp + uy * sp;
                T t = uz * x + sx * h;
                T p0 = 1, p1 = t, d1 = 1;
                T a = rt[0], g = 0;
                if (d.lmax >= 1) {
                    a += rt[1] * t;
                    g = rt[1];
                }
                for (int l = 2; l <= d.lmax; ++l) {
                    T p2 = tb.rc1[l] * t * p1 - tb.rc2[l] * p0;
                    T d2 = (T)l * p1 + t * d1;
                    a += rt[l] * p2;
                    g += rt[l] * d2;
                    p0 = p1;
                    p1 = p2;
                    d1 = d2;
                }
                T dxt = uz - tb.xsx[u] * h;
                T dpt = sx * (uy * cp - ux * sp);
                T fI = sf[uv], fX = sf[d.UV + uv], fP = sf[2 * d.UV + uv];
                sa[s] += a * fI;
                sb[s] += g * (dpt * fX - dxt * fP);
            }
        }
    }
    T *Sa = smem;
    T *Sb = Sa + d.UV;
    T *Tm = Sb + d.UV;
#pragma unroll
    for (int s = 0; s < NPT; ++s) {
        int uv = threadIdx.x + s * kThreads;
        if (uv < d.UV) {
            Sa[uv] = sa[s];
            Sb[uv] = sb[s];
        }
    }
    __syncthreads();
    analysis2(tb, Sa, Sb, Tm, Ta + br * d.K, Tb + br * d.K);
}

// Separated edge synthesis (Eqs. msgpass-FE, msgpass-AE and the derivative
// passes): per edge, the real SH of the bond direction, E[k] = Rt_l Y_k(rhat),
// the Legendre pass and the Fourier pass at every grid point.
template <typename T>
__device__ void edge_sh(const Tabs<T> &tb, T ux, T uy, T uz, T *Y)
{
    const Dims &d = tb.d;
    // one thread per order m >= 0 walks its column in l
    for (int m = threadIdx.x; m <= d.lmax; m += blockDim.x) {
        T s = sqrt(ux * ux + uy * uy);
        T cph = s > 0 ? ux / s : (T)1, sph = s > 0 ? uy / s : (T)0;
        T cm = 1, sm = 0;  // cos(m phi), sin(m phi)
        for (int k = 0; k < m; ++k) {
            T c2 = cm * cph - sm * sph;
            sm = sm * cph + cm * sph;
            cm = c2;
        }
        T pmm = tb.ymm[0];
        for (int k = 1; k <= m; ++k) pmm *= tb.ymm[k] * s;
        const T r2 = (T)1.4142135623730950488;
        T pl2 = 0, pl1 = pmm;
        for (int l = m; l <= d.lmax; ++l) {
            T v;
            int idx = l * (l + 1) / 2 + m;
            if (l == m) v = pmm;
            else if (l == m + 1) v = tb.ya[idx] * uz * pmm;
            else v = tb.ya[idx] * (uz * pl1 - tb.yb[idx] * pl2);
            if (l > m) {
                pl2 = pl1;
                pl1 = v;
            }
            if (m == 0) {
                Y[l * l + l] = v;
            } else {
                Y[l * l + l + m] = r2 * v * cm;
                Y[l * l + l - m] = r2 * v * sm;
            }
        }
    }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void k_receiver_separated(
    Tabs<T> tb, int R, const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
    const T *__restrict__ unit, const T *__restrict__ Rt, const T *__restrict__ SF,
    T *__restrict__ Ta, T *__restrict__ Tb)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    const int64_t br = blockIdx.x;
    const int64_t i = br / R;
    const int r = (int)(br - i * R);
    const int MU = d.M * d.U;
    T *Sa = smem;
    T *Sb = Sa + d.UV;
    T *Y = Sb + d.UV;
    T *F = Y + d.K;
    T *Fx = F + MU;
    for (int uv = threadIdx.x; uv < d.UV; uv += blockDim.x) Sa[uv] = Sb[uv] = 0;
    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    for (int e = e0; e < e1; ++e) {
        const int64_t j = col[e];
        T ux, uy, uz;
        load_unit(unit, e, ux, uy, uz);
        __syncthreads();  // previous edge done with Y / F
        edge_sh(tb, ux, uy, uz, Y);
        __syncthreads();
        const T *rt = Rt + ((int64_t)e * R + r) * d.L;
        for (int k = threadIdx.x; k < d.K; k += blockDim.x) Y[k] *= rt[degree_of(k)];
        __syncthreads();
        legendre_synth(tb, Y, F, Fx);
        __syncthreads();
        const T *sf = SF + (j * R + r) * 3 * (int64_t)d.UV;
        for (int uv = threadIdx.x; uv < d.UV; uv += blockDim.x) {
            int u = uv / d.V, v = uv - u * d.V;
            T a, ax, ap;
            fourier_point(tb, F, Fx, u, v, a, ax, ap);
            Sa[uv] += a * sf[uv];
            Sb[uv] += ap * sf[d.UV + uv] - ax * sf[2 * d.UV + uv];
        }
    }
    __syncthreads();
    analysis2(tb, Sa, Sb, F /* Tm scratch, 2 MU */, Ta + br * d.K, Tb + br * d.K);
}

template <typename T>
hipError_t launch_receiver(const Tabs<T> &tb, bool separated, int64_t N, int R,
                           const int32_t *row_ptr, const int32_t *col, const T *unit,
                           const T *Rt, const T *SF, T *Ta, T *Tb, hipStream_t s)
{
    int64_t blocks = N * R;
    if (blocks == 0) return hipSuccess;
    const Dims &d = tb.d;
    if (separated) {
        size_t sh = sizeof(T) * (2 * d.UV + d.K + 2 * d.M * d.U);
        hipLaunchKernelGGL(k_receiver_separated<T>, dim3((unsigned)blocks), dim3(kThreads), sh, s,
                           tb, R, row_ptr, col, unit, Rt, SF, Ta, Tb);
        return hipGetLastError();
    }
    size_t sh = sizeof(T) * (2 * d.UV + 2 * d.M * d.U);
    int npt = (d.UV + kThreads - 1) / kThreads;
#define CGTP_RECV(NP)                                                                         \
    hipLaunchKernelGGL((k_receiver_zonal<T, NP>), dim3((unsigned)blocks), dim3(kThreads), sh, s, \
                       tb, R, row_ptr, col, unit, Rt, SF, Ta, Tb)
    if (npt <= 1) CGTP_RECV(1);
    else if (npt <= 2) CGTP_RECV(2);
    else if (npt <= 4) CGTP_RECV(4);
    else if (npt <= 8) CGTP_RECV(8);
    else CGTP_RECV(11);
#undef CGTP_RECV
    return hipGetLastError();
}

#define CGTP_INSTANTIATE(T)                                                                      \
    template hipError_t launch_contract<T>(int64_t, int, int, int, bool, const T *, int64_t,     \
                                           int64_t, int64_t, const T *, T *, const T *,          \
                                           hipStream_t);                                         \
    template hipError_t launch_sender_fields<T>(const Tabs<T> &, int64_t, int, const T *, T *,   \
                                                hipStream_t);                                    \
    template hipError_t launch_onsite_grid<T>(const Tabs<T> &, int64_t, int, const T *,          \
                                              const T *, T *, T *, hipStream_t);                 \
    template hipError_t launch_receiver<T>(const Tabs<T> &, bool, int64_t, int, const int32_t *, \
                                           const int32_t *, const T *, const T *, const T *,     \
                                           T *, T *, hipStream_t);

CGTP_INSTANTIATE(float)
CGTP_INSTANTIATE(double)

}  // namespace cgtp
