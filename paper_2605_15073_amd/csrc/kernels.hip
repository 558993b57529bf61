// HIP kernels for gfx950 (wave64): grid synthesis, the on-site grid product /
// surface curl, the message-passing receiver pass and the quadrature analysis.
// Templated on the scalar type (fp32, fp64).
//
// Layouts (row-major): coefficients [b][c][K]; stored grid fields [b][r][f][UVs]
// with point index u * V + v and rows padded to UVs (a multiple of 32 elements);
// azimuthal index mi = m + lmax.
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
// q points at the [V][M] Fourier table (staged in LDS by the callers).
template <typename T>
__device__ __forceinline__ void fourier_point(const Tabs<T> &tb, const T *q, const T *F,
                                              const T *Fx, int u, int v, T &a, T &ax, T &ap)
{
    const Dims &d = tb.d;
    const T *qv = q + v * d.M;
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

// Value-only Legendre synthesis (Eq. struct-F): F[mi][u] = sum_{l>=|m|} Pt_l^|m|(x_u) H[l,m].
template <typename T>
__device__ void legendre_value(const Tabs<T> &tb, const T *H, T *F)
{
    const Dims &d = tb.d;
    for (int idx = threadIdx.x; idx < d.M * d.U; idx += blockDim.x) {
        int mi = idx / d.U, u = idx - mi * d.U;
        int m = mi - d.lmax, am = m < 0 ? -m : m;
        const T *pu = tb.p + (size_t)u * d.P;
        T f = 0;
        for (int l = am; l <= d.lmax; ++l) f += pu[l * (l + 1) / 2 + am] * H[l * l + l + m];
        F[idx] = f;
    }
}

// Value-only Fourier synthesis at one grid point (Eq. struct-tildeA).
template <typename T>
__device__ __forceinline__ T fourier_value(const Tabs<T> &tb, const T *q, const T *F, int u, int v)
{
    const Dims &d = tb.d;
    const T *qv = q + v * d.M;
    T a = 0;
    for (int mi = 0; mi < d.M; ++mi) a += qv[mi] * F[mi * d.U + u];
    return a;
}

// Quadrature analysis (Eqs. struct-Tmu, struct-Tlm) of one grid field S [UV] held on chip,
// through Tm scratch [M][U]; writes out [K].
template <typename T>
__device__ void analysis1(const Tabs<T> &tb, const T *q, const T *S, T *Tm, T *out)
{
    const Dims &d = tb.d;
    for (int idx = threadIdx.x; idx < d.M * d.U; idx += blockDim.x) {
        int mi = idx / d.U, u = idx - mi * d.U;
        const T *row = S + u * d.V;
        T s = 0;
        for (int v = 0; v < d.V; ++v) s += q[v * d.M + mi] * row[v];
        Tm[idx] = s;
    }
    __syncthreads();
    for (int k = threadIdx.x; k < d.K; k += blockDim.x) {
        int l = degree_of(k), m = k - l * l - l, am = m < 0 ? -m : m;
        const T *tm = Tm + (m + d.lmax) * d.U;
        int pi = l * (l + 1) / 2 + am;
        T s = 0;
        for (int u = 0; u < d.U; ++u) s += tb.wq[u] * tb.p[(size_t)u * d.P + pi] * tm[u];
        out[k] = s;
    }
}

// Quadrature analysis (Eqs. struct-Tmu, struct-Tlm) of two grid fields S1, S2
// [UV] held on chip, through Tm scratch [2][M][U]; writes out1/out2 [K].
template <typename T>
__device__ void analysis2(const Tabs<T> &tb, const T *q, const T *S1, const T *S2, T *Tm, T *out1,
                          T *out2)
{
    const Dims &d = tb.d;
    const int MU = d.M * d.U;
    for (int idx = threadIdx.x; idx < 2 * MU; idx += blockDim.x) {
        int which = idx >= MU;
        int rem = idx - which * MU;
        int mi = rem / d.U, u = rem - mi * d.U;
        const T *S = (which ? S2 : S1) + u * d.V;
        T s = 0;
        for (int v = 0; v < d.V; ++v) s += q[v * d.M + mi] * S[v];
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

// Quadrature analysis of the curl product in the moved-derivative form, plus a value field:
// Sv, S1, S2 [UV] on chip (Sv may be null, and S1, S2 both null), through Tm scratch
// [3][M][U]; writes
//   out[l, m] = sum_u wq_u [ Pt_l^|m|(x_u) (Fv[m][u] - m F1[-m][u]) - dPt_l^|m|/dx(x_u) F2[m][u] ]
// with F_f[m][u] = sum_v q_vm S_f[u][v]. The first term is the analysis of Sv (Eqs.
// struct-Tmu, struct-Tlm). The others are the analysis of the surface curl of Eq.
// poisson-S2-x after moving both derivatives onto the test function: on the sphere, with
// {f, g} = f_phi g_x - f_x g_phi, the integral of Y {A, B} equals that of B {Y, A}, and the
// grid integrates both exactly, so with S1 = sum_j B_j dA_j/dx and S2 = sum_j B_j dA_j/dphi
// the curl's coefficient is the analysis of S1 against dY/dphi minus that of S2 against dY/dx.
// dY_lm/dphi = Pt_l^|m| times the order-swapped Fourier factor -m q_{-m}.
template <typename T>
__device__ void analysis_moved(const Tabs<T> &tb, const T *q, const T *Sv, const T *S1,
                               const T *S2, T *Tm, T *out)
{
    const Dims &d = tb.d;
    const int MU = d.M * d.U;
    const bool hv = Sv != nullptr, hc = S1 != nullptr;
    const int f0 = hv ? 0 : 1, f1 = hc ? 3 : 1;  // the fields present: f0 <= f < f1
    for (int idx = threadIdx.x; idx < (f1 - f0) * MU; idx += blockDim.x) {
        const int f = f0 + idx / MU, rem = idx - (f - f0) * MU;
        const int mi = rem / d.U, u = rem - mi * d.U;
        const T *S = (f == 0 ? Sv : f == 1 ? S1 : S2) + u * d.V;
        T s = 0;
        for (int v = 0; v < d.V; ++v) s += q[v * d.M + mi] * S[v];
        Tm[f * MU + rem] = s;
    }
    __syncthreads();
    for (int k = threadIdx.x; k < d.K; k += blockDim.x) {
        const int l = degree_of(k), m = k - l * l - l, am = m < 0 ? -m : m;
        const T *tv = Tm + (m + d.lmax) * d.U;
        const T *t1 = Tm + MU + (d.lmax - m) * d.U;
        const T *t2 = Tm + 2 * MU + (m + d.lmax) * d.U;
        const int pi = l * (l + 1) / 2 + am;
        const T fm = (T)m;
        T s = 0;
        for (int u = 0; u < d.U; ++u) {
            const T p = tb.p[(size_t)u * d.P + pi];
            T t = 0;
            if (hv) t += p * tv[u];
            if (hc) t += -fm * p * t1[u] - tb.dp[(size_t)u * d.P + pi] * t2[u];
            s += tb.wq[u] * t;
        }
        out[k] = s;
    }
}

// Copy the [V][M] Fourier table into LDS (callers synchronise afterwards).
template <typename T>
__device__ __forceinline__ void stage_q(const Tabs<T> &tb, T *qs)
{
    for (int k = threadIdx.x; k < tb.d.V * tb.d.M; k += blockDim.x) qs[k] = tb.q[k];
}

// ---------------------------------------------------------------------------
// Sender (node-side) grid fields: SF[b][r][0..2][UV] = (A, dA/dx, dA/dphi); only the fields
// whose bit is set in `planes` are stored (bit 8: A into plane 1).
// One block per (node, rb consecutive ranks): the Legendre pass of all rb ranks,
// then every thread writes the three fields of its grid points for each rank.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void k_sender_fields(Tabs<T> tb, int R, int rb,
                                                            const T *__restrict__ H,
                                                            T *__restrict__ SF, int planes)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    const int MU = d.M * d.U;
    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    T *qs = smem;               // [V][M]
    T *Hs = qs + d.V * d.M;     // [rb][K]
    T *F = Hs + rb * d.K;       // [rb][M][U]
    T *Fx = F + rb * MU;        // [rb][M][U]
    stage_q(tb, qs);
    const T *hsrc = H + (b * R + r0) * (int64_t)d.K;
    for (int k = threadIdx.x; k < nr * d.K; k += blockDim.x) Hs[k] = hsrc[k];
    __syncthreads();
    for (int q = 0; q < nr; ++q) legendre_synth(tb, Hs + q * d.K, F + q * MU, Fx + q * MU);
    __syncthreads();
    T *out = SF + (b * R + r0) * 3 * (int64_t)d.UVs;
    for (int uv = threadIdx.x; uv < d.UV; uv += blockDim.x) {
        const int u = uv / d.V, v = uv - u * d.V;
        for (int q = 0; q < nr; ++q) {
            T a, ax, ap;
            fourier_point(tb, qs, F + q * MU, Fx + q * MU, u, v, a, ax, ap);
            T *o = out + (int64_t)q * 3 * d.UVs + uv;
            if (planes & 1) o[0] = a;
            if (planes & 2) o[d.UVs] = ax;
            if (planes & 4) o[2 * d.UVs] = ap;
            if (planes & 8) o[d.UVs] = a;
        }
    }
}

template <typename T>
hipError_t launch_sender_fields(const Tabs<T> &tb, int64_t B, int R, const T *H, T *SF,
                                hipStream_t s, int planes)
{
    if (B == 0) return hipSuccess;
    if constexpr (sizeof(T) == 4) {
        hipError_t e = launch_sender_mfma(tb, B, R, H, SF, false, s, planes);
        if (e != hipErrorNotSupported) return e;
    }
    const size_t per_rank = tb.d.K + 2 * (size_t)tb.d.M * tb.d.U;
    const size_t fixed = (size_t)tb.d.V * tb.d.M;
    int rb = (int)((48 * 1024 / sizeof(T) - fixed) / per_rank);
    if (rb > 8) rb = 8;
    if (rb < 1) rb = 1;
    if (rb > R) rb = R;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    const size_t sh = sizeof(T) * (fixed + rb * per_rank);
    hipLaunchKernelGGL(k_sender_fields<T>, dim3((unsigned)blocks), dim3(kThreads), sh, s, tb, R,
                       rb, H, SF, planes);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// On-site: per (node, rank) synthesise both operands, form
//   S_alpha = A1 A2 (Eq. struct-S)  and
//   S_beta  = dA1/dphi dA2/dx - dA1/dx dA2/dphi (Eq. poisson-S2-x),
// then analyse both back to (l, m).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void k_onsite_grid(Tabs<T> tb, int R, int q_in_lds,
                                                          const T *__restrict__ HA,
                                                          const T *__restrict__ HB,
                                                          T *__restrict__ Ta, T *__restrict__ Tb)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    const int64_t br = blockIdx.x;
    const int MU = d.M * d.U;
    // the Fourier table is staged in LDS unless that would exceed the workgroup's LDS
    T *qs = smem;
    T *H1 = qs + (q_in_lds ? d.V * d.M : 0);
    T *H2 = H1 + d.K;
    T *F1 = H2 + d.K;
    T *F1x = F1 + MU;
    T *F2 = F1x + MU;
    T *F2x = F2 + MU;
    T *Sa = F2x + MU;
    T *Sb = Sa + d.UV;
    if (q_in_lds) stage_q(tb, qs);
    const T *q = q_in_lds ? qs : tb.q;
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
        fourier_point(tb, q, F1, F1x, u, v, a1, a1x, a1p);
        fourier_point(tb, q, F2, F2x, u, v, a2, a2x, a2p);
        Sa[uv] = a1 * a2;
        Sb[uv] = a1p * a2x - a1x * a2p;
    }
    __syncthreads();
    analysis2(tb, q, Sa, Sb, F1 /* reused as Tm scratch [2][M][U] */, Ta + br * d.K,
              Tb + br * d.K);
}

template <typename T>
hipError_t launch_onsite_grid(const Tabs<T> &tb, int64_t B, int R, const T *HA, const T *HB,
                              T *Ta, T *Tb, hipStream_t s)
{
    int64_t blocks = B * R;
    if (blocks == 0) return hipSuccess;
    if constexpr (sizeof(T) == 4) {
        if (tb.d.lmax >= kOnsiteMfmaMinL) {
            hipError_t e = launch_onsite_mfma(tb, B, R, HA, HB, Ta, Tb, s);
            if (e != hipErrorNotSupported) return e;
        }
        if (tb.d.lmax <= kOnsiteFoldedMaxL) {
            hipError_t e = launch_onsite_folded(tb, B, R, HA, HB, Ta, Tb, s);
            if (e != hipErrorNotSupported && e != hipErrorInvalidValue) return e;
        }
    }
    const size_t base = 2 * tb.d.K + 4 * tb.d.M * tb.d.U + 2 * tb.d.UV;
    const size_t with_q = base + tb.d.V * tb.d.M;
    const int q_in_lds = sizeof(T) * with_q <= (size_t)tb.d.lds_max ? 1 : 0;
    const size_t sh = sizeof(T) * (q_in_lds ? with_q : base);
    hipLaunchKernelGGL(k_onsite_grid<T>, dim3((unsigned)blocks), dim3(kThreads), sh, s, tb, R,
                       q_in_lds, HA, HB, Ta, Tb);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// nu-body on-site product: per (node, rank) synthesise the values of the nu operands'
// fields, multiply them pointwise on the grid and analyse the product back to (l, m) (the
// grid product extended to nu operands, one inverse transform). The plan's grid must be fine
// enough for the (nu + 1) lmax integrand.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void k_nbody_grid(Tabs<T> tb, int R, int nu, int q_in_lds,
                                                         NbodyOperands<T> H, T *__restrict__ Tout)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    const int64_t br = blockIdx.x;
    const int MU = d.M * d.U;
    T *qs = smem;
    T *Hs = qs + (q_in_lds ? d.V * d.M : 0);  // [nu][K]
    T *F = Hs + nu * d.K;                       // [nu][M][U]
    T *S = F + nu * MU;                         // [UV]
    T *Tm = S + d.UV;                           // [M][U]
    if (q_in_lds) stage_q(tb, qs);
    const T *q = q_in_lds ? qs : tb.q;
    for (int t = 0; t < nu; ++t)
        for (int k = threadIdx.x; k < d.K; k += blockDim.x) Hs[t * d.K + k] = H.h[t][br * d.K + k];
    __syncthreads();
    for (int t = 0; t < nu; ++t) legendre_value(tb, Hs + t * d.K, F + t * MU);
    __syncthreads();
    for (int uv = threadIdx.x; uv < d.UV; uv += blockDim.x) {
        const int u = uv / d.V, v = uv - u * d.V;
        T prod = fourier_value(tb, q, F, u, v);
        for (int t = 1; t < nu; ++t) prod *= fourier_value(tb, q, F + t * MU, u, v);
        S[uv] = prod;
    }
    __syncthreads();
    analysis1(tb, q, S, Tm, Tout + br * d.K);
}

template <typename T>
hipError_t launch_nbody_grid(const Tabs<T> &tb, int64_t B, int R, int nu,
                             const NbodyOperands<T> &H, T *Tout, hipStream_t s)
{
    const int64_t blocks = B * R;
    if (blocks == 0) return hipSuccess;
    if (nu < 1 || nu > kMaxNu) return hipErrorInvalidValue;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    if constexpr (sizeof(T) == 4) {
        hipError_t e = launch_nbody_folded(tb, B, R, nu, H, Tout, s);
        if (e != hipErrorNotSupported) return e;
    }
    const size_t MU = (size_t)tb.d.M * tb.d.U;
    const size_t base = nu * (tb.d.K + MU) + tb.d.UV + MU;
    const size_t with_q = base + (size_t)tb.d.V * tb.d.M;
    const int q_in_lds = sizeof(T) * with_q <= (size_t)tb.d.lds_max ? 1 : 0;
    const size_t sh = sizeof(T) * (q_in_lds ? with_q : base);
    if (sh > (size_t)tb.d.lds_max) return hipErrorNotSupported;
    hipLaunchKernelGGL(k_nbody_grid<T>, dim3((unsigned)blocks), dim3(kThreads), sh, s, tb, R, nu,
                       q_in_lds, H, Tout);
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
    // renormalised: fp32 by the hardware reciprocal square root (within 1 ulp), fp64 exactly
    T inv;
    if constexpr (sizeof(T) == 4) inv = __builtin_amdgcn_rsqf(ux * ux + uy * uy + uz * uz);
    else inv = (T)1 / sqrt(ux * ux + uy * uy + uz * uz);
    ux *= inv;
    uy *= inv;
    uz *= inv;
}

// Block = (receiver i, RB consecutive ranks); thread = NPT fixed grid points.
// Per edge, the Legendre recurrence in t = rhat . Omega runs once per point and
// serves all RB ranks; the 3 RB sender values of a point are loaded before the
// arithmetic so that their latency overlaps it.
constexpr int kRecvMaxThreads = 1024;
constexpr int kRecvEdgeChunk = 16;  // edges whose coefficients a receiver block stages at once

// Raw buffer loads: one descriptor per edge over the sender's rank block; every
// load of a grid point shares its VGPR byte offset and differs only in a scalar
// offset. Out-of-range offsets read 0 (num_records bounds the block).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

template <typename T>
__device__ __forceinline__ T buf_load(__amdgpu_buffer_rsrc_t rs, unsigned voff, unsigned soff);

template <>
__device__ __forceinline__ float buf_load<float>(__amdgpu_buffer_rsrc_t rs, unsigned voff,
                                                 unsigned soff)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, 0));
}

template <>
__device__ __forceinline__ double buf_load<double>(__amdgpu_buffer_rsrc_t rs, unsigned voff,
                                                   unsigned soff)
{
    return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(rs, voff, soff, 0));
}

// TWO: the senders carry a second, parity-flipped node slot SFf (same layout as SF). By
// Table 1 its Gaunt product then feeds Tb and its curl product Ta.
// SPLIT: the curl product takes the edge coefficients Rtg (its own CP factors) for the
// derivative sum g, the Gaunt product Rt for the value sum a.
// VAL: the curl product in the moved-derivative form of analysis_moved. The senders then
// only need their value plane (plane 0 of each rank's three; with SPLIT the curl factors'
// values in plane 1): per point and rank the block accumulates the Gaunt sum a B and the two
// sums B dA/dx, B dA/dphi of the edge field's derivatives.
template <typename T, int RB, int NPT, bool FULL, bool TWO, bool SPLIT, bool VAL>
__global__ __launch_bounds__(kRecvMaxThreads) void k_receiver_zonal(
    Tabs<T> tb, int R, int64_t N, const int32_t *__restrict__ row_ptr,
    const int32_t *__restrict__ col, const int32_t *__restrict__ order,
    const T *__restrict__ unit, const T *__restrict__ Rt, const T *__restrict__ Rtg,
    const T *__restrict__ SF, const T *__restrict__ SFf, T *__restrict__ Ta, T *__restrict__ Tb,
    T *__restrict__ Sg)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    const int UV = d.UV, L = d.L, lmax = d.lmax;
    // Block order (recv_block): the slices are the rank blocks.
    int64_t c, i;
    if (!recv_block(N, order, c, i)) return;
    const int r0 = (int)c * RB;
    // FULL: R is a multiple of RB, so every rank of the block exists (no guards)
    const int nr = FULL ? RB : ((R - r0 < RB) ? (R - r0) : RB);

    int uvs[NPT];
    T px[NPT], psx[NPT], pxsx[NPT], pcp[NPT], psp[NPT];
#pragma unroll
    for (int s = 0; s < NPT; ++s) {
        int uv = threadIdx.x + s * blockDim.x;
        uvs[s] = uv;
        int uvc = uv < UV ? uv : 0;
        int u = uvc / d.V, v = uvc - u * d.V;
        px[s] = tb.x[u];
        psx[s] = tb.sx[u];
        pxsx[s] = tb.xsx[u];
        pcp[s] = tb.cphi[v];
        psp[s] = tb.sphi[v];
    }
    // VAL: sa, sb the Gaunt sums into Ta, Tb; (ca1, ca2) the moved curl sums into Ta (the
    // flipped slot's, TWO), (cb1, cb2) into Tb (the natural slot's)
    T sa[NPT][RB], sb[NPT][RB], ca1[NPT][RB], ca2[NPT][RB], cb1[NPT][RB], cb2[NPT][RB];
#pragma unroll
    for (int s = 0; s < NPT; ++s)
#pragma unroll
        for (int q = 0; q < RB; ++q) sa[s][q] = sb[s][q] = ca1[s][q] = ca2[s][q] = cb1[s][q] = cb2[s][q] = 0;

    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    // the next edge's sender index and direction are fetched one iteration ahead
    // (the sender index is the same for the whole block: readfirstlane keeps it, and the
    // per-edge base address, in scalar registers)
    int jn = 0;
    T uxn = 0, uyn = 0, uzn = 1;
    if (e0 < e1) {
        jn = __builtin_amdgcn_readfirstlane(col[e0]);
        load_unit(unit, e0, uxn, uyn, uzn);
    }
    // SPLIT (two coefficient sets per edge): the block's edge coefficients are staged in LDS
    // kRecvEdgeChunk edges at a time, as Rs[edge][set][l][q] (set 1: the curl's Rtg; ranks
    // past nr zero), and read from there as broadcasts; one set is read from global memory
    // as uniform (scalar) loads, which keep the single-set kernels at fewer registers
    constexpr bool STAGE = SPLIT;
    constexpr int NSET = SPLIT ? 2 : 1;
    const int rstride = STAGE ? RB : R;  // between the degrees of one edge's coefficients
    T *Rs = smem;
    for (int ec = e0; ec < e1; ec += (STAGE ? kRecvEdgeChunk : e1 - e0)) {
        const int ne = STAGE ? ((e1 - ec < kRecvEdgeChunk) ? (e1 - ec) : kRecvEdgeChunk)
                             : e1 - e0;
        if (STAGE) {
            __syncthreads();  // the previous chunk is consumed
            for (int k = threadIdx.x; k < ne * NSET * L * RB; k += blockDim.x) {
                const int q = k % RB, rest = k / RB;
                const int l = rest % L, es = rest / L;
                const int set = es % NSET, ee = es / NSET;
                const T *src = set ? Rtg : Rt;
                Rs[k] = (FULL || q < nr) ? src[((int64_t)(ec + ee) * L + l) * R + r0 + q]
                                         : (T)0;
            }
            __syncthreads();
        }
        for (int e = ec; e < ec + ne; ++e) {
            const int64_t j = jn;
            const T ux = uxn, uy = uyn, uz = uzn;
            if (e + 1 < e1) {
                jn = __builtin_amdgcn_readfirstlane(col[e + 1]);
                load_unit(unit, e + 1, uxn, uyn, uzn);
            }
            // rt[l * rstride + q] = Rt[e][l][r0 + q], rtg the same of Rtg
            const T *rt = STAGE ? Rs + (e - ec) * NSET * L * RB : Rt + (int64_t)e * L * R + r0;
            const T *rtg = SPLIT ? rt + L * RB : rt;
            const int UVs = d.UVs;
            const __amdgpu_buffer_rsrc_t sfr = make_rsrc(SF + (j * R + r0) * 3 * (int64_t)UVs,
                                                         (unsigned)(nr * 3 * UVs * sizeof(T)));
            const __amdgpu_buffer_rsrc_t sff =
                make_rsrc((TWO ? SFf : SF) + (j * R + r0) * 3 * (int64_t)UVs,
                          (unsigned)(nr * 3 * UVs * sizeof(T)));
            const unsigned fstride = (unsigned)(UVs * sizeof(T));
#pragma unroll
            for (int s = 0; s < NPT; ++s) {
                const int uv = uvs[s];
                if (uv >= UV) continue;
                const unsigned voff = (unsigned)(uv * sizeof(T));
                T fI[RB], fX[RB], fP[RB], gI[RB], gX[RB], gP[RB];
#pragma unroll
                for (int q = 0; q < RB; ++q) {
                    // ranks past nr fall outside the descriptor's range and read 0
                    fI[q] = buf_load<T>(sfr, voff, (3 * q) * fstride);
                    if (!VAL || SPLIT) fX[q] = buf_load<T>(sfr, voff, (3 * q + 1) * fstride);
                    if (!VAL) fP[q] = buf_load<T>(sfr, voff, (3 * q + 2) * fstride);
                    if (TWO) {
                        gI[q] = buf_load<T>(sff, voff, (3 * q) * fstride);
                        if (!VAL) {
                            gX[q] = buf_load<T>(sff, voff, (3 * q + 1) * fstride);
                            gP[q] = buf_load<T>(sff, voff, (3 * q + 2) * fstride);
                        }
                    }
                }
        const T h = ux * pcp[s] + uy * psp[s];
                const T t = uz * px[s] + psx[s] * h;
                T a[RB], g[RB];
#pragma unroll
                for (int q = 0; q < RB; ++q) {
                    a[q] = (FULL || q < nr) ? rt[q] : (T)0;
                    g[q] = 0;
                }
                if (lmax >= 1) {
#pragma unroll
                    for (int q = 0; q < RB; ++q) {
                        T c = (FULL || q < nr) ? rt[rstride + q] : (T)0;
                        a[q] += c * t;
                        g[q] = SPLIT ? ((FULL || q < nr) ? rtg[rstride + q] : (T)0) : c;
                    }
                }
                T p0 = 1, p1 = t, d1 = 1;
                for (int l = 2; l <= lmax; ++l) {
                    const T p2 = tb.rc1[l] * t * p1 - tb.rc2[l] * p0;
                    const T d2 = (T)l * p1 + t * d1;
#pragma unroll
                    for (int q = 0; q < RB; ++q) {
                        T c = (FULL || q < nr) ? rt[l * rstride + q] : (T)0;
                        T cg = SPLIT ? ((FULL || q < nr) ? rtg[l * rstride + q] : (T)0) : c;
                        a[q] += c * p2;
                        g[q] += cg * d2;
                    }
                    p0 = p1;
                    p1 = p2;
                    d1 = d2;
                }
                const T dxt = uz - pxsx[s] * h;
                const T dpt = psx[s] * (uy * pcp[s] - ux * psp[s]);
#pragma unroll
                for (int q = 0; q < RB; ++q) {
                    if (VAL) {
                        // dA/dx = g dxt and dA/dphi = g dpt of the edge field
                        sa[s][q] += a[q] * fI[q];
                        // SPLIT: the curl takes the curl factors' values (plane 1)
                        const T gf = g[q] * (SPLIT ? fX[q] : fI[q]);
                        cb1[s][q] += dxt * gf;
                        cb2[s][q] += dpt * gf;
                        if (TWO) {
                            sb[s][q] += a[q] * gI[q];
                            const T gg = g[q] * gI[q];
                            ca1[s][q] += dxt * gg;
                            ca2[s][q] += dpt * gg;
                        }
                    } else {
                        sa[s][q] += a[q] * fI[q];
                        sb[s][q] += g[q] * (dpt * fX[q] - dxt * fP[q]);
                        if (TWO) {
                            sa[s][q] += g[q] * (dpt * gX[q] - dxt * gP[q]);
                            sb[s][q] += a[q] * gI[q];
                        }
                    }
                }
            }
        }
    }
    if (STAGE) __syncthreads();  // the staged coefficients are consumed before the analysis
    if (VAL && Sg) {
        // the sums go to Sg [N][R][NF][UVs] for the MFMA analysis: (Gaunt sum into Ta, moved
        // curl pair into Tb), or with two slots (value sum, moved pair) for Ta, then for Tb
        constexpr int NF = TWO ? 6 : 3;
        const int UVs = d.UVs;
#pragma unroll
        for (int q = 0; q < RB; ++q) {
            if (!FULL && q >= nr) break;
            T *o = Sg + (i * R + r0 + q) * NF * (int64_t)UVs;
#pragma unroll
            for (int s = 0; s < NPT; ++s) {
                const int uv = uvs[s];
                if (uv >= UV) continue;
                o[uv] = sa[s][q];
                if (TWO) {
                    o[UVs + uv] = ca1[s][q];
                    o[2 * UVs + uv] = ca2[s][q];
                    o[3 * UVs + uv] = sb[s][q];
                    o[4 * UVs + uv] = cb1[s][q];
                    o[5 * UVs + uv] = cb2[s][q];
                } else {
                    o[UVs + uv] = cb1[s][q];
                    o[2 * UVs + uv] = cb2[s][q];
                }
            }
        }
        return;
    }
    // inverse transforms, one rank at a time through LDS
    T *qs = smem;
    T *Sa = qs + d.V * d.M;
    T *Sb = Sa + UV;
    T *Tm = Sb + UV;
    stage_q(tb, qs);
    if (VAL) {
        // one output at a time: its value sum (if any) and moved curl pair (if any)
        T *S1 = Sb + UV, *Tm3 = S1 + UV;
#pragma unroll
        for (int q = 0; q < RB; ++q) {
            if (q >= nr) break;
            const int64_t br = i * R + r0 + q;
#pragma unroll
            for (int o = 0; o < 2; ++o) {
                const bool hv = o == 0 || TWO, hc = o == 1 || TWO;
#pragma unroll
                for (int s = 0; s < NPT; ++s) {
                    if (uvs[s] < UV) {
                        Sa[uvs[s]] = o ? sb[s][q] : sa[s][q];
                        S1[uvs[s]] = o ? cb1[s][q] : ca1[s][q];
                        Sb[uvs[s]] = o ? cb2[s][q] : ca2[s][q];
                    }
                }
                __syncthreads();
                analysis_moved(tb, qs, hv ? Sa : (const T *)nullptr, hc ? S1 : (const T *)nullptr,
                               hc ? Sb : (const T *)nullptr, Tm3, (o ? Tb : Ta) + br * d.K);
                __syncthreads();
            }
        }
        return;
    }
#pragma unroll
    for (int q = 0; q < RB; ++q) {
        if (q >= nr) break;
#pragma unroll
        for (int s = 0; s < NPT; ++s) {
            if (uvs[s] < UV) {
                Sa[uvs[s]] = sa[s][q];
                Sb[uvs[s]] = sb[s][q];
            }
        }
        __syncthreads();
        const int64_t br = i * R + r0 + q;
        analysis2(tb, qs, Sa, Sb, Tm, Ta + br * d.K, Tb + br * d.K);
        __syncthreads();
    }
}

// Read-pattern ceiling of k_receiver_zonal in its value-only form (the moved-derivative curl):
// the same blocks in the same order, the same wave-uniform sender index per edge and the
// same raw buffer loads of the RB sender values of every grid point, with nothing computed
// from them but a running sum. sink
// receives a value only if that sum equals a constant no finite input sums to by chance,
// which keeps every load live.
template <int RB>
__global__ __launch_bounds__(kRecvMaxThreads) void k_gather_probe(
    int UV, int UVs, int R, int64_t N, const int32_t *__restrict__ row_ptr,
    const int32_t *__restrict__ col, const int32_t *__restrict__ order,
    const float *__restrict__ SF, float *__restrict__ sink)
{
    int64_t c, i;
    if (!recv_block(N, order, c, i)) return;
    const int r0 = (int)c * RB;
    const int nr = (R - r0 < RB) ? (R - r0) : RB;
    const int uv = threadIdx.x;
    const unsigned voff = (unsigned)(uv * sizeof(float));
    const unsigned fstride = (unsigned)(UVs * sizeof(float));
    float acc = 0.f;
    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    for (int e = e0; e < e1; ++e) {
        const int64_t j = __builtin_amdgcn_readfirstlane(col[e]);
        const __amdgpu_buffer_rsrc_t sfr = make_rsrc(SF + (j * R + r0) * 3 * (int64_t)UVs,
                                                     (unsigned)(nr * 3 * UVs * sizeof(float)));
        if (uv < UV) {
#pragma unroll
            for (int q = 0; q < RB; ++q) acc += buf_load<float>(sfr, voff, (3 * q) * fstride);
        }
    }
    if (acc == -1.2345678e30f) sink[0] = acc;
}

hipError_t launch_gather_probe(const Dims &d, int64_t N, int R, const int32_t *row_ptr,
                               const int32_t *col, const int32_t *order, const float *SF,
                               float *sink, hipStream_t s)
{
    // the rank block of the fp32 value-only receiver at one point per thread: 16 ranks when
    // they divide R, else 8
    if (d.UV > kRecvMaxThreads) return hipErrorNotSupported;
    const int threads = (d.UV + 63) / 64 * 64;
    const int rb = R % 16 == 0 ? 16 : 8;
    if (N == 0 || R == 0) return hipSuccess;
    const int64_t nb = recv_blocks(N, (R + rb - 1) / rb);
    if (nb > 0x7fffffffLL) return hipErrorInvalidValue;
    if (rb == 16)
        hipLaunchKernelGGL(k_gather_probe<16>, dim3((unsigned)nb), dim3(threads), 0, s, d.UV,
                           d.UVs, R, N, row_ptr, col, order, SF, sink);
    else
        hipLaunchKernelGGL(k_gather_probe<8>, dim3((unsigned)nb), dim3(threads), 0, s, d.UV,
                           d.UVs, R, N, row_ptr, col, order, SF, sink);
    return hipGetLastError();
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
    Tabs<T> tb, int R, int64_t N, const int32_t *__restrict__ row_ptr,
    const int32_t *__restrict__ col, const int32_t *__restrict__ order,
    const T *__restrict__ unit, const T *__restrict__ Rt, const T *__restrict__ SF,
    T *__restrict__ Ta, T *__restrict__ Tb)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    // Block order (recv_block): the slices are the ranks.
    int64_t rr, i;
    if (!recv_block(N, order, rr, i)) return;
    const int r = (int)rr;
    const int64_t br = i * R + r;
    const int MU = d.M * d.U;
    T *qs = smem;
    T *Sa = qs + d.V * d.M;
    T *Sb = Sa + d.UV;
    T *Y = Sb + d.UV;
    T *F = Y + d.K;
    T *Fx = F + MU;
    stage_q(tb, qs);
    for (int uv = threadIdx.x; uv < d.UV; uv += blockDim.x) Sa[uv] = Sb[uv] = 0;
    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    for (int e = e0; e < e1; ++e) {
        const int64_t j = col[e];
        T ux, uy, uz;
        load_unit(unit, e, ux, uy, uz);
        __syncthreads();  // previous edge done with Y / F
        edge_sh(tb, ux, uy, uz, Y);
        __syncthreads();
        const T *rt = Rt + (int64_t)e * d.L * R + r;   // Rt[e][l][r] = rt[l * R]
        for (int k = threadIdx.x; k < d.K; k += blockDim.x) Y[k] *= rt[degree_of(k) * R];
        __syncthreads();
        legendre_synth(tb, Y, F, Fx);
        __syncthreads();
        const T *sf = SF + (j * R + r) * 3 * (int64_t)d.UVs;
        for (int uv = threadIdx.x; uv < d.UV; uv += blockDim.x) {
            int u = uv / d.V, v = uv - u * d.V;
            T a, ax, ap;
            fourier_point(tb, qs, F, Fx, u, v, a, ax, ap);
            Sa[uv] += a * sf[uv];
            Sb[uv] += ap * sf[d.UVs + uv] - ax * sf[2 * d.UVs + uv];
        }
    }
    __syncthreads();
    analysis2(tb, qs, Sa, Sb, F /* Tm scratch, 2 MU */, Ta + br * d.K, Tb + br * d.K);
}

// Receiver for a general per-edge field (two parity-bearing fields, Eq. twoparity-phi):
// the edge field no longer factors as R Y, so its channel-contracted coefficients
// HE[e][r][K] go through the Legendre and Fourier syntheses (Eqs. msgpass-FI, msgpass-AI
// and their derivative passes, applied on the edge side) and multiply the streamed sender
// fields (Eqs. msgpass-S, cat-beta-curl). One workgroup per (receiver, RB ranks), one
// thread per grid point (NPT points per thread). Per edge the RB ranks' coefficients sit in
// LDS (double-buffered: the next edge's are loaded while this one is transformed), the
// Legendre stage F, dF/dx is shared through LDS (with the Legendre tables in LDS when LT),
// and each thread forms the Fourier sums at its points and accumulates in registers. The
// sender fields of an edge are requested before its Legendre stage, so their latency is
// hidden behind it. Blocks run rank block by rank block, all receivers inside one, as in
// k_receiver_zonal.
constexpr int kFieldsKpt = 8;  // staged coefficients per thread and edge, at most

template <typename T, int RB, int NPT, bool FULL, bool LT>
__global__ __launch_bounds__(kRecvMaxThreads) void k_receiver_fields(
    Tabs<T> tb, int R, int64_t N, const int32_t *__restrict__ row_ptr,
    const int32_t *__restrict__ col, const int32_t *__restrict__ order,
    const T *__restrict__ HE, const T *__restrict__ SF, T *__restrict__ Ta, T *__restrict__ Tb)
{
    extern __shared__ unsigned char smem_raw[];
    T *smem = reinterpret_cast<T *>(smem_raw);
    const Dims &d = tb.d;
    const int UV = d.UV, UVs = d.UVs, K = d.K, MU = d.M * d.U, lmax = d.lmax, P = d.P;
    int64_t c, i;
    if (!recv_block(N, order, c, i)) return;
    const int r0 = (int)c * RB;
    const int nr = FULL ? RB : ((R - r0 < RB) ? (R - r0) : RB);
    const int nk = nr * K;  // staged coefficients of one edge
    T *qs = smem;                        // [V][M]
    T *Pt = qs + d.V * d.M;              // LT: [U][P] Pt_l^m(x_u), then [U][P] dPt/dx
    T *Dt = Pt + (LT ? d.U * P : 0);
    T *Hs = Dt + (LT ? d.U * P : 0);     // [2][RB][K] coefficients of this / the next edge
    T *F = Hs + 2 * RB * K;              // [RB][M][U]
    T *Fx = F + RB * MU;                 // [RB][M][U]
    stage_q(tb, qs);
    if (LT) {
        for (int k = threadIdx.x; k < d.U * P; k += blockDim.x) {
            Pt[k] = tb.p[k];
            Dt[k] = tb.dp[k];
        }
    }
    const T *ptab = LT ? Pt : tb.p;
    const T *dtab = LT ? Dt : tb.dp;

    int uvs[NPT], us[NPT], vs[NPT];
#pragma unroll
    for (int s = 0; s < NPT; ++s) {
        const int uv = threadIdx.x + s * blockDim.x;
        const int uvc = uv < UV ? uv : 0;
        uvs[s] = uv;
        us[s] = uvc / d.V;
        vs[s] = uvc - us[s] * d.V;
    }
    T sa[NPT][RB], sb[NPT][RB];
#pragma unroll
    for (int s = 0; s < NPT; ++s)
#pragma unroll
        for (int q = 0; q < RB; ++q) sa[s][q] = sb[s][q] = 0;

    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    if (e0 < e1) {
        const T *he = HE + ((int64_t)e0 * R + r0) * K;
        for (int k = threadIdx.x; k < nk; k += blockDim.x) Hs[k] = he[k];
    }
    for (int e = e0; e < e1; ++e) {
        const int cur = (e - e0) & 1;
        __syncthreads();  // this edge's coefficients are staged; the previous F is consumed
        const int64_t j = __builtin_amdgcn_readfirstlane(col[e]);
        // this edge's sender fields, consumed after the Legendre stage
        T fI[NPT][RB], fX[NPT][RB], fP[NPT][RB];
        const T *sf = SF + (j * R + r0) * 3 * (int64_t)UVs;
#pragma unroll
        for (int s = 0; s < NPT; ++s) {
            const int uvc = uvs[s] < UV ? uvs[s] : 0;
#pragma unroll
            for (int q = 0; q < RB; ++q) {
                const bool ok = FULL || q < nr;
                const T *f = sf + (int64_t)(ok ? q : 0) * 3 * UVs + uvc;
                fI[s][q] = ok ? f[0] : (T)0;
                fX[s][q] = ok ? f[UVs] : (T)0;
                fP[s][q] = ok ? f[2 * UVs] : (T)0;
            }
        }
        // the next edge's coefficients, stored after the Legendre stage
        T hn[kFieldsKpt];
        const bool more = e + 1 < e1;
        if (more) {
            const T *he = HE + ((int64_t)(e + 1) * R + r0) * K;
#pragma unroll
            for (int t = 0; t < kFieldsKpt; ++t) {
                const int k = threadIdx.x + t * blockDim.x;
                hn[t] = k < nk ? he[k] : (T)0;
            }
        }
        // Legendre stage of the RB ranks: F[q][mi][u] = sum_l Pt_l^|m|(x_u) HE[q][l, m]
        const T *hc = Hs + cur * RB * K;
        for (int idx = threadIdx.x; idx < RB * MU; idx += blockDim.x) {
            const int q = idx / MU, rem = idx - q * MU;
            const int mi = rem / d.U, u = rem - mi * d.U;
            const int m = mi - lmax, am = m < 0 ? -m : m;
            const T *pu = ptab + u * P;
            const T *dpu = dtab + u * P;
            const T *h = hc + q * K;
            T f = 0, fx = 0;
            if (FULL || q < nr) {
                for (int l = am; l <= lmax; ++l) {
                    const T hv = h[l * l + l + m];
                    const int pi = l * (l + 1) / 2 + am;
                    f += pu[pi] * hv;
                    fx += dpu[pi] * hv;
                }
            }
            F[idx] = f;
            Fx[idx] = fx;
        }
        if (more) {
            T *hnext = Hs + (cur ^ 1) * RB * K;
#pragma unroll
            for (int t = 0; t < kFieldsKpt; ++t) {
                const int k = threadIdx.x + t * blockDim.x;
                if (k < nk) hnext[k] = hn[t];
            }
        }
        __syncthreads();
#pragma unroll
        for (int s = 0; s < NPT; ++s) {
            if (uvs[s] >= UV) continue;
#pragma unroll
            for (int q = 0; q < RB; ++q) {
                if (!FULL && q >= nr) break;
                T a, ax, ap;
                fourier_point(tb, qs, F + q * MU, Fx + q * MU, us[s], vs[s], a, ax, ap);
                sa[s][q] += a * fI[s][q];
                sb[s][q] += ap * fX[s][q] - ax * fP[s][q];
            }
        }
    }
    // inverse transforms, one rank at a time through LDS (reusing the edge staging)
    T *Sa = Hs;
    T *Sb = Sa + UV;
    T *Tm = Sb + UV;
#pragma unroll
    for (int q = 0; q < RB; ++q) {
        if (q >= nr) break;
        __syncthreads();
#pragma unroll
        for (int s = 0; s < NPT; ++s) {
            if (uvs[s] < UV) {
                Sa[uvs[s]] = sa[s][q];
                Sb[uvs[s]] = sb[s][q];
            }
        }
        __syncthreads();
        const int64_t br = i * R + r0 + q;
        analysis2(tb, qs, Sa, Sb, Tm, Ta + br * K, Tb + br * K);
    }
}

template <typename T>
hipError_t launch_receiver_fields(const Tabs<T> &tb, int64_t N, int R, const int32_t *row_ptr,
                                  const int32_t *col, const int32_t *order, const T *HE,
                                  const T *SF, T *Ta, T *Tb, hipStream_t s)
{
    if (N == 0 || R == 0) return hipSuccess;
    const Dims &d = tb.d;
    const size_t MU = (size_t)d.M * d.U;
    const int npt = (d.UV + kRecvMaxThreads - 1) / kRecvMaxThreads;
    if (npt > 3) return hipErrorNotSupported;
    const int threads = ((d.UV + npt - 1) / npt + 63) / 64 * 64;
    // ranks per block and table staging: the largest RB whose registers (five values per
    // rank and point) and LDS (the workgroup's; the analysis reuses the edge staging, 2 UV +
    // 2 MU elements) fit, with the Legendre tables in LDS when they fit too
    const size_t analysis = 2 * (size_t)d.UV + 2 * MU;
    int rb = 0;
    bool lt = false;
    size_t sh = 0;
    // (at most two ranks per thread: the per-point Fourier sums keep about 60 registers live
    // per rank and the 1024-thread bound leaves 128)
    for (int cand : {2, 1}) {
        if (cand * npt > 2 || (size_t)cand * d.K > (size_t)kFieldsKpt * threads) continue;
        const size_t stage = cand * (2 * (size_t)d.K + 2 * MU);
        const size_t base = (size_t)d.V * d.M + (stage > analysis ? stage : analysis);
        const size_t tabs = 2 * (size_t)d.U * d.P;
        if (sizeof(T) * (base + tabs) <= (size_t)d.lds_max) {
            rb = cand, lt = true, sh = sizeof(T) * (base + tabs);
            break;
        }
        if (sizeof(T) * base <= (size_t)d.lds_max) {
            rb = cand, lt = false, sh = sizeof(T) * base;
            break;
        }
    }
    if (rb == 0) return hipErrorNotSupported;
    const int64_t blocks = recv_blocks(N, (R + rb - 1) / rb);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
#define CGTP_FIELDS(RBV, NP, LTV)                                                              \
    do {                                                                                       \
        if (R % RBV == 0)                                                                      \
            hipLaunchKernelGGL((k_receiver_fields<T, RBV, NP, true, LTV>),                     \
                               dim3((unsigned)blocks), dim3(threads), sh, s, tb, R, N,         \
                               row_ptr, col, order, HE, SF, Ta, Tb);                           \
        else                                                                                   \
            hipLaunchKernelGGL((k_receiver_fields<T, RBV, NP, false, LTV>),                    \
                               dim3((unsigned)blocks), dim3(threads), sh, s, tb, R, N,         \
                               row_ptr, col, order, HE, SF, Ta, Tb);                           \
    } while (0)
#define CGTP_FIELDS_LT(RBV, NP)                          \
    do {                                                 \
        if (lt) CGTP_FIELDS(RBV, NP, true);              \
        else CGTP_FIELDS(RBV, NP, false);                \
    } while (0)
    if (npt == 1) {
        if (rb == 2) CGTP_FIELDS_LT(2, 1);
        else CGTP_FIELDS_LT(1, 1);
    } else if (npt == 2) {
        CGTP_FIELDS_LT(1, 2);
    } else {
        CGTP_FIELDS_LT(1, 3);
    }
#undef CGTP_FIELDS_LT
#undef CGTP_FIELDS
    return hipGetLastError();
}

template <typename T>
hipError_t launch_receiver(const Tabs<T> &tb, bool separated, int64_t N, int R,
                           const int32_t *row_ptr, const int32_t *col, const int32_t *order,
                           const T *unit, const T *Rt, const T *Rtg, const T *SF, const T *SFf,
                           T *Ta, T *Tb, hipStream_t s, bool values_only, T *Sg, bool analyse)
{
    if (N == 0 || R == 0) return hipSuccess;
    const int64_t blocks = recv_blocks(N, R);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    const Dims &d = tb.d;
    if (SFf && Rtg) return hipErrorNotSupported;
    if (values_only && separated) return hipErrorInvalidValue;
    if (Sg && (!values_only || sizeof(T) != 4)) return hipErrorInvalidValue;
    if (separated) {
        if (SFf || Rtg) return hipErrorNotSupported;
        size_t sh = sizeof(T) * (d.V * d.M + 2 * d.UV + d.K + 2 * d.M * d.U);
        hipLaunchKernelGGL(k_receiver_separated<T>, dim3((unsigned)blocks), dim3(kThreads), sh, s,
                           tb, R, N, row_ptr, col, order, unit, Rt, SF, Ta, Tb);
        return hipGetLastError();
    }
    // the analysis buffers: two grid fields and two Fourier row sets, three of each with
    // values_only
    // (none when the analysis follows on MFMA)
    const int nf = values_only ? 3 : 2;
    size_t sh = Sg ? 0 : sizeof(T) * (d.V * d.M + nf * d.UV + nf * d.M * d.U);
    const int npt = (d.UV + kRecvMaxThreads - 1) / kRecvMaxThreads;
    const int threads = ((d.UV + npt - 1) / npt + 63) / 64 * 64;
    // LDS: the analysis buffers, or (split) one chunk of staged edge coefficients if larger
#define CGTP_RECV_TW(RBV, NP, TW, SP, VL)                                                      \
    do {                                                                                       \
        const int64_t nb = recv_blocks(N, (R + RBV - 1) / RBV);                                \
        if (nb > 0x7fffffffLL) return hipErrorInvalidValue;                                    \
        const size_t chunk = SP ? sizeof(T) * kRecvEdgeChunk * 2 * d.L * RBV : 0;              \
        const size_t shc = chunk > sh ? chunk : sh;                                            \
        if (shc > (size_t)d.lds_max) return hipErrorNotSupported;                              \
        if (R % RBV == 0)                                                                      \
            hipLaunchKernelGGL((k_receiver_zonal<T, RBV, NP, true, TW, SP, VL>),               \
                               dim3((unsigned)nb), dim3(threads), shc, s, tb, R, N, row_ptr,   \
                               col, order, unit, Rt, Rtg, SF, SFf, Ta, Tb, Sg);                \
        else                                                                                   \
            hipLaunchKernelGGL((k_receiver_zonal<T, RBV, NP, false, TW, SP, VL>),              \
                               dim3((unsigned)nb), dim3(threads), shc, s, tb, R, N, row_ptr,   \
                               col, order, unit, Rt, Rtg, SF, SFf, Ta, Tb, Sg);                \
    } while (0)
#define CGTP_RECV(RBV, NP)                                                  \
    do {                                                                    \
        if (values_only) {                                                  \
            if (SFf) CGTP_RECV_TW(RBV, NP, true, false, true);              \
            else if (Rtg) CGTP_RECV_TW(RBV, NP, false, true, true);         \
            else CGTP_RECV_TW(RBV, NP, false, false, true);                 \
        } else if (SFf) CGTP_RECV_TW(RBV, NP, true, false, false);          \
        else if (Rtg) CGTP_RECV_TW(RBV, NP, false, true, false);            \
        else CGTP_RECV_TW(RBV, NP, false, false, false);                    \
    } while (0)
    // ranks per block: sized so the per-thread accumulators and in-flight loads fit in
    // registers without spilling (fp64 values take two registers)
    constexpr int rb1 = sizeof(T) == 4 ? 8 : 4;
    constexpr int rb2 = sizeof(T) == 4 ? 4 : 2;
    if (npt <= 1) CGTP_RECV(rb1, 1);
    else if (npt <= 2) CGTP_RECV(rb2, 2);
    else CGTP_RECV(2, 3);
#undef CGTP_RECV
#undef CGTP_RECV_TW
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !Sg || !analyse) return e;
    if constexpr (sizeof(T) == 4)
        return launch_analysis_mfma(tb, N, R, Sg, Ta, Tb, s, SFf ? 2 : 1);
    return hipErrorInvalidValue;
}

#define CGTP_INSTANTIATE(T)                                                                      \
    template hipError_t launch_sender_fields<T>(const Tabs<T> &, int64_t, int, const T *, T *,   \
                                                hipStream_t, int);                               \
    template hipError_t launch_onsite_grid<T>(const Tabs<T> &, int64_t, int, const T *,          \
                                              const T *, T *, T *, hipStream_t);                 \
    template hipError_t launch_receiver<T>(const Tabs<T> &, bool, int64_t, int, const int32_t *, \
                                           const int32_t *, const int32_t *, const T *,          \
                                           const T *, const T *, const T *, const T *, T *, T *, \
                                           hipStream_t, bool, T *, bool);                        \
    template hipError_t launch_receiver_fields<T>(const Tabs<T> &, int64_t, int, const int32_t *, \
                                                  const int32_t *, const int32_t *, const T *,    \
                                                  const T *, T *, T *, hipStream_t);              \
    template hipError_t launch_nbody_grid<T>(const Tabs<T> &, int64_t, int, int,                  \
                                             const NbodyOperands<T> &, T *, hipStream_t);

CGTP_INSTANTIATE(float)
CGTP_INSTANTIATE(double)

}  // namespace cgtp
