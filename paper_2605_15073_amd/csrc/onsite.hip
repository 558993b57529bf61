// On-site grid stage, fp32, lmax <= kOnsiteFoldedMaxL: one workgroup per
// (node, block of rb ranks), one thread per (rank, Gauss-Legendre node u).
//
// A thread keeps the Legendre coefficients F[m] and dF/dx[m] of both operands in
// registers (Eq. struct-F and its x-derivative pass), then sweeps the azimuth in
// pairs (v, V - v): cos(m phi) is the same at both points and sin(m phi) changes
// sign, so the cosine part C and the sine part S of each synthesised field
// (Eq. struct-tildeA) give A(v) = C + S and A(V - v) = C - S. At both points it
// forms the product (Eq. struct-S) and the surface curl (Eq. poisson-S2-x), and
// accumulates the Fourier analysis (Eq. struct-Tmu) in registers with the same
// pairing. The Gauss-Legendre analysis across u (Eq. struct-Tlm) goes through LDS, one
// output field at a time, in the space the coefficient rows held (they are dead once the
// Legendre pass is in registers): the workgroup's LDS is then about half of what both
// fields' Fourier rows next to the coefficient rows took, so more ranks and workgroups fit
// per CU.
//
// With per-block factors (general parameterization) the Gaunt product takes the values of the
// Gaunt factors' contractions HA, HB and the surface curl the derivative fields of the curl
// factors' contractions HAc, HBc; that kernel sweeps the two one after the other, with both
// output rows in registers and the same LDS reuse.
#include "internal.h"

namespace cgtp {

namespace {

// qg, qdg: the Fourier factors q_vm [V][M] and their phi-derivative weights as read-only
// arguments: the azimuth sweep reads one row of each per step, the same for every thread, as
// scalar loads (operands from scalar registers, no LDS traffic in the sweep).
template <int LM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(LM == 12 || LM == 13 ? 3 : 1)))
void k_onsite_folded(Tabs<float> tb, int R, int rb,
                                                       const float *__restrict__ qg,
                                                       const float *__restrict__ qdg,
                                                       const float *__restrict__ HA,
                                                       const float *__restrict__ HB,
                                                       float *__restrict__ Ta,
                                                       float *__restrict__ Tb)
{
    constexpr int M = 2 * LM + 1, L = LM + 1, K = L * L, P = L * (L + 1) / 2;
    extern __shared__ float smem[];
    const int U = tb.d.U, V = tb.d.V;
    float *ps = smem;              // [U][P]
    float *dps = ps + U * P;       // [U][P]
    float *Hs = dps + U * P;       // [2][rb][K], then reused as
    float *Tm = Hs;                // [rb][M][U]: one field's Fourier rows

    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    for (int k = threadIdx.x; k < U * P; k += blockDim.x) {
        ps[k] = tb.p[k];
        dps[k] = tb.dp[k];
    }
    const float *ha = HA + (b * R + r0) * (int64_t)K;
    const float *hb = HB + (b * R + r0) * (int64_t)K;
    for (int k = threadIdx.x; k < nr * K; k += blockDim.x) {
        Hs[k] = ha[k];
        Hs[rb * K + k] = hb[k];
    }
    __syncthreads();

    const int q = threadIdx.x / U, u = threadIdx.x - q * U;
    const bool active = q < nr;
    float TA[M], TB[M];
#pragma unroll
    for (int mi = 0; mi < M; ++mi) TA[mi] = TB[mi] = 0.f;
    float FA[M], FxA[M], FB[M], FxB[M];
    if (active) {
        const float *h1 = Hs + q * K, *h2 = Hs + (rb + q) * K;
        const float *pu = ps + u * P, *dpu = dps + u * P;
#pragma unroll
        for (int mi = 0; mi < M; ++mi) {
            const int m = mi - LM, am = m < 0 ? -m : m;
            float f1 = 0.f, g1 = 0.f, f2 = 0.f, g2 = 0.f;
#pragma unroll
            for (int l = am; l <= LM; ++l) {
                const float p = pu[l * (l + 1) / 2 + am], dp = dpu[l * (l + 1) / 2 + am];
                const float c1 = h1[l * l + l + m], c2 = h2[l * l + l + m];
                f1 += p * c1;
                g1 += dp * c1;
                f2 += p * c2;
                g2 += dp * c2;
            }
            FA[mi] = f1;
            FxA[mi] = g1;
            FB[mi] = f2;
            FxB[mi] = g2;
        }
    }
    __syncthreads();  // every thread has its coefficients: Hs is free for Tm
    if (active) {
        for (int v = 0; 2 * v <= V; ++v) {
            const int pv = v == 0 ? 0 : V - v;
            const bool paired = v != 0 && pv != v;
            const float *qr = qg + v * M, *qdr = qdg + v * M;
            // cosine (C) and sine (S) parts of A, dA/dx, dA/dphi for both operands
            float aC = FA[LM], aS = 0.f, axC = FxA[LM], axS = 0.f, apC = 0.f, apS = 0.f;
            float bC = FB[LM], bS = 0.f, bxC = FxB[LM], bxS = 0.f, bpC = 0.f, bpS = 0.f;
#pragma unroll
            for (int k = 1; k <= LM; ++k) {
                const float c = qr[LM + k], s = qr[LM - k];
                const float kc = qdr[LM + k], mks = qdr[LM - k];  // k cos, -k sin
                aC += c * FA[LM + k];
                aS += s * FA[LM - k];
                axC += c * FxA[LM + k];
                axS += s * FxA[LM - k];
                apC += kc * FA[LM - k];
                apS += mks * FA[LM + k];
                bC += c * FB[LM + k];
                bS += s * FB[LM - k];
                bxC += c * FxB[LM + k];
                bxS += s * FxB[LM - k];
                bpC += kc * FB[LM - k];
                bpS += mks * FB[LM + k];
            }
            float sa0 = (aC + aS) * (bC + bS);
            float sb0 = (apC + apS) * (bxC + bxS) - (axC + axS) * (bpC + bpS);
            float sa1 = 0.f, sb1 = 0.f;
            if (paired) {
                sa1 = (aC - aS) * (bC - bS);
                sb1 = (apC - apS) * (bxC - bxS) - (axC - axS) * (bpC - bpS);
            }
            const float saP = sa0 + sa1, saM = sa0 - sa1, sbP = sb0 + sb1, sbM = sb0 - sb1;
            TA[LM] += saP;
            TB[LM] += sbP;
#pragma unroll
            for (int k = 1; k <= LM; ++k) {
                const float c = qr[LM + k], s = qr[LM - k];
                TA[LM + k] += c * saP;
                TA[LM - k] += s * saM;
                TB[LM + k] += c * sbP;
                TB[LM - k] += s * sbM;
            }
        }
    }
    // Gauss-Legendre analysis, one field at a time: T[k] = sum_u w_u (2 pi / V) Pt_l^|m|(x_u)
    // Tm[m][u]
#pragma unroll
    for (int which = 0; which < 2; ++which) {
        if (active) {
            float *tm = Tm + q * M * U;
#pragma unroll
            for (int mi = 0; mi < M; ++mi) tm[mi * U + u] = which ? TB[mi] : TA[mi];
        }
        __syncthreads();
        for (int idx = threadIdx.x; idx < nr * K; idx += blockDim.x) {
            const int qq = idx / K, k = idx - qq * K;
            int l = (int)sqrtf((float)k);
            while (l * l > k) --l;
            while ((l + 1) * (l + 1) <= k) ++l;
            const int m = k - l * l - l, am = m < 0 ? -m : m;
            const float *tm = Tm + qq * M * U + (m + LM) * U;
            const int pi = l * (l + 1) / 2 + am;
            float s = 0.f;
            for (int uu = 0; uu < U; ++uu) s += tb.wq[uu] * ps[uu * P + pi] * tm[uu];
            (which ? Tb : Ta)[(b * R + r0 + qq) * (int64_t)K + k] = s;
        }
        __syncthreads();  // Tm is read before the next field overwrites it
    }
}

template <int LM>
hipError_t launch_folded(const Tabs<float> &tb, int64_t B, int R, const float *HA,
                         const float *HB, float *Ta, float *Tb, hipStream_t s)
{
    constexpr int M = 2 * LM + 1, L = LM + 1, K = L * L, P = L * (L + 1) / 2;
    const int U = tb.d.U;
    int rb = 256 / U;
    if (rb > R) rb = R;
    if (rb < 1) return hipErrorInvalidValue;
    auto lds = [&](int r) {
        const int shared = 2 * r * K > r * M * U ? 2 * r * K : r * M * U;  // Hs, then Tm
        return sizeof(float) * (2 * U * P + shared);
    };
    while (rb > 1 && lds(rb) > (size_t)tb.d.lds_max) --rb;
    if (lds(rb) > (size_t)tb.d.lds_max) return hipErrorInvalidValue;
    const int threads = (rb * U + 63) / 64 * 64;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    hipLaunchKernelGGL((k_onsite_folded<LM>), dim3((unsigned)blocks), dim3(threads), lds(rb), s,
                       tb, R, rb, tb.q, tb.qd, HA, HB, Ta, Tb);
    return hipGetLastError();
}

// Azimuth sweep of one row at latitude u for the Gaunt product (Eq. struct-S): synthesise
// A from FA and B from FB at each pair (v, V - v) and add the Fourier analysis (Eq.
// struct-Tmu) of A B into T. qs row v holds cos(k phi_v) at LM + k and sin(k phi_v) at
// LM - k: the plan's table, passed down from a read-only kernel argument so that each row is
// read with scalar loads.
template <int LM>
__device__ __forceinline__ void sweep_product(const float *FA, const float *FB,
                                              const float *qs, int V, float *T)
{
    constexpr int M = 2 * LM + 1;
    for (int v = 0; 2 * v <= V; ++v) {
        const bool paired = v != 0 && 2 * v != V;
        const float *qr = qs + v * M;
        float aC = FA[LM], aS = 0.f, bC = FB[LM], bS = 0.f;
#pragma unroll
        for (int k = 1; k <= LM; ++k) {
            const float c = qr[LM + k], s = qr[LM - k];
            aC += c * FA[LM + k];
            aS += s * FA[LM - k];
            bC += c * FB[LM + k];
            bS += s * FB[LM - k];
        }
        const float s0 = (aC + aS) * (bC + bS);
        const float s1 = paired ? (aC - aS) * (bC - bS) : 0.f;
        const float sP = s0 + s1, sM = s0 - s1;
        T[LM] += sP;
#pragma unroll
        for (int k = 1; k <= LM; ++k) {
            T[LM + k] += qr[LM + k] * sP;
            T[LM - k] += qr[LM - k] * sM;
        }
    }
}

// The same sweep for the surface curl (Eq. poisson-S2-x): dA/dphi dB/dx - dA/dx dB/dphi,
// with the phi-derivatives taken from FA, FB by swapping the cosine and sine halves.
template <int LM>
__device__ __forceinline__ void sweep_curl(const float *FA, const float *FxA, const float *FB,
                                           const float *FxB, const float *qs, const float *qds,
                                           int V, float *T)
{
    constexpr int M = 2 * LM + 1;
    for (int v = 0; 2 * v <= V; ++v) {
        const bool paired = v != 0 && 2 * v != V;
        const float *qr = qs + v * M, *qdr = qds + v * M;
        float axC = FxA[LM], axS = 0.f, apC = 0.f, apS = 0.f;
        float bxC = FxB[LM], bxS = 0.f, bpC = 0.f, bpS = 0.f;
#pragma unroll
        for (int k = 1; k <= LM; ++k) {
            const float c = qr[LM + k], s = qr[LM - k];
            const float kc = qdr[LM + k], mks = qdr[LM - k];  // k cos, -k sin
            axC += c * FxA[LM + k];
            axS += s * FxA[LM - k];
            apC += kc * FA[LM - k];
            apS += mks * FA[LM + k];
            bxC += c * FxB[LM + k];
            bxS += s * FxB[LM - k];
            bpC += kc * FB[LM - k];
            bpS += mks * FB[LM + k];
        }
        const float s0 = (apC + apS) * (bxC + bxS) - (axC + axS) * (bpC + bpS);
        const float s1 =
            paired ? (apC - apS) * (bxC - bxS) - (axC - axS) * (bpC - bpS) : 0.f;
        const float sP = s0 + s1, sM = s0 - s1;
        T[LM] += sP;
#pragma unroll
        for (int k = 1; k <= LM; ++k) {
            T[LM + k] += qr[LM + k] * sP;
            T[LM - k] += qr[LM - k] * sM;
        }
    }
}

// Per-block factors: the workgroup stages the Gaunt rows HA, HB and the curl rows HAc, HBc
// once; each (rank, u) thread sweeps the surface curl from the second pair (values and
// x-derivatives), then the Gaunt product from the first (values only: the smaller register set
// while the curl's Fourier row is held), keeping both Fourier rows in registers. Once every thread has its coefficients the staged rows are dead and their LDS
// holds one output field's Fourier rows at a time for the Gauss-Legendre analysis, as in
// k_onsite_folded.
template <int LM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(LM >= 11 && LM <= 13 ? 3 : 1)))
void k_onsite_split(Tabs<float> tb, int R, int rb, const float *__restrict__ qg,
                    const float *__restrict__ qdg, const float *__restrict__ HA,
                    const float *__restrict__ HB, const float *__restrict__ HAc,
                    const float *__restrict__ HBc, float *__restrict__ Ta,
                    float *__restrict__ Tb)
{
    constexpr int M = 2 * LM + 1, L = LM + 1, K = L * L, P = L * (L + 1) / 2;
    extern __shared__ float smem[];
    const int U = tb.d.U, V = tb.d.V;
    float *ps = smem;              // [U][P]
    float *dps = ps + U * P;       // [U][P]
    float *Hs = dps + U * P;       // [4][rb][K]: HA, HB, HAc, HBc rows, then reused as
    float *Tm = Hs;                // [rb][M][U]: one field's Fourier rows

    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    for (int k = threadIdx.x; k < U * P; k += blockDim.x) {
        ps[k] = tb.p[k];
        dps[k] = tb.dp[k];
    }
    const int64_t row0 = (b * R + r0) * (int64_t)K;
    for (int k = threadIdx.x; k < nr * K; k += blockDim.x) {
        Hs[k] = HA[row0 + k];
        Hs[rb * K + k] = HB[row0 + k];
        Hs[2 * rb * K + k] = HAc[row0 + k];
        Hs[3 * rb * K + k] = HBc[row0 + k];
    }
    __syncthreads();

    const int q = threadIdx.x / U, u = threadIdx.x - q * U;
    const bool active = q < nr;
    float TA[M], TB[M];
#pragma unroll
    for (int mi = 0; mi < M; ++mi) TA[mi] = TB[mi] = 0.f;
    if (active) {
        const float *pu = ps + u * P, *dpu = dps + u * P;
        {
            const float *h1 = Hs + (2 * rb + q) * K, *h2 = Hs + (3 * rb + q) * K;
            float FA[M], FxA[M], FB[M], FxB[M];
#pragma unroll
            for (int mi = 0; mi < M; ++mi) {
                const int m = mi - LM, am = m < 0 ? -m : m;
                float f1 = 0.f, g1 = 0.f, f2 = 0.f, g2 = 0.f;
#pragma unroll
                for (int l = am; l <= LM; ++l) {
                    const float p = pu[l * (l + 1) / 2 + am], dp = dpu[l * (l + 1) / 2 + am];
                    const float c1 = h1[l * l + l + m], c2 = h2[l * l + l + m];
                    f1 += p * c1;
                    g1 += dp * c1;
                    f2 += p * c2;
                    g2 += dp * c2;
                }
                FA[mi] = f1;
                FxA[mi] = g1;
                FB[mi] = f2;
                FxB[mi] = g2;
            }
            sweep_curl<LM>(FA, FxA, FB, FxB, qg, qdg, V, TB);
        }
        {
            const float *h1 = Hs + q * K, *h2 = Hs + (rb + q) * K;
            float FA[M], FB[M];
#pragma unroll
            for (int mi = 0; mi < M; ++mi) {
                const int m = mi - LM, am = m < 0 ? -m : m;
                float f1 = 0.f, f2 = 0.f;
#pragma unroll
                for (int l = am; l <= LM; ++l) {
                    const float p = pu[l * (l + 1) / 2 + am];
                    f1 += p * h1[l * l + l + m];
                    f2 += p * h2[l * l + l + m];
                }
                FA[mi] = f1;
                FB[mi] = f2;
            }
            sweep_product<LM>(FA, FB, qg, V, TA);
        }
    }
    __syncthreads();  // every thread has its Fourier rows: Hs is free for Tm
    // Gauss-Legendre analysis, one field at a time: T[k] = sum_u w_u (2 pi / V) Pt_l^|m|(x_u)
    // Tm[m][u]
#pragma unroll
    for (int which = 0; which < 2; ++which) {
        if (active) {
            float *tm = Tm + q * M * U;
#pragma unroll
            for (int mi = 0; mi < M; ++mi) tm[mi * U + u] = which ? TB[mi] : TA[mi];
        }
        __syncthreads();
        float *dst = which ? Tb : Ta;
        for (int idx = threadIdx.x; idx < nr * K; idx += blockDim.x) {
            const int qq = idx / K, k = idx - qq * K;
            int l = (int)sqrtf((float)k);
            while (l * l > k) --l;
            while ((l + 1) * (l + 1) <= k) ++l;
            const int m = k - l * l - l, am = m < 0 ? -m : m;
            const float *tm = Tm + qq * M * U + (m + LM) * U;
            const int pi = l * (l + 1) / 2 + am;
            float s = 0.f;
            for (int uu = 0; uu < U; ++uu) s += tb.wq[uu] * ps[uu * P + pi] * tm[uu];
            dst[(b * R + r0 + qq) * (int64_t)K + k] = s;
        }
        __syncthreads();  // Tm is read before the next field overwrites it
    }
}

// LDS bytes of k_onsite_split with rb ranks per block: both Legendre tables and the four
// staged row sets, whose space then holds one field's Fourier rows.
size_t split_lds(const Dims &d, int rb)
{
    const size_t M = 2 * d.lmax + 1, L = d.lmax + 1, K = L * L, P = L * (L + 1) / 2;
    const size_t rows = 4 * K > M * d.U ? 4 * K : M * d.U;
    return sizeof(float) * (2 * d.U * P + rb * rows);
}

template <int LM>
hipError_t launch_split(const Tabs<float> &tb, int64_t B, int R, const float *HA,
                        const float *HB, const float *HAc, const float *HBc, float *Ta,
                        float *Tb, hipStream_t s)
{
    const int U = tb.d.U;
    int rb = 256 / U;
    if (rb > R) rb = R;
    if (rb < 1) return hipErrorInvalidValue;
    auto lds = [&](int r) { return split_lds(tb.d, r); };
    while (rb > 1 && lds(rb) > (size_t)tb.d.lds_max) --rb;
    if (lds(rb) > (size_t)tb.d.lds_max) return hipErrorInvalidValue;
    const int threads = (rb * U + 63) / 64 * 64;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    hipLaunchKernelGGL((k_onsite_split<LM>), dim3((unsigned)blocks), dim3(threads), lds(rb), s,
                       tb, R, rb, tb.q, tb.qd, HA, HB, HAc, HBc, Ta, Tb);
    return hipGetLastError();
}

// nu-body product in the folded form (fp32, lmax <= kNbodyFoldedMaxL, NU operands): one
// thread per (rank, Gauss-Legendre node u) keeps the Legendre coefficients F_t[m] of every
// operand in registers (Eq. struct-F), sweeps the azimuth in pairs (v, V - v) forming each
// field's value at both points from its cosine and sine parts, multiplies the NU values at
// each point and accumulates the Fourier analysis (Eq. struct-Tmu) of the product in
// registers with the same pairing. The Gauss-Legendre analysis across u (Eq. struct-Tlm)
// goes through LDS. The grid (U, V) is the plan's, exact for the (NU + 1) lmax integrand.
template <int LM, int NU>
__global__ __launch_bounds__(256) void k_nbody_folded(Tabs<float> tb, int R, int rb,
                                                      const float *__restrict__ qg,
                                                      NbodyOperands<float> H,
                                                      float *__restrict__ Tout)
{
    constexpr int M = 2 * LM + 1, L = LM + 1, K = L * L, P = L * (L + 1) / 2;
    extern __shared__ float smem[];
    const int U = tb.d.U, V = tb.d.V;
    float *ps = smem;              // [U][P]
    float *Hs = ps + U * P;        // [NU][rb][K]
    float *Tm = Hs + NU * rb * K;  // [rb][M][U]

    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    for (int k = threadIdx.x; k < U * P; k += blockDim.x) ps[k] = tb.p[k];
#pragma unroll
    for (int t = 0; t < NU; ++t) {
        const float *h = H.h[t] + (b * R + r0) * (int64_t)K;
        for (int k = threadIdx.x; k < nr * K; k += blockDim.x) Hs[t * rb * K + k] = h[k];
    }
    __syncthreads();

    const int q = threadIdx.x / U, u = threadIdx.x - q * U;
    if (q < nr) {
        float F[NU][M];
        const float *pu = ps + u * P;
#pragma unroll
        for (int t = 0; t < NU; ++t) {
            const float *h = Hs + (t * rb + q) * K;
#pragma unroll
            for (int mi = 0; mi < M; ++mi) {
                const int m = mi - LM, am = m < 0 ? -m : m;
                float f = 0.f;
#pragma unroll
                for (int l = am; l <= LM; ++l) f += pu[l * (l + 1) / 2 + am] * h[l * l + l + m];
                F[t][mi] = f;
            }
        }
        float T[M];
#pragma unroll
        for (int mi = 0; mi < M; ++mi) T[mi] = 0.f;
        for (int v = 0; 2 * v <= V; ++v) {
            const int pv = v == 0 ? 0 : V - v;
            const bool paired = v != 0 && pv != v;
            const float *qr = qg + v * M;
            float p0 = 1.f, p1 = 1.f;  // the product at v and at V - v
#pragma unroll
            for (int t = 0; t < NU; ++t) {
                float c0 = F[t][LM], s0 = 0.f;
#pragma unroll
                for (int k = 1; k <= LM; ++k) {
                    c0 += qr[LM + k] * F[t][LM + k];
                    s0 += qr[LM - k] * F[t][LM - k];
                }
                p0 *= c0 + s0;
                p1 *= c0 - s0;
            }
            if (!paired) p1 = 0.f;
            const float sP = p0 + p1, sM = p0 - p1;
            T[LM] += sP;
#pragma unroll
            for (int k = 1; k <= LM; ++k) {
                T[LM + k] += qr[LM + k] * sP;
                T[LM - k] += qr[LM - k] * sM;
            }
        }
        float *tm = Tm + q * M * U;
#pragma unroll
        for (int mi = 0; mi < M; ++mi) tm[mi * U + u] = T[mi];
    }
    __syncthreads();
    // Gauss-Legendre analysis: T[k] = sum_u w_u (2 pi / V) Pt_l^|m|(x_u) Tm[m][u]
    for (int idx = threadIdx.x; idx < nr * K; idx += blockDim.x) {
        const int qq = idx / K, k = idx - qq * K;
        int l = (int)sqrtf((float)k);
        while (l * l > k) --l;
        while ((l + 1) * (l + 1) <= k) ++l;
        const int m = k - l * l - l, am = m < 0 ? -m : m;
        const float *tm = Tm + qq * M * U + (m + LM) * U;
        const int pi = l * (l + 1) / 2 + am;
        float s = 0.f;
        for (int uu = 0; uu < U; ++uu) s += tb.wq[uu] * ps[uu * P + pi] * tm[uu];
        Tout[(b * R + r0 + qq) * (int64_t)K + k] = s;
    }
}

template <int LM, int NU>
hipError_t launch_nbody_folded_lm(const Tabs<float> &tb, int64_t B, int R,
                                  const NbodyOperands<float> &H, float *Tout, hipStream_t s)
{
    constexpr int M = 2 * LM + 1, L = LM + 1, K = L * L, P = L * (L + 1) / 2;
    const int U = tb.d.U;
    int rb = 256 / U;
    if (rb > R) rb = R;
    if (rb < 1) return hipErrorNotSupported;
    auto lds = [&](int r) { return sizeof(float) * (U * P + NU * r * K + r * M * U); };
    while (rb > 1 && lds(rb) > (size_t)tb.d.lds_max) --rb;
    if (lds(rb) > (size_t)tb.d.lds_max) return hipErrorNotSupported;
    const int threads = (rb * U + 63) / 64 * 64;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_nbody_folded<LM, NU>), dim3((unsigned)blocks), dim3(threads), lds(rb),
                       s, tb, R, rb, tb.q, H, Tout);
    return hipGetLastError();
}

template <int LM>
hipError_t launch_nbody_folded_nu(const Tabs<float> &tb, int64_t B, int R, int nu,
                                  const NbodyOperands<float> &H, float *Tout, hipStream_t s)
{
    switch (nu) {
    case 2: return launch_nbody_folded_lm<LM, 2>(tb, B, R, H, Tout, s);
    case 3: return launch_nbody_folded_lm<LM, 3>(tb, B, R, H, Tout, s);
    case 4: return launch_nbody_folded_lm<LM, 4>(tb, B, R, H, Tout, s);
    default: return hipErrorNotSupported;
    }
}

}  // namespace

bool onsite_split_supported(const Dims &d)
{
    return d.lmax <= kOnsiteFoldedMaxL && d.U <= 256 && split_lds(d, 1) <= (size_t)d.lds_max;
}

hipError_t launch_onsite_folded(const Tabs<float> &tb, int64_t B, int R, const float *HA,
                                const float *HB, float *Ta, float *Tb, hipStream_t s,
                                const float *HAc, const float *HBc)
{
    if (B == 0) return hipSuccess;
    if ((HAc == nullptr) != (HBc == nullptr)) return hipErrorInvalidValue;
    const bool split = HAc != nullptr;
    switch (tb.d.lmax) {
#define CGTP_CASE(LMV) \
    case LMV: \
        return split ? launch_split<LMV>(tb, B, R, HA, HB, HAc, HBc, Ta, Tb, s) \
                     : launch_folded<LMV>(tb, B, R, HA, HB, Ta, Tb, s);
        CGTP_CASE(0) CGTP_CASE(1) CGTP_CASE(2) CGTP_CASE(3) CGTP_CASE(4) CGTP_CASE(5)
        CGTP_CASE(6) CGTP_CASE(7) CGTP_CASE(8) CGTP_CASE(9) CGTP_CASE(10) CGTP_CASE(11)
        CGTP_CASE(12) CGTP_CASE(13) CGTP_CASE(14)
#undef CGTP_CASE
    default: return hipErrorNotSupported;
    }
}

hipError_t launch_nbody_folded(const Tabs<float> &tb, int64_t B, int R, int nu,
                               const NbodyOperands<float> &H, float *Tout, hipStream_t s)
{
    if (B == 0) return hipSuccess;
    switch (tb.d.lmax) {
#define CGTP_CASE(LMV) \
    case LMV: return launch_nbody_folded_nu<LMV>(tb, B, R, nu, H, Tout, s);
        CGTP_CASE(0) CGTP_CASE(1) CGTP_CASE(2) CGTP_CASE(3) CGTP_CASE(4) CGTP_CASE(5)
        CGTP_CASE(6) CGTP_CASE(7) CGTP_CASE(8) CGTP_CASE(9) CGTP_CASE(10)
#undef CGTP_CASE
    default: return hipErrorNotSupported;
    }
}

}  // namespace cgtp
