// Azimuthal transforms on MFMA (fp32, v_mfma_f32_16x16x4f32), specialised per lmax on the
// default grid (U = ceil((3 lmax + 2)/2) Gauss-Legendre nodes, V = 3 lmax + 1 azimuths).
//
// k_sender_mfma: node-side synthesis of the grid fields A, dA/dx, dA/dphi
//   (Eqs. msgpass-FI, msgpass-AI and the derivative passes of Eq. cat-beta-curl).
//   A workgroup owns one node and rb ranks; the product rows are (rank q, node u), the
//   columns azimuths v, and the reduction runs over the order m:
//     field[(q,u)][v] = sum_m Fs[q][m][u] q_vm,
//   with Fs = F, dF/dx, and for d/dphi the slot-swapped coefficients m F[-m]
//   (App. C: d/dphi maps cos(k phi) to -k sin(k phi) and sin(k phi) to k cos(k phi)).
//   Every lane forms exactly the A-operand values it feeds to the matrix core: lane
//   (g, n) at reduction step kk needs F, dF/dx and F[-m] of row n at m = 4 kk + g - lmax,
//   and sums them over l from the transposed Legendre tables (Eq. msgpass-FI), so the
//   Legendre stage needs no LDS.
// k_analysis_mfma: inverse transforms (Eqs. msgpass-Tmu, msgpass-Tlm) of the summed grid
//   fields S [N][R][2][UVs]: rows of S are staged in LDS, then
//     Tm[(q,u)][m] = sum_v S[q][u V + v] q_vm
//   runs on MFMA and the Gauss-Legendre sum over u reads the weighted transposed
//   Legendre table with 16-byte loads.
//
// MFMA 16x16x4 operand layout (wave64): lane = 16 g + n supplies A[row n][k g] and
// B[k g][col n]; the result lane holds D[rows 4 g + j][col n], j = 0..3.
#include "internal.h"

namespace cgtp {

namespace {

typedef float float4_t __attribute__((ext_vector_type(4)));

template <int LM>
struct Grid {
    static constexpr int L = LM + 1, M = 2 * LM + 1, K = L * L, P = L * (L + 1) / 2;
    static constexpr int U = (3 * LM + 3) / 2 < 1 ? 1 : (3 * LM + 3) / 2;
    static constexpr int V = 3 * LM + 1;
    static constexpr int UV = U * V, UVs = (UV + 31) / 32 * 32;
    static constexpr int Ut = (U + 3) / 4 * 4;        // row length of pt, dpt, wpt
    static constexpr int KM = (M + 3) / 4;            // synthesis reduction steps over m
    static constexpr int VT = (V + 15) / 16;          // synthesis column tiles over v
    static constexpr int QW = VT * 16;
    static constexpr int KV = (V + 3) / 4, VP = 4 * KV;  // analysis reduction steps over v
    static constexpr int VS = (VP + 31) / 32 * 32 + 2;  // LDS row stride: <= 2-way conflicts
    static constexpr int MT = (M + 15) / 16, MW = MT * 16;  // analysis column tiles over m
};

constexpr size_t kLdsTarget = 40 * 1024;  // keeps several workgroups resident per CU

// Largest rank block (<= 16) within the LDS target, else the largest within 64 KiB.
int pick_rb(int R, size_t fixed, size_t per_rank)
{
    int rb = R < 16 ? R : 16;
    while (rb > 1 && sizeof(float) * (fixed + rb * per_rank) > kLdsTarget) --rb;
    while (rb > 0 && sizeof(float) * (fixed + rb * per_rank) > 65536) --rb;
    return rb;
}

template <int LM>
__global__ __launch_bounds__(256) void k_sender_mfma(Tabs<float> tb, int R, int rb,
                                                     const float *__restrict__ H,
                                                     float *__restrict__ SF)
{
    using G = Grid<LM>;
    extern __shared__ float smem[];
    float *qs = smem;                    // [4 KM][QW]: q_vm as [m][v], zero padded
    float *Hs = qs + 4 * G::KM * G::QW;  // [rb][K]
    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    const int tid = threadIdx.x;
    for (int k = tid; k < 4 * G::KM * G::QW; k += 256) {
        const int m = k / G::QW, v = k - m * G::QW;
        qs[k] = (m < G::M && v < G::V) ? tb.q[v * G::M + m] : 0.f;
    }
    const float *h = H + (b * R + r0) * (int64_t)G::K;
    for (int k = tid; k < nr * G::K; k += 256) Hs[k] = h[k];
    __syncthreads();

    const int lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, n = lane & 15;
    const int rows = nr * G::U;
    const int rtiles = (rows + 15) / 16;
    for (int rt = wave; rt < rtiles; rt += 4) {
        const int ra = rt * 16 + n;  // this lane's A-operand row (q, u)
        const bool ok = ra < rows;
        const int qa = ok ? ra / G::U : 0, ua = ok ? ra - qa * G::U : 0;
        const float *hq = Hs + qa * G::K;
        const float *ptu = tb.pt + ua, *dptu = tb.dpt + ua;
        float4_t acc[3][G::VT];
#pragma unroll
        for (int t = 0; t < G::VT; ++t)
            acc[0][t] = acc[1][t] = acc[2][t] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
        for (int kk = 0; kk < G::KM; ++kk) {
            const int m = 4 * kk + g4 - LM, am = m < 0 ? -m : m;
            // lowest |m| over the four lane groups: the loop bound is wave-uniform
            const int lo = 4 * kk - LM, hi = lo + 3;
            const int am0 = (lo <= 0 && hi >= 0) ? 0 : (lo > 0 ? lo : -hi);
            float fa = 0.f, fx = 0.f, fn = 0.f;
#pragma unroll 4
            for (int l = am0; l <= LM; ++l) {
                if (l >= am) {  // also false for the padding orders |m| > lmax
                    const int pi = l * (l + 1) / 2 + am;
                    const float pv = ptu[pi * G::Ut], dv = dptu[pi * G::Ut];
                    const float cp = hq[l * l + l + m], cn = hq[l * l + l - m];
                    fa += pv * cp;
                    fx += dv * cp;
                    fn += pv * cn;
                }
            }
            const float fp = ok ? (float)m * fn : 0.f;
            if (!ok) fa = fx = 0.f;
            const float *qr = qs + (4 * kk + g4) * G::QW + n;
#pragma unroll
            for (int t = 0; t < G::VT; ++t) {
                const float bq = qr[t * 16];
                acc[0][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa, bq, acc[0][t], 0, 0, 0);
                acc[1][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(fx, bq, acc[1][t], 0, 0, 0);
                acc[2][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(fp, bq, acc[2][t], 0, 0, 0);
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int ro = rt * 16 + 4 * g4 + j;
            if (ro < rows) {
                const int qo = ro / G::U, uo = ro - qo * G::U;
                float *o = SF + (b * R + r0 + qo) * 3 * (int64_t)G::UVs + uo * G::V + n;
#pragma unroll
                for (int t = 0; t < G::VT; ++t) {
                    if (t * 16 + n < G::V) {
                        o[t * 16] = acc[0][t][j];
                        o[G::UVs + t * 16] = acc[1][t][j];
                        o[2 * G::UVs + t * 16] = acc[2][t][j];
                    }
                }
            }
        }
    }
}

template <int LM>
__global__ __launch_bounds__(256) void k_analysis_mfma(Tabs<float> tb, int R, int rb,
                                                       const float *__restrict__ S,
                                                       float *__restrict__ Ta,
                                                       float *__restrict__ Tb)
{
    using G = Grid<LM>;
    extern __shared__ float smem[];
    float *qs = smem;                       // [VP][MW]: q_vm as [v][m], zero padded
    float *Ss = qs + G::VP * G::MW;         // [rb U][VS]
    float *Tm = Ss + (rb * G::U * G::VS + 3) / 4 * 4;  // [rb][M][Ut], 16-byte aligned
    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, n = lane & 15;
    for (int k = tid; k < G::VP * G::MW; k += 256) {
        const int v = k / G::MW, m = k - v * G::MW;
        qs[k] = (m < G::M && v < G::V) ? tb.q[v * G::M + m] : 0.f;
    }
    const int rows = nr * G::U;
    const int rtiles = (rows + 15) / 16;
    constexpr int pad = G::VP - G::V;
    if (pad > 0)
        for (int k = tid; k < rows * pad; k += 256) {
            const int ro = k / pad;
            Ss[ro * G::VS + G::V + (k - ro * pad)] = 0.f;
        }
    constexpr int tpad = G::Ut - G::U;
    if (tpad > 0)
        for (int k = tid; k < nr * G::M * tpad; k += 256) {
            const int ro = k / tpad;
            Tm[ro * G::Ut + G::U + (k - ro * tpad)] = 0.f;
        }
    constexpr int R4 = G::UVs / 4;  // 16-byte words per stored row
    for (int which = 0; which < 2; ++which) {
        // stage rows (q, u) of S as Ss[q U + u][v]
        for (int k = tid; k < nr * R4; k += 256) {
            const int q = k / R4, r = 4 * (k - q * R4);
            if (r < G::UV) {
                const float4_t x = *reinterpret_cast<const float4_t *>(
                    S + ((b * R + r0 + q) * 2 + which) * (int64_t)G::UVs + r);
                int u = r / G::V, v = r - u * G::V;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (r + e < G::UV) Ss[(q * G::U + u) * G::VS + v] = x[e];
                    if (++v == G::V) {
                        v = 0;
                        ++u;
                    }
                }
            }
        }
        __syncthreads();
        for (int rt = wave; rt < rtiles; rt += 4) {
            const int ra = rt * 16 + n;
            const bool ok = ra < rows;
            const float *sa = Ss + (ok ? ra : 0) * G::VS + g4;
            const float *qc = qs + g4 * G::MW + n;
            float4_t acc[G::MT];
#pragma unroll
            for (int t = 0; t < G::MT; ++t) acc[t] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
            for (int kk = 0; kk < G::KV; ++kk) {
                const float av = ok ? sa[4 * kk] : 0.f;
#pragma unroll
                for (int t = 0; t < G::MT; ++t)
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                        av, qc[4 * kk * G::MW + t * 16], acc[t], 0, 0, 0);
            }
#pragma unroll
            for (int t = 0; t < G::MT; ++t) {
                const int mi = t * 16 + n;
                if (mi < G::M) {
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int ro = rt * 16 + 4 * g4 + j;
                        if (ro < rows) {
                            const int qo = ro / G::U, uo = ro - qo * G::U;
                            Tm[(qo * G::M + mi) * G::Ut + uo] = acc[t][j];
                        }
                    }
                }
            }
        }
        __syncthreads();
        // Gauss-Legendre analysis: T[k] = sum_u w_u (2 pi / V) Pt_l^|m|(x_u) Tm[m][u]
        float *out = which ? Tb : Ta;
        for (int idx = tid; idx < nr * G::K; idx += 256) {
            const int qq = idx / G::K, k = idx - qq * G::K;
            int l = (int)sqrtf((float)k);
            while (l * l > k) --l;
            while ((l + 1) * (l + 1) <= k) ++l;
            const int m = k - l * l - l, am = m < 0 ? -m : m;
            const float4_t *w4 =
                reinterpret_cast<const float4_t *>(tb.wpt + (l * (l + 1) / 2 + am) * G::Ut);
            const float4_t *t4 =
                reinterpret_cast<const float4_t *>(Tm + (qq * G::M + m + LM) * G::Ut);
            float s = 0.f;
#pragma unroll
            for (int c = 0; c < G::Ut / 4; ++c) {
                const float4_t w = w4[c], t = t4[c];
                s += w[0] * t[0] + w[1] * t[1] + w[2] * t[2] + w[3] * t[3];
            }
            out[(b * R + r0 + qq) * (int64_t)G::K + k] = s;
        }
        __syncthreads();
    }
}

template <int LM>
hipError_t sender_lm(const Tabs<float> &tb, int64_t B, int R, const float *H, float *SF,
                     hipStream_t s)
{
    using G = Grid<LM>;
    const size_t fixed = (size_t)4 * G::KM * G::QW;
    const int rb = pick_rb(R, fixed, G::K);
    if (rb < 1) return hipErrorNotSupported;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_sender_mfma<LM>), dim3((unsigned)blocks), dim3(256),
                       sizeof(float) * (fixed + rb * (size_t)G::K), s, tb, R, rb, H, SF);
    return hipGetLastError();
}

template <int LM>
hipError_t analysis_lm(const Tabs<float> &tb, int64_t B, int R, const float *S, float *Ta,
                       float *Tb, hipStream_t s)
{
    using G = Grid<LM>;
    const size_t fixed = (size_t)G::VP * G::MW + 3;  // + alignment of the Tm region
    const size_t per_rank = (size_t)G::U * G::VS + (size_t)G::M * G::Ut;
    const int rb = pick_rb(R, fixed, per_rank);
    if (rb < 1) return hipErrorNotSupported;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_analysis_mfma<LM>), dim3((unsigned)blocks), dim3(256),
                       sizeof(float) * (fixed + rb * per_rank), s, tb, R, rb, S, Ta, Tb);
    return hipGetLastError();
}

bool default_grid(const Dims &d)
{
    const int u = (3 * d.lmax + 3) / 2;
    return d.U == (u < 1 ? 1 : u) && d.V == 3 * d.lmax + 1;
}

}  // namespace

#define CGTP_LMAX_CASES(X)                                                                   \
    X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15)     \
    X(16) X(17) X(18) X(19) X(20) X(21) X(22) X(23) X(24)

hipError_t launch_sender_mfma(const Tabs<float> &tb, int64_t B, int R, const float *H, float *SF,
                              hipStream_t s)
{
    if (B == 0) return hipSuccess;
    if (!default_grid(tb.d)) return hipErrorNotSupported;
    switch (tb.d.lmax) {
#define CGTP_CASE(LMV) \
    case LMV: return sender_lm<LMV>(tb, B, R, H, SF, s);
        CGTP_LMAX_CASES(CGTP_CASE)
#undef CGTP_CASE
    default: return hipErrorNotSupported;
    }
}

hipError_t launch_analysis_mfma(const Tabs<float> &tb, int64_t B, int R, const float *S, float *Ta,
                                float *Tb, hipStream_t s)
{
    if (B == 0) return hipSuccess;
    if (!default_grid(tb.d)) return hipErrorNotSupported;
    switch (tb.d.lmax) {
#define CGTP_CASE(LMV) \
    case LMV: return analysis_lm<LMV>(tb, B, R, S, Ta, Tb, s);
        CGTP_LMAX_CASES(CGTP_CASE)
#undef CGTP_CASE
    default: return hipErrorNotSupported;
    }
}

}  // namespace cgtp
