// Register-resident, azimuth-folded inverse transforms (fp32): one thread per
// (rank, GL node u) analyses the summed grid fields S [N][R][2][UVs] into Ta, Tb
// [N][R][K] (Eqs. msgpass-Tmu, msgpass-Tlm). The azimuth is swept in pairs
// (v, V - v): cos(m phi) is equal at the two points and sin(m phi) changes sign, so
// each coefficient accumulates c (x(v) + x(V-v)) for cosine slots and
// s (x(v) - x(V-v)) for sine slots. The Fourier table stays in LDS and is read as a
// broadcast (all lanes of a wave share v).
#include "internal.h"

namespace cgtp {

namespace {

template <int LM>
__global__ __launch_bounds__(256) void k_analysis_folded(Tabs<float> tb, int R, int rb,
                                                         const float *__restrict__ S,
                                                         float *__restrict__ Ta,
                                                         float *__restrict__ Tb)
{
    constexpr int M = 2 * LM + 1, L = LM + 1, K = L * L, P = L * (L + 1) / 2;
    extern __shared__ float smem[];
    const int U = tb.d.U, V = tb.d.V, UVs = tb.d.UVs;
    float *qs = smem;              // [V][M]
    float *ps = qs + V * M;        // [U][P]
    float *Tm = ps + U * P;        // [rb][M][U]
    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    for (int k = threadIdx.x; k < V * M; k += blockDim.x) qs[k] = tb.q[k];
    for (int k = threadIdx.x; k < U * P; k += blockDim.x) ps[k] = tb.p[k];
    __syncthreads();
    const int q = threadIdx.x / U, u = threadIdx.x - q * U;
    for (int which = 0; which < 2; ++which) {
        if (q < nr) {
            const float *row = S + ((b * R + r0 + q) * 2 + which) * (int64_t)UVs + u * V;
            float T[M];
#pragma unroll
            for (int mi = 0; mi < M; ++mi) T[mi] = 0.f;
            for (int v = 0; 2 * v <= V; ++v) {
                const int pv = v == 0 ? 0 : V - v;
                const bool paired = v != 0 && pv != v;
                const float x0 = row[v], x1 = paired ? row[pv] : 0.f;
                const float xp = x0 + x1, xm = x0 - x1;
                const float *qr = qs + v * M;
                T[LM] += xp;
#pragma unroll
                for (int k = 1; k <= LM; ++k) {
                    T[LM + k] += qr[LM + k] * xp;
                    T[LM - k] += qr[LM - k] * xm;
                }
            }
            float *tm = Tm + q * M * U;
#pragma unroll
            for (int mi = 0; mi < M; ++mi) tm[mi * U + u] = T[mi];
        }
        __syncthreads();
        float *out = which ? Tb : Ta;
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
            out[(b * R + r0 + qq) * (int64_t)K + k] = s;
        }
        __syncthreads();
    }
}

template <int LM>
int pick_rb(int U, int R, size_t fixed, size_t per_rank, int lds_max)
{
    int rb = 256 / U;
    if (rb > 16) rb = 16;
    if (rb > R) rb = R;
    while (rb > 1 && sizeof(float) * (fixed + rb * per_rank) > (size_t)lds_max) --rb;
    return rb;
}

template <int LM>
hipError_t launch_analysis_lm(const Tabs<float> &tb, int64_t B, int R, const float *S, float *Ta,
                              float *Tb, hipStream_t s)
{
    constexpr int M = 2 * LM + 1, L = LM + 1, P = L * (L + 1) / 2;
    const int U = tb.d.U, V = tb.d.V;
    const size_t fixed = (size_t)V * M + (size_t)U * P;
    const int rb = pick_rb<LM>(U, R, fixed, (size_t)M * U, tb.d.lds_max);
    if (sizeof(float) * (fixed + rb * (size_t)M * U) > (size_t)tb.d.lds_max)
        return hipErrorNotSupported;
    const int threads = (rb * U + 63) / 64 * 64;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    hipLaunchKernelGGL((k_analysis_folded<LM>), dim3((unsigned)blocks), dim3(threads),
                       sizeof(float) * (fixed + rb * (size_t)M * U), s, tb, R, rb, S, Ta, Tb);
    return hipGetLastError();
}

}  // namespace

#define CGTP_LMAX_CASES(X)                                                                   \
    X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15)     \
    X(16) X(17) X(18) X(19) X(20) X(21) X(22) X(23) X(24)

hipError_t launch_analysis_folded(const Tabs<float> &tb, int64_t B, int R, const float *S,
                                  float *Ta, float *Tb, hipStream_t s)
{
    if (B == 0) return hipSuccess;
    switch (tb.d.lmax) {
#define CGTP_CASE(LMV) \
    case LMV: return launch_analysis_lm<LMV>(tb, B, R, S, Ta, Tb, s);
        CGTP_LMAX_CASES(CGTP_CASE)
#undef CGTP_CASE
    default: return hipErrorNotSupported;
    }
}

}  // namespace cgtp
