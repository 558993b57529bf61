// Message-passing receiver pass with the edge-field synthesis on MFMA (fp32).
//
// For an edge e the zonal edge field and its t-derivative at grid point p are
//   a[r][p] = sum_l Rt[e][l][r] P_l(t_p),   g[r][p] = sum_l Rt[e][l][r] P_l'(t_p),
// t_p = rhat_e . Omega_p (addition theorem; the (2l+1)/(4 pi) weights are folded
// into Rt). Both are [16 ranks x L] x [L x 16 points] products, one
// v_mfma_f32_16x16x4f32 per 4 degrees. A workgroup owns one receiver, 16 ranks
// and 64 * TPW grid points (4 waves, TPW 16-point tiles per wave). Per edge the
// first 64 * TPW threads run the Legendre recurrence, one point each, into LDS (the
// B operand),
// the wave multiplies, and each lane combines its 4 ranks x 1 point of a and g
// with the streamed sender fields (Eqs. msgpass-S and cat-beta-curl), all in
// registers. The summed grid fields go to S [N][R][2][UVs]; the folded analysis
// (k_analysis_rows when it does not fit)
// then runs the inverse transforms (Eqs. msgpass-Tmu, msgpass-Tlm).
#include "internal.h"

namespace cgtp {

namespace {

typedef float float4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ float bload(__amdgpu_buffer_rsrc_t rs, unsigned voff, unsigned soff)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, 0));
}

constexpr int kRT = 16;  // ranks per workgroup (MFMA rows)

template <int TPW>
__global__ __launch_bounds__(256) void k_receiver_mfma(Tabs<float> tb, int R, int nchunks,
                                                       const int32_t *__restrict__ row_ptr,
                                                       const int32_t *__restrict__ col,
                                                       const float *__restrict__ unit,
                                                       const float *__restrict__ Rt,
                                                       const float *__restrict__ SF,
                                                       float *__restrict__ S)
{
    constexpr int PC = 64 * TPW;  // grid points per workgroup
    const Dims &d = tb.d;
    const int UV = d.UV, UVs = d.UVs, L = d.L, lmax = d.lmax;
    const int KS = (L + 3) / 4;  // K steps of 4 degrees
    extern __shared__ float smem[];
    float *Pl = smem;                 // [4 KS][PC]  P_l(t_p)
    float *Dl = Pl + 4 * KS * PC;     // [4 KS][PC]  P_l'(t_p)
    float *dxs = Dl + 4 * KS * PC;    // [PC] dt/dx
    float *dps = dxs + PC;            // [PC] dt/dphi

    // XCD-aware order: the blocks of one receiver share an XCD (block b runs on XCD b % 8)
    const int64_t nblk = gridDim.x, per = nblk / 8, rem = nblk % 8;
    const int64_t xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int64_t lb = (xcd < rem) ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
    const int nrt = R / kRT;
    const int64_t i = lb / ((int64_t)nrt * nchunks);
    const int rest = (int)(lb - i * (int64_t)nrt * nchunks);
    const int r0 = (rest / nchunks) * kRT;
    const int p0 = (rest % nchunks) * PC;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, n = lane & 15;
    // degrees beyond lmax stay zero in the B operand
    for (int k = tid; k < 4 * KS * PC; k += 256) {
        Pl[k] = 0.f;
        Dl[k] = 0.f;
    }
    // this thread's recurrence point (threads tid < PC)
    const int pr = p0 + tid;
    const int prc = pr < UV ? pr : 0;
    const int ur = prc / d.V, vr = prc - ur * d.V;
    const float rx = tb.x[ur], rsx = tb.sx[ur], rxsx = tb.xsx[ur], rcp = tb.cphi[vr],
                rsp = tb.sphi[vr];

    float4_t sa[TPW], sb[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        sa[t] = float4_t{0.f, 0.f, 0.f, 0.f};
        sb[t] = float4_t{0.f, 0.f, 0.f, 0.f};
    }
    // lane's points: p0 + (wave * TPW + t) * 16 + n; lane's ranks: r0 + 4 g + jj
    const int pl0 = (wave * TPW) * 16 + n;  // local index of tile 0
    const unsigned voff = (unsigned)((12 * g * UVs + p0 + pl0) * 4);
    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    for (int e = e0; e < e1; ++e) {
        const int64_t j = __builtin_amdgcn_readfirstlane(col[e]);
        // sender rank block [16][3][UVs], read with one VGPR offset per lane
        const __amdgpu_buffer_rsrc_t sfr =
            rsrc(SF + (j * R + r0) * 3 * (int64_t)UVs, (unsigned)(kRT * 3 * UVs * 4));
        float fI[TPW][4], fX[TPW][4], fP[TPW][4];
#pragma unroll
        for (int t = 0; t < TPW; ++t)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const unsigned so = (unsigned)(((jj * 3) * UVs + t * 16) * 4);
                fI[t][jj] = bload(sfr, voff, so);
                fX[t][jj] = bload(sfr, voff, so + UVs * 4);
                fP[t][jj] = bload(sfr, voff, so + 2 * UVs * 4);
            }
        float ux = unit[3 * (int64_t)e], uy = unit[3 * (int64_t)e + 1], uz = unit[3 * (int64_t)e + 2];
        const float inv = 1.f / sqrtf(ux * ux + uy * uy + uz * uz);
        ux *= inv;
        uy *= inv;
        uz *= inv;
        // A operand: Rt[e][4 kk + g][r0 + n]
        const float *rte = Rt + (int64_t)e * L * R + r0 + n;
        float A[8];
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) {
            const int l = 4 * kk + g;
            A[kk] = (kk < KS && l <= lmax) ? rte[l * R] : 0.f;
        }
        __syncthreads();  // previous edge done with Pl / Dl
        if (tid < PC) {
            const float h = ux * rcp + uy * rsp;
            const float t = uz * rx + rsx * h;
            float p0v = 1.f, p1v = t, d1 = 1.f;
            Pl[tid] = 1.f;
            Dl[tid] = 0.f;
            if (lmax >= 1) {
                Pl[PC + tid] = t;
                Dl[PC + tid] = 1.f;
            }
            for (int l = 2; l <= lmax; ++l) {
                const float p2 = tb.rc1[l] * t * p1v - tb.rc2[l] * p0v;
                const float d2 = (float)l * p1v + t * d1;
                Pl[l * PC + tid] = p2;
                Dl[l * PC + tid] = d2;
                p0v = p1v;
                p1v = p2;
                d1 = d2;
            }
            dxs[tid] = uz - rxsx * h;
            dps[tid] = rsx * (uy * rcp - ux * rsp);
        }
        __syncthreads();
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            const int pl = pl0 + 16 * t;
            float4_t a = float4_t{0.f, 0.f, 0.f, 0.f}, gg = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < 8; ++kk) {
                if (kk < KS) {
                    const float bp = Pl[(4 * kk + g) * PC + pl];
                    const float bd = Dl[(4 * kk + g) * PC + pl];
                    a = __builtin_amdgcn_mfma_f32_16x16x4f32(A[kk], bp, a, 0, 0, 0);
                    gg = __builtin_amdgcn_mfma_f32_16x16x4f32(A[kk], bd, gg, 0, 0, 0);
                }
            }
            const float dxt = dxs[pl], dpt = dps[pl];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                sa[t][jj] += a[jj] * fI[t][jj];
                sb[t][jj] += gg[jj] * (dpt * fX[t][jj] - dxt * fP[t][jj]);
            }
        }
    }
    // S[i][r0 + 4 g + jj][0 / 1][p]
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        const int p = p0 + pl0 + 16 * t;
        if (p >= UV) continue;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            float *o = S + ((i * R + r0 + 4 * g + jj) * 2) * (int64_t)UVs + p;
            o[0] = sa[t][jj];
            o[UVs] = sb[t][jj];
        }
    }
}

// Inverse transforms of stored grid fields S [B][R][2][UVs] -> Ta, Tb [B][R][K]:
// one workgroup per (node, block of ranks), one rank at a time through LDS.
__global__ __launch_bounds__(256) void k_analysis_rows(Tabs<float> tb, int R, int rb,
                                                       const float *__restrict__ S,
                                                       float *__restrict__ Ta,
                                                       float *__restrict__ Tb)
{
    const Dims &d = tb.d;
    extern __shared__ float smem[];
    float *qs = smem;                  // [V][M]
    float *Sa = qs + d.V * d.M;        // [UV]
    float *Sb = Sa + d.UV;             // [UV]
    float *Tm = Sb + d.UV;             // [2][M][U]
    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    for (int k = threadIdx.x; k < d.V * d.M; k += blockDim.x) qs[k] = tb.q[k];
    for (int q = 0; q < nr; ++q) {
        const float *src = S + ((b * R + r0 + q) * 2) * (int64_t)d.UVs;
        for (int k = threadIdx.x; k < d.UV; k += blockDim.x) {
            Sa[k] = src[k];
            Sb[k] = src[d.UVs + k];
        }
        __syncthreads();
        const int MU = d.M * d.U;
        for (int idx = threadIdx.x; idx < 2 * MU; idx += blockDim.x) {
            const int which = idx >= MU;
            const int r = idx - which * MU;
            const int mi = r / d.U, u = r - mi * d.U;
            const float *row = (which ? Sb : Sa) + u * d.V;
            float s = 0.f;
            for (int v = 0; v < d.V; ++v) s += qs[v * d.M + mi] * row[v];
            Tm[idx] = s;
        }
        __syncthreads();
        const int64_t br = b * R + r0 + q;
        for (int idx = threadIdx.x; idx < 2 * d.K; idx += blockDim.x) {
            const int which = idx >= d.K;
            const int k = idx - which * d.K;
            int l = (int)sqrtf((float)k);
            while (l * l > k) --l;
            while ((l + 1) * (l + 1) <= k) ++l;
            const int m = k - l * l - l, am = m < 0 ? -m : m;
            const float *tm = Tm + which * MU + (m + d.lmax) * d.U;
            const int pi = l * (l + 1) / 2 + am;
            float s = 0.f;
            for (int u = 0; u < d.U; ++u) s += tb.wq[u] * tb.p[(size_t)u * d.P + pi] * tm[u];
            (which ? Tb : Ta)[br * d.K + k] = s;
        }
        __syncthreads();
    }
}

}  // namespace

bool receiver_mfma_supported(const Dims &d, int R)
{
    return R % kRT == 0 && d.L <= 32;
}

size_t receiver_mfma_ws_elems(const Dims &d, int64_t N, int R)
{
    return (size_t)N * R * 2 * d.UVs;
}

hipError_t launch_receiver_mfma(const Tabs<float> &tb, int64_t N, int R, const int32_t *row_ptr,
                                const int32_t *col, const float *unit, const float *Rt,
                                const float *SF, float *S, float *Ta, float *Tb, hipStream_t s)
{
    if (N == 0) return hipSuccess;
    const Dims &d = tb.d;
    if (!receiver_mfma_supported(d, R)) return hipErrorNotSupported;
    constexpr int TPW = 2, PC = 64 * TPW;
    const int KS = (d.L + 3) / 4;
    const int nchunks = (d.UV + PC - 1) / PC;
    const int64_t blocks = N * (R / kRT) * nchunks;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    const size_t sh = sizeof(float) * (2 * 4 * KS * PC + 2 * PC);
    hipLaunchKernelGGL(k_receiver_mfma<TPW>, dim3((unsigned)blocks), dim3(256), sh, s, tb, R,
                       nchunks, row_ptr, col, unit, Rt, SF, S);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_analysis_folded(tb, N, R, S, Ta, Tb, s);
    if (e != hipErrorNotSupported) return e;
    int rb = 8;
    if (rb > R) rb = R;
    const size_t sh2 = sizeof(float) * (d.V * d.M + 2 * d.UV + 2 * d.M * d.U);
    const int64_t blocks2 = N * ((R + rb - 1) / rb);
    hipLaunchKernelGGL(k_analysis_rows, dim3((unsigned)blocks2), dim3(256), sh2, s, tb, R, rb, S,
                       Ta, Tb);
    return hipGetLastError();
}

}  // namespace cgtp
