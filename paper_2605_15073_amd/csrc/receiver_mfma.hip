// Message-passing receiver pass with the edge-field synthesis on MFMA (fp32).
//
// For an edge e the zonal edge field and its t-derivative at grid point p are
//   a[r][p] = sum_l Rt[e][l][r] P_l(t_p),   g[r][p] = sum_l Rt[e][l][r] P_l'(t_p),
// t_p = rhat_e . Omega_p (addition theorem; the (2l+1)/(4 pi) weights are folded
// into Rt). Both are [16 points x L] x [L x 16 ranks] products, one
// v_mfma_f32_16x16x4f32 per 4 degrees. A workgroup owns one receiver, 16 ranks
// and 64 * TPW grid points (4 waves, TPW 16-point tiles per wave). Each wave is
// self-contained: per edge it runs the Legendre recurrence for its own 16 * TPW
// points into wave-private LDS (the B operand; lanes split P and P'), multiplies,
// and each lane combines its 4 points x 1 rank of a and g
// with the streamed sender fields (Eqs. msgpass-S and cat-beta-curl), all in
// registers. The summed grid fields go to S [N][R][2][UVs]; the folded analysis
// (k_analysis_rows when it does not fit)
// then runs the inverse transforms (Eqs. msgpass-Tmu, msgpass-Tlm).
// With VAL the surface curl takes the moved-derivative form (integration by parts on the
// sphere: the curl's coefficient is the analysis of S1 = sum_j B_j dA_j/dx against dY/dphi
// minus that of S2 = sum_j B_j dA_j/dphi against dY/dx): a lane reads only the value plane of
// its sender fields and accumulates the Gaunt sum a B and the pair (S1, S2); S is then
// [N][R][3][UVs] (six planes with two node slots) for the MFMA analysis in its moved modes.
#include "internal.h"

namespace cgtp {

namespace {

typedef float float4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ float4_t bload4(__amdgpu_buffer_rsrc_t rs, unsigned voff, unsigned soff)
{
    return __builtin_bit_cast(float4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, 0));
}

constexpr int kRT = 16;  // ranks per workgroup (MFMA columns)

// Wave-scope ordering of LDS writes before reads by other lanes of the same wave
// (LDS operations of a wave complete in order; the fences keep the compiler from
// moving accesses across).
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Wave-private LDS of k_receiver_mfma in floats: P_l rows (4 KS) and P_l' rows (4 KSG) of 64
// points, then dt/dx and dt/dphi at those points.
constexpr int recv_lds_floats(int lm)
{
    const int ks = (lm + 4) / 4, ksg = (lm + 1 - ((lm > 0 && lm % 4 == 0) ? 1 : 0) + 3) / 4;
    return 4 * (ks + ksg) * 64 + 2 * 64;
}

// Waves per SIMD the register allocation of k_receiver_mfma aims at (values-only form), at
// least: 4 with one set of sums at lmax 3 to 7 (where it needs no spill), else 3 (2 at lmax
// 24), and 2 with six sums (two node slots) or two coefficient sets from lmax 9 (which would
// spill at 3).
template <bool VAL, bool TWO, bool SPLIT>
constexpr int kRecvWaves(int lm)
{
    return !VAL ? 1
           : TWO ? 2
           : SPLIT ? (lm >= 9 ? 2 : 3)
                   : (lm >= 3 && lm <= 7 ? 4 : lm >= 24 ? 2 : 3);
}

// LM is lmax: the recurrence is unrolled with compile-time coefficients. A workgroup
// is WPB waves; each wave owns PW = 64 grid points, one per lane: per edge a lane runs
// the Legendre recurrence for P_l and P_l' at its own point (both in the same lane) into
// wave-private LDS, then the wave multiplies those [64 points x L] values with the
// [L x 16 ranks] edge coefficients on the matrix cores.
// TWO: the senders carry a second, parity-flipped node slot SFf (same layout as SF); by
// Table 1 its curl product then feeds S_alpha's slot (natural parity) and its Gaunt
// product S_beta's. Its six sums keep it at 2 waves per SIMD.
// SPLIT: the curl product's edge coefficients are Rtg (its own CP factors): the derivative
// sum g multiplies P' with those, the value sum a P with Rt.
// VAL: value planes only, moved-derivative curl (above). With SPLIT the senders carry the
// Gaunt factors' values in plane 0 and the curl factors' in plane 1.
template <int WPB, int LM, bool TWO, bool SPLIT, bool VAL>
__global__ __launch_bounds__(64 * WPB)
__attribute__((amdgpu_waves_per_eu(kRecvWaves<VAL, TWO, SPLIT>(LM)))) void k_receiver_mfma(Tabs<float> tb, int R, int nchunks,
                                                            int64_t N,
                                                            const int32_t *__restrict__ row_ptr,
                                                            const int32_t *__restrict__ col,
                                                            const int32_t *__restrict__ order,
                                                            const float *__restrict__ unit,
                                                            const float *__restrict__ Rt,
                                                            const float *__restrict__ Rtg,
                                                            const float *__restrict__ SF,
                                                            const float *__restrict__ SFf,
                                                            int sf_nc, float *__restrict__ S)
{
    constexpr int TPW = 4;           // 16-point tiles per wave
    constexpr int PW = 16 * TPW;     // grid points per wave: one per lane
    constexpr int PC = WPB * PW;     // grid points per workgroup
    constexpr int L = LM + 1;
    constexpr int KS = (L + 3) / 4;  // K steps of 4 degrees
    // P_0' = 0: when lmax is a multiple of 4 the derivative sum starts at degree DO = 1 and
    // takes one K step fewer (KSG) than the value sum; its LDS row j holds degree j + DO
    constexpr int DO = (LM > 0 && LM % 4 == 0) ? 1 : 0;
    constexpr int KSG = (L - DO + 3) / 4;
    // LDS rows of 64 points; point p of row j sits at column p ^ 16 (j & 3). A 64-lane LDS
    // read is served as two halves of 32 lanes over the 32 banks: the two rows a half reads at
    // once (lane groups g = 2 h, 2 h + 1 at j = 4 kk + g) then fall on different halves of the
    // banks, and the recurrence's writes of one row stay a permutation of them
    constexpr int RS = PW;
    const Dims &d = tb.d;
    const int UV = d.UV, UVs = d.UVs;
    // the wave index, uniform across the wave (so the buffer resources built from it are too)
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, n = lane & 15;
    // wave-private LDS: P_l and P_l' at the wave's points, then dt/dx and dt/dphi
    extern __shared__ float smem[];
    constexpr int wstride = recv_lds_floats(LM);
    float *Pl = smem + wave * wstride;  // [4 KS][RS]
    float *Dl = Pl + 4 * KS * RS;       // [4 KSG][RS]
    float *dxs = Dl + 4 * KSG * RS;     // [PW]
    float *dps = dxs + PW;              // [PW]
    auto slot = [](int j, int p) { return j * RS + (p ^ ((j & 3) << 4)); };

    // Block order (recv_block): the slices are (rank tile, point chunk) pairs.
    int64_t slice, i;
    if (!recv_block(N, order, slice, i)) return;
    const int rest = (int)slice;
    const int r0 = (rest / nchunks) * kRT;
    const int pw0 = (rest % nchunks) * PC + wave * PW;  // first point of this wave
    // a wave wholly past the grid (the padding of the last chunk, e.g. at lmax 7, 12, 14, 18)
    // has nothing to compute or store; waves synchronise only within themselves
    if (pw0 >= UV) return;

    // degrees beyond lmax stay zero in the A operand
    for (int k = lane; k < 4 * (KS + KSG) * RS; k += 64) Pl[k] = 0.f;
    // this lane's recurrence point (points past the grid compute on point 0, never stored)
    const int pr = pw0 + lane;
    const int prc = pr < UV ? pr : 0;
    const int ur = prc / d.V, vr = prc - ur * d.V;
    const float rx = tb.x[ur], rsx = tb.sx[ur], rxsx = tb.xsx[ur], rcp = tb.cphi[vr],
                rsp = tb.sphi[vr];

    // D[row = point 4 g + j][col = rank n]: a lane holds 4 consecutive points of one
    // rank, so its sender values are 16-byte loads and its S values 16-byte stores.
    // VAL: sa, sb the Gaunt sums into S_alpha, S_beta; (ca1, ca2) the moved curl pair into
    // S_alpha (the flipped slot's, TWO), (cb1, cb2) into S_beta (the natural slot's)
    float4_t sa[TPW], sb[TPW], ca1[TPW], ca2[TPW], cb1[TPW], cb2[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        sa[t] = float4_t{0.f, 0.f, 0.f, 0.f};
        sb[t] = float4_t{0.f, 0.f, 0.f, 0.f};
        ca1[t] = ca2[t] = cb1[t] = cb2[t] = float4_t{0.f, 0.f, 0.f, 0.f};
    }
    // lane's points: pw0 + 16 t + 4 g + (0..3); lane's rank: r0 + n. The sender fields are
    // either SF [N][R][3][UVs] (a sender's 16-rank block is [16][3][UVs]) or, with sf_nc
    // chunks, SF [R/16][sf_nc][N][16][3][64] (this wave's 64 points of a sender are one
    // contiguous [16][3][64] run).
    const int fstride = sf_nc ? kSfChunk : UVs;  // field stride, elements
    const unsigned voff = sf_nc ? (unsigned)((n * 3 * kSfChunk + 4 * g) * 4)
                                : (unsigned)((n * 3 * UVs + pw0 + 4 * g) * 4);
    const int64_t sfo = sf_nc ? ((int64_t)(r0 / kRT) * sf_nc + pw0 / kSfChunk) * N * (kRT * 3 * kSfChunk)
                              : (int64_t)r0 * 3 * UVs;
    const float *sfb = SF + sfo;
    const float *sfbf = (TWO ? SFf : SF) + sfo;
    const int64_t jstride = sf_nc ? (int64_t)kRT * 3 * kSfChunk : (int64_t)R * 3 * UVs;
    const unsigned sfbytes = (unsigned)(kRT * 3 * fstride * 4);
    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    // lanes whose 4 points all lie past the grid (the padding of the last chunk: up to 18% of
    // the points at lmax 7-8) load through an offset past the resource, which returns zeros
    // without a memory request (2^31: past the resource with or without the scalar offsets
    // below, which stay under 2 UVs x 4 + 192 bytes, and far from wrapping)
    unsigned vofft[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) vofft[t] = pw0 + 16 * t + 4 * g < UV ? voff : 0x80000000u;
    // Edge data in batches of 64 edges: lane k holds the sender index and the normalised
    // direction of edge eb + k, read out per edge with readlane, so no per-edge load of them
    // sits on the critical path.
    int colv = 0;
    float uxv = 0.f, uyv = 0.f, uzv = 1.f;
    auto load_batch = [&](int eb) {
        const int e = eb + lane;
        if (e < e1) {
            colv = col[e];
            const float x = unit[3 * (int64_t)e], y = unit[3 * (int64_t)e + 1],
                        z = unit[3 * (int64_t)e + 2];
            // renormalised by the hardware reciprocal square root (within 1 ulp)
            const float inv = __builtin_amdgcn_rsqf(x * x + y * y + z * z);
            uxv = x * inv;
            uyv = y * inv;
            uzv = z * inv;
        }
    };
    auto lane_f = [](float v, int k) {
        return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), k));
    };
    auto load_fields = [&](const float *base, int k, float4_t *fI, float4_t *fX, float4_t *fP) {
        const int64_t j = __builtin_amdgcn_readlane(colv, k);
        const __amdgpu_buffer_rsrc_t sfr = rsrc(base + j * jstride, sfbytes);
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            const unsigned so = (unsigned)(t * 16 * 4);
            fI[t] = bload4(sfr, vofft[t], so);
            if (!VAL || SPLIT) fX[t] = bload4(sfr, vofft[t], so + fstride * 4);
            if (!VAL) fP[t] = bload4(sfr, vofft[t], so + 2 * fstride * 4);
        }
    };
    // B operands: Rt[e][4 kk + g][r0 + n] for the value sum; for the derivative sum the rows
    // from degree DO on, of Rtg with SPLIT (else the same as the value sum's when DO = 0)
    auto load_b = [&](int e, float *bv, float *bg) {
        const float *rte = Rt + (int64_t)e * L * R + r0 + n;
        const float *rtg = SPLIT ? Rtg + (int64_t)e * L * R + r0 + n : rte;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            const int l = 4 * kk + g;
            bv[kk] = l <= LM ? rte[l * R] : 0.f;
        }
        if (SPLIT || DO) {
#pragma unroll
            for (int kk = 0; kk < KSG; ++kk) {
                const int l = 4 * kk + g + DO;
                bg[kk] = l <= LM ? rtg[l * R] : 0.f;
            }
        }
    };
    // A wave loads an edge's sender fields when the edge starts and hides their latency behind
    // the other waves of its SIMD: prefetching them an edge ahead would take the registers of
    // a wave (4 waves per SIMD in the values-only form at low degrees, 3 with the prefetch,
    // which measured slower). At low degrees (PRE_B) the next edge's B operand, a few
    // registers, is loaded one edge ahead.
    constexpr bool PRE_B = KS <= 2 && !TWO && !SPLIT;
    float nBv[KS], nBg[KS];
    if (e0 < e1) {
        load_batch(e0);
        if (PRE_B) load_b(e0, nBv, nBg);
    }
    for (int e = e0; e < e1; ++e) {
        const int k = (e - e0) & 63;
        float4_t fI[TPW], fX[TPW], fP[TPW], hI[TPW], hX[TPW], hP[TPW];
        float Bv[KS], Bg[KS];
        if (PRE_B) {
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) Bv[kk] = nBv[kk];
#pragma unroll
            for (int kk = 0; kk < KSG; ++kk) Bg[kk] = DO ? nBg[kk] : nBv[kk];
        } else {
            load_b(e, Bv, Bg);
            if (!SPLIT && !DO)
#pragma unroll
                for (int kk = 0; kk < KS; ++kk) Bg[kk] = Bv[kk];
        }
        const float ux = lane_f(uxv, k), uy = lane_f(uyv, k), uz = lane_f(uzv, k);
        load_fields(sfb, k, fI, fX, fP);
        if (TWO) load_fields(sfbf, k, hI, hX, hP);
        if (e + 1 < e1) {
            if (k == 63) load_batch(e + 1);
            if (PRE_B) load_b(e + 1, nBv, nBg);
        }
        wave_sync();  // this wave is done reading the previous edge's P, P'
        {
            // t = rhat . Omega at this lane's point; P_l(t) and P_l'(t) by the Legendre and
            // derivative recurrences
            const float h = ux * rcp + uy * rsp;
            const float t = uz * rx + rsx * h;
            float p0v = 1.f, p1v = t, d1 = 1.f;
            Pl[slot(0, lane)] = 1.f;
            if (!DO) Dl[slot(0, lane)] = 0.f;
            if (LM >= 1) {
                Pl[slot(1, lane)] = t;
                Dl[slot(1 - DO, lane)] = 1.f;
            }
#pragma unroll
            for (int l = 2; l <= LM; ++l) {
                const float c1 = (float)(2 * l - 1) / (float)l, c2 = (float)(l - 1) / (float)l;
                const float p2 = c1 * t * p1v - c2 * p0v;
                const float d2 = (float)l * p1v + t * d1;
                Pl[slot(l, lane)] = p2;
                Dl[slot(l - DO, lane)] = d2;
                p0v = p1v;
                p1v = p2;
                d1 = d2;
            }
            dxs[lane] = uz - rxsx * h;
            dps[lane] = rsx * (uy * rcp - ux * rsp);
        }
        wave_sync();
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            // A operands: P_{4 kk + g}(t_p) and P'_{4 kk + g + DO}(t_p) at point p = 16 t + n
            // (rows are points)
            float4_t a = float4_t{0.f, 0.f, 0.f, 0.f}, gg = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) {
                const float ap = Pl[slot(4 * kk + g, 16 * t + n)];
                a = __builtin_amdgcn_mfma_f32_16x16x4f32(ap, Bv[kk], a, 0, 0, 0);
                if (kk < KSG) {
                    const float ad = Dl[slot(4 * kk + g, 16 * t + n)];
                    gg = __builtin_amdgcn_mfma_f32_16x16x4f32(ad, Bg[kk], gg, 0, 0, 0);
                }
            }
            // this lane's 4 points' dt/dx and dt/dphi: one 16-byte LDS read each
            const float4_t dx4 = *reinterpret_cast<const float4_t *>(dxs + 16 * t + 4 * g);
            const float4_t dp4 = *reinterpret_cast<const float4_t *>(dps + 16 * t + 4 * g);
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const float dxt = dx4[jj], dpt = dp4[jj];
                if (VAL) {
                    // dA/dx = g dxt and dA/dphi = g dpt of the edge field
                    sa[t][jj] += a[jj] * fI[t][jj];
                    // SPLIT: the curl takes the curl factors' values (plane 1)
                    const float gf = gg[jj] * (SPLIT ? fX[t][jj] : fI[t][jj]);
                    cb1[t][jj] += dxt * gf;
                    cb2[t][jj] += dpt * gf;
                    if (TWO) {
                        sb[t][jj] += a[jj] * hI[t][jj];
                        const float gh = gg[jj] * hI[t][jj];
                        ca1[t][jj] += dxt * gh;
                        ca2[t][jj] += dpt * gh;
                    }
                } else {
                    sa[t][jj] += a[jj] * fI[t][jj];
                    sb[t][jj] += gg[jj] * (dpt * fX[t][jj] - dxt * fP[t][jj]);
                    if (TWO) {
                        sa[t][jj] += gg[jj] * (dpt * hX[t][jj] - dxt * hP[t][jj]);
                        sb[t][jj] += a[jj] * hI[t][jj];
                    }
                }
            }
        }
    }
    // S[i][r0 + n][plane][p .. p + 3]: planes (S_alpha, S_beta), or with VAL the Gaunt sum and
    // moved pair (sa, cb1, cb2), with two slots (sa, ca1, ca2, sb, cb1, cb2)
    constexpr int NF = VAL ? (TWO ? 6 : 3) : 2;
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        const int p = pw0 + 16 * t + 4 * g;
        float *o = S + ((i * R + r0 + n) * NF) * (int64_t)UVs + p;
        float4_t pl[NF];
        if (!VAL) {
            pl[0] = sa[t];
            pl[1] = sb[t];
        } else if (!TWO) {
            pl[0] = sa[t];
            pl[1] = cb1[t];
            pl[2] = cb2[t];
        } else {
            pl[0] = sa[t];
            pl[1] = ca1[t];
            pl[2] = ca2[t];
            pl[3] = sb[t];
            pl[4] = cb1[t];
            pl[5] = cb2[t];
        }
        if (p + 3 < UV) {
#pragma unroll
            for (int f = 0; f < NF; ++f) *reinterpret_cast<float4_t *>(o + f * UVs) = pl[f];
        } else {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
                if (p + jj < UV) {
#pragma unroll
                    for (int f = 0; f < NF; ++f) o[f * UVs + jj] = pl[f][jj];
                }
        }
    }
}

// Read-pattern ceiling of k_receiver_mfma in its values-only form on the plain sender layout
// [N][R][3][UVs]: the same blocks in the same order, the same wave-uniform sender index per
// edge and the same 16-byte loads of the value plane (one per 16-point tile and lane), with
// nothing computed from them but a running sum; sink receives a value only if that sum equals
// a constant no finite input sums to by chance, which keeps every load live.
template <int WPB>
__global__ __launch_bounds__(64 * WPB) void k_gather_probe_mfma(int UV, int UVs, int R,
                                                                int nchunks, int64_t N,
                                                                const int32_t *__restrict__ row_ptr,
                                                                const int32_t *__restrict__ col,
                                                                const int32_t *__restrict__ order,
                                                                const float *__restrict__ SF,
                                                                float *__restrict__ sink)
{
    constexpr int TPW = 4, PW = 16 * TPW, PC = WPB * PW;
    // the wave index, uniform across the wave (so the buffer resources built from it are too)
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, n = lane & 15;
    int64_t slice, i;
    if (!recv_block(N, order, slice, i)) return;
    const int rest = (int)slice;
    const int r0 = (rest / nchunks) * kRT;
    const int pw0 = (rest % nchunks) * PC + wave * PW;
    if (pw0 >= UV) return;
    const unsigned voff = (unsigned)((n * 3 * UVs + pw0 + 4 * g) * 4);
    unsigned vofft[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) vofft[t] = pw0 + 16 * t + 4 * g < UV ? voff : 0x80000000u;
    const float *sfb = SF + (int64_t)r0 * 3 * UVs;
    const int64_t jstride = (int64_t)R * 3 * UVs;
    const unsigned sfbytes = (unsigned)(kRT * 3 * UVs * 4);
    float4_t acc = float4_t{0.f, 0.f, 0.f, 0.f};
    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    for (int e = e0; e < e1; ++e) {
        const int64_t j = __builtin_amdgcn_readfirstlane(col[e]);
        const __amdgpu_buffer_rsrc_t sfr = rsrc(sfb + j * jstride, sfbytes);
#pragma unroll
        for (int t = 0; t < TPW; ++t) acc += bload4(sfr, vofft[t], (unsigned)(t * 16 * 4));
    }
    const float sum = acc[0] + acc[1] + acc[2] + acc[3];
    if (sum == -1.2345678e30f) sink[0] = sum;
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

hipError_t launch_gather_probe_mfma(const Dims &d, int64_t N, int R, const int32_t *row_ptr,
                                    const int32_t *col, const int32_t *order, const float *SF,
                                    float *sink, hipStream_t s)
{
    if (!receiver_mfma_supported(d, R)) return hipErrorNotSupported;
    constexpr int WPB = 2, PC = WPB * 64;  // as launch_receiver_mfma
    const int nchunks = (d.UV + PC - 1) / PC;
    if (N == 0) return hipSuccess;
    const int64_t blocks = recv_blocks(N, (int64_t)(R / kRT) * nchunks);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_gather_probe_mfma<WPB>), dim3((unsigned)blocks), dim3(64 * WPB), 0, s,
                       d.UV, d.UVs, R, nchunks, N, row_ptr, col, order, SF, sink);
    return hipGetLastError();
}

size_t receiver_mfma_ws_elems(const Dims &d, int64_t N, int R, int planes)
{
    return (size_t)N * R * planes * d.UVs;
}

hipError_t launch_receiver_mfma(const Tabs<float> &tb, int64_t N, int R, const int32_t *row_ptr,
                                const int32_t *col, const int32_t *order, const float *unit,
                                const float *Rt, const float *Rtg, const float *SF,
                                const float *SFf, bool sf_chunked, float *S, float *Ta, float *Tb,
                                hipStream_t s, bool values_only, bool analyse)
{
    if (N == 0) return hipSuccess;
    const Dims &d = tb.d;
    if (!receiver_mfma_supported(d, R)) return hipErrorNotSupported;
    if (SFf && Rtg) return hipErrorNotSupported;
    if (values_only && SFf && Rtg) return hipErrorInvalidValue;
    // Waves per workgroup: two (128 grid points); one with two node slots up to lmax 8, whose
    // six sums leave two waves per SIMD (there more, smaller workgroups measured 2.8% faster
    // at lmax 6, but 4% slower at lmax 20 and 2.6% slower with one slot).
    constexpr int PW = 64;
    const int wpb = SFf && d.lmax <= 8 ? 1 : 2, PC = wpb * PW;
    const int nchunks = (d.UV + PC - 1) / PC;
    const size_t sh = sizeof(float) * wpb * (size_t)recv_lds_floats(d.lmax);
    const int64_t blocks = recv_blocks(N, (int64_t)(R / kRT) * nchunks);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    static_assert(PW == kSfChunk, "a receiver wave reads one chunk of the chunked layout");
    const int sf_nc = sf_chunked ? sf_chunks(d) : 0;
#define CGTP_LAUNCH(LMV, TW, SP, VL)                                                            \
    hipLaunchKernelGGL((k_receiver_mfma<TW && LMV <= 8 ? 1 : 2, LMV, TW, SP, VL>),            \
                       dim3((unsigned)blocks),                                                  \
                       dim3(64 * wpb), sh, s, tb, R, nchunks, N, row_ptr, col, order, unit, Rt, \
                       Rtg, SF, SFf, sf_nc, S)
    switch (d.lmax) {
#define CGTP_CASE(LMV)                                                 \
    case LMV:                                                          \
        if (values_only) {                                             \
            if (SFf) CGTP_LAUNCH(LMV, true, false, true);              \
            else if (Rtg) CGTP_LAUNCH(LMV, false, true, true);         \
            else CGTP_LAUNCH(LMV, false, false, true);                 \
        } else if (LMV < kMfmaRecvMinL) {                              \
            return hipErrorNotSupported;                               \
        } else if (SFf) {                                              \
            CGTP_LAUNCH(LMV, true, false, false);                      \
        } else if (Rtg) {                                              \
            CGTP_LAUNCH(LMV, false, true, false);                      \
        } else {                                                       \
            CGTP_LAUNCH(LMV, false, false, false);                     \
        }                                                              \
        break;
        CGTP_CASE(0) CGTP_CASE(1) CGTP_CASE(2) CGTP_CASE(3) CGTP_CASE(4) CGTP_CASE(5) CGTP_CASE(6)
        CGTP_CASE(7) CGTP_CASE(8) CGTP_CASE(9) CGTP_CASE(10) CGTP_CASE(11) CGTP_CASE(12) CGTP_CASE(13) CGTP_CASE(14)
        CGTP_CASE(15) CGTP_CASE(16) CGTP_CASE(17) CGTP_CASE(18) CGTP_CASE(19) CGTP_CASE(20)
        CGTP_CASE(21) CGTP_CASE(22) CGTP_CASE(23) CGTP_CASE(24)
#undef CGTP_CASE
#undef CGTP_LAUNCH
    default: return hipErrorNotSupported;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !analyse) return e;
    return launch_summed_analysis(tb, N, R, S, Ta, Tb, s, values_only ? (SFf ? 2 : 1) : 0);
}

hipError_t launch_summed_analysis(const Tabs<float> &tb, int64_t N, int R, const float *S,
                                  float *Ta, float *Tb, hipStream_t s, int mode)
{
    if (N == 0) return hipSuccess;
    const Dims &d = tb.d;
    if (mode != 0) return launch_analysis_mfma(tb, N, R, S, Ta, Tb, s, mode);
    hipError_t e = launch_analysis_mfma(tb, N, R, S, Ta, Tb, s);
    if (e != hipErrorNotSupported) return e;
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
