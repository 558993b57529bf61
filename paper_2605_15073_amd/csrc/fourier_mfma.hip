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
//   fields S [N][R][2][UVs]: rows of S are staged in LDS one field at a time (so that a
//   workgroup's LDS holds more ranks), then
//     Tm[(q,u)][m] = sum_v S[q][u V + v] q_vm
//   runs on MFMA and the Gauss-Legendre sum over u reads the weighted transposed
//   Legendre table with 16-byte loads.
//
// k_onsite_mfma: the whole on-site grid stage for a node and rb ranks (Eqs. struct-F,
//   struct-tildeA, struct-S, poisson-S2-x, struct-Tmu, struct-Tlm). The synthesis runs
//   with the operands swapped, D[v][(q,u)] = sum_m q_vm F[(q,u)][m], so a lane ends up
//   holding, for its row (q,u), the field values at v = 16 t + 4 g + j. Those are exactly
//   the A operands the analysis product Tm[(q,u)][m] = sum_v S[(q,u)][v] q_vm needs when
//   its reduction over v is visited in the order (t, j): the pointwise product and the
//   surface curl are formed in registers and never leave the wave. Only Tm goes through
//   LDS, for the Gauss-Legendre sum.
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
    static constexpr int Ut = (U + 3) / 4 * 4;           // row length of pt, wpt
    static constexpr int KM = (M + 3) / 4;               // synthesis reduction steps over m
    static constexpr int VT = (V + 15) / 16;             // synthesis tiles over v
    static constexpr int KV = (V + 3) / 4, VP = 4 * KV;  // analysis reduction steps over v
    static constexpr int MT = (M + 15) / 16, MW = MT * 16;  // analysis tiles over m
    // coefficient rows with margins: orders of the padded reduction run over
    // m = -lmax .. lmax + 3, so l^2 + l +- m stays in [-(lmax + 3), K + 2]
    static constexpr int HL = LM + 3, HR = HL + K + 3;
    // LDS row strides of the staged Fourier tables. A 64-lane LDS read is served in two
    // halves of 32 lanes (n = 0..15, two lane groups g); each stride puts the two groups
    // of a half on disjoint banks.
    static constexpr int QB = (VT * 16 + 31) / 32 * 32 + 16;  // [m][v], read at g QB + n
    static constexpr int QS = (MW + 31) / 32 * 32 + 2;        // [v][m], read at n QS + g
                                                              // (and at 4 g QS + n: 2-way)
    static constexpr int VS = (VP + 31) / 32 * 32 + 2;        // staged S rows, read at n VS + g
    // Tm rows [m][TS]: written at 16 mt + n (stride TS: 2-way), read as 16-byte words by
    // consecutive m (stride TS / 4 words, odd: conflict-free)
    static constexpr int TS = Ut + (Ut % 8 == 0 ? 4 : 0);
};

// LDS per workgroup that keeps four workgroups resident on a compute unit
inline size_t lds_target(const Dims &d) { return (size_t)d.lds_cu / 4; }
constexpr int64_t kDenseSynthBlocks = 512;  // dense-synthesis workgroups if occupancy is unknown

// Largest rank block (<= 16) within the LDS target, else the largest within a workgroup's
// LDS.
int pick_rb(const Dims &d, int R, size_t fixed, size_t per_rank)
{
    int rb = R < 16 ? R : 16;
    while (rb > 1 && sizeof(float) * (fixed + rb * per_rank) > lds_target(d)) --rb;
    while (rb > 0 && sizeof(float) * (fixed + rb * per_rank) > (size_t)d.lds_max) --rb;
    return rb;
}

// Workgroup size: one wave per 16-row tile, at most four.
int waves_for(int rows)
{
    const int t = (rows + 15) / 16;
    return t < 4 ? t : 4;
}

// Stages q_vm (zero padded) as table[i][j] with row stride ld, where (v, m) = (i, j) when
// v_major, else (j, i).
template <int LM>
__device__ __forceinline__ void stage_q(const Tabs<float> &tb, float *table, int rows, int ld,
                                        bool v_major)
{
    using G = Grid<LM>;
    for (int k = threadIdx.x; k < rows * ld; k += blockDim.x) {
        const int i = k / ld, j = k - i * ld;
        const int v = v_major ? i : j, m = v_major ? j : i;
        table[k] = (m < G::M && v < G::V) ? tb.q[v * G::M + m] : 0.f;
    }
}

// Legendre recurrence coefficients per (l, m >= 0) pair, staged in LDS as
// {a_lm, b_lm, c_lm, 0}: Pt_l = a (x Pt_{l-1} - b Pt_{l-2}) and
// (1 - x^2) dPt_l/dx = c Pt_{l-1} - l x Pt_l.
template <int LM>
__device__ __forceinline__ void stage_coefs(const Tabs<float> &tb, float4_t *cf)
{
    constexpr int P = (LM + 1) * (LM + 2) / 2;
    for (int k = threadIdx.x; k < P; k += blockDim.x)
        cf[k] = float4_t{tb.ya[k], tb.yb[k], tb.yc[k], 0.f};
}

// Copies nr coefficient rows src[q][K] into margin-padded rows dst[q][HR] (margins zero).
template <int LM>
__device__ __forceinline__ void stage_rows(const float *src, float *dst, int nr)
{
    using G = Grid<LM>;
    for (int k = threadIdx.x; k < nr * G::HR; k += blockDim.x) {
        const int q = k / G::HR, i = k - q * G::HR - G::HL;
        dst[k] = (i >= 0 && i < G::K) ? src[q * G::K + i] : 0.f;
    }
}

// Legendre pass of one lane at reduction step KK (order m = 4 KK + g - lmax), for NOP
// operands whose margin-padded coefficient rows start at h[o] (index 0 = (l, m) = (0, 0)):
// fa = sum_l Pt_l^|m|(x) h[l, m], fx = the same with dPt/dx, fn = sum_l Pt_l^|m|(x) h[l, -m]
// (Eq. msgpass-FI and its x-derivative). The functions come from the three-term recurrence
// in l, started by adding seed = Pt_|m|^|m|(x) at l = |m| (seed 0 for the padding orders
// |m| > lmax). Below l = |m| a lane carries zeros. The loop is unrolled from the lowest
// |m| of the step, so every table offset is a constant. VO: the values fa alone (fx, fn
// untouched).
// Degrees a lane visits at reduction step kk (orders 4 kk - lmax .. 4 kk - lmax + 3):
// l = a0(kk) .. lmax, the lowest |m| of the step upwards; base(kk) counts the (step, degree)
// pairs of the steps before kk.
template <int LM>
struct LegendreSteps {
    static constexpr int a0(int kk)
    {
        const int lo = 4 * kk - LM, hi = lo + 3;
        return (lo <= 0 && hi >= 0) ? 0 : (lo > 0 ? lo : -hi);
    }
    static constexpr int base(int kk)
    {
        int b = 0;
        for (int k = 0; k < kk; ++k) b += LM - a0(k) + 1;
        return b;
    }
    static constexpr int N = base(Grid<LM>::KM);
};

template <int LM, int KK, int NOP, bool VO = false>
__device__ __forceinline__ void legendre_step(const float4_t *cf, const float *const *h, float seed,
                                              float x, float r, int m, float *fa, float *fx,
                                              float *fn)
{
    constexpr int A0 = LegendreSteps<LM>::a0(KK);
    const int am = m < 0 ? (-m < LM ? -m : LM) : (m < LM ? m : LM);
    const float4_t *ca = cf + am;
    float p1 = 0.f, p2 = 0.f;
#pragma unroll
    for (int l = A0; l <= LM; ++l) {
        const float4_t c = ca[l * (l + 1) / 2];
        const float inj = (l == am) ? seed : 0.f;
        const float pv = c[0] * (x * p1 - c[1] * p2) + inj;
#pragma unroll
        for (int o = 0; o < NOP; ++o) {
            const float cp = h[o][l * l + l + m];
            fa[o] += pv * cp;
            if constexpr (!VO) {
                const float dv = (c[2] * p1 - (float)l * x * pv) * r;
                fx[o] += dv * cp;
                fn[o] += pv * h[o][l * l + l - m];
            }
        }
        p2 = p1;
        p1 = pv;
    }
}

// Seeds Pt_|m|^|m|(x_u) of the KM reduction steps of one lane.
template <int LM>
__device__ __forceinline__ void load_seeds(const Tabs<float> &tb, int g4, int ua, float *seed)
{
    using G = Grid<LM>;
#pragma unroll
    for (int kk = 0; kk < G::KM; ++kk) {
        const int m = 4 * kk + g4 - LM, am = m < 0 ? -m : m;
        seed[kk] = am <= LM ? tb.pt[(am * (am + 1) / 2 + am) * G::Ut + ua] : 0.f;
    }
}

// ---------------------------------------------------------------- sender fields

// Legendre pass of all reduction steps of one lane for NOP operands: bf[kk][o][f] holds
// F, dF/dx and m F[-m] (the d/dphi slot swap) of operand o at order m = 4 kk + g - lmax
// (VO: F alone, in f = 0).
template <int LM, int NOP>
struct LaneRows {
    const float4_t *cf;
    const float *h[NOP];
    const float *seed;
    float x, r;
    int g4;
};

template <int LM, int NOP, int KK, bool VO = false>
__device__ __forceinline__ void legendre_all(const LaneRows<LM, NOP> &c,
                                             float (&bf)[Grid<LM>::KM][NOP][3])
{
    if constexpr (KK < Grid<LM>::KM) {
        const int m = 4 * KK + c.g4 - LM;
        float fa[NOP], fx[NOP], fn[NOP];
#pragma unroll
        for (int o = 0; o < NOP; ++o) fa[o] = fx[o] = fn[o] = 0.f;
        legendre_step<LM, KK, NOP, VO>(c.cf, c.h, c.seed[KK], c.x, c.r, m, fa, fx, fn);
#pragma unroll
        for (int o = 0; o < NOP; ++o) {
            bf[KK][o][0] = fa[o];
            if constexpr (!VO) {
                bf[KK][o][1] = fx[o];
                bf[KK][o][2] = (float)m * fn[o];
            }
        }
        // keep the scheduler from hoisting the next step's loads over this one: the straight
        // line code would otherwise hold every step's operands in registers at once
        __builtin_amdgcn_sched_barrier(0);
        legendre_all<LM, NOP, KK + 1, VO>(c, bf);
    }
}

// The functions legendre_step forms, tabulated for one lane and every step: pv[base(KK) + l -
// a0(KK)] = Pt_l^|m|(x) and dv[...] = dPt_l^|m|/dx at the step's order m (zero below l = |m|),
// by the same recurrence and arithmetic. They depend on the lane's node and orders only, so a
// lane that runs the Legendre pass once per edge forms them once.
template <int LM, int KK>
__device__ __forceinline__ void legendre_tabulate(const float4_t *cf, const float *seed, float x,
                                                  float r, int g4,
                                                  float (&pv)[LegendreSteps<LM>::N],
                                                  float (&dv)[LegendreSteps<LM>::N])
{
    if constexpr (KK < Grid<LM>::KM) {
        constexpr int A0 = LegendreSteps<LM>::a0(KK), B = LegendreSteps<LM>::base(KK);
        const int m = 4 * KK + g4 - LM;
        const int am = m < 0 ? (-m < LM ? -m : LM) : (m < LM ? m : LM);
        const float4_t *ca = cf + am;
        float p1 = 0.f, p2 = 0.f;
#pragma unroll
        for (int l = A0; l <= LM; ++l) {
            const float4_t c = ca[l * (l + 1) / 2];
            const float inj = (l == am) ? seed[KK] : 0.f;
            const float p = c[0] * (x * p1 - c[1] * p2) + inj;
            pv[B + l - A0] = p;
            dv[B + l - A0] = (c[2] * p1 - (float)l * x * p) * r;
            p2 = p1;
            p1 = p;
        }
        legendre_tabulate<LM, KK + 1>(cf, seed, x, r, g4, pv, dv);
    }
}

// legendre_all over tabulated functions (legendre_tabulate): the same sums in the same order.
template <int LM, int NOP, int KK>
__device__ __forceinline__ void legendre_all_tab(const float *const *h, int g4,
                                                 const float (&pv)[LegendreSteps<LM>::N],
                                                 const float (&dv)[LegendreSteps<LM>::N],
                                                 float (&bf)[Grid<LM>::KM][NOP][3])
{
    if constexpr (KK < Grid<LM>::KM) {
        constexpr int A0 = LegendreSteps<LM>::a0(KK), B = LegendreSteps<LM>::base(KK);
        const int m = 4 * KK + g4 - LM;
        float fa[NOP], fx[NOP], fn[NOP];
#pragma unroll
        for (int o = 0; o < NOP; ++o) fa[o] = fx[o] = fn[o] = 0.f;
#pragma unroll
        for (int l = A0; l <= LM; ++l) {
            const float p = pv[B + l - A0], d = dv[B + l - A0];
#pragma unroll
            for (int o = 0; o < NOP; ++o) {
                const float cp = h[o][l * l + l + m];
                fa[o] += p * cp;
                fx[o] += d * cp;
                fn[o] += p * h[o][l * l + l - m];
            }
        }
#pragma unroll
        for (int o = 0; o < NOP; ++o) {
            bf[KK][o][0] = fa[o];
            bf[KK][o][1] = fx[o];
            bf[KK][o][2] = (float)m * fn[o];
        }
        __builtin_amdgcn_sched_barrier(0);
        legendre_all_tab<LM, NOP, KK + 1>(h, g4, pv, dv, bf);
    }
}

template <int LM, bool V1>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void k_sender_mfma(Tabs<float> tb, int R, int rb, int nc,
                                                     const float *__restrict__ H,
                                                     float *__restrict__ SF, int planes)
{
    using G = Grid<LM>;
    extern __shared__ float smem[];
    float4_t *cf = reinterpret_cast<float4_t *>(smem);  // [P] recurrence coefficients
    float *qs = smem + 4 * G::P;                         // [4 KM][QB]: q_vm as [m][v]
    float *Hs = qs + 4 * G::KM * G::QB;                  // [rb][HR]
    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    stage_q<LM>(tb, qs, 4 * G::KM, G::QB, false);
    stage_rows<LM>(H + (b * R + r0) * (int64_t)G::K, Hs, nr);
    stage_coefs<LM>(tb, cf);
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int g4 = lane >> 4, n = lane & 15;
    const int rows = nr * G::U;
    const int rtiles = (rows + 15) / 16;
    for (int rt = wave; rt < rtiles; rt += nw) {
        // this lane's A-operand row (q, u); rows past the end compute on row 0 and are
        // never stored (a result row depends on its own A row only)
        const int ra = rt * 16 + n;
        const int qa = ra < rows ? ra / G::U : 0, ua = ra < rows ? ra - qa * G::U : 0;
        float seed[G::KM];
        load_seeds<LM>(tb, g4, ua, seed);
        LaneRows<LM, 1> c;
        c.cf = cf;
        c.h[0] = Hs + qa * G::HR + G::HL;
        c.seed = seed;
        const float sxu = tb.sx[ua];
        c.x = tb.x[ua];
        c.r = 1.f / (sxu * sxu);
        c.g4 = g4;
        // V1: the value field alone (planes 1 and 8), without the derivative passes
        constexpr int NFD = V1 ? 1 : 3;
        float bf[G::KM][1][3];
        legendre_all<LM, 1, 0, V1>(c, bf);
        // Fourier pass: D[(q,u)][v] = sum_m F[(q,u)][m] q_vm, one v tile at a time
        float4_t acc[3][G::VT];
#pragma unroll
        for (int t = 0; t < G::VT; ++t) {
            acc[0][t] = acc[1][t] = acc[2][t] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < G::KM; ++kk) {
                const float bq = qs[(4 * kk + g4) * G::QB + t * 16 + n];
#pragma unroll
                for (int f = 0; f < NFD; ++f)
                    acc[f][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(bf[kk][0][f], bq, acc[f][t],
                                                                     0, 0, 0);
            }
        }
        // D[(q,u) = 16 rt + 4 g + j][v = 16 t + n]
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int ro = rt * 16 + 4 * g4 + j;
            if (ro < rows) {
                const int qo = ro / G::U, uo = ro - qo * G::U;
                if (nc == 0) {  // SF [B][R][3][UVs]
                    float *o = SF + (b * R + r0 + qo) * 3 * (int64_t)G::UVs + uo * G::V + n;
#pragma unroll
                    for (int t = 0; t < G::VT; ++t) {
                        if (t * 16 + n < G::V) {
                            if (planes & 1) o[t * 16] = acc[0][t][j];
                            if (!V1 && (planes & 2)) o[G::UVs + t * 16] = acc[1][t][j];
                            if (!V1 && (planes & 4)) o[2 * G::UVs + t * 16] = acc[2][t][j];
                            if (planes & 8) o[G::UVs + t * 16] = acc[0][t][j];
                        }
                    }
                } else {  // SF [R/16][nc][B][16][3][64]
                    const int r = r0 + qo;
                    const int64_t nb = gridDim.x / nrb;  // B
#pragma unroll
                    for (int t = 0; t < G::VT; ++t) {
                        const int p = uo * G::V + t * 16 + n;
                        if (t * 16 + n < G::V) {
                            const int c = p / kSfChunk, pp = p - c * kSfChunk;
                            float *o = SF + ((((int64_t)(r >> 4) * nc + c) * nb + b) * 16 + (r & 15)) *
                                                3 * kSfChunk + pp;
                            if (planes & 1) o[0] = acc[0][t][j];
                            if (!V1 && (planes & 2)) o[kSfChunk] = acc[1][t][j];
                            if (!V1 && (planes & 4)) o[2 * kSfChunk] = acc[2][t][j];
                            if (planes & 8) o[kSfChunk] = acc[0][t][j];
                        }
                    }
                }
            }
        }
    }
}

// Dense synthesis (lmax <= kDenseSynthMaxL, layout [B][R][3][UVs]): the three grid fields
// of a row (b, r) are one product of its coefficients with the plan's table of the real
// harmonics and their x- and phi-derivatives on the grid,
//   SF[(b,r)][f UVs + p] = sum_k H[(b,r)][k] ysyn[k][f UVs + p].
// At these degrees this costs K x 3 UV matrix-core products per row and no Legendre pass
// on the vector ALUs, which outweighs the separated form's smaller count. The 16-row tiles
// of rows (b, r) are dealt to persistent workgroups of NW waves (12 when the column tiles
// split evenly that way, so that every SIMD carries three waves between the per-tile
// barriers; else 6); wave w owns the column tiles [w CTW, (w + 1) CTW) and holds their
// table operands in registers for the whole launch. A row tile (16 K contiguous floats) is loaded once
// per workgroup with coalesced loads into a double-buffered LDS tile while the previous
// one is multiplied. The product is formed transposed, D[column][row] = table^T H^T, so a
// lane holds four consecutive columns of one row and stores them as one 16-byte vector.
// V1: the value field only (the first UVs columns; the receivers that take the curl in its
// moved-derivative form read nothing else).
// Waves per workgroup. All three fields: 12 when the column tiles split evenly that way,
// else 6 (UVs is a multiple of 32, so CT = 6 UVs / 32 splits over six), either way a whole
// number of a wave's tiles per field, so a wave's tiles lie in one field (its store mask is
// per field). The value field alone: the largest even split up to 12.
constexpr int dense_waves(int ct, bool v1)
{
    if (!v1) return ct % 12 == 0 ? 12 : 6;
    for (int nw = 12; nw > 1; --nw)
        if (ct % nw == 0 && nw != 11 && nw != 9 && nw != 7) return nw;
    return 1;
}

template <int LM, bool V1 = false>
struct DenseSyn {
    using G = Grid<LM>;
    static constexpr int KP = (G::K + 3) / 4 * 4, KS = KP / 4;  // reduction steps of 4
    static constexpr int NCOL = 3 * G::UVs;                     // table and output row length
    static constexpr int CT = (V1 ? G::UVs : NCOL) / 16;        // computed 16-column tiles
    static constexpr int NW = dense_waves(CT, V1), NT = 64 * NW, CTW = CT / NW, WC = 16 * CTW;
    static_assert(CT % NW == 0, "column tiles split evenly over the waves");
    static_assert(V1 || (G::UVs / 16) % CTW == 0, "a wave's column tiles lie in one field");
    // LDS row stride of a staged A row: KA / 2 odd (KP is a multiple of 4) puts the 16 rows x
    // 2 lane groups of each 32-lane half of an operand read on distinct banks
    static constexpr int KA = KP + 2;
    static constexpr int NLA = (16 * G::K + NT - 1) / NT;  // tile loads per thread
};

template <int LM, bool V1>
__global__ __launch_bounds__((64 * DenseSyn<LM, V1>::NW)) __attribute__((amdgpu_waves_per_eu(3))) void k_sender_dense(
    const float *__restrict__ Ys, int64_t rows, const float *__restrict__ H,
    float *__restrict__ SF, int planes)
{
    using G = Grid<LM>;
    using D = DenseSyn<LM, V1>;
    __shared__ float as[2][16 * D::KA];  // staged rows of H (columns past K stay 0)
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g4 = lane >> 4, n = lane & 15;
    for (int i = tid; i < 2 * 16 * D::KA; i += D::NT) (&as[0][0])[i] = 0.f;
    const int t0 = wave * D::CTW;
    const int f = (t0 * 16) / G::UVs;   // the field of this wave's columns (CTW tiles lie in one)
    // V1: the value field, into plane 0 (planes bit 0) or plane 1 (bit 3)
    const bool store = V1 ? (planes & 9) != 0 : ((planes >> f) & 1) != 0;
    const int pofs = V1 && (planes & 8) ? G::UVs : 0;
    // A operand of column tile t at reduction step kk: ysyn[4 kk + g][16 (t0 + t) + n]
    float bq[D::CTW][D::KS];
#pragma unroll
    for (int t = 0; t < D::CTW; ++t)
#pragma unroll
        for (int kk = 0; kk < D::KS; ++kk)
            bq[t][kk] = Ys[(4 * kk + g4) * D::NCOL + (t0 + t) * 16 + n];
    const int64_t ntiles = (rows + 15) / 16, nel = rows * G::K;
    // row tile rt is H[16 K rt, 16 K (rt + 1)); this thread's elements e = tid + NT s, staged
    // as the B operand H[16 rt + n][4 kk + g]
    float xr[D::NLA];
    auto load = [&](int64_t rt) {
#pragma unroll
        for (int s2 = 0; s2 < D::NLA; ++s2) {
            const int e = tid + D::NT * s2;
            const int64_t ge = rt * 16 * G::K + e;
            xr[s2] = (rt < ntiles && e < 16 * G::K && ge < nel) ? H[ge] : 0.f;
        }
    };
    auto stage = [&](float *dst) {
#pragma unroll
        for (int s2 = 0; s2 < D::NLA; ++s2) {
            const int e = tid + D::NT * s2;
            if (e < 16 * G::K) {
                const int rr = e / G::K;
                dst[rr * D::KA + (e - rr * G::K)] = xr[s2];
            }
        }
    };
    load(blockIdx.x);
    stage(as[0]);
    __syncthreads();
    int buf = 0;
    for (int64_t rt = blockIdx.x; rt < ntiles; rt += gridDim.x) {
        load(rt + gridDim.x);  // the next tile, in flight during the products
        float a[D::KS];
#pragma unroll
        for (int kk = 0; kk < D::KS; ++kk) a[kk] = as[buf][n * D::KA + 4 * kk + g4];
        float4_t acc[D::CTW];
#pragma unroll
        for (int t = 0; t < D::CTW; ++t) acc[t] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < D::KS; ++kk)
#pragma unroll
            for (int t = 0; t < D::CTW; ++t)
                acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(bq[t][kk], a[kk], acc[t], 0, 0, 0);
        // D[column 16 t + 4 g + j][row n]: columns 4 g .. 4 g + 3 of row 16 rt + n
        const int64_t row = rt * 16 + n;
        if (store && row < rows) {
            float *dst = SF + row * D::NCOL + pofs + t0 * 16 + 4 * g4;
#pragma unroll
            for (int t = 0; t < D::CTW; ++t) *reinterpret_cast<float4_t *>(dst + 16 * t) = acc[t];
        }
        // the other buffer was last read before the previous barrier
        stage(as[buf ^ 1]);
        __syncthreads();
        buf ^= 1;
    }
}

// ------------------------------------------------------ edge-field receiver (MP)

// Ranks per workgroup of k_receiver_fields_mfma: one wave per 16-row tile of (rank, node u)
// rows, at most 4 waves, so that several workgroups share a CU and one waiting at its
// per-edge barrier leaves the others running.
template <int LM>
struct FieldsTiles {
    using G = Grid<LM>;
    static constexpr int RB = (64 / G::U) < 1 ? 1 : ((64 / G::U) < 16 ? (64 / G::U) : 16);
    // prefetched coefficients per thread, edge and row set: rb rows of HR elements over
    // 64 ceil(rb U / 16) >= 4 rb U threads
    static constexpr int KPT = (G::HR + 4 * G::U - 1) / (4 * G::U);
};

// Raw buffer resource over [base, base + bytes): loads past the end return 0 without a memory
// request.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t fields_rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ float fields_load(__amdgpu_buffer_rsrc_t rs, unsigned voff,
                                             unsigned soff)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, 0));
}

// A byte offset past every resource here, also with the scalar offsets added (which stay far
// below 2^31): such loads return 0.
constexpr unsigned kFieldsOutside = 0x80000000u;

// Receiver for a general per-edge field (two parity-bearing fields, Eq. twoparity-phi):
// a workgroup owns one receiver and rb ranks, one wave per 16-row tile of rows (rank q,
// node u). Per edge each wave synthesises its rows of the edge field's grid fields exactly
// as k_sender_mfma does for a node (the Legendre sums formed in the A-operand registers, the
// Fourier product on MFMA; columns v) and each lane multiplies its D values, rows
// 16 rt + 4 g + j at v = 16 t + n, with the sender values at the same (q, u, v) (Eq.
// msgpass-S; 16 lanes read 64 contiguous bytes of a row). The surface curl takes the
// moved-derivative form (integration by parts on the sphere, as k_receiver_mfma): the edge
// field's x- and phi-derivatives times the sender values are summed into S1, S2, which the
// analysis takes against dY/dphi and dY/dx, so the senders' derivative fields are never
// read. A lane requests its sender values and its share of the next edge's coefficient rows
// when the edge starts,
// so both arrive while it computes; the rows are double-buffered in LDS (one barrier per
// edge). Both are buffer loads whose per-lane byte offsets are fixed over the CSR row and
// computed once (rows and columns past the block read 0 from past the resource); only the
// wave-uniform resources change per edge. The products accumulate in registers over the CSR
// row; the sums (S^alpha, S1, S2) go to S [N][R][3][UVs] for k_analysis_mfma in its moved
// mode. Blocks run in the receiver block order (recv_block), rank block by rank block.
// SPLIT: the value field comes from the rows HE (Gaunt factors) and the two derivative
// fields from the rows HEc (curl factors); both row sets are staged and the Legendre pass
// runs over both. The senders then carry the Gaunt factors' values in plane 0 and the curl
// factors' in plane 1, which the derivative fields multiply.
template <int LM, bool SPLIT>
__global__ __launch_bounds__(512) void k_receiver_fields_mfma(Tabs<float> tb, int R, int rb,
                                                              int64_t N,
                                                              const int32_t *__restrict__ row_ptr,
                                                              const int32_t *__restrict__ col,
                                                              const int32_t *__restrict__ order,
                                                              const float *__restrict__ HE,
                                                              const float *__restrict__ HEc,
                                                              const float *__restrict__ SF,
                                                              float *__restrict__ S)
{
    using G = Grid<LM>;
    constexpr int KPT = FieldsTiles<LM>::KPT;
    constexpr int NS = SPLIT ? 2 : 1;  // coefficient row sets per edge
    extern __shared__ float smem[];
    float4_t *cf = reinterpret_cast<float4_t *>(smem);  // [P] recurrence coefficients
    float *qs = smem + 4 * G::P;                         // [4 KM][QB]: q_vm as [m][v]
    float *Hs = qs + 4 * G::KM * G::QB;                  // [2][NS][rb][HR] this / the next edge
    int64_t slice, i;
    if (!recv_block(N, order, slice, i)) return;
    const int r0 = (int)slice * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    const int nh = nr * G::HR;          // staged elements of one row set
    const int hset = rb * G::HR;        // LDS stride of a row set
    stage_q<LM>(tb, qs, 4 * G::KM, G::QB, false);
    stage_coefs<LM>(tb, cf);

    const int lane = threadIdx.x & 63;
    const int rt = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // this wave's row tile (uniform)
    const int g4 = lane >> 4, n = lane & 15;
    const int rows = nr * G::U;
    // this lane's A row (qa, ua) and its Legendre seeds; its four D rows 16 rt + 4 g + j
    const int ra = rt * 16 + n;
    const int qa = ra < rows ? ra / G::U : 0, ua = ra < rows ? ra - qa * G::U : 0;
    float seed[G::KM];
    load_seeds<LM>(tb, g4, ua, seed);
    const float sxu = tb.sx[ua];
    LaneRows<LM, NS> c;
    c.cf = cf;
    c.seed = seed;
    c.x = tb.x[ua];
    c.r = 1.f / (sxu * sxu);
    c.g4 = g4;
    int off[4];  // offset of D row j in a sender's rank block [rb][3][UVs], -1 if none
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int ro = rt * 16 + 4 * g4 + j;
        const int qo = ro / G::U, uo = ro - qo * G::U;
        off[j] = ro < rows ? qo * 3 * G::UVs + uo * G::V : -1;
    }
    // sender-field byte offsets of D row j at v = 16 t + n: tile t at the scalar offset 64 t,
    // the last tile (whose columns may pass V) with offsets of its own
    constexpr int VL = G::V - 16 * (G::VT - 1);  // valid columns of the last tile
    unsigned foff[4], flast[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        foff[j] = off[j] >= 0 ? (unsigned)(off[j] + n) * 4u : kFieldsOutside;
        flast[j] = off[j] >= 0 && n < VL ? foff[j] : kFieldsOutside;
    }
    const unsigned fbytes = (unsigned)(nr * 3 * G::UVs * 4);
    // staged element kk = tid + t blockDim of a row set is element ii = kk % HR - HL of
    // margin-padded row q = kk / HR: coefficient q K + ii of the edge's rank block, or a
    // margin (0)
    unsigned hoff[KPT];
#pragma unroll
    for (int t = 0; t < KPT; ++t) {
        const int kk = threadIdx.x + t * blockDim.x;
        const int q = kk / G::HR, ii = kk - q * G::HR - G::HL;
        hoff[t] = kk < nh && ii >= 0 && ii < G::K ? (unsigned)(q * G::K + ii) * 4u
                                                   : kFieldsOutside;
    }
    const unsigned hbytes = (unsigned)(nr * G::K * 4);
    auto fetch_rows = [&](int64_t e, float (&hv)[NS][KPT]) {
#pragma unroll
        for (int set = 0; set < NS; ++set) {
            const __amdgpu_buffer_rsrc_t rs =
                fields_rsrc((set ? HEc : HE) + (e * R + r0) * G::K, hbytes);
#pragma unroll
            for (int t = 0; t < KPT; ++t) hv[set][t] = fields_load(rs, hoff[t], 0);
        }
    };
    auto store_rows = [&](float *buf, const float (&hv)[NS][KPT]) {
#pragma unroll
        for (int set = 0; set < NS; ++set)
#pragma unroll
            for (int t = 0; t < KPT; ++t) {
                const int kk = threadIdx.x + t * blockDim.x;
                if (kk < nh) buf[set * hset + kk] = hv[set][t];
            }
    };
    float4_t sa[G::VT], s1[G::VT], s2[G::VT];
#pragma unroll
    for (int t = 0; t < G::VT; ++t) sa[t] = s1[t] = s2[t] = float4_t{0.f, 0.f, 0.f, 0.f};

    const int e0 = row_ptr[i], e1 = row_ptr[i + 1];
    if (e0 < e1) {
        float h0[NS][KPT];
        fetch_rows(e0, h0);
        store_rows(Hs, h0);
    }
    __syncthreads();
    // small lmax: the lane's Legendre functions in registers, formed once for the CSR row
    constexpr int NT = LegendreSteps<LM>::N;
    constexpr bool TAB = 2 * NT <= 44;
    float pvt[NT], dvt[NT];
    if constexpr (TAB) legendre_tabulate<LM, 0>(cf, seed, c.x, c.r, g4, pvt, dvt);
    for (int e = e0; e < e1; ++e) {
        const int cur = (e - e0) & 1;
        const int64_t j = __builtin_amdgcn_readfirstlane(col[e]);
        // this edge's sender fields at the lane's D rows and columns
        const __amdgpu_buffer_rsrc_t sfr = fields_rsrc(SF + (j * R + r0) * 3 * (int64_t)G::UVs,
                                                       fbytes);
        // the sender values (plane 0); SPLIT: the curl factors' values too (plane 1)
        float fI[G::VT][4], fC[G::VT][4];
#pragma unroll
        for (int t = 0; t < G::VT; ++t) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const unsigned vo = t == G::VT - 1 ? flast[jj] : foff[jj];
                const unsigned so = (unsigned)(t * 16 * 4);
                fI[t][jj] = fields_load(sfr, vo, so);
                fC[t][jj] = SPLIT ? fields_load(sfr, vo, so + G::UVs * 4) : fI[t][jj];
            }
        }
        // the next edge's coefficient rows, stored after this edge's Legendre pass
        float hn[NS][KPT];
        const bool more = e + 1 < e1;
        if (more) fetch_rows(e + 1, hn);
        if (rt * 16 < rows) {  // wave-uniform: waves past the last tile only help stage rows
            float *hcur = Hs + cur * NS * hset;
            c.h[0] = hcur + qa * G::HR + G::HL;
            if (SPLIT) c.h[NS - 1] = hcur + hset + qa * G::HR + G::HL;
            float bfa[G::KM][NS][3];
            if constexpr (TAB) legendre_all_tab<LM, NS, 0>(c.h, g4, pvt, dvt, bfa);
            else legendre_all<LM, NS, 0>(c, bfa);
            // value from the first row set, the derivative fields from the last
            float bf[G::KM][1][3];
#pragma unroll
            for (int kk = 0; kk < G::KM; ++kk) {
                bf[kk][0][0] = bfa[kk][0][0];
                bf[kk][0][1] = bfa[kk][NS - 1][1];
                bf[kk][0][2] = bfa[kk][NS - 1][2];
            }
#pragma unroll
            for (int t = 0; t < G::VT; ++t) {
                float4_t acc[3] = {float4_t{0.f, 0.f, 0.f, 0.f}, float4_t{0.f, 0.f, 0.f, 0.f},
                                   float4_t{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
                for (int kk = 0; kk < G::KM; ++kk) {
                    const float bq = qs[(4 * kk + g4) * G::QB + t * 16 + n];
#pragma unroll
                    for (int f = 0; f < 3; ++f)
                        acc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(bf[kk][0][f], bq, acc[f], 0,
                                                                      0, 0);
                }
                // the Gaunt sum and the curl's moved-derivative pair: the edge field's x- and
                // phi-derivatives times the sender values
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    sa[t][jj] += acc[0][jj] * fI[t][jj];
                    s1[t][jj] += acc[1][jj] * fC[t][jj];
                    s2[t][jj] += acc[2][jj] * fC[t][jj];
                }
            }
        }
        if (more) store_rows(Hs + (cur ^ 1) * NS * hset, hn);
        __syncthreads();  // the next rows are staged; this edge's rows are consumed
    }
    float *Sr = S + (i * R + r0) * 3 * (int64_t)G::UVs;
#pragma unroll
    for (int t = 0; t < G::VT; ++t) {
        const int v = t * 16 + n;
        if (v >= G::V) continue;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            if (off[jj] < 0) continue;
            const int ro = rt * 16 + 4 * g4 + jj;
            const int qo = ro / G::U, uo = ro - qo * G::U;
            float *o = Sr + qo * 3 * G::UVs + uo * G::V + v;
            o[0] = sa[t][jj];
            o[G::UVs] = s1[t][jj];
            o[2 * G::UVs] = s2[t][jj];
        }
    }
}

// ------------------------------------------------------ inverse transforms (MP)

// Grid fields per (node, rank) of S for k_analysis_mfma: MODE 0 the summed Gaunt product and
// surface curl (into Ta, Tb); MODE 1 the Gaunt sum into Ta and the curl's moved-derivative
// pair (S1, S2 of analysis_moved) into Tb; MODE 2 (two node slots) a value sum and a moved
// pair for each of Ta and Tb.
constexpr int analysis_fields(int mode) { return mode == 0 ? 2 : mode == 1 ? 3 : 6; }

template <int LM, int MODE>
__global__ __launch_bounds__(256) void k_analysis_mfma(Tabs<float> tb, int R, int rb,
                                                       const float *__restrict__ S,
                                                       float *__restrict__ Ta,
                                                       float *__restrict__ Tb)
{
    using G = Grid<LM>;
    constexpr int NF = analysis_fields(MODE);
    extern __shared__ float smem[];
    float *Ss = smem;                                  // [rb U][VS]: one field's rows at a time
    float *Tm = Ss + (rb * G::U * G::VS + 3) / 4 * 4;  // [rb][NF][M][TS], 16-byte aligned
    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    const int tid = threadIdx.x, nt = blockDim.x;
    const int lane = tid & 63, wave = tid >> 6, nw = nt >> 6, g4 = lane >> 4, n = lane & 15;
    const int rows = nr * G::U;
    const int rtiles = (rows + 15) / 16;
    constexpr int pad = G::VP - G::V;
    if (pad > 0)
        for (int k = tid; k < rb * G::U * pad; k += nt) {
            const int ro = k / pad;
            Ss[ro * G::VS + G::V + (k - ro * pad)] = 0.f;
        }
    constexpr int tpad = G::Ut - G::U;
    if (tpad > 0)
        for (int k = tid; k < nr * NF * G::M * tpad; k += nt) {
            const int ro = k / tpad;
            Tm[ro * G::TS + G::U + (k - ro * tpad)] = 0.f;
        }
    // B operand q[v = 4 kk + g][m = 16 t + n], the same for every tile: held in registers
    float qb[G::KV][G::MT];
#pragma unroll
    for (int kk = 0; kk < G::KV; ++kk)
#pragma unroll
        for (int t = 0; t < G::MT; ++t) {
            const int v = 4 * kk + g4, m = 16 * t + n;
            qb[kk][t] = (v < G::V && m < G::M) ? tb.q[v * G::M + m] : 0.f;
        }
    constexpr int R4 = G::UVs / 4;  // 16-byte words per stored row
    // A thread's 16-byte words k = tid + j nt of a field; the first kPre of them are loaded
    // into registers one field ahead, so their latency overlaps the previous field's products.
    constexpr int kPre = 4;
    auto word = [&](int f, int k) {
        const int q = k / R4, r = 4 * (k - q * R4);
        return *reinterpret_cast<const float4_t *>(S + ((b * R + r0 + q) * NF + f) * (int64_t)G::UVs + r);
    };
    // rows (q, u) of a field as Ss[q U + u][v]; columns V .. VP - 1 stay zero
    auto put = [&](int k, const float4_t &x) {
        const int q = k / R4, r = 4 * (k - q * R4);
        float *dst = Ss + q * G::U * G::VS;
        int u = r / G::V, v = r - u * G::V;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (r + e < G::UV) dst[u * G::VS + v] = x[e];
            if (++v == G::V) {
                v = 0;
                ++u;
            }
        }
    };
    auto live = [&](int k) { return k < nr * R4 && 4 * (k % R4) < G::UV; };
    float4_t pre[kPre];
#pragma unroll
    for (int j = 0; j < kPre; ++j) {
        const int k = tid + j * nt;
        if (live(k)) pre[j] = word(0, k);
    }
    for (int f = 0; f < NF; ++f) {
        // stage field f: the prefetched words, then any further ones directly
#pragma unroll
        for (int j = 0; j < kPre; ++j) {
            const int k = tid + j * nt;
            if (live(k)) put(k, pre[j]);
        }
        for (int k = tid + kPre * nt; k < nr * R4; k += nt)
            if (live(k)) put(k, word(f, k));
        if (f + 1 < NF) {
#pragma unroll
            for (int j = 0; j < kPre; ++j) {
                const int k = tid + j * nt;
                if (live(k)) pre[j] = word(f + 1, k);
            }
        }
        __syncthreads();
        // Tm[(q,u)][m] = sum_v S[(q,u)][v] q_vm (Eq. msgpass-Tmu)
        for (int rt = wave; rt < rtiles; rt += nw) {
            const int ra = rt * 16 + n;
            const float *sa = Ss + (ra < rows ? ra : 0) * G::VS + g4;
            float4_t acc[G::MT];
#pragma unroll
            for (int t = 0; t < G::MT; ++t) acc[t] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < G::KV; ++kk) {
                const float av = sa[4 * kk];
#pragma unroll
                for (int t = 0; t < G::MT; ++t)
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, qb[kk][t], acc[t], 0, 0, 0);
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
                            Tm[((qo * NF + f) * G::M + mi) * G::TS + uo] = acc[t][j];
                        }
                    }
                }
            }
        }
        __syncthreads();  // Ss is read before the next field is staged; Tm is complete
    }
    // Gauss-Legendre analysis: T[k] = sum_u w_u (2 pi / V) Pt_l^|m|(x_u) Tm[m][u] (Eq.
    // msgpass-Tlm) of each value field; a moved-derivative pair (F1, F2) adds
    // -m sum_u w_u (2 pi / V) Pt_l^|m|(x_u) F1[-m][u] - sum_u w_u (2 pi / V) dPt_l^|m|/dx(x_u) F2[m][u]
    // Up to lmax 7 (at most 12 GL nodes and K <= 64) a thread keeps one (l, m) and its weight
    // rows in registers over the ranks it serves, nt / K rank groups side by side (the threads
    // past them idle in this phase); above, where the rows cost more registers and K nears the
    // workgroup size, threads take (rank, k) pairs in turn, which keeps them evenly loaded.
    constexpr bool HOLD = G::Ut <= 12;
    if constexpr (HOLD) {
        constexpr int NC = G::Ut / 4;
        const int gq = G::K < nt ? nt / G::K : 1;
        for (int kq = tid; kq < G::K * gq; kq += nt) {
            const int q0 = kq / G::K, k = kq - q0 * G::K;
            // sqrt(k + 1/2) lies at least 1/(4 (l + 1)) from an integer, far more than the
            // hardware square root's error at these k
            const int l = (int)__builtin_amdgcn_sqrtf((float)k + 0.5f);
            const int m = k - l * l - l, am = m < 0 ? -m : m;
            const int pi = l * (l + 1) / 2 + am;
            const float4_t *w4 = reinterpret_cast<const float4_t *>(tb.wpt + pi * G::Ut);
            const float4_t *wd4 = reinterpret_cast<const float4_t *>(tb.wdpt + pi * G::Ut);
            float4_t wv[NC], wdv[NC];  // the weighted Legendre row and its x-derivative
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                wv[c] = w4[c];
                if (MODE != 0) wdv[c] = wd4[c];
            }
            const float fm = (float)m;
            for (int q = q0; q < nr; q += gq) {
                auto row = [&](int f, int mm) {
                    return reinterpret_cast<const float4_t *>(Tm + ((q * NF + f) * G::M + mm + LM) * G::TS);
                };
                auto dot = [&](const float4_t *w, const float4_t *x) {
                    float sum = 0.f;
#pragma unroll
                    for (int c = 0; c < NC; ++c) {
                        const float4_t a = w[c], y = x[c];
                        sum += a[0] * y[0] + a[1] * y[1] + a[2] * y[2] + a[3] * y[3];
                    }
                    return sum;
                };
                // the moved pair's term, formed alike in every mode: a zero flipped slot (mode
                // 2) then gives exactly the one-slot result (mode 1)
                auto curl = [&](int f1) { return -fm * dot(wv, row(f1, -m)) - dot(wdv, row(f1 + 1, m)); };
                float s0, s1;
                if constexpr (MODE == 0) {
                    s0 = dot(wv, row(0, m));
                    s1 = dot(wv, row(1, m));
                } else if constexpr (MODE == 1) {
                    s0 = dot(wv, row(0, m));
                    s1 = curl(1);
                } else {
                    s0 = dot(wv, row(0, m)) + curl(1);
                    s1 = dot(wv, row(3, m)) + curl(4);
                }
                Ta[(b * R + r0 + q) * (int64_t)G::K + k] = s0;
                Tb[(b * R + r0 + q) * (int64_t)G::K + k] = s1;
            }
        }
    } else {
        for (int idx = tid; idx < nr * G::K; idx += nt) {
            const int q = idx / G::K, k = idx - q * G::K;
            const int l = (int)sqrtf((float)k + 0.5f);  // exact for k < 2^20
            const int m = k - l * l - l, am = m < 0 ? -m : m;
            const int pi = l * (l + 1) / 2 + am;
            const float4_t *w4 = reinterpret_cast<const float4_t *>(tb.wpt + pi * G::Ut);
            const float4_t *wd4 = reinterpret_cast<const float4_t *>(tb.wdpt + pi * G::Ut);
            auto row = [&](int f, int mm) {
                return reinterpret_cast<const float4_t *>(Tm + ((q * NF + f) * G::M + mm + LM) * G::TS);
            };
            auto dot = [&](const float4_t *w, const float4_t *x) {
                float sum = 0.f;
#pragma unroll
                for (int c = 0; c < G::Ut / 4; ++c) {
                    const float4_t a = w[c], y = x[c];
                    sum += a[0] * y[0] + a[1] * y[1] + a[2] * y[2] + a[3] * y[3];
                }
                return sum;
            };
            const float fm = (float)m;
            // the moved pair's term, formed alike in every mode: a zero flipped slot (mode 2)
            // then gives exactly the one-slot result (mode 1)
            auto curl = [&](int f1) { return -fm * dot(w4, row(f1, -m)) - dot(wd4, row(f1 + 1, m)); };
            float s0, s1;
            if constexpr (MODE == 0) {
                s0 = dot(w4, row(0, m));
                s1 = dot(w4, row(1, m));
            } else if constexpr (MODE == 1) {
                s0 = dot(w4, row(0, m));
                s1 = curl(1);
            } else {
                s0 = dot(w4, row(0, m)) + curl(1);
                s1 = dot(w4, row(3, m)) + curl(4);
            }
            Ta[(b * R + r0 + q) * (int64_t)G::K + k] = s0;
            Tb[(b * R + r0 + q) * (int64_t)G::K + k] = s1;
        }
    }
}

// ------------------------------------------------------------- on-site grid stage

template <int LM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(LM <= 16 ? 3 : 1))) void k_onsite_mfma(Tabs<float> tb, int R, int rb,
                                                     const float *__restrict__ HA,
                                                     const float *__restrict__ HB,
                                                     float *__restrict__ Ta,
                                                     float *__restrict__ Tb)
{
    using G = Grid<LM>;
    constexpr int QR = G::VT * 16;     // rows (v) of the staged Fourier tables
    extern __shared__ float smem[];
    float4_t *cf = reinterpret_cast<float4_t *>(smem);  // [P] recurrence coefficients
    float *qs = smem + 4 * G::P;                         // [QR][QS]: q_vm as [v][m]
    float *Hs = qs + QR * G::QS;                         // [2][rb][HR]
    float *Tm = Hs + (2 * rb * G::HR + 3) / 4 * 4;       // [rb][2][M][TS], 16-byte aligned
    const int nrb = (R + rb - 1) / rb;
    const int64_t b = blockIdx.x / nrb;
    const int r0 = (int)(blockIdx.x - b * nrb) * rb;
    const int nr = (R - r0 < rb) ? (R - r0) : rb;
    const int tid = threadIdx.x, nt = blockDim.x;
    stage_q<LM>(tb, qs, QR, G::QS, true);
    stage_rows<LM>(HA + (b * R + r0) * (int64_t)G::K, Hs, nr);
    stage_rows<LM>(HB + (b * R + r0) * (int64_t)G::K, Hs + rb * G::HR, nr);
    stage_coefs<LM>(tb, cf);
    constexpr int tpad = G::Ut - G::U;
    if (tpad > 0)
        for (int k = tid; k < nr * 2 * G::M * tpad; k += nt) {
            const int ro = k / tpad;
            Tm[ro * G::TS + G::U + (k - ro * tpad)] = 0.f;
        }
    __syncthreads();

    const int lane = tid & 63, wave = tid >> 6, nw = nt >> 6, g4 = lane >> 4, n = lane & 15;
    const int rows = nr * G::U;
    const int rtiles = (rows + 15) / 16;
    for (int rt = wave; rt < rtiles; rt += nw) {
        // this lane's row (q, u); rows past the end compute on row 0 and are never stored
        const int ra = rt * 16 + n;
        const int qa = ra < rows ? ra / G::U : 0, ua = ra < rows ? ra - qa * G::U : 0;
        float seed[G::KM];
        load_seeds<LM>(tb, g4, ua, seed);
        LaneRows<LM, 2> c;
        c.cf = cf;
        c.h[0] = Hs + qa * G::HR + G::HL;
        c.h[1] = Hs + (rb + qa) * G::HR + G::HL;
        c.seed = seed;
        const float sxu = tb.sx[ua];
        c.x = tb.x[ua];
        c.r = 1.f / (sxu * sxu);
        c.g4 = g4;
        float bf[G::KM][2][3];
        legendre_all<LM, 2, 0>(c, bf);
        // per v tile: synthesis with the operands swapped, D[v = 16 t + 4 g + j][(q,u) = n]
        // for both operands and the three fields; the products S_alpha = A1 A2
        // (Eq. struct-S) and S_beta = dA1/dphi dA2/dx - dA1/dx dA2/dphi (Eq. poisson-S2-x) at
        // this lane's row; and their share of the analysis Tm[(q,u)][m] = sum_v S q_vm,
        // whose reduction over v is visited as (t, j)
        float4_t ta[G::MT], tbv[G::MT];
#pragma unroll
        for (int mt = 0; mt < G::MT; ++mt) ta[mt] = tbv[mt] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < G::VT; ++t) {
            float4_t a[2][3];
#pragma unroll
            for (int f = 0; f < 3; ++f) a[0][f] = a[1][f] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < G::KM; ++kk) {
                const float aq = qs[(t * 16 + n) * G::QS + 4 * kk + g4];
#pragma unroll
                for (int f = 0; f < 3; ++f) {
                    a[0][f] = __builtin_amdgcn_mfma_f32_16x16x4f32(aq, bf[kk][0][f], a[0][f], 0, 0, 0);
                    a[1][f] = __builtin_amdgcn_mfma_f32_16x16x4f32(aq, bf[kk][1][f], a[1][f], 0, 0, 0);
                }
            }
            const float4_t sal = a[0][0] * a[1][0];
            const float4_t sbe = a[0][2] * a[1][1] - a[0][1] * a[1][2];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float *qb = qs + (t * 16 + 4 * g4 + j) * G::QS + n;
#pragma unroll
                for (int mt = 0; mt < G::MT; ++mt) {
                    const float bq = qb[mt * 16];
                    ta[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(sal[j], bq, ta[mt], 0, 0, 0);
                    tbv[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(sbe[j], bq, tbv[mt], 0, 0, 0);
                }
            }
        }
        // D[(q,u) = 16 rt + 4 g + j][m = 16 mt + n]
#pragma unroll
        for (int mt = 0; mt < G::MT; ++mt) {
            const int mi = mt * 16 + n;
            if (mi < G::M) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int ro = rt * 16 + 4 * g4 + j;
                    if (ro < rows) {
                        const int qo = ro / G::U, uo = ro - qo * G::U;
                        Tm[((qo * 2) * G::M + mi) * G::TS + uo] = ta[mt][j];
                        Tm[((qo * 2 + 1) * G::M + mi) * G::TS + uo] = tbv[mt][j];
                    }
                }
            }
        }
    }
    __syncthreads();
    // Gauss-Legendre analysis: T[k] = sum_u w_u (2 pi / V) Pt_l^|m|(x_u) Tm[m][u]
    for (int idx = tid; idx < 2 * nr * G::K; idx += nt) {
        const int qf = idx / G::K, k = idx - qf * G::K;  // qf = 2 q + field
        const int l = (int)sqrtf((float)k + 0.5f);        // exact for k < 2^20
        const int m = k - l * l - l, am = m < 0 ? -m : m;
        const float4_t *w4 =
            reinterpret_cast<const float4_t *>(tb.wpt + (l * (l + 1) / 2 + am) * G::Ut);
        const float4_t *t4 = reinterpret_cast<const float4_t *>(Tm + (qf * G::M + m + LM) * G::TS);
        float sum = 0.f;
#pragma unroll
        for (int c = 0; c < G::Ut / 4; ++c) {
            const float4_t w = w4[c], tv = t4[c];
            sum += w[0] * tv[0] + w[1] * tv[1] + w[2] * tv[2] + w[3] * tv[3];
        }
        const int q = qf >> 1;
        ((qf & 1) ? Tb : Ta)[(b * R + r0 + q) * (int64_t)G::K + k] = sum;
    }
}

template <int LM>
hipError_t onsite_lm(const Tabs<float> &tb, int64_t B, int R, const float *HA, const float *HB,
                     float *Ta, float *Tb, hipStream_t s)
{
    using G = Grid<LM>;
    const size_t fixed = 4 * (size_t)G::P + (size_t)G::VT * 16 * G::QS + 4;
    const size_t per_rank = 2 * (size_t)G::HR + 2 * (size_t)G::M * G::TS;
    const int rb = pick_rb(tb.d, R, fixed, per_rank);
    if (rb < 1) return hipErrorNotSupported;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_onsite_mfma<LM>), dim3((unsigned)blocks), dim3(64 * waves_for(rb * G::U)),
                       sizeof(float) * (fixed + rb * per_rank), s, tb, R, rb, HA, HB, Ta, Tb);
    return hipGetLastError();
}

// The dense synthesis as persistent workgroups, as many as the device holds at once.
template <int LM, bool V1>
hipError_t launch_dense(const Tabs<float> &tb, int64_t rows, const float *H, float *SF, int planes,
                        hipStream_t s)
{
    using D = DenseSyn<LM, V1>;
    const int64_t ntiles = (rows + 15) / 16;
    static const int64_t resident = [] {
        int dev = 0, cus = 0, per = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &per, reinterpret_cast<const void *>(&k_sender_dense<LM, V1>), 64 * D::NW, 0) !=
                hipSuccess ||
            cus < 1 || per < 1)
            return kDenseSynthBlocks;
        return (int64_t)cus * per;
    }();
    const int64_t grid = ntiles < resident ? ntiles : resident;
    hipLaunchKernelGGL((k_sender_dense<LM, V1>), dim3((unsigned)grid), dim3(64 * D::NW), 0, s,
                       tb.ysyn, rows, H, SF, planes);
    return hipGetLastError();
}

template <int LM>
hipError_t sender_lm(const Tabs<float> &tb, int64_t B, int R, const float *H, float *SF,
                     bool chunked, hipStream_t s, int planes)
{
    using G = Grid<LM>;
    const size_t fixed = 4 * (size_t)G::P + 4 * (size_t)G::KM * G::QB;
    const int rb = pick_rb(tb.d, R, fixed, G::HR);
    if (rb < 1) return hipErrorNotSupported;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    if (chunked && R % 16 != 0) return hipErrorInvalidValue;
    if constexpr (LM >= 1 && LM <= kDenseSynthMaxL) {
        if (!chunked) {
            if (planes == 1 || planes == 8) return launch_dense<LM, true>(tb, B * R, H, SF, planes, s);
            return launch_dense<LM, false>(tb, B * R, H, SF, planes, s);
        }
    }
    const int nc = chunked ? sf_chunks(tb.d) : 0;
    const dim3 grid((unsigned)blocks), block(64 * waves_for(rb * G::U));
    const size_t sh = sizeof(float) * (fixed + rb * (size_t)G::HR);
    if ((planes & ~9) == 0)  // the value field alone (planes 0 and/or 1)
        hipLaunchKernelGGL((k_sender_mfma<LM, true>), grid, block, sh, s, tb, R, rb, nc, H, SF,
                           planes);
    else
        hipLaunchKernelGGL((k_sender_mfma<LM, false>), grid, block, sh, s, tb, R, rb, nc, H, SF,
                           planes);
    return hipGetLastError();
}

template <int LM>
hipError_t analysis_lm(const Tabs<float> &tb, int64_t B, int R, const float *S, float *Ta,
                       float *Tb, hipStream_t s, int mode)
{
    using G = Grid<LM>;
    const size_t fixed = 3;  // alignment of the Tm region
    const size_t per_rank =
        (size_t)G::U * G::VS + (size_t)analysis_fields(mode) * G::M * G::TS;
    const int rb = pick_rb(tb.d, R, fixed, per_rank);
    if (rb < 1) return hipErrorNotSupported;
    const int64_t blocks = B * ((R + rb - 1) / rb);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks), block(64 * waves_for(rb * G::U));
    const size_t sh = sizeof(float) * (fixed + rb * per_rank);
    if (mode == 0)
        hipLaunchKernelGGL((k_analysis_mfma<LM, 0>), grid, block, sh, s, tb, R, rb, S, Ta, Tb);
    else if (mode == 1)
        hipLaunchKernelGGL((k_analysis_mfma<LM, 1>), grid, block, sh, s, tb, R, rb, S, Ta, Tb);
    else
        hipLaunchKernelGGL((k_analysis_mfma<LM, 2>), grid, block, sh, s, tb, R, rb, S, Ta, Tb);
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

bool sender_mfma_supported(const Dims &d) { return default_grid(d) && d.lmax <= 24; }

hipError_t launch_sender_mfma(const Tabs<float> &tb, int64_t B, int R, const float *H, float *SF,
                              bool chunked, hipStream_t s, int planes)
{
    if (B == 0) return hipSuccess;
    if (!sender_mfma_supported(tb.d)) return hipErrorNotSupported;
    switch (tb.d.lmax) {
#define CGTP_CASE(LMV) \
    case LMV: return sender_lm<LMV>(tb, B, R, H, SF, chunked, s, planes);
        CGTP_LMAX_CASES(CGTP_CASE)
#undef CGTP_CASE
    default: return hipErrorNotSupported;
    }
}

template <int LM>
hipError_t receiver_fields_lm(const Tabs<float> &tb, int64_t N, int R, const int32_t *row_ptr,
                              const int32_t *col, const int32_t *order, const float *HE,
                              const float *HEc, const float *SF, float *S, hipStream_t s)
{
    using G = Grid<LM>;
    const int ns = HEc ? 2 : 1;
    int rb = FieldsTiles<LM>::RB;
    if (rb > R) rb = R;
    if (rb < 1) return hipErrorNotSupported;
    const int waves = (rb * G::U + 15) / 16;
    // every staged row element is fetched by some thread's prefetch, and the buffer offsets of
    // a rank block's coefficients and sender fields stay below 2^31
    if ((size_t)rb * G::HR > (size_t)FieldsTiles<LM>::KPT * 64 * waves ||
        (size_t)rb * 3 * G::UVs * 4 >= (size_t)kFieldsOutside)
        return hipErrorNotSupported;
    const size_t sh = sizeof(float) * (4 * (size_t)G::P + 4 * (size_t)G::KM * G::QB +
                                       2 * (size_t)ns * rb * G::HR);
    if (sh > (size_t)tb.d.lds_max) return hipErrorNotSupported;
    const int64_t blocks = recv_blocks(N, (R + rb - 1) / rb);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    if (HEc)
        hipLaunchKernelGGL((k_receiver_fields_mfma<LM, true>), dim3((unsigned)blocks),
                           dim3(64 * waves), sh, s, tb, R, rb, N, row_ptr, col, order, HE, HEc,
                           SF, S);
    else
        hipLaunchKernelGGL((k_receiver_fields_mfma<LM, false>), dim3((unsigned)blocks),
                           dim3(64 * waves), sh, s, tb, R, rb, N, row_ptr, col, order, HE, HEc,
                           SF, S);
    return hipGetLastError();
}

hipError_t launch_receiver_fields_mfma(const Tabs<float> &tb, int64_t N, int R,
                                       const int32_t *row_ptr, const int32_t *col,
                                       const int32_t *order, const float *HE, const float *HEc,
                                       const float *SF, float *S, float *Ta, float *Tb,
                                       hipStream_t s, bool analyse)
{
    if (N == 0) return hipSuccess;
    if (!sender_mfma_supported(tb.d)) return hipErrorNotSupported;
    hipError_t e = hipErrorNotSupported;
    switch (tb.d.lmax) {
#define CGTP_CASE(LMV) \
    case LMV: e = receiver_fields_lm<LMV>(tb, N, R, row_ptr, col, order, HE, HEc, SF, S, s); break;
        CGTP_LMAX_CASES(CGTP_CASE)
#undef CGTP_CASE
    default: return hipErrorNotSupported;
    }
    if (e != hipSuccess || !analyse) return e;
    return launch_analysis_mfma(tb, N, R, S, Ta, Tb, s, 1);
}

hipError_t launch_onsite_mfma(const Tabs<float> &tb, int64_t B, int R, const float *HA,
                              const float *HB, float *Ta, float *Tb, hipStream_t s)
{
    if (B == 0) return hipSuccess;
    if (!default_grid(tb.d)) return hipErrorNotSupported;
    switch (tb.d.lmax) {
#define CGTP_CASE(LMV) \
    case LMV: return onsite_lm<LMV>(tb, B, R, HA, HB, Ta, Tb, s);
        CGTP_LMAX_CASES(CGTP_CASE)
#undef CGTP_CASE
    default: return hipErrorNotSupported;
    }
}

hipError_t launch_analysis_mfma(const Tabs<float> &tb, int64_t B, int R, const float *S, float *Ta,
                                float *Tb, hipStream_t s, int mode)
{
    if (B == 0) return hipSuccess;
    if (!default_grid(tb.d) || mode < 0 || mode > 2) return hipErrorNotSupported;
    switch (tb.d.lmax) {
#define CGTP_CASE(LMV) \
    case LMV: return analysis_lm<LMV>(tb, B, R, S, Ta, Tb, s, mode);
        CGTP_LMAX_CASES(CGTP_CASE)
#undef CGTP_CASE
    default: return hipErrorNotSupported;
    }
}

}  // namespace cgtp
