// Per-degree channel contraction (Eqs. struct-H, msgpass-HI, msgpass-tildeR and
// the lambda projection struct-phi / cat-alpha-phi / cat-beta-phi):
//
//   Y[b*y_sb + o*y_so + k*y_sk] (+)= scale[l(k)] * sum_i W[l(k)*w_sl + i*w_si + o*w_so]
//                                                   * X[b*x_sb + i*K + k]
//
// (with accumulate the result is added to Y). For a fixed degree l this is a GEMM
// Y_l[o][c] = sum_i W_l[i][o] X_l[i][c] over the columns c = (b, m), m = 0..2l (or c = b
// when k is the degree itself).
//
// fp32 path: MFMA tiles (v_mfma_f32_16x16x4f32). k_contract_mfma: a block owns 64
// output rows and 64 columns of one degree of a group of 64 nodes; the blocks of a group
// run back to back over all degrees, so the group's input lines are reused from L2. A
// group of 64 nodes has 64(2l+1) columns of degree l, a whole number of 64-wide tiles,
// so no tile straddles two degrees and only the last group has a ragged edge.
// k_contract_kdeg: the case where k is the degree itself (the edge side).
// fp64 path: one thread per output (verification build).
#include "internal.h"

namespace cgtp {

namespace {

constexpr int kTile = 64;      // output rows (o) and columns (c) per block
constexpr int kThreadsC = 256; // 4 waves, each a 32 x 32 sub-tile (2 x 2 MFMA 16 x 16)

__device__ __forceinline__ int isqrt_small(int t)
{
    int l = (int)sqrtf((float)t);
    while (l * l > t) --l;
    while ((l + 1) * (l + 1) <= t) ++l;
    return l;
}

typedef float float4_t __attribute__((ext_vector_type(4)));

// Raw buffer resource over [base, base + bytes): loads past the end return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ float bload(__amdgpu_buffer_rsrc_t rs, unsigned voff)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, voff, 0, 0));
}

constexpr unsigned kOutside = 0xfffffff0u;  // a buffer offset past every resource: reads 0

// One reduction slice of kCs inputs per LDS stage; each thread prefetches its share of
// the next slice into registers while the matrix cores work on the current one. WT: the
// weights are contiguous along the input index i (w_si == 1) and are staged as
// Ws[o][i] (row stride kSWt = 2 mod 32); otherwise as Ws[i][o] (row stride kSWo = 16 mod
// 32). Either way the global reads are coalesced and the A-operand reads of a half-wave
// hit distinct banks. X is staged as Xs[i][c] (row stride kSWo).
constexpr int kCs = 32;
constexpr int kSWo = kTile + 16;
constexpr int kSWt = kCs + 2;
constexpr int kNS = kTile * kCs / kThreadsC;  // staged elements per thread, per operand

// OT output rows per block (64 or 128): wave (wo, wc) owns OT / 2 rows x 32 columns, i.e.
// OT / 32 x 2 MFMA tiles, so a block with OT = 128 stages each X slice once for 128 outputs.
// GATHER: input rows [c rows, (c + 1) rows) come from xg.base[c] (each with row stride x_sb
// and its rows at stride K); rows is a multiple of the slice kCs, so a slice reads one source.
template <bool WT, int OT, bool GATHER>
__global__ __launch_bounds__(kThreadsC) void k_contract_mfma(
    int64_t B, int Cin, int Cout, int K, int tiles_per_group, int otiles,
    const float *__restrict__ W, int64_t w_sl, int64_t w_si, int64_t w_so,
    const float *__restrict__ X, int64_t x_sb, float *__restrict__ Y, int64_t y_sb, int64_t y_so,
    int64_t y_sk, const float *__restrict__ scale, bool accumulate, XGather xg, Pair2 second)
{
    constexpr int SWo = OT + 16;                 // LDS row stride of Ws[i][o]: 16 mod 32
    constexpr int NW = OT * kCs / kThreadsC;     // staged W elements per thread
    constexpr int OTW = OT / 32;                 // 16-row MFMA tiles per wave
    __shared__ float Ws[WT ? OT * kSWt : kCs * SWo];
    __shared__ float Xs[kCs * kSWo];

    // Blocks are dealt round-robin to the 8 XCDs (block b runs on XCD b % 8), each with
    // its own L2. Remap so that each XCD gets a contiguous range of tiles: the tiles of a
    // node group, which read the same input lines, then share one L2.
    const int64_t nblk = gridDim.x;
    const int64_t per = nblk / 8, rem = nblk % 8;
    const int64_t xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    int64_t bid = (xcd < rem) ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
    // a paired launch runs the second problem (same sizes and strides) on blocks past nper
    if (second.nper > 0 && bid >= second.nper) {
        bid -= second.nper;
        W = second.W;
        X = second.X;
        Y = second.Y;
    }
    const int ot = (int)(bid % otiles);
    const int64_t rest = bid / otiles;
    const int t = (int)(rest % tiles_per_group);
    const int64_t g = rest / tiles_per_group;
    const int l = isqrt_small(t);
    const int sub = t - l * l, width = 2 * l + 1, kofs = l * l;
    const int64_t b0 = g * kTile;                      // first node of the group
    const int64_t nb = (B - b0 < kTile) ? (B - b0) : kTile;
    const int ncols = (int)nb * width;                 // columns of degree l in this group
    const int c0 = sub * kTile;
    const int o0 = ot * OT;
    const float *Wl = W + l * w_sl;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int osub = (wave >> 1) * (OT / 2);
    const int csub = (wave & 1) * 32;
    const int gg = lane >> 4, n = lane & 15;

    float4_t acc[OTW][2];
#pragma unroll
    for (int a = 0; a < OTW; ++a)
        for (int bb = 0; bb < 2; ++bb) acc[a][bb] = float4_t{0.f, 0.f, 0.f, 0.f};

    // this thread's column of X (fixed over the reduction): c = tid % 64, rows i = tid / 64 + 4 s
    const int lc = tid & (kTile - 1), li = tid >> 6;
    const int cg = c0 + lc;
    const bool c_ok = cg < ncols;
    const int bl = c_ok ? cg / width : 0;
    const int mm = c_ok ? cg - bl * width : 0;
    const int64_t xoff = (b0 + bl) * x_sb + kofs + mm;
    float wr[NW], xr[kNS];
    auto fetch = [&](int i0) {
        // the slice's source and its first row there (the whole slice lies in one source)
        const int src = GATHER ? i0 / xg.rows : 0;
        const float *xcol = (GATHER ? xg.base[src] : X) + xoff;
        const int ib = GATHER ? i0 - src * xg.rows : i0;
#pragma unroll
        for (int s2 = 0; s2 < kNS; ++s2) {
            const int ig = i0 + li + 4 * s2;
            xr[s2] = (ig < Cin && c_ok) ? xcol[(int64_t)(ib + li + 4 * s2) * K] : 0.f;
        }
#pragma unroll
        for (int s2 = 0; s2 < NW; ++s2) {
            if (WT) {  // k = tid + 256 s -> (o, i), i fastest
                const int k = tid + kThreadsC * s2, o = k / kCs, i = k - o * kCs;
                wr[s2] = (i0 + i < Cin && o0 + o < Cout) ? Wl[(i0 + i) + (int64_t)(o0 + o) * w_so] : 0.f;
            } else {   // (i, o), o fastest: rows li + 4 (s % kNS), outputs lc + 64 (s / kNS)
                const int ig = i0 + li + 4 * (s2 % kNS), oo = lc + 64 * (s2 / kNS);
                wr[s2] = (ig < Cin && o0 + oo < Cout) ? Wl[(int64_t)ig * w_si + (o0 + oo) * w_so] : 0.f;
            }
        }
    };
    fetch(0);
    for (int i0 = 0; i0 < Cin; i0 += kCs) {
        __syncthreads();  // the previous slice is consumed
#pragma unroll
        for (int s2 = 0; s2 < kNS; ++s2) Xs[(li + 4 * s2) * kSWo + lc] = xr[s2];
#pragma unroll
        for (int s2 = 0; s2 < NW; ++s2) {
            if (WT) {
                const int k = tid + kThreadsC * s2, o = k / kCs, ii = k - o * kCs;
                Ws[o * kSWt + ii] = wr[s2];
            } else {
                Ws[(li + 4 * (s2 % kNS)) * SWo + lc + 64 * (s2 / kNS)] = wr[s2];
            }
        }
        __syncthreads();
        if (i0 + kCs < Cin) fetch(i0 + kCs);
#pragma unroll
        for (int kk = 0; kk < kCs; kk += 4) {
            const int ki = kk + gg;
            float av[OTW];
#pragma unroll
            for (int a = 0; a < OTW; ++a)
                av[a] = WT ? Ws[(osub + 16 * a + n) * kSWt + ki] : Ws[ki * SWo + osub + 16 * a + n];
            const float b0v = Xs[ki * kSWo + csub + n];
            const float b1v = Xs[ki * kSWo + csub + 16 + n];
#pragma unroll
            for (int a = 0; a < OTW; ++a) {
                acc[a][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a], b0v, acc[a][0], 0, 0, 0);
                acc[a][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a], b1v, acc[a][1], 0, 0, 0);
            }
        }
    }

    const float sc = scale ? scale[l] : 1.f;
    // D[row][col] of a 16 x 16 tile: lane holds rows 4*(lane/16) + j, column lane % 16
#pragma unroll
    for (int a = 0; a < OTW; ++a)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb) {
            int c = c0 + csub + 16 * bb + n;
            if (c >= ncols) continue;
            int bcol = c / width;
            int m = c - bcol * width;
            float *ycol = Y + (b0 + bcol) * y_sb + (int64_t)(kofs + m) * y_sk;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                int o = o0 + osub + 16 * a + 4 * gg + j;
                if (o < Cout) {
                    float v = acc[a][bb][j] * sc;
                    if (accumulate) v += ycol[(int64_t)o * y_so];
                    ycol[(int64_t)o * y_so] = v;
                }
            }
        }
}

// kdeg contraction (the edge side, Eq. msgpass-tildeR): Y[b][o][l] over the L degree
// slots of X [B][Cin][L]. A workgroup owns 64 rows b and 64 outputs o for a group of kLG
// degrees, so a row's input block is read once for all of those degrees (four: with their
// 64 accumulator registers four waves fit per SIMD, which hides the loads better than
// seven degrees at two waves, even though a group of 7 then leaves one slot idle). The reduction
// runs in slices of kCk inputs: each thread prefetches its share of the next slice into
// registers while the matrix cores work on the current one from LDS. X rows keep their
// natural (i, l) order in LDS (row stride kSB = 2 mod 32: the A-operand reads of a half-wave
// meet at most two to a bank, the fewest any padded stride gives, since the two lane groups
// of a half-wave read slots 4 apart); W is staged as Ws[l][i][o]. Wave (wb, wo) accumulates
// its 32 x 32 sub-tile of D[b][o] for every degree of the group (A = X rows, B = W
// columns, so 16 lanes write 64 contiguous bytes of a row of Y).
constexpr int kCk = 8;           // reduction slice per LDS stage
constexpr int kLG = 4;           // degrees per workgroup
constexpr int kSB = 34;          // LDS row stride of a staged X row (kCk * kLG = 32 used)
constexpr int kSW = kTile + 16;  // LDS row stride of Ws: lane groups of a half-wave apart
constexpr int kNX = kTile * kCk * kLG / kThreadsC;  // staged elements per thread and slice

__global__ __launch_bounds__(kThreadsC, 4) void k_contract_kdeg(
    int64_t B, int Cin, int Cout, int L, int otiles, int lgroups, const float *__restrict__ W,
    unsigned w_bytes, int w_sl, int w_si, int w_so, const float *__restrict__ X, int x_sb,
    float *__restrict__ Y, int64_t y_sb, int64_t y_so, int64_t y_sk,
    const float *__restrict__ scale, bool accumulate)
{
    __shared__ float Xs[kTile * kSB];
    __shared__ float Ws[kLG][kCk][kSW];
    // XCD-aware order (block b runs on XCD b % 8): the output tiles and degree groups of a
    // row group, which read the same input lines, get consecutive ids on one XCD.
    const int64_t nblk = gridDim.x, per = nblk / 8, rem = nblk % 8;
    const int64_t xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int64_t bid = (xcd < rem) ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
    const int ot = (int)(bid % otiles);
    const int64_t rest = bid / otiles;
    const int lg = (int)(rest % lgroups);
    const int64_t grp = rest / lgroups;
    const int64_t b0 = grp * kTile;
    const int o0 = ot * kTile;
    const int l0 = lg * kLG;
    const int nl = (L - l0 < kLG) ? (L - l0) : kLG;
    const int nb = (B - b0 < kTile) ? (int)(B - b0) : kTile;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, n = lane & 15;
    const int wb = (wave >> 1) * 32, wo = (wave & 1) * 32;
    float4_t acc[kLG][2][2];
#pragma unroll
    for (int l = 0; l < kLG; ++l)
#pragma unroll
        for (int a = 0; a < 2; ++a) acc[l][a][0] = acc[l][a][1] = float4_t{0.f, 0.f, 0.f, 0.f};

    // the row group's inputs (reads past its last row return 0) and the weights
    const __amdgpu_buffer_rsrc_t xs =
        rsrc(X + b0 * (int64_t)x_sb, (unsigned)(((int64_t)(nb - 1) * x_sb + (int64_t)Cin * L) * 4));
    const __amdgpu_buffer_rsrc_t ws = rsrc(W, w_bytes);
    // Staged elements of this thread, k = tid + 256 s. X: row b = k / (kCk kLG) = tid / 32 +
    // 8 s, slot r = k % (kCk kLG) = tid % 32 = i kLG + l of the row's slice (consecutive
    // threads read consecutive slots of a row): one base offset, rows 8 apart. Rows past the
    // group's last lie past the resource and read 0. W: output o = tid % 64 for the
    // wave-uniform (l, i) pairs p = wave + 4 s, l = p / kCk, i = p % kCk.
    static_assert(kThreadsC % (kCk * kLG) == 0, "a thread keeps its slot over s");
    constexpr int kRowStep = kThreadsC / (kCk * kLG);
    const int xi = (tid % (kCk * kLG)) / kLG, xl = tid % kLG;
    const bool x_ok = xl < nl;
    const unsigned xbase = (unsigned)((tid / (kCk * kLG)) * x_sb + xi * L + l0 + xl) * 4u;
    const unsigned xstep = (unsigned)(kRowStep * x_sb) * 4u;
    const int xlds = (tid / (kCk * kLG)) * kSB + tid % (kCk * kLG);
    const bool full_i = Cin % kCk == 0;  // every slice has kCk inputs
    const bool o_ok = o0 + (tid & 63) < Cout;
    const unsigned wcol = (unsigned)((o0 + (tid & 63)) * w_so) * 4u;
    float xr[kNX], wr[kNX];
    auto fetch = [&](int i0) {
        const unsigned di = (unsigned)(i0 * L) * 4u;
        const bool ok = x_ok && (full_i || i0 + xi < Cin);
#pragma unroll
        for (int s2 = 0; s2 < kNX; ++s2) {
            xr[s2] = bload(xs, ok ? xbase + s2 * xstep + di : kOutside);
            const int p = wave + 4 * s2, lw = p / kCk, iw = p % kCk;  // wave-uniform
            const unsigned wo4 = (o_ok && lw < nl && i0 + iw < Cin)
                                     ? wcol + (unsigned)((l0 + lw) * w_sl + (i0 + iw) * w_si) * 4u
                                     : kOutside;
            wr[s2] = bload(ws, wo4);
        }
    };
    fetch(0);
    for (int i0 = 0; i0 < Cin; i0 += kCk) {
        __syncthreads();  // the previous slice is consumed
#pragma unroll
        for (int s2 = 0; s2 < kNX; ++s2) {
            Xs[xlds + s2 * kRowStep * kSB] = xr[s2];
            const int p = wave + 4 * s2;
            Ws[p / kCk][p % kCk][tid & 63] = wr[s2];
        }
        __syncthreads();
        if (i0 + kCk < Cin) fetch(i0 + kCk);
#pragma unroll
        for (int l = 0; l < kLG; ++l)
#pragma unroll
            for (int kk = 0; kk < kCk; kk += 4) {
                const int xo = (kk + g) * kLG + l;
                const float a0 = Xs[(wb + n) * kSB + xo], a1 = Xs[(wb + 16 + n) * kSB + xo];
                const float b0v = Ws[l][kk + g][wo + n], b1v = Ws[l][kk + g][wo + 16 + n];
                acc[l][0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b0v, acc[l][0][0], 0, 0, 0);
                acc[l][0][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b1v, acc[l][0][1], 0, 0, 0);
                acc[l][1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b0v, acc[l][1][0], 0, 0, 0);
                acc[l][1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b1v, acc[l][1][1], 0, 0, 0);
            }
    }
    // D[b = 4 g + j][o = n] of each 16 x 16 tile
#pragma unroll
    for (int l = 0; l < kLG; ++l) {
        if (l >= nl) break;
        const float sc = scale ? scale[l0 + l] : 1.f;
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int o = o0 + wo + 16 * c + n;
                if (o >= Cout) continue;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int b = wb + 16 * a + 4 * g + j;
                    if (b < nb) {
                        float *y = Y + (b0 + b) * y_sb + (int64_t)o * y_so + (int64_t)(l0 + l) * y_sk;
                        float v = acc[l][a][c][j] * sc;
                        if (accumulate) v += *y;
                        *y = v;
                    }
                }
            }
    }
}

template <typename T>
__global__ __launch_bounds__(256) void k_contract_simple(int64_t B, int Cin, int Cout, int K,
                                                         int kdeg, const T *__restrict__ W,
                                                         int64_t w_sl, int64_t w_si, int64_t w_so,
                                                         const T *__restrict__ X, int64_t x_sb,
                                                         T *__restrict__ Y, int64_t y_sb,
                                                         int64_t y_so, int64_t y_sk,
                                                         const T *__restrict__ scale,
                                                         bool accumulate)
{
    const int64_t total = B * (int64_t)Cout * K;
    for (int64_t idx = blockIdx.x * (int64_t)256 + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * 256) {
        int k = (int)(idx % K);
        int64_t rest = idx / K;
        int o = (int)(rest % Cout);
        int64_t b = rest / Cout;
        int l = kdeg ? k : isqrt_small(k);
        const T *w = W + l * w_sl + o * w_so;
        const T *x = X + b * x_sb + k;
        T acc = 0;
        for (int i = 0; i < Cin; ++i) acc += w[i * w_si] * x[(int64_t)i * K];
        if (scale) acc *= scale[l];
        T *y = Y + b * y_sb + o * y_so + (int64_t)k * y_sk;
        *y = accumulate ? *y + acc : acc;
    }
}

}  // namespace

template <>
hipError_t launch_contract<float>(int64_t B, int Cin, int Cout, int K, bool kdeg, const float *W,
                                  int64_t w_sl, int64_t w_si, int64_t w_so, const float *X,
                                  int64_t x_sb, float *Y, int64_t y_sb, int64_t y_so, int64_t y_sk,
                                  const float *scale, bool accumulate, hipStream_t s)
{
    if (B == 0 || Cout == 0 || K == 0) return hipSuccess;
    if (x_sb < (int64_t)Cin * K) return hipErrorInvalidValue;
    if (kdeg) {
        const int64_t groups = (B + kTile - 1) / kTile;
        const int otiles = (Cout + kTile - 1) / kTile;
        const int lgroups = (K + kLG - 1) / kLG;
        const int64_t blocks = groups * otiles * lgroups;
        if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
        // 32-bit buffer offsets: the row group's inputs and every weight index must fit
        const int64_t w_span = 4 * ((K - 1) * w_sl + (int64_t)(Cin - 1) * w_si +
                                    (int64_t)(Cout - 1) * w_so + 1);
        if (w_span >= (int64_t)kOutside ||
            4 * ((int64_t)(kTile - 1) * x_sb + (int64_t)Cin * K) >= (int64_t)kOutside ||
            w_sl < 0 || w_si < 0 || w_so < 0)
            return hipErrorNotSupported;
        hipLaunchKernelGGL(k_contract_kdeg, dim3((unsigned)blocks), dim3(kThreadsC), 0, s, B,
                           Cin, Cout, K, otiles, lgroups, W, (unsigned)w_span, (int)w_sl,
                           (int)w_si, (int)w_so, X, (int)x_sb, Y, y_sb, y_so, y_sk, scale,
                           accumulate);
        return hipGetLastError();
    }
    const int64_t groups = (B + kTile - 1) / kTile;
    const int tiles_per_group = K;  // sum over degrees of the (2l+1) tiles of 64 columns
    // 128 outputs per block once there are that many: each X slice is staged once for them
    const bool wide = Cout >= 128;
    const int ot_rows = wide ? 128 : kTile;
    const int otiles = (Cout + ot_rows - 1) / ot_rows;
    const int64_t blocks = groups * tiles_per_group * otiles;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    const XGather none{};
#define CGTP_CONTRACT(WTV, OTV)                                                                  \
    hipLaunchKernelGGL((k_contract_mfma<WTV, OTV, false>), dim3((unsigned)blocks),               \
                       dim3(kThreadsC), 0, s, B, Cin, Cout, K, tiles_per_group, otiles, W, w_sl, \
                       w_si, w_so, X, x_sb, Y, y_sb, y_so, y_sk, scale, accumulate, none, Pair2{})
    if (w_si == 1) {
        if (wide) CGTP_CONTRACT(true, 128);
        else CGTP_CONTRACT(true, 64);
    } else {
        if (wide) CGTP_CONTRACT(false, 128);
        else CGTP_CONTRACT(false, 64);
    }
#undef CGTP_CONTRACT
    return hipGetLastError();
}

hipError_t launch_contract_gather(int64_t B, int Cout, int K, const float *W, int64_t w_sl,
                                  int64_t w_si, int64_t w_so, const XGather &xg, int nsrc,
                                  int64_t x_sb, float *Y, int64_t y_sb, int64_t y_so,
                                  int64_t y_sk, hipStream_t s)
{
    if (B == 0 || Cout == 0 || K == 0 || nsrc == 0) return hipSuccess;
    if (nsrc > kMaxGather || xg.rows <= 0 || xg.rows % kCs != 0) return hipErrorNotSupported;
    const int Cin = nsrc * xg.rows;
    if (x_sb < (int64_t)xg.rows * K) return hipErrorInvalidValue;
    const int64_t groups = (B + kTile - 1) / kTile;
    const bool wide = Cout >= 128;
    const int otiles = (Cout + (wide ? 128 : kTile) - 1) / (wide ? 128 : kTile);
    const int64_t blocks = groups * K * otiles;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
#define CGTP_CONTRACT(WTV, OTV)                                                                  \
    hipLaunchKernelGGL((k_contract_mfma<WTV, OTV, true>), dim3((unsigned)blocks),                \
                       dim3(kThreadsC), 0, s, B, Cin, Cout, K, K, otiles, W, w_sl, w_si, w_so,   \
                       nullptr, x_sb, Y, y_sb, y_so, y_sk, nullptr, false, xg, Pair2{})
    if (w_si == 1) {
        if (wide) CGTP_CONTRACT(true, 128);
        else CGTP_CONTRACT(true, 64);
    } else {
        if (wide) CGTP_CONTRACT(false, 128);
        else CGTP_CONTRACT(false, 64);
    }
#undef CGTP_CONTRACT
    return hipGetLastError();
}

hipError_t launch_contract_pair(int64_t B, int Cin, int Cout, int K, const float *W0,
                                const float *W1, int64_t w_sl, int64_t w_si, int64_t w_so,
                                const float *X0, const float *X1, int64_t x_sb, float *Y0,
                                float *Y1, int64_t y_sb, int64_t y_so, int64_t y_sk, hipStream_t s)
{
    if (B == 0 || Cout == 0 || K == 0) return hipSuccess;
    if (x_sb < (int64_t)Cin * K) return hipErrorInvalidValue;
    const int64_t groups = (B + kTile - 1) / kTile;
    const bool wide = Cout >= 128;
    const int otiles = (Cout + (wide ? 128 : kTile) - 1) / (wide ? 128 : kTile);
    const int64_t per = groups * K * otiles;  // blocks of one problem
    if (2 * per > 0x7fffffffLL) return hipErrorInvalidValue;
    const XGather none{};
    const Pair2 second{W1, X1, Y1, per};
#define CGTP_CONTRACT(WTV, OTV)                                                                  \
    hipLaunchKernelGGL((k_contract_mfma<WTV, OTV, false>), dim3((unsigned)(2 * per)),            \
                       dim3(kThreadsC), 0, s, B, Cin, Cout, K, K, otiles, W0, w_sl, w_si, w_so,  \
                       X0, x_sb, Y0, y_sb, y_so, y_sk, nullptr, false, none, second)
    if (w_si == 1) {
        if (wide) CGTP_CONTRACT(true, 128);
        else CGTP_CONTRACT(true, 64);
    } else {
        if (wide) CGTP_CONTRACT(false, 128);
        else CGTP_CONTRACT(false, 64);
    }
#undef CGTP_CONTRACT
    return hipGetLastError();
}

template <>
hipError_t launch_contract<double>(int64_t B, int Cin, int Cout, int K, bool kdeg,
                                   const double *W, int64_t w_sl, int64_t w_si, int64_t w_so,
                                   const double *X, int64_t x_sb, double *Y, int64_t y_sb,
                                   int64_t y_so, int64_t y_sk, const double *scale,
                                   bool accumulate, hipStream_t s)
{
    int64_t total = B * (int64_t)Cout * K;
    if (total == 0) return hipSuccess;
    if (x_sb < (int64_t)Cin * K) return hipErrorInvalidValue;
    int64_t blocks = (total + 255) / 256;
    if (blocks > (1 << 20)) blocks = 1 << 20;
    hipLaunchKernelGGL(k_contract_simple<double>, dim3((unsigned)blocks), dim3(256), 0, s, B, Cin,
                       Cout, K, kdeg ? 1 : 0, W, w_sl, w_si, w_so, X, x_sb, Y, y_sb, y_so, y_sk,
                       scale, accumulate);
    return hipGetLastError();
}

}  // namespace cgtp
