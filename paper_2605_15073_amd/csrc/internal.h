// Internal declarations shared by the host plan code and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "cgtp.h"

namespace cgtp {

// Grid sizes derived from lmax and the (possibly overridden) grid.
struct Dims {
    int lmax;  // band limit
    int L;     // lmax + 1
    int K;     // (lmax + 1)^2 flattened SH coefficients
    int M;     // 2 lmax + 1 azimuthal orders
    int P;     // (lmax + 1)(lmax + 2)/2 Legendre (l, m >= 0) pairs
    int U;     // Gauss-Legendre nodes in x = cos(theta)
    int V;     // equispaced phi nodes
    int UV;    // U * V grid points
    int UVs;   // row stride of stored grid fields: UV rounded up to 32 elements, so every
               // row starts on a 128-byte line
    int lds_max;  // LDS bytes one workgroup may use on the plan's device (queried when the
                  // plan is created; 64 KiB until then)
    int lds_cu;   // LDS bytes of one compute unit (the same query)
};

bool resolve_grid(int lmax, int n_theta, int n_phi, int *U, int *V);
Dims make_dims(int lmax, int U, int V);

// fp64 host tables (see cgtp_host_tables in cgtp.h for the layouts).
void gauss_legendre(int n, double *x, double *w);
void legendre_tables(int lmax, int U, const double *x, double *p, double *dp);
void fourier_table(int lmax, int V, double *q);

// Device tables, all in the plan's scalar type T, one allocation per plan.
template <typename T>
struct Tabs {
    const T *x;     // [U] cos(theta_u)
    const T *sx;    // [U] sin(theta_u)
    const T *xsx;   // [U] cos/sin, for d(rhat.Omega)/dx
    const T *wq;    // [U] w_u * 2 pi / V (quadrature weight of a grid point)
    const T *p;     // [U][P] Pt_l^m(x_u)
    const T *dp;    // [U][P] dPt_l^m/dx(x_u)
    const T *q;     // [V][M] real Fourier factor q_vm, column m + lmax
    const T *cphi;  // [V] cos(phi_v)
    const T *sphi;  // [V] sin(phi_v)
    const T *cl;    // [L] (2l+1)/(4 pi): addition theorem weight
    const T *rc1;   // [L] (2l-1)/l  Legendre recurrence, l >= 1
    const T *rc2;   // [L] (l-1)/l
    const T *ya;    // [P] normalised-Legendre recurrence factor a_lm (edge SH)
    const T *yb;    // [P] normalised-Legendre recurrence factor b_lm (edge SH)
    const T *ymm;   // [L] sqrt((2m+1)/(2m)) diagonal step (edge SH), ymm[0] = 1/sqrt(4 pi)
    const T *pt;    // [P][Ut] p transposed, Ut = U rounded up to 4, zero padded
    const T *dpt;   // [P][Ut] dp transposed
    const T *wpt;   // [P][Ut] wq[u] * p transposed (Gauss-Legendre analysis weights)
    const T *wdpt;  // [P][Ut] wq[u] * dp transposed
    const T *yc;    // [P] sqrt((2l+1)(l^2-m^2)/(2l-1)): (1-x^2) dPt_l^m/dx
                    //     = yc Pt_{l-1}^m - l x Pt_l^m
    const T *qd;    // [V][M] the phi-derivative weights of q: column LM + k holds k q[v][LM + k],
                    // column LM - k holds -k q[v][LM - k] (k >= 1), column LM zero
    const T *ysyn;  // [KP][3 UVs] for lmax <= kDenseSynthMaxL (else empty): row k = (l, m),
                    // KP = K rounded up to 4 (rows past K zero); column f UVs + u V + v holds
                    // Y_k (f = 0), dY_k/dx (f = 1) and dY_k/dphi (f = 2) at grid point (u, v),
                    // with zeros past UV in each block

    Dims d;
};

// Degrees up to which the plan builds the dense synthesis table ysyn (the sender fields of
// a row are then one product of its coefficients with that table).
constexpr int kDenseSynthMaxL = 6;

// Number of T elements of each table region, in the order of Tabs.
size_t table_elems(const Dims &d);
void fill_tables(const Dims &d, double *host);  // host fp64 image, table_elems(d) long
template <typename T>
Tabs<T> bind_tables(const Dims &d, const void *dev);

// Generic per-degree channel contraction (Eq. struct-H / struct-phi / msgpass-tildeR):
//   Y[b*y_sb + o*y_so + k*y_sk] (+)= scale[l(k)] * sum_i W[l(k)*w_sl + i*w_si + o*w_so]
//                                                   * X[b*x_sb + i*K + k]
// for rows b < B, inputs i < Cin, outputs o < Cout; x_sb >= Cin*K (Cin*K when X is a packed
// [B][Cin][K]); l(k) = k when kdeg, else the degree of the flattened index k. scale may be
// null. With accumulate the result is added to Y instead of overwriting it. fp32: MFMA
// tiles; fp64: one thread per output (both specialised in contract.hip).
template <typename T>
hipError_t launch_contract(int64_t B, int Cin, int Cout, int K, bool kdeg, const T *W,
                           int64_t w_sl, int64_t w_si, int64_t w_so, const T *X, int64_t x_sb,
                           T *Y, int64_t y_sb, int64_t y_so, int64_t y_sk, const T *scale,
                           bool accumulate, hipStream_t s);
template <>
hipError_t launch_contract<float>(int64_t, int, int, int, bool, const float *, int64_t, int64_t,
                                  int64_t, const float *, int64_t, float *, int64_t, int64_t,
                                  int64_t, const float *, bool, hipStream_t);
template <>
hipError_t launch_contract<double>(int64_t, int, int, int, bool, const double *, int64_t, int64_t,
                                   int64_t, const double *, int64_t, double *, int64_t, int64_t,
                                   int64_t, const double *, bool, hipStream_t);

// fp32 contraction whose Cin = nsrc * xg.rows input rows come from nsrc sources: rows
// [c rows, (c + 1) rows) of node b are xg.base[c] + b * x_sb + i * K (i < rows), otherwise as
// launch_contract (never accumulating, no scale). rows must be a multiple of 32 and
// nsrc <= kMaxGather; hipErrorNotSupported otherwise.
constexpr int kMaxGather = 8;
struct XGather {
    const float *base[kMaxGather];
    int rows;
};
hipError_t launch_contract_gather(int64_t B, int Cout, int K, const float *W, int64_t w_sl,
                                  int64_t w_si, int64_t w_so, const XGather &xg, int nsrc,
                                  int64_t x_sb, float *Y, int64_t y_sb, int64_t y_so,
                                  int64_t y_sk, hipStream_t s);

// Two fp32 contractions of the same sizes and strides (never accumulating, no scale) in one
// launch: Y0 from (W0, X0) and Y1 from (W1, X1), each as launch_contract with kdeg false.
// Small problems are bound by the latency of their few workgroups; one launch overlaps both.
struct Pair2 {
    const float *W;
    const float *X;
    float *Y;
    int64_t nper;  // blocks of the first problem; 0: a single problem
};
hipError_t launch_contract_pair(int64_t B, int Cin, int Cout, int K, const float *W0,
                                const float *W1, int64_t w_sl, int64_t w_si, int64_t w_so,
                                const float *X0, const float *X1, int64_t x_sb, float *Y0,
                                float *Y1, int64_t y_sb, int64_t y_so, int64_t y_sk,
                                hipStream_t s);

// Node-side synthesis of the three grid fields (A, dA/dx, dA/dphi) of H[b][r][K]:
// SF[b][r][3][UVs] (Eqs. struct-F, struct-tildeA plus the derivative passes). Only the
// fields whose bit is set in planes (1: A, 2: dA/dx, 4: dA/dphi) are written; bit 8 writes A
// into plane 1 (the curl factors' values of the moved-derivative form with per-block factors).
template <typename T>
hipError_t launch_sender_fields(const Tabs<T> &tb, int64_t B, int R, const T *H, T *SF,
                                hipStream_t s, int planes = 7);

// On-site grid product and surface curl followed by the inverse transforms:
// Ta/Tb[b][r][K] from HA/HB[b][r][K].
template <typename T>
hipError_t launch_onsite_grid(const Tabs<T> &tb, int64_t B, int R, const T *HA, const T *HB,
                              T *Ta, T *Tb, hipStream_t s);

// fp32 on-site grid stage for lmax <= kOnsiteFoldedMaxL (onsite.hip); returns
// hipErrorNotSupported above that.
// HAc, HBc: NULL, or the curl factors' contractions (then HA, HB are the Gaunt factors': the
// product takes the values of HA, HB and the curl the derivative fields of HAc, HBc).
constexpr int kOnsiteFoldedMaxL = 14;
hipError_t launch_onsite_folded(const Tabs<float> &tb, int64_t B, int R, const float *HA,
                                const float *HB, float *Ta, float *Tb, hipStream_t s,
                                const float *HAc = nullptr, const float *HBc = nullptr);
// Whether the split form (HAc, HBc given) fits this grid: lmax in range and one rank's rows,
// tables and coefficients within a workgroup's LDS.
bool onsite_split_supported(const Dims &d);

// Block order of the receiver passes. Their work is split into slices (a rank block, and a
// chunk of grid points where a pass has them) times receivers. Slices run one after another
// and inside a slice all receivers, so blocks in flight read one slice of the sender fields.
// The hardware hands the blocks of a launch to the kXcds XCDs in turn (block b to XCD
// b mod kXcds); here XCD x takes the x-th of kXcds contiguous spans of the receiver sequence of
// each slice. order[pos] gives the receiver at sequence position pos (NULL: the identity);
// under a locality-preserving order (cgtp_receiver_order) the receivers one XCD runs at once
// are close in space, share most of their senders, and those senders' fields stay in that
// XCD's L2 instead of being fetched again for every edge.
constexpr int kXcds = 8;
__host__ __device__ inline int64_t recv_span(int64_t N) { return (N + kXcds - 1) / kXcds; }
// Blocks of a receiver launch with `slices` slices (at most kXcds - 1 idle per slice).
inline int64_t recv_blocks(int64_t N, int64_t slices) { return kXcds * recv_span(N) * slices; }
// This block's slice and receiver; false for the idle blocks past the last receiver.
__device__ inline bool recv_block(int64_t N, const int32_t *order, int64_t &slice, int64_t &i)
{
    const int64_t m = recv_span(N);
    const int64_t b = blockIdx.x;
    const int64_t k = b / kXcds;
    slice = k / m;
    const int64_t pos = (b - k * kXcds) * m + (k - slice * m);
    if (pos >= N) return false;
    i = order ? (int64_t)order[pos] : pos;
    return true;
}

// Message-passing receiver pass: per receiver, synthesise the edge fields, multiply
// with the streamed sender fields, sum over the CSR row, then the inverse transforms.
// Rt is the edge-radial contraction in the layout [E][L][R].
// order: the receiver sequence of the block order above (NULL: the identity); every
// receiver pass below takes it.
// Rtg: NULL, or separate edge coefficients of the curl product (same layout; zonal edge
// field, one node slot).
// SFf: NULL, or the sender fields of the parity-flipped node slot (two-slot message
// passing; not with the separated edge field).
// values_only: the curl in the moved-derivative form, which reads only the value plane of the
// sender fields (the others need not be written); not with the separated edge field or Rtg.
// Sg (fp32, values_only, default grid): the summed fields go to Sg [N][R][3][UVs] ([6] with
// SFf) and the MFMA analysis follows; NULL: the analysis runs inside the receiver.
template <typename T>
hipError_t launch_receiver(const Tabs<T> &tb, bool separated, int64_t N, int R,
                           const int32_t *row_ptr, const int32_t *col, const int32_t *order,
                           const T *unit, const T *Rt, const T *Rtg, const T *SF, const T *SFf,
                           T *Ta, T *Tb,
                           hipStream_t s, bool values_only = false, T *Sg = nullptr,
                           bool analyse = true);

// Receiver pass for a general per-edge field (two parity-bearing fields): HE [E][R][K] are
// the edge field's channel-contracted coefficients (edge e = row_ptr order), SF the sender
// fields [N][R][3][UVs]; per receiver, the edge syntheses, products with the sender fields,
// the sum over the CSR row and the inverse transforms into Ta, Tb [N][R][K].
// hipErrorNotSupported when the LDS staging does not fit (fp64 at the highest degrees).
template <typename T>
hipError_t launch_receiver_fields(const Tabs<T> &tb, int64_t N, int R, const int32_t *row_ptr,
                                  const int32_t *col, const int32_t *order, const T *HE,
                                  const T *SF, T *Ta, T *Tb, hipStream_t s);

// fp32 edge-field receiver on MFMA (fourier_mfma.hip), default grid, with the curl in the
// moved-derivative form: the summed grid fields (S^alpha, S1, S2) go to S [N][R][3][UVs] and
// the inverse transforms (launch_analysis_mfma mode 1) into Ta, Tb follow. SF in the layout
// [N][R][3][UVs], of which only the sender values (plane 0) are read.
// hipErrorNotSupported off the default grid.
// HEc: NULL, or the edge coefficients of the curl factors (then HE holds the Gaunt factors'
// and gives the value field, HEc the two derivative fields, which multiply the curl factors'
// sender values in plane 1 of SF).
hipError_t launch_receiver_fields_mfma(const Tabs<float> &tb, int64_t N, int R,
                                       const int32_t *row_ptr, const int32_t *col,
                                       const int32_t *order, const float *HE, const float *HEc,
                                       const float *SF, float *S, float *Ta, float *Tb,
                                       hipStream_t s, bool analyse = true);

// nu-body on-site grid product (kernels.hip): Tout[b][r][K] = the analysis of the pointwise
// product of the nu fields synthesised from H.h[t][b][r][K]. The grid of tb must be fine
// enough for the (nu + 1) lmax integrand (checked by the caller).
constexpr int kMaxNu = 8;
template <typename T>
struct NbodyOperands {
    const T *h[kMaxNu];
};
template <typename T>
hipError_t launch_nbody_grid(const Tabs<T> &tb, int64_t B, int R, int nu,
                             const NbodyOperands<T> &H, T *Tout, hipStream_t s);
// fp32 folded form of the same (onsite.hip) for lmax <= 10 and nu = 2 .. 4;
// hipErrorNotSupported otherwise.
hipError_t launch_nbody_folded(const Tabs<float> &tb, int64_t B, int R, int nu,
                               const NbodyOperands<float> &H, float *Tout, hipStream_t s);

// fp32 folded inverse transforms (folded.hip), lmax <= 24; hipErrorNotSupported when
// the LDS staging does not fit.
hipError_t launch_analysis_folded(const Tabs<float> &tb, int64_t B, int R, const float *S,
                                  float *Ta, float *Tb, hipStream_t s);

// fp32 azimuthal transforms on MFMA (fourier_mfma.hip): the sender-field synthesis
// (same output as launch_sender_fields) and the inverse transforms of S [N][R][2][UVs]
// into Ta, Tb. hipErrorNotSupported when the grid is wider than their tiling
// (V > 80) or the LDS staging does not fit.
// With chunked set, SF is written in the layout the MFMA receiver reads:
// [R/16][NC][B][16][3][64], NC = ceil(UV / 64) chunks of 64 grid points, so the fields a
// receiver wave needs from one sender (16 ranks x 3 fields x 64 points) are one
// contiguous 12 KiB run. Requires R % 16 == 0.
constexpr int kSfChunk = 64;
inline int sf_chunks(const Dims &d) { return (d.UV + kSfChunk - 1) / kSfChunk; }
bool sender_mfma_supported(const Dims &d);
hipError_t launch_sender_mfma(const Tabs<float> &tb, int64_t B, int R, const float *H, float *SF,
                              bool chunked, hipStream_t s, int planes = 7);
// Inverse transforms on MFMA of the summed grid fields S [B][R][NF][UVs] into Ta, Tb
// (default grid): mode 0, NF = 2 (Gaunt product, surface curl); mode 1, NF = 3 (Gaunt sum;
// the curl's moved-derivative pair S1, S2); mode 2, NF = 6 (per output a value sum and a
// moved pair, two node slots). hipErrorNotSupported off the default grid.
hipError_t launch_analysis_mfma(const Tabs<float> &tb, int64_t B, int R, const float *S,
                                float *Ta, float *Tb, hipStream_t s, int mode = 0);
// fp32 on-site grid stage on MFMA (fourier_mfma.hip), default grid only: the same
// contract as launch_onsite_grid. Used from kOnsiteMfmaMinL up; below it the
// register-resident folded kernel is faster.
constexpr int kOnsiteMfmaMinL = 15;
hipError_t launch_onsite_mfma(const Tabs<float> &tb, int64_t B, int R, const float *HA,
                              const float *HB, float *Ta, float *Tb, hipStream_t s);

// fp32 receiver pass with the edge synthesis on MFMA (receiver_mfma.hip): writes the
// summed grid fields to S [N][R][2][UVs] and then runs the inverse transforms into
// Ta, Tb. Requires R % 16 == 0.
constexpr int kMfmaRecvMinL = 7;  // three-plane form: below this the per-thread SIMT receiver
bool receiver_mfma_supported(const Dims &d, int R);
// S [N][R][planes][UVs]: 2 planes, or with values_only 3 (6 with SFf).
size_t receiver_mfma_ws_elems(const Dims &d, int64_t N, int R, int planes);
// values_only (not with Rtg; default grid): the moved-derivative curl, reading only the value
// plane of SF (and SFf); every lmax. Otherwise lmax >= kMfmaRecvMinL.
hipError_t launch_receiver_mfma(const Tabs<float> &tb, int64_t N, int R, const int32_t *row_ptr,
                                const int32_t *col, const int32_t *order, const float *unit,
                                const float *Rt, const float *Rtg, const float *SF,
                                const float *SFf, bool sf_chunked, float *S, float *Ta, float *Tb,
                                hipStream_t s, bool values_only = false, bool analyse = true);
// The inverse transforms of the summed grid fields S of a receiver (analyse = false above)
// into Ta, Tb: mode as launch_analysis_mfma; mode 0 also off the default grid.
hipError_t launch_summed_analysis(const Tabs<float> &tb, int64_t N, int R, const float *S,
                                  float *Ta, float *Tb, hipStream_t s, int mode);

// Read-pattern ceiling of the per-thread receiver (kernels.hip): the sender-field loads of
// k_receiver_zonal in its value-only form (fp32, one grid point per thread, blocks of 16
// ranks when they divide R, else 8; plane 0 of SF [N][R][3][UVs]), in its block order, and no
// arithmetic. hipErrorNotSupported for grids of
// more than 1024 points.
hipError_t launch_gather_probe(const Dims &d, int64_t N, int R, const int32_t *row_ptr,
                               const int32_t *col, const int32_t *order, const float *SF,
                               float *sink, hipStream_t s);
// The same for the MFMA receiver in its values-only form on the plain sender layout
// (receiver_mfma.hip): its blocks, block order and 16-byte value-plane loads.
hipError_t launch_gather_probe_mfma(const Dims &d, int64_t N, int R, const int32_t *row_ptr,
                                    const int32_t *col, const int32_t *order, const float *SF,
                                    float *sink, hipStream_t s);

// Status reporting shared by the entry points of every source file: report() stores the
// detail message returned by cgtp_last_error() on this thread and passes the status through.
int report(int status, const char *fmt, ...);
void clear_error();

// The on-site call on a caller-fixed scratch buffer (plan.cpp): the workspace is never
// grown and no stage events are recorded; CGTP_ERR_WORKSPACE when the scratch is too small.
int onsite_fixed_scratch(cgtp_plan plan, int64_t n_nodes, const void *A, const void *B,
                         const void *U_A, const void *U_B, const void *U_out_even,
                         const void *U_out_odd, void *out_even, void *out_odd, void *scratch,
                         size_t scratch_bytes, void *stream);

// Resolves the device address of the fixed scratch of cgtp_onsite_noalloc for device dev,
// which must be current (noalloc.hip). Called by cgtp_plan_create; the result is kept per
// device and later calls return it.
hipError_t noalloc_setup(int dev);

}  // namespace cgtp
