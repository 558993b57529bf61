// C-ABI entry points: plan lifetime, argument validation, workspace layout and
// the stream-ordered launch sequences of the on-site and message-passing paths.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "internal.h"

namespace {
constexpr int kMaxStages = 7;
constexpr int kNumOps = 7;  // CGTP_OP_ONSITE .. CGTP_OP_ONSITE_NBODY
// HIP events bracketing the kernel stages of one call (CGTP_TIME_STAGES).
struct EventSet {
    hipEvent_t ev[kMaxStages + 1];
    int op;
    int n_stages;
    bool complete;
};
}  // namespace

struct cgtp_plan_s {
    cgtp::Dims d;
    int C, R, dtype;
    unsigned flags;
    int device;
    void *tables;        // device table image (plan dtype)
    void *own_ws;        // workspace grown by the plan when the caller passes none
    size_t own_ws_bytes;
    std::vector<EventSet> timers;  // reused across calls; timers_used are pending
    size_t timers_used;
    double stage_acc[kNumOps][kMaxStages];  // drained sums per op (CGTP_OP_*)
    int stage_calls[kNumOps];
    int32_t *order;      // receiver sequence of the message-passing passes (plan-owned device
    int64_t order_n;     // copy of cgtp_plan_set_receiver_order's), NULL: the identity
};

namespace {

thread_local char g_err[512];

int fail(int status, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return status;
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(CGTP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// Largest dynamic LDS any kernel of the plan asks for, in bytes.
size_t max_lds_bytes(const cgtp::Dims &d, size_t es)
{
    size_t qtab = (size_t)d.V * d.M;
    size_t onsite = es * (2 * d.K + 4 * (size_t)d.M * d.U + 2 * (size_t)d.UV);  // q may stay global
    size_t recv_sep = es * (qtab + 2 * (size_t)d.UV + d.K + 2 * (size_t)d.M * d.U);
    size_t sender = es * (qtab + d.K + 2 * (size_t)d.M * d.U);
    if (sender > recv_sep) recv_sep = sender;
    size_t m = onsite > recv_sep ? onsite : recv_sep;
    return m;
}

struct Layout {
    size_t off[6];
    size_t total;
    size_t hf = 0, sff = 0;  // offsets of the second HI / SF (flipped slot or curl factors)
    size_t rtf = 0;          // offset of the second Rt (curl factors)
    size_t wc = 0;           // concatenated factor blocks of a run of rank groups [L][C][R]
};

// Receiver on MFMA in its values-only form (the moved-derivative curl: only the senders'
// values are read, plane 0, and with per-block factors (split) the curl factors' values in
// plane 1): fp32, zonal edge field, R a multiple of 16, the default grid (for the MFMA
// analysis of its moved planes); every lmax.
bool mfma_values_only(const cgtp_plan_s *p, int R, bool split)
{
    (void)split;
    return p->dtype == CGTP_F32 && !(p->flags & CGTP_EDGE_SEPARATED) &&
           cgtp::receiver_mfma_supported(p->d, R) && cgtp::sender_mfma_supported(p->d);
}

// Receiver on MFMA: the values-only form above, else (three sender planes) fp32, zonal edge
// field, R a multiple of 16, lmax high enough that the per-thread recurrence sums would make
// the SIMT receiver compute-bound.
bool use_mfma_receiver(const cgtp_plan_s *p, int R, bool split = false)
{
    return mfma_values_only(p, R, split) ||
           (p->dtype == CGTP_F32 && !(p->flags & CGTP_EDGE_SEPARATED) &&
            p->d.lmax >= cgtp::kMfmaRecvMinL && cgtp::receiver_mfma_supported(p->d, R));
}

// Whether the receiver takes the curl in the moved-derivative form (senders then write only
// their values): the zonal edge field, on the per-thread receiver or on the MFMA one in its
// values-only form.
bool values_only_form(const cgtp_plan_s *p, int R, bool split)
{
    if (p->flags & CGTP_EDGE_SEPARATED) return false;
    return !use_mfma_receiver(p, R, split) || mfma_values_only(p, R, split);
}

// The MFMA receiver reads the sender fields in 64-point chunks when the MFMA sender writes
// them (fp32, default grid, from kMfmaRecvMinL on; below it the dense sender writes the plain
// layout).
bool sf_chunked(const cgtp_plan_s *p, int R, bool split = false)
{
    return use_mfma_receiver(p, R, split) && p->d.lmax >= cgtp::kMfmaRecvMinL &&
           cgtp::sender_mfma_supported(p->d);
}

// On-site workspace: HA, HB, Ta, Tb, each [N][R][K] (R: the plan's rank, or the total
// rank of the groups of the general path), with split factors then HAc, HBc (the curl
// factors' contractions), and the concatenated factor blocks of a run of groups.
Layout onsite_layout(const cgtp_plan_s *p, int R, int64_t N, bool split = false)
{
    size_t es = p->dtype == CGTP_F64 ? 8 : 4;
    size_t blk = align256(es * (size_t)N * R * p->d.K);
    const int nb = split ? 6 : 4;
    Layout l{};
    for (int i = 0; i < 6; ++i) l.off[i] = i * blk;  // HA, HB, Ta, Tb (, HAc, HBc)
    l.wc = nb * blk;
    l.total = nb * blk + align256(es * (size_t)p->d.L * p->C * R);
    return l;
}

// The general on-site call splits its rank groups (one per slot pair, Gaunt and curl
// factors apart) on the folded kernel: fp32, lmax within its range and a grid whose tables
// fit its LDS (a plan with a larger grid override takes the unsplit groups).
bool onsite_split_ok(const cgtp_plan_s *p)
{
    return p->dtype == CGTP_F32 && cgtp::onsite_split_supported(p->d);
}

// The zonal receiver (values-only form, fp32, default grid) hands its summed fields to the
// MFMA analysis through S [N][R][3][UVs] ([6] with two node slots).
bool zonal_mfma_analysis(const cgtp_plan_s *p, int R, bool split)
{
    return p->dtype == CGTP_F32 && !(p->flags & CGTP_EDGE_SEPARATED) &&
           !use_mfma_receiver(p, R, split) && cgtp::sender_mfma_supported(p->d);
}

// Message-passing workspace: HI [N][R][K], SF [N][R][3][UVs], Rt [E][L][R], Ta, Tb [N][R][K],
// and the summed grid fields S: [N][R][2][UVs] for the MFMA receiver, [N][R][3 or 6][UVs] for
// the zonal one handing over to the MFMA analysis. With two node slots,
// HI and SF hold the natural slot followed by the flipped one. With split factors (general
// path), HI and Rt hold the Gaunt factors' contraction followed by the curl factors'. Last,
// room for one sector's output weights concatenated over the groups (the general path's
// gathered projection).
Layout mp_layout(const cgtp_plan_s *p, int R, int64_t N, int64_t E, bool two = false,
                 bool split = false)
{
    size_t es = p->dtype == CGTP_F64 ? 8 : 4;
    const size_t nh = (two || split) ? 2 : 1, nsf = two ? 2 : 1, nrt = split ? 2 : 1;
    size_t h = align256(es * (size_t)N * R * p->d.K);
    const size_t sf_pts = sf_chunked(p, R, split) ? (size_t)cgtp::sf_chunks(p->d) * cgtp::kSfChunk : p->d.UVs;
    size_t sf = align256(es * (size_t)N * R * 3 * sf_pts);
    size_t rt = align256(es * (size_t)E * R * p->d.L);
    const int sg_planes = values_only_form(p, R, split) ? (two ? 6 : 3) : 2;
    size_t sg = use_mfma_receiver(p, R, split)
                    ? align256(es * cgtp::receiver_mfma_ws_elems(p->d, N, R, sg_planes))
                : zonal_mfma_analysis(p, R, split)
                    ? align256(es * (size_t)N * R * sg_planes * p->d.UVs)
                    : 0;
    Layout l{};
    l.off[0] = 0;
    l.off[1] = nh * h;
    l.off[2] = nh * h + nsf * sf;
    l.off[3] = l.off[2] + nrt * rt;
    l.off[4] = l.off[3] + h;
    l.off[5] = l.off[4] + h;
    l.wc = l.off[5] + sg;  // the output weights of a sector's groups, concatenated
    l.total = l.wc + align256(es * (size_t)p->d.L * p->C * R);
    l.hf = h;
    l.sff = sf;
    l.rtf = rt;
    return l;
}

// The edge-field receiver on MFMA (fp32, default grid) writes the summed grid fields
// S [N][R][2][UVs] before the inverse transforms.
bool use_mfma_fields(const cgtp_plan_s *p)
{
    return p->dtype == CGTP_F32 && cgtp::sender_mfma_supported(p->d);
}

// Workspace of message passing with a general edge field: HI [N][R][K], SF [N][R][3][UVs],
// HE [E][R][K], Ta, Tb [N][R][K], S [N][R][2][UVs] for the MFMA receiver, and the
// concatenated factor blocks. With split factors HI and HE are followed by the curl
// factors' contractions.
Layout mpf_layout(const cgtp_plan_s *p, int R, int64_t N, int64_t E, bool split = false)
{
    size_t es = p->dtype == CGTP_F64 ? 8 : 4;
    const size_t ns = split ? 2 : 1;
    size_t h = align256(es * (size_t)N * R * p->d.K);
    size_t sf = align256(es * (size_t)N * R * 3 * p->d.UVs);
    size_t he = align256(es * (size_t)E * R * p->d.K);
    // the MFMA edge-field receiver's sums: the Gaunt sum and the curl's moved pair
    size_t sg = use_mfma_fields(p) ? align256(es * (size_t)N * R * 3 * p->d.UVs) : 0;
    Layout l{};
    l.off[0] = 0;
    l.off[1] = ns * h;
    l.off[2] = ns * h + sf;
    l.off[3] = l.off[2] + ns * he;
    l.off[4] = l.off[3] + h;
    l.off[5] = l.off[4] + h;
    l.hf = h;
    l.rtf = he;
    l.wc = l.off[5] + sg;
    l.total = l.wc + align256(es * (size_t)p->d.L * p->C * R);
    return l;
}

// Workspace of the nu-body product: the nu operand contractions H [N][R][K] each, then
// T [N][R][K].
Layout nbody_layout(const cgtp_plan_s *p, int64_t N, int nu)
{
    size_t es = p->dtype == CGTP_F64 ? 8 : 4;
    size_t h = align256(es * (size_t)N * p->R * p->d.K);
    Layout l{};
    l.off[0] = 0;
    l.off[1] = (size_t)nu * h;
    l.total = (size_t)(nu + 1) * h;
    l.hf = h;
    return l;
}

// Smallest grid on which the product of nu fields of degree lmax, projected onto degree
// lmax, is integrated exactly: Gauss-Legendre with 2 U - 1 >= (nu + 1) lmax, V > (nu + 1) lmax.
void nbody_min_grid(int lmax, int nu, int *U, int *V)
{
    const int deg = (nu + 1) * lmax;
    *U = (deg + 2) / 2;
    if (*U < 1) *U = 1;
    *V = deg + 1;
}

// A receiver order set on the plan must be for the call's node count.
int check_order(const cgtp_plan_s *p, int64_t n_nodes)
{
    if (p->order && p->order_n != n_nodes)
        return fail(CGTP_ERR_ARG, "the plan's receiver order is for %lld nodes, the call has %lld",
                    (long long)p->order_n, (long long)n_nodes);
    return CGTP_OK;
}

int check_device(const cgtp_plan_s *p)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != p->device)
        return fail(CGTP_ERR_ARG, "plan was created on device %d, current device is %d", p->device,
                    dev);
    return CGTP_OK;
}

// Resolve the workspace: the caller's, or the plan's own (grown on demand).
int get_workspace(cgtp_plan_s *p, size_t need, void *ws, size_t ws_bytes, void **out)
{
    if (ws) {
        if (reinterpret_cast<uintptr_t>(ws) % 256 != 0)
            return fail(CGTP_ERR_ARG, "workspace %p is not 256-byte aligned", ws);
        if (ws_bytes < need)
            return fail(CGTP_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, need);
        *out = ws;
        return CGTP_OK;
    }
    if (p->own_ws_bytes < need) {
        if (p->own_ws) {
            hipError_t e = hipDeviceSynchronize();
            if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
            (void)hipFree(p->own_ws);
            p->own_ws = nullptr;
            p->own_ws_bytes = 0;
        }
        hipError_t e = hipMalloc(&p->own_ws, need);
        if (e != hipSuccess) {
            p->own_ws = nullptr;
            return hip_fail(e, "hipMalloc(workspace)");
        }
        p->own_ws_bytes = need;
    }
    *out = p->own_ws;
    return CGTP_OK;
}

// Fold the pending event sets into the plan's running sums.
int drain_timers(cgtp_plan_s *p)
{
    int status = CGTP_OK;
    for (size_t i = 0; i < p->timers_used; ++i) {
        EventSet &es = p->timers[i];
        if (!es.complete) continue;
        hipError_t e = hipEventSynchronize(es.ev[es.n_stages]);
        double t_stage[kMaxStages] = {0};
        for (int k = 0; e == hipSuccess && k < es.n_stages; ++k) {
            float t = 0.f;
            e = hipEventElapsedTime(&t, es.ev[k], es.ev[k + 1]);
            t_stage[k] = t;
        }
        if (e != hipSuccess) {
            status = hip_fail(e, "stage events");
            continue;
        }
        for (int k = 0; k < es.n_stages; ++k) p->stage_acc[es.op][k] += t_stage[k];
        p->stage_calls[es.op] += 1;
    }
    p->timers_used = 0;
    return status;
}

constexpr size_t kMaxPendingTimers = 1024;

// Records the stage boundaries of one call when the plan times its stages.
struct StageRec {
    EventSet *set = nullptr;
    hipStream_t s = nullptr;
    int next = 0;

    int begin(cgtp_plan_s *p, int op, int n_stages, hipStream_t stream)
    {
        if (!(p->flags & CGTP_TIME_STAGES)) return CGTP_OK;
        if (p->timers_used == kMaxPendingTimers) {
            int st = drain_timers(p);
            if (st) return st;
        }
        if (p->timers_used == p->timers.size()) {
            EventSet es{};
            for (int i = 0; i <= kMaxStages; ++i) {
                hipError_t e = hipEventCreate(&es.ev[i]);
                if (e != hipSuccess) {
                    for (int j = 0; j < i; ++j) (void)hipEventDestroy(es.ev[j]);
                    return hip_fail(e, "hipEventCreate");
                }
            }
            p->timers.push_back(es);
        }
        set = &p->timers[p->timers_used++];
        set->op = op;
        set->n_stages = n_stages;
        set->complete = false;
        s = stream;
        next = 0;
        hipError_t e = hipEventRecord(set->ev[0], s);
        return e == hipSuccess ? CGTP_OK : hip_fail(e, "hipEventRecord");
    }
    // stage `next` has been enqueued (or skipped)
    void mark()
    {
        if (!set) return;
        (void)hipEventRecord(set->ev[++next], s);
        if (next == set->n_stages) set->complete = true;
    }
};

// Eq. struct-phi / cat-alpha-phi / cat-beta-phi: out[n][k] (+)= sum_r Uout[l][n][r] T[r][k]
// over R ranks of T, whose rows are x_sb elements apart.
template <typename T>
hipError_t project(int64_t N, int C, int R, int K, const void *Uout, const T *Tsrc, int64_t x_sb,
                   void *out, bool accumulate, hipStream_t s)
{
    return cgtp::launch_contract<T>(N, R, C, K, false, (const T *)Uout, (int64_t)C * R, 1, R, Tsrc,
                                    x_sb, (T *)out, (int64_t)C * K, K, 1, nullptr, accumulate, s);
}

// Eq. struct-H / msgpass-HI: H[b][r][k] = sum_n U[l][n][r] X[b][n][k] into rows of H that are
// h_sb elements apart.
template <typename T>
hipError_t contract_in(int64_t N, int C, int R, int K, const void *U, const void *X, T *H,
                       int64_t h_sb, hipStream_t s)
{
    return cgtp::launch_contract<T>(N, C, R, K, false, (const T *)U, (int64_t)C * R, R, 1,
                                    (const T *)X, (int64_t)C * K, H, h_sb, K, 1, nullptr, false, s);
}

template <typename T>
int run_onsite(cgtp_plan_s *p, int op, int64_t N, const void *A, const void *B, const void *UA,
               const void *UB, const void *Uoe, const void *Uoo, void *oe, void *oo, char *ws,
               hipStream_t s, bool timed = true)
{
    const cgtp::Dims &d = p->d;
    const int C = p->C, R = p->R;
    cgtp::Tabs<T> tb = cgtp::bind_tables<T>(d, p->tables);
    Layout lay = onsite_layout(p, R, N);
    T *HA = reinterpret_cast<T *>(ws + lay.off[0]);
    T *HB = reinterpret_cast<T *>(ws + lay.off[1]);
    T *Ta = reinterpret_cast<T *>(ws + lay.off[2]);
    T *Tb = reinterpret_cast<T *>(ws + lay.off[3]);
    const int64_t hs = (int64_t)R * d.K;
    StageRec rec;
    int st = timed ? rec.begin(p, op, 3, s) : CGTP_OK;
    if (st) return st;
    hipError_t e;
    // Eq. struct-H for both operands (shared when the operands coincide); in fp32 the two
    // contractions run as one launch
    const bool shared = A == B && UA == UB;
    const T *HBp = shared ? HA : HB;
    if (sizeof(T) == 4 && !shared) {
        e = cgtp::launch_contract_pair(N, C, R, d.K, (const float *)UA, (const float *)UB,
                                       (int64_t)C * R, R, 1, (const float *)A, (const float *)B,
                                       (int64_t)C * d.K, (float *)HA, (float *)HB, hs, d.K, 1, s);
    } else {
        e = contract_in<T>(N, C, R, d.K, UA, A, HA, hs, s);
        if (e == hipSuccess && !shared) e = contract_in<T>(N, C, R, d.K, UB, B, HB, hs, s);
    }
    if (e != hipSuccess) return hip_fail(e, "contract operands");
    rec.mark();
    e = cgtp::launch_onsite_grid<T>(tb, N, R, HA, HBp, Ta, Tb, s);
    if (e != hipSuccess) return hip_fail(e, "onsite grid");
    rec.mark();
    // Eqs. struct-phi / cat-beta-phi for the slots asked for (both in one fp32 launch)
    if (sizeof(T) == 4 && oe && oo) {
        e = cgtp::launch_contract_pair(N, R, C, d.K, (const float *)Uoe, (const float *)Uoo,
                                       (int64_t)C * R, 1, R, (const float *)Ta, (const float *)Tb,
                                       hs, (float *)oe, (float *)oo, (int64_t)C * d.K, d.K, 1, s);
    } else {
        e = hipSuccess;
        if (oe) e = project<T>(N, C, R, d.K, Uoe, Ta, hs, oe, false, s);
        if (e == hipSuccess && oo) e = project<T>(N, C, R, d.K, Uoo, Tb, hs, oo, false, s);
    }
    if (e != hipSuccess) return hip_fail(e, "project");
    rec.mark();
    return CGTP_OK;
}

template <typename T>
int run_mp(cgtp_plan_s *p, int op, int64_t N, int64_t E, const int32_t *row_ptr,
           const int32_t *col, const void *unit, const void *rad, const void *I, const void *If,
           const void *UE, const void *UI, const void *Uoe, const void *Uoo, void *oe, void *oo,
           char *ws, hipStream_t s)
{
    const cgtp::Dims &d = p->d;
    const int C = p->C, R = p->R;
    const bool separated = (p->flags & CGTP_EDGE_SEPARATED) != 0;
    const bool two = If != nullptr;
    cgtp::Tabs<T> tb = cgtp::bind_tables<T>(d, p->tables);
    Layout lay = mp_layout(p, R, N, E, two);
    T *HI = reinterpret_cast<T *>(ws + lay.off[0]);
    T *SF = reinterpret_cast<T *>(ws + lay.off[1]);
    T *Rt = reinterpret_cast<T *>(ws + lay.off[2]);
    T *Ta = reinterpret_cast<T *>(ws + lay.off[3]);
    T *Tb = reinterpret_cast<T *>(ws + lay.off[4]);
    T *HIf = two ? reinterpret_cast<T *>(ws + lay.off[0] + lay.hf) : nullptr;
    T *SFf = two ? reinterpret_cast<T *>(ws + lay.off[1] + lay.sff) : nullptr;
    const int64_t hs = (int64_t)R * d.K;
    // the zonal receiver takes the curl in the moved-derivative form: the senders' value plane
    // is all it reads
    const bool values_only = values_only_form(p, R, false);
    StageRec rec;
    int st = rec.begin(p, op, 7, s);
    if (st) return st;
    hipError_t e;
    // Eq. msgpass-HI, then the node-side forward transforms (Eqs. msgpass-FI, msgpass-AI),
    // for each node slot
    for (int slot = 0; slot < (two ? 2 : 1); ++slot) {
        e = contract_in<T>(N, C, R, d.K, UI, slot ? If : I, slot ? HIf : HI, hs, s);
        if (e != hipSuccess) return hip_fail(e, "contract node features");
    }
    rec.mark();
    for (int slot = 0; slot < (two ? 2 : 1); ++slot) {
        T *h = slot ? HIf : HI, *sf = slot ? SFf : SF;
        const int planes = values_only ? 1 : 7;
        if constexpr (sizeof(T) == 4) {
            if (sf_chunked(p, R))
                e = cgtp::launch_sender_mfma(tb, N, R, h, sf, true, s, planes);
            else
                e = cgtp::launch_sender_fields<T>(tb, N, R, h, sf, s, planes);
        } else {
            e = cgtp::launch_sender_fields<T>(tb, N, R, h, sf, s, planes);
        }
        if (e != hipSuccess) return hip_fail(e, "sender fields");
    }
    rec.mark();
    // Eq. msgpass-tildeR into Rt [E][L][R] (the zonal form folds in the addition-theorem
    // weight (2l+1)/(4 pi))
    e = cgtp::launch_contract<T>(E, C, R, d.L, true, (const T *)UE, (int64_t)C * R, R, 1,
                                 (const T *)rad, (int64_t)C * d.L, Rt, (int64_t)d.L * R, 1, R,
                                 separated ? nullptr : tb.cl, false, s);
    if (e != hipSuccess) return hip_fail(e, "contract edge radial");
    rec.mark();
    {
        // the receiver pass (stage 3); the inverse transforms of its summed fields S (stage 4)
        // when they run as a kernel of their own, else inside the receiver (the stage is empty)
        T *Sg = reinterpret_cast<T *>(ws + lay.off[5]);
        int amode = -1;  // analysis mode of S (launch_analysis_mfma), -1: none
        bool mfma = false;
        if constexpr (sizeof(T) == 4) {
            mfma = use_mfma_receiver(p, R);
            if (mfma) {
                e = cgtp::launch_receiver_mfma(tb, N, R, row_ptr, col, p->order,
                                               (const float *)unit, Rt, nullptr, SF, SFf,
                                               sf_chunked(p, R), Sg, Ta, Tb, s, values_only, false);
                if (e != hipSuccess) return hip_fail(e, "receiver (mfma)");
                amode = values_only ? (two ? 2 : 1) : 0;
            }
        }
        if (!mfma) {
            const bool hand_over = values_only && zonal_mfma_analysis(p, R, false);
            e = cgtp::launch_receiver<T>(tb, separated, N, R, row_ptr, col, p->order,
                                         (const T *)unit, Rt, nullptr, SF, SFf, Ta, Tb, s,
                                         values_only, hand_over ? Sg : nullptr, false);
            if (e != hipSuccess) return hip_fail(e, "receiver");
            if (hand_over) amode = two ? 2 : 1;
        }
        rec.mark();
        if constexpr (sizeof(T) == 4) {
            if (amode >= 0) {
                e = cgtp::launch_summed_analysis(tb, N, R, Sg, Ta, Tb, s, amode);
                if (e != hipSuccess) return hip_fail(e, "analysis");
            }
        }
        rec.mark();
    }
    if (oe) {
        e = project<T>(N, C, R, d.K, Uoe, Ta, hs, oe, false, s);
        if (e != hipSuccess) return hip_fail(e, "project even");
    }
    rec.mark();
    if (oo) {
        e = project<T>(N, C, R, d.K, Uoo, Tb, hs, oo, false, s);
        if (e != hipSuccess) return hip_fail(e, "project odd");
    }
    rec.mark();
    return CGTP_OK;
}

// ---------------------------------------------------------------------------------------
// General parameterization (Eqs. msgpass-cp-alpha, msgpass-cp-beta; Table 1): every
// coupling category (0 Gaunt, 1 curl) and output sector (0 out_even, 1 out_odd) may carry
// its own input factors and output weights: block b = 2 category + sector. Operands may
// carry a parity-flipped slot. A slot pair of relative parity rel (0 equal, 1 mixed)
// sends its Gaunt coupling to sector rel and its curl coupling to sector 1 - rel.
//
// The general call is lowered onto the fused kernels by stacking rank groups: group g
// holds the ranks [g R, (g+1) R) of one slot pair, contracted with the factors of the
// blocks it feeds, so one launch of the grid stage at rank G R computes every group's
// Gaunt product (into Ta) and curl (into Tb). Each block then projects the groups that
// feed it, through Ta for a Gaunt block and Tb for a curl block, accumulating into its
// sector's output. With shared input factors a group feeds one Gaunt and one curl block.
// Message passing with per-block factors splits each group: the Gaunt product reads the
// sender value and the edge value sum contracted with its block's factors, the curl
// product the sender derivatives and edge derivative sum contracted with its own; so a
// slot is one group and nothing is computed twice. On-site (both grid operands from one
// contraction per group) and the separated edge field use one group per (slot pair,
// block) instead, and each group's product of the other category is not used.

constexpr int kMaxGroups = 8;

struct Group {
    int s1, s2;  // slots of the first and second operand (0 natural, 1 flipped)
    int bg, bc;  // blocks fed by the group's Gaunt / curl product (-1: none); their input
                 // factors contract the operands
};

struct Groups {
    int n = 0;
    bool split = false;  // groups take different factors for their Gaunt and curl products
    Group g[kMaxGroups];
};

int block_of(int cat, int rel) { return 2 * cat + (cat ? 1 - rel : rel); }

// Whether group g's product of block b's category feeds block b.
bool feeds(const Group &g, int b) { return (b >> 1 ? g.bc : g.bg) == b; }

// f1 / f2: the first / second operand has a flipped slot (message passing: f1 = false, the
// edge field); in_blocks: 1 (shared factors), 2 (per category) or 4 (per block); split:
// per-block factors may differ between a group's two products. Groups are ordered by slot
// pair, so the groups that contract the same operand slot are runs of consecutive groups.
Groups make_groups(bool f1, bool f2, int in_blocks, bool split)
{
    Groups G;
    auto present = [&](int s1, int s2) { return (s1 == 0 || f1) && (s2 == 0 || f2); };
    const int pairs[4][2] = {{0, 0}, {0, 1}, {1, 0}, {1, 1}};
    G.split = split && in_blocks > 1;
    for (const auto &pr : pairs) {
        if (!present(pr[0], pr[1])) continue;
        const int rel = pr[0] != pr[1];
        if (in_blocks == 1 || G.split) {
            G.g[G.n++] = Group{pr[0], pr[1], block_of(0, rel), block_of(1, rel)};
        } else {
            G.g[G.n++] = Group{pr[0], pr[1], block_of(0, rel), -1};
            G.g[G.n++] = Group{pr[0], pr[1], -1, block_of(1, rel)};
        }
    }
    return G;
}

// The block whose input factors contract a group's operands when it has one contraction.
int group_block(const Group &g) { return g.bg >= 0 ? g.bg : g.bc; }

// Factor pointers of the general entry points, resolved per block.
struct Factors {
    const void *in1[4], *in2[4];  // input factors of the first / second operand per block
    const void *out[4];           // output weights per block
};

Factors resolve_factors(const cgtp_plan_s *p, int in_blocks, const void *U1, const void *U2,
                        int out_blocks, const void *Uoe, const void *Uoo)
{
    const size_t es = p->dtype == CGTP_F64 ? 8 : 4;
    const size_t blk = es * (size_t)p->d.L * p->C * p->R;
    Factors f{};
    for (int b = 0; b < 4; ++b) {
        const int cat = b >> 1, sec = b & 1;
        const int ib = in_blocks == 1 ? 0 : (in_blocks == 2 ? cat : b);
        f.in1[b] = static_cast<const char *>(U1) + ib * blk;
        f.in2[b] = static_cast<const char *>(U2) + ib * blk;
        const void *base = sec ? Uoo : Uoe;
        f.out[b] = base ? static_cast<const char *>(base) + (out_blocks == 2 ? cat : 0) * blk
                        : nullptr;
    }
    return f;
}

// Projection of each output sector (Eqs. cat-alpha-phi, cat-beta-phi): the sum over the
// groups' products that feed one of its blocks, each with that block's weights. fp32 with
// R a multiple of 32: one contraction per sector over all of its contributions, the rows
// gathered from Ta / Tb and the weights concatenated along the rank into wcat [L][C][n R];
// otherwise one accumulating contraction per contribution.
template <typename T>
int project_blocks(const cgtp_plan_s *p, const Groups &G, int64_t N, const Factors &f,
                   const T *Ta, const T *Tb, void *oe, void *oo, T *wcat, hipStream_t s,
                   StageRec &rec)
{
    const cgtp::Dims &d = p->d;
    const int C = p->C, R = p->R;
    const int64_t rs = (int64_t)G.n * R * d.K;  // row stride of Ta / Tb
    const size_t es = sizeof(T);
    void *outs[2] = {oe, oo};
    for (int sec = 0; sec < 2; ++sec) {
        const T *src[2 * kMaxGroups];
        int blk[2 * kMaxGroups], n = 0;
        for (int cat = 0; cat < 2 && outs[sec]; ++cat) {
            const int b = 2 * cat + sec;
            for (int gi = 0; gi < G.n; ++gi) {
                if (!feeds(G.g[gi], b)) continue;
                src[n] = (cat ? Tb : Ta) + (int64_t)gi * R * d.K;
                blk[n++] = b;
            }
        }
        const char *what = sec ? "project odd" : "project even";
        hipError_t e = hipSuccess;
        if (sizeof(T) == 4 && n > 1 && n <= cgtp::kMaxGather && R % 32 == 0) {
            cgtp::XGather xg{};
            xg.rows = R;
            for (int c = 0; c < n && e == hipSuccess; ++c) {
                xg.base[c] = reinterpret_cast<const float *>(src[c]);
                e = hipMemcpy2DAsync(wcat + (size_t)c * R, es * n * R, f.out[blk[c]], es * R,
                                     es * R, (size_t)d.L * C, hipMemcpyDeviceToDevice, s);
            }
            if (e == hipSuccess)
                e = cgtp::launch_contract_gather(N, C, d.K, reinterpret_cast<const float *>(wcat),
                                                 (int64_t)C * n * R, 1, (int64_t)n * R, xg, n, rs,
                                                 static_cast<float *>(outs[sec]),
                                                 (int64_t)C * d.K, d.K, 1, s);
            if (e != hipSuccess) return hip_fail(e, what);
        } else {
            for (int c = 0; c < n; ++c) {
                e = project<T>(N, C, R, d.K, f.out[blk[c]], src[c], rs, outs[sec], c > 0, s);
                if (e != hipSuccess) return hip_fail(e, what);
            }
        }
        rec.mark();
    }
    return CGTP_OK;
}

// Channel contraction of every group's operand (first when first, else second) into
// H [rows][G R][K]: one launch per run of consecutive groups that read the same operand slot,
// with the runs' factor blocks concatenated along the rank into wcat [L][C][n R].
// side: 0 the group's one contraction (group_block), 1 its Gaunt factors (bg), 2 its curl
// factors (bc).
template <typename T>
hipError_t contract_runs(const cgtp_plan_s *p, const Groups &G, int64_t rows, bool first,
                         const void *const X[2], const void *const fac[4], T *H, T *wcat,
                         hipStream_t s, int side = 0)
{
    auto blk = [&](const Group &g) { return side == 1 ? g.bg : side == 2 ? g.bc : group_block(g); };
    const cgtp::Dims &d = p->d;
    const int C = p->C, R = p->R, Rg = G.n * R;
    const size_t es = sizeof(T);
    int g0 = 0;
    while (g0 < G.n) {
        const int slot = first ? G.g[g0].s1 : G.g[g0].s2;
        int g1 = g0 + 1;
        while (g1 < G.n && (first ? G.g[g1].s1 : G.g[g1].s2) == slot) ++g1;
        const int n = g1 - g0;
        const T *W = static_cast<const T *>(fac[blk(G.g[g0])]);
        if (n > 1) {
            for (int gi = g0; gi < g1; ++gi) {
                hipError_t e = hipMemcpy2DAsync(wcat + (size_t)(gi - g0) * R, es * n * R,
                                                fac[blk(G.g[gi])], es * R, es * R,
                                                (size_t)d.L * C, hipMemcpyDeviceToDevice, s);
                if (e != hipSuccess) return e;
            }
            W = wcat;
        }
        hipError_t e = cgtp::launch_contract<T>(rows, C, n * R, d.K, false, W, (int64_t)C * n * R,
                                                n * R, 1, static_cast<const T *>(X[slot]),
                                                (int64_t)C * d.K, H + (int64_t)g0 * R * d.K,
                                                (int64_t)Rg * d.K, d.K, 1, nullptr, false, s);
        if (e != hipSuccess) return e;
        g0 = g1;
    }
    return hipSuccess;
}

template <typename T>
int run_onsite_groups(cgtp_plan_s *p, const Groups &G, int64_t N, const void *const X1[2],
                      const void *const X2[2], const Factors &f, void *oe, void *oo, char *ws,
                      hipStream_t s)
{
    const cgtp::Dims &d = p->d;
    const int Rg = G.n * p->R;
    cgtp::Tabs<T> tb = cgtp::bind_tables<T>(d, p->tables);
    Layout lay = onsite_layout(p, Rg, N, G.split);
    T *HA = reinterpret_cast<T *>(ws + lay.off[0]);
    T *HB = reinterpret_cast<T *>(ws + lay.off[1]);
    T *Ta = reinterpret_cast<T *>(ws + lay.off[2]);
    T *Tb = reinterpret_cast<T *>(ws + lay.off[3]);
    T *HAc = G.split ? reinterpret_cast<T *>(ws + lay.off[4]) : nullptr;
    T *HBc = G.split ? reinterpret_cast<T *>(ws + lay.off[5]) : nullptr;
    StageRec rec;
    int st = rec.begin(p, CGTP_OP_ONSITE_GENERAL, 5, s);
    if (st) return st;
    hipError_t e;
    T *wc = reinterpret_cast<T *>(ws + lay.wc);
    const int side = G.split ? 1 : 0;  // split: Gaunt factors first, then the curl factors
    e = contract_runs<T>(p, G, N, true, X1, f.in1, HA, wc, s, side);
    if (e == hipSuccess && G.split) e = contract_runs<T>(p, G, N, true, X1, f.in1, HAc, wc, s, 2);
    if (e != hipSuccess) return hip_fail(e, "contract first operand");
    rec.mark();
    e = contract_runs<T>(p, G, N, false, X2, f.in2, HB, wc, s, side);
    if (e == hipSuccess && G.split) e = contract_runs<T>(p, G, N, false, X2, f.in2, HBc, wc, s, 2);
    if (e != hipSuccess) return hip_fail(e, "contract second operand");
    rec.mark();
    if constexpr (sizeof(T) == 4) {
        if (G.split) {
            e = cgtp::launch_onsite_folded(tb, N, Rg, HA, HB, Ta, Tb, s, HAc, HBc);
            if (e != hipSuccess) return hip_fail(e, "onsite grid (split)");
            rec.mark();
            return project_blocks<T>(p, G, N, f, Ta, Tb, oe, oo, wc, s, rec);
        }
    }
    e = cgtp::launch_onsite_grid<T>(tb, N, Rg, HA, HB, Ta, Tb, s);
    if (e != hipSuccess) return hip_fail(e, "onsite grid");
    rec.mark();
    return project_blocks<T>(p, G, N, f, Ta, Tb, oe, oo, wc, s, rec);
}

template <typename T>
int run_mp_groups(cgtp_plan_s *p, const Groups &G, int64_t N, int64_t E, const int32_t *row_ptr,
                  const int32_t *col, const void *unit, const void *rad, const void *const X2[2],
                  const Factors &f, void *oe, void *oo, char *ws, hipStream_t s)
{
    const cgtp::Dims &d = p->d;
    const int C = p->C, R = p->R, Rg = G.n * R;
    const bool separated = (p->flags & CGTP_EDGE_SEPARATED) != 0;
    cgtp::Tabs<T> tb = cgtp::bind_tables<T>(d, p->tables);
    Layout lay = mp_layout(p, Rg, N, E, false, G.split);
    T *wc = reinterpret_cast<T *>(ws + lay.wc);
    T *HI = reinterpret_cast<T *>(ws + lay.off[0]);
    T *SF = reinterpret_cast<T *>(ws + lay.off[1]);
    T *Rt = reinterpret_cast<T *>(ws + lay.off[2]);
    T *Ta = reinterpret_cast<T *>(ws + lay.off[3]);
    T *Tb = reinterpret_cast<T *>(ws + lay.off[4]);
    // split: the curl products' node contraction and edge coefficients
    T *HIc = G.split ? reinterpret_cast<T *>(ws + lay.off[0] + lay.hf) : nullptr;
    T *Rtc = G.split ? reinterpret_cast<T *>(ws + lay.off[2] + lay.rtf) : nullptr;
    StageRec rec;
    int st = rec.begin(p, CGTP_OP_MESSAGE_PASS_GENERAL, 7, s);
    if (st) return st;
    hipError_t e;
    for (int gi = 0; gi < G.n; ++gi) {
        const Group &g = G.g[gi];
        const int64_t off = (int64_t)gi * R * d.K, hs = (int64_t)Rg * d.K;
        e = contract_in<T>(N, C, R, d.K, f.in2[G.split ? g.bg : group_block(g)], X2[g.s2],
                           HI + off, hs, s);
        if (e == hipSuccess && G.split)
            e = contract_in<T>(N, C, R, d.K, f.in2[g.bc], X2[g.s2], HIc + off, hs, s);
        if (e != hipSuccess) return hip_fail(e, "contract node features");
    }
    rec.mark();
    // split: the Gaunt factors' contraction gives the sender values (plane 0); the curl
    // factors' give the two derivative fields (planes 1, 2), or in the moved-derivative form
    // their values (plane 1)
    const bool values_only = values_only_form(p, Rg, G.split);
    for (int pass = 0; pass < (G.split ? 2 : 1); ++pass) {
        const T *h = pass ? HIc : HI;
        const int planes =
            G.split ? (pass ? (values_only ? 8 : 6) : 1) : (values_only ? 1 : 7);
        if constexpr (sizeof(T) == 4) {
            if (sf_chunked(p, Rg, G.split))
                e = cgtp::launch_sender_mfma(tb, N, Rg, h, SF, true, s, planes);
            else
                e = cgtp::launch_sender_fields<T>(tb, N, Rg, h, SF, s, planes);
        } else {
            e = cgtp::launch_sender_fields<T>(tb, N, Rg, h, SF, s, planes);
        }
        if (e != hipSuccess) return hip_fail(e, "sender fields");
    }
    rec.mark();
    for (int gi = 0; gi < G.n; ++gi) {
        const Group &g = G.g[gi];
        for (int pass = 0; pass < (G.split ? 2 : 1); ++pass) {
            const int blk = G.split ? (pass ? g.bc : g.bg) : group_block(g);
            e = cgtp::launch_contract<T>(E, C, R, d.L, true, (const T *)f.in1[blk],
                                         (int64_t)C * R, R, 1, (const T *)rad, (int64_t)C * d.L,
                                         (pass ? Rtc : Rt) + (int64_t)gi * R, (int64_t)d.L * Rg,
                                         1, Rg, separated ? nullptr : tb.cl, false, s);
            if (e != hipSuccess) return hip_fail(e, "contract edge radial");
        }
    }
    rec.mark();
    // the receiver pass (stage 3), then the inverse transforms of its summed fields S (stage 4)
    // when they run as a kernel of their own
    T *Sg = reinterpret_cast<T *>(ws + lay.off[5]);
    int amode = -1;  // analysis mode of S (launch_analysis_mfma), -1: none
    bool mfma = false;
    if constexpr (sizeof(T) == 4) {
        mfma = use_mfma_receiver(p, Rg, G.split);
        if (mfma) {
            e = cgtp::launch_receiver_mfma(tb, N, Rg, row_ptr, col, p->order, (const float *)unit,
                                           Rt, Rtc, SF, nullptr, sf_chunked(p, Rg, G.split), Sg, Ta,
                                           Tb, s, values_only, false);
            if (e != hipSuccess) return hip_fail(e, "receiver (mfma)");
            amode = values_only ? 1 : 0;
        }
    }
    if (!mfma) {
        const bool hand_over = values_only && zonal_mfma_analysis(p, Rg, G.split);
        e = cgtp::launch_receiver<T>(tb, separated, N, Rg, row_ptr, col, p->order,
                                     (const T *)unit, Rt, Rtc, SF, nullptr, Ta, Tb, s, values_only,
                                     hand_over ? Sg : nullptr, false);
        if (e != hipSuccess) return hip_fail(e, "receiver");
        if (hand_over) amode = 1;
    }
    rec.mark();
    if constexpr (sizeof(T) == 4) {
        if (amode >= 0) {
            e = cgtp::launch_summed_analysis(tb, N, Rg, Sg, Ta, Tb, s, amode);
            if (e != hipSuccess) return hip_fail(e, "analysis");
        }
    }
    rec.mark();
    return project_blocks<T>(p, G, N, f, Ta, Tb, oe, oo, wc, s, rec);
}

// Message passing with two parity-bearing fields (Eq. twoparity-phi): rank groups as for
// the on-site contraction (slot pairs of the edge and node fields); the edge field's
// coefficients are contracted per edge (the analogue of Eq. msgpass-HI on the edge side)
// and synthesised on the grid inside the receiver.
template <typename T>
int run_mp_fields(cgtp_plan_s *p, const Groups &G, int64_t N, int64_t E, const int32_t *row_ptr,
                  const int32_t *col, const void *const X1[2], const void *const X2[2],
                  const Factors &f, void *oe, void *oo, char *ws, hipStream_t s)
{
    const cgtp::Dims &d = p->d;
    const int Rg = G.n * p->R;
    cgtp::Tabs<T> tb = cgtp::bind_tables<T>(d, p->tables);
    Layout lay = mpf_layout(p, Rg, N, E, G.split);
    T *HI = reinterpret_cast<T *>(ws + lay.off[0]);
    T *SF = reinterpret_cast<T *>(ws + lay.off[1]);
    T *HE = reinterpret_cast<T *>(ws + lay.off[2]);
    T *Ta = reinterpret_cast<T *>(ws + lay.off[3]);
    T *Tb = reinterpret_cast<T *>(ws + lay.off[4]);
    // split: the curl factors' node and edge contractions
    T *HIc = G.split ? reinterpret_cast<T *>(ws + lay.off[0] + lay.hf) : nullptr;
    T *HEc = G.split ? reinterpret_cast<T *>(ws + lay.off[2] + lay.rtf) : nullptr;
    StageRec rec;
    int st = rec.begin(p, CGTP_OP_MESSAGE_PASS_FIELDS, 7, s);
    if (st) return st;
    hipError_t e;
    T *wc = reinterpret_cast<T *>(ws + lay.wc);
    e = contract_runs<T>(p, G, N, false, X2, f.in2, HI, wc, s, G.split ? 1 : 0);
    if (e == hipSuccess && G.split) e = contract_runs<T>(p, G, N, false, X2, f.in2, HIc, wc, s, 2);
    if (e != hipSuccess) return hip_fail(e, "contract node features");
    rec.mark();
    // The MFMA receiver takes the curl in the moved-derivative form and reads sender values
    // only: plane 0, and with split factors the curl factors' values in plane 1. The
    // per-thread receiver reads all three fields; split: the Gaunt factors' contraction gives
    // the sender values, the curl factors' the two derivative fields.
    const bool moved = sizeof(T) == 4 && use_mfma_fields(p);
    e = cgtp::launch_sender_fields<T>(tb, N, Rg, HI, SF, s, moved || G.split ? 1 : 7);
    if (e == hipSuccess && G.split)
        e = cgtp::launch_sender_fields<T>(tb, N, Rg, HIc, SF, s, moved ? 8 : 6);
    if (e != hipSuccess) return hip_fail(e, "sender fields");
    rec.mark();
    e = contract_runs<T>(p, G, E, true, X1, f.in1, HE, wc, s, G.split ? 1 : 0);
    if (e == hipSuccess && G.split) e = contract_runs<T>(p, G, E, true, X1, f.in1, HEc, wc, s, 2);
    if (e != hipSuccess) return hip_fail(e, "contract edge field");
    rec.mark();
    if constexpr (sizeof(T) == 4) {
        if (use_mfma_fields(p)) {
            // the receiver pass (stage 3), then the inverse transforms of its sums (stage 4)
            float *Sg = reinterpret_cast<float *>(ws + lay.off[5]);
            e = cgtp::launch_receiver_fields_mfma(tb, N, Rg, row_ptr, col, p->order, HE, HEc, SF,
                                                  Sg, Ta, Tb, s, false);
            if (e != hipSuccess) return hip_fail(e, "receiver (edge field, mfma)");
            rec.mark();
            e = cgtp::launch_summed_analysis(tb, N, Rg, Sg, Ta, Tb, s, 1);
            if (e != hipSuccess) return hip_fail(e, "analysis");
            rec.mark();
            return project_blocks<T>(p, G, N, f, Ta, Tb, oe, oo, wc, s, rec);
        }
    }
    e = cgtp::launch_receiver_fields<T>(tb, N, Rg, row_ptr, col, p->order, HE, SF, Ta, Tb, s);
    if (e == hipErrorNotSupported)
        return fail(CGTP_ERR_UNSUPPORTED,
                    "edge-field receiver: a grid of %d points (at most 2048 off the fp32 default "
                    "grid) or its LDS staging (beyond a workgroup's LDS) is out of range",
                    p->d.UV);
    if (e != hipSuccess) return hip_fail(e, "receiver (edge field)");
    rec.mark();
    rec.mark();  // the analysis ran inside the receiver
    return project_blocks<T>(p, G, N, f, Ta, Tb, oe, oo, wc, s, rec);
}

// nu-body on-site product: one channel contraction per distinct (operand, factor) pair,
// then the fused grid product and analysis, then the projection.
template <typename T>
int run_nbody(cgtp_plan_s *p, int64_t N, int nu, const void *const *X, const void *const *U,
              const void *Uout, void *out, char *ws, hipStream_t s)
{
    const cgtp::Dims &d = p->d;
    const int C = p->C, R = p->R;
    cgtp::Tabs<T> tb = cgtp::bind_tables<T>(d, p->tables);
    Layout lay = nbody_layout(p, N, nu);
    T *Tn = reinterpret_cast<T *>(ws + lay.off[1]);
    const int64_t hs = (int64_t)R * d.K;
    StageRec rec;
    int st = rec.begin(p, CGTP_OP_ONSITE_NBODY, 3, s);
    if (st) return st;
    cgtp::NbodyOperands<T> H{};
    for (int t = 0; t < nu; ++t) {
        int same = -1;  // identical operand and factors: share the contraction
        for (int u = 0; u < t && same < 0; ++u)
            if (X[u] == X[t] && U[u] == U[t]) same = u;
        if (same >= 0) {
            H.h[t] = H.h[same];
            continue;
        }
        T *h = reinterpret_cast<T *>(ws + lay.off[0] + (size_t)t * lay.hf);
        hipError_t e = contract_in<T>(N, C, R, d.K, U[t], X[t], h, hs, s);
        if (e != hipSuccess) return hip_fail(e, "contract operand");
        H.h[t] = h;
    }
    rec.mark();
    hipError_t e = cgtp::launch_nbody_grid<T>(tb, N, R, nu, H, Tn, s);
    if (e == hipErrorNotSupported)
        return fail(CGTP_ERR_UNSUPPORTED, "nu-body grid staging exceeds a workgroup's LDS");
    if (e != hipSuccess) return hip_fail(e, "nu-body grid product");
    rec.mark();
    e = project<T>(N, C, R, d.K, Uout, Tn, hs, out, false, s);
    if (e != hipSuccess) return hip_fail(e, "project");
    rec.mark();
    return CGTP_OK;
}

// How a general call runs: on the fused single-group kernels when the factors are shared
// and each output sector reads one set of weights, else through rank groups.
struct GeneralRoute {
    bool fused;   // run_onsite / run_mp with the plan's rank
    Groups G;     // otherwise: the rank groups
    size_t ws;    // workspace bytes
};

GeneralRoute route_onsite(const cgtp_plan_s *p, int64_t N, bool f1, bool f2, int in_blocks)
{
    GeneralRoute r{};
    r.fused = in_blocks == 1 && !f1 && !f2;
    if (r.fused) {
        r.ws = onsite_layout(p, p->R, N).total;
    } else {
        r.G = make_groups(f1, f2, in_blocks, onsite_split_ok(p));
        r.ws = onsite_layout(p, r.G.n * p->R, N, r.G.split).total;
    }
    return r;
}

GeneralRoute route_mp(const cgtp_plan_s *p, int64_t N, int64_t E, bool flip, int in_blocks,
                      int out_blocks)
{
    GeneralRoute r{};
    // one slot: each sector holds one coupling, so per-category weights change nothing
    r.fused = in_blocks == 1 && (!flip || out_blocks == 1) &&
              !(flip && (p->flags & CGTP_EDGE_SEPARATED));
    if (r.fused) {
        r.ws = mp_layout(p, p->R, N, E, flip).total;
    } else {
        r.G = make_groups(false, flip, in_blocks, !(p->flags & CGTP_EDGE_SEPARATED));
        r.ws = mp_layout(p, r.G.n * p->R, N, E, false, r.G.split).total;
    }
    return r;
}

bool valid_blocks(int in_blocks, int out_blocks)
{
    return (in_blocks == 1 || in_blocks == 2 || in_blocks == 4) &&
           (out_blocks == 1 || out_blocks == 2);
}

int validate_csr(int64_t N, int64_t E, const int32_t *row_ptr, const int32_t *col, hipStream_t s)
{
    std::vector<int32_t> rp((size_t)N + 1), cl((size_t)E);
    hipError_t e = hipMemcpyAsync(rp.data(), row_ptr, sizeof(int32_t) * (N + 1),
                                  hipMemcpyDeviceToHost, s);
    if (e == hipSuccess && E > 0)
        e = hipMemcpyAsync(cl.data(), col, sizeof(int32_t) * E, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "CSR copy");
    if (rp[0] != 0) return fail(CGTP_ERR_CSR, "row_ptr[0] = %d, expected 0", rp[0]);
    for (int64_t i = 0; i < N; ++i)
        if (rp[i + 1] < rp[i])
            return fail(CGTP_ERR_CSR, "row_ptr decreases at row %lld", (long long)i);
    if (rp[N] != E) return fail(CGTP_ERR_CSR, "row_ptr[N] = %d, expected %lld", rp[N], (long long)E);
    for (int64_t k = 0; k < E; ++k)
        if (cl[k] < 0 || cl[k] >= N)
            return fail(CGTP_ERR_CSR, "col[%lld] = %d out of [0, %lld)", (long long)k, cl[k],
                        (long long)N);
    return CGTP_OK;
}

}  // namespace

extern "C" {

int cgtp_plan_create(const cgtp_desc *desc, cgtp_plan *plan)
{
    g_err[0] = 0;
    if (!plan) return fail(CGTP_ERR_ARG, "plan output pointer is NULL");
    *plan = nullptr;
    if (!desc) return fail(CGTP_ERR_ARG, "descriptor is NULL");
    if (desc->lmax < 0 || desc->lmax > CGTP_MAX_LMAX)
        return fail(CGTP_ERR_ARG, "lmax %d outside [0, %d]", desc->lmax, CGTP_MAX_LMAX);
    if (desc->channels < 1 || desc->rank < 1)
        return fail(CGTP_ERR_ARG, "channels (%d) and rank (%d) must be >= 1", desc->channels,
                    desc->rank);
    if (desc->dtype != CGTP_F32 && desc->dtype != CGTP_F64)
        return fail(CGTP_ERR_ARG, "unknown dtype %d", desc->dtype);
    if (desc->flags & ~(CGTP_VALIDATE_CSR | CGTP_EDGE_SEPARATED | CGTP_TIME_STAGES))
        return fail(CGTP_ERR_ARG, "unknown flags 0x%x", desc->flags);
    int U, V;
    if (desc->n_theta < 0 || desc->n_phi < 0 ||
        !cgtp::resolve_grid(desc->lmax, desc->n_theta, desc->n_phi, &U, &V))
        return fail(CGTP_ERR_ARG, "grid %d x %d invalid for lmax %d (minimum %d x %d)",
                    desc->n_theta, desc->n_phi, desc->lmax, (3 * desc->lmax + 2) / 2,
                    3 * desc->lmax + 1);
    cgtp::Dims d = cgtp::make_dims(desc->lmax, U, V);
    size_t es = desc->dtype == CGTP_F64 ? 8 : 4;
    if (d.UV > 11 * 256)
        return fail(CGTP_ERR_UNSUPPORTED, "grid of %d points exceeds 2816", d.UV);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    // the LDS of a workgroup and of a compute unit size the kernels' rank blocks
    e = hipDeviceGetAttribute(&d.lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&d.lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                                  dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute(shared memory)");
    if (max_lds_bytes(d, es) > (size_t)d.lds_max)
        return fail(CGTP_ERR_UNSUPPORTED,
                    "grid %d x %d at lmax %d needs %zu B of LDS (the device's workgroups have "
                    "%d)", U, V, desc->lmax, max_lds_bytes(d, es), d.lds_max);
    // the fixed scratch of cgtp_onsite_noalloc is resolved once per device, here, with the
    // plan's device current; a failure is reported by that entry point, not here
    (void)cgtp::noalloc_setup(dev);
    size_t n = cgtp::table_elems(d);
    std::vector<double> host(n);
    cgtp::fill_tables(d, host.data());
    void *dt = nullptr;
    e = hipMalloc(&dt, n * es);
    if (e != hipSuccess) return hip_fail(e, "hipMalloc(tables)");
    if (desc->dtype == CGTP_F64) {
        e = hipMemcpy(dt, host.data(), n * es, hipMemcpyHostToDevice);
    } else {
        std::vector<float> hf(n);
        for (size_t i = 0; i < n; ++i) hf[i] = (float)host[i];
        e = hipMemcpy(dt, hf.data(), n * es, hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) {
        (void)hipFree(dt);
        return hip_fail(e, "hipMemcpy(tables)");
    }
    cgtp_plan_s *p = new (std::nothrow) cgtp_plan_s();
    if (!p) {
        (void)hipFree(dt);
        return fail(CGTP_ERR_ARG, "out of host memory");
    }
    p->d = d;
    p->C = desc->channels;
    p->R = desc->rank;
    p->dtype = desc->dtype;
    p->flags = desc->flags;
    p->device = dev;
    p->tables = dt;
    p->own_ws = nullptr;
    p->own_ws_bytes = 0;
    p->timers_used = 0;
    p->order = nullptr;
    p->order_n = 0;
    *plan = p;
    return CGTP_OK;
}

int cgtp_plan_grid(cgtp_plan plan, int *n_theta, int *n_phi)
{
    if (!plan) return fail(CGTP_ERR_ARG, "plan is NULL");
    if (n_theta) *n_theta = plan->d.U;
    if (n_phi) *n_phi = plan->d.V;
    return CGTP_OK;
}

int cgtp_workspace_bytes(cgtp_plan plan, int op, int64_t n_nodes, int64_t n_edges, size_t *bytes)
{
    if (!plan || !bytes) return fail(CGTP_ERR_ARG, "NULL argument");
    if (n_nodes < 0 || n_edges < 0) return fail(CGTP_ERR_ARG, "negative size");
    if (op == CGTP_OP_ONSITE) *bytes = onsite_layout(plan, plan->R, n_nodes).total;
    else if (op == CGTP_OP_MESSAGE_PASS) *bytes = mp_layout(plan, plan->R, n_nodes, n_edges).total;
    else if (op == CGTP_OP_MESSAGE_PASS_TWO_SLOT)
        *bytes = mp_layout(plan, plan->R, n_nodes, n_edges, true).total;
    else return fail(CGTP_ERR_ARG, "unknown op %d (general ops: cgtp_workspace_bytes_general)", op);
    return CGTP_OK;
}

}  // extern "C"

namespace {

// Shared by cgtp_onsite and the fixed-scratch entry point. fixed: the workspace is the
// caller's fixed buffer (never grown by the plan) and no stage events are recorded, so
// nothing is allocated.
int onsite_impl(cgtp_plan plan, int64_t n_nodes, const void *A, const void *B, const void *U_A,
                const void *U_B, const void *U_out_even, const void *U_out_odd, void *out_even,
                void *out_odd, void *workspace, size_t ws_bytes, void *stream, bool fixed)
{
    if (!plan) return fail(CGTP_ERR_ARG, "plan is NULL");
    if (n_nodes < 0) return fail(CGTP_ERR_ARG, "n_nodes < 0");
    if (n_nodes == 0) return CGTP_OK;
    if (!out_even && !out_odd) return fail(CGTP_ERR_ARG, "both outputs are NULL");
    if (!A || !B || !U_A || !U_B) return fail(CGTP_ERR_ARG, "NULL input");
    if ((out_even && !U_out_even) || (out_odd && !U_out_odd))
        return fail(CGTP_ERR_ARG, "NULL output projection");
    if (n_nodes * (int64_t)plan->R > 0x7fffffffLL)
        return fail(CGTP_ERR_UNSUPPORTED, "n_nodes * rank exceeds 2^31 - 1");
    int st = check_device(plan);
    if (st) return st;
    void *ws = nullptr;
    const size_t need = onsite_layout(plan, plan->R, n_nodes).total;
    if (fixed && (!workspace || ws_bytes < need))
        return fail(CGTP_ERR_WORKSPACE,
                    "%lld nodes need %zu bytes of scratch; the fixed scratch holds %zu",
                    (long long)n_nodes, need, workspace ? ws_bytes : (size_t)0);
    st = get_workspace(plan, need, workspace, ws_bytes, &ws);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (plan->dtype == CGTP_F64)
        return run_onsite<double>(plan, CGTP_OP_ONSITE, n_nodes, A, B, U_A, U_B, U_out_even,
                                  U_out_odd, out_even, out_odd, static_cast<char *>(ws), s,
                                  !fixed);
    return run_onsite<float>(plan, CGTP_OP_ONSITE, n_nodes, A, B, U_A, U_B, U_out_even, U_out_odd,
                             out_even, out_odd, static_cast<char *>(ws), s, !fixed);
}

}  // namespace

namespace cgtp {

int onsite_fixed_scratch(cgtp_plan plan, int64_t n_nodes, const void *A, const void *B,
                         const void *U_A, const void *U_B, const void *U_out_even,
                         const void *U_out_odd, void *out_even, void *out_odd, void *scratch,
                         size_t scratch_bytes, void *stream)
{
    return onsite_impl(plan, n_nodes, A, B, U_A, U_B, U_out_even, U_out_odd, out_even, out_odd,
                       scratch, scratch_bytes, stream, true);
}

int report(int status, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return status;
}

void clear_error() { g_err[0] = 0; }

}  // namespace cgtp

extern "C" {

int cgtp_onsite(cgtp_plan plan, int64_t n_nodes, const void *A, const void *B, const void *U_A,
                const void *U_B, const void *U_out_even, const void *U_out_odd, void *out_even,
                void *out_odd, void *workspace, size_t ws_bytes, void *stream)
{
    g_err[0] = 0;
    return onsite_impl(plan, n_nodes, A, B, U_A, U_B, U_out_even, U_out_odd, out_even, out_odd,
                       workspace, ws_bytes, stream, false);
}

namespace {

// Shared by the one- and two-slot entry points (node_flip NULL for one slot).
int message_pass_impl(cgtp_plan plan, int64_t n_nodes, int64_t n_edges, const int32_t *row_ptr,
                      const int32_t *col, const void *edge_unit, const void *edge_radial,
                      const void *node_feat, const void *node_flip, const void *U_E,
                      const void *U_I, const void *U_out_even, const void *U_out_odd,
                      void *out_even, void *out_odd, void *workspace, size_t ws_bytes,
                      void *stream)
{
    g_err[0] = 0;
    if (!plan) return fail(CGTP_ERR_ARG, "plan is NULL");
    if (n_nodes < 0 || n_edges < 0) return fail(CGTP_ERR_ARG, "negative size");
    if (n_edges >= 0x7fffffffLL) return fail(CGTP_ERR_ARG, "n_edges must be below 2^31 - 1");
    if (n_nodes == 0) {
        if (n_edges != 0) return fail(CGTP_ERR_ARG, "edges without nodes");
        return CGTP_OK;
    }
    if (!out_even && !out_odd) return fail(CGTP_ERR_ARG, "both outputs are NULL");
    if (!row_ptr || !node_feat || !U_E || !U_I) return fail(CGTP_ERR_ARG, "NULL input");
    if (n_edges > 0 && (!col || !edge_unit || !edge_radial))
        return fail(CGTP_ERR_ARG, "NULL edge input");
    if ((out_even && !U_out_even) || (out_odd && !U_out_odd))
        return fail(CGTP_ERR_ARG, "NULL output projection");
    if (n_nodes * (int64_t)plan->R > 0x7fffffffLL)
        return fail(CGTP_ERR_UNSUPPORTED, "n_nodes * rank exceeds 2^31 - 1");
    const bool two = node_flip != nullptr;
    if (two && (plan->flags & CGTP_EDGE_SEPARATED))
        return fail(CGTP_ERR_UNSUPPORTED,
                    "two node slots are built for the zonal edge field, not CGTP_EDGE_SEPARATED");
    int st = check_device(plan);
    if (!st) st = check_order(plan, n_nodes);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (plan->flags & CGTP_VALIDATE_CSR) {
        st = validate_csr(n_nodes, n_edges, row_ptr, col, s);
        if (st) return st;
    }
    void *ws = nullptr;
    st = get_workspace(plan, mp_layout(plan, plan->R, n_nodes, n_edges, two).total, workspace,
                       ws_bytes, &ws);
    if (st) return st;
    const int op = two ? CGTP_OP_MESSAGE_PASS_TWO_SLOT : CGTP_OP_MESSAGE_PASS;
    if (plan->dtype == CGTP_F64)
        return run_mp<double>(plan, op, n_nodes, n_edges, row_ptr, col, edge_unit, edge_radial,
                              node_feat, node_flip, U_E, U_I, U_out_even, U_out_odd, out_even,
                              out_odd, static_cast<char *>(ws), s);
    return run_mp<float>(plan, op, n_nodes, n_edges, row_ptr, col, edge_unit, edge_radial,
                         node_feat, node_flip, U_E, U_I, U_out_even, U_out_odd, out_even, out_odd,
                         static_cast<char *>(ws), s);
}

}  // namespace

int cgtp_message_pass(cgtp_plan plan, int64_t n_nodes, int64_t n_edges, const int32_t *row_ptr,
                      const int32_t *col, const void *edge_unit, const void *edge_radial,
                      const void *node_feat, const void *U_E, const void *U_I,
                      const void *U_out_even, const void *U_out_odd, void *out_even, void *out_odd,
                      void *workspace, size_t ws_bytes, void *stream)
{
    return message_pass_impl(plan, n_nodes, n_edges, row_ptr, col, edge_unit, edge_radial,
                             node_feat, nullptr, U_E, U_I, U_out_even, U_out_odd, out_even,
                             out_odd, workspace, ws_bytes, stream);
}

int cgtp_message_pass_two_slot(cgtp_plan plan, int64_t n_nodes, int64_t n_edges,
                               const int32_t *row_ptr, const int32_t *col, const void *edge_unit,
                               const void *edge_radial, const void *node_feat,
                               const void *node_flip, const void *U_E, const void *U_I,
                               const void *U_out_even, const void *U_out_odd, void *out_even,
                               void *out_odd, void *workspace, size_t ws_bytes, void *stream)
{
    if (n_nodes > 0 && !node_flip) {
        g_err[0] = 0;
        return fail(CGTP_ERR_ARG, "NULL input (node_flip)");
    }
    return message_pass_impl(plan, n_nodes, n_edges, row_ptr, col, edge_unit, edge_radial,
                             node_feat, node_flip, U_E, U_I, U_out_even, U_out_odd, out_even,
                             out_odd, workspace, ws_bytes, stream);
}

int cgtp_workspace_bytes_general(cgtp_plan plan, int op, int64_t n_nodes, int64_t n_edges,
                                 int flips, int in_blocks, int out_blocks, size_t *bytes)
{
    if (!plan || !bytes) return fail(CGTP_ERR_ARG, "NULL argument");
    if (n_nodes < 0 || n_edges < 0) return fail(CGTP_ERR_ARG, "negative size");
    if (!valid_blocks(in_blocks, out_blocks) || (flips & ~3))
        return fail(CGTP_ERR_ARG, "in_blocks %d / out_blocks %d / flips %d invalid", in_blocks,
                    out_blocks, flips);
    if (op == CGTP_OP_ONSITE_GENERAL)
        *bytes = route_onsite(plan, n_nodes, flips & 1, flips & 2, in_blocks).ws;
    else if (op == CGTP_OP_MESSAGE_PASS_GENERAL)
        *bytes = route_mp(plan, n_nodes, n_edges, flips & 2, in_blocks, out_blocks).ws;
    else if (op == CGTP_OP_MESSAGE_PASS_FIELDS) {
        Groups G = make_groups(flips & 1, flips & 2, in_blocks, use_mfma_fields(plan));
        *bytes = mpf_layout(plan, G.n * plan->R, n_nodes, n_edges, G.split).total;
    }
    else return fail(CGTP_ERR_ARG, "unknown general op %d", op);
    return CGTP_OK;
}

int cgtp_onsite_general(cgtp_plan plan, int64_t n_nodes, const void *A, const void *A_flip,
                        const void *B, const void *B_flip, int in_blocks, const void *U_A,
                        const void *U_B, int out_blocks, const void *U_out_even,
                        const void *U_out_odd, void *out_even, void *out_odd, void *workspace,
                        size_t ws_bytes, void *stream)
{
    g_err[0] = 0;
    if (!plan) return fail(CGTP_ERR_ARG, "plan is NULL");
    if (n_nodes < 0) return fail(CGTP_ERR_ARG, "n_nodes < 0");
    if (!valid_blocks(in_blocks, out_blocks))
        return fail(CGTP_ERR_ARG, "in_blocks %d / out_blocks %d invalid", in_blocks, out_blocks);
    if (n_nodes == 0) return CGTP_OK;
    if (!out_even && !out_odd) return fail(CGTP_ERR_ARG, "both outputs are NULL");
    if (!A || !B || !U_A || !U_B) return fail(CGTP_ERR_ARG, "NULL input");
    if ((out_even && !U_out_even) || (out_odd && !U_out_odd))
        return fail(CGTP_ERR_ARG, "NULL output projection");
    GeneralRoute r = route_onsite(plan, n_nodes, A_flip != nullptr, B_flip != nullptr, in_blocks);
    const int Rg = r.fused ? plan->R : r.G.n * plan->R;
    if (n_nodes * (int64_t)Rg > 0x7fffffffLL)
        return fail(CGTP_ERR_UNSUPPORTED, "n_nodes * total rank exceeds 2^31 - 1");
    int st = check_device(plan);
    if (st) return st;
    void *ws = nullptr;
    st = get_workspace(plan, r.ws, workspace, ws_bytes, &ws);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    Factors f = resolve_factors(plan, in_blocks, U_A, U_B, out_blocks, U_out_even, U_out_odd);
    char *w = static_cast<char *>(ws);
    if (r.fused) {  // one slot each: out_even holds block 0 (Gaunt), out_odd block 3 (curl)
        if (plan->dtype == CGTP_F64)
            return run_onsite<double>(plan, CGTP_OP_ONSITE_GENERAL, n_nodes, A, B, U_A, U_B,
                                      f.out[0], f.out[3], out_even, out_odd, w, s);
        return run_onsite<float>(plan, CGTP_OP_ONSITE_GENERAL, n_nodes, A, B, U_A, U_B, f.out[0],
                                 f.out[3], out_even, out_odd, w, s);
    }
    const void *X1[2] = {A, A_flip}, *X2[2] = {B, B_flip};
    if (plan->dtype == CGTP_F64)
        return run_onsite_groups<double>(plan, r.G, n_nodes, X1, X2, f, out_even, out_odd, w, s);
    return run_onsite_groups<float>(plan, r.G, n_nodes, X1, X2, f, out_even, out_odd, w, s);
}

int cgtp_message_pass_general(cgtp_plan plan, int64_t n_nodes, int64_t n_edges,
                              const int32_t *row_ptr, const int32_t *col, const void *edge_unit,
                              const void *edge_radial, const void *node_feat,
                              const void *node_flip, int in_blocks, const void *U_E,
                              const void *U_I, int out_blocks, const void *U_out_even,
                              const void *U_out_odd, void *out_even, void *out_odd,
                              void *workspace, size_t ws_bytes, void *stream)
{
    g_err[0] = 0;
    if (!plan) return fail(CGTP_ERR_ARG, "plan is NULL");
    if (n_nodes < 0 || n_edges < 0) return fail(CGTP_ERR_ARG, "negative size");
    if (n_edges >= 0x7fffffffLL) return fail(CGTP_ERR_ARG, "n_edges must be below 2^31 - 1");
    if (!valid_blocks(in_blocks, out_blocks))
        return fail(CGTP_ERR_ARG, "in_blocks %d / out_blocks %d invalid", in_blocks, out_blocks);
    if (n_nodes == 0) {
        if (n_edges != 0) return fail(CGTP_ERR_ARG, "edges without nodes");
        return CGTP_OK;
    }
    if (!out_even && !out_odd) return fail(CGTP_ERR_ARG, "both outputs are NULL");
    if (!row_ptr || !node_feat || !U_E || !U_I) return fail(CGTP_ERR_ARG, "NULL input");
    if (n_edges > 0 && (!col || !edge_unit || !edge_radial))
        return fail(CGTP_ERR_ARG, "NULL edge input");
    if ((out_even && !U_out_even) || (out_odd && !U_out_odd))
        return fail(CGTP_ERR_ARG, "NULL output projection");
    const bool flip = node_flip != nullptr;
    GeneralRoute r = route_mp(plan, n_nodes, n_edges, flip, in_blocks, out_blocks);
    const int Rg = r.fused ? plan->R : r.G.n * plan->R;
    if (n_nodes * (int64_t)Rg > 0x7fffffffLL)
        return fail(CGTP_ERR_UNSUPPORTED, "n_nodes * total rank exceeds 2^31 - 1");
    int st = check_device(plan);
    if (!st) st = check_order(plan, n_nodes);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (plan->flags & CGTP_VALIDATE_CSR) {
        st = validate_csr(n_nodes, n_edges, row_ptr, col, s);
        if (st) return st;
    }
    void *ws = nullptr;
    st = get_workspace(plan, r.ws, workspace, ws_bytes, &ws);
    if (st) return st;
    Factors f = resolve_factors(plan, in_blocks, U_E, U_I, out_blocks, U_out_even, U_out_odd);
    char *w = static_cast<char *>(ws);
    if (r.fused) {  // out_even: blocks 0 (+ 2), out_odd: blocks 3 (+ 1), one weight set each
        if (plan->dtype == CGTP_F64)
            return run_mp<double>(plan, CGTP_OP_MESSAGE_PASS_GENERAL, n_nodes, n_edges, row_ptr,
                                  col, edge_unit, edge_radial, node_feat, node_flip, U_E, U_I,
                                  f.out[0], f.out[3], out_even, out_odd, w, s);
        return run_mp<float>(plan, CGTP_OP_MESSAGE_PASS_GENERAL, n_nodes, n_edges, row_ptr, col,
                             edge_unit, edge_radial, node_feat, node_flip, U_E, U_I, f.out[0],
                             f.out[3], out_even, out_odd, w, s);
    }
    const void *X2[2] = {node_feat, node_flip};
    if (plan->dtype == CGTP_F64)
        return run_mp_groups<double>(plan, r.G, n_nodes, n_edges, row_ptr, col, edge_unit,
                                     edge_radial, X2, f, out_even, out_odd, w, s);
    return run_mp_groups<float>(plan, r.G, n_nodes, n_edges, row_ptr, col, edge_unit, edge_radial,
                                X2, f, out_even, out_odd, w, s);
}

int cgtp_message_pass_fields(cgtp_plan plan, int64_t n_nodes, int64_t n_edges,
                             const int32_t *row_ptr, const int32_t *col, const void *edge_feat,
                             const void *edge_flip, const void *node_feat, const void *node_flip,
                             int in_blocks, const void *U_E, const void *U_I, int out_blocks,
                             const void *U_out_even, const void *U_out_odd, void *out_even,
                             void *out_odd, void *workspace, size_t ws_bytes, void *stream)
{
    g_err[0] = 0;
    if (!plan) return fail(CGTP_ERR_ARG, "plan is NULL");
    if (n_nodes < 0 || n_edges < 0) return fail(CGTP_ERR_ARG, "negative size");
    if (n_edges >= 0x7fffffffLL) return fail(CGTP_ERR_ARG, "n_edges must be below 2^31 - 1");
    if (!valid_blocks(in_blocks, out_blocks))
        return fail(CGTP_ERR_ARG, "in_blocks %d / out_blocks %d invalid", in_blocks, out_blocks);
    if (n_nodes == 0) {
        if (n_edges != 0) return fail(CGTP_ERR_ARG, "edges without nodes");
        return CGTP_OK;
    }
    if (!out_even && !out_odd) return fail(CGTP_ERR_ARG, "both outputs are NULL");
    if (!row_ptr || !node_feat || !U_E || !U_I) return fail(CGTP_ERR_ARG, "NULL input");
    if (n_edges > 0 && (!col || !edge_feat)) return fail(CGTP_ERR_ARG, "NULL edge input");
    if ((out_even && !U_out_even) || (out_odd && !U_out_odd))
        return fail(CGTP_ERR_ARG, "NULL output projection");
    Groups G = make_groups(edge_flip != nullptr, node_flip != nullptr, in_blocks,
                           use_mfma_fields(plan));
    const int Rg = G.n * plan->R;
    if ((n_nodes > n_edges ? n_nodes : n_edges) * (int64_t)Rg > 0x7fffffffLL)
        return fail(CGTP_ERR_UNSUPPORTED, "rows * total rank exceeds 2^31 - 1");
    int st = check_device(plan);
    if (!st) st = check_order(plan, n_nodes);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (plan->flags & CGTP_VALIDATE_CSR) {
        st = validate_csr(n_nodes, n_edges, row_ptr, col, s);
        if (st) return st;
    }
    void *ws = nullptr;
    st = get_workspace(plan, mpf_layout(plan, Rg, n_nodes, n_edges, G.split).total, workspace,
                       ws_bytes, &ws);
    if (st) return st;
    Factors f = resolve_factors(plan, in_blocks, U_E, U_I, out_blocks, U_out_even, U_out_odd);
    const void *X1[2] = {edge_feat, edge_flip}, *X2[2] = {node_feat, node_flip};
    char *w = static_cast<char *>(ws);
    if (plan->dtype == CGTP_F64)
        return run_mp_fields<double>(plan, G, n_nodes, n_edges, row_ptr, col, X1, X2, f, out_even,
                                     out_odd, w, s);
    return run_mp_fields<float>(plan, G, n_nodes, n_edges, row_ptr, col, X1, X2, f, out_even,
                                out_odd, w, s);
}

int cgtp_workspace_bytes_nbody(cgtp_plan plan, int64_t n_nodes, int nu, size_t *bytes)
{
    if (!plan || !bytes) return fail(CGTP_ERR_ARG, "NULL argument");
    if (n_nodes < 0) return fail(CGTP_ERR_ARG, "negative size");
    if (nu < 1 || nu > CGTP_MAX_NU) return fail(CGTP_ERR_ARG, "nu %d outside [1, %d]", nu, CGTP_MAX_NU);
    *bytes = nbody_layout(plan, n_nodes, nu).total;
    return CGTP_OK;
}

int cgtp_onsite_nbody(cgtp_plan plan, int64_t n_nodes, int nu, const void *const *X,
                      const void *const *U, const void *U_out, void *out, void *workspace,
                      size_t ws_bytes, void *stream)
{
    g_err[0] = 0;
    if (!plan) return fail(CGTP_ERR_ARG, "plan is NULL");
    if (n_nodes < 0) return fail(CGTP_ERR_ARG, "n_nodes < 0");
    if (nu < 1 || nu > CGTP_MAX_NU) return fail(CGTP_ERR_ARG, "nu %d outside [1, %d]", nu, CGTP_MAX_NU);
    int Umin, Vmin;
    nbody_min_grid(plan->d.lmax, nu, &Umin, &Vmin);
    if (plan->d.U < Umin || plan->d.V < Vmin)
        return fail(CGTP_ERR_ARG,
                    "grid %d x %d too coarse for a %d-fold product at lmax %d: create the plan "
                    "with n_theta >= %d and n_phi >= %d",
                    plan->d.U, plan->d.V, nu, plan->d.lmax, Umin, Vmin);
    if (n_nodes == 0) return CGTP_OK;
    if (!X || !U || !U_out || !out) return fail(CGTP_ERR_ARG, "NULL argument");
    for (int t = 0; t < nu; ++t)
        if (!X[t] || !U[t]) return fail(CGTP_ERR_ARG, "NULL operand %d", t);
    if (n_nodes * (int64_t)plan->R > 0x7fffffffLL)
        return fail(CGTP_ERR_UNSUPPORTED, "n_nodes * rank exceeds 2^31 - 1");
    int st = check_device(plan);
    if (st) return st;
    void *ws = nullptr;
    st = get_workspace(plan, nbody_layout(plan, n_nodes, nu).total, workspace, ws_bytes, &ws);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    char *w = static_cast<char *>(ws);
    if (plan->dtype == CGTP_F64) return run_nbody<double>(plan, n_nodes, nu, X, U, U_out, out, w, s);
    return run_nbody<float>(plan, n_nodes, nu, X, U, U_out, out, w, s);
}

int cgtp_gather_probe(cgtp_plan plan, int64_t n_nodes, int64_t n_edges, const int32_t *row_ptr,
                      const int32_t *col, const void *fields, size_t fields_bytes, void *sink,
                      void *stream)
{
    g_err[0] = 0;
    if (!plan) return fail(CGTP_ERR_ARG, "plan is NULL");
    if (n_nodes < 0 || n_edges < 0 || n_edges >= 0x7fffffffLL)
        return fail(CGTP_ERR_ARG, "bad sizes");
    // the receiver of cgtp_message_pass on this plan: the MFMA one in its values-only form on
    // the plain sender layout, or the per-thread zonal one
    const bool mfma = use_mfma_receiver(plan, plan->R);
    const bool mfma_plain = mfma && mfma_values_only(plan, plan->R, false) && !sf_chunked(plan, plan->R);
    if (plan->dtype != CGTP_F32 || (plan->flags & CGTP_EDGE_SEPARATED) || (mfma && !mfma_plain) ||
        (!mfma && plan->d.UV > 1024))
        return fail(CGTP_ERR_UNSUPPORTED,
                    "the probe replays the fp32 message-passing receiver in its values-only form "
                    "(MFMA below lmax %d on the default grid, else per-thread on grids of at "
                    "most 1024 points)", cgtp::kMfmaRecvMinL);
    if (n_nodes == 0) return CGTP_OK;
    if (!row_ptr || !fields || !sink || (n_edges > 0 && !col))
        return fail(CGTP_ERR_ARG, "NULL argument");
    const size_t need = sizeof(float) * (size_t)n_nodes * plan->R * 3 * plan->d.UVs;
    if (fields_bytes < need)
        return fail(CGTP_ERR_ARG, "fields buffer of %zu bytes, %zu needed", fields_bytes, need);
    int st = check_device(plan);
    if (!st) st = check_order(plan, n_nodes);
    if (st) return st;
    hipError_t e =
        mfma_plain ? cgtp::launch_gather_probe_mfma(plan->d, n_nodes, plan->R, row_ptr, col,
                                                    plan->order,
                                                    static_cast<const float *>(fields),
                                                    static_cast<float *>(sink),
                                                    static_cast<hipStream_t>(stream))
                   : cgtp::launch_gather_probe(plan->d, n_nodes, plan->R, row_ptr, col,
                                               plan->order, static_cast<const float *>(fields),
                                               static_cast<float *>(sink),
                                               static_cast<hipStream_t>(stream));
    return e == hipSuccess ? CGTP_OK : hip_fail(e, "gather probe");
}

int cgtp_plan_set_receiver_order(cgtp_plan plan, int64_t n_nodes, const int32_t *order)
{
    g_err[0] = 0;
    if (!plan) return fail(CGTP_ERR_ARG, "plan is NULL");
    if (n_nodes < 0 || n_nodes >= 0x7fffffffLL) return fail(CGTP_ERR_ARG, "bad n_nodes");
    int st = check_device(plan);
    if (st) return st;
    if (!order || n_nodes == 0) {  // back to the identity
        if (plan->order) {
            hipError_t e = hipDeviceSynchronize();  // calls in flight may still read it
            (void)hipFree(plan->order);
            plan->order = nullptr;
            plan->order_n = 0;
            if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
        }
        return CGTP_OK;
    }
    std::vector<unsigned char> seen((size_t)n_nodes, 0);
    for (int64_t k = 0; k < n_nodes; ++k) {
        const int32_t v = order[k];
        if (v < 0 || v >= n_nodes || seen[(size_t)v])
            return fail(CGTP_ERR_ARG, "order is not a permutation of the %lld nodes (order[%lld] = %d)",
                        (long long)n_nodes, (long long)k, v);
        seen[(size_t)v] = 1;
    }
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    if (plan->order) {
        (void)hipFree(plan->order);
        plan->order = nullptr;
        plan->order_n = 0;
    }
    int32_t *dev = nullptr;
    e = hipMalloc(&dev, sizeof(int32_t) * (size_t)n_nodes);
    if (e != hipSuccess) return hip_fail(e, "hipMalloc(receiver order)");
    e = hipMemcpy(dev, order, sizeof(int32_t) * (size_t)n_nodes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(dev);
        return hip_fail(e, "hipMemcpy(receiver order)");
    }
    plan->order = dev;
    plan->order_n = n_nodes;
    return CGTP_OK;
}

int cgtp_destroy(cgtp_plan plan)
{
    if (!plan) return CGTP_OK;
    hipError_t e = hipDeviceSynchronize();
    if (plan->own_ws) (void)hipFree(plan->own_ws);
    if (plan->tables) (void)hipFree(plan->tables);
    if (plan->order) (void)hipFree(plan->order);
    for (EventSet &es : plan->timers)
        for (int i = 0; i <= kMaxStages; ++i) (void)hipEventDestroy(es.ev[i]);
    delete plan;
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    return CGTP_OK;
}

int cgtp_stage_times(cgtp_plan plan, int op, double *ms, int cap, int *n_stages, int *n_calls)
{
    if (!plan || !ms || !n_stages || !n_calls) return fail(CGTP_ERR_ARG, "NULL argument");
    if (!(plan->flags & CGTP_TIME_STAGES))
        return fail(CGTP_ERR_ARG, "plan was created without CGTP_TIME_STAGES");
    int ns;
    if (op == CGTP_OP_ONSITE_NBODY || op == CGTP_OP_ONSITE) ns = 3;
    else if (op == CGTP_OP_ONSITE_GENERAL) ns = 5;
    else if (op == CGTP_OP_MESSAGE_PASS || op == CGTP_OP_MESSAGE_PASS_TWO_SLOT ||
             op == CGTP_OP_MESSAGE_PASS_GENERAL || op == CGTP_OP_MESSAGE_PASS_FIELDS)
        ns = 7;
    else return fail(CGTP_ERR_ARG, "unknown op %d", op);
    int status = drain_timers(plan);
    for (int k = 0; k < ns && k < cap; ++k) ms[k] = plan->stage_acc[op][k];
    *n_stages = ns;
    *n_calls = plan->stage_calls[op];
    for (int k = 0; k < kMaxStages; ++k) plan->stage_acc[op][k] = 0.0;
    plan->stage_calls[op] = 0;
    return status;
}

const char *cgtp_status_string(int status)
{
    switch (status) {
    case CGTP_OK: return "ok";
    case CGTP_ERR_ARG: return "invalid argument";
    case CGTP_ERR_WORKSPACE: return "workspace too small";
    case CGTP_ERR_CSR: return "invalid CSR neighbour list";
    case CGTP_ERR_HIP: return "HIP runtime error";
    case CGTP_ERR_UNSUPPORTED: return "unsupported size";
    default: return "unknown status";
    }
}

const char *cgtp_last_error(void) { return g_err; }

int cgtp_host_tables(int lmax, int n_theta, int n_phi, double *x, double *w, double *p, double *dp,
                     double *q)
{
    int U, V;
    if (n_theta < 0 || n_phi < 0 || !cgtp::resolve_grid(lmax, n_theta, n_phi, &U, &V))
        return fail(CGTP_ERR_ARG, "invalid lmax / grid");
    std::vector<double> xs(U), ws(U);
    cgtp::gauss_legendre(U, xs.data(), ws.data());
    if (x) std::memcpy(x, xs.data(), sizeof(double) * U);
    if (w) std::memcpy(w, ws.data(), sizeof(double) * U);
    const size_t P = (size_t)(lmax + 1) * (lmax + 2) / 2;
    std::vector<double> pp(U * P), dd(U * P);
    cgtp::legendre_tables(lmax, U, xs.data(), pp.data(), dd.data());
    if (p) std::memcpy(p, pp.data(), sizeof(double) * U * P);
    if (dp) std::memcpy(dp, dd.data(), sizeof(double) * U * P);
    if (q) cgtp::fourier_table(lmax, V, q);
    return CGTP_OK;
}

}  // extern "C"
