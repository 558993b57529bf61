// C-ABI entry points: plan lifetime, argument validation, workspace layout and
// the stream-ordered launch sequences of the on-site and message-passing paths.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "internal.h"

namespace {
constexpr int kMaxStages = 6;
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
    double stage_acc[3][kMaxStages];  // drained sums per op (onsite, message pass, two-slot)
    int stage_calls[3];
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
    size_t hf = 0, sff = 0;  // offsets of the flipped slot from HI and from SF (two slots)
};

// Receiver on MFMA: fp32, zonal edge field, R a multiple of 16, lmax high enough that the
// per-thread recurrence sums would make the SIMT receiver compute-bound.
bool use_mfma_receiver(const cgtp_plan_s *p)
{
    return p->dtype == CGTP_F32 && !(p->flags & CGTP_EDGE_SEPARATED) &&
           p->d.lmax >= cgtp::kMfmaRecvMinL && cgtp::receiver_mfma_supported(p->d, p->R);
}

// The MFMA receiver reads the sender fields in 64-point chunks when the MFMA sender writes
// them (fp32, default grid).
bool sf_chunked(const cgtp_plan_s *p)
{
    return use_mfma_receiver(p) && cgtp::sender_mfma_supported(p->d);
}

// On-site workspace: HA, HB, Ta, Tb, each [N][R][K].
Layout onsite_layout(const cgtp_plan_s *p, int64_t N)
{
    size_t es = p->dtype == CGTP_F64 ? 8 : 4;
    size_t blk = align256(es * (size_t)N * p->R * p->d.K);
    Layout l{};
    for (int i = 0; i < 4; ++i) l.off[i] = i * blk;
    l.total = 4 * blk;
    return l;
}

// Message-passing workspace: HI [N][R][K], SF [N][R][3][UVs], Rt [E][L][R], Ta, Tb [N][R][K],
// and, for the MFMA receiver, the summed grid fields S [N][R][2][UVs]. With two node slots,
// HI and SF hold the natural slot followed by the flipped one.
Layout mp_layout(const cgtp_plan_s *p, int64_t N, int64_t E, bool two = false)
{
    size_t es = p->dtype == CGTP_F64 ? 8 : 4;
    const size_t slots = two ? 2 : 1;
    size_t h = align256(es * (size_t)N * p->R * p->d.K);
    const size_t sf_pts = sf_chunked(p) ? (size_t)cgtp::sf_chunks(p->d) * cgtp::kSfChunk : p->d.UVs;
    size_t sf = align256(es * (size_t)N * p->R * 3 * sf_pts);
    size_t rt = align256(es * (size_t)E * p->R * p->d.L);
    size_t sg = use_mfma_receiver(p) ? align256(es * cgtp::receiver_mfma_ws_elems(p->d, N, p->R)) : 0;
    Layout l{};
    l.off[0] = 0;
    l.off[1] = slots * h;
    l.off[2] = slots * (h + sf);
    l.off[3] = slots * (h + sf) + rt;
    l.off[4] = slots * (h + sf) + rt + h;
    l.off[5] = slots * (h + sf) + rt + 2 * h;
    l.total = slots * (h + sf) + rt + 2 * h + sg;
    l.hf = h;
    l.sff = sf;
    return l;
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

template <typename T>
int run_onsite(cgtp_plan_s *p, int64_t N, const void *A, const void *B, const void *UA,
               const void *UB, const void *Uoe, const void *Uoo, void *oe, void *oo, char *ws,
               hipStream_t s)
{
    const cgtp::Dims &d = p->d;
    const int C = p->C, R = p->R;
    cgtp::Tabs<T> tb = cgtp::bind_tables<T>(d, p->tables);
    Layout lay = onsite_layout(p, N);
    T *HA = reinterpret_cast<T *>(ws + lay.off[0]);
    T *HB = reinterpret_cast<T *>(ws + lay.off[1]);
    T *Ta = reinterpret_cast<T *>(ws + lay.off[2]);
    T *Tb = reinterpret_cast<T *>(ws + lay.off[3]);
    const int64_t sl = (int64_t)C * R;
    StageRec rec;
    int st = rec.begin(p, CGTP_OP_ONSITE, 5, s);
    if (st) return st;
    hipError_t e;
    // Eq. struct-H for both operands (shared when the operands coincide)
    e = cgtp::launch_contract<T>(N, C, R, d.K, false, (const T *)UA, sl, R, 1, (const T *)A, HA,
                                 (int64_t)R * d.K, d.K, 1, nullptr, s);
    if (e != hipSuccess) return hip_fail(e, "contract A");
    rec.mark();
    const T *HBp = HA;
    if (!(A == B && UA == UB)) {
        e = cgtp::launch_contract<T>(N, C, R, d.K, false, (const T *)UB, sl, R, 1, (const T *)B,
                                     HB, (int64_t)R * d.K, d.K, 1, nullptr, s);
        if (e != hipSuccess) return hip_fail(e, "contract B");
        HBp = HB;
    }
    rec.mark();
    e = cgtp::launch_onsite_grid<T>(tb, N, R, HA, HBp, Ta, Tb, s);
    if (e != hipSuccess) return hip_fail(e, "onsite grid");
    rec.mark();
    // Eq. struct-phi: out[b][n][k] = sum_r Uout[l][n][r] T[b][r][k]
    if (oe) {
        e = cgtp::launch_contract<T>(N, R, C, d.K, false, (const T *)Uoe, sl, 1, R, Ta, (T *)oe,
                                     (int64_t)C * d.K, d.K, 1, nullptr, s);
        if (e != hipSuccess) return hip_fail(e, "project even");
    }
    rec.mark();
    if (oo) {
        e = cgtp::launch_contract<T>(N, R, C, d.K, false, (const T *)Uoo, sl, 1, R, Tb, (T *)oo,
                                     (int64_t)C * d.K, d.K, 1, nullptr, s);
        if (e != hipSuccess) return hip_fail(e, "project odd");
    }
    rec.mark();
    return CGTP_OK;
}

template <typename T>
int run_mp(cgtp_plan_s *p, int64_t N, int64_t E, const int32_t *row_ptr, const int32_t *col,
           const void *unit, const void *rad, const void *I, const void *If, const void *UE,
           const void *UI, const void *Uoe, const void *Uoo, void *oe, void *oo, char *ws,
           hipStream_t s)
{
    const cgtp::Dims &d = p->d;
    const int C = p->C, R = p->R;
    const bool separated = (p->flags & CGTP_EDGE_SEPARATED) != 0;
    const bool two = If != nullptr;
    cgtp::Tabs<T> tb = cgtp::bind_tables<T>(d, p->tables);
    Layout lay = mp_layout(p, N, E, two);
    T *HI = reinterpret_cast<T *>(ws + lay.off[0]);
    T *SF = reinterpret_cast<T *>(ws + lay.off[1]);
    T *Rt = reinterpret_cast<T *>(ws + lay.off[2]);
    T *Ta = reinterpret_cast<T *>(ws + lay.off[3]);
    T *Tb = reinterpret_cast<T *>(ws + lay.off[4]);
    T *HIf = two ? reinterpret_cast<T *>(ws + lay.off[0] + lay.hf) : nullptr;
    T *SFf = two ? reinterpret_cast<T *>(ws + lay.off[1] + lay.sff) : nullptr;
    const int64_t sl = (int64_t)C * R;
    StageRec rec;
    int st = rec.begin(p, two ? CGTP_OP_MESSAGE_PASS_TWO_SLOT : CGTP_OP_MESSAGE_PASS, 6, s);
    if (st) return st;
    hipError_t e;
    // Eq. msgpass-HI, then the node-side forward transforms (Eqs. msgpass-FI, msgpass-AI),
    // for each node slot
    for (int slot = 0; slot < (two ? 2 : 1); ++slot) {
        e = cgtp::launch_contract<T>(N, C, R, d.K, false, (const T *)UI, sl, R, 1,
                                     (const T *)(slot ? If : I), slot ? HIf : HI,
                                     (int64_t)R * d.K, d.K, 1, nullptr, s);
        if (e != hipSuccess) return hip_fail(e, "contract node features");
    }
    rec.mark();
    for (int slot = 0; slot < (two ? 2 : 1); ++slot) {
        T *h = slot ? HIf : HI, *sf = slot ? SFf : SF;
        if constexpr (sizeof(T) == 4) {
            if (sf_chunked(p))
                e = cgtp::launch_sender_mfma(tb, N, R, h, sf, true, s);
            else
                e = cgtp::launch_sender_fields<T>(tb, N, R, h, sf, s);
        } else {
            e = cgtp::launch_sender_fields<T>(tb, N, R, h, sf, s);
        }
        if (e != hipSuccess) return hip_fail(e, "sender fields");
    }
    rec.mark();
    // Eq. msgpass-tildeR into Rt [E][L][R] (the zonal form folds in the addition-theorem
    // weight (2l+1)/(4 pi))
    e = cgtp::launch_contract<T>(E, C, R, d.L, true, (const T *)UE, sl, R, 1, (const T *)rad, Rt,
                                 (int64_t)d.L * R, 1, R, separated ? nullptr : tb.cl, s);
    if (e != hipSuccess) return hip_fail(e, "contract edge radial");
    rec.mark();
    if constexpr (sizeof(T) == 4) {
        if (use_mfma_receiver(p)) {
            float *Sg = reinterpret_cast<float *>(ws + lay.off[5]);
            e = cgtp::launch_receiver_mfma(tb, N, R, row_ptr, col, (const float *)unit, Rt, SF,
                                           SFf, sf_chunked(p), Sg, Ta, Tb, s);
            if (e != hipSuccess) return hip_fail(e, "receiver (mfma)");
            rec.mark();
            goto projections;
        }
    }
    e = cgtp::launch_receiver<T>(tb, separated, N, R, row_ptr, col, (const T *)unit, Rt, SF, SFf,
                                 Ta, Tb, s);
    if (e != hipSuccess) return hip_fail(e, "receiver");
    rec.mark();
projections:
    if (oe) {
        e = cgtp::launch_contract<T>(N, R, C, d.K, false, (const T *)Uoe, sl, 1, R, Ta, (T *)oe,
                                     (int64_t)C * d.K, d.K, 1, nullptr, s);
        if (e != hipSuccess) return hip_fail(e, "project even");
    }
    rec.mark();
    if (oo) {
        e = cgtp::launch_contract<T>(N, R, C, d.K, false, (const T *)Uoo, sl, 1, R, Tb, (T *)oo,
                                     (int64_t)C * d.K, d.K, 1, nullptr, s);
        if (e != hipSuccess) return hip_fail(e, "project odd");
    }
    rec.mark();
    return CGTP_OK;
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
    if (max_lds_bytes(d, es) > 65536)
        return fail(CGTP_ERR_UNSUPPORTED, "grid %d x %d at lmax %d needs %zu B of LDS (> 64 KiB)",
                    U, V, desc->lmax, max_lds_bytes(d, es));
    if (d.UV > 11 * 256)
        return fail(CGTP_ERR_UNSUPPORTED, "grid of %d points exceeds 2816", d.UV);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
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
    if (op == CGTP_OP_ONSITE) *bytes = onsite_layout(plan, n_nodes).total;
    else if (op == CGTP_OP_MESSAGE_PASS) *bytes = mp_layout(plan, n_nodes, n_edges).total;
    else if (op == CGTP_OP_MESSAGE_PASS_TWO_SLOT)
        *bytes = mp_layout(plan, n_nodes, n_edges, true).total;
    else return fail(CGTP_ERR_ARG, "unknown op %d", op);
    return CGTP_OK;
}

int cgtp_onsite(cgtp_plan plan, int64_t n_nodes, const void *A, const void *B, const void *U_A,
                const void *U_B, const void *U_out_even, const void *U_out_odd, void *out_even,
                void *out_odd, void *workspace, size_t ws_bytes, void *stream)
{
    g_err[0] = 0;
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
    st = get_workspace(plan, onsite_layout(plan, n_nodes).total, workspace, ws_bytes, &ws);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (plan->dtype == CGTP_F64)
        return run_onsite<double>(plan, n_nodes, A, B, U_A, U_B, U_out_even, U_out_odd, out_even,
                                  out_odd, static_cast<char *>(ws), s);
    return run_onsite<float>(plan, n_nodes, A, B, U_A, U_B, U_out_even, U_out_odd, out_even,
                             out_odd, static_cast<char *>(ws), s);
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
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (plan->flags & CGTP_VALIDATE_CSR) {
        st = validate_csr(n_nodes, n_edges, row_ptr, col, s);
        if (st) return st;
    }
    void *ws = nullptr;
    st = get_workspace(plan, mp_layout(plan, n_nodes, n_edges, two).total, workspace, ws_bytes,
                       &ws);
    if (st) return st;
    if (plan->dtype == CGTP_F64)
        return run_mp<double>(plan, n_nodes, n_edges, row_ptr, col, edge_unit, edge_radial,
                              node_feat, node_flip, U_E, U_I, U_out_even, U_out_odd, out_even,
                              out_odd, static_cast<char *>(ws), s);
    return run_mp<float>(plan, n_nodes, n_edges, row_ptr, col, edge_unit, edge_radial, node_feat,
                         node_flip, U_E, U_I, U_out_even, U_out_odd, out_even, out_odd,
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

int cgtp_destroy(cgtp_plan plan)
{
    if (!plan) return CGTP_OK;
    hipError_t e = hipDeviceSynchronize();
    if (plan->own_ws) (void)hipFree(plan->own_ws);
    if (plan->tables) (void)hipFree(plan->tables);
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
    if (op == CGTP_OP_ONSITE) ns = 5;
    else if (op == CGTP_OP_MESSAGE_PASS || op == CGTP_OP_MESSAGE_PASS_TWO_SLOT) ns = 6;
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
