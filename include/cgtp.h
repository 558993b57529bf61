/*
 * cgtp.h - contracted Clebsch-Gordan tensor products on a structured
 * Gauss-Legendre x Fourier S^2 grid, for AMD Instinct MI355X (gfx950).
 *
 * Method: Bochkarev, Lysogorskiy, Drautz, "Fast contracted Clebsch-Gordan tensor
 * products for equivariant graph neural networks" (SCALE-CG). The library
 * evaluates, for CP-factorised channel mixing (Eq. cp-decomp),
 *
 *   on-site (Eq. phi-cg, natural-parity inputs):
 *     out_even = Category alpha (Gaunt product, l1+l2+l even), parity (-1)^l
 *     out_odd  = Category beta  (surface curl / spherical Poisson bracket
 *                {A,B} = r.(grad A x grad B), Eq. poisson-S2-x; l1+l2+l odd),
 *                parity -(-1)^l
 *   message passing (Eq. msgpass-parity-start, single natural-parity node slot,
 *   edge feature R_{n l1}(r_ji) Y_{l1 m1}(rhat_ji)):
 *     out_even/out_odd as above, summed over the neighbours j of receiver i.
 *
 * Both follow the structured pipelines (Sec. "Optimized computational
 * pipelines": Eqs. struct-H..struct-phi and msgpass-tildeR..cat-beta-phi) in
 * the real SH basis of App. C (Eq. realY, no Condon-Shortley phase):
 *   Y_{l,m>0} = sqrt2 Pt_l^m(cos th) cos(m ph), Y_{l,0} = Pt_l^0(cos th),
 *   Y_{l,m<0} = sqrt2 Pt_l^|m|(cos th) sin(|m| ph),
 *   Pt_l^m = sqrt((2l+1)/(4 pi) (l-m)!/(l+m)!) P_l^m.
 * With H1 = U_1^T X1, H2 = U_2^T X2 per degree (Eq. struct-H), the outputs are
 *   out_even[n][k] = sum_r U_out_even[l][n][r] sum_{k1,k2} G[k1,k2,k] H1[r][k1] H2[r][k2]
 *   out_odd [n][k] = sum_r U_out_odd [l][n][r] sum_{k1,k2} Q[k1,k2,k] H1[r][k1] H2[r][k2]
 * where G = int Y_k1 Y_k2 Y_k (Eq. gaunt) and Q = int {Y_k1, Y_k2} Y_k (Eq. Q-def)
 * are the real-basis Gaunt and curl tables. The prefactors f and kappa of
 * Eqs. msgpass-cp-alpha/beta are absorbed in the learnable factors, as the paper
 * parameterises them. The first operand of the bracket is A (on-site) or the
 * edge field (message passing); exchanging the operands negates out_odd.
 *
 * Conventions for every entry point:
 *  - All tensors are dense, row-major, contiguous, in device memory, of the
 *    plan's dtype (fp32, or fp64 for a CGTP_F64 plan), except the int32 CSR
 *    arrays. The flattened SH index is k = l*l + l + m, K = (lmax+1)^2 and
 *    L = lmax+1. Factor matrices are [L][C][R]: U[l][n][r] with n the radial
 *    channel and r the CP rank.
 *  - The caller owns every buffer it passes. Inputs are read only. Outputs are
 *    fully overwritten (no accumulation into existing contents).
 *  - Calls are asynchronous on `stream` (a hipStream_t cast to void*, NULL for
 *    the default stream): they return after enqueueing the kernels.
 *  - Every function returns CGTP_OK (0) or a negative status; none aborts or
 *    throws. cgtp_last_error() gives the detail of the last failure on the
 *    calling thread. A plan is not thread-safe: use it from one host thread and
 *    one stream at a time.
 */
#ifndef CGTP_H
#define CGTP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CGTP_MAX_LMAX 24

/* status codes */
#define CGTP_OK 0
#define CGTP_ERR_ARG (-1)         /* NULL pointer, negative size, bad descriptor */
#define CGTP_ERR_WORKSPACE (-2)   /* caller workspace smaller than cgtp_workspace_bytes() */
#define CGTP_ERR_CSR (-3)         /* CSR rejected (only checked with CGTP_VALIDATE_CSR) */
#define CGTP_ERR_HIP (-4)         /* HIP runtime / launch failure; see cgtp_last_error() */
#define CGTP_ERR_UNSUPPORTED (-5) /* valid request this build does not support */

/* dtypes */
#define CGTP_F32 0
#define CGTP_F64 1

/* plan flags */
#define CGTP_VALIDATE_CSR 1u   /* copy the CSR to the host and check it before launching */
#define CGTP_EDGE_SEPARATED 2u /* edge field by separated Legendre+Fourier synthesis
                                  (Eqs. msgpass-FE, msgpass-AE) instead of the zonal
                                  addition-theorem form; same values, more work */
#define CGTP_TIME_STAGES 4u    /* record HIP events between the kernel stages of every call
                                  (read with cgtp_stage_times) */

/* operations for cgtp_workspace_bytes and cgtp_stage_times */
#define CGTP_OP_ONSITE 0
#define CGTP_OP_MESSAGE_PASS 1
#define CGTP_OP_MESSAGE_PASS_TWO_SLOT 2
#define CGTP_OP_ONSITE_GENERAL 3        /* cgtp_workspace_bytes_general / cgtp_stage_times */
#define CGTP_OP_MESSAGE_PASS_GENERAL 4
#define CGTP_OP_MESSAGE_PASS_FIELDS 5
#define CGTP_OP_ONSITE_NBODY 6

#define CGTP_MAX_NU 8   /* largest body order of cgtp_onsite_nbody */

typedef struct cgtp_plan_s *cgtp_plan;

typedef struct {
    int lmax;       /* band limit, 0 <= lmax <= CGTP_MAX_LMAX */
    int channels;   /* C >= 1 radial channels (input = output, as in the paper's benchmark) */
    int rank;       /* R >= 1 CP rank */
    int n_theta;    /* Gauss-Legendre nodes; 0 => ceil((3 lmax + 2)/2); otherwise must be
                       >= ceil((3 lmax + 1)/2), the exactness bound of Sec. "Representation
                       using Structured Tensor-Product Grids" */
    int n_phi;      /* equispaced phi nodes phi_v = 2 pi v / n_phi; 0 => 3 lmax + 1; otherwise
                       must be >= 3 lmax + 1 */
    int dtype;      /* CGTP_F32 or CGTP_F64 */
    unsigned flags; /* CGTP_VALIDATE_CSR | CGTP_EDGE_SEPARATED | CGTP_TIME_STAGES */
} cgtp_desc;

/* Create a plan: validates the descriptor, builds the grid tables on the host in
 * fp64 (Gauss-Legendre nodes/weights, Pt_l^m and dPt_l^m/dx at the nodes, real
 * Fourier factors q_vm of Eq. realq) and uploads them in the plan's dtype to the
 * current HIP device. The plan owns these tables (and any workspace it grows
 * itself) until cgtp_destroy. Errors: CGTP_ERR_ARG (bad descriptor or NULL out),
 * CGTP_ERR_UNSUPPORTED (a size whose on-chip staging exceeds the kernel limits),
 * CGTP_ERR_HIP (allocation/copy failure). *plan is NULL on failure. */
int cgtp_plan_create(const cgtp_desc *desc, cgtp_plan *plan);

/* Grid actually used by the plan (after defaults). Any pointer may be NULL. */
int cgtp_plan_grid(cgtp_plan plan, int *n_theta, int *n_phi);

/* Bytes of device workspace an operation needs for n_nodes nodes and n_edges
 * edges (n_edges ignored for CGTP_OP_ONSITE). A caller workspace must start on a
 * 256-byte boundary (kernels store 16-byte vectors into it); a misaligned one is
 * rejected with CGTP_ERR_ARG. */
int cgtp_workspace_bytes(cgtp_plan plan, int op, int64_t n_nodes, int64_t n_edges,
                         size_t *bytes);

/* On-site contraction, Eq. phi-cg with Eq. cp-decomp, by the structured
 * pipeline (Eqs. struct-H, struct-F, struct-tildeA, struct-S, struct-Tmu,
 * struct-Tlm, struct-phi) plus the surface-curl channel (Eq. cat-beta-curl with
 * the neighbour sum dropped, as in the on-site paragraph of the same section).
 *   A, B                  [N][C][K] natural-parity coefficients; B may equal A.
 *   U_A, U_B              [L][C][R] first-operand and second-operand CP factors.
 *   U_out_even, U_out_odd [L][C][R] output projections (lambda); may alias.
 *   out_even, out_odd     [N][C][K]; either may be NULL to skip that channel (not both).
 *   workspace, ws_bytes   device scratch of at least cgtp_workspace_bytes(ONSITE);
 *                         workspace == NULL => the plan allocates and keeps one.
 * n_nodes == 0 is a no-op (pointers may then be NULL).
 * Errors: CGTP_ERR_ARG, CGTP_ERR_WORKSPACE, CGTP_ERR_HIP. */
int cgtp_onsite(cgtp_plan plan, int64_t n_nodes, const void *A, const void *B,
                const void *U_A, const void *U_B, const void *U_out_even,
                const void *U_out_odd, void *out_even, void *out_odd, void *workspace,
                size_t ws_bytes, void *stream);

/* Size in bytes of the fixed device scratch of cgtp_onsite_noalloc (64 MiB). */
#define CGTP_NOALLOC_SCRATCH_BYTES 67108864u

/* cgtp_onsite for callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc. Same arguments, results and errors as
 * cgtp_onsite, except that there is no workspace argument: the workspace is a fixed array of
 * CGTP_NOALLOC_SCRATCH_BYTES in device memory, one per GPU, resolved by cgtp_plan_create on
 * the plan's device (the first plan on a device sets it up) and held until the process ends.
 * The call allocates nothing (no hipMalloc/hipFree, no events: stage times are not recorded
 * for it). A call whose workspace, cgtp_workspace_bytes(CGTP_OP_ONSITE, n_nodes), exceeds
 * the scratch returns CGTP_ERR_WORKSPACE before anything is enqueued. Every call on one GPU
 * shares that GPU's scratch: calls that may overlap on one GPU (several host threads, or
 * several streams without an ordering between them) race and must be serialised by the
 * caller. Nothing in the scratch needs to start at zero; it keeps the last call's contents. */
int cgtp_onsite_noalloc(cgtp_plan plan, int64_t n_nodes, const void *A, const void *B,
                        const void *U_A, const void *U_B, const void *U_out_even,
                        const void *U_out_odd, void *out_even, void *out_odd, void *stream);

/* Message passing, Eq. msgpass-parity-start, by the parity-aware pipeline
 * (Eqs. msgpass-tildeR, msgpass-HI, msgpass-FI, msgpass-AI, msgpass-S,
 * cat-beta-curl, msgpass-Tmu, msgpass-Tlm, cat-alpha-phi, cat-beta-phi) for a
 * single natural-parity node slot, where Case A feeds out_even and Case B
 * feeds out_odd (Table 1).
 *   row_ptr [N+1], col [E]  int32 CSR by receiver i: edges e in [row_ptr[i],
 *                           row_ptr[i+1]) carry messages from sender j = col[e] to i.
 *   edge_unit   [E][3]      direction of r_ji = r_j - r_i (renormalised; must be non-zero).
 *   edge_radial [E][C][L]   radial features R_{n l1}(|r_ji|).
 *   node_feat   [N][C][K]   sender features I_j (natural parity).
 *   U_E, U_I                [L][C][R] CP factors of the edge and node operands.
 *   U_out_even, U_out_odd   [L][C][R] output projections; may alias.
 *   out_even, out_odd       [N][C][K]; either may be NULL (not both). Receivers
 *                           with no edges get zeros.
 * n_nodes == 0 (with n_edges == 0) is a no-op; with n_edges == 0 the edge pointers
 * may be NULL. Preconditions (checked only with CGTP_VALIDATE_CSR): row_ptr[0] = 0,
 * non-decreasing, row_ptr[N] = E, 0 <= col[e] < N; E < 2^31.
 * Errors: CGTP_ERR_ARG, CGTP_ERR_WORKSPACE, CGTP_ERR_CSR, CGTP_ERR_HIP. */
int cgtp_message_pass(cgtp_plan plan, int64_t n_nodes, int64_t n_edges,
                      const int32_t *row_ptr, const int32_t *col, const void *edge_unit,
                      const void *edge_radial, const void *node_feat, const void *U_E,
                      const void *U_I, const void *U_out_even, const void *U_out_odd,
                      void *out_even, void *out_odd, void *workspace, size_t ws_bytes,
                      void *stream);

/* Message passing with both node parity slots (Table 1, Cases A-D; Eqs.
 * cat-alpha-slot and cat-beta-slot): each sender carries a natural-parity slot
 * node_feat (parity (-1)^l2) and a parity-flipped slot node_flip (parity -(-1)^l2),
 * contracted with the same factors U_I. The edge feature R Y has natural parity,
 * so by the parity rule p = p1 p2 the outputs of degree l are
 *   out_even (parity (-1)^l)  = Gaunt(edge, node_feat) + curl(edge, node_flip)
 *   out_odd  (parity -(-1)^l) = curl(edge, node_feat)  + Gaunt(edge, node_flip)
 * (Cases A and D feed out_even, Cases B and C out_odd), each projected with its own
 * factors U_out_even / U_out_odd. Arguments are those of cgtp_message_pass plus
 *   node_flip [N][C][K]      sender features in the parity-flipped slot.
 * The workspace is cgtp_workspace_bytes(CGTP_OP_MESSAGE_PASS_TWO_SLOT). With
 * node_flip all zero the result equals cgtp_message_pass on node_feat.
 * Errors: those of cgtp_message_pass; CGTP_ERR_UNSUPPORTED for a plan created
 * with CGTP_EDGE_SEPARATED. */
int cgtp_message_pass_two_slot(cgtp_plan plan, int64_t n_nodes, int64_t n_edges,
                               const int32_t *row_ptr, const int32_t *col, const void *edge_unit,
                               const void *edge_radial, const void *node_feat,
                               const void *node_flip, const void *U_E, const void *U_I,
                               const void *U_out_even, const void *U_out_odd, void *out_even,
                               void *out_odd, void *workspace, size_t ws_bytes, void *stream);

/* General parameterization (Eqs. msgpass-cp-alpha and msgpass-cp-beta; Table 1; the
 * on-site contraction with parity-labelled inputs). Each coupling category (Gaunt,
 * Category alpha; surface curl, Category beta) and each output parity sector (out_even,
 * parity (-1)^l; out_odd, parity -(-1)^l) has its own CP input factors and output weights:
 * block b = 2 * category + sector (0 Gaunt->even, 1 Gaunt->odd, 2 curl->even,
 * 3 curl->odd). An operand may carry, besides its natural-parity slot (parity (-1)^l), a
 * parity-flipped slot (parity -(-1)^l). By p = p1 p2 a slot pair of equal relative parity
 * sends its Gaunt coupling to out_even and its curl coupling to out_odd; a mixed pair the
 * other way round. Every pair is contracted with the factors of the block it feeds:
 *   out_s = sum_{cat} sum_r Uout[cat, s][l][n][r] T_{2 cat + s}[r][k],
 *   T_b   = sum over the slot pairs (s1, s2) routed to b of the block-b coupling of
 *           U1[b]^T X1[s1] and U2[b]^T X2[s2] (Gaunt table G or curl table Q).
 * Factor layouts: in_blocks = 1: U [L][C][R] shared by every block; 2: U [2][L][C][R]
 * (Gaunt, curl); 4: U [4][L][C][R] indexed by b. out_blocks = 1: U_out_even and U_out_odd
 * [L][C][R] serve both categories; 2: each is [2][L][C][R] (Gaunt, curl).
 * With in_blocks = 1, out_blocks = 1 and no flipped slots these are cgtp_onsite /
 * cgtp_message_pass. Other cases stack one rank group per (slot pair, factor block) and
 * run the same kernels at a multiple of the plan's rank (at most 8x on-site, 4x for
 * message passing), so the workspace grows accordingly: query it with
 * cgtp_workspace_bytes_general. Preconditions, ownership, streams and errors are those of
 * cgtp_onsite / cgtp_message_pass; CGTP_ERR_UNSUPPORTED also when n_nodes times the
 * stacked rank exceeds 2^31 - 1. */

/* Workspace of a general call. op: CGTP_OP_ONSITE_GENERAL, CGTP_OP_MESSAGE_PASS_GENERAL or
 * CGTP_OP_MESSAGE_PASS_FIELDS; flips: bit 0 set when the first operand (on-site A, or the
 * edge field of cgtp_message_pass_fields) has a flipped slot, bit 1 when the second operand
 * (on-site B, or the node feature) has one; in_blocks, out_blocks as in the calls. */
int cgtp_workspace_bytes_general(cgtp_plan plan, int op, int64_t n_nodes, int64_t n_edges,
                                 int flips, int in_blocks, int out_blocks, size_t *bytes);

/* On-site contraction with general parity.
 *   A, B            [N][C][K] natural-parity slots; A_flip, B_flip [N][C][K] or NULL.
 *   U_A, U_B        input factors, in_blocks blocks of [L][C][R].
 *   U_out_even, U_out_odd  output weights, out_blocks blocks of [L][C][R] each.
 *   out_even, out_odd      [N][C][K]; either may be NULL (not both). */
int cgtp_onsite_general(cgtp_plan plan, int64_t n_nodes, const void *A, const void *A_flip,
                        const void *B, const void *B_flip, int in_blocks, const void *U_A,
                        const void *U_B, int out_blocks, const void *U_out_even,
                        const void *U_out_odd, void *out_even, void *out_odd, void *workspace,
                        size_t ws_bytes, void *stream);

/* Message passing with general parity: the edge feature R Y is the first operand (natural
 * parity only), the node feature the second (node_flip: its flipped slot, or NULL).
 *   U_E, U_I        input factors of the edge radial and node operands, in_blocks blocks.
 * Other arguments as in cgtp_message_pass; U_out_* as in cgtp_onsite_general. */
int cgtp_message_pass_general(cgtp_plan plan, int64_t n_nodes, int64_t n_edges,
                              const int32_t *row_ptr, const int32_t *col, const void *edge_unit,
                              const void *edge_radial, const void *node_feat,
                              const void *node_flip, int in_blocks, const void *U_E,
                              const void *U_I, int out_blocks, const void *U_out_even,
                              const void *U_out_odd, void *out_even, void *out_odd,
                              void *workspace, size_t ws_bytes, void *stream);

/* Message passing with two parity-bearing fields (Eq. twoparity-phi): the edge operand is a
 * general per-edge feature with its own parity slots (a message that has gathered parity
 * content in earlier layers) instead of R Y. Its channel contraction runs per edge (the
 * analogue of Eq. msgpass-HI) and its grid fields come from the full Legendre and Fourier
 * syntheses, so the zonal form does not apply. Every (edge slot, node slot) pair is routed
 * to the factor blocks exactly as the on-site slot pairs of cgtp_onsite_general:
 *   out_s = sum_{cat} sum_r Uout[cat, s] T_{2 cat + s},  T_b = sum over the edges
 *           (j -> i) and the slot pairs routed to b of the block-b coupling of
 *           U_E[b]^T I^(E)_e[s1] and U_I[b]^T I^(N)_j[s2].
 *   edge_feat [E][C][K]   natural-parity slot of the edge field (edge e in CSR order);
 *   edge_flip [E][C][K]   its parity-flipped slot, or NULL;
 *   node_feat, node_flip  [N][C][K] node field slots (node_flip may be NULL);
 *   U_E, U_I              input factors of the edge and node fields, in_blocks blocks;
 *   U_out_even, U_out_odd output weights, out_blocks blocks each (cgtp_onsite_general).
 * Rank groups are stacked as in cgtp_onsite_general (up to 8x the plan's rank); query the
 * workspace with cgtp_workspace_bytes_general(CGTP_OP_MESSAGE_PASS_FIELDS). Other
 * arguments, preconditions and errors as in cgtp_message_pass; CGTP_ERR_UNSUPPORTED also
 * when the per-point receiver (fp64, or fp32 on a grid other than the default) meets a grid
 * of more than 2048 points or LDS staging beyond what a workgroup of the device holds (160 KiB
 * on MI355X; fp64 at the highest degrees). */
int cgtp_message_pass_fields(cgtp_plan plan, int64_t n_nodes, int64_t n_edges,
                             const int32_t *row_ptr, const int32_t *col, const void *edge_feat,
                             const void *edge_flip, const void *node_feat, const void *node_flip,
                             int in_blocks, const void *U_E, const void *U_I, int out_blocks,
                             const void *U_out_even, const void *U_out_odd, void *out_even,
                             void *out_odd, void *workspace, size_t ws_bytes, void *stream);

/* nu-body on-site product: the grid pointwise product extended to nu operands, followed by
 * a single inverse transform (the ACE-style higher-body-order extension the paper sketches
 * after its comparison with other algorithms; nu = 2 is the Gaunt part of Eq. phi-cg):
 *   H_t[r][k] = sum_n U[t][l][n][r] X[t][n][k],   t = 0 .. nu-1   (Eq. struct-H)
 *   out[n][k] = sum_r U_out[l][n][r] int Y_k prod_t (sum_k' H_t[r][k'] Y_k') dOmega.
 * With natural-parity inputs the output has natural parity (only Gaunt couplings).
 *   nu         1 .. CGTP_MAX_NU;
 *   X, U       host arrays of nu device pointers: X[t] [N][C][K], U[t] [L][C][R]; entries may
 *              repeat (an operand with the same pointer and factors is contracted once);
 *   U_out      [L][C][R]; out [N][C][K] (overwritten).
 * Exactness needs a finer grid than the bilinear product: the plan must have been created
 * with n_theta >= ((nu + 1) lmax + 2) / 2 (integer division) and n_phi >= (nu + 1) lmax + 1
 * (CGTP_ERR_ARG otherwise, with the sizes in cgtp_last_error). The workspace is
 * cgtp_workspace_bytes_nbody. n_nodes == 0 is a no-op. Errors: CGTP_ERR_ARG,
 * CGTP_ERR_WORKSPACE, CGTP_ERR_UNSUPPORTED (LDS staging beyond a workgroup's), CGTP_ERR_HIP.
 * Stages for cgtp_stage_times (CGTP_OP_ONSITE_NBODY): 0 contract operands, 1 grid product
 * and analysis, 2 project. */
int cgtp_workspace_bytes_nbody(cgtp_plan plan, int64_t n_nodes, int nu, size_t *bytes);
int cgtp_onsite_nbody(cgtp_plan plan, int64_t n_nodes, int nu, const void *const *X,
                      const void *const *U, const void *U_out, void *out, void *workspace,
                      size_t ws_bytes, void *stream);

/* Per-stage GPU time of the calls made since the previous cgtp_stage_times on
 * this plan (plan created with CGTP_TIME_STAGES), in the spirit of the paper's
 * per-step breakdown (App. D, Table 4). Waits for the recorded events, writes the
 * summed milliseconds of each stage of `op` to ms[0 .. *n_stages) (at most cap
 * entries) and the number of calls to *n_calls, then resets the accumulation.
 * Stages of CGTP_OP_ONSITE: 0 contract both operands, 1 grid product+curl and
 * analysis, 2 project both output slots. Stages of CGTP_OP_MESSAGE_PASS:
 * 0 contract node features, 1 sender grid fields, 2 contract edge radial,
 * 3 receiver pass (edge synthesis, products, neighbour sum), 4 analysis of the summed grid
 * fields (0 where the receiver runs it itself: fp64, grids off the default one),
 * 5 project even, 6 project odd. CGTP_OP_MESSAGE_PASS_TWO_SLOT has the same seven
 * stages, each covering both node slots; CGTP_OP_ONSITE_GENERAL: 0 contract first
 * operand, 1 contract second operand, 2 grid product+curl and analysis, 3 project even,
 * 4 project odd; CGTP_OP_MESSAGE_PASS_GENERAL those of CGTP_OP_MESSAGE_PASS; both cover
 * every rank group; CGTP_OP_MESSAGE_PASS_FIELDS: 0 contract node features, 1 sender grid
 * fields, 2 contract edge field, 3 receiver pass, 4 analysis, 5 project even, 6 project odd.
 * A skipped stage counts as 0.
 * Errors: CGTP_ERR_ARG (NULL, flag not set, unknown op), CGTP_ERR_HIP. */
int cgtp_stage_times(cgtp_plan plan, int op, double *ms, int cap, int *n_stages, int *n_calls);

/* Measurement helper, not part of the method: the read-pattern ceiling of the message-passing
 * receiver. Replays, for the CSR (row_ptr, col) of cgtp_message_pass, exactly the sender-field
 * loads of the plan's receiver, in its block order, over fields [n_nodes][R][3][UVs]
 * (UVs = n_theta * n_phi rounded up to 32; contents arbitrary), and computes nothing from them;
 * sink is a device float written at most once. Its time is the floor the receiver's gather
 * pattern sets on the memory path. The receivers take the surface curl with both derivatives
 * moved onto the analysis (integration by parts on the sphere), so they read only the value
 * plane (plane 0) of each sender rank, once per edge: 4 R n_theta n_phi bytes per edge.
 * Supported for fp32 plans whose receiver is the MFMA one on the plain sender layout (the
 * default grid below lmax 7, R a multiple of 16) or the per-thread one (grids of at most 1024
 * points). Asynchronous on stream.
 * Errors: CGTP_ERR_ARG (NULL, sizes, fields_bytes too small), CGTP_ERR_UNSUPPORTED (another
 * receiver), CGTP_ERR_HIP. */
int cgtp_gather_probe(cgtp_plan plan, int64_t n_nodes, int64_t n_edges, const int32_t *row_ptr,
                      const int32_t *col, const void *fields, size_t fields_bytes, void *sink,
                      void *stream);

/* Scheduling aid, not an operation of the paper: the order in which the message-passing
 * receivers run. The neighbour sum of a receiver (Eq. msgpass-S) is the same whatever order
 * the receivers are processed in, so the outputs of every message-passing call are bitwise
 * the same with or without an order; a locality-preserving one lets the receivers that run at
 * the same time share their senders, whose grid fields then stay in the GPU's L2.
 *
 * cgtp_receiver_order (host only, no GPU needed) computes such an order for the CSR of a
 * message-passing call: row_ptr[n_nodes + 1], col[n_edges] and edge_vec[n_edges][3] are HOST
 * arrays, order[n_nodes] a host array it fills with a permutation of 0 .. n_nodes - 1.
 * edge_vec is the edge direction of cgtp_message_pass (or the displacement vector); positions
 * are rebuilt from it along a breadth-first spanning tree of each connected component, and
 * the nodes sorted by component, then by the Hilbert index of the rebuilt position. edge_vec
 * may be NULL (e.g. for cgtp_message_pass_fields): the order is then the breadth-first
 * discovery order. Deterministic. Cost O(n_edges + n_nodes log n_nodes) on one host thread;
 * compute it once per graph. Errors: CGTP_ERR_ARG (NULL, sizes), CGTP_ERR_CSR (row_ptr not
 * non-decreasing from 0 to n_edges, or col out of range).
 *
 * cgtp_plan_set_receiver_order copies order[n_nodes] (a HOST array, checked to be a
 * permutation) to device memory the plan owns; from then on every message-passing call and
 * cgtp_gather_probe on the plan runs its receivers in that order and must pass exactly
 * n_nodes nodes (CGTP_ERR_ARG otherwise). order NULL or n_nodes 0 clears it (the identity).
 * Synchronises the device. Setting or clearing an order frees the previous device copy, so
 * a HIP graph captured from calls under that order must not be replayed afterwards.
 * Errors: CGTP_ERR_ARG (NULL plan, not a permutation, wrong device), CGTP_ERR_HIP
 * (allocation or copy). */
int cgtp_receiver_order(int64_t n_nodes, int64_t n_edges, const int32_t *row_ptr,
                        const int32_t *col, const float *edge_vec, int32_t *order);
int cgtp_plan_set_receiver_order(cgtp_plan plan, int64_t n_nodes, const int32_t *order);

/* Release the plan and everything it owns. Synchronises the device first.
 * cgtp_destroy(NULL) is a no-op. */
int cgtp_destroy(cgtp_plan plan);

/* Static description of a status code. */
const char *cgtp_status_string(int status);

/* Detail message of the last failing call on this host thread ("" if none). */
const char *cgtp_last_error(void);

/* Host-only (no GPU needed): the fp64 grid tables a plan would upload, for
 * testing. Sizes with U = n_theta, V = n_phi, P = (lmax+1)(lmax+2)/2:
 *   x[U], w[U]         Gauss-Legendre nodes cos(theta_u) and weights (sum 2)
 *   p[U][P], dp[U][P]  Pt_l^m(x_u) and dPt_l^m/dx(x_u), index l(l+1)/2 + m, m >= 0
 *   q[V][2 lmax + 1]   real Fourier factors q_vm of Eq. realq, column m + lmax
 * Any output pointer may be NULL. n_theta / n_phi follow the cgtp_desc rules. */
int cgtp_host_tables(int lmax, int n_theta, int n_phi, double *x, double *w, double *p,
                     double *dp, double *q);

#ifdef __cplusplus
}
#endif

#endif /* CGTP_H */
