/*
 * e2f.h -- C ABI of libe2f: the Wigner-6j convolution of E2Former
 * (arXiv 2501.19216) on AMD MI355X (gfx950).
 *
 * The layer (Def. 3.1 with attention weights, App. D.2 setup; Alg. 1 I/O):
 *   y_i^(o)[m,c] = sum_{j in N(i)} alpha[e(i,j), c / (C/H)] sum_{a,f} w[a][f][o]
 *                  [h_j^(a) (x) R^(f)(r_i - r_j)]^(o)_m [c]
 *   out_i^(o)[m,c'] = sum_c W[o][c'][c] y_i^(o)[m,c]              (App. F self-mix)
 * with real regular solid harmonics R^(f) (Def. 2.1), real-basis
 * Clebsch-Gordan coupling [.](o) (Def. 2.2), a, f, o <= L.
 *
 * Conventions:
 *   - irrep features are float32 [N][(L+1)^2][C], index l*l+l+m, m = -l..l,
 *     real basis with m<0 <-> sin(|m| phi), m>0 <-> cos(m phi), no
 *     Condon-Shortley sign; R^(1)(v) = (v_y, v_z, v_x) and
 *     R^(l) = [R^(l-1) (x) R^(1)]^(l) (stretched power);
 *   - channel c belongs to head c / (C/H);
 *   - positions are float32 [N][3] in Angstrom; the radius graph compares
 *     squared distances exactly on the 2^-16 A grid (positions are rounded
 *     to it for that comparison only);
 *   - the graph is CSR: row_ptr int64 [N+1], col_idx int32 [E]; row i holds
 *     the senders j of receiver i in ascending order; attention weights are
 *     float32 [E][H] in the same order.
 *
 * Memory: every pointer argument is HIP device memory owned by the caller
 * unless it is marked "host".  The library never frees caller memory.  A
 * context owns its coefficient tables: the structure tables of every degree
 * (uploaded by e2f_create) and one set of path-weighted coefficients per
 * path-weight vector it has seen (uploaded on first use, at most 16 per
 * degree).  The Wigner-6j forward works in a workspace the caller provides
 * (e2f_wigner6j_workspace_size); the other layer entry points (edge-TP
 * baseline with mixing, dense and global forms, backward, node TP) keep an
 * internal workspace that grows on demand (hipMalloc) and is released by
 * e2f_destroy.
 *
 * Streams: `stream` is a hipStream_t passed as void* (NULL = null stream).
 * Work is enqueued on it; calls marked (sync) also wait for it.  Calls not
 * marked (sync) neither wait for the device nor read anything back from it.
 *
 * Errors: functions return e2f_status and never throw.  Arguments are
 * checked on the host before any device work; on E2F_EINVAL no output is
 * written.  e2f_last_error() gives the message of the last failing call on
 * the calling thread.  A context is not safe for concurrent use from two
 * threads, and calls on one context must not overlap on two streams.
 */
#ifndef E2F_H
#define E2F_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  E2F_OK = 0,
  E2F_EINVAL = 1,       /* bad argument (null pointer, bad size, non-finite) */
  E2F_ECAPACITY = 2,    /* output buffer too small; the needed size is returned */
  E2F_ENOMEM = 3,       /* device allocation failed */
  E2F_EDEVICE = 4,      /* HIP error, or a context without a device */
  E2F_EUNSUPPORTED = 5  /* L, C or problem size outside what is compiled in */
} e2f_status;

typedef enum { E2F_F32 = 0, E2F_BF16 = 1 } e2f_dtype;
typedef enum { E2F_FORM_AUTO = 0, E2F_FORM_SPLIT = 1, E2F_FORM_FUSED = 2 } e2f_form;

typedef struct e2f_ctx e2f_ctx;

/* Create a context for degrees up to lmax_max (0..6) on HIP device `device`.
 * device = -1 makes a host-only context (tables and argument checks only;
 * every device call then returns E2F_EDEVICE).  (sync) */
e2f_status e2f_create(int lmax_max, int device, e2f_ctx** out);
void e2f_destroy(e2f_ctx* ctx);
/* Message of the last failing call on this thread ("" if none). */
const char* e2f_last_error(void);

/* Number of rows of the j-side node tensor product T_j for degree L: the
 * blocks [h^(a) (x) R^(b)]^(d), a,b <= L, |a-b| <= d <= a+b, that some
 * i-side degree u <= L-b and output o <= L use (Thm. 3.3).  -1 if L is out
 * of range.  58 / 183 / 454 / 1767 for L = 2 / 3 / 4 / 6. */
int64_t e2f_node_tp_dim(int lmax);

/* Host utilities (host memory, no context). */
/* Real-basis CG tensor for (l1,l2,l3), l <= 12: out[(2l1+1)][(2l2+1)][(2l3+1)] (Def. 2.2). */
e2f_status e2f_real_cg(int l1, int l2, int l3, double* out /* host */);
/* Recoupling weight X_d of [A (x) [C (x) B]^(b+u)]^(o) = sum_d X_d [C (x) [A (x) B]^(d)]^(o)
 * for A, B, C of degrees a, b, u (Def. 2.3). */
double e2f_recoupling_weight(int a, int b, int u, int o, int d);

/* Radius graph (Alg. 1 step 2): every ordered pair (i, j), i != j, with
 * |r_i - r_j| < cutoff (strict, exact on the 2^-16 A grid) and, if graph_id
 * is given, graph_id[i] == graph_id[j].  Rows are sorted ascending.
 * graph_id: [N] or NULL.  row_ptr: [N+1] (always written).  col_idx:
 * [capacity] or NULL.  *n_edges (host) receives E.  If col_idx is NULL or
 * E > capacity, returns E2F_ECAPACITY after writing row_ptr and *n_edges
 * (a size query).  Positions must satisfy |x| < 16384 A.  (sync) */
e2f_status e2f_neighbor_list(e2f_ctx* ctx, const float* pos, const int32_t* graph_id, int32_t n, float cutoff,
                             int64_t* row_ptr, int32_t* col_idx, int64_t capacity, int64_t* n_edges,
                             void* stream);

/* k-nearest-neighbour graph (the sparse graphs of the scaling study, Sec. 4.1
 * and Fig. 2): row i holds the min(k, n_g - 1) atoms j != i of i's graph (n_g
 * atoms; all atoms if graph_id is NULL) that come first in the order of
 * (squared distance on the 2^-16 A grid, compared exactly, then index j),
 * listed by ascending j.  1 <= k <= 512 (E2F_EUNSUPPORTED above).  Arguments,
 * capacity protocol and errors as for e2f_neighbor_list; graph ids must be
 * below 2^24.  Every candidate pair is examined (O(N^2) work).  (sync) */
e2f_status e2f_knn_graph(e2f_ctx* ctx, const float* pos, const int32_t* graph_id, int32_t n, int32_t k,
                         int64_t* row_ptr, int32_t* col_idx, int64_t capacity, int64_t* n_edges, void* stream);

/* Attention weights of the graph's edges, the input alpha of Alg. 1 (App. E:
 * logits from the scalar features and a radial basis, softmax over the
 * neighbours).  For the edge e = (i, j) of row i and head h:
 *   logit = sum_t q[i][h][t] k[j][h][t] + sum_r rbf_w[h][r] exp(-((d - mu_r)/sigma)^2),
 *   mu_r = r cutoff / (n_rbf - 1), sigma = cutoff / (n_rbf - 1), d = |r_i - r_j|,
 *   alpha[e][h] = (cos(pi d / cutoff) + 1)/2 * exp(logit) / (sum over row i of exp(logit)),
 * with the envelope 0 for d >= cutoff.  q, k: [N][heads][dk] float32 (unused
 * if dk = 0); rbf_w: [heads][n_rbf] float32 (n_rbf = 0: no radial term, else
 * 2..32); CSR as from e2f_neighbor_list / e2f_knn_graph; out alpha [E][heads].
 * heads <= 64.  fp32, deterministic. */
e2f_status e2f_attention_weights(e2f_ctx* ctx, const float* pos, const float* q, const float* k, int32_t n,
                                 int32_t heads, int32_t dk, const float* rbf_w, int32_t n_rbf, float cutoff,
                                 const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges, float* alpha,
                                 void* stream);

/* Real regular solid harmonics (Def. 2.1) of p_i = pos_i - origins[origin_id[i]]
 * (origin 0 if origin_id is NULL; the zero vector if origins is NULL),
 * evaluated in float64 and rounded: out [N][(lmax+1)^2] float32. */
e2f_status e2f_solid_harmonics(e2f_ctx* ctx, const float* pos, const float* origins, const int32_t* origin_id,
                               int32_t n, int lmax, float* out, void* stream);

/* j-side node tensor product (Alg. 1 clebsch_gorden_tp; red box of Thm. 3.3):
 * out[i][row][c] = [h_i^(a) (x) R^(b)(p_i)]^(d)_delta [c] for the rows of
 * e2f_node_tp_dim(lmax) blocks, ordered by (a, b, d), then delta.
 * p_i as in e2f_solid_harmonics.  feat [N][(L+1)^2][C], out [N][dimT][C].
 * C must be a multiple of 4. */
e2f_status e2f_node_tp(e2f_ctx* ctx, const float* pos, const float* origins, const int32_t* origin_id,
                       const float* feat, int32_t n, int32_t channels, int lmax, float* out, void* stream);

/* Attention-weighted aggregation of stored node tensors, on its own (the
 * aggregation of Alg. 1, its einsum "ijh,jhds->ihds" restricted to the
 * graph's edges, with T_j already made): for every receiver i, head h, row
 * k < rows and channel t < C/heads of the head,
 *     S[i][h][k][t] = sum over the edges e = (i, j) of row i of alpha[e][h] T[j][h][k][t].
 * T, S: device [n][heads][rows][C/heads] float32 (head-major: a head's
 * rows * C/heads values contiguous; S is written whole, isolated receivers
 * get zeros).  row_ptr [n+1], col_idx [n_edges]: CSR whose rows list their
 * senders strictly ascending (as e2f_neighbor_list writes them).  alpha:
 * [n_edges][heads] in CSR order, or NULL (ones).  C/heads a multiple of 4;
 * n_edges < 2^31.  Blocks of 16 receivers, consecutive in `order` (device
 * [n], a permutation of 0..n-1; NULL = index order), aggregate the union of
 * their senders on the matrix cores (A = the block's weights, B = the
 * union's rows of T), so each row of T read from L2 serves every receiver of
 * the block that has it as a neighbour: an order that keeps close atoms
 * together (a cell or Morton order of the positions) makes the unions small.
 * If some block has more than 8192 edges every receiver is summed on its own
 * instead.  The graph is checked first (the bits of e2f_validate_graph, 16
 * for a row not strictly ascending, 32 for an order that is not a
 * permutation: E2F_EINVAL, nothing written).  workspace:
 * e2f_aggregate_workspace_size bytes, 256-byte aligned (E2F_ECAPACITY
 * below).  Deterministic for a given order.  (sync: one read-back of the
 * check and the largest block) */
e2f_status e2f_aggregate_workspace_size(e2f_ctx* ctx, int32_t n, int64_t n_edges, int32_t heads, size_t* bytes);
e2f_status e2f_aggregate(e2f_ctx* ctx, const float* T, int32_t n, int32_t rows, int32_t channels, int32_t heads,
                         const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges, const float* alpha,
                         const int32_t* order, float* S, void* workspace, size_t workspace_bytes, void* stream);

typedef struct {
  int lmax;              /* L, 0..6 */
  int32_t channels;      /* C, a multiple of 4, <= 1024 */
  int32_t heads;         /* H, C % H == 0 and (C/H) % 4 == 0 (a head wider than the aggregation's
                            tile is split into channel groups that share its weights) */
  float cutoff;          /* r_c of the graph, used for default weights and tiles */
  const double* path_w;  /* host [(L+1)^3] w[a][f][o]; NULL => cutoff^-f on triangle-valid paths */
  const void* mix_w;     /* device [(L+1)][C][C] W[o][c_out][c_in] of mix_dtype; NULL => no mixing */
  e2f_dtype mix_dtype;   /* E2F_F32, or E2F_BF16 (mixing inputs rounded to bf16, fp32 accumulate) */
  float tile_side;       /* side of the receiver tiles whose centres serve as local origins;
                            0 => cutoff * (8, 8, 8, 6, 4, 3, 2) for L = 0..6 (fp32 precision of
                            the binomial expansion; the cost does not depend on it) */
  int32_t y_norm;        /* 0: the layer above.  1: Alg. 1's per-degree attention weights
                            alpha_ij / D_ij^f on the paths of filter degree f, D_ij = |r_i - r_j|
                            (filters Y^(f) of the unit vector; the path f takes 0 at D = 0 for
                            f > 0).  The factorised forward then aggregates once per f (L+1
                            times the aggregation work).  The weights 1/D^f no longer damp the
                            rounding of the binomial expansion (about eps ((|p_i| + |p_j|) /
                            D_ij)^f per edge), so the tile side is capped at 2.31 times the
                            shortest nonzero edge (found on the device), keeping that ratio
                            below 5.  Forward entry points only (the backward returns
                            E2F_EUNSUPPORTED) */
  int32_t form;          /* which form of the aggregation and recouple the forward runs (e2f_form):
                            E2F_FORM_FUSED: up to L = 4, with heads whose width is a multiple of 16,
                            the aggregation applies the i-side recouple itself (with y_norm, per
                            filter degree f with the weights alpha / D^f and the terms b + u = f,
                            at L = 4 in two passes: degrees 3 and 2, then 4, 1 and 0) (the
                            j-side coupling and the recouple of Thm. 3.3 composed into one
                            (L+1)^2 x (L+1)^4 matrix per receiver), so S is never stored;
                            elsewhere the split form.  E2F_FORM_SPLIT: S is written and recoupled
                            by a second kernel.  E2F_FORM_AUTO (0): fused wherever it applies with
                            y_norm (the split form then aggregates once per degree), and at L = 4
                            where the split form's S (n dimT C floats) would exceed 256 MiB
                            (beyond the on-die cache its round trip through HBM outweighs the
                            fused form's extra matrix-core work per receiver), else split.  All forms give the same
                            result up to rounding order: the fused form multiplies on the bf16
                            matrix cores with each float operand split into three bf16 parts
                            (x = hi + mid + lo exactly) and the six cross products that reach
                            2^-24 of the product accumulated in float, i.e. float products to
                            within float rounding */
} e2f_conv_params;

/* Workspace of e2f_wigner6j_conv_forward for n atoms and n_edges edges:
 * *bytes (host) = the size with which every receiver's S fits at once (one
 * aggregation pass), about E (L+1)^2 4 + N dimT C 4 bytes plus the plan
 * (N (L+1)^2 8 + 40 N bytes and the sort's scratch), E H 4 for the attention
 * weights ((L+1) times that with y_norm) and N (L+1)^2 C 4 with mixing. */
e2f_status e2f_wigner6j_workspace_size(e2f_ctx* ctx, const e2f_conv_params* params, int32_t n, int64_t n_edges,
                                       size_t* bytes);
/* The smallest workspace the forward accepts: the plan and per-edge arrays
 * plus S for 256 receivers; any size between this and
 * e2f_wigner6j_workspace_size works (receivers are then aggregated and
 * recoupled in slices that fit, in the same order and with the same result). */
e2f_status e2f_wigner6j_workspace_min(e2f_ctx* ctx, const e2f_conv_params* params, int32_t n, int64_t n_edges,
                                      size_t* bytes);
/* Uploads what the forward needs for these parameters (the coefficient set
 * of the path weights, the aggregation's coupling schedule) so that later
 * forwards with them do no host-to-device copy.  The forward does the same
 * on first use.  (sync) */
e2f_status e2f_wigner6j_prepare(e2f_ctx* ctx, const e2f_conv_params* params);

/* Wigner-6j convolution forward (Thm. 3.3, Alg. 1): the layer above computed
 * by node factorisation.  Each receiver i takes as local origin o the centre
 * of its tile (a cube of side tile_side of its graph's bounding box).  With
 * p = r - o, the forward aggregates the uncoupled products of the neighbours,
 *   G_i = sum_j alpha_ij R(p_j) (x) h_j   (the j-side node product before
 *   its CG coupling, Alg. 1 clebsch_gorden_tp; linear in h_j (x) R(p_j)),
 * couples them into S_i^(a,b,d) = [h (x) R^(b)]^(d) summed over j (the
 * einsum "ijh,jhds->ihds"), and recouples at the receiver,
 *   y_i = sum K(a,b,d,u,o) [R^(u)(p_i) (x) S_i^(a,b,d)]^(o)   (Wigner6jTP),
 * then mixes.  graph_id: [N] or NULL (must match the graph's).  alpha:
 * [E][H] or NULL (all ones).  out: [N][(L+1)^2][C].  Isolated atoms get zero
 * rows.
 * workspace: device memory of workspace_bytes >= e2f_wigner6j_workspace_min
 * (else E2F_ECAPACITY), 256-byte aligned; its contents on entry do not
 * matter and are overwritten.  Not needed (may be NULL) when n_edges = 0.
 * Asynchronous: no host wait, no device allocation or host-to-device copy
 * once the path weights are resident (e2f_wigner6j_prepare), so the call can
 * be captured in a HIP graph.  The plan (bounding box, tiles, receiver order)
 * is derived on the device: positions must be finite with |x| < 16384 A (an
 * atom outside that range is placed in the nearest tile and its outputs are
 * not meaningful; nothing is reported).  The CSR is trusted for values but
 * read with clamped indices (a malformed graph gives wrong outputs, never an
 * access outside the buffers); e2f_validate_graph checks one.
 * Deterministic: no floating-point atomics. */
e2f_status e2f_wigner6j_conv_forward(e2f_ctx* ctx, const e2f_conv_params* params, const float* pos,
                                     const int32_t* graph_id, const float* feat, int32_t n, const int64_t* row_ptr,
                                     const int32_t* col_idx, int64_t n_edges, const float* alpha, float* out,
                                     void* workspace, size_t workspace_bytes, void* stream);

/* e2f_wigner6j_conv_forward for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same computation and result, in a scratch area of
 * 128 MiB that the library holds in every GPU it runs on (a static device
 * array, resolved per device by e2f_create) instead of a caller workspace.
 * It calls no hipMalloc, hipFree, host-to-device copy or allocating library
 * routine: the path weights' coefficient set and the coupling schedule must
 * already be resident (e2f_wigner6j_prepare, or an earlier forward with the
 * same parameters), else E2F_EINVAL.  Inputs whose smallest workspace
 * (e2f_wigner6j_workspace_min) exceeds 128 MiB return E2F_ECAPACITY.  All
 * calls on one GPU share its scratch area: calls that overlap on one GPU
 * (two streams, two threads, two contexts) race and must be serialised by
 * the caller.  Nothing in it needs to start at zero; it keeps the last
 * call's contents. */
e2f_status e2f_wigner6j_conv_forward_noalloc(e2f_ctx* ctx, const e2f_conv_params* params, const float* pos,
                                             const int32_t* graph_id, const float* feat, int32_t n,
                                             const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges,
                                             const float* alpha, float* out, void* stream);

/* Checks a CSR graph of n atoms: *bad (host) = 0 if row_ptr[0] = 0, row_ptr
 * never decreases, row_ptr[n] = n_edges and every col_idx is in [0, n); else
 * the OR of 1 (row_ptr[0]), 2 (a decreasing row_ptr), 4 (row_ptr[n]), 8 (a
 * sender out of range).  Launches no layer kernel.  (sync) */
e2f_status e2f_validate_graph(e2f_ctx* ctx, int32_t n, const int64_t* row_ptr, const int32_t* col_idx,
                              int64_t n_edges, int32_t* bad /* host */, void* stream);

/* The layer on a dense graph (every atom attends to every other atom; the
 * dense graphs of the scaling study, Sec. 4.1, and Alg. 1 with its attention
 * tensor alpha in R^{N x N x H}): the sum runs over all j != i.
 * alpha [N][N][H] float32 (receiver i, sender j, head); alpha[i][i][*] is
 * ignored; NULL => 1 for every pair.  One origin, the centre of the bounding
 * box (found on the device).  T_j is stored for every atom and the
 * aggregation S_h = A_h T_h is a dense product per head on the matrix cores
 * (fp32, a hand-written tiled kernel).  tile_side and cutoff serve only the
 * default path weights (cutoff^-f).  N^2 H must stay below 4e9.  Internal
 * workspace: about N (2 dimT C + N H) floats.  Positions must be finite with
 * |x| < 16384 A (not reported). */
e2f_status e2f_wigner6j_conv_forward_dense(e2f_ctx* ctx, const e2f_conv_params* params, const float* pos,
                                           const float* feat, int32_t n, const float* alpha, float* out,
                                           void* stream);

/* Uniform attention over the whole graph (the global-moment special case of
 * App. G): alpha = 1 for every pair i, j of the N atoms, j = i included, so
 * the aggregation collapses to the moments M = sum_j [h_j (x) R^(b)(r_j - o)]^(d)
 * of all atoms, summed once, and every atom contracts M with its own
 * R^(u)(r_i - o) (Thm. 3.3): O(N).  o is the centre of the bounding box; the
 * self term of j = i is R^(f)(0) = [f == 0].  heads only sets the layout of
 * the intermediates (every head sees the same weights); tile_side is unused.
 * out: [N][(L+1)^2][C].  The moments are taken of the uncoupled products,
 * G = sum_j R(r_j - o) (x) h_j, summed in float64 in a fixed order
 * (deterministic), and coupled once.  Internal workspace: N (L+1)^2 doubles
 * plus float64 partial sums of G (about 2048 (L+1)^2 * 256 doubles, some
 * 10-25 MB).  The centre is found on the device: positions must be finite
 * with |x| < 16384 A (not reported). */
e2f_status e2f_wigner6j_conv_forward_global(e2f_ctx* ctx, const e2f_conv_params* params, const float* pos,
                                            const float* feat, int32_t n, float* out, void* stream);

/* Backward of e2f_wigner6j_conv_forward (same parameters and graph): the
 * vector-Jacobian products for the output gradient grad_out [N][(L+1)^2][C].
 * The layer is linear in the features and in the attention weights:
 *   grad_feat [N][(L+1)^2][C]: the adjoint, itself a Wigner-6j convolution
 *     (Thm. 3.3) of the unmixed output gradient on the transposed graph (rows
 *     = senders), with path weights w[a][f][o] kappa(a,f,o) (-1)^f, kappa the
 *     ratio of the real CG tensors of (a,f,o) and (o,f,a) (computed from the
 *     tables); the mixing contributes W^(o) transposed;
 *   grad_alpha [E][H]: per edge and head, the dot product of the unmixed
 *     output gradient of the receiver with the edge's message; needs feat
 *     and C <= 256;
 *   grad_pos [N][3]: the gradient with respect to the positions (the graph
 *     and alpha held fixed; forces are its negative).  Per edge (i, j) the
 *     message depends on r_i - r_j only, through R^(f); its derivative uses
 *     the gradient of the solid harmonics, and the edge's vector adds to i and
 *     subtracts from j (per atom in a fixed order: deterministic); needs feat
 *     and C <= 256.
 * Both per-edge products use that the edge filter is linear in R(r_i - r_j):
 * the receiver's output gradient is contracted with the filter coefficients
 * once per receiver, and one product with the senders' features per head
 * gives the contraction against R (grad_alpha) and against its gradient
 * weighted by alpha (grad_pos) for every edge of the receiver.
 * Any of the outputs may be NULL (not all).  Not available with y_norm. */
e2f_status e2f_wigner6j_conv_backward(e2f_ctx* ctx, const e2f_conv_params* params, const float* pos,
                                      const int32_t* graph_id, const float* feat, const float* grad_out, int32_t n,
                                      const int64_t* row_ptr, const int32_t* col_idx, int64_t n_edges,
                                      const float* alpha, float* grad_feat, float* grad_alpha, float* grad_pos,
                                      void* stream);

/* The conventional per-edge SO(3) convolution (Def. 3.1): the same layer
 * computed edge by edge with R^(f)(r_i - r_j) and the CG product per edge.
 * Same arguments and output as e2f_wigner6j_conv_forward; graph_id unused. */
e2f_status e2f_edge_tp_conv_forward(e2f_ctx* ctx, const e2f_conv_params* params, const float* pos,
                                    const int32_t* graph_id, const float* feat, int32_t n, const int64_t* row_ptr,
                                    const int32_t* col_idx, int64_t n_edges, const float* alpha, float* out,
                                    void* stream);

/* Number of receiver slices the last e2f_wigner6j_conv_forward on this
 * context ran (1 when the workspace held every receiver's S).  Host output. */
e2f_status e2f_last_slices(const e2f_ctx* ctx, int64_t* slices /* host */);

/* Kernel timing.  e2f_profile(ctx, 1) waits for the device, clears the
 * records and starts bracketing every launch group of this context with HIP
 * events on its stream (bbox, nl_count, nl_fill, tile_plan, sh, node_tp,
 * aggregate, recouple, mix, edge_tp); e2f_profile(ctx, 0) stops.  (sync) */
e2f_status e2f_profile(e2f_ctx* ctx, int enable);
/* Text "name launches total_ms" per line for the records so far, into buf
 * (host, `bytes` long, NUL-terminated); E2F_ECAPACITY if too small.  (sync) */
e2f_status e2f_profile_read(e2f_ctx* ctx, char* buf /* host */, size_t bytes);

#ifdef __cplusplus
}
#endif

#endif /* E2F_H */
