// Kernel launchers of libe2f (implemented in neighbor.hip, plan.hip, conv.hip
// and attention.hip).
// All sizes are checked by the callers in abi.cpp before these run.
#pragma once

#include <hip/hip_runtime.h>

#include "e2f_internal.h"

namespace e2f {

// stats[0..2] = min grid coordinate, stats[3..5] = max, stats[6] = max
// graph id, stats[7] = error bits (1: bad position, 2: negative graph id).
constexpr int kStatsInts = 8;
// rows of padding after the forward's per-edge arrays (harmonics of the
// edges, head-major attention weights): the fused aggregation's staging
// loads whole chunks of edges without a bound check
constexpr int kEdgePad = 128;
hipError_t launch_bbox(const float* pos, const int32_t* graph_id, int n, int* stats, hipStream_t s);

// ---- device-side plan of the factorised forward (plan.hip)
// Tile grid on the 2^-16 A lattice, shared by every graph: cell (cx, cy, cz)
// covers lo + [c span / dim, (c+1) span / dim) per axis; its centre is the
// local origin of the receivers in it.
struct TileGridDev {
  int lo[3];
  int dim[3];
  int64_t span[3];
  int ncell;
  int pad;
};
// stats as for launch_bbox (initialised here); dmin (or NULL) receives the
// shortest nonzero edge length as fp32 bits after launch_plan_dmin
hipError_t launch_plan_bbox(const float* pos, const int32_t* graph_id, int n, int* stats, unsigned* dmin,
                            hipStream_t s);
hipError_t launch_plan_dmin(const float* pos, const int32_t* rows, const int32_t* col, int n, int64_t n_edges,
                            unsigned* dmin, hipStream_t s);
// origin [3] float64 = the centre of the bounding box in stats
hipError_t launch_plan_centre(const int* stats, double* origin, hipStream_t s);
// side in grid units; with dmin, side = min(side, dmin_scale * shortest edge)
hipError_t launch_plan_grid(const int* stats, const unsigned* dmin, double side, double dmin_scale,
                            TileGridDev* grid, hipStream_t s);
size_t plan_sort_tmp_bytes(int n);
// stats and *dmin initialised alone (the small plan computes the box itself)
hipError_t launch_plan_init(int* stats, unsigned* dmin, hipStream_t s);
// The whole plan of a graph of at most kPlanSmallMax atoms in one workgroup:
// stats, grid, tile_of and order as launch_plan_bbox + launch_plan_grid +
// launch_plan_order give them (dmin as for launch_plan_grid)
constexpr int kPlanSmallMax = 8192;
hipError_t launch_plan_small(const float* pos, const int32_t* graph_id, int n, const unsigned* dmin, double side,
                             double dmin_scale, int* stats, TileGridDev* grid, int32_t* tile_of, int32_t* order,
                             hipStream_t s);
// tile_of [n] = the grid cell of every atom; order [n] = receivers sorted by
// (graph, Morton index of 4 A cells)
hipError_t launch_plan_order(const float* pos, const int32_t* graph_id, int n, const TileGridDev* grid,
                             int32_t* tile_of, uint64_t* keys, uint64_t* keys_out, int32_t* vals, int32_t* order,
                             void* tmp, size_t tmp_bytes, hipStream_t s);
// Rr [n][nk] float64 (receivers) and Re [E][nk] float32 (senders, CSR order),
// both about the receiver's tile centre; rows [E]: the receiver of every
// edge (launch_plan_edge_rows)
hipError_t launch_plan_sh(const DevTables& t, const float* pos, const int32_t* rows, const int32_t* col, int n,
                          int64_t n_edges, const int32_t* tile_of, const TileGridDev* grid, double* Rr, float* Re,
                          hipStream_t s);
// rows [E] = the receiver of every edge; with alpha (and alpha_hm), the same
// launch copies the weights [E][H] head-major into alpha_hm [H][E]
hipError_t launch_plan_edge_rows(const int64_t* row_ptr, int n, int64_t n_edges, int32_t* rows, const float* alpha,
                                 int H, float* alpha_hm, hipStream_t s);
hipError_t launch_fill(float* p, int64_t count, float v, hipStream_t s);
// *bad (device int) = 0, or the bits of k_validate_*: 1 row_ptr[0] != 0,
// 2 a decreasing row_ptr, 4 row_ptr[n] != n_edges, 8 a sender outside [0, n)
hipError_t launch_validate_graph(const int64_t* row_ptr, const int32_t* col, int n, int64_t n_edges, int* bad,
                                 hipStream_t s);

// ---- radius graph
struct CellGrid {
  int lo[3];
  int64_t side;   // cell side in grid units (>= cutoff)
  int dim[3];
  int64_t ncell;
};
size_t nl_scratch_bytes(int n, const CellGrid& g);  // cell tables and counts
// max_degree: device int, receives the largest row length
hipError_t launch_nl_count(const float* pos, const int32_t* graph_id, int n, double r2, const CellGrid& g,
                           void* scratch, int64_t* row_ptr, int* max_degree, hipStream_t s);
// After the count: sorts n+1 counts into row_ptr (exclusive scan).  Part of launch_nl_count.
// rows up to 1024 long are sorted in LDS; longer graphs go through `unsorted`
// and a segmented sort
hipError_t launch_nl_fill(const float* pos, const int32_t* graph_id, int n, double r2, const CellGrid& g,
                          void* scratch, const int64_t* row_ptr, int32_t* unsorted, int32_t* col_idx, int64_t E,
                          int max_degree, void* sort_tmp, size_t sort_tmp_bytes, hipStream_t s);
size_t nl_sort_tmp_bytes(int n, int64_t E);
// k-nearest-neighbour graph: row sizes min(k, graph size - 1) into row_ptr
// (graph ids in [0, ngraph)), then the rows (k <= kKnnMaxK).
constexpr int kKnnMaxK = 512;
size_t knn_scratch_bytes(int n, int ngraph);
hipError_t launch_knn_count(const int32_t* graph_id, int n, int k, int ngraph, void* scratch, int64_t* row_ptr,
                            hipStream_t s);
hipError_t launch_knn_fill(const float* pos, const int32_t* graph_id, int n, int k, const int64_t* row_ptr,
                           int32_t* col_idx, hipStream_t s);

// ---- solid harmonics: out[item][k], item -> node node_of[item] (or item),
// origin origins[origin_id[item] % origin_mod] (or 0 / zero vector)
hipError_t launch_sh(const DevTables& t, const float* pos, const int32_t* node_of, const double* origins_d,
                     const float* origins_f, const int32_t* origin_id, int origin_mod, int n, double* out_d,
                     float* out_f, hipStream_t s);

// ---- factorised layer
// T stored head-major: T[item][c / dh][row][c % dh] (dh = C: plain [row][c])
hipError_t launch_node_tp(const DevTables& t, const double* R, const int32_t* node_of, const float* feat,
                          int n_items, int C, int dh, float* T, hipStream_t s);
// Receiver blocks of 16 consecutive entries of `order`: block edge counts
// (blk_count [nblk+1]) and offsets (blk_off [nblk+1]), the sorted union of the
// T rows each block reads (uni [E], block b at blk_off[b]), union sizes
// (ucount [nblk+1]) and the union position of every edge (edge_slot [E]).  Requires 16 * (largest
// degree) <= 8192.
constexpr int kBlockMaxDegree = 512;
size_t blocks_tmp_bytes(int nblk);
hipError_t launch_block_union(const int64_t* row_ptr, const int32_t* col_pair, const int32_t* order, int n,
                              int32_t* blk_count, int32_t* blk_off, int32_t* uni, int32_t* ucount, int32_t* edge_slot,
                              void* tmp, size_t tmp_bytes, hipStream_t s);
// S[r] for the n receivers order[0..n) (S rows follow that order); T holds the
// pairs from pair_base on.  use_blocks: MFMA form over the block plan (built
// for the same n receivers; the attention operand is assembled from the
// head-major weights alpha_hm [H][n_edges] and edge_slot); else per-receiver
// rows from L2 with alpha [n_edges][H].  Null weights mean all ones.  n_edges
// and n_total are the whole graph's edges and atoms (mean degree).
// Standalone aggregation plan checks (receivers in index order): bit 16 of
// *bad for a row whose senders are not strictly ascending; *maxc = the
// largest edge count of a block of 16 consecutive receivers (the block path
// of launch_aggregate takes blocks of at most a3_union_max() edges)
hipError_t launch_a3_checks(const int64_t* row_ptr, const int32_t* col, int n, int64_t n_edges, int* bad,
                            int* maxc, hipStream_t s);
int a3_union_max();
// bit 32 of *bad unless order is a permutation of 0..n-1 (cnt: n ints of scratch)
hipError_t launch_a3_order_check(const int32_t* order, int n, int* cnt, int* bad, hipStream_t s);
hipError_t launch_aggregate(const float* T, int pair_base, const int64_t* row_ptr, const int32_t* col_pair,
                            const float* alpha, const float* alpha_hm, int64_t n_edges, int n_total,
                            const int32_t* order, const int32_t* uni, const int32_t* blk_off,
                            const int32_t* ucount, const int32_t* edge_slot, bool use_blocks, int n, int dimT, int C,
                            int H, float* S, hipStream_t s);
// alpha_f[(f*H + h)*E + e] = alpha[e][h] / |r_i - r_j|^f for f <= L (rows:
// E ints, the receiver of every edge, filled here unless row_ptr is NULL,
// then read as given); alpha NULL means ones
hipError_t launch_alpha_dnorm(const float* pos, const int64_t* row_ptr, const int32_t* col, const float* alpha, int n,
                              int64_t n_edges, int H, int L, int32_t* rows, float* alpha_f, hipStream_t s);
// alpha_hm[h][e] = alpha[e][h]
hipError_t launch_alpha_head_major(const float* alpha, int64_t n_edges, int H, float* alpha_hm, hipStream_t s);
// S rows r < n (receivers order[r]) by aggregating the uncoupled node products
// alpha_ij R(p_j) (x) h_j and coupling per receiver (no T): Re [E][nk] float32
// (launch_plan_sh), alpha_hm [H][n_edges] or NULL (ones); H heads of C/H
// channels, each of the caller's heads split into hdiv (the attention weight
// of head h is alpha_hm[h / hdiv]); n_nodes bounds the senders
// with the coupling schedule of couple_schedule(tables, outer_agg_groups(L, C, H))
// (its packed form pmeta/ptab, ntab > 0, is staged in LDS when it exists)
bool outer_agg_supported(int L, int C, int H);
int outer_agg_groups(int L, int C, int H);
hipError_t launch_outer_agg(const DevTables& t, const float* Re, const int64_t* row_ptr, const int32_t* col,
                            const float* alpha_hm, int64_t n_edges, const float* feat,
                            const int32_t* order, const int* cmeta, const float* ccoef, const int* pmeta,
                            const float* ptab, int ntab, int ck, int cgroups, int n, int C, int H, int hdiv,
                            int n_nodes, float* S, hipStream_t s);
// Fused aggregation and recouple (L <= kFuseMaxL, H virtual heads of 16
// channels, C = 16 H): F rows r < n (receivers order[r]) of fuse_stride(nk)
// floats from the fused table (fptr/fidx/fcoef, fuse_table) and R [N][nk]
// float64; then y[order[r]] directly from the aggregated products and F row r
// (other arguments as for launch_outer_agg)
// (L <= kFuseMaxL, C = 16 H, and the re-laid features of n_nodes atoms
// addressable with 32-bit entry offsets)
bool outer_fused_supported(int L, int C, int H, int64_t n_nodes);
// nkr: the K rows of the table's layout (fuse_stride(nk, nkr) floats a row)
hipError_t launch_fuse_build(int L, int nkr, const int* fptr, const int* fidx, const double* fcoef,
                             const double* R, const int32_t* order, int n, float* F, hipStream_t s);
// featq: the features re-laid and split into bfloat16 parts by
// launch_feat_qmajor, n_nodes * C * 6 * fuse_groups(L) floats of space (a
// 16-byte and an 8-byte array of n_nodes * C / 16 * fuse_groups(L) * 16
// entries each)
int fuse_groups(int L);
hipError_t launch_feat_qmajor(int L, const float* feat, int n, int C, float* featq, hipStream_t s);
// The segments of the K rows of one fused aggregation (nkr rows, F from a
// table of that layout): segment q, from K row start[q] to the next start
// (or nkr), holds the components 0 .. of R(p_j) weighted by alpha_hm[q]
// ([H / hdiv][n_edges] head-major, NULL: weight 1).  The plain layer: one
// segment of nk rows; alpha / D^f: a segment per filter degree f of the
// table, (f+1)^2 rows with the weights alpha / D^f.
constexpr int kFusedSegs = 5;
struct FusedSegs {
  const float* alpha_hm[kFusedSegs];
  int start[kFusedSegs];  // start[0] = 0, increasing; no segment longer than nk
  int n;                  // 1 .. kFusedSegs
};
// K row counts the fused aggregation is built for: nk, and those of the
// stacked alpha / D^f passes (5, 14, 30 at L = 1, 2, 3; 30 at L = 4)
bool fused_krows_supported(int L, int nkr);
// accumulate: the result is added to y (the sum over the filter degrees of
// alpha / D^f), else stored
hipError_t launch_outer_fused(int L, int nkr, const float* Re, const int64_t* row_ptr, const int32_t* col,
                              const FusedSegs& sg, int64_t n_edges, const float* featq, const int32_t* order,
                              const float* F, int n, int C, int H, int hdiv, int n_nodes, bool accumulate, float* y,
                              hipStream_t s);
// y[order[r]] from S row r (head-major like T), r < n; shared_s: every r
// reads S row 0; accumulate: y += the product instead of y = (one writer per
// element)
hipError_t launch_recouple(const DevTables& t, const double* R, const float* S, bool shared_s, const int32_t* order,
                           int n, int C, int dh, float* y, hipStream_t s, bool accumulate = false);
// The global moment of every atom's uncoupled products, coupled into one S
// row M32 [H][dimT][dh]: part holds global_groups(n, nk, C) * nk * nk * C
// doubles, G64 nk * nk * C doubles; R [n][nk] float64 (one origin)
int global_groups(int n, int nk, int C);
hipError_t launch_global_moment(const DevTables& t, const double* R, const float* feat, int n, int C, int dh,
                                double* part, double* G64, float* M32, hipStream_t s);

// ---- attention weights [E][H] (H <= 64, 2 <= R <= kAttnMaxRbf radial functions)
constexpr int kAttnMaxRbf = 32;
hipError_t launch_attention(const float* pos, const float* q, const float* k, int n, int H, int dk,
                            const float* rbf_w, int R, float rc, const int64_t* row_ptr, const int32_t* col_idx,
                            float* alpha, hipStream_t s);

// ---- backward
// Both per-edge backward products in one pass (either output may be NULL):
// galpha[e][h] = sum_{c of h} <gy_i[.][c], (K_e h_j)[.][c]> [E][H] and the
// position gradient per edge gedge [E][3]; needs 4 | C/H and C <= 256.
// launch_force_gather then sums per atom the edges it receives minus those it
// sends (rowT, perm: the transposed graph).
bool edge_geom_supported(int C, int H);
// LDS bytes of the backward kernel for qc filter rows per pass and a
// schedule of gtot entries (staged in LDS up to L = 4)
size_t edge_geom_lds(int L, int dh, int qc, int gtot);
hipError_t launch_edge_geom(const DevTables& t, const float* pos, const float* feat, const float* gy,
                            const int64_t* row_ptr, const int32_t* col_idx, const float* alpha, int n, int C, int H,
                            int qc, const int* gmeta, const float* gunit, const int* goc, int gtot, const float* Gt,
                            int64_t n_edges, float* galpha, float* gedge, hipStream_t s);
// Gt [3][nk][E]: the harmonic gradients of every edge (rows: the receiver of
// each edge), read by launch_edge_geom when not NULL
hipError_t launch_edge_shgrad(const DevTables& t, const float* pos, const int32_t* rows, const int32_t* col,
                              int64_t n_edges, float* Gt, hipStream_t s);
hipError_t launch_force_gather(const int64_t* row_ptr, const int64_t* rowT, const int32_t* perm, const float* gedge,
                               int n, float* gpos, hipStream_t s);
// transposed CSR (row = sender, ascending receivers) and alpha in its order;
// scratch: rows, iota, keys_out, perm [E], cnt [n+1]
size_t transpose_tmp_bytes(int n, int64_t E);
hipError_t launch_transpose_graph(const int64_t* row_ptr, const int32_t* col_idx, const float* alpha, int n,
                                  int64_t E, int H, int32_t* rows, int32_t* iota, int32_t* keys_out, int32_t* perm,
                                  int64_t* cnt, int64_t* rowT_ptr, int32_t* colT, float* alphaT, void* tmp,
                                  size_t tmp_bytes, hipStream_t s);
// WT[o][c][c'] = W[o][c'][c], float32 or bf16 elements
hipError_t launch_transpose_mix(const void* W, bool bf16, int L, int C, void* WT, hipStream_t s);

// ---- dense graphs (dense.hip): A[h][i][j] = alpha[i][j][h] (1 if alpha is
// NULL), 0 for i == j, rows of dense_lda(n) floats (zero padding)
int dense_lda(int n);
hipError_t launch_dense_alpha(const float* alpha, int n, int H, float* A, hipStream_t s);
// S_h = A_h T_h per head on MFMA: T and S head-major [n][H][dimT][C/H]
hipError_t launch_dense_aggregate(const float* A, int n, const float* T, int dimT, int C, int H, float* S,
                                  hipStream_t s);
hipError_t launch_iota(int n, int32_t* v, hipStream_t s);

// ---- per-irrep channel mixing and the edge baseline
hipError_t launch_mix(int L, const float* y, const void* W, bool w_bf16, int n, int C, float* out, hipStream_t s);
hipError_t launch_edge_tp(const DevTables& t, const float* pos, const float* feat, const int64_t* row_ptr,
                          const int32_t* col_idx, const float* alpha, int n, int64_t n_edges, int C, int H, float* y,
                          hipStream_t s, bool y_norm = false);

}  // namespace e2f
