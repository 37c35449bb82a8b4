// Internal declarations shared by the host code (tables, C ABI) and the HIP
// kernels of libe2f.  Nothing here is part of the public ABI (include/e2f.h).
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

namespace e2f {

constexpr int kMaxL = 6;          // largest supported degree L
constexpr double kGrid = 65536.0; // positions are compared on a 2^-16 A grid

inline int nk_of(int L) { return (L + 1) * (L + 1); }

// ---------------------------------------------------------------- host tables
// Real-basis Clebsch-Gordan tensor C[m1][m2][m3] for (l1,l2,l3), row-major,
// built from the explicit CG formula and the real change of basis (tables.cpp).
std::vector<double> real_cg(int l1, int l2, int l3);
// Recoupling weight X(a,b,u,o;d) of [A (x) [C (x) B]^(b+u)]^(o) onto
// [C (x) [A (x) B]^(d)]^(o) (Def. 2.3), closed form from the Wigner 6j symbol.
double recoupling_weight(int a, int b, int u, int o, int d);
double wigner6j(int j1, int j2, int j3, int j4, int j5, int j6);

// Structure of the factorised layer for one L: every table is independent of
// the path weights except the *_coef arrays, which the context refreshes when
// the caller's path weights change.
// Thread count of the schedules that build per-node matrices in LDS.
constexpr int kSchedThreads = 256;
// Rows of T per chunk of the recouple's per-node matrix: 192 at L <= 4 (a
// 37 KB tile, four workgroups per CU: 1.18 vs 1.20 ms with 256 rows and three),
// 128 at L = 5, 120 at L = 6 (a 38.4 KB tile: four workgroups per CU instead
// of three with 128 rows, 46.9 vs 49.7 ms at 200k atoms).
constexpr int rc_rows(int nk) { return nk > 36 ? 120 : (nk > 25 ? 128 : 192); }
// Row stride (floats) of the recouple's per-node matrix tile in LDS: the
// 16*ceil(nk/16) used columns padded to 16 mod 32, so the MFMA operand reads
// of 4 rows x 16 columns fall in distinct banks.
constexpr int rc_qstride(int nk) {
  return 16 * ((nk + 15) / 16) + (((nk + 15) / 16) % 2 == 0 ? 16 : 0);
}

// A per-node matrix built by 256 threads from a fixed schedule: in chunk c,
// thread t walks entries k = 0..k[c]-1 at index off[c] + k*256 + t, each
// adding coef * R[ridx] and, on the last entry of a slot, storing the sum to
// LDS position dest.  meta packs dest (bits 0-19), ridx (20-26), last (31).
// Monomials of degree l, and the offset of degree l's block in the dense
// solid-harmonic table (rows 2l'+1 by columns sh_monos(l') for every l' < l).
constexpr int sh_monos(int l) { return (l + 1) * (l + 2) / 2; }
constexpr int sh_dense_off(int l) { return l <= 0 ? 0 : sh_dense_off(l - 1) + (2 * l - 1) * sh_monos(l - 1); }

struct Schedule {
  std::vector<int> k, off;
  std::vector<int> meta;
  std::vector<int> path;      // path-weight index of each entry (-1: none)
  std::vector<double> unit;   // coefficient without the path weight
};

struct Block {
  int a, b, d, toff;  // T_j^(a,b,d) occupies rows toff .. toff+2d
};

struct LayerTables {
  int L = 0, nk = 0, dimT = 0;
  std::vector<Block> blocks;        // sorted by (a, b, d)
  std::vector<int> a_row_start;     // [L+2] first T row of each a
  // solid harmonics as polynomials: component k = sum_t coef_t x^ex y^ey z^ez
  std::vector<int> sh_ptr;          // [nk+1]
  std::vector<int> sh_pow;          // packed ex | ey<<4 | ez<<8
  std::vector<double> sh_coef;
  // the same polynomials dense per degree l: rows m < 2l+1, columns the
  // monomials x^ex y^ey z^(l-ex-ey) in (ex, ey) order, ex and ey ascending;
  // the block of degree l starts at sh_dense_off(l)
  std::vector<double> sh_dense;
  // j-side per-node matrix M: row r of T has (2a+1) slots starting at m_rowoff[r]
  std::vector<int> m_rowoff;        // [dimT+1]
  std::vector<int> m_ptr;           // [nslots+1] entries of each slot
  std::vector<int> m_ridx;          // index into R (l*l + l + m)
  std::vector<double> m_coef;       // CG value
  // i-side per-node matrix Q_o, (2o+1) x ncol[o], for each output degree o
  std::vector<int> q_ncol;          // [L+1]
  std::vector<int> q_coloff;        // [L+2] offset of o's column list in q_cols
  std::vector<int> q_cols;          // T row index of each column
  std::vector<int> q_slotoff;       // [L+2] offset of o's slots
  std::vector<int> q_ptr;           // [nslots+1]
  std::vector<int> q_ridx;
  std::vector<int> q_path;          // (a*(L+1)+f)*(L+1)+o of the path weight
  std::vector<double> q_unit;       // coefficient without the path weight
  // edge tensor product filter K[k][q] (dense nk x nk)
  std::vector<int> k_ptr;           // [nk*nk+1]
  std::vector<int> k_ridx;
  std::vector<int> k_path;
  std::vector<double> k_unit;
  // node TP: one chunk; the matrix of degree a is stored transposed at
  // tp_mo[a], entry (al, row) at al*tp_rs[a] + row - a_row_start[a], with
  // 2a+1 rows of tp_rs[a] floats (tp_rs = 16 mod 32)
  Schedule tp_sched;
  std::vector<int> tp_rs, tp_mo;    // [L+1], [L+2]
  Schedule rc_sched;                // recouple: chunks of rc_rows T rows, dest = row*rc_qstride + (o*o+m)
  // recouple restricted to the terms of filter degree f = b + u, one schedule
  // per f (attention weights alpha / D^f need one aggregation per f)
  std::vector<Schedule> rcf_sched;  // [L+1]
  // j-side coupling of aggregated uncoupled products: S[row] = sum over the
  // row's entries of coef * G[be][q], entries ag_ptr[row] .. ag_ptr[row+1]
  // with ag_idx = be << 6 | q (be, q < (L+1)^2)
  std::vector<int> ag_ptr, ag_idx;
  std::vector<float> ag_coef;
  int max_qslots = 0;               // largest (2o+1)*ncol[o]
  int m_slots() const { return m_rowoff.back(); }
};

LayerTables build_layer_tables(int L);

// The coupling after aggregation as a thread-balanced schedule for `groups`
// groups of threads (one thread per channel in a group): entry k of group g
// at k*groups + g; meta = gidx (bits 0-11, be << 6 | q) | row << 12 | last
// (bit 31); rows are spread over the groups by entry count.
struct CoupleSchedule {
  int groups = 0, k = 0;
  std::vector<int> meta;
  std::vector<float> coef;
  // the same entries packed for LDS when dimT <= 512 and the coefficients take
  // at most 1024 distinct values (L <= 4): pmeta = gidx | row << 12 (9 bits) |
  // coefficient index << 21 (10 bits) | last (bit 31), tab = the coefficients
  // (empty otherwise)
  std::vector<int> pmeta;
  std::vector<float> tab;
};
CoupleSchedule couple_schedule(const LayerTables& t, int groups);

// Schedule of the per-receiver filter contraction of the backward,
// Z[be][q][c] = sum_k w(path) unit * gy[k][c], for filter rows q taken qc at a
// time (chunk ch covers q in [ch*qc, min(nk, (ch+1)*qc))).  Per chunk the
// keys (be, q) are spread over kGeomGroups groups by entry count; group g
// walks entries off[ch] + k*kGeomGroups + g for k < ck[ch]; meta = k (bits
// 0-5) | be << 6 | (q - ch*qc) << 12 | path << 18 | last (bit 31); a key
// without entries stores its zero from one entry of unit 0; padding entries
// are all zero and follow the group's last store.
constexpr int kGeomGroups = 32;
struct GeomSchedule {
  int qc = 0, nchunk = 0;
  std::vector<int> off, ck;
  std::vector<int> meta;
  std::vector<float> unit;
};
GeomSchedule geom_schedule(const LayerTables& t, int qc);
int64_t node_tp_dim(int L);

// ---------------------------------------------------------------- fused recouple
// Up to L = 4 the j-side coupling and the i-side recouple compose into one
// per-receiver matrix F_i = Q_i CG of (L+1)^2 rows k = (o, m) and (L+1)^4
// columns (be, q), be the component of R(p_j) and q that of h_j:
//     y_i[k][c] = sum_{be, q} F_i[k][be, q] G_i[be][q][c],
//     G_i[be][q][c] = sum_j alpha_ij R_be(p_j) h_j[q][c].
// F_i = sum_x R_x(p_i) K_x with fixed tensors K_x (x a component of R(p_i)),
// K_x[k][be, q] = sum over T rows r of Q_i's coefficient of R_x in entry
// (k, r) times CG[r][be, q].  F_i is stored per receiver in the order in which
// the aggregation's waves read it as the A operand of v_mfma_f32_16x16x4f32:
// per q a block of (row tile rt, K tile mt) sub-blocks, each [k4 < kc][l16 <
// rows][s < 4] holding F[16 rt + l16][be][q] at K position 4 k4 + s =
// fuse_kpos(be) of be's tile (zero at positions no component takes).  A tile
// of r components uses kc = ceil(r / 4) groups k4 and ks = ceil(r / kc)
// steps s each (component j of the tile at k4 = j / ks, s = j % ks), so where
// r <= 12 the steps s >= ks hold only zeros and F_i G_i skips them (at
// L = 4 the second tile's 9 components take s < 3).
constexpr int kFuseMaxL = 4;
constexpr int fuse_rows(int nk, int rt) { return nk - 16 * rt < 16 ? nk - 16 * rt : 16; }
constexpr int fuse_kc(int nk, int mt) { return (fuse_rows(nk, mt) + 3) / 4; }
constexpr int fuse_tiles(int nk) { return (nk + 15) / 16; }
constexpr int fuse_ks(int nk, int mt) { return (fuse_rows(nk, mt) + fuse_kc(nk, mt) - 1) / fuse_kc(nk, mt); }
// K position (0 .. 15) of component be inside its tile be / 16
constexpr int fuse_kpos(int nk, int be) {
  return 4 * ((be % 16) / fuse_ks(nk, be / 16)) + (be % 16) % fuse_ks(nk, be / 16);
}
static_assert(fuse_ks(25, 1) == 3 && fuse_kpos(25, 24) == 10 && fuse_kpos(25, 19) == 4 && fuse_kpos(25, 7) == 7 &&
                  fuse_ks(16, 0) == 4 && fuse_ks(1, 0) == 1 && fuse_ks(9, 0) == 3,
              "K positions of the fused layout");
// The K rows of F may stack several filter degrees (alpha / D^f, one pass
// over the edges for several degrees): nkr rows, in segments of (f+1)^2 rows
// per degree f, the j-side component be of degree f's segment at row
// start + be (the plain layer: one segment, nkr = nk).  Rows k stay the nk
// output components; the functions below with nk take rows k or, with nkr,
// K rows.
// offset (floats) of sub-block (rt, mt) inside a q block, rt-major
constexpr int fuse_blk(int nk, int nkr, int rt, int mt) {
  int off = 0;
  for (int a = 0; a < fuse_tiles(nk); ++a)
    for (int b = 0; b < fuse_tiles(nkr); ++b) {
      if (a == rt && b == mt) return off;
      off += 4 * fuse_kc(nkr, b) * fuse_rows(nk, a);
    }
  return off;
}
constexpr int fuse_qblock(int nk, int nkr) { return fuse_blk(nk, nkr, fuse_tiles(nk), 0); }
// floats of one receiver's F, rounded up to 64 (256-byte rows)
constexpr int fuse_stride(int nk, int nkr) { return (nk * fuse_qblock(nk, nkr) + 63) / 64 * 64; }
// position of F[k][kr][q] (kr a K row) in a receiver's row
constexpr int fuse_pos(int nk, int nkr, int k, int kr, int q) {
  return q * fuse_qblock(nk, nkr) + fuse_blk(nk, nkr, k / 16, kr / 16) +
         (fuse_kpos(nkr, kr) / 4 * fuse_rows(nk, k / 16) + k % 16) * 4 + fuse_kpos(nkr, kr) % 4;
}
// K rows of the stacked degrees degs[0 .. nd) (a degree -1: every filter
// degree in one segment of nk rows)
inline int fuse_krows(int nk, const int* degs, int nd) {
  int r = 0;
  for (int s = 0; s < nd; ++s) r += degs[s] < 0 ? nk : (degs[s] + 1) * (degs[s] + 1);
  return r;
}
// The alpha / D^f passes of the fused aggregation, each a set of filter
// degrees stacked in the K rows: below L = 4 one pass of every degree (L, L-1,
// .. 0: 30 K rows at L = 3); at L = 4 (55 rows in all) two passes within two
// K tiles, degrees 3 and 2 (25 rows), then 4, 1 and 0 (30 rows).
struct YnormPass {
  int nd;                   // segments
  int degs[kFuseMaxL + 1];  // their filter degrees
};
constexpr int kYnormMaxPasses = 2;
inline int ynorm_passes(int L, YnormPass* out) {
  if (L == 4) {
    out[0] = YnormPass{2, {3, 2, 0, 0, 0}};
    out[1] = YnormPass{3, {4, 1, 0, 0, 0}};
    return 2;
  }
  out[0] = YnormPass{L + 1, {0, 0, 0, 0, 0}};
  for (int s = 0; s <= L; ++s) out[0].degs[s] = L - s;
  return 1;
}
// K_x by position of F (CSR over the positions 0 .. fuse_stride - 1): the
// entries of position p are idx[e] (the component x) and coef[e] (float64,
// path weights w[a][f][o] included) for e in ptr[p] .. ptr[p+1] - 1.
struct FuseTable {
  std::vector<int> ptr;
  std::vector<int> idx;
  std::vector<double> coef;
};
// degs[0 .. nd): the segments of K rows (fuse_krows): a degree f >= 0 takes
// only the terms of filter degree f (the T rows of j-side degree b with the
// receiver's harmonics of degree u = f - b), for the per-degree weights
// alpha / D^f, at rows start + be of its segment; -1 takes every term (the
// plain layer).  nkr >= fuse_krows: the K rows of the layout (rows past the
// segments hold zeros), so that one degree alone can use the plain layout.
FuseTable fuse_table(const LayerTables& t, const std::vector<double>& w, const int* degs, int nd, int nkr);

// ---------------------------------------------------------------- device side
// Device copies of one LayerTables (pointers into one allocation).
struct DevTables {
  int L, nk, dimT;
  const int* a_row_start;
  const int* sh_ptr; const int* sh_pow; const double* sh_coef;
  const double* sh_dense;  // LayerTables::sh_dense
  const int* m_rowoff; const int* m_ptr; const int* m_ridx; const double* m_coef;
  const int* q_ncol; const int* q_coloff; const int* q_cols; const int* q_slotoff;
  const int* q_ptr; const int* q_ridx; const double* q_coef; // q_coef includes path weights
  const int* k_ptr; const int* k_ridx; const float* k_coef;  // k_coef includes path weights
  const int* tp_k; const int* tp_off; const int* tp_meta; const double* tp_coef;
  const int* rc_k; const int* rc_off; const int* rc_meta; const double* rc_coef;  // rc_coef includes path weights
  const int* ag_ptr; const int* ag_idx; const float* ag_coef;
  const float* w_f;  // path weights w[(a*(L+1) + f)*(L+1) + o] as float
  int max_qslots, m_slots;
  int tp_rs[kMaxL + 1], tp_mo[kMaxL + 2];
};

}  // namespace e2f
