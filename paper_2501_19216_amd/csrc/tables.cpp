// Host-side coefficient tables of libe2f.
//
// * Complex Clebsch-Gordan coefficients from the explicit (Racah) CG formula,
//   mapped to the real basis of Def. 2.1 (m<0 <-> sin, m>0 <-> cos, no
//   Condon-Shortley sign in the real functions).  The mapped tensor is purely
//   real when l1+l2+l3 is even and purely imaginary when odd; the nonzero part
//   is kept, which fixes the per-triple sign.
// * Wigner 6j symbols from Racah's single-sum formula, and the recoupling
//   weights of Def. 2.3 in closed form:
//     X(a,b,u,o;d) = (-1)^(a+b+d) sqrt((2d+1)(2f+1)) {a b d; u o f},  f = b+u,
//   times -1 when a+b+d and u+d+o are both odd (the real basis multiplies
//   odd-parity CG tensors by -i, and the four tensors of the two coupling trees
//   meet that factor an even number of times except in that case).
// * Real regular solid harmonics (Def. 2.1) as explicit polynomials of the
//   stretched power R^(l) = [R^(l-1) (x) R^(1)]^(l), R^(1)(v) = (y, z, x).
// * The index structure of the node-factorised layer (Thm. 3.3, Alg. 1):
//   j-side blocks T^(a,b,d) = [h^(a) (x) R^(b)(p_j)]^(d) kept when some
//   i-side degree u <= L-b and output o <= L can use them, and the i-side
//   coefficient K = w_{a,b+u,o} (-1)^b binom(b+u,u) X(a,b,u,o;d) of the binomial
//   expansion (Thm. 3.2) recoupled by Def. 2.3.
#include <algorithm>
#include <cmath>
#include <complex>
#include <cstdlib>
#include <map>
#include <tuple>

#include "e2f_internal.h"

namespace e2f {
namespace {

long double factorial(int n) {
  long double r = 1.0L;
  for (int k = 2; k <= n; ++k) r *= k;
  return r;
}

bool tri(int a, int b, int c) { return c >= std::abs(a - b) && c <= a + b; }

// <j1 m1; j2 m2 | J M>, Condon-Shortley phase, explicit single-sum form.
double cg_complex(int j1, int m1, int j2, int m2, int J, int M) {
  if (M != m1 + m2 || !tri(j1, j2, J)) return 0.0;
  if (std::abs(m1) > j1 || std::abs(m2) > j2 || std::abs(M) > J) return 0.0;
  long double pre = (2.0L * J + 1.0L) * factorial(J + j1 - j2) * factorial(J - j1 + j2) * factorial(j1 + j2 - J) /
                    factorial(j1 + j2 + J + 1);
  long double pm = factorial(J + M) * factorial(J - M) * factorial(j1 - m1) * factorial(j1 + m1) *
                   factorial(j2 - m2) * factorial(j2 + m2);
  long double sum = 0.0L;
  for (int k = 0; k <= j1 + j2 - J; ++k) {
    int d1 = j1 - m1 - k, d2 = j2 + m2 - k, d3 = J - j2 + m1 + k, d4 = J - j1 - m2 + k;
    if (d1 < 0 || d2 < 0 || d3 < 0 || d4 < 0) continue;
    long double den = factorial(k) * factorial(j1 + j2 - J - k) * factorial(d1) * factorial(d2) * factorial(d3) *
                      factorial(d4);
    sum += ((k & 1) ? -1.0L : 1.0L) / den;
  }
  return (double)(std::sqrt(pre * pm) * sum);
}

// Coefficient of Y^m in the real function S_p of degree l.
std::complex<double> to_real(int p, int m) {
  const double s = 1.0 / std::sqrt(2.0);
  if (p == 0) return m == 0 ? 1.0 : 0.0;
  if (p > 0) {
    if (m == p) return ((p & 1) ? -s : s);
    if (m == -p) return s;
    return 0.0;
  }
  int mu = -p;
  if (m == -mu) return {0.0, s};
  if (m == mu) return {0.0, (mu & 1) ? s : -s};
  return 0.0;
}

long double tri_coef(int a, int b, int c) {
  return std::sqrt(factorial(a + b - c) * factorial(a - b + c) * factorial(-a + b + c) / factorial(a + b + c + 1));
}

using Poly = std::map<std::tuple<int, int, int>, double>;

}  // namespace

std::vector<double> real_cg(int l1, int l2, int l3) {
  const int n1 = 2 * l1 + 1, n2 = 2 * l2 + 1, n3 = 2 * l3 + 1;
  std::vector<double> out((size_t)n1 * n2 * n3, 0.0);
  if (!tri(l1, l2, l3)) return out;
  const bool odd = (l1 + l2 + l3) & 1;
  for (int p1 = -l1; p1 <= l1; ++p1)
    for (int p2 = -l2; p2 <= l2; ++p2)
      for (int p3 = -l3; p3 <= l3; ++p3) {
        std::complex<double> acc = 0.0;
        for (int m1 = -l1; m1 <= l1; ++m1)
          for (int m2 = -l2; m2 <= l2; ++m2) {
            int m3 = m1 + m2;
            if (std::abs(m3) > l3) continue;
            std::complex<double> w = std::conj(to_real(p1, m1)) * std::conj(to_real(p2, m2)) * to_real(p3, m3);
            if (w == 0.0) continue;
            acc += w * cg_complex(l1, m1, l2, m2, l3, m3);
          }
        out[((size_t)(p1 + l1) * n2 + (p2 + l2)) * n3 + (p3 + l3)] = odd ? acc.imag() : acc.real();
      }
  return out;
}

double wigner6j(int j1, int j2, int j3, int j4, int j5, int j6) {
  if (!tri(j1, j2, j3) || !tri(j1, j5, j6) || !tri(j4, j2, j6) || !tri(j4, j5, j3)) return 0.0;
  const int a1 = j1 + j2 + j3, a2 = j1 + j5 + j6, a3 = j4 + j2 + j6, a4 = j4 + j5 + j3;
  const int b1 = j1 + j2 + j4 + j5, b2 = j2 + j3 + j5 + j6, b3 = j3 + j1 + j6 + j4;
  long double s = 0.0L;
  for (int t = std::max(std::max(a1, a2), std::max(a3, a4)); t <= std::min(b1, std::min(b2, b3)); ++t) {
    long double den = factorial(t - a1) * factorial(t - a2) * factorial(t - a3) * factorial(t - a4) *
                      factorial(b1 - t) * factorial(b2 - t) * factorial(b3 - t);
    s += ((t & 1) ? -1.0L : 1.0L) * factorial(t + 1) / den;
  }
  return (double)(tri_coef(j1, j2, j3) * tri_coef(j1, j5, j6) * tri_coef(j4, j2, j6) * tri_coef(j4, j5, j3) * s);
}

double recoupling_weight(int a, int b, int u, int o, int d) {
  const int f = b + u;
  if (!tri(a, f, o) || !tri(a, b, d) || !tri(u, d, o)) return 0.0;
  double x = (((a + b + d) & 1) ? -1.0 : 1.0) * std::sqrt((2.0 * d + 1.0) * (2.0 * f + 1.0)) * wigner6j(a, b, d, u, o, f);
  if (((a + b + d) & 1) && ((u + d + o) & 1)) x = -x;
  return x;
}

namespace {

struct Entry {
  int ridx, path;
  double unit;
};
struct Slot {
  int dest;
  std::vector<Entry> e;
};

// Balance the slots of every chunk over the threads (largest first to the
// least loaded thread) and lay the entries out transposed.
Schedule make_schedule(const std::vector<std::vector<Slot>>& chunks) {
  Schedule s;
  const int T = kSchedThreads;
  for (const auto& slots : chunks) {
    std::vector<int> order(slots.size());
    for (size_t q = 0; q < slots.size(); ++q) order[q] = (int)q;
    std::stable_sort(order.begin(), order.end(),
                     [&](int x, int y) { return slots[x].e.size() > slots[y].e.size(); });
    std::vector<std::vector<const Slot*>> per(T);
    std::vector<size_t> load(T, 0);
    for (int q : order) {
      if (slots[q].e.empty()) continue;
      int best = 0;
      for (int th = 1; th < T; ++th)
        if (load[th] < load[best]) best = th;
      per[best].push_back(&slots[q]);
      load[best] += slots[q].e.size();
    }
    size_t K = 0;
    for (int th = 0; th < T; ++th) K = std::max(K, load[th]);
    s.off.push_back((int)s.meta.size());
    s.k.push_back((int)K);
    const size_t base = s.meta.size();
    s.meta.resize(base + K * T, 0);
    s.path.resize(base + K * T, -1);
    s.unit.resize(base + K * T, 0.0);
    for (int th = 0; th < T; ++th) {
      size_t k = 0;
      for (const Slot* sl : per[th])
        for (size_t q = 0; q < sl->e.size(); ++q, ++k) {
          const size_t at = base + k * T + th;
          const bool last = q + 1 == sl->e.size();
          s.meta[at] = sl->dest | (sl->e[q].ridx << 20) | (last ? (int)0x80000000u : 0);
          s.path[at] = sl->e[q].path;
          s.unit[at] = sl->e[q].unit;
        }
    }
  }
  return s;
}

}  // namespace

static bool block_used(int L, int a, int b, int d) {
  for (int u = 0; u <= L - b; ++u)
    for (int o = 0; o <= L; ++o)
      if (tri(a, b + u, o) && tri(u, d, o)) return true;
  return false;
}

int64_t node_tp_dim(int L) {
  if (L < 0 || L > kMaxL) return -1;
  int64_t n = 0;
  for (int a = 0; a <= L; ++a)
    for (int b = 0; b <= L; ++b)
      for (int d = std::abs(a - b); d <= a + b; ++d)
        if (block_used(L, a, b, d)) n += 2 * d + 1;
  return n;
}

LayerTables build_layer_tables(int L) {
  LayerTables t;
  t.L = L;
  t.nk = nk_of(L);
  const int L1 = L + 1;
  // cached real CG tensors
  std::map<std::tuple<int, int, int>, std::vector<double>> cgs;
  auto CG = [&](int l1, int l2, int l3) -> const std::vector<double>& {
    auto key = std::make_tuple(l1, l2, l3);
    auto it = cgs.find(key);
    if (it == cgs.end()) it = cgs.emplace(key, real_cg(l1, l2, l3)).first;
    return it->second;
  };

  // ---- solid harmonics as polynomials (stretched power)
  std::vector<Poly> R(t.nk);
  R[0][{0, 0, 0}] = 1.0;
  if (L >= 1) {
    R[1][{0, 1, 0}] = 1.0;  // m=-1: y
    R[2][{0, 0, 1}] = 1.0;  // m= 0: z
    R[3][{1, 0, 0}] = 1.0;  // m=+1: x
  }
  const int e1[3][3] = {{0, 1, 0}, {0, 0, 1}, {1, 0, 0}};
  for (int l = 2; l <= L; ++l) {
    const auto& c = CG(l - 1, 1, l);
    for (int m3 = 0; m3 < 2 * l + 1; ++m3) {
      Poly acc;
      for (int m1 = 0; m1 < 2 * l - 1; ++m1)
        for (int m2 = 0; m2 < 3; ++m2) {
          double w = c[((size_t)m1 * 3 + m2) * (2 * l + 1) + m3];
          if (w == 0.0) continue;
          for (auto& kv : R[(l - 1) * (l - 1) + m1]) {
            auto [ex, ey, ez] = kv.first;
            acc[{ex + e1[m2][0], ey + e1[m2][1], ez + e1[m2][2]}] += w * kv.second;
          }
        }
      for (auto it = acc.begin(); it != acc.end();) it = (std::fabs(it->second) < 1e-15) ? acc.erase(it) : std::next(it);
      R[l * l + m3] = acc;
    }
  }
  t.sh_ptr.push_back(0);
  for (int k = 0; k < t.nk; ++k) {
    for (auto& kv : R[k]) {
      auto [ex, ey, ez] = kv.first;
      t.sh_pow.push_back(ex | (ey << 4) | (ez << 8));
      t.sh_coef.push_back(kv.second);
    }
    t.sh_ptr.push_back((int)t.sh_coef.size());
  }
  t.sh_dense.assign(sh_dense_off(L + 1), 0.0);
  for (int l = 0; l <= L; ++l)
    for (int m = 0; m < 2 * l + 1; ++m)
      for (auto& kv : R[l * l + m]) {
        auto [ex, ey, ez] = kv.first;
        if (ex + ey + ez != l) continue;  // never: R^(l) is homogeneous of degree l by its construction
        int q = 0;  // column of (ex, ey): the monomials of smaller ex, then ey
        for (int a = 0; a < ex; ++a) q += l - a + 1;
        q += ey;
        t.sh_dense[sh_dense_off(l) + m * sh_monos(l) + q] += kv.second;
      }

  // ---- j-side blocks, sorted by (a, b, d)
  int toff = 0;
  t.a_row_start.assign(L + 2, 0);
  for (int a = 0; a <= L; ++a) {
    t.a_row_start[a] = toff;
    for (int b = 0; b <= L; ++b)
      for (int d = std::abs(a - b); d <= a + b; ++d)
        if (block_used(L, a, b, d)) {
          t.blocks.push_back({a, b, d, toff});
          toff += 2 * d + 1;
        }
  }
  t.a_row_start[L + 1] = toff;
  t.dimT = toff;

  // ---- j-side matrix M: T[r] = sum_al M[r][al] h^(a)[al],  M[r][al] = sum_be C^{d de}_{a al, b be} R^(b)_be
  t.m_rowoff.push_back(0);
  t.m_ptr.push_back(0);
  for (const Block& B : t.blocks) {
    const auto& c = CG(B.a, B.b, B.d);
    for (int de = 0; de < 2 * B.d + 1; ++de) {
      for (int al = 0; al < 2 * B.a + 1; ++al) {
        for (int be = 0; be < 2 * B.b + 1; ++be) {
          double w = c[((size_t)al * (2 * B.b + 1) + be) * (2 * B.d + 1) + de];
          if (w == 0.0) continue;
          t.m_ridx.push_back(B.b * B.b + be);
          t.m_coef.push_back(w);
        }
        t.m_ptr.push_back((int)t.m_coef.size());
      }
      t.m_rowoff.push_back(t.m_rowoff.back() + 2 * B.a + 1);
    }
  }

  // ---- the same CG entries by row, for the coupling after aggregation
  t.ag_ptr.assign(1, 0);
  for (int r = 0; r < t.dimT; ++r) {
    const int s0 = t.m_rowoff[r], s1 = t.m_rowoff[r + 1];
    const int a = (s1 - s0 - 1) / 2;
    for (int sl = s0; sl < s1; ++sl)
      for (int e = t.m_ptr[sl]; e < t.m_ptr[sl + 1]; ++e) {
        t.ag_idx.push_back((t.m_ridx[e] << 6) | (a * a + sl - s0));
        t.ag_coef.push_back((float)t.m_coef[e]);
      }
    t.ag_ptr.push_back((int)t.ag_idx.size());
  }

  // ---- i-side matrices Q_o: y^(o)[m] = sum_cols Q_o[m][col] S[col]
  t.q_ncol.assign(L1, 0);
  t.q_coloff.assign(L1 + 1, 0);
  t.q_slotoff.assign(L1 + 1, 0);
  t.q_ptr.push_back(0);
  for (int o = 0; o <= L; ++o) {
    t.q_coloff[o] = (int)t.q_cols.size();
    t.q_slotoff[o] = (int)t.q_ptr.size() - 1;
    std::vector<const Block*> comp;
    for (const Block& B : t.blocks) {
      bool ok = false;
      for (int u = 0; u <= L - B.b; ++u) ok = ok || (tri(B.a, B.b + u, o) && tri(u, B.d, o));
      if (ok) comp.push_back(&B);
    }
    for (const Block* B : comp)
      for (int de = 0; de < 2 * B->d + 1; ++de) t.q_cols.push_back(B->toff + de);
    const int ncol = (int)t.q_cols.size() - t.q_coloff[o];
    t.q_ncol[o] = ncol;
    t.max_qslots = std::max(t.max_qslots, (2 * o + 1) * ncol);
    for (int m = 0; m < 2 * o + 1; ++m)
      for (const Block* B : comp)
        for (int de = 0; de < 2 * B->d + 1; ++de) {
          for (int u = 0; u <= L - B->b; ++u) {
            const int f = B->b + u;
            if (!tri(B->a, f, o) || !tri(u, B->d, o)) continue;
            double binom = 1.0;
            for (int s = 1; s <= u; ++s) binom = binom * (f - u + s) / s;
            const double K = ((B->b & 1) ? -1.0 : 1.0) * binom * recoupling_weight(B->a, B->b, u, o, B->d);
            if (K == 0.0) continue;
            const auto& c = CG(u, B->d, o);
            for (int ga = 0; ga < 2 * u + 1; ++ga) {
              double w = c[((size_t)ga * (2 * B->d + 1) + de) * (2 * o + 1) + m];
              if (w == 0.0) continue;
              t.q_ridx.push_back(u * u + ga);
              t.q_path.push_back((B->a * L1 + f) * L1 + o);
              t.q_unit.push_back(K * w);
            }
          }
          t.q_ptr.push_back((int)t.q_unit.size());
        }
  }
  t.q_coloff[L1] = (int)t.q_cols.size();
  t.q_slotoff[L1] = (int)t.q_ptr.size() - 1;
  // ---- build schedules of the per-node matrices
  {
    // node TP: one chunk over all degrees, transposed per-degree matrices
    t.tp_rs.assign(L + 1, 0);
    t.tp_mo.assign(L + 2, 0);
    for (int a = 0; a <= L; ++a) {
      int rs = (t.a_row_start[a + 1] - t.a_row_start[a] + 15) / 16 * 16;
      if ((rs / 16) % 2 == 0) rs += 16;
      t.tp_rs[a] = rs;
      t.tp_mo[a + 1] = t.tp_mo[a] + (2 * a + 1) * rs;
    }
    std::vector<std::vector<Slot>> chunks(1);
    for (int a = 0; a <= L; ++a)
      for (int r = t.a_row_start[a]; r < t.a_row_start[a + 1]; ++r)
        for (int al = 0; al < 2 * a + 1; ++al) {
          const int s = t.m_rowoff[r] + al;
          Slot sl{t.tp_mo[a] + al * t.tp_rs[a] + (r - t.a_row_start[a]), {}};
          for (int e = t.m_ptr[s]; e < t.m_ptr[s + 1]; ++e) sl.e.push_back({t.m_ridx[e], -1, t.m_coef[e]});
          chunks[0].push_back(std::move(sl));
        }
    t.tp_sched = make_schedule(chunks);
    // recouple: chunks of rc_rows T rows; Q rows padded to rc_qstride
    const int QS = rc_qstride(t.nk), RR = rc_rows(t.nk);
    std::vector<std::vector<Slot>> rchunks((t.dimT + RR - 1) / RR);
    for (int o = 0; o <= L; ++o) {
      const int ncol = t.q_ncol[o];
      for (int m = 0; m < 2 * o + 1; ++m)
        for (int col = 0; col < ncol; ++col) {
          const int s = t.q_slotoff[o] + m * ncol + col;
          const int row = t.q_cols[t.q_coloff[o] + col];
          Slot sl{(row % RR) * QS + o * o + m, {}};
          for (int e = t.q_ptr[s]; e < t.q_ptr[s + 1]; ++e) sl.e.push_back({t.q_ridx[e], t.q_path[e], t.q_unit[e]});
          rchunks[row / RR].push_back(std::move(sl));
        }
    }
    t.rc_sched = make_schedule(rchunks);
    // per filter degree f: the entries of the same slots whose u = f - b
    std::vector<int> row_b(t.dimT, 0);
    for (const Block& B : t.blocks)
      for (int de = 0; de < 2 * B.d + 1; ++de) row_b[B.toff + de] = B.b;
    auto degree_of = [](int ridx) {  // ridx = u*u + gamma, gamma < 2u+1
      int u = 0;
      while ((u + 1) * (u + 1) <= ridx) ++u;
      return u;
    };
    t.rcf_sched.clear();
    for (int f = 0; f <= L; ++f) {
      std::vector<std::vector<Slot>> fchunks((t.dimT + RR - 1) / RR);
      for (int o = 0; o <= L; ++o) {
        const int ncol = t.q_ncol[o];
        for (int m = 0; m < 2 * o + 1; ++m)
          for (int col = 0; col < ncol; ++col) {
            const int s = t.q_slotoff[o] + m * ncol + col;
            const int row = t.q_cols[t.q_coloff[o] + col];
            Slot sl{(row % RR) * QS + o * o + m, {}};
            for (int e = t.q_ptr[s]; e < t.q_ptr[s + 1]; ++e)
              if (row_b[row] + degree_of(t.q_ridx[e]) == f) sl.e.push_back({t.q_ridx[e], t.q_path[e], t.q_unit[e]});
            if (!sl.e.empty()) fchunks[row / RR].push_back(std::move(sl));
          }
      }
      t.rcf_sched.push_back(make_schedule(fchunks));
    }
  }

  // ---- edge filter K[k][q] = sum_f w_afo sum_mf C^{o m}_{a al, f mf} R^(f)_mf(r_ij)
  t.k_ptr.push_back(0);
  for (int o = 0; o <= L; ++o)
    for (int m = 0; m < 2 * o + 1; ++m)
      for (int a = 0; a <= L; ++a)
        for (int al = 0; al < 2 * a + 1; ++al) {
          for (int f = 0; f <= L; ++f) {
            if (!tri(a, f, o)) continue;
            const auto& c = CG(a, f, o);
            for (int mf = 0; mf < 2 * f + 1; ++mf) {
              double w = c[((size_t)al * (2 * f + 1) + mf) * (2 * o + 1) + m];
              if (w == 0.0) continue;
              t.k_ridx.push_back(f * f + mf);
              t.k_path.push_back((a * L1 + f) * L1 + o);
              t.k_unit.push_back(w);
            }
          }
          t.k_ptr.push_back((int)t.k_unit.size());
        }
  return t;
}

CoupleSchedule couple_schedule(const LayerTables& t, int groups) {
  CoupleSchedule cs;
  cs.groups = groups;
  std::vector<int> order(t.dimT);
  for (int r = 0; r < t.dimT; ++r) order[r] = r;
  auto len = [&](int r) { return t.ag_ptr[r + 1] - t.ag_ptr[r]; };
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return len(x) > len(y); });
  std::vector<std::vector<int>> per(groups);
  std::vector<int> load(groups, 0);
  for (int r : order) {
    int best = 0;
    for (int g = 1; g < groups; ++g)
      if (load[g] < load[best]) best = g;
    per[best].push_back(r);
    load[best] += std::max(1, len(r));  // an empty row still stores its zero
  }
  int K = 0;
  for (int g = 0; g < groups; ++g) K = std::max(K, load[g]);
  cs.k = K;
  cs.meta.assign((size_t)K * groups, 0);
  cs.coef.assign((size_t)K * groups, 0.0f);
  for (int g = 0; g < groups; ++g) {
    int k = 0;
    for (int r : per[g]) {
      const int a0 = t.ag_ptr[r], a1 = t.ag_ptr[r + 1];
      if (a0 == a1) {  // no entry: store 0
        cs.meta[(size_t)k * groups + g] = (r << 12) | (int)0x80000000u;
        ++k;
        continue;
      }
      for (int e = a0; e < a1; ++e, ++k) {
        const bool last = e + 1 == a1;
        cs.meta[(size_t)k * groups + g] = t.ag_idx[e] | (r << 12) | (last ? (int)0x80000000u : 0);
        cs.coef[(size_t)k * groups + g] = t.ag_coef[e];
      }
    }
  }
  if (t.dimT <= 512) {
    std::map<float, int> idx;  // exact values (padding entries carry 0.0f)
    cs.pmeta.resize(cs.meta.size());
    for (size_t q = 0; q < cs.meta.size(); ++q) {
      auto it = idx.emplace(cs.coef[q], (int)idx.size()).first;
      const int m = cs.meta[q];
      cs.pmeta[q] = (m & 0xfff) | (((m >> 12) & 511) << 12) | (it->second << 21) | (m & (int)0x80000000u);
    }
    if (idx.size() > 1024) {
      cs.pmeta.clear();
    } else {
      cs.tab.resize(idx.size());
      for (const auto& kv : idx) cs.tab[kv.second] = kv.first;
    }
  }
  return cs;
}

GeomSchedule geom_schedule(const LayerTables& t, int qc) {
  GeomSchedule gs;
  const int nk = t.nk, G = kGeomGroups;
  gs.qc = qc;
  gs.nchunk = (nk + qc - 1) / qc;
  // entries (k, unit, path) of each key (be, q), in ascending k
  struct Ent { int k, path; double unit; };
  std::vector<std::vector<Ent>> ent((size_t)nk * nk);
  for (int sidx = 0; sidx < nk * nk; ++sidx)
    for (int e = t.k_ptr[sidx]; e < t.k_ptr[sidx + 1]; ++e)
      ent[(size_t)t.k_ridx[e] * nk + sidx % nk].push_back({sidx / nk, t.k_path[e], t.k_unit[e]});
  for (int ch = 0; ch < gs.nchunk; ++ch) {
    const int q0 = ch * qc, nq = std::min(qc, nk - q0);
    std::vector<int> keys;
    for (int be = 0; be < nk; ++be)
      for (int qq = 0; qq < nq; ++qq) keys.push_back(be * nk + q0 + qq);
    auto len = [&](int key) { return std::max<int>(1, (int)ent[key].size()); };
    std::stable_sort(keys.begin(), keys.end(), [&](int x, int y) { return len(x) > len(y); });
    std::vector<std::vector<int>> per(G);
    std::vector<int> load(G, 0);
    for (int key : keys) {
      int best = 0;
      for (int g = 1; g < G; ++g)
        if (load[g] < load[best]) best = g;
      per[best].push_back(key);
      load[best] += len(key);
    }
    const int K = *std::max_element(load.begin(), load.end());
    const size_t base = gs.meta.size();
    gs.off.push_back((int)base);
    gs.ck.push_back(K);
    gs.meta.resize(base + (size_t)K * G, 0);
    gs.unit.resize(base + (size_t)K * G, 0.0f);
    for (int g = 0; g < G; ++g) {
      int k = 0;
      for (int key : per[g]) {
        const int be = key / nk, qq = key % nk - q0;
        const int kb = (be << 6) | (qq << 12);
        if (ent[key].empty()) {
          gs.meta[base + (size_t)k * G + g] = kb | (int)0x80000000u;
          ++k;
          continue;
        }
        for (size_t e = 0; e < ent[key].size(); ++e, ++k) {
          const bool last = e + 1 == ent[key].size();
          gs.meta[base + (size_t)k * G + g] =
              ent[key][e].k | kb | (ent[key][e].path << 18) | (last ? (int)0x80000000u : 0);
          gs.unit[base + (size_t)k * G + g] = (float)ent[key][e].unit;
        }
      }
    }
  }
  return gs;
}

FuseTable fuse_table(const LayerTables& t, const std::vector<double>& w, const int* degs, int nd, int nkr) {
  const int nk = t.nk;
  FuseTable ft;
  if (t.L > kFuseMaxL || nkr < fuse_krows(nk, degs, nd)) return ft;
  // first K row of each filter degree's segment (-1: not in this table),
  // and of the segment that takes every term (the plain layer: b + u up to 2L)
  int start[kFuseMaxL + 1], start_all = -1;
  for (int f = 0; f <= kFuseMaxL; ++f) start[f] = -1;
  for (int s = 0, r = 0; s < nd; ++s) {
    if (degs[s] < 0) start_all = r;
    else start[degs[s]] = r;
    r += degs[s] < 0 ? nk : (degs[s] + 1) * (degs[s] + 1);
  }
  std::vector<int> row_b(t.dimT, 0);  // j-side degree of every T row
  for (const Block& B : t.blocks)
    for (int de = 0; de < 2 * B.d + 1; ++de) row_b[B.toff + de] = B.b;
  // dense K[pos][x], accumulated over the T rows r that link a recouple entry
  // (k, r) with a coupling entry (r, be, q)
  const int np = fuse_stride(nk, nkr);
  std::vector<double> K((size_t)np * nk, 0.0), mag((size_t)np * nk, 0.0);
  for (int o = 0; o <= t.L; ++o) {
    const int ncol = t.q_ncol[o];
    for (int m = 0; m < 2 * o + 1; ++m)
      for (int col = 0; col < ncol; ++col) {
        const int s = t.q_slotoff[o] + m * ncol + col;
        const int r = t.q_cols[t.q_coloff[o] + col];
        const int k = o * o + m;
        const int s0 = t.m_rowoff[r], s1 = t.m_rowoff[r + 1];
        const int a = (s1 - s0 - 1) / 2;
        for (int e = t.q_ptr[s]; e < t.q_ptr[s + 1]; ++e) {
          const double cq = t.q_unit[e] * w[t.q_path[e]];
          const int x = t.q_ridx[e];
          int u = 0;  // x = u^2 + gamma: the degree of the receiver's harmonic
          while ((u + 1) * (u + 1) <= x) ++u;
          const int deg = row_b[r] + u;
          int shift = start_all;  // K row of a j-side component be: shift + be
          if (shift < 0) {
            if (deg > kFuseMaxL || start[deg] < 0) continue;
            shift = start[deg];
          }
          for (int sl = s0; sl < s1; ++sl)
            for (int e2 = t.m_ptr[sl]; e2 < t.m_ptr[sl + 1]; ++e2) {
              const size_t at = (size_t)fuse_pos(nk, nkr, k, t.m_ridx[e2] + shift, a * a + sl - s0) * nk + x;
              K[at] += cq * t.m_coef[e2];
              mag[at] += std::fabs(cq * t.m_coef[e2]);
            }
        }
      }
  }
  // sums that cancel to rounding level are zeros of the exact tensor
  ft.ptr.assign(1, 0);
  for (int p = 0; p < np; ++p) {
    for (int x = 0; x < nk; ++x) {
      const double v = K[(size_t)p * nk + x];
      if (v != 0.0 && std::fabs(v) > 1e-13 * mag[(size_t)p * nk + x]) {
        ft.idx.push_back(x);
        ft.coef.push_back(v);
      }
    }
    ft.ptr.push_back((int)ft.idx.size());
  }
  return ft;
}

}  // namespace e2f
