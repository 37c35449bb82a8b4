// Host check of the fused recouple tables (built with g++ against the
// library's tables.cpp by test_fuse_tables.py; no GPU).  For L = 0 .. 4 and
// random path weights it verifies that
//   * the table of filter degree f has entries only at K rows be < (f+1)^2
//     (the terms of degree f = b + u read the j-side components of degree
//     b <= f);
//   * the per-degree tables sum to the plain layer's table (the degrees f =
//     0 .. L partition its terms);
//   * each pass of ynorm_passes (its degrees in segments of (f+1)^2 K rows)
//     equals the per-degree tables moved to the segment's rows, entry by
//     entry, with nothing else in it, and the passes cover every degree once.
// Prints one line per check, "ok" or "FAIL", and exits 1 on a failure.
#include <cmath>
#include <cstdio>
#include <random>
#include "e2f_internal.h"

using namespace e2f;

static std::vector<double> dense(const FuseTable& ft, int np, int nk, bool& ok) {
  std::vector<double> D((size_t)np * nk, 0.0);
  if ((int)ft.ptr.size() != np + 1) {
    ok = false;
    return D;
  }
  for (int p = 0; p < np; ++p)
    for (int e = ft.ptr[p]; e < ft.ptr[p + 1]; ++e) D[(size_t)p * nk + ft.idx[e]] += ft.coef[e];
  return D;
}

int main() {
  bool all_ok = true;
  for (int L = 0; L <= kFuseMaxL; ++L) {
    const LayerTables t = build_layer_tables(L);
    const int nk = t.nk, np = fuse_stride(nk, nk);
    std::mt19937 g(11 + L);
    std::uniform_real_distribution<double> U(0.2, 1.0);
    std::vector<double> w((size_t)(L + 1) * (L + 1) * (L + 1));
    for (double& v : w) v = U(g);
    bool ok = true;
    const int all[1] = {-1};
    const std::vector<double> full = dense(fuse_table(t, w, all, 1, nk), np, nk, ok);
    std::vector<std::vector<double>> ff;
    for (int f = 0; f <= L; ++f) ff.push_back(dense(fuse_table(t, w, &f, 1, nk), np, nk, ok));
    // degree f only at K rows be < (f+1)^2
    size_t outside = 0;
    for (int f = 0; f <= L; ++f)
      for (int k = 0; k < nk; ++k)
        for (int be = (f + 1) * (f + 1); be < nk; ++be)
          for (int q = 0; q < nk; ++q)
            for (int x = 0; x < nk; ++x)
              if (ff[f][(size_t)fuse_pos(nk, nk, k, be, q) * nk + x] != 0.0) ++outside;
    double dsum = 0.0, fmax = 0.0;
    for (size_t a = 0; a < full.size(); ++a) {
      double s = 0.0;
      for (int f = 0; f <= L; ++f) s += ff[f][a];
      dsum = std::max(dsum, std::fabs(s - full[a]));
      fmax = std::max(fmax, std::fabs(full[a]));
    }
    const bool ok1 = ok && outside == 0 && fmax > 0.0 && dsum <= 1e-12 * fmax;
    std::printf("L=%d per-degree rows and sum: %s (entries outside %zu, |sum - plain| %.3e of %.3e)\n", L,
                ok1 ? "ok" : "FAIL", outside, dsum, fmax);
    all_ok = all_ok && ok1;
    YnormPass yps[kYnormMaxPasses];
    const int nyp = ynorm_passes(L, yps);
    std::vector<int> seen(L + 1, 0);
    for (int q = 0; q < nyp; ++q)
      for (int s = 0; s < yps[q].nd; ++s) ++seen[yps[q].degs[s]];
    bool cover = true;
    for (int f = 0; f <= L; ++f) cover = cover && seen[f] == 1;
    std::printf("L=%d passes cover every degree once: %s\n", L, cover ? "ok" : "FAIL");
    all_ok = all_ok && cover;
    for (int q = 0; q < nyp; ++q) {
      const YnormPass& yp = yps[q];
      const int nkr = fuse_krows(nk, yp.degs, yp.nd);
      bool okp = true;
      const std::vector<double> P = dense(fuse_table(t, w, yp.degs, yp.nd, nkr), fuse_stride(nk, nkr), nk, okp);
      std::vector<char> hit(P.size(), 0);
      double err = 0.0;
      for (int s = 0, st = 0; s < yp.nd; ++s) {
        const int f = yp.degs[s], nr = (f + 1) * (f + 1);
        for (int k = 0; k < nk; ++k)
          for (int be = 0; be < nr; ++be)
            for (int qq = 0; qq < nk; ++qq)
              for (int x = 0; x < nk; ++x) {
                const size_t a = (size_t)fuse_pos(nk, nkr, k, st + be, qq) * nk + x;
                err = std::max(err, std::fabs(P[a] - ff[f][(size_t)fuse_pos(nk, nk, k, be, qq) * nk + x]));
                hit[a] = 1;
              }
        st += nr;
      }
      size_t stray = 0;
      for (size_t a = 0; a < P.size(); ++a)
        if (!hit[a] && P[a] != 0.0) ++stray;
      const bool ok2 = okp && err == 0.0 && stray == 0;
      std::printf("L=%d stacked pass %d (%d K rows): %s (max diff %.3e, stray entries %zu)\n", L, q, nkr,
                  ok2 ? "ok" : "FAIL", err, stray);
      all_ok = all_ok && ok2;
    }
  }
  return all_ok ? 0 : 1;
}
