"""Pins of the fp64 oracle against closed forms and invariants (CPU only).

Each test names the passage of arXiv 2501.19216 (or the textbook identity)
that fixes the expected value.  A plausible mistake anywhere in the oracle
(a dropped term, a wrong sign or index, a transposed operand) fails one of
them.
"""
import itertools
import math
import os

import numpy as np
import pytest
from scipy.special import lpmv

import e2f_synth as syn
import oracle as o


def tri(a, b, c):
    return abs(a - b) <= c <= a + b


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.lstrip().startswith("#")]


# ---------------------------------------------------------------- 3j / CG
def test_wigner_symbols_tabulated():
    # tests/golden/wigner_symbols_tabulated.txt: exact tabulated 3j and 6j values
    rows = golden_lines("wigner_symbols_tabulated.txt")
    assert len(rows) >= 9
    for r in rows:
        j = [int(v) for v in r[1:7]]
        sign, num, den = int(r[7]), int(r[8]), int(r[9])
        want = sign * math.sqrt(num / den)
        got = o.wigner3j(*j) if r[0] == "3j" else o.wigner6j(*j)
        assert got == pytest.approx(want, abs=1e-15), r


def test_3j_textbook_values():
    assert o.cg_complex(1, 0, 1, 0, 0, 0) == pytest.approx(-1 / math.sqrt(3), abs=1e-15)
    assert o.cg_complex(1, 1, 1, 0, 2, 1) == pytest.approx(1 / math.sqrt(2), abs=1e-15)
    # selection rules (App. C.1)
    assert o.wigner3j(1, 1, 1, 1, 0, 0) == 0.0
    assert o.wigner3j(1, 1, 3, 0, 0, 0) == 0.0


def test_3j_special_closed_forms():
    for j in range(0, 9):
        for m in range(-j, j + 1):
            # (j j 0; m -m 0) = (-1)^(j-m)/sqrt(2j+1)
            assert o.wigner3j(j, j, 0, m, -m, 0) == pytest.approx((-1) ** (j - m) / math.sqrt(2 * j + 1), abs=1e-14)
    f = math.factorial
    for j1, j2 in itertools.product(range(5), range(5)):
        J = j1 + j2
        for m1 in range(-j1, j1 + 1):
            for m2 in range(-j2, j2 + 1):
                M = m1 + m2
                # stretched coupling, closed form
                v = (-1) ** (j1 - j2 + M) * math.sqrt(f(2 * j1) * f(2 * j2) * f(J + M) * f(J - M) /
                                                     (f(2 * J + 1) * f(j1 + m1) * f(j1 - m1) * f(j2 + m2) * f(j2 - m2)))
                assert o.wigner3j(j1, j2, J, m1, m2, -M) == pytest.approx(v, abs=1e-14)
    # coupling with j2 = 1, m2 = 0 (Condon-Shortley closed forms)
    for j in range(1, 9):
        for m in range(-j, j + 1):
            assert o.cg_complex(j, m, 1, 0, j + 1, m) == pytest.approx(
                math.sqrt((j - m + 1) * (j + m + 1) / ((2 * j + 1) * (j + 1))), abs=1e-14)
            assert o.cg_complex(j, m, 1, 0, j, m) == pytest.approx(m / math.sqrt(j * (j + 1)), abs=1e-14)
            assert o.cg_complex(j, m, 1, 0, j - 1, m) == pytest.approx(
                -math.sqrt((j - m) * (j + m) / (j * (2 * j + 1))), abs=1e-14)


def test_3j_symmetries_and_orthogonality():
    # App. C.1: column permutations, m reversal, both orthogonality sums
    for j1, j2, j3 in itertools.product(range(5), repeat=3):
        if not tri(j1, j2, j3):
            continue
        ph = (-1) ** (j1 + j2 + j3)
        for m1 in range(-j1, j1 + 1):
            for m2 in range(-j2, j2 + 1):
                m3 = -m1 - m2
                if abs(m3) > j3:
                    continue
                v = o.wigner3j(j1, j2, j3, m1, m2, m3)
                assert o.wigner3j(j2, j3, j1, m2, m3, m1) == pytest.approx(v, abs=1e-14)
                assert o.wigner3j(j2, j1, j3, m2, m1, m3) == pytest.approx(ph * v, abs=1e-14)
                assert o.wigner3j(j1, j2, j3, -m1, -m2, -m3) == pytest.approx(ph * v, abs=1e-14)
    for j1, j2 in itertools.product(range(4), repeat=2):
        for j3 in range(abs(j1 - j2), j1 + j2 + 1):
            for j3p in range(abs(j1 - j2), j1 + j2 + 1):
                for m3 in range(-j3, j3 + 1):
                    for m3p in range(-j3p, j3p + 1):
                        s = sum((2 * j3 + 1) * o.wigner3j(j1, j2, j3, m1, m2, m3) * o.wigner3j(j1, j2, j3p, m1, m2, m3p)
                                for m1 in range(-j1, j1 + 1) for m2 in range(-j2, j2 + 1))
                        assert s == pytest.approx(float(j3 == j3p and m3 == m3p), abs=1e-13)
        for m1, m2, m1p, m2p in itertools.product(range(-j1, j1 + 1), range(-j2, j2 + 1), range(-j1, j1 + 1), range(-j2, j2 + 1)):
            s = sum((2 * j3 + 1) * o.wigner3j(j1, j2, j3, m1, m2, m3) * o.wigner3j(j1, j2, j3, m1p, m2p, m3)
                    for j3 in range(abs(j1 - j2), j1 + j2 + 1) for m3 in range(-j3, j3 + 1))
            assert s == pytest.approx(float(m1 == m1p and m2 == m2p), abs=1e-13)


# ---------------------------------------------------------------- solid harmonics
def sh_closed_form(lmax, v):
    """Real regular solid harmonics from associated Legendre functions
    (Def. 2.1 case formula): R^(l)_m = sqrt(l!/(2l-1)!!) * C_lm with the
    Racah-normalised C_lm = sqrt(4pi/(2l+1)) r^l Y_lm, sin for m<0, cos
    for m>0, and no Condon-Shortley sign."""
    x, y, z = v
    r = math.sqrt(x * x + y * y + z * z)
    ct = z / r
    phi = math.atan2(y, x)
    out = []
    for l in range(lmax + 1):
        dfact = 1
        for k in range(2 * l - 1, 0, -2):
            dfact *= k
        s = math.sqrt(math.factorial(l) / dfact)
        for m in range(-l, l + 1):
            am = abs(m)
            P = (-1) ** am * lpmv(am, l, ct)  # remove scipy's Condon-Shortley phase
            if m == 0:
                c = r ** l * P
            else:
                nrm = math.sqrt(2.0 * math.factorial(l - am) / math.factorial(l + am))
                c = nrm * r ** l * P * (math.cos(am * phi) if m > 0 else math.sin(am * phi))
            out.append(s * c)
    return np.array(out)


def test_solid_harmonics_closed_form():
    rng = np.random.default_rng(11)
    for _ in range(20):
        v = rng.standard_normal(3) * rng.uniform(0.3, 3.0)
        got = o.solid_harmonics(6, v)
        ref = sh_closed_form(6, v)
        assert np.max(np.abs(got - ref)) <= 1e-11 * max(1.0, np.max(np.abs(ref)))


def test_solid_harmonics_paper_shapes():
    # Def. 2.1: R^(1)(v) proportional to (y, z, x); the degree-2 example the
    # paper prints (tests/golden/real_sh_degree2_cartesian.txt): each R^(2)_m
    # is a fixed positive multiple of its Cartesian form
    v = np.array([0.37, -1.21, 0.83])
    x, y, z = v
    R = o.solid_harmonics(2, v)
    assert np.allclose(R[1:4], [y, z, x], atol=1e-15)
    forms = {}
    for r in golden_lines("real_sh_degree2_cartesian.txt"):
        terms = []
        for tok in r[1:]:
            c, e = tok.split(":")
            terms.append((float(c), [int(k) for k in e.split(",")]))
        forms[int(r[0])] = terms
    assert sorted(forms) == [-2, -1, 0, 1, 2]

    def form(m, p):
        return sum(c * p[0] ** e[0] * p[1] ** e[1] * p[2] ** e[2] for c, e in forms[m])

    rng = np.random.default_rng(7)
    pts = rng.standard_normal((6, 3))
    for m in range(-2, 3):
        ratios = [o.solid_harmonics(2, p)[4 + m + 2] / form(m, p) for p in pts]
        assert min(ratios) > 0 and max(ratios) - min(ratios) <= 1e-12 * max(ratios), (m, ratios)
    # the constants of the stretched-power convention (C_l scaled by sqrt(l!/(2l-1)!!))
    scale = np.array([math.sqrt(2), math.sqrt(2), 1 / math.sqrt(6), math.sqrt(2), 1 / math.sqrt(2)])
    assert np.allclose(R[4:9], scale * np.array([form(m, v) for m in range(-2, 3)]), atol=1e-14)
    # value on the z axis: R^(l)_0(z) = sqrt(l!/(2l-1)!!)
    Rz = o.solid_harmonics(6, np.array([0.0, 0.0, 1.0]))
    for l in range(7):
        dfact = 1
        for k in range(2 * l - 1, 0, -2):
            dfact *= k
        assert Rz[l * l + l] == pytest.approx(math.sqrt(math.factorial(l) / dfact), abs=1e-14)
    assert Rz[2 * 2 + 2] == pytest.approx(math.sqrt(2.0 / 3.0), abs=1e-15)


def test_solid_harmonics_invariants():
    rng = np.random.default_rng(5)
    p, q = rng.standard_normal(3), rng.standard_normal(3)
    # R^(1) is linear: R1(p - q) = R1(p) - R1(q) (Def. 2.1), and only l = 1 is
    Rp, Rq, Rpq = o.solid_harmonics(3, p), o.solid_harmonics(3, q), o.solid_harmonics(3, p - q)
    assert np.allclose(Rpq[1:4], Rp[1:4] - Rq[1:4], atol=1e-14)
    assert not np.allclose(Rpq[4:9], Rp[4:9] - Rq[4:9], atol=1e-3)
    v = rng.standard_normal(3)
    R = o.solid_harmonics(6, v)
    for l in range(7):
        s = slice(l * l, (l + 1) ** 2)
        # homogeneity and parity
        assert np.allclose(o.solid_harmonics(6, 1.7 * v)[s], 1.7 ** l * R[s], rtol=1e-13, atol=1e-13)
        assert np.allclose(o.solid_harmonics(6, -v)[s], (-1) ** l * R[s], atol=1e-13)
        # squared norm = l!/(2l-1)!! |v|^(2l)
        dfact = 1
        for k in range(2 * l - 1, 0, -2):
            dfact *= k
        assert np.sum(R[s] ** 2) == pytest.approx(math.factorial(l) / dfact * (v @ v) ** l, rel=1e-13)
    # harmonic: the Laplacian vanishes (central differences, fp64)
    h = 1e-3
    lap = -6 * R
    for k in range(3):
        e = np.zeros(3)
        e[k] = h
        lap = lap + o.solid_harmonics(6, v + e) + o.solid_harmonics(6, v - e)
    assert np.max(np.abs(lap / (h * h))) < 1e-4


def test_binomial_local_expansion():
    # Thm. 3.2: R^(l)(p - q) = sum_u (-1)^(l-u) binom(l,u) [R^(u)(p) (x) R^(l-u)(q)]^(l)
    rng = np.random.default_rng(2)
    for l in range(7):
        for _ in range(3):
            p, q = rng.standard_normal(3) * 2, rng.standard_normal(3) * 2
            Rp, Rq = o.solid_harmonics(6, p), o.solid_harmonics(6, q)
            acc = np.zeros(2 * l + 1)
            for u in range(l + 1):
                c = o.cg_real(u, l - u, l)
                acc += (-1) ** (l - u) * math.comb(l, u) * np.einsum(
                    "abc,a,b->c", c, Rp[u * u:(u + 1) ** 2], Rq[(l - u) ** 2:(l - u + 1) ** 2])
            ref = o.solid_harmonics(l, p - q)[l * l:]
            assert np.max(np.abs(acc - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


# ---------------------------------------------------------------- real CG
def closed_form_d(lmax, Q):
    """Wigner D^(l)(Q) fitted from the Legendre closed-form harmonics
    (independent of the oracle's CG tables)."""
    rng = np.random.default_rng(3)
    v = rng.standard_normal((40, 3))
    A = np.array([sh_closed_form(lmax, x) for x in v])
    B = np.array([sh_closed_form(lmax, Q @ x) for x in v])
    Ds = []
    for l in range(lmax + 1):
        s = slice(l * l, (l + 1) ** 2)
        Dt, *_ = np.linalg.lstsq(A[:, s], B[:, s], rcond=None)
        Ds.append(Dt.T)
    return Ds


def test_real_cg_orthogonal_and_equivariant():
    Q = o.random_rotation(17)
    D = closed_form_d(4, Q)
    # l = 1 is the rotation matrix itself in (y, z, x) order
    P = np.array([[0, 1, 0], [0, 0, 1], [1, 0, 0]])
    assert np.allclose(D[1], P @ Q @ P.T, atol=1e-12)
    for l1, l2 in itertools.product(range(5), repeat=2):
        blocks = []
        for l3 in range(abs(l1 - l2), l1 + l2 + 1):
            c = o.cg_real(l1, l2, l3)  # raises if the real/imaginary split fails
            M = c.reshape(-1, 2 * l3 + 1)
            assert np.allclose(M.T @ M, np.eye(2 * l3 + 1), atol=1e-13)
            blocks.append(M)
            if l3 <= 4:
                # coupling commutes with rotation: C(D1 x, D2 y) = D3 C(x, y)
                lhs = np.einsum("ia,jb,ijk->abk", D[l1], D[l2], c)
                rhs = np.einsum("kq,abq->abk", D[l3], c)
                assert np.max(np.abs(lhs - rhs)) < 1e-10, (l1, l2, l3)
        full = np.concatenate(blocks, axis=1)  # completeness: square orthogonal
        assert np.allclose(full @ full.T, np.eye(full.shape[0]), atol=1e-13)
    for l1, l2, l3 in itertools.product(range(4), repeat=3):
        if tri(l1, l2, l3):
            # swap symmetry inherited from the complex basis
            a, b = o.cg_real(l1, l2, l3), o.cg_real(l2, l1, l3)
            assert np.allclose(a, (-1) ** (l1 + l2 - l3) * b.transpose(1, 0, 2), atol=1e-14)


# ---------------------------------------------------------------- 6j and X
def sixj_from_3j(j1, j2, j3, j4, j5, j6):
    """6j as the contraction of four 3j symbols (standard form)."""
    s = 0.0
    for m1, m2, m4, m5 in itertools.product(range(-j1, j1 + 1), range(-j2, j2 + 1), range(-j4, j4 + 1), range(-j5, j5 + 1)):
        m3 = -m1 - m2  # from the first symbol (-m1 -m2 -m3)
        m6 = m5 - m1   # from (j1 j5 j6; m1 -m5 m6)
        if abs(m3) > j3 or abs(m6) > j6:
            continue
        ph = (-1) ** (j1 + j2 + j3 + j4 + j5 + j6 - m1 - m2 - m3 - m4 - m5 - m6)
        s += ph * (o.wigner3j(j1, j2, j3, -m1, -m2, -m3) * o.wigner3j(j1, j5, j6, m1, -m5, m6) *
                   o.wigner3j(j4, j2, j6, m4, m2, -m6) * o.wigner3j(j4, j5, j3, -m4, m5, m3))
    return s


def test_6j_against_four_3j_sum():
    for js in [(1, 1, 1, 1, 1, 1), (2, 1, 1, 1, 2, 2), (2, 2, 2, 2, 2, 2), (3, 2, 1, 2, 3, 2), (1, 2, 3, 3, 2, 1),
               (2, 3, 3, 1, 2, 2), (4, 2, 2, 2, 4, 2), (3, 3, 2, 2, 1, 3)]:
        assert o.wigner6j(*js) == pytest.approx(sixj_from_3j(*js), abs=1e-13), js


def test_6j_special_value_symmetries_orthogonality():
    for a, b, c in itertools.product(range(5), repeat=3):
        if tri(a, b, c):
            # {a b c; 0 c b} = (-1)^(a+b+c) / sqrt((2b+1)(2c+1))
            assert o.wigner6j(a, b, c, 0, c, b) == pytest.approx((-1) ** (a + b + c) / math.sqrt((2 * b + 1) * (2 * c + 1)), abs=1e-14)
    # App. C.2: the 24 tetrahedral symmetries
    rng = np.random.default_rng(0)
    for _ in range(30):
        j = [int(x) for x in rng.integers(0, 5, size=6)]
        v = o.wigner6j(*j)
        cols = [(j[0], j[3]), (j[1], j[4]), (j[2], j[5])]
        for perm in itertools.permutations(range(3)):
            pc = [cols[k] for k in perm]
            for flip in [(), (0, 1), (0, 2), (1, 2)]:
                cc = [(c[1], c[0]) if k in flip else c for k, c in enumerate(pc)]
                assert o.wigner6j(cc[0][0], cc[1][0], cc[2][0], cc[0][1], cc[1][1], cc[2][1]) == pytest.approx(v, abs=1e-14)
    # App. C.2 orthogonality
    for j1, j2, j4, j5 in itertools.product(range(4), repeat=4):
        for j6 in range(0, 7):
            for j6p in range(0, 7):
                s = sum((2 * j3 + 1) * (2 * j6 + 1) * o.wigner6j(j1, j2, j3, j4, j5, j6) * o.wigner6j(j1, j2, j3, j4, j5, j6p)
                        for j3 in range(0, 8))
                want = float(j6 == j6p and tri(j1, j5, j6) and tri(j4, j2, j6))
                assert s == pytest.approx(want, abs=1e-12)


def test_recoupling_weights():
    rng = np.random.default_rng(9)
    L = 4
    for a, b, u in itertools.product(range(L + 1), repeat=3):
        f = b + u
        if f > L:
            continue
        for oo in range(abs(a - f), min(a + f, L) + 1):
            xs = {d: o.recoupling_x(a, b, u, oo, d) for d in range(abs(a - b), a + b + 1)}
            for d, x in xs.items():
                # closed form of Def. 2.3 with the standard phase (-1)^(a+b+d)
                # (the printed (-1)^(a+b+c+d) is a misprint), times -1 in the
                # real basis when a+b+d and u+d+o are both odd
                cf = (-1) ** (a + b + d) * math.sqrt((2 * d + 1) * (2 * f + 1)) * o.wigner6j(a, b, d, u, oo, f)
                if (a + b + d) % 2 and (u + d + oo) % 2:
                    cf = -cf
                assert x == pytest.approx(cf, abs=1e-12)
                if u == 0:
                    assert x == pytest.approx(float(d == oo), abs=1e-13)
                if b == 0:
                    assert x == pytest.approx(float(d == a) * (-1) ** (a + u - oo), abs=1e-13)
            # the recoupling identity on random tensors
            A, B, C = rng.standard_normal(2 * a + 1), rng.standard_normal(2 * b + 1), rng.standard_normal(2 * u + 1)
            cb = np.einsum("gbk,g,b->k", o.cg_real(u, b, f), C, B)
            lhs = np.einsum("ako,a,k->o", o.cg_real(a, f, oo), A, cb)
            rhs = np.zeros(2 * oo + 1)
            for d, x in xs.items():
                if tri(u, d, oo):
                    ab = np.einsum("abd,a,b->d", o.cg_real(a, b, d), A, B)
                    rhs += x * np.einsum("gdo,g,d->o", o.cg_real(u, d, oo), C, ab)
            assert np.allclose(lhs, rhs, atol=1e-12)


# ---------------------------------------------------------------- radius graph
def test_neighbor_list_exact_predicate_and_cells():
    rng = np.random.default_rng(4)
    pos = syn.quantize(rng.uniform(0, 12, size=(300, 3)))
    gid = rng.integers(0, 3, size=300).astype(np.int32)
    for g in [None, gid]:
        rp1, c1 = o.neighbor_list(pos, 3.0, g, method="brute")
        rp2, c2 = o.neighbor_list(pos, 3.0, g, method="cells")
        assert np.array_equal(rp1, rp2) and np.array_equal(c1, c2)
        pairs = set()
        for i in range(300):
            row = c1[rp1[i]:rp1[i + 1]]
            assert np.all(np.diff(row) > 0) and i not in row
            for j in row:
                pairs.add((i, int(j)))
                if g is not None:
                    assert g[i] == g[j]
        assert all((j, i) in pairs for (i, j) in pairs)
        # brute force in float64 on the grid agrees
        d2 = np.sum((pos[:, None, :].astype(np.float64) - pos[None, :, :]) ** 2, axis=2)
        want = (d2 < 9.0) & ~np.eye(300, dtype=bool)
        if g is not None:
            want &= g[:, None] == g[None, :]
        assert len(pairs) == int(want.sum())
    # strict inequality exactly at the cutoff on the grid
    two = np.array([[0, 0, 0], [0, 0, 3.0], [0, 3.0 - 2.0 ** -16, 0]], dtype=np.float32)
    rp, c = o.neighbor_list(two, 3.0)
    assert list(c[rp[0]:rp[1]]) == [2]


# ---------------------------------------------------------------- the layer
def small_graph(L, n, C, H, seed, box=4.0, cutoff=3.0):
    rng = np.random.default_rng(seed)
    pos = syn.quantize(rng.uniform(0, box, size=(n, 3)))
    rp, ci = o.neighbor_list(pos, cutoff)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.1, 1.0, size=(len(ci), H)).astype(np.float32)
    w = rng.uniform(0.5, 1.5, size=(L + 1) ** 3)
    return pos, rp, ci, feat, alpha, w


def test_attention_weights_closed_forms():
    """Attention weights (App. E): softmax over a row times the cosine envelope."""
    rng = np.random.default_rng(9)
    n, H, dk, R, rc = 60, 3, 4, 6, 5.0
    pos = syn.quantize(rng.uniform(0, 9, size=(n, 3)))
    rp, ci = o.neighbor_list(pos, rc)
    q = rng.standard_normal((n, H, dk)).astype(np.float32)
    k = rng.standard_normal((n, H, dk)).astype(np.float32)
    w = rng.standard_normal((H, R)).astype(np.float32)
    a = o.attention_weights(pos, q, k, w, rc, rp, ci)
    recv = np.repeat(np.arange(n), np.diff(rp))
    d = np.linalg.norm(pos[recv].astype(np.float64) - pos[ci], axis=1)
    env = 0.5 * (np.cos(np.pi * d / rc) + 1.0)
    # rows of alpha / envelope sum to one (every edge is inside the cutoff)
    s = np.zeros((n, H))
    np.add.at(s, recv, a / env[:, None])
    has = np.diff(rp) > 0
    assert np.allclose(s[has], 1.0, atol=2e-6)
    # equal logits (no q.k, no radial weights): envelope / degree
    z = o.attention_weights(pos, np.zeros_like(q), k, np.zeros_like(w), rc, rp, ci)
    assert np.allclose(z, (env / np.diff(rp)[recv])[:, None], rtol=1e-6)
    # one neighbour per row: the envelope alone
    rp1 = np.arange(n + 1, dtype=np.int64)
    ci1 = ((np.arange(n) + 1) % n).astype(np.int32)
    a1 = o.attention_weights(pos, q, k, w, 50.0, rp1, ci1)
    d1 = np.linalg.norm(pos.astype(np.float64) - pos[ci1], axis=1)
    assert np.allclose(a1, (0.5 * (np.cos(np.pi * d1 / 50.0) + 1.0))[:, None], rtol=1e-6)
    # beyond the cutoff the weight is zero
    a2 = o.attention_weights(pos, q, k, w, 0.5 * float(d1.min()), rp1, ci1)
    assert np.all(a2 == 0)
    # invariant under rotations and translations (logits depend on distances only)
    Q = o.random_rotation(3)
    pr = (pos.astype(np.float64) @ Q.T + 11.0).astype(np.float32)
    assert np.allclose(o.attention_weights(pr, q, k, w, rc, rp, ci), a, atol=1e-5)
    # the synthetic generator's weights are the case dk = 1, q = k = species embedding
    species = rng.integers(0, 5, size=n)
    ref = syn.attention_weights(pos, species, rp, ci, H, rc, 5, 17)
    g = np.random.default_rng(0xA1FA0000 + 17)
    emb = g.standard_normal((5, H))
    rho = g.standard_normal((H, 8)) / math.sqrt(8.0)
    e = emb[species][:, :, None].astype(np.float32)
    got = o.attention_weights(pos, e, e, rho.astype(np.float32), rc, rp, ci)
    assert np.allclose(got, ref, rtol=1e-5, atol=1e-7)


@pytest.mark.parametrize("L", [0, 2, 3])
def test_layer_vjp_adjoint_identities(L):
    """The backward of the layer (with respect to the features and to the
    attention weights) is pinned by the adjoint identities of a linear map:
    <gy, y(h, alpha)> = <gfeat(gy), h> = sum_e alpha_e . galpha_e, and the
    directional derivative in alpha is exact."""
    rng = np.random.default_rng(30 + L)
    n, C, H = 40, 8, 2
    pos = syn.quantize(rng.uniform(0, 7, size=(n, 3)))
    rp, ci = o.neighbor_list(pos, 4.0)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.1, 1.0, size=(len(ci), H)).astype(np.float32)
    w = rng.uniform(0.2, 1.0, size=(L + 1) ** 3)
    gy = rng.standard_normal((n, (L + 1) ** 2, C))
    y = o.conv_edge(L, H, pos, feat, rp, ci, alpha, w)
    gf, ga = o.conv_edge_vjp(L, H, pos, feat, gy, rp, ci, alpha, w)
    lhs = float((gy * y).sum())
    assert abs(float((gf * feat.astype(np.float64)).sum()) - lhs) <= 1e-10 * abs(lhs)
    assert abs(float((ga * alpha.astype(np.float64)).sum()) - lhs) <= 1e-10 * abs(lhs)
    d = rng.standard_normal(alpha.shape).astype(np.float32) * np.float32(0.25)
    y2 = o.conv_edge(L, H, pos, feat, rp, ci, (alpha + d).astype(np.float32), w)
    dl = float((gy * (y2 - y)).sum())
    da = (alpha + d).astype(np.float64) - alpha.astype(np.float64)  # the perturbation as stored in float32
    assert abs(dl - float((ga * da).sum())) <= 1e-9 * max(1.0, abs(dl))
    # mixing: the adjoint of out = W^(o) y is W^(o)T
    mix = rng.standard_normal((L + 1, C, C))
    out = o.mix(L, y, mix)
    back = o.mix(L, gy, np.transpose(mix, (0, 2, 1)))
    assert abs(float((gy * out).sum()) - float((back * y).sum())) <= 1e-10 * abs(float((gy * out).sum()))


def test_knn_graph_closed_forms():
    """kNN graph (Sec. 4.1 sparse workloads): lattice distances are known in
    closed form (a, a*sqrt2, a*sqrt3), so the selected sets are too, ties
    included (equal distances are taken in index order)."""
    a = 1.5  # exact on the 2^-16 grid
    g = np.array(list(itertools.product(range(5), repeat=3)), dtype=np.float32) * a  # index = 25x + 5y + z
    idx = lambda x, y, z: 25 * x + 5 * y + z
    c = idx(2, 2, 2)
    faces = {idx(2 + dx, 2 + dy, 2 + dz) for dx, dy, dz in itertools.product((-1, 0, 1), repeat=3)
             if abs(dx) + abs(dy) + abs(dz) == 1}
    edges = {idx(2 + dx, 2 + dy, 2 + dz) for dx, dy, dz in itertools.product((-1, 0, 1), repeat=3)
             if abs(dx) + abs(dy) + abs(dz) == 2}
    corners = {idx(2 + dx, 2 + dy, 2 + dz) for dx, dy, dz in itertools.product((-1, 0, 1), repeat=3)
               if abs(dx) + abs(dy) + abs(dz) == 3}
    for k, want in [(6, faces), (7, faces | {min(edges)}), (18, faces | edges), (26, faces | edges | corners),
                    (20, faces | edges | set(sorted(corners)[:2]))]:
        rp, ci = o.knn_graph(g, k)
        row = ci[rp[c]:rp[c + 1]]
        assert list(row) == sorted(want), k
        assert np.all(np.diff(rp) == k)
    # corner atom (0,0,0): 3 at a, 3 at sqrt2 a, then (1,1,1) at sqrt3 a, closer
    # than the three at 2a
    rp, ci = o.knn_graph(g, 7)
    row = set(ci[rp[0]:rp[1]])
    assert row == {idx(1, 0, 0), idx(0, 1, 0), idx(0, 0, 1), idx(1, 1, 0), idx(1, 0, 1), idx(0, 1, 1), idx(1, 1, 1)}


def test_knn_graph_invariants():
    rng = np.random.default_rng(5)
    pos = syn.quantize(rng.uniform(0, 12, size=(150, 3)))
    gid = np.repeat(np.arange(3), 50).astype(np.int32)
    gid[-1] = 7  # a graph of one atom: empty row
    for k, graph in [(9, None), (9, gid), (200, None)]:
        rp, ci = o.knn_graph(pos, k, graph)
        n = len(pos)
        for i in range(n):
            row = ci[rp[i]:rp[i + 1]]
            same = [j for j in range(n) if j != i and (graph is None or graph[j] == graph[i])]
            assert len(row) == min(k, len(same))
            assert np.all(np.diff(row) > 0) and i not in row
            if k >= len(same):
                assert list(row) == same  # complete graph of the component
            else:
                # every chosen atom precedes every other in (distance, index) order
                X = np.rint(pos.astype(np.float64) * 65536.0).astype(np.int64)
                key = lambda j: (int(((X[i] - X[j]) ** 2).sum()), j)
                worst = max(key(j) for j in row)
                assert all(key(j) > worst for j in same if j not in set(row))


@pytest.mark.parametrize("L", [0, 1, 2, 3, 4])
def test_factorised_equals_definition(L):
    # Thm. 3.3 and Sec. 4.1: the node-factorised layer gives identical outputs
    n = 8 if L < 4 else 5
    pos, rp, ci, feat, alpha, w = small_graph(L, n, 4, 2, seed=10 + L)
    y1 = o.conv_edge(L, 2, pos, feat, rp, ci, alpha, w)
    for origin in ([0, 0, 0], [-3.1, 2.2, 7.5], pos[0].astype(np.float64)):
        y2 = o.conv_factorised(L, 2, pos, feat, rp, ci, alpha, w, np.array(origin, dtype=np.float64))
        # the binomial expansion cancels terms of size |p|^f down to |r_ij|^f,
        # so fp64 rounding grows like (max|p| / cutoff)^L
        maxp = np.max(np.linalg.norm(pos.astype(np.float64) - np.array(origin), axis=1))
        tol = 1e-13 * max(1.0, maxp / 3.0) ** L
        assert np.max(np.abs(y1 - y2)) <= tol * np.max(np.abs(y1))


@pytest.mark.parametrize("L", [0, 2, 3, 4])
def test_global_moment_equals_definition(L):
    # App. G: with alpha = 1 on every pair (self included) the moments
    # M = sum_j h_j (x) R(p_j) are shared by all nodes; the O(n) form equals
    # the layer's definition on the complete graph with self edges
    n, C = (7, 3) if L < 4 else (5, 2)
    pos, _, _, feat, _, w = small_graph(L, n, C, 1, seed=40 + L)
    rp = np.arange(n + 1, dtype=np.int64) * n
    ci = np.tile(np.arange(n, dtype=np.int32), n)
    y1 = o.conv_edge(L, 1, pos, feat, rp, ci, np.ones((n * n, 1), np.float32), w)
    for origin in ([0, 0, 0], [-2.5, 1.0, 6.0]):
        y2 = o.conv_global(L, pos, feat, w, np.array(origin, dtype=np.float64))
        maxp = np.max(np.linalg.norm(pos.astype(np.float64) - np.array(origin), axis=1))
        tol = 1e-13 * max(1.0, maxp / 3.0) ** L
        assert np.max(np.abs(y1 - y2)) <= tol * np.max(np.abs(y1))
    sub = np.array([n - 1, 0, 2], dtype=np.int32)
    assert np.array_equal(o.conv_global(L, pos, feat, w, np.array(origin, dtype=np.float64), rows=sub), y2[sub])
    if L == 0:
        # closed form: every node receives w_000 * sum_j h_j
        assert np.allclose(y2[:, 0, :], w[0] * feat[:, 0, :].astype(np.float64).sum(0)[None, :], rtol=1e-13)


def test_y_norm_closed_forms():
    # Alg. 1's per-degree weights alpha / D^f: on a lattice whose edges all
    # have length D the variant equals the plain layer with w_afo D^-f; scaling
    # every position by 2 leaves it unchanged, while the plain layer's path f
    # grows by 2^f
    L, H, C = 3, 2, 4
    g = np.array(list(itertools.product(range(4), repeat=3)), dtype=np.float32) * 1.5
    rp, ci = o.neighbor_list(g, 1.6)  # the six nearest neighbours, all at 1.5
    rng = np.random.default_rng(3)
    feat = rng.standard_normal((len(g), (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.2, 1.0, size=(len(ci), H)).astype(np.float32)
    w = rng.uniform(0.5, 1.5, size=(L + 1) ** 3)
    fpow = np.array([f for a in range(L + 1) for f in range(L + 1) for oo in range(L + 1)], dtype=float)
    yn = o.conv_edge(L, H, g, feat, rp, ci, alpha, w, y_norm=True)
    yp = o.conv_edge(L, H, g, feat, rp, ci, alpha, w * 1.5 ** -fpow)
    assert np.max(np.abs(yn - yp)) <= 1e-13 * np.max(np.abs(yp))
    pos, rp2, ci2, feat2, alpha2, w2 = small_graph(L, 9, C, H, seed=77)
    a = o.conv_edge(L, H, pos, feat2, rp2, ci2, alpha2, w2, y_norm=True)
    b = o.conv_edge(L, H, pos * 2, feat2, rp2, ci2, alpha2, w2, y_norm=True)
    assert np.max(np.abs(a - b)) <= 1e-13 * np.max(np.abs(a))
    c = o.conv_edge(L, H, pos * 2, feat2, rp2, ci2, alpha2, w2)
    d = o.conv_edge(L, H, pos, feat2, rp2, ci2, alpha2, w2 * 2.0 ** fpow)
    assert np.max(np.abs(c - d)) <= 1e-13 * np.max(np.abs(c))
    assert np.max(np.abs(a - o.conv_edge(L, H, pos, feat2, rp2, ci2, alpha2, w2))) > 1e-3 * np.max(np.abs(a))


def test_solid_harmonics_gradient():
    # central differences in float64, and Euler's identity for the
    # homogeneous polynomials R^(l): sum_x v_x dR^(l)/dv_x = l R^(l)
    L = 6
    rng = np.random.default_rng(12)
    for _ in range(5):
        v = rng.uniform(-2.0, 2.0, size=3)
        d = o.solid_harmonics_grad(L, v)
        for x in range(3):
            e = np.zeros(3)
            e[x] = 1e-5
            fd = (o.solid_harmonics(L, v + e) - o.solid_harmonics(L, v - e)) / 2e-5
            assert np.allclose(d[x], fd, rtol=1e-7, atol=1e-7 * np.abs(fd).max())
        deg = np.array([l for l in range(L + 1) for _ in range(2 * l + 1)], dtype=float)
        assert np.allclose(v @ d, deg * o.solid_harmonics(L, v), rtol=1e-12, atol=1e-12)


def test_forces_definition():
    # the position gradient of sum(gy * layer) with the graph and alpha fixed:
    # finite differences of the layer (actual float32 steps), zero net force
    # (the layer depends on differences of positions), rotation covariance
    L, H, C = 3, 2, 4
    pos, rp, ci, feat, alpha, w = small_graph(L, 10, C, H, seed=31)
    gy = np.random.default_rng(4).standard_normal((10, (L + 1) ** 2, C))
    g = o.conv_edge_grad_pos(L, H, pos, feat, gy, rp, ci, alpha, w)
    assert np.allclose(g.sum(0), 0.0, atol=1e-11 * np.abs(g).max())
    loss = lambda p: float((gy * o.conv_edge(L, H, p, feat, rp, ci, alpha, w)).sum())
    for a, x in ((0, 0), (3, 1), (7, 2), (9, 0)):
        up, dn = pos.copy(), pos.copy()
        up[a, x] = np.float32(pos[a, x] + np.float32(1e-3))
        dn[a, x] = np.float32(pos[a, x] - np.float32(1e-3))
        fd = (loss(up) - loss(dn)) / (float(up[a, x]) - float(dn[a, x]))
        assert abs(fd - g[a, x]) <= 1e-5 * np.abs(g).max(), (a, x, fd, g[a, x])
    sub = np.array([9, 2, 5], dtype=np.int32)
    assert np.array_equal(o.conv_edge_grad_pos(L, H, pos, feat, gy, rp, ci, alpha, w, atoms=sub), g[sub])
    Q = o.random_rotation(8)
    D = o.wigner_d(L, Q)
    rot = lambda t: np.concatenate([np.einsum("mn,inc->imc", D[l], t[:, l * l:(l + 1) ** 2]) for l in range(L + 1)], 1)
    center = pos.astype(np.float64).mean(0)
    pos_r = ((pos.astype(np.float64) - center) @ Q.T + center).astype(np.float32)
    g_r = o.conv_edge_grad_pos(L, H, pos_r, rot(feat).astype(np.float32), rot(gy), rp, ci, alpha, w)
    assert np.allclose(g_r, g @ Q.T, atol=2e-5 * np.abs(g).max())


def test_layer_equivariance_and_translation():
    # Lemma (equivariance, App. E): rotating positions and features rotates
    # every output irrep by D^(o); a translation changes nothing.
    L, H, C = 3, 2, 4
    pos, rp, ci, feat, alpha, w = small_graph(L, 9, C, H, seed=21)
    W = np.random.default_rng(1).standard_normal((L + 1, C, C)).astype(np.float32)
    y = o.layer(L, H, pos, feat, rp, ci, alpha, w, W)
    Q = o.random_rotation(5)
    D = o.wigner_d(L, Q)
    for l in range(L + 1):
        assert np.allclose(D[l] @ D[l].T, np.eye(2 * l + 1), atol=1e-12)
    center = np.array([1.0, 2.0, -0.5])
    pos_r = ((pos.astype(np.float64) - center) @ Q.T + center).astype(np.float32)
    feat_r = feat.astype(np.float64).copy()
    for l in range(L + 1):
        s = slice(l * l, (l + 1) ** 2)
        feat_r[:, s, :] = np.einsum("mk,nkc->nmc", D[l], feat[:, s, :])
    y_r = o.layer(L, H, pos_r, feat_r.astype(np.float32), rp, ci, alpha, w, W)
    want = y.copy()
    for l in range(L + 1):
        s = slice(l * l, (l + 1) ** 2)
        want[:, s, :] = np.einsum("mk,nkc->nmc", D[l], y[:, s, :])
    # float32 rounding of the rotated inputs bounds the agreement
    assert np.max(np.abs(y_r - want)) <= 2e-5 * np.max(np.abs(want))
    shift = np.array([3.0, -1.25, 0.5], dtype=np.float32)  # a grid vector
    y_t = o.layer(L, H, pos + shift, feat, rp, ci, alpha, w, W)
    assert np.array_equal(y_t, y)


def test_layer_special_cases():
    rng = np.random.default_rng(8)
    L, H, C = 2, 2, 4
    pos, rp, ci, feat, alpha, _ = small_graph(L, 10, C, H, seed=31)
    n = pos.shape[0]
    recv = np.repeat(np.arange(n), np.diff(rp))
    head = np.arange(C) // (C // H)
    a_full = alpha[:, head]  # [E, C]
    # only the f = 0 paths (a, 0, a): y^(a) = sum_j alpha_ij h_j^(a), a plain SpMM
    w = np.zeros((L + 1,) * 3)
    for a in range(L + 1):
        w[a, 0, a] = 1.0
    y = o.conv_edge(L, H, pos, feat, rp, ci, alpha, w.reshape(-1))
    want = np.zeros((n, (L + 1) ** 2, C))
    np.add.at(want, recv, a_full[:, None, :] * feat[ci].astype(np.float64))
    assert np.allclose(y, want, atol=1e-12)
    # only (0, 1, 1): y^(1) = sum_j alpha_ij h_j^(0) (r_i - r_j) in (y, z, x) order
    w = np.zeros((L + 1,) * 3)
    w[0, 1, 1] = 1.0
    y = o.conv_edge(L, H, pos, feat, rp, ci, alpha, w.reshape(-1))
    rij = pos[recv].astype(np.float64) - pos[ci]
    vec = rij[:, [1, 2, 0]]
    want = np.zeros((n, 3, C))
    np.add.at(want, recv, vec[:, :, None] * (a_full * feat[ci, 0, :])[:, None, :])
    assert np.allclose(y[:, 1:4, :], want, atol=1e-12)
    assert np.all(y[:, 0, :] == 0) and np.all(y[:, 4:, :] == 0)
    # isolated atom: zero row
    lonely = np.concatenate([pos, np.array([[40.0, 40.0, 40.0]], dtype=np.float32)])
    rp2, ci2 = o.neighbor_list(lonely, 3.0)
    f2 = rng.standard_normal((n + 1, (L + 1) ** 2, C)).astype(np.float32)
    a2 = rng.uniform(size=(len(ci2), H)).astype(np.float32)
    y2 = o.conv_edge(L, H, lonely, f2, rp2, ci2, a2, rng.uniform(size=(L + 1) ** 3))
    assert np.all(y2[n] == 0)


def test_row_subset_and_mixing():
    L, H, C = 2, 2, 4
    pos, rp, ci, feat, alpha, w = small_graph(L, 10, C, H, seed=41)
    y = o.conv_edge(L, H, pos, feat, rp, ci, alpha, w)
    rows = np.array([7, 2, 9], dtype=np.int32)
    assert np.array_equal(o.conv_edge(L, H, pos, feat, rp, ci, alpha, w, rows), y[rows])
    W = np.random.default_rng(2).standard_normal((L + 1, C, C)).astype(np.float32)
    out = o.mix(L, y, W)
    for l in range(L + 1):
        s = slice(l * l, (l + 1) ** 2)
        assert np.allclose(out[:, s, :], np.einsum("pc,nmc->nmp", W[l].astype(np.float64), y[:, s, :]), atol=1e-13)


def test_mixing_closed_forms():
    # App. F: the self-mix is one C x C matrix per output degree o, applied to
    # the channels of every m of that degree, W stored [o][c_out][c_in].
    L, C, n = 3, 5, 4
    rng = np.random.default_rng(77)
    y = rng.standard_normal((n, (L + 1) ** 2, C))
    # W^(o) = (o + 1) I: each degree's rows are scaled by their own factor,
    # which fixes the assignment of the blocks of W to the degrees
    W = np.zeros((L + 1, C, C), np.float32)
    for l in range(L + 1):
        W[l] = (l + 1) * np.eye(C, dtype=np.float32)
    out = o.mix(L, y, W)
    for l in range(L + 1):
        s = slice(l * l, (l + 1) ** 2)
        assert np.array_equal(out[:, s, :], (l + 1) * y[:, s, :])
    # a single entry W^(o)[1][0] = 1: output channel 1 of degree o receives
    # input channel 0 and nothing else is written, which fixes the orientation
    # (row = output channel, column = input channel)
    for l in range(L + 1):
        W = np.zeros((L + 1, C, C), np.float32)
        W[l, 1, 0] = 1.0
        out = o.mix(L, y, W)
        s = slice(l * l, (l + 1) ** 2)
        want = np.zeros_like(y)
        want[:, s, 1] = y[:, s, 0]
        assert np.array_equal(out, want)
    # a cyclic channel shift on degree 2 only: out[c'] = y[(c' + 1) % C]
    W = np.zeros((L + 1, C, C), np.float32)
    for cp in range(C):
        W[2, cp, (cp + 1) % C] = 1.0
    out = o.mix(L, y, W)
    assert np.array_equal(out[:, 4:9, :], np.roll(y[:, 4:9, :], -1, axis=2))
    assert np.all(out[:, :4, :] == 0) and np.all(out[:, 9:, :] == 0)


def test_global_moment_equals_definition_larger():
    # App. G at a size where a dropped or misindexed moment term cannot hide:
    # 40 atoms, every pair and the self term, against the definition
    L, C, n = 3, 3, 40
    rng = np.random.default_rng(91)
    pos = (rng.uniform(-4.0, 4.0, size=(n, 3)) * 65536.0).round() / 65536.0
    pos = pos.astype(np.float32)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    w = rng.uniform(0.5, 1.5, size=(L + 1) ** 3)
    rp = np.arange(n + 1, dtype=np.int64) * n
    ci = np.tile(np.arange(n, dtype=np.int32), n)
    y1 = o.conv_edge(L, 1, pos, feat, rp, ci, np.ones((n * n, 1), np.float32), w)
    origin = np.array([0.3, -0.2, 0.1])
    y2 = o.conv_global(L, pos, feat, w, origin)
    assert np.max(np.abs(y1 - y2)) <= 1e-11 * np.max(np.abs(y1))


def test_aggregate_equals_dense_einsum_and_hand_example():
    # Alg. 1's aggregation written as the paper's dense einsum "ijh,jhds->ihds"
    # (alpha scattered into an N x N x H tensor, zero off the graph) against
    # the oracle's edge loop; plus a three-atom example summed by hand
    rng = np.random.default_rng(21)
    n, H, K, dh = 23, 3, 5, 4
    pos = rng.uniform(0, 6, size=(n, 3)).astype(np.float32)
    rp, ci = o.neighbor_list(pos, 3.0)
    T = rng.standard_normal((n, H, K, dh)).astype(np.float32)
    alpha = rng.uniform(0, 1, size=(len(ci), H)).astype(np.float32)
    A = np.zeros((n, n, H))
    for i in range(n):
        for e in range(rp[i], rp[i + 1]):
            A[i, ci[e]] = alpha[e]
    dense = np.einsum("ijh,jhkd->ihkd", A, T.astype(np.float64))
    got = o.aggregate(T, rp, ci, alpha)
    assert np.max(np.abs(got - dense)) <= 1e-12 * np.max(np.abs(dense))
    rows = np.array([n - 1, 0, 7], dtype=np.int32)
    assert np.array_equal(o.aggregate(T, rp, ci, alpha, rows=rows), got[rows])
    ones = o.aggregate(T, rp, ci, None)
    assert np.allclose(ones, np.einsum("ijh,jhkd->ihkd", (A != 0).astype(np.float64), T.astype(np.float64)),
                       rtol=0, atol=1e-12)
    # 0 <- {1, 2}, 1 <- {0}, 2 isolated; one head of two values
    T3 = np.array([[[1.0, 2.0]], [[3.0, 5.0]], [[7.0, 11.0]]], dtype=np.float32)[:, :, None, :]
    rp3 = np.array([0, 2, 3, 3], dtype=np.int64)
    ci3 = np.array([1, 2, 0], dtype=np.int32)
    a3 = np.array([[0.5], [2.0], [4.0]], dtype=np.float32)
    S3 = o.aggregate(T3, rp3, ci3, a3)
    assert np.array_equal(S3[0, 0, 0], [0.5 * 3 + 2 * 7, 0.5 * 5 + 2 * 11])
    assert np.array_equal(S3[1, 0, 0], [4.0 * 1, 4.0 * 2])
    assert np.array_equal(S3[2], np.zeros((1, 1, 2)))
