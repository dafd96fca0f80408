"""Pins of the G' oracle (``oracle/network.py``) to things other than itself:
exact rational solutions of the circuit written independently here, hand
derived closed forms, textbook ladder reductions, invariants of resistive
networks, and the paper's worked sneak-path example (Sec. IV-A)."""

import json
import os
from fractions import Fraction as Fr

import numpy as np
import pytest

from oracle.network import gprime_nodal, gprime_paper, gprime_rowsweep, node_voltages

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# exact rational references
# ---------------------------------------------------------------------------

def _solve_exact(A, B):
    """Gauss-Jordan with exact rationals; A n x n, B n x k (lists)."""
    n = len(A)
    k = len(B[0])
    T = [list(A[i]) + list(B[i]) for i in range(n)]
    for c in range(n):
        p = next(r for r in range(c, n) if T[r][c] != 0)
        T[c], T[p] = T[p], T[c]
        inv = 1 / T[c][c]
        T[c] = [v * inv for v in T[c]]
        for r in range(n):
            if r != c and T[r][c] != 0:
                f = T[r][c]
                T[r] = [vr - f * vc for vr, vc in zip(T[r], T[c])]
    return [row[n:n + k] for row in T]


def exact_gprime_device_voltages(G, rd, rs, rr, rc):
    """Exact G' from Kirchhoff's voltage law written on the device voltages
    V[i][j] = Va - Vb: walking from source i along row i to node a[i][j], down
    through device (i,j) and along column j to ground,
        Vin_i = (rd + rr*(j+1))*(row current through segment 1..j+1)...
    expanded here term by term: every device current G[i][x] V[i][x] of row i
    crosses the first min(j,x)+1 row segments, and every device current
    G[y][j] V[y][j] of column j crosses the column segments below row
    max(i, y) and the sense resistor."""
    M, N = len(G), len(G[0])
    idx = lambda i, j: i * N + j
    A = [[Fr(0)] * (M * N) for _ in range(M * N)]
    for i in range(M):
        for j in range(N):
            e = idx(i, j)
            A[e][e] += 1
            for x in range(N):
                A[e][idx(i, x)] += (rd + rr * (min(j, x) + 1)) * G[i][x]
            for y in range(M):
                A[e][idx(y, j)] += (rs + rc * (M - 1 - max(i, y))) * G[y][j]
    B = [[Fr(1) if i == s else Fr(0) for s in range(M)] for i in range(M) for _ in range(N)]
    V = _solve_exact(A, B)
    return [[sum(G[y][j] * V[idx(y, j)][i] for y in range(M)) for j in range(N)]
            for i in range(M)]


def exact_gprime_nodal(G, rd, rs, rr, rc):
    """Exact G' from KCL at every node (all resistances > 0)."""
    M, N = len(G), len(G[0])
    a = lambda i, j: i * N + j
    b = lambda i, j: M * N + i * N + j
    n = 2 * M * N
    Y = [[Fr(0)] * n for _ in range(n)]
    rhs = [[Fr(0)] * M for _ in range(n)]

    def el(p, q, g):
        Y[p][p] += g; Y[q][q] += g; Y[p][q] -= g; Y[q][p] -= g

    for i in range(M):
        g1 = 1 / (rd + rr)
        Y[a(i, 0)][a(i, 0)] += g1
        rhs[a(i, 0)][i] += g1
        for j in range(N - 1):
            el(a(i, j), a(i, j + 1), 1 / rr)
        for j in range(N):
            el(a(i, j), b(i, j), G[i][j])
    for j in range(N):
        for i in range(M - 1):
            el(b(i, j), b(i + 1, j), 1 / rc)
        Y[b(M - 1, j)][b(M - 1, j)] += 1 / rs
    V = _solve_exact(Y, rhs)
    return [[V[b(M - 1, j)][i] / rs for j in range(N)] for i in range(M)]


def _rand_exact(rng, M, N):
    # conductances k * 1e-6 S with k in 5..50 (the [5, 50] uS device range)
    return [[Fr(int(rng.integers(5, 51)), 10 ** 6) for _ in range(N)] for _ in range(M)]


RES_EXACT = (Fr(1000), Fr(1000), Fr(5, 2), Fr(5, 2))


@pytest.mark.parametrize("M,N", [(1, 1), (1, 3), (3, 1), (2, 2), (3, 2), (2, 3), (3, 3), (4, 4)])
def test_exact_rational_tiny(M, N):
    rng = np.random.default_rng(100 + 10 * M + N)
    Gq = _rand_exact(rng, M, N)
    # two independent exact formulations agree exactly
    e1 = exact_gprime_device_voltages(Gq, *RES_EXACT)
    e2 = exact_gprime_nodal(Gq, *RES_EXACT)
    assert e1 == e2
    ref = np.array([[float(v) for v in row] for row in e1])
    G = np.array([[float(v) for v in row] for row in Gq])
    res = tuple(float(r) for r in RES_EXACT)
    for fn in (gprime_nodal, gprime_paper, gprime_rowsweep):
        got = fn(G, *res)
        assert np.max(np.abs(got - ref) / np.abs(ref)) < 1e-12, fn.__name__


@pytest.mark.parametrize("res", [(0, 300, 0, 40), (500, 0, 7, 0), (0, 0, 3, 0), (0, 0, 0, 9)])
def test_exact_rational_with_zero_elements(res):
    """Ideal (zero-resistance) elements merge nodes; checked against the
    device-voltage form, which needs no conductance of a wire."""
    rng = np.random.default_rng(7)
    Gq = _rand_exact(rng, 3, 3)
    ref = np.array([[float(v) for v in row]
                    for row in exact_gprime_device_voltages(Gq, *(Fr(r) for r in res))])
    G = np.array([[float(v) for v in row] for row in Gq])
    for fn in (gprime_nodal, gprime_paper):
        got = fn(G, *map(float, res))
        assert np.max(np.abs(got - ref) / ref) < 1e-12, fn.__name__


@pytest.mark.parametrize("M,N", [(2, 2), (3, 3), (4, 4)])
def test_exact_rational_open_devices(M, N):
    """Devices of zero conductance (a variation factor of 0 makes them) are
    open circuits; both exact formulations and every oracle solver agree on
    arrays that hold some, and a column whose devices are all open carries
    no current."""
    rng = np.random.default_rng(300 + 10 * M + N)
    Gq = _rand_exact(rng, M, N)
    Gq[0][0] = Fr(0)
    Gq[M - 1][N - 2] = Fr(0)
    for i in range(M):
        Gq[i][N - 1] = Fr(0)                      # the last column is open throughout
    e1 = exact_gprime_device_voltages(Gq, *RES_EXACT)
    e2 = exact_gprime_nodal(Gq, *RES_EXACT)
    assert e1 == e2
    assert all(e1[i][N - 1] == 0 for i in range(M))
    ref = np.array([[float(v) for v in row] for row in e1])
    G = np.array([[float(v) for v in row] for row in Gq])
    res = tuple(float(r) for r in RES_EXACT)
    scale = np.abs(ref).max()
    for fn in (gprime_nodal, gprime_paper, gprime_rowsweep):
        got = fn(G, *res)
        assert np.all(np.abs(got - ref) <= 1e-12 * np.maximum(np.abs(ref), 1e-10 * scale)), \
            fn.__name__


def test_open_device_is_the_limit_of_small_conductance():
    """G = 0 is the continuous limit G -> 0+ (40 x 40, nodal and row sweep)."""
    rng = np.random.default_rng(5)
    G = rng.uniform(5e-6, 50e-6, size=(40, 40))
    G[rng.random(G.shape) < 0.05] = 0.0
    Gs = np.where(G == 0.0, 1e-24, G)
    res = (1000.0, 1000.0, 2.5, 2.5)
    a = gprime_nodal(G, *res)
    b = gprime_nodal(Gs, *res)
    c = gprime_rowsweep(G, *res)
    assert np.all(np.isfinite(a)) and np.all(a >= -1e-20)
    assert np.max(np.abs(a - b)) <= 1e-12 * np.max(np.abs(b))
    assert np.max(np.abs(a - c)) <= 1e-11 * np.max(np.abs(a))
    for fn in (gprime_nodal, gprime_rowsweep):
        with pytest.raises(ValueError):
            fn(-G, *res)


# ---------------------------------------------------------------------------
# closed forms and textbook ladders
# ---------------------------------------------------------------------------

@pytest.fixture
def Grand():
    return np.random.default_rng(11).uniform(5e-6, 50e-6, size=(7, 6))


@pytest.mark.parametrize("fn", [gprime_nodal, gprime_paper])
def test_zero_parasitics_is_ideal(fn, Grand):
    # Eq. 1: with no parasitic resistance the crossbar is the ideal G
    assert np.array_equal(fn(Grand, 0.0, 0.0, 0.0, 0.0), Grand)


@pytest.mark.parametrize("fn", [gprime_nodal, gprime_paper])
def test_sense_only(fn, Grand):
    # each column is its devices in parallel, in series with R_sense; the
    # column node voltage is R_s * Iout_j
    Rs = 1000.0
    want = Grand / (1.0 + Rs * Grand.sum(axis=0, keepdims=True))
    np.testing.assert_allclose(fn(Grand, 0.0, Rs, 0.0, 0.0), want, rtol=1e-13)


@pytest.mark.parametrize("fn", [gprime_nodal, gprime_paper])
def test_driver_only_is_divider(fn, Grand):
    # the DAC output divided by its load (Sec. IV-A 'Non-ideal DAC'):
    # row node voltage Vin / (1 + R_d sum_j G_ij)
    Rd = 1000.0
    want = Grand / (1.0 + Rd * Grand.sum(axis=1, keepdims=True))
    np.testing.assert_allclose(fn(Grand, Rd, 0.0, 0.0, 0.0), want, rtol=1e-13)


@pytest.mark.parametrize("fn", [gprime_nodal, gprime_paper, gprime_rowsweep])
def test_one_by_one(fn):
    G = np.array([[3.3e-5]])
    # a 1x1 array has no column segment: source, R_d + r_row, device, R_sense
    want = 1.0 / (1.0 / 3.3e-5 + 1000.0 + 2.5 + 700.0)
    np.testing.assert_allclose(fn(G, 1000.0, 700.0, 2.5, 4.0), [[want]], rtol=1e-13)


@pytest.mark.parametrize("fn", [gprime_nodal, gprime_paper])
def test_orientation_two_rows(fn):
    # 2x1 array, column wire only: row 0 is farthest from the sense amplifier,
    # so its device current crosses r_col; row 1's node b is the grounded one.
    G1, G2, rc = 2e-5, 4e-5, 150.0
    got = fn(np.array([[G1], [G2]]), 0.0, 0.0, 0.0, rc)
    np.testing.assert_allclose(got, [[1.0 / (1.0 / G1 + rc)], [G2]], rtol=1e-13)


def _row_ladder(Gs, rd, rr, rs):
    """Textbook ladder reduction of a 1 x N array: source, R_d + r_row, then
    N shunt branches (device in series with R_sense) separated by r_row."""
    N = len(Gs)
    h = [1.0 / (1.0 / g + rs) for g in Gs]            # branch conductances
    Z = [0.0] * N                                      # impedance looking right
    Z[N - 1] = 1.0 / h[N - 1]
    for k in range(N - 2, -1, -1):
        Z[k] = 1.0 / (h[k] + 1.0 / (rr + Z[k + 1]))
    I = 1.0 / (rd + rr + Z[0])
    V = I * Z[0]
    out = []
    for k in range(N):
        out.append(V * h[k])
        if k + 1 < N:
            I_next = V / (rr + Z[k + 1])
            V = V - rr * I_next
    return np.array([out])


def _column_ladder(Gs, rd, rr, rc, rs):
    """Textbook ladder reduction of an M x 1 array: a chain b_0 -r_col- ... -
    b_{M-1} -R_sense- ground, with a branch (R_d + r_row + 1/G_x) from each
    b_x to its (grounded or 1 V) source."""
    M = len(Gs)
    h = [1.0 / (rd + rr + 1.0 / g) for g in Gs]
    out = np.zeros((M, 1))
    for i in range(M):
        # impedance seen from b_x looking up (towards row 0) / down (to ground)
        up = [None] * M
        up[0] = 1.0 / h[0]
        for x in range(1, M):
            up[x] = 1.0 / (h[x] + 1.0 / (rc + up[x - 1]))
        down = [None] * M
        down[M - 1] = 1.0 / (h[M - 1] + 1.0 / rs)
        for x in range(M - 2, -1, -1):
            down[x] = 1.0 / (h[x] + 1.0 / (rc + down[x + 1]))
        # load at b_i excluding its own source branch
        y = 0.0
        if i > 0:
            y += 1.0 / (rc + up[i - 1])
        y += (1.0 / (rc + down[i + 1])) if i < M - 1 else 1.0 / rs
        Zl = 1.0 / y
        V = Zl / (1.0 / h[i] + Zl)
        # walk the current down to the sense resistor
        for x in range(i, M - 1):
            I_seg = V / (rc + down[x + 1])
            V = V - rc * I_seg
        out[i, 0] = V / rs
    return out


@pytest.mark.parametrize("fn", [gprime_nodal, gprime_paper, gprime_rowsweep])
def test_row_ladder(fn):
    Gs = np.random.default_rng(3).uniform(5e-6, 5e-5, 9)
    got = fn(Gs[None, :], 1000.0, 800.0, 2.5, 77.0)    # r_col unused for M = 1
    np.testing.assert_allclose(got, _row_ladder(Gs, 1000.0, 2.5, 800.0), rtol=1e-12)


@pytest.mark.parametrize("fn", [gprime_nodal, gprime_paper, gprime_rowsweep])
def test_column_ladder(fn):
    Gs = np.random.default_rng(4).uniform(5e-6, 5e-5, 8)
    got = fn(Gs[:, None], 1000.0, 900.0, 2.5, 30.0)
    np.testing.assert_allclose(got, _column_ladder(Gs, 1000.0, 2.5, 30.0, 900.0), rtol=1e-12)


def test_nodal_matches_paper_32x32():
    G = np.random.default_rng(5).uniform(5e-6, 5e-5, size=(24, 20))
    a = gprime_nodal(G, 1000.0, 1000.0, 2.5, 2.5)
    b = gprime_paper(G, 1000.0, 1000.0, 2.5, 2.5)
    assert np.max(np.abs(a - b) / a) < 1e-11


@pytest.mark.parametrize("M,N,res", [
    (1, 17, (1000.0, 1000.0, 2.5, 2.5)),
    (19, 1, (1000.0, 1000.0, 2.5, 2.5)),
    (13, 29, (1000.0, 1000.0, 2.5, 2.5)),
    (40, 33, (0.0, 1000.0, 1.0, 5.0)),
    (64, 64, (1000.0, 1000.0, 1.0, 1.0)),
])
def test_rowsweep_matches_nodal(M, N, res):
    """The row sweep (large-array oracle) solves the same KCL equations as the
    nodal solve by a different elimination."""
    G = np.random.default_rng(M * 100 + N).uniform(5e-6, 5e-5, size=(M, N))
    a = gprime_nodal(G, *res)
    b = gprime_rowsweep(G, *res)
    assert np.max(np.abs(a - b) / a) < 1e-9


def test_rowsweep_rejects_zero_wire():
    with pytest.raises(ValueError):
        gprime_rowsweep(np.full((3, 3), 1e-5), 1000.0, 1000.0, 0.0, 2.5)


def test_rowsweep_invariants_128():
    """At 128 x 128 (the size of the stacked workloads): positivity, the row
    and column sum bounds, and Rayleigh monotonicity of 1^T G' 1 in the wire
    resistance."""
    G = np.random.default_rng(13).uniform(5e-6, 5e-5, size=(128, 128))
    gp = gprime_rowsweep(G, 1000.0, 1000.0, 1.0, 1.0)
    assert np.all(gp > 0)
    assert np.all(gp.sum(axis=1) <= G.sum(axis=1))
    assert np.all(gp.sum(axis=0) <= G.sum(axis=0))
    gp2 = gprime_rowsweep(G, 1000.0, 1000.0, 2.5, 2.5)
    assert gp2.sum() < gp.sum()


# ---------------------------------------------------------------------------
# invariants of passive resistive networks
# ---------------------------------------------------------------------------

def test_invariants_random():
    rng = np.random.default_rng(8)
    for _ in range(5):
        M, N = rng.integers(2, 12, size=2)
        G = rng.uniform(5e-6, 5e-5, size=(M, N))
        res = rng.uniform(0.5, 2000.0, 4) * np.array([1, 1, 1e-3, 1e-3])
        gp = gprime_nodal(G, *res)
        assert np.all(gp > 0)                                    # maximum principle
        assert np.all(gp.sum(axis=1) <= G.sum(axis=1) * (1 + 1e-12))
        assert np.all(gp.sum(axis=0) <= G.sum(axis=0) * (1 + 1e-12))


def test_rayleigh_monotone():
    """The conductance between the shorted sources and ground, 1^T G' 1, can
    only fall when any resistance rises (Rayleigh's monotonicity law).  (Single
    entries of G' are not monotone in general.)"""
    G = np.random.default_rng(9).uniform(5e-6, 5e-5, size=(10, 9))
    base = [1000.0, 1000.0, 2.5, 2.5]
    for k in range(4):
        vals = []
        for f in (0.0, 0.5, 1.0, 2.0, 8.0):
            r = list(base)
            r[k] = base[k] * f
            vals.append(gprime_nodal(G, *r).sum())
        assert all(vals[i + 1] <= vals[i] * (1 + 1e-13) for i in range(len(vals) - 1)), k


def test_error_grows_with_size():
    """Sec. IV-B, sensitivity to crossbar size: with all devices at G_min or at
    G_max the relative loss of the array grows with its dimension."""
    for g in (5e-6, 5e-5):
        loss = []
        for n in (4, 8, 16, 32):
            gp = gprime_nodal(np.full((n, n), g), 1000.0, 1000.0, 2.5, 2.5)
            loss.append(1.0 - gp.sum() / (g * n * n))
        assert all(loss[i] < loss[i + 1] for i in range(len(loss) - 1))


def test_superposition():
    G = np.random.default_rng(12).uniform(5e-6, 5e-5, size=(5, 4))
    res = (1000.0, 1000.0, 2.5, 2.5)
    v1, v2 = np.array([0.1, 0.0, 0.2, 0.05, 0.0]), np.array([0.0, 0.3, 0.01, 0.0, 0.2])
    a1, b1 = node_voltages(G, v1, *res)
    a2, b2 = node_voltages(G, v2, *res)
    a3, b3 = node_voltages(G, v1 + v2, *res)
    np.testing.assert_allclose(a3, a1 + a2, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(b3, b1 + b2, rtol=1e-12, atol=1e-15)
    # the column outputs are V . G' (Eq. 14)
    gp = gprime_nodal(G, *res)
    i_out = (G * (a3 - b3)).sum(axis=0)
    np.testing.assert_allclose(i_out, (v1 + v2) @ gp, rtol=1e-12)


# ---------------------------------------------------------------------------
# the paper's worked example
# ---------------------------------------------------------------------------

def test_sneak_path_example():
    ex = json.load(open(os.path.join(GOLDEN, "sneak_path_3x2.json")))
    G = np.full((ex["rows"], ex["cols"]), 1.0 / ex["device_ohm"])
    i, j = (v - 1 for v in ex["reversed_device_1based"])
    va, vb = node_voltages(G, ex["vin_volt"], 1000.0, 1000.0, 2.5, 2.5)
    assert va[i, j] - vb[i, j] < 0          # current flows from b22 towards Vin2
    # rows driven at 0.2 V conduct in the expected direction
    assert np.all((va - vb)[[0, 2], :] > 0)
    # the reversal is produced by the sense resistance; wires alone do not flip it
    va, vb = node_voltages(G, ex["vin_volt"], 0.0, 0.0, 2.5, 2.5)
    assert va[i, j] - vb[i, j] > 0
