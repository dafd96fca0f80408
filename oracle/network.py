"""Oracle: the equivalent non-ideal conductance matrix G' of one crossbar.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The crossbar is the resistive network of Sec. V-B (equivalent circuit of an
M x N array).  Tile-local indices are 0-based here; row 0 is the paper's row 1
and column 0 the paper's column 1.

Topology (the reading of Eqs. 2-8; the circuit figure itself is not available):

* Row i: an ideal source ``Vin_i`` drives node ``a[i,0]`` through the driver
  resistance in series with the first row-wire segment (``r_driver + r_row``);
  consecutive row nodes ``a[i,j]`` -- ``a[i,j+1]`` are joined by ``r_row``.
  The far end of the row is open.  (The driver resistance is one of the
  non-idealities listed in Sec. IV-A; Eqs. 2-14 omit it, and the reading used
  here puts it in series with the first row segment.)
* Column j: ``b[i,j]`` -- ``b[i+1,j]`` are joined by ``r_col``; the last row's
  node ``b[M-1,j]`` reaches the virtual ground of the sense amplifier through
  ``r_sense``.  Row 0 is therefore the row farthest from the sense amplifier
  (the paper's J vector in Eq. 2 has ``R_sense + (M-1) r_col`` for row 1).
* Device ``G[i,j]`` joins ``a[i,j]`` and ``b[i,j]``.
* ``Iout_j`` is the current through column j's sense resistor, which by KCL on
  the column equals the sum of the column's device currents (Eq. 3).
* ``G'[i,j] = Iout_j`` when ``Vin = e_i`` (1 V on row i, 0 V on the other rows,
  whose drivers stay connected).  The paper states that G' reproduces the
  network exactly (Sec. V-A, generator step 3) and uses it as
  ``Iout = Vin . G'`` (Eq. 14).

Functions
---------
gprime_nodal(G, ...)   KCL at every node, library sparse LU.  Pinned by the
                       exact-rational and closed-form tests in
                       ``tests/test_oracle_network.py``.
node_voltages(G, Vin, ...)  The node voltages of the same nodal solve, used by
                       the sneak-path example of Sec. IV-A.
gprime_paper(G, ...)   The paper's Eqs. 2-14, dense.  Pinned by the same tests
                       and against ``gprime_nodal``.
gprime_rowsweep(G, ...)  The same nodal equations solved row by row (block
                       tridiagonal elimination), O(M N^3): the oracle for
                       large arrays.  Needs positive wire and sense
                       resistances.  Pinned against ``gprime_nodal`` and the
                       exact rational solutions, and by the network
                       invariants at 128 x 128.
"""

from __future__ import annotations

import numpy as np
import scipy.linalg as sla
import scipy.sparse as sp
import scipy.sparse.linalg as spla


# ---------------------------------------------------------------------------
# Nodal analysis (the plain definition)
# ---------------------------------------------------------------------------

def _edges(G, r_driver, r_sense, r_row, r_col):
    """List the two-terminal elements of the network.

    Returns (n_nodes, src, gnd, res_edges, dev_edges) where res_edges holds
    (p, q, resistance) and dev_edges holds (p, q, conductance).
    """
    M, N = G.shape
    a = lambda i, j: i * N + j
    b = lambda i, j: M * N + i * N + j
    src = [2 * M * N + i for i in range(M)]
    gnd = 2 * M * N + M
    res = []
    for i in range(M):
        res.append((src[i], a(i, 0), r_driver + r_row))
        for j in range(N - 1):
            res.append((a(i, j), a(i, j + 1), r_row))
    for j in range(N):
        for i in range(M - 1):
            res.append((b(i, j), b(i + 1, j), r_col))
        res.append((b(M - 1, j), gnd, r_sense))
    dev = [(a(i, j), b(i, j), float(G[i, j])) for i in range(M) for j in range(N)]
    return 2 * M * N + M + 1, src, gnd, res, dev


def _solve_nodal(G, Vin_cols, r_driver, r_sense, r_row, r_col):
    """Node voltages for each column of ``Vin_cols`` (M x K source patterns).

    Zero-resistance elements are ideal wires: their two terminals are the same
    node, so they are merged before KCL is written.  KCL is then written at
    every node group that is not held by a source or by ground.
    """
    G = np.asarray(G, dtype=np.float64)
    M, N = G.shape
    if not np.all(np.isfinite(G)) or np.any(G < 0):
        raise ValueError("device conductances must be finite and >= 0 (0: an open device)")
    for r in (r_driver, r_sense, r_row, r_col):
        if r < 0:
            raise ValueError("resistances must be non-negative")
    n, src, gnd, res, dev = _edges(G, r_driver, r_sense, r_row, r_col)

    parent = list(range(n))

    def find(x):
        while parent[x] != x:
            parent[x] = parent[parent[x]]
            x = parent[x]
        return x

    cond = []  # (p, q, conductance) between distinct groups
    for p, q, r in res:
        if r == 0.0:
            parent[find(p)] = find(q)
        else:
            cond.append((p, q, 1.0 / r))
    cond += dev
    root = [find(x) for x in range(n)]

    # fixed groups: a source group holds Vin_i, the ground group holds 0 V
    K = Vin_cols.shape[1]
    fixed = {}
    for i, s in enumerate(src):
        fixed.setdefault(root[s], []).append(("src", i))
    fixed.setdefault(root[gnd], []).append(("gnd", 0))
    for g, tags in fixed.items():
        if len(tags) > 1:
            raise ValueError("a source is shorted to another source or ground")

    groups = sorted(set(root))
    free = [g for g in groups if g not in fixed]
    fidx = {g: k for k, g in enumerate(free)}

    def fixed_value(g):
        kind, i = fixed[g][0]
        if kind == "gnd":
            return np.zeros(K)
        return Vin_cols[i, :].astype(np.float64)

    rows, cols, vals = [], [], []
    rhs = np.zeros((len(free), K))
    for p, q, g in cond:
        gp, gq = root[p], root[q]
        if gp == gq:
            raise ValueError("an element is shorted by ideal wires")
        for x, y in ((gp, gq), (gq, gp)):
            if x in fidx:
                rows.append(fidx[x]); cols.append(fidx[x]); vals.append(g)
                if y in fidx:
                    rows.append(fidx[x]); cols.append(fidx[y]); vals.append(-g)
                else:
                    rhs[fidx[x], :] += g * fixed_value(y)
    Y = sp.csc_matrix((vals, (rows, cols)), shape=(len(free), len(free)))
    Vf = spla.splu(Y).solve(rhs) if len(free) else np.zeros((0, K))

    V = np.empty((n, K))
    for x in range(n):
        g = root[x]
        V[x, :] = Vf[fidx[g], :] if g in fidx else fixed_value(g)
    Va = V[: M * N, :].reshape(M, N, K)
    Vb = V[M * N: 2 * M * N, :].reshape(M, N, K)
    return Va, Vb


def node_voltages(G, Vin, r_driver, r_sense, r_row, r_col):
    """Voltages of the row nodes ``a`` and column nodes ``b`` (M x N each) for
    one input vector ``Vin`` (length M)."""
    Vin = np.asarray(Vin, dtype=np.float64).reshape(-1, 1)
    Va, Vb = _solve_nodal(G, Vin, r_driver, r_sense, r_row, r_col)
    return Va[:, :, 0], Vb[:, :, 0]


def gprime_nodal(G, r_driver, r_sense, r_row, r_col):
    """G' by nodal analysis: ``G'[i,j]`` = column-j output current (Eq. 3) for
    1 V on row i and 0 V on the others.  fp64, M x N."""
    G = np.asarray(G, dtype=np.float64)
    M, N = G.shape
    Va, Vb = _solve_nodal(G, np.eye(M), r_driver, r_sense, r_row, r_col)
    # Va[x, j, i]: voltage of a[x, j] for source pattern e_i
    dev_current = G[:, :, None] * (Va - Vb)          # [x, j, i]
    return dev_current.sum(axis=0).T                  # [i, j]


# ---------------------------------------------------------------------------
# The paper's derivation, Sec. V-B Eqs. 2-14 (dense)
# ---------------------------------------------------------------------------

def gprime_paper(G, r_driver, r_sense, r_row, r_col):
    """G' following the six steps of Sec. V-B.

    Unknowns are the device voltages ``V[i,j] = Va[i,j] - Vb[i,j]``.

    Step 1 (Eqs. 2-4), column system of column j.  KCL at the column nodes
    gives ``Va[:,j] = Atil_j V[:,j] + J Iout_j`` with ``Iout_j = K_j V[:,j]``
    (Eq. 3).  ``Atil_j`` is the paper's ``A_j`` with the opposite overall sign:
    identity on the diagonal and ``-(x-i) r_col G[x,j]`` above it.  With the
    matrix exactly as printed, Eq. 4 yields ``G' = -G`` for a wire-free array,
    so the printed overall sign is read as a slip (the reading is recorded with
    the other readings of the paper).  ``J[i] = R_sense + (M-1-i) r_col``.
    Step 2 (Eqs. 5-6): direct sums ``COLmat = (+)_j (Atil_j + J K_j)`` and
    ``Gmat = (+)_j K_j`` over the column-ordered unknown vector ``CVcol``.
    Step 3 (Eq. 7): row system ``B_i Vrow_i = VrowIN_i - VArow_i`` with
    ``B_i[j,x] = (r_driver + r_row (min(j,x)+1)) G[i,x]`` (0-based; the driver
    resistance is added to every entry because every row current crosses it).
    Step 4 (Eq. 8): ``ROWmat = (+)_i B_i`` over the row-ordered vector.
    Step 5 (Eqs. 9-12): reorder the row system into column order,
    ``ROWmatA = P ROWmat P^T``, ``CVrowINA = P CVrowIN``, so that
    ``(COLmat + ROWmatA) CVcol = CVrowINA`` and
    ``NETmat = Gmat (COLmat + ROWmatA)^-1``.
    Step 6 (Eqs. 13-14): add the columns of NETmat that multiply the same
    ``Vin_i`` to get ``NETmatC`` (N x M); ``G' = NETmatC^T``.
    """
    G = np.asarray(G, dtype=np.float64)
    M, N = G.shape
    MN = M * N
    # column-ordered index of (i, j): j*M + i ; row-ordered index: i*N + j
    colmat = np.zeros((MN, MN))
    gmat = np.zeros((N, MN))
    Jv = np.array([r_sense + (M - 1 - i) * r_col for i in range(M)])
    for j in range(N):
        Kj = G[:, j]
        Atil = np.eye(M)
        for i in range(M):
            for x in range(i + 1, M):
                Atil[i, x] = -(x - i) * G[x, j] * r_col
        blk = Atil + np.outer(Jv, Kj)
        colmat[j * M:(j + 1) * M, j * M:(j + 1) * M] = blk
        gmat[j, j * M:(j + 1) * M] = Kj
    rowmat = np.zeros((MN, MN))
    for i in range(M):
        Bi = np.empty((N, N))
        for jj in range(N):
            for x in range(N):
                Bi[jj, x] = (r_driver + r_row * (min(jj, x) + 1)) * G[i, x]
        rowmat[i * N:(i + 1) * N, i * N:(i + 1) * N] = Bi
    # permutation from row order to column order: (P v)[j*M+i] = v[i*N+j]
    perm = np.empty(MN, dtype=np.int64)
    for i in range(M):
        for j in range(N):
            perm[j * M + i] = i * N + j
    P = np.zeros((MN, MN))
    P[np.arange(MN), perm] = 1.0
    rowmatA = P @ rowmat @ P.T
    netmat = gmat @ np.linalg.inv(colmat + rowmatA)        # Eq. 12
    # CVrowINA[j*M+i] = Vin_i : compress columns sharing the same Vin_i (Eq. 13)
    netmatC = np.zeros((N, M))
    for j in range(N):
        for i in range(M):
            netmatC[:, i] += netmat[:, j * M + i]
    return netmatC.T                                         # Eq. 14


# ---------------------------------------------------------------------------
# Row sweep of the nodal equations (large arrays)
# ---------------------------------------------------------------------------

def gprime_rowsweep(G, r_driver, r_sense, r_row, r_col):
    """G' from the KCL equations of ``_solve_nodal``, eliminated one row at a
    time.

    Row i's nodes a[i, :] form a chain: KCL there reads
    ``T_i a_i = g_in Vin_i e_0 + D_i b_i`` with ``D_i = diag(G[i, :])`` and
    ``T_i`` the chain's tridiagonal conductance matrix (``g_in = 1 / (r_driver
    + r_row)`` to the source at node 0, ``1 / r_row`` between neighbours) plus
    ``D_i``.  Substituting ``a_i`` into KCL at the column nodes b[i, :] leaves
    a block tridiagonal system in the b rows:

        ``(S_i + g_col n_i I + [i = M-1] g_sense I) b_i - g_col b_(i-1)
          - g_col b_(i+1) = f_i Vin_i``

    with ``S_i = D_i - D_i T_i^-1 D_i``, ``f_i = g_in D_i T_i^-1 e_0`` and
    ``n_i`` the number of column segments at row i.  Forward elimination over
    the rows carries every source pattern ``Vin = e_k`` at once; the last row
    gives ``G'[k, j] = b_(M-1, j) / r_sense``.  fp64, M x N.
    """
    G = np.asarray(G, dtype=np.float64)
    M, N = G.shape
    if not np.all(np.isfinite(G)) or np.any(G < 0):
        raise ValueError("device conductances must be finite and >= 0 (0: an open device)")
    if not (r_row > 0 and r_col > 0 and r_sense > 0 and r_driver >= 0):
        raise ValueError("the row sweep needs positive wire and sense resistances")
    g_in, g_r, g_c, g_s = 1.0 / (r_driver + r_row), 1.0 / r_row, 1.0 / r_col, 1.0 / r_sense
    # chain conductance matrix of one row without the devices, in the banded
    # storage of scipy.linalg.solve_banded: (upper, diagonal, lower)
    lap_diag = np.zeros(N)
    lap_diag[0] += g_in
    lap_diag[:-1] += g_r
    lap_diag[1:] += g_r
    band = np.zeros((3, N))
    band[0, 1:] = -g_r
    band[2, :-1] = -g_r
    rhs_e0 = np.zeros((N, N + 1))
    A_prev_inv = None
    rhs = None          # N x M: the eliminated right-hand side of every pattern
    for i in range(M):
        band[1] = lap_diag + G[i]
        rhs_e0[:, :N] = np.diag(G[i])
        rhs_e0[:, N] = 0.0
        rhs_e0[0, N] = 1.0
        sol = sla.solve_banded((1, 1), band, rhs_e0)     # T_i^-1 [D_i | e_0]
        S = np.diag(G[i]) - G[i][:, None] * sol[:, :N]
        f = g_in * (G[i] * sol[:, N])
        n_seg = (1 if i > 0 else 0) + (1 if i + 1 < M else 0)
        A = S + g_c * n_seg * np.eye(N)
        if i == M - 1:
            A += g_s * np.eye(N)
        r_i = np.zeros((N, M))
        r_i[:, i] = f
        if i > 0:
            A = A - g_c * g_c * A_prev_inv
            r_i = r_i + g_c * (A_prev_inv @ rhs)
        A_prev_inv = np.linalg.inv(A)
        rhs = r_i
    b_last = A_prev_inv @ rhs            # N x M: b[M-1, j] for pattern e_k
    return (g_s * b_last).T
