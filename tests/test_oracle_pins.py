"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every check here is independent of the oracle's own formulas: worked examples
derived by hand, invariants the paper states (Sec. "Permutohedral Lattice",
Eq. splat / Eq. slice), brute-force Delaunay search on tiny inputs, closed
forms (affine reproduction, isometry), and library routines.
"""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from datagen.clouds import conv_weight, random_cloud
from oracle import lattice_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _random_hyperplane_points(d, n, seed, spread=12.0):
    rng = np.random.default_rng(seed)
    x = rng.uniform(-spread, spread, size=(n, d + 1))
    x -= x.mean(axis=1, keepdims=True)
    return x.astype(np.float32)


# --------------------------------------------------------------------------
# elevation (Sec. "Permutohedral Lattice", Sec. "Method": G / sigma)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("d", [1, 2, 3, 4])
def test_elevation_is_scaled_isometry_onto_hyperplane(d):
    """alpha E is alpha times an isometry from R^d onto H_d: columns orthogonal,
    norm alpha, each summing to zero (so every elevated point lies on H_d)."""
    sigma = np.ones(d, dtype=np.float32)
    alpha = 1.0
    fac = O.scale_factors(d, sigma, alpha)
    cols = O.elevate(np.eye(d, dtype=np.float32), fac).astype(np.float64)  # row j = column j of E
    G = cols @ cols.T
    assert np.allclose(G, np.eye(d), atol=1e-6)
    assert np.allclose(cols.sum(axis=1), 0.0, atol=1e-6)


@pytest.mark.parametrize("d", [2, 3, 4])
def test_elevation_norm_and_sum(d):
    rng = np.random.default_rng(7)
    g = rng.uniform(-3, 3, size=(500, d)).astype(np.float32)
    sigma = rng.uniform(0.2, 2.0, size=d).astype(np.float32)
    alpha = O.default_alpha(d)
    x = O.elevate(g, O.scale_factors(d, sigma, alpha)).astype(np.float64)
    s = g.astype(np.float64) / sigma.astype(np.float64)
    assert np.allclose(np.linalg.norm(x, axis=1), alpha * np.linalg.norm(s, axis=1), rtol=2e-6)
    assert np.all(np.abs(x.sum(axis=1)) <= 1e-5 * np.abs(x).max(axis=1) + 1e-6)


def test_scale_factor_values():
    f = O.scale_factors(3, [0.5, 0.25, 2.0], alpha=1.0)
    expect = [1 / (0.5 * np.sqrt(2)), 1 / (0.25 * np.sqrt(6)), 1 / (2.0 * np.sqrt(12))]
    assert np.allclose(f, expect, rtol=1e-7)
    assert f.dtype == np.float32
    # sigma given as a scalar broadcasts over the d axes
    assert np.array_equal(O.scale_factors(3, 0.3), O.scale_factors(3, [0.3] * 3))


# --------------------------------------------------------------------------
# enclosing simplex, keys, barycentric weights
# --------------------------------------------------------------------------

def test_worked_examples():
    cases = json.load(open(os.path.join(GOLDEN, "simplex_worked_examples.json")))["cases"]
    for c in cases:
        x = np.array([c["x"]], dtype=np.float32)
        r, rank = O.enclosing_simplex(x)
        b = O.barycentric(x, r, rank)[0]
        keys = O.simplex_keys(r, rank)[0]
        got = {tuple(int(v) for v in k): float(w) for k, w in zip(keys, b)}
        listed = 0.0
        for v, (num, den) in zip(c["vertices"], c["weights"]):
            assert tuple(v) in got, c["name"]
            assert abs(got[tuple(v)] - float(Fraction(num, den))) < 2e-7, c["name"]
            listed += float(Fraction(num, den))
        assert abs(listed - 1.0) < 1e-12
        for k, w in got.items():
            if list(k) not in c["vertices"]:
                assert abs(w) < 1e-7, c["name"]


@pytest.mark.parametrize("d", [1, 2, 3, 4])
def test_key_invariants(d):
    """Keys sum to 0; vertex k is congruent to k mod (d+1); consecutive simplex
    vertices differ by -n_j with j running over a permutation of 0..d."""
    x = _random_hyperplane_points(d, 2000, seed=d)
    r, rank = O.enclosing_simplex(x)
    keys = O.simplex_keys(r, rank)
    assert np.all(keys.sum(axis=2) == 0)
    for k in range(d + 1):
        assert np.all(np.mod(keys[:, k, :] - k, d + 1) == 0)
    n = (d + 1) * np.eye(d + 1, dtype=np.int64) - 1
    cyc = np.concatenate([keys, keys[:, :1, :]], axis=1)
    for p in range(0, 2000, 7):
        js = []
        for k in range(d + 1):
            diff = cyc[p, k + 1] - cyc[p, k]   # k = d closes the cycle back to remainder 0
            # -n_j: all ones except -d at coordinate j
            j = int(np.argmin(diff))
            assert np.array_equal(diff, -n[j]), (p, k, diff)
            js.append(j)
        assert sorted(js) == list(range(d + 1))


@pytest.mark.parametrize("d", [1, 2, 3, 4])
def test_barycentric_reconstruction(d):
    """b >= 0, sum b = 1 and sum_k b_k c_k = x: x lies in the simplex spanned by the keys."""
    x = _random_hyperplane_points(d, 5000, seed=10 + d)
    r, rank = O.enclosing_simplex(x)
    b = O.barycentric(x, r, rank)
    keys = O.simplex_keys(r, rank).astype(np.float64)
    assert b.min() >= -1e-6
    assert np.allclose(b.sum(axis=1), 1.0, atol=1e-12)
    rec = np.einsum("pk,pki->pi", b, keys)
    x64 = x.astype(np.float64)
    # x in fp32 is off H_d by rounding; compare on H_d
    x64 = x64 - x64.mean(axis=1, keepdims=True)
    assert np.allclose(rec, x64, atol=1e-5)


def _delaunay_simplex(x, d, n_near=3):
    """Brute force: the (d+1)-set of A*_d points, one per remainder class,
    that contains x and whose circumsphere holds no lattice point."""
    x = x.astype(np.float64)
    x = x - x.mean()
    dp1 = d + 1
    cands, cls = [], []
    for k in range(dp1):
        u = (x - k) / dp1
        base = np.floor(u[:d]).astype(np.int64)
        for off in itertools.product(range(-2, 3), repeat=d):
            z = base + np.array(off)
            zd = -k - z.sum()
            c = k + dp1 * np.append(z, zd)
            cands.append(c)
            cls.append(k)
    cands = np.array(cands, dtype=np.float64)
    cls = np.array(cls)
    dist = np.linalg.norm(cands - x, axis=1)
    near = [np.argsort(np.where(cls == k, dist, np.inf))[:n_near] for k in range(dp1)]
    found = []
    for combo in itertools.product(*near):
        P = cands[list(combo)]                          # [d+1, d+1]
        A = np.vstack([P.T, np.ones(dp1)])              # (d+2) x (d+1)
        if np.linalg.matrix_rank(A) < dp1:              # affinely dependent: not a d-simplex
            continue
        lam, *_ = np.linalg.lstsq(A, np.append(x, 1.0), rcond=None)
        if lam.min() < -1e-9 or np.abs(A @ lam - np.append(x, 1.0)).max() > 1e-9:
            continue
        M = np.vstack([2 * (P[1:] - P[0]), np.ones(dp1)])
        rhs = np.append((P[1:] ** 2).sum(1) - (P[0] ** 2).sum(), 0.0)
        o = np.linalg.solve(M, rhs)
        R2 = ((P[0] - o) ** 2).sum()
        inside = ((cands - o) ** 2).sum(1) < R2 * (1 - 1e-9)
        if inside.any():
            continue
        found.append((P, lam))
    return found


@pytest.mark.parametrize("d", [1, 2, 3, 4])
def test_enclosing_simplex_matches_brute_force_delaunay(d):
    x = _random_hyperplane_points(d, 60 if d == 4 else 120, seed=100 + d, spread=9.0)
    r, rank = O.enclosing_simplex(x)
    keys = O.simplex_keys(r, rank)
    b = O.barycentric(x, r, rank)
    checked = 0
    for p in range(x.shape[0]):
        if b[p].min() < 1e-4:      # within rounding of a face: several simplices are correct
            continue
        found = _delaunay_simplex(x[p], d)
        assert len(found) == 1, (p, len(found))
        P, lam = found[0]
        assert {tuple(v) for v in P.astype(np.int64)} == {tuple(v) for v in keys[p]}
        order = {tuple(v): w for v, w in zip(P.astype(np.int64), lam)}
        for k in range(d + 1):
            assert abs(order[tuple(keys[p, k])] - b[p, k]) < 1e-5
        checked += 1
    assert checked > x.shape[0] // 2


def test_rank_ties_lower_index_first():
    """All Delta equal: ranks follow the coordinate index; the simplex is still valid."""
    x = np.zeros((1, 4), dtype=np.float32)
    r, rank = O.enclosing_simplex(x)
    assert rank.tolist() == [[0, 1, 2, 3]]
    assert r.tolist() == [[0, 0, 0, 0]]
    b = O.barycentric(x, r, rank)
    assert b.tolist() == [[1.0, 0.0, 0.0, 0.0]]


# --------------------------------------------------------------------------
# splat / slice (Eq. splat, Eq. slice)
# --------------------------------------------------------------------------

def _small_lattice(d=3, m=3000, seed=3, C=5, n_batch=0):
    w = random_cloud(m, d, seed, extent=1.0, C=C, n_batch=n_batch)
    lat = O.build(w.pos, 0.15, batch=w.batch)
    return w, lat


def test_splat_mass_conservation():
    w, lat = _small_lattice()
    vals, wt, _ = O.splat(lat, w.feat)
    assert np.allclose(vals.sum(0), w.feat.astype(np.float64).sum(0), rtol=1e-10, atol=1e-9)
    assert abs(wt.sum() - w.m) < 1e-8


def test_splat_normalised_constant_field():
    w, lat = _small_lattice()
    const = np.full((w.m, 3), 2.5, dtype=np.float32)
    vals, wt, _ = O.splat(lat, const, normalize=True)
    nz = wt > 0
    assert np.allclose(vals[nz], 2.5, rtol=1e-12)
    assert np.all(vals[~nz] == 0)


def test_splat_then_slice_of_constant_is_constant():
    w, lat = _small_lattice()
    const = np.full((w.m, 2), -1.25, dtype=np.float32)
    vals, _, _ = O.splat(lat, const, normalize=True)
    out, _ = O.slice_(lat, vals)
    # zero-weight vertices of a simplex carry 0 but also get weight 0 in the slice
    assert np.allclose(out, -1.25, rtol=1e-12)


def test_single_point_splat_equals_weights():
    pos = np.array([[0.123, -0.456, 0.789]], dtype=np.float32)
    lat = O.build(pos, 0.1)
    vals, wt, _ = O.splat(lat, np.array([[3.0]], dtype=np.float32))
    assert lat.V == 4
    for k in range(4):
        v = lat.idx[0, k]
        assert np.isclose(vals[v, 0], 3.0 * lat.bary[0, k])
        assert np.isclose(wt[v], lat.bary[0, k])


def test_slice_reproduces_affine_field():
    """Barycentric interpolation is exact for affine functions: y_v = a . c_v + b0
    slices to a . x_p + b0 (splat/slice are piecewise linear, Sec. "Permutohedral Lattice")."""
    w, lat = _small_lattice(d=4, m=2000, seed=5)
    rng = np.random.default_rng(0)
    a = rng.standard_normal((lat.d + 1, 3))
    b0 = rng.standard_normal(3)
    y = lat.keys.astype(np.float64) @ a + b0
    out, _ = O.slice_(lat, y)
    expect = lat.x.astype(np.float64) @ a + b0
    # fp32 x is off H_d by rounding; project before comparing
    xh = lat.x.astype(np.float64)
    xh = xh - xh.mean(axis=1, keepdims=True)
    expect = xh @ a + b0
    assert np.allclose(out, expect, atol=1e-4 * np.abs(expect).max())


def test_splat_slice_adjoint():
    """<S f, y> = <f, Y y>: splat and slice use the same weights (Sec. "Common Operations")."""
    w, lat = _small_lattice(C=4)
    rng = np.random.default_rng(1)
    y = rng.standard_normal((lat.V, 4))
    Sf, _, _ = O.splat(lat, w.feat)
    Yy, _ = O.slice_(lat, y)
    lhs = (Sf * y).sum()
    rhs = (w.feat.astype(np.float64) * Yy).sum()
    assert np.isclose(lhs, rhs, rtol=1e-10)


def test_point_on_vertex_slices_vertex_value():
    """A point on a remainder-0 lattice vertex has weight 1 there."""
    d = 3
    c = np.array([4, -4, 8, -8], dtype=np.float64)
    # invert the elevation: g = sigma * E^T c / alpha, E from elevating unit vectors
    fac = O.scale_factors(d, 1.0, 1.0)
    E = O.elevate(np.eye(d, dtype=np.float32), fac).astype(np.float64).T   # [d+1, d]
    g = (E.T @ c)[None, :].astype(np.float32)
    lat = O.build(g, 1.0, alpha=1.0)
    k0 = [k for k in range(4) if np.array_equal(lat.keys[lat.idx[0, k]], c.astype(np.int64))]
    assert len(k0) == 1
    assert lat.bary[0, k0[0]] > 1 - 1e-5


def test_batched_lattice_is_concatenation_of_independent_lattices():
    w = random_cloud(3000, 3, 11, extent=1.0, C=3, n_batch=4)
    lat = O.build(w.pos, 0.2, batch=w.batch)
    start = 0
    for bb in range(4):
        sel = w.batch == bb
        sub = O.build(w.pos[sel], 0.2)
        assert np.array_equal(lat.keys[start:start + sub.V], sub.keys)
        assert np.all(lat.vbatch[start:start + sub.V] == bb)
        vals, _, _ = O.splat(lat, w.feat)
        svals, _, _ = O.splat(sub, w.feat[sel])
        assert np.allclose(vals[start:start + sub.V], svals, rtol=1e-12, atol=1e-12)
        start += sub.V
    assert start == lat.V
    nbr = O.neighbors(lat)
    present = nbr >= 0
    rows = np.repeat(np.arange(lat.V)[:, None], nbr.shape[1], axis=1)
    assert np.all(lat.vbatch[nbr[present]] == lat.vbatch[rows[present]])


# --------------------------------------------------------------------------
# neighbours (Sec. "Permutohedral Lattice": 2(d+1) neighbours at +-n_j)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("d", [2, 3, 4])
def test_neighbour_offsets_symmetry_and_presence(d):
    w = random_cloud(1500, d, 20 + d, extent=1.0, C=1)
    lat = O.build(w.pos, 0.2)
    nbr = O.neighbors(lat)
    T = 2 * (d + 1) + 1
    assert nbr.shape == (lat.V, T)
    assert np.array_equal(nbr[:, 0], np.arange(lat.V))
    keyset = {tuple(k) for k in lat.keys}
    n = (d + 1) * np.eye(d + 1, dtype=np.int64) - 1
    for v in range(0, lat.V, 3):
        for j in range(d + 1):
            for t, sgn in ((1 + j, 1), (d + 2 + j, -1)):
                q = tuple(lat.keys[v] + sgn * n[j])
                u = nbr[v, t]
                if q in keyset:
                    assert u >= 0 and tuple(lat.keys[u]) == q
                    back = d + 2 + j if sgn == 1 else 1 + j
                    assert nbr[u, back] == v
                else:
                    assert u == -1


@pytest.mark.parametrize("d", [2, 3, 4])
def test_simplex_edges_are_one_ring_taps(d):
    """Cyclically consecutive simplex vertices k, k+1 differ by -n_j (the edge
    vectors of the lattice): vertex k+1 must be tap d+2+j of vertex k."""
    w = random_cloud(800, d, 30 + d, extent=1.0, C=1)
    lat = O.build(w.pos, 0.2)
    nbr = O.neighbors(lat)
    for p in range(w.m):
        for k in range(d + 1):
            a = lat.idx[p, k]
            b = lat.idx[p, (k + 1) % (d + 1)]
            taps = np.nonzero(nbr[a] == b)[0]
            assert len(taps) == 1
            t = int(taps[0])
            assert t >= 1
            diff = lat.keys[b] - lat.keys[a]
            off = O.neighbor_offsets(d)[t]
            assert np.array_equal(diff, off)


# --------------------------------------------------------------------------
# convolution (Sec. "Common Operations": Convolving)
# --------------------------------------------------------------------------

def test_conv_identity_centre_tap():
    w, lat = _small_lattice(C=6)
    nbr = O.neighbors(lat)
    x = np.random.default_rng(2).standard_normal((lat.V, 6))
    W = np.zeros((6, nbr.shape[1], 6))
    W[:, 0, :] = np.eye(6)
    y, _ = O.conv(x, nbr, W)
    assert np.allclose(y, x, rtol=0, atol=0)


def test_conv_impulse_pins_tap_order_and_sign():
    """One non-zero vertex u (value e_i): a vertex v whose tap t reaches u
    receives W[:, t, i]; every other vertex receives 0."""
    d = 3
    w, lat = _small_lattice(d=d, C=2)
    nbr = O.neighbors(lat)
    T = nbr.shape[1]
    W = conv_weight(3, 4, d, seed=9).astype(np.float64)
    u = lat.V // 2
    x = np.zeros((lat.V, 3))
    x[u, 1] = 1.0
    y, _ = O.conv(x, nbr, W)
    offs = O.neighbor_offsets(d)
    keyidx = {tuple(k): i for i, k in enumerate(lat.keys)}
    expect = np.zeros_like(y)
    for t in range(T):
        v = keyidx.get(tuple(lat.keys[u] - offs[t]))   # key_v + off_t = key_u
        if v is not None:
            expect[v] += W[:, t, 1]
    assert np.allclose(y, expect, atol=0)
    assert np.abs(expect).sum() > 0


def test_conv_equals_dense_im2col_matmul():
    """The per-tap sum equals one dense [V, T C_in] x [T C_in, C_out] product."""
    w, lat = _small_lattice(C=3)
    nbr = O.neighbors(lat)
    T = nbr.shape[1]
    rng = np.random.default_rng(4)
    x = rng.standard_normal((lat.V, 5))
    W = rng.standard_normal((7, T, 5))
    Z = np.zeros((lat.V, T, 5))
    for t in range(T):
        ok = nbr[:, t] >= 0
        Z[ok, t] = x[nbr[ok, t]]
    dense = Z.reshape(lat.V, T * 5) @ W.reshape(7, T * 5).T
    y, _ = O.conv(x, nbr, W)
    assert np.allclose(y, dense, rtol=1e-12, atol=1e-12)


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    a = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-6, 6, 100000),
        # exact ties between two bf16 neighbours, both parities
        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0, -0.0, 65504.0], dtype=np.float32),
    ]).astype(np.float32)
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()
    got = O.round_bf16(a)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


# --------------------------------------------------------------------------
# DeformSlice + classifier (Sec. "Proposed Operations": DeformSlicing;
# Sec. "Implementation": fused with the last linear layer)
# --------------------------------------------------------------------------

def test_deform_slice_worked_examples():
    """Hand-derived tanh arguments (golden file) pin the Gather / MaxPool /
    SubtractMax / Linear order; f and the logits follow by direct sums."""
    import math
    with open(os.path.join(GOLDEN, "deform_slice_worked_examples.json")) as fh:
        ex = json.load(fh)["examples"]
    for e in ex:
        b = e["bary"]
        rows = e["rows"]
        dp1, C = len(rows), len(rows[0])
        delta = [math.tanh(a) for a in e["args"]]
        f = [sum((b[k] + delta[k]) * rows[k][c] for k in range(dp1)) for c in range(C)]
        X = np.array(rows)
        idx = np.arange(dp1)[None, :]
        out, dl, _ = O.deform_slice(idx, np.array([b]), X, np.array(e["w_delta"]), e["b_delta"])
        np.testing.assert_allclose(dl[0], delta, rtol=0, atol=1e-15)
        np.testing.assert_allclose(out[0], f, rtol=0, atol=1e-13)
        if "w_cls" in e:
            logits, _, _ = O.deform_slice(idx, np.array([b]), X, np.array(e["w_delta"]), e["b_delta"],
                                          np.array(e["w_cls"]), np.array(e["b_cls"]))
            np.testing.assert_allclose(logits[0], [f[0], f[1] + 1.0, f[0] + f[1] - 1.0], rtol=0, atol=1e-13)


def test_deform_slice_reduces_to_slice_and_saturates():
    """Zero offset weights and bias give Eq. (slice); a large bias drives
    every offset to +-1, adding +- the plain sum of the simplex's rows."""
    w = random_cloud(300, 3, seed=61, extent=1.0, C=1)
    lat = O.build(w.pos, 0.2)
    X = np.random.default_rng(62).standard_normal((lat.V, 5))
    f0, d0, _ = O.deform_slice(lat.idx, lat.bary, X, np.zeros(5), 0.0)
    ref, _ = O.slice_(lat, X)
    assert np.all(d0 == 0.0)
    np.testing.assert_allclose(f0, ref, rtol=0, atol=1e-12)
    rowsum = np.zeros((lat.m, 5))
    for p in range(lat.m):
        for k in range(4):
            rowsum[p] += X[lat.idx[p, k]]
    for sgn in (1.0, -1.0):
        f, dl, _ = O.deform_slice(lat.idx, lat.bary, X, np.ones(5), sgn * 40.0)
        assert np.all(dl == sgn)
        np.testing.assert_allclose(f, ref + sgn * rowsum, rtol=0, atol=1e-12)


def test_deform_slice_is_permutation_equivariant():
    """Enumerating a simplex's vertices in another order permutes the
    offsets the same way and leaves f unchanged (the max is symmetric)."""
    w = random_cloud(200, 2, seed=63, extent=1.0, C=1)
    lat = O.build(w.pos, 0.3)
    rng = np.random.default_rng(64)
    X = rng.standard_normal((lat.V, 6))
    wd = rng.standard_normal(6)
    f, dl, _ = O.deform_slice(lat.idx, lat.bary, X, wd, 0.3)
    perm = np.argsort(rng.random(lat.idx.shape), axis=1)
    idx_p = np.take_along_axis(lat.idx, perm, axis=1)
    bary_p = np.take_along_axis(lat.bary, perm, axis=1)
    f2, dl2, _ = O.deform_slice(idx_p, bary_p, X, wd, 0.3)
    np.testing.assert_allclose(f2, f, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dl2, np.take_along_axis(dl, perm, axis=1), rtol=0, atol=0)


@pytest.mark.parametrize("with_cls,invalid", [(True, False), (False, False), (True, True)])
def test_deform_slice_backward_matches_autograd(with_cls, invalid):
    """The hand-written backward of DeformSlice (and its classifier) against
    torch autograd of the forward's formula in float64 (torch's max sends
    its gradient to the index it returns, the first maximum, as the oracle
    does).  Some simplex slots set to -1 (a failed insertion) read zero rows
    and receive nothing."""
    import torch

    w = random_cloud(300, 3, seed=67, extent=1.0, C=1)
    lat = O.build(w.pos, 0.15)
    rng = np.random.default_rng(68)
    C, n_cls = 6, 4
    X = rng.standard_normal((lat.V, C))
    wd = rng.standard_normal(C)
    bd = 0.2
    Wc = rng.standard_normal((n_cls, C)) if with_cls else None
    bc = rng.standard_normal(n_cls) if with_cls else None
    idx = lat.idx.copy()
    if invalid:
        idx[rng.random(idx.shape) < 0.05] = -1
    G = rng.standard_normal((idx.shape[0], n_cls if with_cls else C))
    (dX, dwd, dbd, dWc, dbc), _ = O.deform_slice_backward(idx, lat.bary, X, wd, bd, G, lat.V, Wc, bc)

    Xt = torch.tensor(X, requires_grad=True)
    wt = torch.tensor(wd, requires_grad=True)
    bdt = torch.tensor(bd, dtype=torch.float64, requires_grad=True)
    it = torch.tensor(idx)
    b = torch.tensor(lat.bary)
    rows = Xt[it.clamp(min=0)] * (it >= 0)[..., None]
    q = b[..., None] * rows
    mx, _ = q.max(dim=1)
    delta = torch.tanh(bdt + (q - mx[:, None, :]) @ wt)
    f = ((b + delta)[..., None] * rows).sum(1)
    if with_cls:
        Wct = torch.tensor(Wc, requires_grad=True)
        bct = torch.tensor(bc, requires_grad=True)
        out = f @ Wct.T + bct
    else:
        out = f
    (out * torch.tensor(G)).sum().backward()
    np.testing.assert_allclose(dX, Xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dwd, wt.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.isclose(dbd, bdt.grad.item(), rtol=1e-10)
    if with_cls:
        np.testing.assert_allclose(dWc, Wct.grad.numpy(), rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(dbc, bct.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_deform_slice_backward_max_routes_to_first_fp32_maximum():
    """Two vertices whose products b x tie in float32 (but not in float64):
    the max's gradient goes to the lower slot, by the float32 decision."""
    idx = np.array([[0, 1]])
    b = np.array([[0.5, 0.5]])
    x0 = 1.0
    x1 = 1.0 + 2.0 ** -30                  # equal to x0 in float32, larger in float64
    X = np.array([[x0], [x1]])
    G = np.array([[1.0]])
    (dX, _, _, _, _), _ = O.deform_slice_backward(idx, b, X, np.array([1.0]), 0.0, G, 2)
    # forward (float64): mx = q_1, db_0 = tanh(0.5 (x0 - x1)), db_1 = 0, gf = 1;
    # dx_pk = (b + db_k) gf + b darg_k w - b S w [k == k*], darg_k = x_k (1 - db_k^2),
    # S = darg_0 + darg_1, and k* = 0 (the float32 tie goes to the first slot)
    db0 = np.tanh(0.5 * (x0 - x1))
    darg = np.array([x0 * (1.0 - db0 ** 2), x1])
    S = darg.sum()
    want = [(0.5 + db0) + 0.5 * darg[0] - 0.5 * S, 0.5 + 0.5 * darg[1]]
    np.testing.assert_allclose(dX[:, 0], want, rtol=0, atol=1e-15)
    # with the decision taken in float64 the gradient would have gone to slot 1
    assert abs(want[0] - (0.5 + db0 + 0.5 * darg[0])) > 0.5


def test_deform_slice_identity_classifier():
    """An identity classifier with zero bias returns f itself."""
    w = random_cloud(100, 3, seed=65, extent=1.0, C=1)
    lat = O.build(w.pos, 0.2)
    rng = np.random.default_rng(66)
    X = rng.standard_normal((lat.V, 4))
    wd = rng.standard_normal(4)
    f, _, _ = O.deform_slice(lat.idx, lat.bary, X, wd, -0.2)
    lg, _, _ = O.deform_slice(lat.idx, lat.bary, X, wd, -0.2, np.eye(4), np.zeros(4))
    np.testing.assert_allclose(lg, f, rtol=0, atol=0)


# --------------------------------------------------------------------------
# backward passes: each gradient is the transpose of the forward's Jacobian.
# Pinned against the Jacobian itself, built column by column from the forward
# oracle (pinned above) on tiny lattices, and against torch autograd.
# --------------------------------------------------------------------------

def _tiny_lattice(d=3, m=40, seed=21, sigma=0.35):
    w = random_cloud(m, d, seed, extent=1.0, C=2)
    return w, O.build(w.pos, sigma)


def _jacobian(f, shape_in):
    """Dense Jacobian of a linear map by applying it to every unit input."""
    n = int(np.prod(shape_in))
    cols = []
    for j in range(n):
        e = np.zeros(n)
        e[j] = 1.0
        cols.append(np.asarray(f(e.reshape(shape_in)), dtype=np.float64).ravel())
    return np.stack(cols, axis=1)


@pytest.mark.parametrize("d", [2, 3, 4])
def test_slice_backward_is_jacobian_transpose(d):
    w, lat = _tiny_lattice(d=d, seed=20 + d)
    C = 2
    J = _jacobian(lambda y: O.slice_(lat, y)[0], (lat.V, C))
    g = np.random.default_rng(d).standard_normal((lat.m, C))
    got, scale = O.slice_backward(lat, g)
    assert np.allclose(got.ravel(), J.T @ g.ravel(), rtol=1e-12, atol=1e-12)
    assert np.all(scale >= np.abs(got) - 1e-12)


@pytest.mark.parametrize("normalize", [False, True])
def test_splat_backward_is_jacobian_transpose(normalize):
    w, lat = _tiny_lattice(d=3, seed=31)
    C = 2
    J = _jacobian(lambda f: O.splat(lat, f, normalize=normalize)[0], (lat.m, C))
    _, wt, _ = O.splat(lat, w.feat)
    g = np.random.default_rng(5).standard_normal((lat.V, C))
    got, _ = O.splat_backward(lat, g, normalize=normalize, weight=wt)
    assert np.allclose(got.ravel(), J.T @ g.ravel(), rtol=1e-12, atol=1e-12)


def test_splat_backward_zero_weight_vertex():
    """A vertex whose every pair has weight 0 holds the constant 0 in the
    normalised splat, so no gradient flows through it."""
    pos = np.array([[0.0, 0.0, 0.0]], dtype=np.float32)   # on a remainder-0 vertex: 3 weights are 0
    lat = O.build(pos, 1.0)
    _, wt, _ = O.splat(lat, np.ones((1, 1), dtype=np.float32))
    assert (wt == 0).sum() == 3
    g = np.ones((lat.V, 1))
    got, _ = O.splat_backward(lat, g, normalize=True, weight=wt)
    assert np.allclose(got, 1.0)  # only the weight-1 vertex contributes, with 1/w = 1


@pytest.mark.parametrize("d", [2, 3])
def test_conv_backward_is_jacobian_transpose(d):
    w, lat = _tiny_lattice(d=d, m=30, seed=40 + d)
    nbr = O.neighbors(lat)
    T = nbr.shape[1]
    rng = np.random.default_rng(d)
    c_in, c_out = 2, 3
    x = rng.standard_normal((lat.V, c_in))
    W = rng.standard_normal((c_out, T, c_in))
    bias = rng.standard_normal(c_out)
    g = rng.standard_normal((lat.V, c_out))
    gx, gw, gb, gx_s, gw_s, gb_s = O.conv_backward(x, nbr, W, g)
    Jx = _jacobian(lambda xx: O.conv(xx, nbr, W)[0], (lat.V, c_in))
    Jw = _jacobian(lambda ww: O.conv(x, nbr, ww)[0], (c_out, T, c_in))
    Jb = _jacobian(lambda bb: O.conv(x, nbr, W, bb)[0] - O.conv(x, nbr, W)[0], (c_out,))
    assert np.allclose(gx.ravel(), Jx.T @ g.ravel(), rtol=1e-11, atol=1e-11)
    assert np.allclose(gw.ravel(), Jw.T @ g.ravel(), rtol=1e-11, atol=1e-11)
    assert np.allclose(gb, Jb.T @ g.ravel(), rtol=1e-11, atol=1e-11)
    for got, s in ((gx, gx_s), (gw, gw_s), (gb, gb_s)):
        assert np.all(s >= np.abs(got) - 1e-9)


def test_backward_matches_torch_autograd():
    """The whole chain splat -> conv -> slice, differentiated by torch autograd
    (float64, CPU) from a forward written with sparse/dense torch products,
    gives the oracle's chained backward."""
    torch = pytest.importorskip("torch")
    w, lat = _small_lattice(d=3, m=600, seed=12, C=3)
    nbr = O.neighbors(lat)
    T = nbr.shape[1]
    rng = np.random.default_rng(3)
    W = rng.standard_normal((4, T, 3))
    gout = rng.standard_normal((lat.m, 4))
    Bd = torch.from_numpy(lat.B.toarray())                          # [m, V]
    f = torch.tensor(w.feat.astype(np.float64), requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    xv = Bd.T @ f                                                   # splat
    Z = torch.zeros((lat.V, T, 3), dtype=torch.float64)
    for t in range(T):
        ok = torch.from_numpy(nbr[:, t] >= 0)
        Z[ok, t] = xv[torch.from_numpy(nbr[nbr[:, t] >= 0, t])]
    y = Z.reshape(lat.V, -1) @ Wt.reshape(4, -1).T                  # conv
    out = Bd @ y                                                    # slice
    (out * torch.from_numpy(gout)).sum().backward()
    gy, _ = O.slice_backward(lat, gout)
    vals, _, _ = O.splat(lat, w.feat)
    gx, gw, _, _, _, _ = O.conv_backward(vals, nbr, W, gy)
    gf, _ = O.splat_backward(lat, gx)
    assert np.allclose(gw, Wt.grad.numpy(), rtol=1e-10, atol=1e-10)
    assert np.allclose(gf, f.grad.numpy(), rtol=1e-10, atol=1e-10)


# --------------------------------------------------------------------------
# downsampling / upsampling (Sec. "Proposed Operations": Downsampling,
# Upsampling; the Coarsen figure: a strided and a transposed convolution)
# --------------------------------------------------------------------------

def _flip_transpose(W, d):
    """W'[i][s][o] = W[o][flip(s)][i], flip exchanging taps +n_j and -n_j."""
    T = W.shape[1]
    flip = [0] + [1 + (d + 1) + j for j in range(d + 1)] + [1 + j for j in range(d + 1)]
    return np.transpose(W[:, flip, :], (2, 1, 0))


def test_d1_down_and_up_are_textbook_stride2_conv_and_transpose():
    """In d = 1 the lattice is the integers a ~ key (a, -a); the ring offsets
    are +-1 (twice), so downsampling is the stride-2 correlation of a 1-D
    signal with a 3-tap kernel and upsampling is the stride-2 transposed
    convolution, here built with scipy.ndimage on a dense signal."""
    from scipy.ndimage import convolve1d, correlate1d

    g = np.linspace(-3.0, 5.0, 4001, dtype=np.float32)[:, None]
    sigma = 0.3
    fine = O.build(g, sigma)
    coarse = O.coarsen(g, sigma)
    a = fine.keys[:, 0]
    ac = coarse.keys[:, 0]
    assert np.array_equal(a, np.arange(a.min(), a.max() + 1))      # every cell occupied
    assert np.array_equal(ac, np.arange(ac.min(), ac.max() + 1))
    rng = np.random.default_rng(0)
    W = rng.standard_normal((1, 5, 1))
    K = {-1: W[0, 2, 0] + W[0, 3, 0], 0: W[0, 0, 0], 1: W[0, 1, 0] + W[0, 4, 0]}
    # dense fine signal on [lo, hi], zero-padded around the lattice's range
    lo, hi = 2 * ac.min() - 2, 2 * ac.max() + 2
    assert lo <= a.min() and hi >= a.max()
    x = rng.standard_normal(fine.V)
    X = np.zeros(hi - lo + 1)
    X[a - lo] = x
    full = correlate1d(X, [K[-1], K[0], K[1]], mode="constant", cval=0.0)
    y, _ = O.downsample(fine, coarse, x[:, None], W)
    assert np.allclose(y[:, 0], full[2 * ac - lo], rtol=1e-12, atol=1e-12)

    U = rng.standard_normal((1, 5, 1))
    k = {-1: U[0, 1, 0] + U[0, 4, 0], 0: U[0, 0, 0], 1: U[0, 2, 0] + U[0, 3, 0]}
    yc = rng.standard_normal(coarse.V)
    Zup = np.zeros(hi - lo + 1)
    Zup[2 * ac - lo] = yc                                      # zero insertion
    Z = convolve1d(Zup, [k[-1], k[0], k[1]], mode="constant", cval=0.0)
    z, _ = O.upsample(coarse, fine, yc[:, None], U)
    assert np.allclose(z[:, 0], Z[a - lo], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("d", [2, 3, 4])
def test_downsample_is_fine_conv_sampled_at_embedded_vertices(d):
    """Where 2c' is itself a fine vertex v, the coarse value equals the fine
    lattice's convolution at v: its taps are v's 1-ring (a strided conv)."""
    w = random_cloud(2500, d, 50 + d, extent=1.0, C=2)
    sigma = {2: 0.08, 3: 0.15, 4: 0.3}[d]
    fine = O.build(w.pos, sigma)
    coarse = O.coarsen(w.pos, sigma)
    nbr = O.neighbors(fine)
    rng = np.random.default_rng(d)
    x = rng.standard_normal((fine.V, 3))
    W = rng.standard_normal((4, nbr.shape[1], 3))
    y, _ = O.downsample(fine, coarse, x, W)
    yf, _ = O.conv(x, nbr, W)
    v = O.lookup(fine, 2 * coarse.keys)
    assert (v >= 0).mean() > 0.3
    assert np.allclose(y[v >= 0], yf[v[v >= 0]], rtol=1e-12, atol=1e-12)
    # coarse keys embed into the fine lattice: 2c' sums to zero, coordinates congruent mod d+1
    e = 2 * coarse.keys
    assert np.all(e.sum(axis=1) == 0) and np.all((e - e[:, :1]) % (d + 1) == 0)


@pytest.mark.parametrize("d,batched", [(2, False), (3, False), (3, True), (4, False)])
def test_upsample_is_adjoint_of_downsample(d, batched):
    """<down_W(x), y> = <x, up_W'(y)> with W' the flipped transposed weights:
    upsampling is the transposed convolution of downsampling."""
    w = random_cloud(2000, d, 60 + d, extent=1.0, C=2, n_batch=3 if batched else 0)
    sigma = {2: 0.08, 3: 0.15, 4: 0.3}[d]
    fine = O.build(w.pos, sigma, batch=w.batch)
    coarse = O.coarsen(w.pos, sigma, batch=w.batch)
    T = 2 * (d + 1) + 1
    rng = np.random.default_rng(7)
    W = rng.standard_normal((3, T, 2))
    x = rng.standard_normal((fine.V, 2))
    y = rng.standard_normal((coarse.V, 3))
    dx, _ = O.downsample(fine, coarse, x, W)
    uy, _ = O.upsample(coarse, fine, y, _flip_transpose(W, d))
    assert np.isclose((dx * y).sum(), (x * uy).sum(), rtol=1e-10)
    # and the taps that exist are not few
    assert (O.up_neighbors(coarse, fine) >= 0).sum() > fine.V // 2


@pytest.mark.parametrize("d,batched", [(2, False), (3, True), (4, False)])
def test_resample_backward_is_the_adjoint_and_the_weight_derivative(d, batched):
    """Both resamplings are bilinear in (input, weights): for random x, W, g
    <op(x, W), g> = <x, grad_x(g)> = <W, grad_w(g)>, and grad_bias = sum_v g_v
    (the derivative of <op(x, W) + bias, g> in bias).  The input gradient of
    each is also the other resampling with the flipped transposed weights,
    the identity the GPU path computes it by."""
    w = random_cloud(1500, d, 80 + d, extent=1.0, C=2, n_batch=2 if batched else 0)
    sigma = {2: 0.08, 3: 0.15, 4: 0.3}[d]
    fine = O.build(w.pos, sigma, batch=w.batch)
    coarse = O.coarsen(w.pos, sigma, batch=w.batch)
    T = 2 * (d + 1) + 1
    rng = np.random.default_rng(90 + d)
    for up in (False, True):
        src, dst = (coarse, fine) if up else (fine, coarse)
        C_in, C_out = 3, 2
        W = rng.standard_normal((C_out, T, C_in))
        x = rng.standard_normal((src.V, C_in))
        g = rng.standard_normal((dst.V, C_out))
        fwd = O.upsample if up else O.downsample
        bwd = O.upsample_backward if up else O.downsample_backward
        y, _ = fwd(src, dst, x, W)
        gx, gw, gb, _, _, _ = bwd(src, dst, x, W, g)
        ip = (y * g).sum()
        assert gx.shape == x.shape and gw.shape == W.shape
        assert np.isclose(ip, (x * gx).sum(), rtol=1e-10)
        assert np.isclose(ip, (W * gw).sum(), rtol=1e-10)
        yb, _ = fwd(src, dst, x, W, bias=np.ones(C_out))
        assert np.allclose(gb, g.sum(axis=0)) and np.isclose(((yb - y) * g).sum(), gb.sum(), rtol=1e-10)
        other = O.downsample if up else O.upsample
        gx2, _ = other(dst, src, g, _flip_transpose(W, d))
        assert np.allclose(gx, gx2, rtol=1e-12, atol=1e-12)


def test_upsample_taps_follow_remainder_parity_in_3d():
    """d = 3: a vertex's coordinates share its remainder mod 4, so an
    even-remainder fine vertex u has u/2 integral and every (u +- n_j)/2
    fractional (centre tap only), and an odd-remainder one the reverse."""
    w = random_cloud(3000, 3, 70, extent=1.0, C=2)
    fine = O.build(w.pos, 0.15)
    coarse = O.coarsen(w.pos, 0.15)
    up = O.up_neighbors(coarse, fine)
    rem = fine.keys[:, 0] % 4
    even = rem % 2 == 0
    assert np.all(up[~even, 0] == -1)
    assert np.all(up[even, 1:] == -1)
    assert (up[even, 0] >= 0).mean() > 0.2 and (up[~even, 1:] >= 0).any(axis=1).mean() > 0.2


# --------------------------------------------------------------------------
# Distribute + PointNet + per-vertex max (Sec. "Proposed Operations":
# Distribute; the PointNet block of the network figure)
# --------------------------------------------------------------------------

def test_distribute_pointnet_worked_example_d1():
    """Two points of one lattice cell in d = 1 (keys (0,0) and (1,-1)), worked
    by hand.  Both vertices receive both points; the local mean is their
    midpoint 0.5, so the distributed rows are (off, f) = (-0.2, 1) and
    (0.2, -3).  Block 1: a = (1, 1), s = (1, 5) (ReLU is then the identity
    here), W = [[1, 0], [-1, 0], [0, 1]], b = (-1, 1, -5) gives (off, -off, f);
    block 2: a = 1, s = 0, W = [[1, 1, 0], [0, 0, 1]], b = 0 gives
    (|off|, relu f).  Rows (0.2, 1) and (0.2, 0): the max is (0.2, 1) at both
    vertices.  Without the mean it would be (0.7, 1); with a weighted mean
    0.28; with a sum (0.4, 1); with [f ; off] concatenated (1, 0.2)."""
    g = np.array([[0.3], [0.7]], dtype=np.float32)
    f = np.array([[1.0], [-3.0]], dtype=np.float32)
    lat = O.build(g, 1.0, alpha=1.0)
    assert lat.V == 2 and sorted(map(tuple, lat.keys)) == [(0, 0), (1, -1)]
    mu = O.local_mean(lat, g)
    assert np.allclose(mu, 0.5, atol=1e-7)
    L1 = (np.ones(2), np.array([1.0, 5.0]), np.array([[1.0, 0.0], [-1.0, 0.0], [0.0, 1.0]]),
          np.array([-1.0, 1.0, -5.0]))
    L2 = (np.ones(3), np.zeros(3), np.array([[1.0, 1.0, 0.0], [0.0, 0.0, 1.0]]), np.zeros(2))
    out, scale, _ = O.distribute_pointnet(lat, g, f, [L1, L2])
    assert np.allclose(out, [[0.2, 1.0], [0.2, 1.0]], atol=1e-6)
    assert np.all(scale >= np.abs(out))


def test_local_mean_offsets_sum_to_zero_and_counts():
    w, lat = _small_lattice(d=3, m=2000, seed=80, C=3)
    mu = O.local_mean(lat, w.pos)
    g = w.pos.astype(np.float64)
    resid = np.zeros_like(mu)
    m, dp1 = lat.idx.shape
    for k in range(dp1):
        np.add.at(resid, lat.idx[:, k], g - mu[lat.idx[:, k]])
    assert np.abs(resid).max() < 1e-9
    # |J_v| from the keys themselves: the points whose simplex has v's key
    keys = O.simplex_keys(*O.enclosing_simplex(lat.x))
    cnt = {}
    for kk in keys.reshape(-1, dp1):
        cnt[tuple(kk)] = cnt.get(tuple(kk), 0) + 1
    n = np.bincount(lat.idx.ravel(), minlength=lat.V)
    assert all(cnt[tuple(lat.keys[v])] == n[v] for v in range(lat.V))


def test_distribute_pointnet_matches_torch_index_reduce():
    """The same network built from torch primitives (float64, CPU):
    index_reduce 'mean' for the local mean, F.linear for the 1x1 layers and
    index_reduce 'amax' for the per-vertex max."""
    torch = pytest.importorskip("torch")
    from datagen.clouds import pointnet_weights

    w, lat = _small_lattice(d=3, m=3000, seed=81, C=4)
    layers = pointnet_weights(3 + 4, 3, 0.15, seed=82)
    out, _, mu = O.distribute_pointnet(lat, w.pos, w.feat, layers)
    m, dp1 = lat.idx.shape
    v = torch.from_numpy(lat.idx.ravel())
    p = torch.arange(m).repeat_interleave(dp1)
    g = torch.from_numpy(w.pos.astype(np.float64))
    f = torch.from_numpy(w.feat.astype(np.float64))
    tmu = torch.zeros((lat.V, 3), dtype=torch.float64).index_reduce_(0, v, g[p], "mean", include_self=False)
    h = torch.cat([g[p] - tmu[v], f[p]], dim=1)
    for a, s, W, b in layers:
        h = torch.nn.functional.linear(torch.relu(torch.from_numpy(a.astype(np.float64)) * h
                                                  + torch.from_numpy(s.astype(np.float64))),
                                       torch.from_numpy(W.astype(np.float64)), torch.from_numpy(b.astype(np.float64)))
    tout = torch.zeros((lat.V, h.shape[1]), dtype=torch.float64).index_reduce_(0, v, h, "amax", include_self=False)
    assert np.allclose(mu, tmu.numpy(), rtol=1e-12, atol=1e-12)
    assert np.allclose(out, tout.numpy(), rtol=1e-12, atol=1e-12)


def test_distribute_pointnet_is_point_permutation_invariant():
    from datagen.clouds import pointnet_weights

    w, lat = _small_lattice(d=4, m=1500, seed=83, C=2)
    layers = pointnet_weights(4 + 2, 4, 0.15, seed=84)
    out, _, _ = O.distribute_pointnet(lat, w.pos, w.feat, layers)
    perm = np.random.default_rng(0).permutation(w.m)
    lat2 = O.build(w.pos[perm], 0.15)
    out2, _, _ = O.distribute_pointnet(lat2, w.pos[perm], w.feat[perm], layers)
    assert np.array_equal(lat.keys, lat2.keys)
    assert np.allclose(out, out2, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------
# Group normalisation in the PointNet of Distribute (Sec. "Implementation":
# every convolution is pre-activated by a group normalisation of 32 groups
# and a ReLU; the network figure's PointNet block is GN, ReLU, 1x1, three
# times, then the max-pool)
# --------------------------------------------------------------------------

def test_default_groups_are_the_largest_divisor_up_to_32():
    assert [O.default_groups(k) for k in (1, 4, 9, 16, 32, 48, 64, 96, 128)] == [1, 4, 9, 16, 32, 24, 32, 32, 32]


@pytest.mark.parametrize("K,groups", [(8, 1), (8, 2), (8, 8), (9, 3), (9, 9), (32, 32), (64, 32)])
def test_group_norm_matches_torch(K, groups):
    """torch.nn.functional.group_norm (float64, CPU) on each sample's rows,
    laid out as one [1, K, N] sample."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(K * 100 + groups)
    N = 500
    h = rng.normal(size=(N, K)) * rng.uniform(0.1, 5.0, size=K) + rng.normal(size=K) * 3
    seg = rng.integers(0, 3, size=N) * 7          # three samples with ids 0, 7, 14
    gamma, beta = rng.normal(size=K), rng.normal(size=K)
    out, means, varis, samples = O.group_norm(h, seg, groups, gamma, beta, eps=1e-5)
    assert list(samples) == [0, 7, 14]
    for i, s in enumerate(samples):
        x = torch.from_numpy(h[seg == s].T.copy())[None]
        ref = torch.nn.functional.group_norm(x, groups, torch.from_numpy(gamma), torch.from_numpy(beta), eps=1e-5)
        assert np.allclose(out[seg == s], ref[0].numpy().T, rtol=1e-12, atol=1e-12)
        xg = x[0].reshape(groups, -1)
        assert np.allclose(means[i], xg.mean(dim=1).numpy(), rtol=1e-12, atol=1e-12)
        assert np.allclose(varis[i], xg.var(dim=1, unbiased=False).numpy(), rtol=1e-12, atol=1e-12)


def test_group_norm_standardises_each_group_and_ignores_its_affine():
    """With gamma = 1, beta = 0 and eps = 0 every (sample, group) comes out
    with mean 0 and variance 1, and scaling a (sample, group) by a positive
    factor and shifting it by a constant changes nothing."""
    rng = np.random.default_rng(5)
    N, K, G = 400, 12, 4
    h = rng.normal(size=(N, K)) * 2 + 1
    seg = (np.arange(N) >= 150).astype(np.int64)
    out, _, _, _ = O.group_norm(h, seg, G, np.ones(K), np.zeros(K), eps=0.0)
    for s in (0, 1):
        for g in range(G):
            x = out[seg == s][:, g * 3:(g + 1) * 3]
            assert abs(x.mean()) < 1e-12 and abs(x.var() - 1.0) < 1e-12
    h2 = h.copy()
    for s in (0, 1):
        for g in range(G):
            a, c = rng.uniform(0.5, 4.0), rng.normal() * 10
            rows = seg == s
            h2[np.ix_(rows, range(g * 3, (g + 1) * 3))] = a * h[np.ix_(rows, range(g * 3, (g + 1) * 3))] + c
    out2, _, _, _ = O.group_norm(h2, seg, G, np.ones(K), np.zeros(K), eps=0.0)
    assert np.allclose(out, out2, rtol=1e-10, atol=1e-10)


def test_distribute_pointnet_gn_worked_example_d1():
    """Three points in d = 1 (alpha = sigma = 1, vertices at g = k sqrt 2),
    worked by hand.  g = 0.3 and 0.7 fall in the cell of keys (0,0), (1,-1);
    g = 2.0 in the cell of (1,-1), (2,-2).  Local means: 0.5, 1.0, 2.0.
    Rows (offset, f) with f = (1, -1, 0): v0 (-0.2, 1), (0.2, -1); v1
    (-0.7, 1), (-0.3, -1), (1.0, 0); v2 (0.0, 0).  One block: GN with two
    groups (one channel each), gamma = 1, beta = 0, eps = 0; ReLU; W = I,
    b = 0.  Over all six rows the offsets have mean 0 (they sum to zero per
    vertex) and variance 1.66 / 6, so they divide by sqrt(0.27667) =
    0.525991; the features have mean 0 and variance 4 / 6, so they divide by
    0.816497.  The max per vertex: v0 (0.2 / 0.525991, 1 / 0.816497) =
    (0.380235, 1.224745); v1 (1.0 / 0.525991, 1.224745) = (1.901173,
    1.224745); v2 (0, 0).  Statistics per vertex instead of per cloud would
    give v0 (1, 1) and no answer at v2 (zero variance)."""
    g = np.array([[0.3], [0.7], [2.0]], dtype=np.float32)
    f = np.array([[1.0], [-1.0], [0.0]], dtype=np.float32)
    lat = O.build(g, 1.0, alpha=1.0)
    assert [tuple(k) for k in lat.keys] == [(0, 0), (1, -1), (2, -2)]
    layer = (np.ones(2), np.zeros(2), np.eye(2), np.zeros(2))
    out, scale, mu = O.distribute_pointnet(lat, g, f, [layer], groups=[2], eps=0.0)
    assert np.allclose(mu.ravel(), [0.5, 1.0, 2.0], atol=1e-7)
    assert np.allclose(out, [[0.380235, 1.224745], [1.901173, 1.224745], [0.0, 0.0]], atol=2e-6)
    assert np.all(scale >= np.abs(out))


def _torch_pointnet_gn(torch, lat, pos, feat, layers, groups, eps):
    """The same network from torch primitives (float64, CPU): index_reduce
    'mean' for the local mean, group_norm per cloud, F.linear, index_reduce
    'amax' for the per-vertex max."""
    m, dp1 = lat.idx.shape
    v = torch.from_numpy(lat.idx.ravel())
    p = torch.arange(m).repeat_interleave(dp1)
    g = torch.from_numpy(pos.astype(np.float64))
    tmu = torch.zeros((lat.V, pos.shape[1]), dtype=torch.float64).index_reduce_(0, v, g[p], "mean",
                                                                               include_self=False)
    h = torch.cat([g[p] - tmu[v], torch.from_numpy(feat.astype(np.float64))[p]], dim=1)
    seg = torch.from_numpy(lat.vbatch)[v] if lat.vbatch is not None else torch.zeros(len(v), dtype=torch.int64)
    for (ga, be, W, b), G in zip(layers, groups):
        hn = torch.empty_like(h)
        for s in torch.unique(seg):
            rows = seg == s
            hn[rows] = torch.nn.functional.group_norm(h[rows].T[None], G, torch.from_numpy(ga.astype(np.float64)),
                                                      torch.from_numpy(be.astype(np.float64)), eps=eps)[0].T
        h = torch.nn.functional.linear(torch.relu(hn), torch.from_numpy(W.astype(np.float64)),
                                       torch.from_numpy(b.astype(np.float64)))
    return torch.zeros((lat.V, h.shape[1]), dtype=torch.float64).index_reduce_(0, v, h, "amax", include_self=False)


@pytest.mark.parametrize("n_batch", [0, 3])
def test_distribute_pointnet_gn_matches_torch(n_batch):
    torch = pytest.importorskip("torch")
    from datagen.clouds import pointnet_gn_weights

    w, lat = _small_lattice(d=3, m=3000, seed=85, C=5, n_batch=n_batch)
    layers = pointnet_gn_weights(3 + 5, seed=86)
    groups = [O.default_groups(k) for k in (8, 16, 32)]
    out, _, _ = O.distribute_pointnet(lat, w.pos, w.feat, layers, groups=groups, eps=1e-5)
    ref = _torch_pointnet_gn(torch, lat, w.pos, w.feat, layers, groups, 1e-5)
    assert np.allclose(out, ref.numpy(), rtol=1e-10, atol=1e-10)
    # coarser groups than the default (block 1: one group of all 8 channels)
    out2, _, _ = O.distribute_pointnet(lat, w.pos, w.feat, layers, groups=[1, 4, 8], eps=1e-5)
    ref2 = _torch_pointnet_gn(torch, lat, w.pos, w.feat, layers, [1, 4, 8], 1e-5)
    assert np.allclose(out2, ref2.numpy(), rtol=1e-10, atol=1e-10)
    assert not np.allclose(out, out2, rtol=1e-3, atol=1e-3)


@pytest.mark.parametrize("n_batch,use_groups", [(0, True), (3, True), (0, False)])
def test_distribute_pointnet_backward_matches_autograd(n_batch, use_groups):
    """The hand-written backward of the PointNet blocks (group normalisation
    or the fixed affine, ReLU, the 1x1 layers, the per-vertex max) against
    torch autograd of the forward built from torch primitives, float64:
    every block's gamma / a, beta / s, W and b.  torch's amax sends the
    gradient to the maximum (evenly among exact ties; random data has none)."""
    torch = pytest.importorskip("torch")
    from datagen.clouds import pointnet_gn_weights

    w, lat = _small_lattice(d=3, m=800, seed=87, C=2, n_batch=n_batch)
    layers = pointnet_gn_weights(3 + 2, seed=88)
    groups = [O.default_groups(k) for k in (5, 16, 32)] if use_groups else None
    rng = np.random.default_rng(89)
    G = rng.standard_normal((lat.V, 64))
    grads, am, h3, v, _, _ = O.distribute_pointnet_backward(lat, w.pos, w.feat, layers, G, groups=groups, eps=1e-5)

    m, dp1 = lat.idx.shape
    vt = torch.from_numpy(lat.idx.ravel())
    p = torch.arange(m).repeat_interleave(dp1)
    g = torch.from_numpy(w.pos.astype(np.float64))
    tmu = torch.zeros((lat.V, 3), dtype=torch.float64).index_reduce_(0, vt, g[p], "mean", include_self=False)
    h = torch.cat([g[p] - tmu[vt], torch.from_numpy(w.feat.astype(np.float64))[p]], dim=1)
    seg = torch.from_numpy(lat.vbatch)[vt] if lat.vbatch is not None else torch.zeros(len(vt), dtype=torch.int64)
    params = []
    for li, (ga, be, W, b) in enumerate(layers):
        ga, be, W, b = (torch.tensor(np.asarray(x, np.float64), requires_grad=True) for x in (ga, be, W, b))
        params.append((ga, be, W, b))
        if use_groups:
            parts = []
            hn = torch.zeros_like(h)
            for s_ in torch.unique(seg):
                rows = torch.nonzero(seg == s_)[:, 0]
                gn = torch.nn.functional.group_norm(h[rows].T[None], groups[li], ga, be, eps=1e-5)[0].T
                hn = hn.index_put((rows,), gn)
        else:
            hn = ga * h + be
        h = torch.nn.functional.linear(torch.relu(hn), W, b)
    out = torch.zeros((lat.V, 64), dtype=torch.float64).index_reduce(0, vt, h, "amax", include_self=False)
    (out * torch.from_numpy(G)).sum().backward()
    for (da, ds, dW, db), (ga, be, W, b) in zip(grads, params):
        np.testing.assert_allclose(da, ga.grad.numpy(), rtol=1e-9, atol=1e-9)
        np.testing.assert_allclose(ds, be.grad.numpy(), rtol=1e-9, atol=1e-9)
        np.testing.assert_allclose(dW, W.grad.numpy(), rtol=1e-9, atol=1e-9)
        np.testing.assert_allclose(db, b.grad.numpy(), rtol=1e-9, atol=1e-9)
    # the max's rows: each vertex's winning row is one of its own, and holds the forward's value
    out_ref, _, _ = O.distribute_pointnet(lat, w.pos, w.feat, layers, groups=groups, eps=1e-5)
    assert np.all(v[am] == np.arange(lat.V)[:, None])
    np.testing.assert_allclose(np.take_along_axis(h3, am, axis=0), out_ref, rtol=0, atol=1e-12)


def test_distribute_pointnet_gn_statistics_are_per_cloud():
    """A batched lattice normalises each batch id over its own rows: the
    output equals the clouds run one by one, and a cloud whose positions are
    shifted and whose features are scaled and shifted (each feature channel
    is its own group in block 1) gives the same output as the original."""
    from datagen.clouds import pointnet_gn_weights

    w = random_cloud(1200, 3, 87, extent=1.0, C=3)
    pos2 = (w.pos + np.float32(3.0)).astype(np.float32)
    feat2 = (w.feat * np.float32(8.0) - np.float32(5.0)).astype(np.float32)
    layers = pointnet_gn_weights(3 + 3, seed=88)
    groups = [O.default_groups(k) for k in (6, 16, 32)]
    lat1 = O.build(w.pos, 0.15)
    out1, _, _ = O.distribute_pointnet(lat1, w.pos, w.feat, layers, groups=groups, eps=0.0)
    pos = np.concatenate([w.pos, pos2])
    feat = np.concatenate([w.feat, feat2])
    batch = np.repeat(np.array([0, 1], dtype=np.int32), w.m)
    latb = O.build(pos, 0.15, batch=batch)
    outb, _, _ = O.distribute_pointnet(latb, pos, feat, layers, groups=groups, eps=0.0)
    lat2 = O.build(pos2, 0.15)
    out2, _, _ = O.distribute_pointnet(lat2, pos2, feat2, layers, groups=groups, eps=0.0)
    assert np.allclose(outb[latb.vbatch == 0], out1, rtol=1e-9, atol=1e-9)
    assert np.allclose(outb[latb.vbatch == 1], out2, rtol=1e-9, atol=1e-9)
    # The shifted cloud has its own lattice (the shift is not a lattice
    # translation), so compare the block-1 normalisation of its feature
    # channels, which does not depend on the vertex set: the same values, to
    # the float32 rounding of 8 f - 5.
    h1, _, _, seg1, _, _ = O.distribute_rows(lat1, w.pos, w.feat)
    h2, _, _, seg2, _, _ = O.distribute_rows(lat2, pos2, feat2)
    n1, _, _, _ = O.group_norm(h1[:, 3:], seg1, 3, np.ones(3), np.zeros(3), eps=0.0)
    n2, _, _, _ = O.group_norm(h2[:, 3:], seg2, 3, np.ones(3), np.zeros(3), eps=0.0)
    assert np.allclose(np.sort(n1, axis=0), np.sort(n2, axis=0), rtol=1e-6, atol=1e-6)
