"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bar (per stage): bit-exact key set, per-point simplex vertices and
neighbour table after canonical ordering; barycentric weights within 1e-5
absolute; fp32 splat / conv / slice within 1e-5 of the sum of |terms| of each
output element; the bf16 MFMA conv within 2e-2 of that sum against the
fp32-input oracle and within 1e-5 against the oracle fed the same
bf16-rounded inputs.
"""
import numpy as np
import pytest
import torch

from datagen.clouds import conv_weight, deform_weights, make_workload, random_cloud, random_rows
from oracle import lattice_oracle as O
from tests.gpu_util import (BARY_ABS, REL_BF16, REL_F32, GpuLattice, assert_close_scaled, check_lattice, dev,
                            to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2108_03917_amd import load_library

    load_library()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _lattice(d, sigma, m, **kw):
    from paper_2108_03917_amd import Lattice

    return Lattice(d, sigma, max_points=max(m, 1), **kw)


# ---------------------------------------------------------------------------
# splat: keys, simplex records, values (Sec. "Permutohedral Lattice", Eq. splat)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d,m,sigma,C", [(1, 3000, 0.05, 3), (2, 5000, 0.08, 5), (3, 6000, 0.15, 64),
                                         (3, 7001, 0.1, 1), (4, 5000, 0.3, 16)])
def test_splat_parity(d, m, sigma, C):
    w = random_cloud(m, d, seed=100 + d, extent=1.0, C=C)
    L = _lattice(d, sigma, m)
    g = GpuLattice(L, w.pos, w.feat)
    lat = O.build(w.pos, sigma)
    check_lattice(g, lat)
    ref, wref, scale = O.splat(lat, w.feat)
    assert_close_scaled(g.values(), ref, scale, REL_F32, "splat values")
    assert_close_scaled(g.weight(), wref, wref, REL_F32, "splat weight")


def _clustered_cloud(seed, C, m_dense=6000, m_sparse=3000):
    """A few tight clusters (vertices hit by thousands of points) plus a
    sparse background (short pair lists), so that one splat exercises both
    the per-vertex and the split-list gather."""
    rng = np.random.default_rng(seed)
    centres = rng.uniform(-0.8, 0.8, size=(3, 3))
    dense = centres[rng.integers(0, 3, m_dense)] + rng.normal(0, 0.01, size=(m_dense, 3))
    sparse = rng.uniform(-1, 1, size=(m_sparse, 3))
    pos = np.concatenate([dense, sparse]).astype(np.float32)[rng.permutation(m_dense + m_sparse)]
    feat = rng.standard_normal((pos.shape[0], C)).astype(np.float32)
    return pos, feat


@pytest.mark.parametrize("C,values_dtype,normalize", [(3, "f32", False), (64, "f32", False), (64, "bf16", False),
                                                      (128, "f32", True), (520, "f32", False), (0, "f32", False),
                                                      (12, "f32", False), (32, "bf16", False), (96, "f32", True),
                                                      (256, "f32", False)])
def test_splat_long_pair_lists(C, values_dtype, normalize):
    """Vertices with up to thousands of (point, vertex) pairs: their lists are
    summed in parts of 32 pairs and the parts added in order; the result must
    not depend on that split.  Two splats in a row on one lattice (the second smaller)
    check that no per-split state leaks from the first.  Channel counts cover
    every group width of the float4 gather (4 to 64 lanes, with idle lanes
    when C / 4 is not a power of two) and the scalar one."""
    sigma = 0.1
    L = _lattice(3, sigma, 9000)
    for rep, (md, ms) in enumerate([(6000, 3000), (2500, 700)]):
        pos, feat = _clustered_cloud(40 + rep, max(C, 1), md, ms)
        feat_in = to_dev(feat) if C > 0 else None
        vals, wt = L.splat(to_dev(pos), feat_in, normalize=normalize, values_dtype=values_dtype,
                           want_weight=True)
        V = L.num_vertices()
        keys = L.keys().cpu().numpy().astype(np.int64)
        from tests.gpu_util import canonical_perm
        perm, rank = canonical_perm(keys, None, 3)
        lat = O.build(pos, sigma)
        assert V == lat.V
        counts = np.bincount(lat.idx.reshape(-1), minlength=lat.V)
        assert counts.max() > 500 and (counts > 32).sum() >= 3 and (counts <= 32).sum() > 100
        ref, wref, scale = O.splat(lat, feat, normalize=normalize)
        gw = wt[:V].cpu().numpy().astype(np.float64)[perm]
        assert_close_scaled(gw, wref, wref, REL_F32, "split-list weight")
        if C == 0:
            continue
        got = vals[:V].float().cpu().numpy().astype(np.float64)[perm]
        tol = (2 if normalize else 1) * REL_F32 * scale
        if values_dtype == "bf16":
            tol = tol + BF16_ULP * np.abs(ref)
        assert_close_scaled(got, ref, tol, 1.0, f"split-list splat C={C} rep={rep}")


def test_splat_normalized_parity():
    w = random_cloud(4000, 3, seed=7, extent=1.0, C=6)
    L = _lattice(3, 0.12, w.m)
    g = GpuLattice(L, w.pos, w.feat, normalize=True)
    lat = O.build(w.pos, 0.12)
    ref, wref, scale = O.splat(lat, w.feat, normalize=True)
    # one more rounding (the division) on top of the sum
    assert_close_scaled(g.values(), ref, scale, 2 * REL_F32, "normalised splat")
    assert_close_scaled(g.weight(), wref, wref, REL_F32, "weight")


def test_splat_batched_parity():
    w = random_cloud(6000, 3, seed=8, extent=1.0, C=8, n_batch=5)
    L = _lattice(3, 0.15, w.m)
    g = GpuLattice(L, w.pos, w.feat, batch=w.batch)
    lat = O.build(w.pos, 0.15, batch=w.batch)
    check_lattice(g, lat)
    ref, _, scale = O.splat(lat, w.feat)
    assert_close_scaled(g.values(), ref, scale, REL_F32, "batched splat")
    nbr = g.neighbors()
    assert np.array_equal(nbr, O.neighbors(lat))


def test_splat_alpha_one():
    w = random_cloud(3000, 3, seed=9, extent=1.0, C=4)
    L = _lattice(3, 0.1, w.m, alpha=1.0)
    g = GpuLattice(L, w.pos, w.feat)
    lat = O.build(w.pos, 0.1, alpha=1.0)
    check_lattice(g, lat)


def test_splat_anisotropic_sigma():
    w = random_cloud(3000, 3, seed=10, extent=1.0, C=2)
    sig = [0.05, 0.2, 0.11]
    L = _lattice(3, sig, w.m)
    g = GpuLattice(L, w.pos, w.feat)
    lat = O.build(w.pos, np.array(sig, dtype=np.float32))
    check_lattice(g, lat)


def test_splat_order_independent():
    """Hash insertion order changes with point order; the canonical lattice does not."""
    w = random_cloud(5000, 3, seed=11, extent=1.0, C=4)
    perm = np.random.default_rng(0).permutation(w.m)
    L = _lattice(3, 0.1, w.m)
    a = GpuLattice(L, w.pos, w.feat)
    va, ia = a.values(), a.idx.copy()
    b = GpuLattice(L, w.pos[perm], w.feat[perm])
    assert np.array_equal(a.keys, b.keys)
    assert np.array_equal(ia[perm], b.idx)
    lat = O.build(w.pos, 0.1)
    _, _, scale = O.splat(lat, w.feat)
    assert_close_scaled(b.values(), va, scale, 2 * REL_F32, "reordered splat")


# ---------------------------------------------------------------------------
# neighbours (Sec. "Permutohedral Lattice": +-[-1,..,d,..,-1])
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d", [1, 2, 3, 4])
def test_neighbors_parity(d):
    w = random_cloud(4000, d, seed=200 + d, extent=1.0, C=1)
    L = _lattice(d, 0.2, w.m)
    g = GpuLattice(L, w.pos, w.feat)
    lat = O.build(w.pos, 0.2)
    assert np.array_equal(g.neighbors(), O.neighbors(lat))


# ---------------------------------------------------------------------------
# conv (Sec. "Common Operations": Convolving over the 1-hop ring)
# ---------------------------------------------------------------------------

CONV_CASES = [
    # d, sigma, m, C_in, C_out, dtype, bias
    (3, 0.05, 4096, 8, 16, "f32", False),     # any-shape MFMA kernel (tiny config shape)
    (3, 0.1, 6000, 64, 64, "f32", False),     # fp32 MFMA, BN = 64
    (3, 0.1, 6000, 32, 128, "f32", True),     # fp32 MFMA, one chunk per tap, BN = 128
    (3, 0.1, 6000, 64, 64, "bf16", False),    # bf16 MFMA, BN = 64
    (3, 0.1, 6000, 64, 128, "bf16", True),    # bf16 MFMA, BN = 128
    (3, 0.1, 5000, 128, 128, "bf16", False),  # two chunks per tap
    (3, 0.1, 5000, 64, 192, "bf16", False),   # three N tiles of 64
    (4, 0.3, 5000, 64, 64, "bf16", False),    # T = 11
    (3, 0.1, 3000, 96, 64, "bf16", False),    # C_in not a multiple of 64: any-shape MFMA kernel
    (2, 0.05, 3000, 5, 7, "f32", True),       # odd channels, d = 2
    (3, 0.1, 3000, 96, 48, "f32", True),      # any-shape, 64 x 64 tiles, C_out tail of 16
    (4, 0.3, 3000, 16, 40, "bf16", True),     # any-shape, T = 11, K = 176 (three chunks, tail)
    (1, 0.05, 2000, 3, 1, "f32", False),      # any-shape, d = 1 (T = 5), one output channel
    (3, 0.1, 3000, 200, 24, "bf16", False),   # any-shape, K = 1800 over 29 chunks, 128 x 32 tiles
    (3, 0.5, 300, 64, 64, "bf16", False),     # V below one tile
]


def _conv_case(d, sigma, m, C_in, C_out, dtype, bias, seed=0):
    w = random_cloud(m, d, seed=300 + seed, extent=1.0, C=1)
    L = _lattice(d, sigma, m)
    g = GpuLattice(L, w.pos, w.feat)
    lat = O.build(w.pos, sigma)
    nbr = O.neighbors(lat)
    x = random_rows(lat.V, C_in, seed=400 + seed)
    W = conv_weight(C_in, C_out, d, seed=500 + seed)
    b = random_rows(1, C_out, seed=600 + seed)[0] if bias else None
    wd = to_dev(W)
    if dtype == "bf16":
        wd = L.weights_to_bf16(wd)
    out = L.conv(g.to_gpu_order(x), wd, dtype=dtype, bias=None if b is None else to_dev(b))
    got = g.from_gpu_order(out)
    return L, g, lat, nbr, x, W, b, got


@pytest.mark.parametrize("case", CONV_CASES, ids=[f"d{c[0]}-{c[3]}x{c[4]}-{c[5]}{'-bias' if c[6] else ''}"
                                                  for c in CONV_CASES])
def test_conv_parity(case):
    d, sigma, m, C_in, C_out, dtype, bias = case
    L, g, lat, nbr, x, W, b, got = _conv_case(*case)
    ref, scale = O.conv(x, nbr, W, b)
    if dtype == "f32":
        assert_close_scaled(got, ref, scale, REL_F32, "f32 conv")
    else:
        assert_close_scaled(got, ref, scale, REL_BF16, "bf16 conv vs fp32 oracle")
        xr = O.round_bf16(x).astype(np.float64)
        Wr = O.round_bf16(W).astype(np.float64)
        ref_b, scale_b = O.conv(xr, nbr, Wr, b)
        assert_close_scaled(got, ref_b, scale_b, REL_F32, "bf16 conv vs bf16-input oracle")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_conv_unaligned_operands(dtype):
    """Rows, weights and output one element past a 16-byte boundary: a
    shape the tiled kernels serve when aligned runs on the any-shape MFMA
    kernel, with the same result."""
    d, sigma, m, C_in, C_out = 3, 0.1, 5000, 64, 64
    w = random_cloud(m, d, seed=950, extent=1.0, C=1)
    L = _lattice(d, sigma, m)
    g = GpuLattice(L, w.pos, w.feat)
    lat = O.build(w.pos, sigma)
    nbr = O.neighbors(lat)
    x = random_rows(lat.V, C_in, seed=951)
    W = conv_weight(C_in, C_out, d, seed=952)
    b = random_rows(1, C_out, seed=953)[0]

    def shifted(t):
        buf = torch.empty(t.numel() + 1, dtype=t.dtype, device=t.device)
        v = buf[1:].view(t.shape)
        v.copy_(t)
        assert v.data_ptr() % 16 != 0
        return v

    wd = to_dev(W)
    if dtype == "bf16":
        wd = L.weights_to_bf16(wd)
    xd = g.to_gpu_order(x)
    ref_aligned = L.conv(xd, wd, dtype=dtype, bias=to_dev(b))
    out = shifted(torch.zeros_like(ref_aligned))
    got = L.conv(shifted(xd), shifted(wd), dtype=dtype, bias=to_dev(b), out=out)
    ref, scale = O.conv(x, nbr, W, b)
    if dtype == "f32":
        assert_close_scaled(g.from_gpu_order(got), ref, scale, REL_F32, "unaligned f32 conv")
    else:
        xr = O.round_bf16(x).astype(np.float64)
        Wr = O.round_bf16(W).astype(np.float64)
        ref_b, scale_b = O.conv(xr, nbr, Wr, b)
        assert_close_scaled(g.from_gpu_order(got), ref_b, scale_b, REL_F32, "unaligned bf16 conv")
    # and the aligned launch (another kernel) agrees within the same bound
    assert_close_scaled(g.from_gpu_order(got), g.from_gpu_order(ref_aligned).astype(np.float64), scale, REL_F32,
                        "unaligned vs aligned")


BF16_ULP = 2.0 ** -8   # bound on the relative error of one round-to-nearest to bf16


@pytest.mark.parametrize("case", [(3, 0.1, 6000, 64, 64), (3, 0.1, 5000, 128, 128), (4, 0.3, 5000, 64, 64),
                                  (3, 0.1, 3000, 96, 32)])
def test_conv_bf16_storage(case):
    """bf16-stored input and output: the input is the bf16 value itself, the
    output is the fp32 result rounded once to bf16."""
    d, sigma, m, C_in, C_out = case
    w = random_cloud(m, d, seed=900, extent=1.0, C=1)
    L = _lattice(d, sigma, m)
    g = GpuLattice(L, w.pos, w.feat)
    lat = O.build(w.pos, sigma)
    nbr = O.neighbors(lat)
    x = O.round_bf16(random_rows(lat.V, C_in, seed=901))
    W = conv_weight(C_in, C_out, d, seed=902)
    xin = g.to_gpu_order(x).to(torch.bfloat16)
    wd = L.weights_to_bf16(to_dev(W))
    ref, scale = O.conv(x, nbr, O.round_bf16(W))
    out32 = L.conv(xin, wd, dtype="bf16")
    assert_close_scaled(g.from_gpu_order(out32), ref, scale, REL_F32, "bf16-in conv")
    out16 = L.conv(xin, wd, dtype="bf16", out_dtype="bf16")
    assert out16.dtype == torch.bfloat16
    got = g.from_gpu_order(out16.float())
    assert_close_scaled(got, ref, REL_F32 * scale + BF16_ULP * np.abs(ref), 1.0, "bf16-out conv")
    # fp32 compute with bf16 output
    xf = g.to_gpu_order(x)
    out16f = L.conv(xf, to_dev(W), dtype="f32", out_dtype="bf16")
    reff, scalef = O.conv(x, nbr, W)
    assert_close_scaled(g.from_gpu_order(out16f.float()), reff, REL_F32 * scalef + BF16_ULP * np.abs(reff), 1.0,
                        "f32 conv, bf16 out")


def test_splat_bf16_storage_and_slice_of_bf16():
    w = random_cloud(6000, 3, seed=910, extent=1.0, C=64)
    L = _lattice(3, 0.1, w.m)
    vals, _ = L.splat(to_dev(w.pos), to_dev(w.feat), values_dtype="bf16")
    assert vals.dtype == torch.bfloat16
    V = L.num_vertices()
    keys = L.keys().cpu().numpy().astype(np.int64)
    from tests.gpu_util import canonical_perm
    perm, rank = canonical_perm(keys, None, 3)
    lat = O.build(w.pos, 0.1)
    ref, _, scale = O.splat(lat, w.feat)
    got = vals[:V].float().cpu().numpy().astype(np.float64)[perm]
    assert_close_scaled(got, ref, REL_F32 * scale + BF16_ULP * np.abs(ref), 1.0, "bf16 splat")
    # slice of bf16-stored vertex values
    y = O.round_bf16(random_rows(lat.V, 64, seed=911))
    yin = to_dev(np.ascontiguousarray(y[rank])).to(torch.bfloat16)
    out = L.slice(yin).cpu().numpy()
    sref, sscale = O.slice_(lat, y)
    assert_close_scaled(out, sref, sscale, REL_F32, "slice of bf16 values")


def test_conv_weights_to_bf16_matches_oracle_rounding():
    L = _lattice(3, 0.1, 10)
    W = conv_weight(64, 128, 3, seed=1)
    got = L.weights_to_bf16(to_dev(W)).float().cpu().numpy()
    assert np.array_equal(got.view(np.uint32), O.round_bf16(W).view(np.uint32))


# ---------------------------------------------------------------------------
# slice (Eq. slice)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d,C", [(3, 1), (3, 3), (3, 16), (3, 64), (3, 128), (4, 64), (2, 12)])
def test_slice_parity(d, C):
    w = random_cloud(5000, d, seed=700 + d, extent=1.0, C=1)
    L = _lattice(d, 0.15, w.m)
    g = GpuLattice(L, w.pos, w.feat)
    lat = O.build(w.pos, 0.15)
    y = random_rows(lat.V, C, seed=800 + C)
    got = L.slice(g.to_gpu_order(y)).cpu().numpy()
    ref, scale = O.slice_(lat, y)
    assert_close_scaled(got, ref, scale, REL_F32, "slice")


# ---------------------------------------------------------------------------
# DeformSlice and the fused classifier (Eq. deformSlice; Sec. "Implementation")
# ---------------------------------------------------------------------------

def _deform_case(d, C, n_cls, values_bf16, seed, m=5000, sigma=0.15):
    w = random_cloud(m, d, seed=1200 + seed, extent=1.0, C=1)
    L = _lattice(d, sigma, w.m)
    g = GpuLattice(L, w.pos, w.feat)
    lat = O.build(w.pos, sigma)
    y = random_rows(lat.V, C, seed=1300 + seed)
    if values_bf16:
        y = O.round_bf16(y).astype(np.float32)
    yd = g.to_gpu_order(y)
    if values_bf16:
        yd = yd.to(torch.bfloat16)
    dw = deform_weights(C, max(n_cls, 1), seed=1400 + seed)
    return L, g, lat, y, yd, dw


def _check_deform(got, delta, lat, y, dw, with_cls, what):
    res = O.deform_slice(lat.idx, lat.bary, y, dw.w_delta, dw.b_delta,
                         dw.w_cls if with_cls else None, dw.b_cls if with_cls else None, with_delta_scale=True)
    ref, dref, scale, dscale = res
    r = assert_close_scaled(got, ref, scale, REL_F32, what)
    # tanh in fp32 adds a few ulps of its value on top of the argument's rounding
    assert_close_scaled(delta, dref, dscale, REL_F32, what + " offsets", atol=4e-7)
    return r


@pytest.mark.parametrize("d,C,n_cls,bf16", [
    (3, 64, 0, False), (3, 64, 50, False), (3, 128, 20, True), (2, 16, 3, False), (4, 64, 26, False),
    (4, 128, 0, True), (3, 3, 20, False), (3, 77, 7, False), (2, 520, 20, False), (3, 1024, 1, True),
    (3, 200, 0, False), (1, 5, 0, False), (3, 256, 64, False)])
def test_deform_slice_parity(d, C, n_cls, bf16):
    """Every kernel shape: float4 rows with one or four chunks per lane,
    scalar rows (C not a multiple of 4) with one or four, bf16 rows, classes
    fewer or more than the lanes per point, and no classifier."""
    L, g, lat, y, yd, dw = _deform_case(d, C, n_cls, bf16, seed=d * 1000 + C + n_cls)
    with_cls = n_cls > 0
    wd = to_dev(dw.w_delta)
    wc = to_dev(dw.w_cls) if with_cls else None
    bc = to_dev(dw.b_cls) if with_cls else None
    out, delta = L.deform_slice(yd, wd, dw.b_delta, wc, bc, want_delta=True)
    assert out.shape == (L.m, n_cls if with_cls else C)
    r = _check_deform(out.cpu().numpy(), delta.cpu().numpy(), lat, y, dw, with_cls,
                      f"deform d={d} C={C} n_cls={n_cls} bf16={bf16}")
    print(f" max rel {r:.2e}", flush=True)


def test_deform_slice_without_offsets_is_slice():
    """Zero offset weights and bias give tanh(0) = 0: the result is the
    plain slice, bit for bit (same products in the same order)."""
    L, g, lat, y, yd, dw = _deform_case(3, 64, 0, False, seed=5)
    z = torch.zeros(64, device=dev())
    out, delta = L.deform_slice(yd, z, 0.0, want_delta=True)
    assert torch.equal(out, L.slice(yd))
    assert torch.count_nonzero(delta).item() == 0


def test_deform_slice_saturated_offsets():
    """A large bias saturates tanh at 1: f = sum_k (b_k + 1) x_k."""
    L, g, lat, y, yd, dw = _deform_case(3, 32, 0, False, seed=6)
    out, delta = L.deform_slice(yd, torch.zeros(32, device=dev()), 40.0, want_delta=True)
    assert torch.all(delta == 1.0)
    ref, _, scale = O.deform_slice(lat.idx, lat.bary, y, np.zeros(32), 40.0)
    assert_close_scaled(out.cpu().numpy(), ref, scale, REL_F32, "saturated deform")


def test_deform_slice_classifier_is_linear_in_features():
    """Fused classifier == the unfused features times W_cls^T plus b_cls
    (computed here in float64 from the kernel's own features)."""
    L, g, lat, y, yd, dw = _deform_case(3, 64, 20, False, seed=7)
    wd = to_dev(dw.w_delta)
    f = L.deform_slice(yd, wd, dw.b_delta).cpu().numpy().astype(np.float64)
    logits = L.deform_slice(yd, wd, dw.b_delta, to_dev(dw.w_cls), to_dev(dw.b_cls)).cpu().numpy()
    ref = f @ dw.w_cls.astype(np.float64).T + dw.b_cls
    scale = np.abs(f) @ np.abs(dw.w_cls.astype(np.float64)).T + np.abs(dw.b_cls)
    assert_close_scaled(logits, ref, scale, REL_F32, "classifier")
    nob = L.deform_slice(yd, wd, dw.b_delta, to_dev(dw.w_cls)).cpu().numpy()
    assert_close_scaled(nob, ref - dw.b_cls, scale, REL_F32, "classifier without bias")


def test_deform_slice_errors_and_empty():
    from paper_2108_03917_amd import LatticeError
    from paper_2108_03917_amd.lattice import E_ARG, E_STATE

    L = _lattice(3, 0.1, 100)
    x = torch.zeros((4, 8), device=dev())
    wd = torch.zeros(8, device=dev())
    with pytest.raises(LatticeError) as ei:
        L.deform_slice(x, wd, 0.0)
    assert ei.value.status == E_STATE
    w = random_cloud(100, 3, seed=8, extent=1.0, C=1)
    L.splat(to_dev(w.pos), to_dev(w.feat))
    V = L.num_vertices()
    lib, h = L._lib, L._h
    out = torch.zeros((100, 300), device=dev())
    vals = torch.zeros((V, 300), device=dev())
    wdd = torch.zeros(300, device=dev())
    wc = torch.zeros((300, 300), device=dev())
    P = lambda t: t.data_ptr()  # noqa: E731
    F32 = 0
    cases = [
        (P(vals), F32, 0, P(wdd), None, None, 0),             # C = 0
        (P(vals), F32, 8, P(wdd), P(wc), None, 0),            # classifier with no classes
        (P(vals), F32, 8, P(wdd), P(wc), None, 257),          # too many classes
        (P(vals), F32, 8, P(wdd), None, P(wc), 0),            # class bias without weights
        (None, F32, 8, P(wdd), None, None, 0),                # no values
        (P(vals), F32, 8, None, None, None, 0),               # no offset weights
        (P(vals), 7, 8, P(wdd), None, None, 0),               # bad storage type
        (P(vals), F32, 1028, P(wdd), None, None, 0),          # above the float4 limit
        (P(vals) + 4, F32, 300, P(wdd), None, None, 0),       # misaligned rows beyond the scalar limit
        (P(vals), F32, 258, P(wdd), None, None, 0),           # not a multiple of 4 beyond the scalar limit
    ]
    for v, dt, C, wdp, wcp, bcp, n in cases:
        st = lib.lattice_deform_slice(h, v, dt, C, wdp, 0.0, wcp, bcp, n, P(out), None)
        assert st == E_ARG, (C, n, st)
    torch.cuda.synchronize()
    # an empty cloud launches nothing and succeeds
    L0 = _lattice(3, 0.1, 16)
    L0.splat(torch.zeros((0, 3), device=dev()), torch.zeros((0, 8), device=dev()))
    o, dl = L0.deform_slice(torch.zeros((1, 8), device=dev()), torch.zeros(8, device=dev()), 0.0, want_delta=True)
    assert o.shape == (0, 8) and dl.shape == (0, 4)


def test_splat_then_slice_constant_is_constant():
    """Normalised splat then slice of a constant field returns the constant."""
    w = random_cloud(5000, 3, seed=12, extent=1.0, C=1)
    L = _lattice(3, 0.1, w.m)
    const = np.full((w.m, 4), 2.5, dtype=np.float32)
    vals, _ = L.splat(to_dev(w.pos), to_dev(const), normalize=True)
    out = L.slice(vals).cpu().numpy()
    assert np.allclose(out, 2.5, rtol=4e-6, atol=0)


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------

def test_empty_cloud():
    L = _lattice(3, 0.1, 16)
    pos = torch.zeros((0, 3), device=dev())
    feat = torch.zeros((0, 8), device=dev())
    vals, _ = L.splat(pos, feat)
    assert L.num_vertices() == 0
    W = L.weights_to_bf16(to_dev(conv_weight(64, 64, 3, seed=0)))
    x = torch.zeros((1, 64), device=dev())
    L.conv(x, W, dtype="bf16")
    out = L.slice(torch.zeros((1, 8), device=dev()))
    assert out.shape == (0, 8)
    assert L.neighbors().shape[0] == 0


def test_single_point_and_duplicates():
    pos = np.array([[0.123, -0.456, 0.789]] * 37, dtype=np.float32)
    feat = random_rows(37, 3, seed=5)
    L = _lattice(3, 0.1, 37)
    g = GpuLattice(L, pos, feat)
    lat = O.build(pos, 0.1)
    assert g.V == 4
    check_lattice(g, lat)
    ref, wref, scale = O.splat(lat, feat)
    assert_close_scaled(g.values(), ref, scale, REL_F32, "duplicate splat")
    assert_close_scaled(g.weight(), wref, wref, REL_F32, "duplicate weight")


@pytest.mark.parametrize("explicit_capacity", [False, True])
def test_sparse_cloud_near_worst_load(explicit_capacity):
    """A cloud so sparse that nearly every (point, vertex) pair creates its
    own vertex: V is close to (d+1) m, the most a table must hold.  The
    default capacity keeps the load at or below 2/3; a table of exactly
    (d+1) m slots runs at a load near 1, where most lookups (the absent ring
    neighbours) probe long chains.  Both give the oracle's keys, simplices
    and neighbour table."""
    d, m, sigma = 3, 4096, 0.0005
    rng = np.random.default_rng(77)
    pos = rng.uniform(0.0, 1.0, (m, d)).astype(np.float32)
    feat = rng.standard_normal((m, 2)).astype(np.float32)
    keys_max = (d + 1) * m
    L = _lattice(d, sigma, m, hash_capacity=keys_max if explicit_capacity else 0)
    if explicit_capacity:
        assert L.hash_capacity == keys_max
    else:
        assert L.hash_capacity >= 1.5 * keys_max
    g = GpuLattice(L, pos, feat)
    lat = O.build(pos, sigma)
    assert lat.V >= 0.99 * keys_max, lat.V
    check_lattice(g, lat)
    assert np.array_equal(g.neighbors(), O.neighbors(lat))


def test_capacity_error_is_reported():
    from paper_2108_03917_amd import LatticeError
    from paper_2108_03917_amd.lattice import E_CAPACITY

    w = random_cloud(4000, 3, seed=13, extent=1.0, C=2)
    L = _lattice(3, 0.05, w.m, hash_capacity=64)
    L.splat(to_dev(w.pos), to_dev(w.feat))
    with pytest.raises(LatticeError) as ei:
        L.num_vertices()
    assert ei.value.status == E_CAPACITY
    # the lattice recovers on the next splat that fits
    small = np.array([[0.0, 0.0, 0.0], [0.01, 0.0, 0.0]], dtype=np.float32)
    L.splat(to_dev(small), to_dev(np.ones((2, 2), dtype=np.float32)))
    assert L.num_vertices() >= 4


def test_resplat_sequence():
    """Clouds of different sizes, an empty cloud and a splat that overflows
    the hash table, one after the other on one lattice: every splat that fits
    matches the oracle (keys, simplices, values, neighbours), whatever the
    splats before it left in the lattice's buffers.  The table is emptied
    slot by slot after a splat of n vertices with 8n < capacity; otherwise,
    and after a failed splat, it is emptied whole.  The sequence takes both
    ways, on a small table and on a large one."""
    from paper_2108_03917_amd import LatticeError
    from paper_2108_03917_amd.lattice import E_CAPACITY

    ways = set()

    def run(L, clouds):
        cap = L.hash_capacity
        prev = None  # vertices of the splat before, None after a failed one
        for i, w in enumerate(clouds):
            if i > 0:
                ways.add("slots" if prev is not None and 8 * prev < cap else "whole")
            if w is None:
                L.splat(torch.zeros((0, 3), device=dev()), torch.zeros((0, 4), device=dev()))
                assert L.num_vertices() == 0, i
                continue  # an empty splat leaves the list of occupied slots as it was
            if w == "overflow":   # 5000 points spread thinly: more than 16384 vertices
                big = random_cloud(5000, 3, seed=34, extent=40.0, C=4)
                L.splat(to_dev(big.pos), to_dev(big.feat))
                with pytest.raises(LatticeError) as ei:
                    L.num_vertices()
                assert ei.value.status == E_CAPACITY
                prev = None
                continue
            g = GpuLattice(L, w.pos, w.feat)
            lat = O.build(w.pos, 0.1)
            check_lattice(g, lat)
            ref, wref, scale = O.splat(lat, w.feat)
            assert_close_scaled(g.values(), ref, scale, REL_F32, f"splat {i}")
            assert np.array_equal(g.neighbors(), O.neighbors(lat)), i
            prev = lat.V

    clouds = [random_cloud(5000, 3, seed=30, extent=1.0, C=4), random_cloud(1200, 3, seed=31, extent=0.5, C=4),
              None, random_cloud(3000, 3, seed=32, extent=2.0, C=4), "overflow",
              random_cloud(5000, 3, seed=30, extent=1.0, C=4), random_cloud(700, 3, seed=33, extent=1.0, C=4)]
    run(_lattice(3, 0.1, 5000, hash_capacity=16384), clouds)
    run(_lattice(3, 0.1, 5000, hash_capacity=1 << 19), [c for c in clouds if not isinstance(c, str)])
    assert ways == {"slots", "whole"}, ways


def test_range_error_is_reported():
    from paper_2108_03917_amd import LatticeError
    from paper_2108_03917_amd.lattice import E_RANGE

    pos = np.array([[0.0, 0.0, 0.0], [5000.0, 0.0, 0.0]], dtype=np.float32)
    L = _lattice(3, 0.01, 2)
    L.splat(to_dev(pos), to_dev(np.ones((2, 1), dtype=np.float32)))
    with pytest.raises(LatticeError) as ei:
        L.num_vertices()
    assert ei.value.status == E_RANGE
    pos2 = np.array([[0.0, 0.0, 0.0], [np.nan, 0.0, 0.0]], dtype=np.float32)
    L.splat(to_dev(pos2), to_dev(np.ones((2, 1), dtype=np.float32)))
    assert L.status() == E_RANGE


def test_batch_id_range_error():
    from paper_2108_03917_amd.lattice import E_RANGE

    pos = np.zeros((2, 3), dtype=np.float32)
    L = _lattice(3, 0.1, 2)
    L.splat(to_dev(pos), to_dev(np.ones((2, 1), dtype=np.float32)),
            batch=to_dev(np.array([0, 70000], dtype=np.int32)))
    assert L.status() == E_RANGE


def test_state_and_argument_errors():
    from paper_2108_03917_amd import LatticeError
    from paper_2108_03917_amd.lattice import E_ARG, E_STATE

    L = _lattice(3, 0.1, 10)
    x = torch.zeros((4, 64), device=dev())
    W = torch.zeros((64, 9, 64), device=dev())
    with pytest.raises(LatticeError) as ei:
        L.conv(x, W)
    assert ei.value.status == E_STATE
    with pytest.raises(LatticeError) as ei:
        L.slice(x)
    assert ei.value.status == E_STATE
    with pytest.raises(LatticeError) as ei:
        L.splat(torch.zeros((11, 3), device=dev()), torch.zeros((11, 2), device=dev()))
    assert ei.value.status == E_ARG
    L4 = _lattice(4, 0.1, 10)
    with pytest.raises(LatticeError) as ei:
        L4.splat(torch.zeros((2, 4), device=dev()), torch.zeros((2, 1), device=dev()),
                 batch=torch.zeros(2, dtype=torch.int32, device=dev()))
    assert ei.value.status == E_ARG


def test_stage_timing_records_every_stage():
    w = random_cloud(3000, 3, seed=14, extent=1.0, C=64)
    L = _lattice(3, 0.1, w.m)
    L.set_timing(1)
    vals, _ = L.splat(to_dev(w.pos), to_dev(w.feat))
    Wb = L.weights_to_bf16(to_dev(conv_weight(64, 64, 3, seed=2)))
    y = L.conv(vals, Wb, dtype="bf16")
    L.slice(y)
    L.deform_slice(y, torch.zeros(64, device=dev()), 0.0)
    t = L.timing()
    assert all(t[s][1] == 1 and t[s][0] > 0 for s in ("splat", "neighbors", "conv", "slice", "deform")), t
    L.set_timing(2)
    assert all(v == (0.0, 0) for v in L.timing().values())
    # the slice and the deform slice are timed at their kernel's start and
    # end; an empty cloud launches no kernel and records nothing
    L.splat(torch.zeros((0, 3), device=dev()), None)
    L.slice(torch.zeros((1, 64), device=dev()))
    L.deform_slice(torch.zeros((1, 64), device=dev()), torch.zeros(64, device=dev()), 0.0)
    t = L.timing()
    assert t["slice"] == (0.0, 0) and t["deform"] == (0.0, 0), t


# ---------------------------------------------------------------------------
# every conv kernel family on a lattice large enough for several tiles per
# workgroup (the pipelined kernels prefetch across tiles) and a ragged tail
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def big_lattices():
    out = {}
    for d, sigma in [(3, 0.05), (4, 0.12)]:
        w = random_cloud(40000, d, seed=970 + d, extent=1.0, C=1)
        L = _lattice(d, sigma, w.m)
        g = GpuLattice(L, w.pos, w.feat)
        lat = O.build(w.pos, sigma)
        out[d] = (L, g, lat, O.neighbors(lat))
    return out


@pytest.mark.parametrize("d,C_in,C_out", [(3, 64, 64), (3, 64, 128), (3, 128, 128), (4, 64, 128), (4, 64, 64),
                                          (3, 128, 64)])
def test_conv_every_path_bf16(big_lattices, d, C_in, C_out):
    L, g, lat, nbr = big_lattices[d]
    assert lat.V > 256 * 64 * 2  # more tiles than two per workgroup for every tiling
    x = O.round_bf16(random_rows(lat.V, C_in, seed=971))
    W = conv_weight(C_in, C_out, d, seed=972)
    b = random_rows(1, C_out, seed=973)[0]
    ref, scale = O.conv(x.astype(np.float64), nbr, O.round_bf16(W).astype(np.float64), b)
    xin = g.to_gpu_order(x).to(torch.bfloat16)
    wd = L.weights_to_bf16(to_dev(W))
    try:
        for path in ("tiled", "ws", "rs"):
            L.set_conv_path(path)
            for out_dtype in ("f32", "bf16"):
                out = L.conv(xin, wd, dtype="bf16", bias=to_dev(b), out_dtype=out_dtype)
                got = g.from_gpu_order(out.float())
                tol = REL_F32 * scale + (BF16_ULP * np.abs(ref) if out_dtype == "bf16" else 0.0)
                assert_close_scaled(got, ref, tol, 1.0, f"{path} conv {C_in}x{C_out} d={d} out {out_dtype}")
    finally:
        L.set_conv_path("auto")


@pytest.mark.parametrize("d,C_in,C_out", [(3, 64, 64), (4, 64, 64), (3, 32, 128)])
def test_conv_every_path_f32(big_lattices, d, C_in, C_out):
    """fp32 rows and weights on every kernel family (the register-resident
    ring kernel covers 64 -> 64 with 9 taps, the others fall back)."""
    L, g, lat, nbr = big_lattices[d]
    x = random_rows(lat.V, C_in, seed=981)
    W = conv_weight(C_in, C_out, d, seed=982)
    b = random_rows(1, C_out, seed=983)[0]
    ref, scale = O.conv(x.astype(np.float64), nbr, W.astype(np.float64), b)
    xin = g.to_gpu_order(x)
    try:
        for path in ("tiled", "ws", "rs"):
            L.set_conv_path(path)
            for out_dtype in ("f32", "bf16"):
                out = L.conv(xin, to_dev(W), dtype="f32", bias=to_dev(b), out_dtype=out_dtype)
                got = g.from_gpu_order(out.float())
                tol = REL_F32 * scale + (BF16_ULP * np.abs(ref) if out_dtype == "bf16" else 0.0)
                assert_close_scaled(got, ref, tol, 1.0, f"{path} f32 conv {C_in}x{C_out} d={d} out {out_dtype}")
    finally:
        L.set_conv_path("auto")


@pytest.mark.parametrize("d,ordered,batched", [(3, True, False), (4, True, False), (3, False, False),
                                               (3, True, True)])
def test_splat_large_cloud_insert_paths(d, ordered, batched):
    """Clouds of at least 256 points per CU take the insert kernel that
    merges each workgroup's keys in LDS first; spatially ordered points (a
    sweep) share most vertices within a workgroup, shuffled ones almost none.
    The point count leaves a ragged last workgroup."""
    m = 70001
    rng = np.random.default_rng(990 + d)
    pos = rng.uniform(-1, 1, size=(m, d)).astype(np.float32)
    if ordered:
        pos = pos[np.lexsort(pos.T[::-1])]  # sorted along the first axis: neighbours in index order
    batch = rng.integers(0, 7, size=m).astype(np.int32) if batched else None
    if batched and ordered:
        batch = np.sort(batch)
    feat = rng.standard_normal((m, 8)).astype(np.float32)
    sigma = 0.08 if d == 3 else 0.25
    L = _lattice(d, sigma, m)
    g = GpuLattice(L, pos, feat, batch=batch)
    lat = O.build(pos, sigma, batch=batch)
    check_lattice(g, lat)
    ref, wref, scale = O.splat(lat, feat)
    assert_close_scaled(g.values(), ref, scale, REL_F32, "large-cloud splat")
    assert_close_scaled(g.weight(), wref, wref, REL_F32, "large-cloud weight")
