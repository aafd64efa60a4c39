"""GPU parity on the five full-size synthetic workloads, and the end-to-end
chain of the benchmark's workload in the benchmark's launch configuration.

Per workload: the lattice (keys, per-point vertices, weights, neighbours) is
compared bit-exactly; splat values within 1e-5 of the sum of |terms|; each of
the workload's convolutions is fed the oracle's splat values and compared on
every vertex; slice is fed the oracle's conv output and compared on every
point; DeformSlice with the fused classifier (the workload's class count) is
fed seeded rows of the last conv's width and compared on every point.  Each
bf16 conv also runs on bf16-stored rows (the benchmark's kernels).  The
benchmark's whole chain runs on every workload.
"""
import numpy as np
import pytest
import torch

from datagen.clouds import N_CLASSES, deform_weights, make_workload, random_rows
from oracle import lattice_oracle as O
from tests.gpu_util import REL_BF16, REL_F32, GpuLattice, assert_close_scaled, check_lattice, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("config", [1, 2, 3, 4, 5])
def test_full_config_parity(config):
    from paper_2108_03917_amd import Lattice

    w = make_workload(config)
    print(f"\nconfig {config}: {w.name} m={w.m} d={w.d} C={w.C}", flush=True)
    L = Lattice(w.d, w.sigma, max_points=w.m)
    g = GpuLattice(L, w.pos, w.feat, batch=w.batch)
    lat = O.build(w.pos, w.sigma, batch=w.batch)
    check_lattice(g, lat)
    vals, wref, scale = O.splat(lat, w.feat)
    r = assert_close_scaled(g.values(), vals, scale, REL_F32, "splat")
    print(f"  V={lat.V} splat max rel {r:.2e}", flush=True)
    nbr = O.neighbors(lat)
    assert np.array_equal(g.neighbors(), nbr)
    x32 = vals.astype(np.float32)
    xin = g.to_gpu_order(x32)
    for cv in w.convs:
        wd = to_dev(cv.weight)
        if cv.dtype == "bf16":
            wd = L.weights_to_bf16(wd)
        out = L.conv(xin, wd, dtype=cv.dtype)
        got = g.from_gpu_order(out)
        if cv.dtype == "f32":
            ref, cscale = O.conv(x32, nbr, cv.weight)
            r = assert_close_scaled(got, ref, cscale, REL_F32, f"conv {cv.c_in}->{cv.c_out} f32")
        else:
            ref, cscale = O.conv(x32, nbr, cv.weight)
            r = assert_close_scaled(got, ref, cscale, REL_BF16, f"conv {cv.c_in}->{cv.c_out} bf16")
            refb, cscaleb = O.conv(O.round_bf16(x32), nbr, O.round_bf16(cv.weight))
            assert_close_scaled(got, refb, cscaleb, REL_F32, f"conv {cv.c_in}->{cv.c_out} bf16-input")
            # the rows stored as bf16, as the benchmark stores them: the
            # register-resident (or ring) kernels it runs there
            xb = xin.to(torch.bfloat16)
            for out_dtype in ("f32", "bf16"):
                outb = L.conv(xb, wd, dtype="bf16", out_dtype=out_dtype)
                gotb = g.from_gpu_order(outb.float())
                extra = 2.0 ** -8 * np.abs(refb) if out_dtype == "bf16" else 0.0
                assert_close_scaled(gotb, refb, REL_F32 * cscaleb + extra, 1.0,
                                    f"conv {cv.c_in}->{cv.c_out} bf16 rows, {out_dtype} out")
        print(f"  conv {cv.c_in}->{cv.c_out} {cv.dtype} max rel {r:.2e}", flush=True)
        y32 = ref.astype(np.float32)
        sl = L.slice(g.to_gpu_order(y32)).cpu().numpy()
        sref, sscale = O.slice_(lat, y32)
        r = assert_close_scaled(sl, sref, sscale, REL_F32, "slice")
        print(f"  slice C={cv.c_out} max rel {r:.2e}", flush=True)
    L.close()


@pytest.mark.parametrize("config", [1, 2, 3, 4, 5])
def test_full_config_deform_every_point(config):
    """DeformSlice with the fused classifier on every point of the workload."""
    from paper_2108_03917_amd import Lattice

    w = make_workload(config)
    L = Lattice(w.d, w.sigma, max_points=w.m)
    g = GpuLattice(L, w.pos, None, batch=w.batch)
    lat = O.build(w.pos, w.sigma, batch=w.batch)
    assert np.array_equal(g.keys, lat.keys)
    c_last = w.convs[-1].c_out
    dw = deform_weights(c_last, N_CLASSES[config], seed=100 + config)
    yv = random_rows(lat.V, c_last, seed=1500 + config)
    got = L.deform_slice(g.to_gpu_order(yv), to_dev(dw.w_delta), dw.b_delta, to_dev(dw.w_cls),
                         to_dev(dw.b_cls)).cpu().numpy()
    # the oracle in slices of points (each point is independent)
    for p0 in range(0, w.m, 100000):
        sl = slice(p0, min(w.m, p0 + 100000))
        ref, _, dscale = O.deform_slice(lat.idx[sl], lat.bary[sl], yv, dw.w_delta, dw.b_delta, dw.w_cls,
                                        dw.b_cls)
        r = assert_close_scaled(got[sl], ref, dscale, REL_F32, f"deform+classifier points {p0}..")
    print(f"\nconfig {config}: deform C={c_last} classes={N_CLASSES[config]} on all {w.m} points, "
          f"last slice max rel {r:.2e}", flush=True)
    L.close()


@pytest.mark.parametrize("config", [1, 2, 3, 4, 5])
def test_bench_workload_end_to_end(config):
    """splat -> every conv of the workload -> slice exactly as bench.py
    launches it (rows stored as bf16 where a bf16 conv reads them), against
    the oracle chain; the tolerance is 2e-2 (bf16) or 3e-5 (fp32 only) of the
    magnitude chain |B| |W|..|W| |B^T| |f|."""
    import bench

    w = make_workload(config)
    step = bench.Pipeline(w)
    res = step.run()
    step.stream.synchronize()   # the pipeline runs on its own stream
    out = res.cpu().numpy().astype(np.float64)
    lat = O.build(w.pos, w.sigma, batch=w.batch)
    x, _, scale = O.splat(lat, w.feat)
    nbr = O.neighbors(lat)
    any_bf16 = False
    for cv in step.convs:
        if cv.dtype == "bf16":
            any_bf16 = True
            x, _ = O.conv(O.round_bf16(x.astype(np.float32)), nbr, O.round_bf16(cv.weight))
            _, scale = O.conv(scale, nbr, np.abs(O.round_bf16(cv.weight).astype(np.float64)))
        else:
            x, _ = O.conv(x, nbr, cv.weight)
            _, scale = O.conv(scale, nbr, np.abs(cv.weight.astype(np.float64)))
    ref, _ = O.slice_(lat, x)
    _, rscale = O.slice_(lat, scale)
    rel = REL_BF16 if any_bf16 else 3 * REL_F32
    r = assert_close_scaled(out, ref, rscale, rel, "end-to-end")
    print(f"\nend-to-end {w.name}: max rel {r:.2e}", flush=True)
