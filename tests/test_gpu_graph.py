"""The benchmark's step captured as a HIP graph: every replay, interleaved
with eager steps and synchronisations, must match the oracle as the eager
step does (the graph holds kernels only, no memset nodes)."""
import numpy as np
import pytest
import torch

from datagen.clouds import make_workload
from oracle import lattice_oracle as O
from tests.gpu_util import REL_BF16, REL_F32, assert_close_scaled

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _oracle_chain(w, convs):
    lat = O.build(w.pos, w.sigma, batch=w.batch)
    x, _, scale = O.splat(lat, w.feat)
    nbr = O.neighbors(lat)
    any_bf16 = False
    for cv in convs:
        if cv.dtype == "bf16":
            any_bf16 = True
            Wr = O.round_bf16(cv.weight)
            x, _ = O.conv(O.round_bf16(x.astype(np.float32)), nbr, Wr)
            _, scale = O.conv(scale, nbr, np.abs(Wr.astype(np.float64)))
        else:
            x, _ = O.conv(x, nbr, cv.weight)
            _, scale = O.conv(scale, nbr, np.abs(cv.weight.astype(np.float64)))
    ref, _ = O.slice_(lat, x)
    _, rscale = O.slice_(lat, scale)
    return lat, ref, rscale, (REL_BF16 if any_bf16 else 3 * REL_F32)


@pytest.mark.parametrize("config", [1, 2])
def test_graph_replays_match_oracle(config):
    import bench

    w = make_workload(config)
    lat, ref, rscale, rel = _oracle_chain(w, w.convs)
    pipe = bench.Pipeline(w)
    res = pipe.run()
    pipe.stream.synchronize()   # the pipeline runs on its own stream
    out = res.clone()
    assert pipe.L.num_vertices() == lat.V
    assert_close_scaled(out.cpu().numpy(), ref, rscale, rel, "eager")
    pipe.capture()
    for i in range(3):
        got = pipe.replay()
        pipe.stream.synchronize()
        assert pipe.L.num_vertices() == lat.V
        assert_close_scaled(got.cpu().numpy(), ref, rscale, rel, f"replay {i}")
        # the program's own eager work between replays
        eager = pipe.run()
        pipe.stream.synchronize()
        assert_close_scaled(eager.cpu().numpy(), ref, rscale, rel, f"eager after replay {i}")
