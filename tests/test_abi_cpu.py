"""CPU-side checks of the C ABI: the library loads, exports every function
that include/lattice.h declares, and rejects bad arguments before touching a
device (so these run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2108_03917_amd import lattice as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lattice.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lattice_[a-z0-9_]+)\s*\(", text)) - {"lattice_status", "lattice_dtype"})


def test_header_declares_the_hot_path():
    names = _declared()
    for n in ("lattice_create", "lattice_splat", "lattice_conv", "lattice_slice", "lattice_deform_slice",
              "lattice_destroy"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(B.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(B.EXPORTS) == _declared()


def test_binding_loads():
    lib = B.load_library()
    assert lib.lattice_status_string(0).decode() == "ok"
    assert lib.lattice_status_string(B.E_CAPACITY).decode() == "hash table full"


def test_create_rejects_bad_arguments_without_device():
    lib = B.load_library()
    out = ctypes.c_void_p()
    sig = (ctypes.c_float * 4)(0.1, 0.1, 0.1, 0.1)
    bad_sig = (ctypes.c_float * 3)(0.1, -1.0, 0.1)
    nan_sig = (ctypes.c_float * 3)(0.1, float("nan"), 0.1)
    cases = [
        (0, sig, 0.0, 10, 0),        # d below 1
        (5, sig, 0.0, 10, 0),        # d above 4
        (3, None, 0.0, 10, 0),       # no sigma
        (3, bad_sig, 0.0, 10, 0),    # sigma <= 0
        (3, nan_sig, 0.0, 10, 0),    # sigma NaN
        (3, sig, 0.0, 0, 0),         # no points
        (3, sig, 0.0, (1 << 28) + 1, 0),  # above 2^28 points (a pair-list entry holds the point in 28 bits)
        (3, sig, 0.0, 10, -1),       # negative capacity
        (3, sig, float("inf"), 10, 0),
    ]
    for d, s, a, mp, cap in cases:
        st = lib.lattice_create(d, s, a, mp, cap, None, ctypes.byref(out))
        assert st == B.E_ARG, (d, a, mp, cap, st)
        assert not out.value
    assert lib.lattice_create(3, sig, 0.0, 10, 0, None, None) == B.E_ARG


def test_null_lattice_is_rejected():
    lib = B.load_library()
    assert lib.lattice_max_vertices(None, 10) == -1
    assert lib.lattice_hash_capacity(None) == -1
    assert lib.lattice_dim(None) == -1
    assert lib.lattice_splat(None, None, None, 0, None, 0, 0, None, 0, None) == B.E_ARG
    assert lib.lattice_conv(None, None, 0, 1, None, 1, 0, None, None, 0) == B.E_ARG
    assert lib.lattice_slice(None, None, 0, 1, None) == B.E_ARG
    assert lib.lattice_deform_slice(None, None, 0, 1, None, 0.0, None, None, 0, None, None) == B.E_ARG
    assert lib.lattice_get_status(None) == B.E_ARG
    V = ctypes.c_int64()
    assert lib.lattice_num_vertices(None, ctypes.byref(V)) == B.E_ARG
    lib.lattice_destroy(None)


def test_no_device_fails_loudly():
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("a device is present")
    lib = B.load_library()
    out = ctypes.c_void_p()
    sig = (ctypes.c_float * 3)(0.1, 0.1, 0.1)
    st = lib.lattice_create(3, sig, 0.0, 10, 0, None, ctypes.byref(out))
    assert st in (B.E_HIP, B.E_NOMEM)
    assert not out.value


def test_resample_binding_passes_source_then_destination(monkeypatch):
    """lattice_downsample(fine, coarse, ...) and lattice_upsample(coarse, fine,
    ...) both take the source lattice first: the binding must pass the
    handles in that order (a swapped upsample indexes rows the input does not
    have)."""
    import torch

    calls = []

    class Stub:
        def lattice_downsample(self, *a):
            calls.append(("down", a[0], a[1]))
            return 0

        def lattice_upsample(self, *a):
            calls.append(("up", a[0], a[1]))
            return 0

    monkeypatch.setattr(B, "_dev", lambda t, dtype, name: t)

    def fake(handle, V):
        L = object.__new__(B.Lattice)
        L._lib, L._h, L.taps, L._V, L.m, L.d = Stub(), handle, 9, V, 10, 3
        return L

    fine, coarse = fake("FINE", 100), fake("COARSE", 40)
    w = torch.zeros((4, 9, 4))
    y = fine.downsample(coarse, torch.zeros((100, 4)), w)
    z = coarse.upsample(fine, torch.zeros((40, 4)), w)
    assert calls == [("down", "FINE", "COARSE"), ("up", "COARSE", "FINE")]
    assert y.shape == (40, 4) and z.shape == (100, 4)


def test_distribute_binding_passes_the_output_storage(monkeypatch):
    """lattice_distribute_pointnet takes the output's storage type right after
    the output pointer: the binding derives it from the out tensor."""
    import torch

    calls = []

    class Stub:
        def lattice_distribute_pointnet(self, *a):
            calls.append(a)
            return 0

    monkeypatch.setattr(B, "_dev", lambda t, dtype, name: t)
    monkeypatch.setattr(B, "_ptr", lambda t: None if t is None else id(t))
    L = object.__new__(B.Lattice)
    L._lib, L._h, L.taps, L._V, L.m, L.d = Stub(), "H", 9, 50, 10, 3
    k0 = 3   # d + f_d: per block a, s, W, b
    params = torch.zeros(2 * k0 + 16 * k0 + 16 + 2 * 16 + 32 * 16 + 32 + 2 * 32 + 64 * 32 + 64)
    for dt, code in ((torch.float32, B.F32), (torch.bfloat16, B.BF16)):
        out = torch.zeros((50, 64), dtype=dt)
        L.distribute_pointnet(torch.zeros((10, 3)), None, params, out=out)
        a = calls[-1]
        assert a[0] == "H" and a[3] == 0 and a[5] == 3
        assert a[7] is None                               # no groups: the caller's affines
        assert a[9] == id(out) and a[10] == code and a[11] is None
    out = L.distribute_pointnet(torch.zeros((10, 3)), None, params, out_dtype="bf16")
    assert out.dtype == torch.bfloat16 and calls[-1][10] == B.BF16
    # group normalisation: three group counts ("default": min(32, K) per block) and eps
    L.distribute_pointnet(torch.zeros((10, 3)), None, params, groups="default", eps=1e-3)
    a = calls[-1]
    assert list(a[7]) == [3, 16, 32] and abs(a[8].value - 1e-3) < 1e-9
    L.distribute_pointnet(torch.zeros((10, 3)), None, params, groups=[1, 4, 8])
    assert list(calls[-1][7]) == [1, 4, 8]
