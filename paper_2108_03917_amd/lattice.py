"""Thin ctypes binding of liblattice.so (include/lattice.h).

Argument marshalling only: tensors are passed to the library as raw device
pointers together with the current HIP stream, and output tensors are
allocated with torch.  Every step of splat, neighbours, conv and slice runs in
the library's HIP kernels.  When the library has not been built, importing
works but every call raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "_lib", "liblattice.so")

OK, E_ARG, E_STATE, E_RANGE, E_CAPACITY, E_NOMEM, E_HIP = range(7)
F32, BF16 = 0, 1
STAGES = ("splat", "neighbors", "conv", "slice", "deform", "slice_backward", "conv_backward", "splat_backward",
          "downsample", "upsample", "distribute", "downsample_backward", "upsample_backward", "deform_backward",
          "distribute_backward")

EXPORTS = (
    "lattice_create", "lattice_destroy", "lattice_max_vertices", "lattice_splat", "lattice_build_neighbors",
    "lattice_conv",
    "lattice_slice", "lattice_weights_to_bf16", "lattice_num_vertices", "lattice_get_status",
    "lattice_get_keys", "lattice_get_neighbors", "lattice_get_point_simplex", "lattice_set_timing",
    "lattice_get_timing", "lattice_hash_capacity", "lattice_dim", "lattice_status_string",
    "lattice_last_error", "lattice_set_conv_path", "lattice_deform_slice", "lattice_slice_backward",
    "lattice_splat_backward", "lattice_conv_backward", "lattice_downsample", "lattice_upsample",
    "lattice_distribute_pointnet", "lattice_conv_backward_noalloc", "lattice_downsample_backward",
    "lattice_upsample_backward", "lattice_deform_slice_backward", "lattice_distribute_pointnet_backward",
)

_lib = None


class LatticeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"[{status}] {message}")
        self.status = status


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load liblattice.so and declare its signatures; raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(python -m paper_2108_03917_amd._build)")
    lib = ctypes.CDLL(path)
    P, I64, I, D, St = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_double, ctypes.c_int
    sig = {
        "lattice_create": (St, [I, P, D, I64, I64, P, ctypes.POINTER(P)]),
        "lattice_destroy": (None, [P]),
        "lattice_max_vertices": (I64, [P, I64]),
        "lattice_splat": (St, [P, P, P, I64, P, I, I, P, I, P]),
        "lattice_build_neighbors": (St, [P]),
        "lattice_conv": (St, [P, P, I, I, P, I, I, P, P, I]),
        "lattice_slice": (St, [P, P, I, I, P]),
        "lattice_deform_slice": (St, [P, P, I, I, P, ctypes.c_float, P, P, I, P, P]),
        "lattice_deform_slice_backward": (St, [P, P, I, I, P, ctypes.c_float, P, I, P, P, I, P, P, P, P]),
        "lattice_slice_backward": (St, [P, P, I, P, I]),
        "lattice_splat_backward": (St, [P, P, I, I, I, P, P]),
        "lattice_conv_backward": (St, [P, P, I, I, P, I, I, P, I, P, I, P, P]),
        "lattice_conv_backward_noalloc": (St, [P, P, I, I, P, I, I, P, I, P, I, P, P]),
        "lattice_distribute_pointnet": (St, [P, P, P, I, P, I, P, P, ctypes.c_float, P, I, P]),
        "lattice_distribute_pointnet_backward": (St, [P, P, P, I, P, I, P, P, ctypes.c_float, P, P]),
        "lattice_downsample": (St, [P, P, P, I, I, P, I, I, P, P, I]),
        "lattice_upsample": (St, [P, P, P, I, I, P, I, I, P, P, I]),
        "lattice_downsample_backward": (St, [P, P, P, I, I, P, I, I, P, I, P, I, P, P]),
        "lattice_upsample_backward": (St, [P, P, P, I, I, P, I, I, P, I, P, I, P, P]),
        "lattice_weights_to_bf16": (St, [P, P, I64, P]),
        "lattice_num_vertices": (St, [P, ctypes.POINTER(I64)]),
        "lattice_get_status": (St, [P]),
        "lattice_get_keys": (St, [P, P, P]),
        "lattice_get_neighbors": (St, [P, P]),
        "lattice_get_point_simplex": (St, [P, P, P]),
        "lattice_set_timing": (St, [P, I]),
        "lattice_set_conv_path": (St, [P, I]),
        "lattice_get_timing": (St, [P, ctypes.POINTER(D), ctypes.POINTER(I64)]),
        "lattice_hash_capacity": (I64, [P]),
        "lattice_dim": (I, [P]),
        "lattice_status_string": (ctypes.c_char_p, [I]),
        "lattice_last_error": (ctypes.c_char_p, [P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


_STORAGE = {torch.float32: F32, torch.bfloat16: BF16}
_TORCH = {"f32": torch.float32, "bf16": torch.bfloat16}


def _dev(t: torch.Tensor, dtype, name: str) -> torch.Tensor:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    allowed = dtype if isinstance(dtype, tuple) else (dtype,)
    if t.dtype not in allowed:
        raise ValueError(f"{name} must be {' or '.join(map(str, allowed))}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


class Lattice:
    """A sparse permutohedral lattice on the current device and stream."""

    def __init__(self, d: int, sigma, alpha: float = 0.0, max_points: int = 1, hash_capacity: int = 0,
                 stream: Optional[torch.cuda.Stream] = None):
        self._lib = load_library()
        sig = torch.as_tensor(sigma, dtype=torch.float32).broadcast_to((d,)).contiguous()
        self.d = d
        self.taps = 2 * (d + 1) + 1
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        self.device = self.stream.device
        self._sigma = (ctypes.c_float * d)(*[float(s) for s in sig])
        h = ctypes.c_void_p()
        st = self._lib.lattice_create(d, self._sigma, float(alpha), int(max_points), int(hash_capacity),
                                      ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h))
        if st != OK:
            raise LatticeError(st, f"lattice_create: {self._lib.lattice_status_string(st).decode()}")
        self._h = h
        self.max_points = int(max_points)
        self.m = 0
        self._V = None   # V of the current lattice once read back, else None

    # -- lifetime ---------------------------------------------------------
    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.lattice_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, st: int, what: str):
        if st != OK:
            msg = self._lib.lattice_last_error(self._h)
            raise LatticeError(st, f"{what}: {self._lib.lattice_status_string(st).decode()}: "
                                   f"{msg.decode() if msg else ''}")

    # -- queries ----------------------------------------------------------
    def max_vertices(self, m: Optional[int] = None) -> int:
        return int(self._lib.lattice_max_vertices(self._h, self.m if m is None else int(m)))

    @property
    def hash_capacity(self) -> int:
        return int(self._lib.lattice_hash_capacity(self._h))

    def num_vertices(self) -> int:
        V = ctypes.c_int64()
        self._check(self._lib.lattice_num_vertices(self._h, ctypes.byref(V)), "num_vertices")
        self._V = int(V.value)
        return self._V

    def _rows_needed(self) -> int:
        """Rows a per-vertex buffer must have: V when it is known on the host,
        else the bound max_vertices(m)."""
        return self._V if self._V is not None else self.max_vertices(self.m)

    def status(self) -> int:
        return int(self._lib.lattice_get_status(self._h))

    # -- the hot path -----------------------------------------------------
    def splat(self, pos: torch.Tensor, feat: Optional[torch.Tensor] = None, batch: Optional[torch.Tensor] = None,
              normalize: bool = False, values: Optional[torch.Tensor] = None,
              weight: Optional[torch.Tensor] = None, want_weight: bool = True, values_dtype: str = "f32"):
        """Build the lattice of ``pos`` [m, d] and splat ``feat`` [m, C].

        Returns (values, weight): [max_vertices, C] and [max_vertices]
        tensors whose first V rows hold the result (V stays on the device).
        ``values_dtype`` "bf16" stores the fp32 sums rounded to bf16."""
        _dev(pos, torch.float32, "pos")
        m = pos.shape[0]
        if pos.dim() != 2 or pos.shape[1] != self.d:
            raise ValueError(f"pos must be [m, {self.d}]")
        C = 0
        if feat is not None:
            _dev(feat, torch.float32, "feat")
            if feat.dim() != 2 or feat.shape[0] != m:
                raise ValueError("feat must be [m, C]")
            C = feat.shape[1]
        if batch is not None:
            _dev(batch, torch.int32, "batch")
            if batch.shape != (m,):
                raise ValueError("batch must be [m]")
        mv = int(self._lib.lattice_max_vertices(self._h, m))
        if C > 0 and values is None:
            values = torch.empty((mv, C), dtype=_TORCH[values_dtype], device=pos.device)
        if want_weight and weight is None:
            weight = torch.empty((max(mv, 1),), dtype=torch.float32, device=pos.device)
        vdt = F32
        if values is not None:
            _dev(values, (torch.float32, torch.bfloat16), "values")
            vdt = _STORAGE[values.dtype]
            if values.numel() < mv * C:
                raise ValueError("values has fewer than max_vertices rows")
        if weight is not None:
            _dev(weight, torch.float32, "weight")
            if weight.numel() < mv:
                raise ValueError("weight has fewer than max_vertices rows")
        st = self._lib.lattice_splat(self._h, _ptr(pos), _ptr(batch), m, _ptr(feat), C, int(bool(normalize)),
                                     _ptr(values), vdt, _ptr(weight))
        self.m = m
        self._V = None
        self._check(st, "splat")
        return values, weight

    def build_neighbors(self):
        """Build the 1-ring neighbour table of the current lattice now."""
        self._check(self._lib.lattice_build_neighbors(self._h), "build_neighbors")

    def conv(self, x: torch.Tensor, w: torch.Tensor, dtype: str = "f32", bias: Optional[torch.Tensor] = None,
             out: Optional[torch.Tensor] = None, out_dtype: str = "f32") -> torch.Tensor:
        """1-ring convolution of vertex values ``x`` [>= V, C_in] (fp32 or bf16
        storage) with weights [C_out, T, C_in] (fp32 for dtype "f32", bf16 for
        "bf16"); the output is stored as ``out_dtype``."""
        _dev(x, (torch.float32, torch.bfloat16), "x")
        if dtype == "f32":
            _dev(w, torch.float32, "w")
            dt = F32
        elif dtype == "bf16":
            _dev(w, torch.bfloat16, "w")
            dt = BF16
        else:
            raise ValueError("dtype must be 'f32' or 'bf16'")
        C_out, T, C_in = w.shape
        if T != self.taps or x.dim() != 2 or x.shape[1] != C_in:
            raise ValueError(f"w must be [C_out, {self.taps}, C_in] with C_in = x.shape[1]")
        if bias is not None:
            _dev(bias, torch.float32, "bias")
            if bias.numel() != C_out:
                raise ValueError("bias must have C_out elements")
        if out is None:
            out = torch.empty((max(x.shape[0], 1), C_out), dtype=_TORCH[out_dtype], device=x.device)
        _dev(out, (torch.float32, torch.bfloat16), "out")
        need = self._rows_needed()
        if x.shape[0] < need or out.dim() != 2 or out.shape[1] != C_out or out.shape[0] < need:
            raise ValueError(f"x and out need >= {need} rows (out [rows, {C_out}])")
        self._check(self._lib.lattice_conv(self._h, _ptr(x), _STORAGE[x.dtype], C_in, _ptr(w), C_out, dt,
                                           _ptr(bias), _ptr(out), _STORAGE[out.dtype]), "conv")
        return out

    def slice(self, values: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Eq. (slice) onto the points of the last splat: [m, C] fp32
        (``values`` stored as fp32 or bf16)."""
        _dev(values, (torch.float32, torch.bfloat16), "values")
        C = values.shape[1]
        if values.dim() != 2 or values.shape[0] < self._rows_needed():
            raise ValueError(f"values needs >= {self._rows_needed()} rows")
        if out is None:
            out = torch.empty((self.m, C), dtype=torch.float32, device=values.device)
        _dev(out, torch.float32, "out")
        if out.numel() < self.m * C:
            raise ValueError("out needs [m, C]")
        self._check(self._lib.lattice_slice(self._h, _ptr(values), _STORAGE[values.dtype], C, _ptr(out)), "slice")
        return out

    def deform_slice(self, values: torch.Tensor, w_delta: torch.Tensor, b_delta: float,
                     w_cls: Optional[torch.Tensor] = None, b_cls: Optional[torch.Tensor] = None,
                     out: Optional[torch.Tensor] = None, delta: Optional[torch.Tensor] = None,
                     want_delta: bool = False):
        """DeformSlice (Eq. deformSlice) onto the points of the last splat,
        fused with the classifier ``f W_cls^T + b_cls`` when ``w_cls`` [n_cls, C]
        is given.  Returns ``out`` ([m, n_cls] logits or [m, C] features, fp32)
        and, with ``want_delta`` or a ``delta`` tensor, the offsets [m, d+1]."""
        _dev(values, (torch.float32, torch.bfloat16), "values")
        if values.dim() != 2 or values.shape[0] < self._rows_needed():
            raise ValueError(f"values needs >= {self._rows_needed()} rows")
        C = values.shape[1]
        _dev(w_delta, torch.float32, "w_delta")
        if w_delta.numel() != C:
            raise ValueError("w_delta needs C entries")
        n_cls = 0
        if w_cls is not None:
            _dev(w_cls, torch.float32, "w_cls")
            if w_cls.dim() != 2 or w_cls.shape[1] != C:
                raise ValueError("w_cls needs [n_cls, C]")
            n_cls = w_cls.shape[0]
            if b_cls is not None:
                _dev(b_cls, torch.float32, "b_cls")
                if b_cls.numel() != n_cls:
                    raise ValueError("b_cls needs n_cls entries")
        elif b_cls is not None:
            raise ValueError("b_cls without w_cls")
        width = n_cls if w_cls is not None else C
        if out is None:
            out = torch.empty((self.m, width), dtype=torch.float32, device=values.device)
        _dev(out, torch.float32, "out")
        if out.numel() < self.m * width:
            raise ValueError(f"out needs [m, {width}]")
        if delta is None and want_delta:
            delta = torch.empty((self.m, self.d + 1), dtype=torch.float32, device=values.device)
        if delta is not None:
            _dev(delta, torch.float32, "delta")
            if delta.numel() < self.m * (self.d + 1):
                raise ValueError("delta needs [m, d+1]")
        self._check(self._lib.lattice_deform_slice(self._h, _ptr(values), _STORAGE[values.dtype], C, _ptr(w_delta),
                                                   float(b_delta), _ptr(w_cls), _ptr(b_cls), n_cls, _ptr(out),
                                                   _ptr(delta)), "deform_slice")
        return (out, delta) if delta is not None else out

    # -- distribute + PointNet ---------------------------------------------
    POINTNET_WIDTHS = (16, 32, 64)

    @staticmethod
    def pack_pointnet(layers) -> torch.Tensor:
        """Pack [(a, s, W, b)] per block (array-likes) into the flat fp32
        layout lattice_distribute_pointnet takes (a, s, W row-major, b per
        block), on the CPU."""
        parts = []
        for a, s, W, b in layers:
            parts += [torch.as_tensor(x, dtype=torch.float32).reshape(-1) for x in (a, s, W, b)]
        return torch.cat(parts)

    def distribute_pointnet(self, pos: torch.Tensor, feat: Optional[torch.Tensor], params: torch.Tensor,
                            out: Optional[torch.Tensor] = None, mean: Optional[torch.Tensor] = None,
                            want_mean: bool = False, out_dtype: str = "f32", groups=None, eps: float = 1e-5):
        """Distribute + PointNet + per-vertex max over the last splat's pairs:
        ``pos`` [m, d] (the positions that were splatted), ``feat`` [m, f_d]
        or None, ``params`` the packed parameters (see pack_pointnet) on the
        device.  With ``groups`` (three group counts, or "default" for
        min(32, K) per block) each block's normalisation is a group
        normalisation computed per cloud and ``params`` holds (gamma, beta, W,
        b) per block; without, the normalisation is the fixed affine (a, s) of
        ``params``.  Returns out [rows, 64], stored as fp32 or bf16 (the dtype
        of ``out``, else ``out_dtype``), and the local means [rows, d] with
        want_mean or a ``mean`` tensor."""
        _dev(pos, torch.float32, "pos")
        if pos.dim() != 2 or pos.shape != (self.m, self.d):
            raise ValueError(f"pos must be the splatted [m = {self.m}, {self.d}] positions")
        f_d = 0
        if feat is not None:
            _dev(feat, torch.float32, "feat")
            if feat.dim() != 2 or feat.shape[0] != self.m:
                raise ValueError("feat must be [m, f_d]")
            f_d = feat.shape[1]
        _dev(params, torch.float32, "params")
        k0 = self.d + f_d
        n_par = 2 * k0 + 16 * k0 + 16 + 2 * 16 + 32 * 16 + 32 + 2 * 32 + 64 * 32 + 64
        if params.numel() != n_par:
            raise ValueError(f"params must hold {n_par} values for d + f_d = {k0}")
        need = self._rows_needed()
        if out is None:
            out = torch.empty((max(need, 1), 64), dtype=_TORCH[out_dtype], device=pos.device)
        _dev(out, (torch.float32, torch.bfloat16), "out")
        if out.dim() != 2 or out.shape[1] != 64 or out.shape[0] < need:
            raise ValueError(f"out needs [>= {need}, 64]")
        if mean is None and want_mean:
            mean = torch.empty((max(need, 1), self.d), dtype=torch.float32, device=pos.device)
        if mean is not None:
            _dev(mean, torch.float32, "mean")
            if mean.numel() < need * self.d:
                raise ValueError(f"mean needs [>= {need}, {self.d}]")
        widths = (ctypes.c_int * 3)(*self.POINTNET_WIDTHS)
        gr = None
        if groups is not None:
            if isinstance(groups, str) and groups == "default":
                groups = [min(32, k) for k in (k0, 16, 32)]
            if len(groups) != 3:
                raise ValueError("groups must hold one group count per block (3)")
            gr = (ctypes.c_int * 3)(*[int(g) for g in groups])
        self._check(self._lib.lattice_distribute_pointnet(self._h, _ptr(pos), _ptr(feat), f_d, _ptr(params), 3,
                                                          widths, gr, ctypes.c_float(eps), _ptr(out),
                                                          _STORAGE[out.dtype], _ptr(mean)),
                    "distribute_pointnet")
        return (out, mean) if mean is not None else out

    def distribute_pointnet_backward(self, pos: torch.Tensor, feat: Optional[torch.Tensor], params: torch.Tensor,
                                     grad_out: torch.Tensor, groups=None, eps: float = 1e-5,
                                     grad_params: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Gradients of ``distribute_pointnet(pos, feat, params, groups=groups,
        eps=eps)`` with respect to ``params`` given ``grad_out`` = dL/dx
        [>= V, 64] fp32: a tensor in the layout of ``params``."""
        _dev(pos, torch.float32, "pos")
        if pos.dim() != 2 or pos.shape != (self.m, self.d):
            raise ValueError(f"pos must be the splatted [m = {self.m}, {self.d}] positions")
        f_d = 0
        if feat is not None:
            _dev(feat, torch.float32, "feat")
            if feat.dim() != 2 or feat.shape[0] != self.m:
                raise ValueError("feat must be [m, f_d]")
            f_d = feat.shape[1]
        _dev(params, torch.float32, "params")
        k0 = self.d + f_d
        n_par = 2 * k0 + 16 * k0 + 16 + 2 * 16 + 32 * 16 + 32 + 2 * 32 + 64 * 32 + 64
        if params.numel() != n_par:
            raise ValueError(f"params must hold {n_par} values for d + f_d = {k0}")
        _dev(grad_out, torch.float32, "grad_out")
        need = self._rows_needed()
        if grad_out.dim() != 2 or grad_out.shape[1] != 64 or grad_out.shape[0] < need:
            raise ValueError(f"grad_out needs [>= {need}, 64]")
        if grad_params is None:
            grad_params = torch.empty_like(params)
        _dev(grad_params, torch.float32, "grad_params")
        if grad_params.numel() != n_par:
            raise ValueError("grad_params needs the layout of params")
        widths = (ctypes.c_int * 3)(*self.POINTNET_WIDTHS)
        gr = None
        if groups is not None:
            if isinstance(groups, str) and groups == "default":
                groups = [min(32, k) for k in (k0, 16, 32)]
            if len(groups) != 3:
                raise ValueError("groups must hold one group count per block (3)")
            gr = (ctypes.c_int * 3)(*[int(g) for g in groups])
        self._check(self._lib.lattice_distribute_pointnet_backward(
            self._h, _ptr(pos), _ptr(feat), f_d, _ptr(params), 3, widths, gr, ctypes.c_float(eps), _ptr(grad_out),
            _ptr(grad_params)), "distribute_pointnet_backward")
        return grad_params

    # -- downsampling / upsampling ----------------------------------------
    def _resample(self, fn, src: "Lattice", dst: "Lattice", x, w, dtype, bias, out, out_dtype, what):
        _dev(x, (torch.float32, torch.bfloat16), "x")
        if dtype == "f32":
            _dev(w, torch.float32, "w")
            dt = F32
        elif dtype == "bf16":
            _dev(w, torch.bfloat16, "w")
            dt = BF16
        else:
            raise ValueError("dtype must be 'f32' or 'bf16'")
        C_out, T, C_in = w.shape
        if T != self.taps or x.dim() != 2 or x.shape[1] != C_in or x.shape[0] < src._rows_needed():
            raise ValueError(f"w must be [C_out, {self.taps}, C_in] and x [>= {src._rows_needed()}, C_in]")
        if bias is not None:
            _dev(bias, torch.float32, "bias")
            if bias.numel() != C_out:
                raise ValueError("bias must have C_out entries")
        need = dst._rows_needed()
        if out is None:
            out = torch.empty((max(need, 1), C_out), dtype=_TORCH[out_dtype], device=x.device)
        _dev(out, (torch.float32, torch.bfloat16), "out")
        if out.dim() != 2 or out.shape[1] != C_out or out.shape[0] < need:
            raise ValueError(f"out needs [>= {need}, {C_out}]")
        # both entry points take (source lattice, destination lattice)
        st = fn(src._h, dst._h, _ptr(x), _STORAGE[x.dtype], C_in, _ptr(w), C_out, dt, _ptr(bias), _ptr(out),
                _STORAGE[out.dtype])
        if st != OK:
            msg = self._lib.lattice_last_error(dst._h)
            raise LatticeError(st, f"{what}: {self._lib.lattice_status_string(st).decode()}: "
                                   f"{msg.decode() if msg else ''}")
        return out

    def downsample(self, coarse: "Lattice", x: torch.Tensor, w: torch.Tensor, dtype: str = "f32",
                   bias: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                   out_dtype: str = "f32") -> torch.Tensor:
        """Strided convolution of this (fine) lattice's values ``x`` onto the
        vertices of ``coarse`` (the same cloud at twice the scale)."""
        return self._resample(self._lib.lattice_downsample, self, coarse, x, w, dtype, bias, out, out_dtype,
                              "downsample")

    def upsample(self, fine: "Lattice", x: torch.Tensor, w: torch.Tensor, dtype: str = "f32",
                 bias: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                 out_dtype: str = "f32") -> torch.Tensor:
        """Transposed convolution of this (coarse) lattice's values ``x`` onto
        the vertices of ``fine``."""
        return self._resample(self._lib.lattice_upsample, self, fine, x, w, dtype, bias, out, out_dtype,
                              "upsample")

    def _resample_backward(self, fn, src: "Lattice", dst: "Lattice", grad_out, w, x, dtype, want_input,
                           want_weight, want_bias, grad_in_dtype, what):
        _dev(grad_out, (torch.float32, torch.bfloat16), "grad_out")
        if dtype == "f32":
            _dev(w, torch.float32, "w")
            dt = F32
        elif dtype == "bf16":
            _dev(w, torch.bfloat16, "w")
            dt = BF16
        else:
            raise ValueError("dtype must be 'f32' or 'bf16'")
        C_out, T, C_in = w.shape
        n_in, n_out = src._rows_needed(), dst._rows_needed()
        if T != self.taps or grad_out.dim() != 2 or grad_out.shape[1] != C_out or grad_out.shape[0] < n_out:
            raise ValueError(f"w must be [C_out, {self.taps}, C_in], grad_out [>= {n_out}, C_out]")
        if x is not None:
            _dev(x, (torch.float32, torch.bfloat16), "x")
            if x.dim() != 2 or x.shape[1] != C_in or x.shape[0] < n_in:
                raise ValueError(f"x must be [>= {n_in}, {C_in}]")
        if (want_weight or want_bias) and x is None:
            raise ValueError("the weight and bias gradients need the forward input x")
        dev_ = grad_out.device
        gi = torch.empty((max(n_in, 1), C_in), dtype=_TORCH[grad_in_dtype], device=dev_) if want_input else None
        gw = torch.empty((C_out, T, C_in), dtype=torch.float32, device=dev_) if want_weight else None
        gb = torch.empty((C_out,), dtype=torch.float32, device=dev_) if want_bias else None
        # both entry points take (source lattice, destination lattice) of the forward call
        st = fn(src._h, dst._h, _ptr(grad_out), _STORAGE[grad_out.dtype], C_out, _ptr(w), C_in, dt, _ptr(x),
                _STORAGE[x.dtype] if x is not None else F32, _ptr(gi), _STORAGE[gi.dtype] if gi is not None else F32,
                _ptr(gw), _ptr(gb))
        if st != OK:
            msg = self._lib.lattice_last_error(dst._h)
            raise LatticeError(st, f"{what}: {self._lib.lattice_status_string(st).decode()}: "
                                   f"{msg.decode() if msg else ''}")
        return gi, gw, gb

    def downsample_backward(self, coarse: "Lattice", grad_out: torch.Tensor, w: torch.Tensor,
                            x: Optional[torch.Tensor] = None, dtype: str = "f32", want_input: bool = True,
                            want_weight: bool = True, want_bias: bool = False, grad_in_dtype: str = "f32"):
        """Gradients of ``self.downsample(coarse, x, w)`` given ``grad_out`` on
        the coarse vertices: (grad_in [rows of this lattice, C_in] or None,
        grad_w [C_out, T, C_in] or None, grad_bias [C_out] or None)."""
        return self._resample_backward(self._lib.lattice_downsample_backward, self, coarse, grad_out, w, x, dtype,
                                       want_input, want_weight, want_bias, grad_in_dtype, "downsample_backward")

    def upsample_backward(self, fine: "Lattice", grad_out: torch.Tensor, w: torch.Tensor,
                          x: Optional[torch.Tensor] = None, dtype: str = "f32", want_input: bool = True,
                          want_weight: bool = True, want_bias: bool = False, grad_in_dtype: str = "f32"):
        """Gradients of ``self.upsample(fine, x, w)`` given ``grad_out`` on the
        fine vertices."""
        return self._resample_backward(self._lib.lattice_upsample_backward, self, fine, grad_out, w, x, dtype,
                                       want_input, want_weight, want_bias, grad_in_dtype, "upsample_backward")

    # -- backward passes ------------------------------------------------
    def slice_backward(self, grad_out: torch.Tensor, out: Optional[torch.Tensor] = None,
                       out_dtype: str = "f32") -> torch.Tensor:
        """Gradient of the slice with respect to the vertex values:
        Eq. (splat) of ``grad_out`` [m, C] over the last splat's pairs.
        Returns [max_vertices, C] (rows 0..V-1 hold the result)."""
        _dev(grad_out, torch.float32, "grad_out")
        if grad_out.dim() != 2 or grad_out.shape[0] != self.m:
            raise ValueError(f"grad_out must be [m = {self.m}, C]")
        C = grad_out.shape[1]
        mv = self.max_vertices(self.m)
        if out is None:
            out = torch.empty((max(mv, 1), C), dtype=_TORCH[out_dtype], device=grad_out.device)
        _dev(out, (torch.float32, torch.bfloat16), "out")
        if out.dim() != 2 or out.shape[1] != C or out.shape[0] < self._rows_needed():
            raise ValueError(f"out needs >= {self._rows_needed()} rows of {C}")
        self._check(self._lib.lattice_slice_backward(self._h, _ptr(grad_out), C, _ptr(out), _STORAGE[out.dtype]),
                    "slice_backward")
        return out

    def splat_backward(self, grad_values: torch.Tensor, normalize: bool = False,
                       weight: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Gradient of the splat with respect to the point features: Eq.
        (slice) of ``grad_values`` [>= V, C] (divided by the splat's weight
        w_v first when ``normalize``).  Returns [m, C] fp32."""
        _dev(grad_values, (torch.float32, torch.bfloat16), "grad_values")
        if grad_values.dim() != 2 or grad_values.shape[0] < self._rows_needed():
            raise ValueError(f"grad_values needs >= {self._rows_needed()} rows")
        C = grad_values.shape[1]
        if normalize:
            if weight is None:
                raise ValueError("the normalised splat's gradient needs its weight w_v")
            _dev(weight, torch.float32, "weight")
            if weight.numel() < self._rows_needed():
                raise ValueError("weight needs >= V entries")
        if out is None:
            out = torch.empty((self.m, C), dtype=torch.float32, device=grad_values.device)
        _dev(out, torch.float32, "out")
        if out.numel() < self.m * C:
            raise ValueError("out needs [m, C]")
        self._check(self._lib.lattice_splat_backward(self._h, _ptr(grad_values), _STORAGE[grad_values.dtype], C,
                                                     int(bool(normalize)), _ptr(weight if normalize else None),
                                                     _ptr(out)), "splat_backward")
        return out

    def conv_backward(self, grad_out: torch.Tensor, w: torch.Tensor, x: Optional[torch.Tensor] = None,
                      dtype: str = "f32", want_input: bool = True, want_weight: bool = True,
                      want_bias: bool = False, grad_in_dtype: str = "f32",
                      grad_in: Optional[torch.Tensor] = None, grad_w: Optional[torch.Tensor] = None,
                      grad_bias: Optional[torch.Tensor] = None, noalloc: bool = False):
        """Gradients of ``conv(x, w)`` given ``grad_out`` [>= V, C_out]:
        returns (grad_in [rows, C_in] or None, grad_w [C_out, T, C_in] fp32
        or None, grad_bias [C_out] fp32 or None).  Preallocated outputs may
        be passed in (then the matching want_* flag is implied).  With
        ``noalloc`` the library's allocation-free entry point runs (its
        scratch in a fixed per-GPU workspace; pass preallocated outputs to
        allocate nothing on this side either)."""
        _dev(grad_out, (torch.float32, torch.bfloat16), "grad_out")
        if dtype == "f32":
            _dev(w, torch.float32, "w")
            dt = F32
        elif dtype == "bf16":
            _dev(w, torch.bfloat16, "w")
            dt = BF16
        else:
            raise ValueError("dtype must be 'f32' or 'bf16'")
        C_out, T, C_in = w.shape
        need = self._rows_needed()
        if T != self.taps or grad_out.dim() != 2 or grad_out.shape[1] != C_out or grad_out.shape[0] < need:
            raise ValueError(f"w must be [C_out, {self.taps}, C_in], grad_out [>= {need}, C_out]")
        if x is not None:
            _dev(x, (torch.float32, torch.bfloat16), "x")
            if x.dim() != 2 or x.shape[1] != C_in or x.shape[0] < need:
                raise ValueError(f"x must be [>= {need}, {C_in}]")
        want_input = want_input or grad_in is not None
        want_weight = want_weight or grad_w is not None
        want_bias = want_bias or grad_bias is not None
        if (want_weight or want_bias) and x is None:
            raise ValueError("the weight and bias gradients need the forward input x")
        gi = grad_in if grad_in is not None else (
            torch.empty((grad_out.shape[0], C_in), dtype=_TORCH[grad_in_dtype], device=grad_out.device)
            if want_input else None)
        gw = grad_w if grad_w is not None else (
            torch.empty((C_out, T, C_in), dtype=torch.float32, device=grad_out.device) if want_weight else None)
        gb = grad_bias if grad_bias is not None else (
            torch.empty((C_out,), dtype=torch.float32, device=grad_out.device) if want_bias else None)
        if gi is not None:
            _dev(gi, (torch.float32, torch.bfloat16), "grad_in")
            if gi.dim() != 2 or gi.shape[1] != C_in or gi.shape[0] < need:
                raise ValueError(f"grad_in needs [>= {need}, {C_in}]")
        if gw is not None:
            _dev(gw, torch.float32, "grad_w")
            if gw.numel() != C_out * T * C_in:
                raise ValueError("grad_w needs [C_out, T, C_in]")
        if gb is not None:
            _dev(gb, torch.float32, "grad_bias")
            if gb.numel() != C_out:
                raise ValueError("grad_bias needs C_out entries")
        fn = self._lib.lattice_conv_backward_noalloc if noalloc else self._lib.lattice_conv_backward
        self._check(fn(
            self._h, _ptr(grad_out), _STORAGE[grad_out.dtype], C_out, _ptr(w), C_in, dt, _ptr(x),
            _STORAGE[x.dtype] if x is not None else F32, _ptr(gi), _STORAGE[gi.dtype] if gi is not None else F32,
            _ptr(gw), _ptr(gb)), "conv_backward_noalloc" if noalloc else "conv_backward")
        return gi, gw, gb

    def deform_slice_backward(self, values: torch.Tensor, w_delta: torch.Tensor, b_delta: float,
                              grad_out: torch.Tensor, w_cls: Optional[torch.Tensor] = None,
                              want_values: bool = True, want_w_delta: bool = True, want_b_delta: bool = True,
                              want_cls: bool = True, grad_dtype: str = "f32"):
        """Gradients of ``deform_slice(values, w_delta, b_delta, w_cls, b_cls)``
        given ``grad_out`` (fp32 [m, n_cls] with ``w_cls``, else [m, C]).
        Returns (grad_values [rows, C], grad_w_delta [C], grad_b_delta [1],
        grad_w_cls [n_cls, C], grad_b_cls [n_cls]); unrequested ones (and the
        classifier's without ``w_cls``) are None."""
        _dev(values, (torch.float32, torch.bfloat16), "values")
        need = self._rows_needed()
        if values.dim() != 2 or values.shape[0] < need:
            raise ValueError(f"values needs >= {need} rows")
        C = values.shape[1]
        _dev(w_delta, torch.float32, "w_delta")
        if w_delta.numel() != C:
            raise ValueError("w_delta needs C entries")
        n_cls = 0
        if w_cls is not None:
            _dev(w_cls, torch.float32, "w_cls")
            if w_cls.dim() != 2 or w_cls.shape[1] != C:
                raise ValueError("w_cls needs [n_cls, C]")
            n_cls = w_cls.shape[0]
        width = n_cls if w_cls is not None else C
        _dev(grad_out, torch.float32, "grad_out")
        if grad_out.numel() < self.m * width:
            raise ValueError(f"grad_out needs [m, {width}]")
        dev_ = values.device
        gv = torch.empty((max(need, 1), C), dtype=_TORCH[grad_dtype], device=dev_) if want_values else None
        gw = torch.empty((C,), dtype=torch.float32, device=dev_) if want_w_delta else None
        gb = torch.empty((1,), dtype=torch.float32, device=dev_) if want_b_delta else None
        with_cls = want_cls and w_cls is not None
        gwc = torch.empty((n_cls, C), dtype=torch.float32, device=dev_) if with_cls else None
        gbc = torch.empty((n_cls,), dtype=torch.float32, device=dev_) if with_cls else None
        self._check(self._lib.lattice_deform_slice_backward(
            self._h, _ptr(values), _STORAGE[values.dtype], C, _ptr(w_delta), float(b_delta), _ptr(w_cls), n_cls,
            _ptr(grad_out), _ptr(gv), _STORAGE[gv.dtype] if gv is not None else F32, _ptr(gw), _ptr(gb), _ptr(gwc),
            _ptr(gbc)), "deform_slice_backward")
        return gv, gw, gb, gwc, gbc

    def weights_to_bf16(self, w: torch.Tensor) -> torch.Tensor:
        """Round fp32 weights to bf16 (nearest even) with the library's kernel."""
        _dev(w, torch.float32, "w")
        out = torch.empty(w.shape, dtype=torch.bfloat16, device=w.device)
        self._check(self._lib.lattice_weights_to_bf16(self._h, _ptr(w), w.numel(), _ptr(out)), "weights_to_bf16")
        return out

    # -- introspection ----------------------------------------------------
    def keys(self, with_batch: bool = False):
        V = self.num_vertices()
        keys = torch.empty((max(V, 1), self.d + 1), dtype=torch.int32, device=self.device)
        b = torch.empty((max(V, 1),), dtype=torch.int32, device=self.device) if with_batch else None
        self._check(self._lib.lattice_get_keys(self._h, _ptr(keys), _ptr(b)), "get_keys")
        return (keys[:V], b[:V]) if with_batch else keys[:V]

    def neighbors(self) -> torch.Tensor:
        V = self.num_vertices()
        nbr = torch.empty((max(V, 1), self.taps), dtype=torch.int32, device=self.device)
        self._check(self._lib.lattice_get_neighbors(self._h, _ptr(nbr)), "get_neighbors")
        return nbr[:V]

    def point_simplex(self):
        idx = torch.empty((max(self.m, 1), self.d + 1), dtype=torch.int32, device=self.device)
        bary = torch.empty((max(self.m, 1), self.d + 1), dtype=torch.float32, device=self.device)
        self._check(self._lib.lattice_get_point_simplex(self._h, _ptr(idx), _ptr(bary)), "get_point_simplex")
        return idx[:self.m], bary[:self.m]

    # -- stage timing -----------------------------------------------------
    CONV_PATHS = {"auto": 0, "tiled": 1, "ws": 2, "rs": 3}

    def set_conv_path(self, path: str):
        """Kernel family of later convs: "auto", "tiled", "ws" or "rs"."""
        self._check(self._lib.lattice_set_conv_path(self._h, self.CONV_PATHS[path]), "set_conv_path")

    def set_timing(self, mode: int):
        self._check(self._lib.lattice_set_timing(self._h, int(mode)), "set_timing")

    def timing(self):
        ms = (ctypes.c_double * len(STAGES))()
        cnt = (ctypes.c_int64 * len(STAGES))()
        self._check(self._lib.lattice_get_timing(self._h, ms, cnt), "get_timing")
        return {s: (float(ms[i]), int(cnt[i])) for i, s in enumerate(STAGES)}


def exported_symbols(path: str = LIB_PATH) -> Sequence[str]:
    """Names from EXPORTS that the built library resolves."""
    lib = ctypes.CDLL(path)
    return [n for n in EXPORTS if hasattr(lib, n)]
