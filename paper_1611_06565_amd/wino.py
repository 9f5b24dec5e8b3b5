"""ctypes binding of libwino (include/wino.h).

Argument marshalling only: every step of the forward runs in the library's
HIP kernels.  Device buffers are torch CUDA (HIP) tensors; calls are enqueued
on torch's current stream.  If the library is not built, every entry point
raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os
import re
from fractions import Fraction

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
HEADER = os.path.join(os.path.dirname(HERE), "include", "wino.h")

WINO_RELU = 1
WINO_NO_SPLIT = 2
WINO_LEAKY_RELU = 4
WINO_NO_FUSE = 8
_STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported (N, m, r)",
           -3: "workspace too small", -4: "device launch failed"}


class WinoError(RuntimeError):
    def __init__(self, status, what=""):
        self.status = int(status)
        super().__init__(f"{what}: {_STATUS.get(self.status, 'unknown')} ({self.status})")


class _Opts(ctypes.Structure):
    _fields_ = [("pad", ctypes.c_int32 * 3), ("points", ctypes.POINTER(ctypes.c_double)),
                ("n_points", ctypes.c_int32), ("flags", ctypes.c_uint32), ("slope", ctypes.c_float),
                ("tile", ctypes.c_int32 * 3)]


class _Desc(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int32), ("m", ctypes.c_int32), ("r", ctypes.c_int32),
                ("alpha", ctypes.c_int32), ("n_xi", ctypes.c_int32),
                ("C", ctypes.c_int32), ("K", ctypes.c_int32),
                ("C_pad", ctypes.c_int32), ("K_pad", ctypes.c_int32),
                ("batch", ctypes.c_int64),
                ("X", ctypes.c_int64 * 3), ("Y", ctypes.c_int64 * 3), ("tiles", ctypes.c_int64 * 3),
                ("T", ctypes.c_int64), ("T_pad", ctypes.c_int64),
                ("block_tiles", ctypes.c_int32), ("block_kernels", ctypes.c_int32),
                ("default_points", ctypes.c_int32), ("channel_group", ctypes.c_int32),
                ("filter_channel_group", ctypes.c_int32), ("gemm_parts", ctypes.c_int32),
                ("gemm_tail_blocks", ctypes.c_int64), ("fused", ctypes.c_int32),
                ("tile", ctypes.c_int32 * 3), ("alpha_axis", ctypes.c_int32 * 3)]


_LIB = None


def library_path():
    return os.path.join(HERE, "libwino.so")


def lib():
    """Load libwino.so (raises if it has not been built)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    P_i64 = ctypes.POINTER(i64)
    P_dbl = ctypes.POINTER(ctypes.c_double)
    sig = {
        "wino_plan": (i32, [i32, i32, i32, i32, i32, P_i64, ctypes.POINTER(_Opts), ctypes.POINTER(vp)]),
        "wino_destroy": (None, [vp]),
        "wino_plan_describe": (i32, [vp, ctypes.POINTER(_Desc)]),
        "wino_filter_bytes": (sz, [vp]),
        "wino_workspace_bytes": (sz, [vp]),
        "wino_forward_workspace_bytes": (sz, [vp]),
        "wino_output_dims": (i32, [vp, P_i64]),
        "wino_get_matrices": (i32, [vp, P_dbl, P_dbl, P_dbl]),
        "wino_transform_filter": (i32, [vp, vp, vp, vp]),
        "wino_transform_input": (i32, [vp, vp, vp, sz, vp]),
        "wino_gemm_inverse": (i32, [vp, vp, sz, vp, vp, vp]),
        "wino_forward": (i32, [vp, vp, vp, vp, vp, sz, vp]),
        "wino_gemm_inverse_ex": (i32, [vp, vp, sz, vp, vp, vp, vp]),
        "wino_forward_ex": (i32, [vp, vp, vp, vp, vp, vp, sz, vp]),
        "wino_forward_noalloc": (i32, [vp, vp, vp, vp, vp, vp]),
        "wino_maxpool3d": (i32, [P_i64, ctypes.POINTER(i32), vp, vp, vp]),
        "wino_forward_pool": (i32, [vp, vp, vp, vp, ctypes.POINTER(i32), vp, vp, sz, vp]),
        "wino_status_string": (ctypes.c_char_p, [i32]),
        "wino_points_error_growth": (i32, [i32, i32, i32, P_dbl, i32, P_dbl]),
        "wino_search_points": (i32, [i32, i32, i32, P_dbl, P_dbl]),
        "wino_plan_adjoint": (i32, [vp, ctypes.POINTER(vp)]),
        "wino_weight_gradient_workspace_bytes": (sz, [vp]),
        "wino_weight_gradient": (i32, [vp, vp, vp, vp, vp, sz, vp]),
        "wino_transform_filter_adjoint": (i32, [vp, vp, vp, vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = L
    return L


def describe_header_symbols(path=HEADER):
    """Names of the functions include/wino.h declares."""
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\s*\*?\s*(wino_\w+)\s*\(", text, flags=re.M)))


def _check(st, what):
    if st != 0:
        raise WinoError(st, what)


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev_ptr(t, what, dtype=None):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{what} must be a CUDA (HIP) tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{what} must be {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _point(p):
    if isinstance(p, (Fraction, str)):
        return float(Fraction(p))
    return float(p)


class Plan:
    """One planned layer: Plan(N, m, r, C, K, dims=[batch, X_1..X_N], pad, points, relu, split, leaky).

    relu=True sets WINO_RELU; leaky=s (a float) sets WINO_LEAKY_RELU with
    slope s (the activation f of eq. 2).  split=False sets WINO_NO_SPLIT: no
    product block is split over several work-groups, whatever the grid size.
    fuse=False sets WINO_NO_FUSE: an F(4^3) forward stays in two stages.
    tile=(m_0, .., m_{N-1}) sets per-axis output tiles (wino_opts.tile)."""

    def __init__(self, N, m, r, C, K, dims, pad=0, points=None, relu=False, split=True, leaky=None,
                 fuse=True, tile=None):
        L = lib()
        dims = [int(d) for d in dims]
        if len(dims) != N + 1:
            raise ValueError("dims must be [batch, X_1..X_N]")
        opts = _Opts()
        pads = [pad] * N if isinstance(pad, int) else list(pad)
        for i, p in enumerate(pads):
            opts.pad[i] = int(p)
        self._pts = None
        if points is not None:
            self._pts = (ctypes.c_double * len(points))(*[_point(p) for p in points])
            opts.points = ctypes.cast(self._pts, ctypes.POINTER(ctypes.c_double))
            opts.n_points = len(points)
        opts.flags = (WINO_RELU if relu else 0) | (0 if split else WINO_NO_SPLIT) | (0 if fuse else WINO_NO_FUSE)
        if leaky is not None:
            opts.flags |= WINO_LEAKY_RELU
            opts.slope = float(leaky)
        if tile is not None:
            if len(tile) != N:
                raise ValueError("one tile extent per axis")
            for i, t in enumerate(tile):
                opts.tile[i] = int(t)
        arr = (ctypes.c_int64 * len(dims))(*dims)
        h = ctypes.c_void_p()
        _check(L.wino_plan(N, m, r, C, K, arr, ctypes.byref(opts), ctypes.byref(h)), "wino_plan")
        self._adopt(L, h, relu)
        self.leaky = leaky

    def _adopt(self, L, h, relu):
        self._h = h
        self._L = L
        d = _Desc()
        _check(L.wino_plan_describe(h, ctypes.byref(d)), "wino_plan_describe")
        self.desc = {f: (list(getattr(d, f)) if f in ("X", "Y", "tiles", "tile", "alpha_axis") else getattr(d, f))
                     for f, _ in _Desc._fields_}
        N, C, K, r = d.N, d.C, d.K, d.r
        self.N, self.m, self.r, self.C, self.K = N, d.m, r, C, K
        self.relu = relu
        self.leaky = None
        out = (ctypes.c_int64 * (N + 2))()
        _check(L.wino_output_dims(h, out), "wino_output_dims")
        self.output_shape = tuple(int(v) for v in out)
        self.input_shape = (int(d.batch), C) + tuple(int(v) for v in list(d.X)[:N])
        self.weight_shape = (K, C) + (r,) * N

    def adjoint(self):
        """The plan of this layer's data gradient dx from dy (wino_plan_adjoint):
        C and K swapped, input extents Y, pads r - 1 - pad; run it with
        transform_filter_adjoint(w) of this layer's kernels and forward(dy, U)."""
        h = ctypes.c_void_p()
        _check(self._L.wino_plan_adjoint(self._h, ctypes.byref(h)), "wino_plan_adjoint")
        p = Plan.__new__(Plan)
        p._pts = None
        p._adopt(self._L, h, False)
        return p

    @property
    def weight_gradient_workspace_bytes(self):
        return int(self._L.wino_weight_gradient_workspace_bytes(self._h))

    def weight_gradient(self, x, dy, dw=None, workspace=None):
        """dw [K][C][r^N] of this layer from its input x and output gradient dy."""
        import torch
        self._check_shape(x, self.input_shape, "x")
        self._check_shape(dy, self.output_shape, "dy")
        if dw is None:
            dw = torch.empty(self.weight_shape, dtype=torch.float32, device="cuda")
        self._check_shape(dw, self.weight_shape, "dw")
        need = self.weight_gradient_workspace_bytes
        if workspace is None:
            workspace = torch.empty(max(need, 4) // 4, dtype=torch.float32, device="cuda")
        _check(self._L.wino_weight_gradient(self._h, _dev_ptr(x, "x", torch.float32),
                                            _dev_ptr(dy, "dy", torch.float32), _dev_ptr(dw, "dw", torch.float32),
                                            _dev_ptr(workspace, "workspace"),
                                            workspace.numel() * workspace.element_size(), _stream()),
               "wino_weight_gradient")
        return dw

    def transform_filter_adjoint(self, w, U=None):
        """U of the flipped, transposed kernels from the forward layer's w [C][K][r^N]
        (this plan's C and K are the forward layer's K and C)."""
        import torch
        self._check_shape(w, (self.C, self.K) + (self.r,) * self.N, "w")
        if U is None:
            U = self.new_filter()
        if U.numel() * 4 < self.filter_bytes:
            raise ValueError("U is too small")
        _check(self._L.wino_transform_filter_adjoint(self._h, _dev_ptr(w, "w", torch.float32),
                                                     _dev_ptr(U, "U", torch.float32), _stream()),
               "wino_transform_filter_adjoint")
        return U

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._L.wino_destroy(h)
            self._h = None

    @property
    def handle(self):
        return self._h

    @property
    def filter_bytes(self):
        return int(self._L.wino_filter_bytes(self._h))

    @property
    def workspace_bytes(self):
        """Workspace of the two-stage API (transform_input + gemm_inverse)."""
        return int(self._L.wino_workspace_bytes(self._h))

    @property
    def forward_workspace_bytes(self):
        """Workspace forward() needs: 0 when the plan fuses the input transform
        into the product, workspace_bytes otherwise."""
        return int(self._L.wino_forward_workspace_bytes(self._h))

    def matrices(self):
        a, m, r = self.desc["alpha"], self.m, self.r
        AT = np.zeros((m, a))
        BT = np.zeros((a, a))
        G = np.zeros((a, r))
        P = ctypes.POINTER(ctypes.c_double)
        _check(self._L.wino_get_matrices(self._h, AT.ctypes.data_as(P), BT.ctypes.data_as(P),
                                         G.ctypes.data_as(P)), "wino_get_matrices")
        return AT, BT, G

    # ---- device calls -------------------------------------------------
    def _check_shape(self, t, shape, what):
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{what} has shape {tuple(t.shape)}, expected {tuple(shape)}")

    def new_filter(self):
        import torch
        return torch.empty(self.filter_bytes // 4, dtype=torch.float32, device="cuda")

    def unpack_filter(self, U):
        """U (device or host) -> numpy [alpha^N][C_pad][K_pad] in plain order."""
        d = self.desc
        cg = d["filter_channel_group"]
        u = U.detach().cpu().numpy() if hasattr(U, "detach") else np.asarray(U)
        u = u.reshape(d["n_xi"], d["C_pad"] // cg, d["K_pad"], cg)
        return u.transpose(0, 1, 3, 2).reshape(d["n_xi"], d["C_pad"], d["K_pad"])

    def unpack_workspace(self, ws):
        """V workspace (device or host) -> numpy [alpha^N][C_pad][T_pad] in plain order."""
        d = self.desc
        cg, b = d["channel_group"], d["block_tiles"]
        v = ws.detach().cpu().numpy() if hasattr(ws, "detach") else np.asarray(ws)
        v = v[: d["n_xi"] * d["C_pad"] * d["T_pad"]]
        v = v.reshape(d["T_pad"] // b, d["C_pad"] // cg, d["n_xi"], b, cg)
        return v.transpose(2, 1, 4, 0, 3).reshape(d["n_xi"], d["C_pad"], d["T_pad"])

    def new_workspace(self):
        import torch
        return torch.empty(self.workspace_bytes // 4, dtype=torch.float32, device="cuda")

    def new_output(self):
        import torch
        return torch.empty(self.output_shape, dtype=torch.float32, device="cuda")

    def transform_filter(self, w, U=None):
        import torch
        self._check_shape(w, self.weight_shape, "w")
        if U is None:
            U = self.new_filter()
        if U.numel() * 4 < self.filter_bytes:
            raise ValueError("U is too small")
        _check(self._L.wino_transform_filter(self._h, _dev_ptr(w, "w", torch.float32),
                                             _dev_ptr(U, "U", torch.float32), _stream()),
               "wino_transform_filter")
        return U

    def transform_input(self, x, ws=None):
        import torch
        self._check_shape(x, self.input_shape, "x")
        if ws is None:
            ws = self.new_workspace()
        _check(self._L.wino_transform_input(self._h, _dev_ptr(x, "x", torch.float32),
                                            _dev_ptr(ws, "workspace"), ws.numel() * ws.element_size(),
                                            _stream()), "wino_transform_input")
        return ws

    def _bias_ptr(self, bias):
        import torch
        if bias is None:
            return ctypes.c_void_p()
        self._check_shape(bias, (self.K,), "bias")
        return _dev_ptr(bias, "bias", torch.float32)

    def gemm_inverse(self, ws, U, y=None, bias=None):
        """bias: optional device [K] float32, b of eq. (2), added before the activation."""
        import torch
        if y is None:
            y = self.new_output()
        self._check_shape(y, self.output_shape, "y")
        _check(self._L.wino_gemm_inverse_ex(self._h, _dev_ptr(ws, "workspace"),
                                            ws.numel() * ws.element_size(),
                                            _dev_ptr(U, "U", torch.float32), self._bias_ptr(bias),
                                            _dev_ptr(y, "y", torch.float32), _stream()),
               "wino_gemm_inverse_ex")
        return y

    def forward(self, x, U, y=None, workspace=None, bias=None):
        """bias: optional device [K] float32, b of eq. (2), added before the activation."""
        import torch
        self._check_shape(x, self.input_shape, "x")
        if y is None:
            y = self.new_output()
        self._check_shape(y, self.output_shape, "y")
        need = self.forward_workspace_bytes
        if workspace is None and need:
            workspace = torch.empty(need // 4, dtype=torch.float32, device="cuda")
        ws_ptr = _dev_ptr(workspace, "workspace") if workspace is not None else ctypes.c_void_p()
        ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
        _check(self._L.wino_forward_ex(self._h, _dev_ptr(x, "x", torch.float32),
                                       _dev_ptr(U, "U", torch.float32), self._bias_ptr(bias),
                                       _dev_ptr(y, "y", torch.float32), ws_ptr, ws_len, _stream()),
               "wino_forward_ex")
        return y

    def pooled_shape(self, window):
        """Output shape of forward_pool: [batch, K, Y_i // window_i]."""
        return tuple(self.output_shape[:2]) + tuple(int(yi) // int(w) for yi, w in
                                                    zip(self.output_shape[2:], window))

    def forward_pool(self, x, U, window, y=None, workspace=None, bias=None):
        """wino_forward_pool: the F(4^3) forward with the max-pool (window =
        stride, (1, 2, 2) or (2, 2, 2)), or the F(2^3) forward with window
        (2, 2, 2), in the product's epilogue; y is the pooled output.  Other
        sizes and windows raise WinoError."""
        import torch
        self._check_shape(x, self.input_shape, "x")
        shape = self.pooled_shape(window)
        if y is None:
            y = torch.empty(shape, dtype=torch.float32, device="cuda")
        self._check_shape(y, shape, "y")
        need = self.forward_workspace_bytes
        if workspace is None and need:
            workspace = torch.empty(need // 4, dtype=torch.float32, device="cuda")
        ws_ptr = _dev_ptr(workspace, "workspace") if workspace is not None else ctypes.c_void_p()
        ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
        win = (ctypes.c_int32 * 3)(*[int(w) for w in window])
        _check(self._L.wino_forward_pool(self._h, _dev_ptr(x, "x", torch.float32),
                                         _dev_ptr(U, "U", torch.float32), self._bias_ptr(bias), win,
                                         _dev_ptr(y, "y", torch.float32), ws_ptr, ws_len, _stream()),
               "wino_forward_pool")
        return y

    def forward_noalloc(self, x, U, y=None, bias=None):
        """wino_forward_noalloc: the forward with the library's static device
        scratch as its workspace (the call allocates nothing; y is allocated
        here only when not given)."""
        import torch
        self._check_shape(x, self.input_shape, "x")
        if y is None:
            y = self.new_output()
        self._check_shape(y, self.output_shape, "y")
        _check(self._L.wino_forward_noalloc(self._h, _dev_ptr(x, "x", torch.float32),
                                            _dev_ptr(U, "U", torch.float32), self._bias_ptr(bias),
                                            _dev_ptr(y, "y", torch.float32), _stream()),
               "wino_forward_noalloc")
        return y


NOALLOC_SCRATCH_BYTES = 64 << 20   # WINO_NOALLOC_SCRATCH_BYTES of include/wino.h


def points_error_growth(N, m, r, points=None):
    """kappa of a point set (None: the default set); see include/wino.h."""
    L = lib()
    g = ctypes.c_double()
    if points is None:
        _check(L.wino_points_error_growth(N, m, r, None, 0, ctypes.byref(g)), "wino_points_error_growth")
    else:
        arr = (ctypes.c_double * len(points))(*[_point(p) for p in points])
        _check(L.wino_points_error_growth(N, m, r, arr, len(points), ctypes.byref(g)),
               "wino_points_error_growth")
    return g.value


def search_points(N, m, r):
    """The symmetric point set with the smallest kappa; returns (points, kappa)."""
    L = lib()
    n = m + r - 2
    arr = (ctypes.c_double * n)()
    g = ctypes.c_double()
    _check(L.wino_search_points(N, m, r, arr, ctypes.byref(g)), "wino_search_points")
    return tuple(arr), g.value


def maxpool3d(x, window, y=None):
    """Max-pool over the trailing three axes with window = stride, floor rounding."""
    import torch
    L = lib()
    lead = int(np.prod(x.shape[:-3])) if x.dim() > 3 else 1
    X = list(x.shape[-3:])
    Y = [xi // pi for xi, pi in zip(X, window)]
    if y is None:
        y = torch.empty(tuple(x.shape[:-3]) + tuple(Y), dtype=torch.float32, device=x.device)
    dims = (ctypes.c_int64 * 4)(lead, *X)
    win = (ctypes.c_int32 * 3)(*[int(p) for p in window])
    _check(L.wino_maxpool3d(dims, win, _dev_ptr(x, "x", torch.float32), _dev_ptr(y, "y", torch.float32),
                            _stream()), "wino_maxpool3d")
    return y
