"""Python binding of the Winograd convolution library (argument marshalling only).

Every step of the computation runs in the native library and its gfx950
kernels; PyTorch supplies device memory and the current HIP stream.  There is
no CPU fallback: without the built library or a GPU the calls raise.

    plan = Plan("0,1,-1,a^2+1,inf", m=4, dtype="f16")   # F(4x4, 3x3), alpha' = 7
    y = plan.conv2d(x, w)          # x [N][H][W][C], w [K][3][3][C] -> y [N][H][W][K]
"""
import ctypes
from fractions import Fraction

import torch

from . import _native as N

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def _stream_handle(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _tensor(t, name, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a GPU device")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.dim() != 4:
        raise ValueError(f"{name} must have 4 dimensions")
    return N.WgTensor(ctypes.c_void_p(t.data_ptr()), *[int(v) for v in (shape or t.shape)])


class Plan:
    """A Winograd plan F(m x m, 3 x 3) built from a modulus set (Algorithms 1, 2)."""

    def __init__(self, moduli, m, dtype="f32", inner="0,-1,inf", r=3, factors="B", path="auto",
                 generic_transforms=False, scaling="none", channel_sum="mfma"):
        """``factors``: where the CRT factors N_i go, "B" (the paper's
        matrices) or "G" (on the kernel residues).  ``path``: "separate"
        (M through memory), "fused" (contraction and output transform in one
        kernel) or "auto" (chosen per layer shape).  ``generic_transforms``:
        never use the built-in constant-coefficient transform kernels.
        ``scaling``: "none" or "l1" (every domain row of G and A divided by
        its 1-norm, compensated in B).  ``channel_sum``: "mfma" (the matrix
        cores' chains) or "pairwise" (a binary tree over 64-byte pieces of the
        channel rows; separate path)."""
        if dtype not in N.DTYPE_CODES:
            raise ValueError(f"dtype must be one of {list(N.DTYPE_CODES)}")
        if factors not in N.FACTOR_CODES:
            raise ValueError(f"factors must be one of {list(N.FACTOR_CODES)}")
        if path not in N.PATH_CODES:
            raise ValueError(f"path must be one of {list(N.PATH_CODES)}")
        if scaling not in N.SCALING_CODES:
            raise ValueError(f"scaling must be one of {list(N.SCALING_CODES)}")
        if channel_sum not in N.CHANNEL_SUM_CODES:
            raise ValueError(f"channel_sum must be one of {list(N.CHANNEL_SUM_CODES)}")
        self._lib = N.lib()
        self._h = ctypes.c_void_p()
        if factors == "B" and path == "auto" and not generic_transforms and scaling == "none" \
                and channel_sum == "mfma":
            N.check(self._lib.winograd_plan_create_str(moduli.encode(), (inner or "").encode(), int(m), int(r),
                                                       N.DTYPE_CODES[dtype], ctypes.byref(self._h)))
        else:
            opts = N.WgPlanOptions(N.FACTOR_CODES[factors], N.PATH_CODES[path], 1 if generic_transforms else 0,
                                   N.SCALING_CODES[scaling], N.CHANNEL_SUM_CODES[channel_sum])
            N.check(self._lib.winograd_plan_create_ex(moduli.encode(), (inner or "").encode(), int(m), int(r),
                                                      N.DTYPE_CODES[dtype], ctypes.byref(opts),
                                                      ctypes.byref(self._h)))
        self.moduli, self.inner, self.dtype, self.factors, self.path = moduli, inner, dtype, factors, path
        self.scaling, self.channel_sum = scaling, channel_sum
        vals = [ctypes.c_int() for _ in range(5)]
        N.check(self._lib.winograd_plan_info(self._h, *[ctypes.byref(v) for v in vals]))
        self.m, self.r, self.alpha, self.tile_in, _ = [v.value for v in vals]
        self._ws = None

    @classmethod
    def from_moduli(cls, moduli, m, dtype="f32", inner_points=None, inner_inf=True, r=3):
        """Build from structured moduli: each item is ``None`` (infinity) or a
        coefficient list (low to high) of Fractions/ints (the struct-based C entry)."""
        mods = (N.WgModulus * len(moduli))()
        for i, c in enumerate(moduli):
            if c is None:
                mods[i].degree = 0
                continue
            mods[i].degree = len(c) - 1
            for k, v in enumerate(c):
                q = Fraction(v)
                mods[i].coef[k] = N.WgRational(q.numerator, q.denominator)
        pts = inner_points or []
        inner = (N.WgRational * max(len(pts), 1))()
        for i, v in enumerate(pts):
            q = Fraction(v)
            inner[i] = N.WgRational(q.numerator, q.denominator)
        ps = N.WgPolySet(len(moduli), mods, len(pts), inner, 1 if inner_inf else 0)
        self = cls.__new__(cls)
        self._lib = N.lib()
        self._h = ctypes.c_void_p()
        N.check(self._lib.winograd_plan_create(ctypes.byref(ps), int(m), int(r), N.DTYPE_CODES[dtype],
                                               ctypes.byref(self._h)))
        self.moduli, self.inner, self.dtype, self.factors, self.path = moduli, inner_points, dtype, "B", "auto"
        vals = [ctypes.c_int() for _ in range(5)]
        N.check(self._lib.winograd_plan_info(self._h, *[ctypes.byref(v) for v in vals]))
        self.m, self.r, self.alpha, self.tile_in, _ = [v.value for v in vals]
        self._ws = None
        return self

    # ------------------------------------------------------------ plan data
    def _shape(self, which):
        return {"G": (self.alpha, self.r), "A": (self.alpha, self.m), "B": (self.tile_in, self.alpha)}[which]

    def matrix(self, which):
        """Exact matrix 'G', 'A' or 'B' as nested lists of Fractions."""
        rows, cols = self._shape(which)
        buf = (N.WgRational * (rows * cols))()
        N.check(self._lib.winograd_plan_matrix(self._h, which.encode(), buf, rows * cols))
        return [[Fraction(buf[i * cols + j].num, buf[i * cols + j].den) for j in range(cols)] for i in range(rows)]

    def matrix_f32(self, which):
        """The fp32 matrix the kernels use, as a list of lists of floats."""
        rows, cols = self._shape(which)
        buf = (ctypes.c_float * (rows * cols))()
        N.check(self._lib.winograd_plan_matrix_f32(self._h, which.encode(), buf, rows * cols))
        return [[buf[i * cols + j] for j in range(cols)] for i in range(rows)]

    @property
    def builtin(self):
        """Index of the built-in plan whose constant-coefficient transform
        kernels this plan uses, or -1."""
        out = ctypes.c_int()
        N.check(self._lib.winograd_plan_builtin(self._h, ctypes.byref(out)))
        return out.value

    @property
    def ratio(self):
        num, den = ctypes.c_int64(), ctypes.c_int64()
        N.check(self._lib.winograd_plan_ratio(self._h, ctypes.byref(num), ctypes.byref(den)))
        return Fraction(num.value, den.value)

    def workspace_bytes(self, N_, H, W, C, K):
        out = ctypes.c_size_t()
        N.check(self._lib.winograd_workspace_bytes(self._h, N_, H, W, C, K, ctypes.byref(out)))
        return out.value

    def conv_path(self, N_, H, W, C, K):
        """"separate", "fused" or "fused_input": the path conv2d takes for this layer shape."""
        out = ctypes.c_int()
        N.check(self._lib.winograd_conv_path(self._h, N_, H, W, C, K, ctypes.byref(out)))
        return N.PATH_NAMES[out.value]

    def conv_chunks(self, N_, H, W, C, K):
        """(launch pairs, images of the largest chunk) conv2d uses for this
        layer: the fused path runs a large batch in chunks of images."""
        n, c = ctypes.c_int64(), ctypes.c_int64()
        N.check(self._lib.winograd_conv_chunks(self._h, N_, H, W, C, K, ctypes.byref(n), ctypes.byref(c)))
        return n.value, c.value

    # ------------------------------------------------------------- compute
    @property
    def torch_dtype(self):
        return TORCH_DTYPES[self.dtype]

    def _check_dtype(self, t, name):
        if t.dtype != self.torch_dtype:
            raise TypeError(f"{name} must be {self.torch_dtype}, got {t.dtype}")

    def bind_workspace(self, ws):
        """Bind a caller-owned uint8 device tensor as the workspace."""
        N.check(self._lib.winograd_plan_set_workspace(self._h, ctypes.c_void_p(ws.data_ptr()), ws.numel()))
        self._ws = ws

    def conv2d(self, x, w, y=None, workspace=None, stream=None):
        """y = conv3x3(x, w), stride 1, padding 1 (NHWC), by eq. (2)."""
        self._check_dtype(x, "x")
        self._check_dtype(w, "w")
        Nn, H, W, C = x.shape
        K = w.shape[0]
        if y is None:
            y = torch.empty((Nn, H, W, K), dtype=x.dtype, device=x.device)
        self._check_dtype(y, "y")
        need = self.workspace_bytes(Nn, H, W, C, K)
        if workspace is None:
            if self._ws is None or self._ws.numel() < need or self._ws.device != x.device:
                self.bind_workspace(torch.empty(need, dtype=torch.uint8, device=x.device))
        else:
            self.bind_workspace(workspace)
        xt, wt, yt = _tensor(x, "x"), _tensor(w, "w"), _tensor(y, "y")
        N.check(self._lib.winograd_conv2d(self._h, ctypes.byref(xt), ctypes.byref(wt), ctypes.byref(yt),
                                          _stream_handle(stream)))
        self._keep_for(stream, y)
        return y

    def _keep_for(self, stream, y):
        """Memory allocated here on the current stream but used on another
        one: keep the caching allocator from reusing it before that stream's
        work is done."""
        if stream is not None and stream != torch.cuda.current_stream(y.device):
            y.record_stream(stream)
            if self._ws is not None:
                self._ws.record_stream(stream)

    def workspace_bytes_1d(self, N_, L, C, K):
        out = ctypes.c_size_t()
        N.check(self._lib.winograd_workspace_bytes_1d(self._h, N_, L, C, K, ctypes.byref(out)))
        return out.value

    def conv1d(self, x, w, y=None, workspace=None, stream=None):
        """1D F(m, 3): y [N][L][K] = conv(x [N][L][C], w [K][3][C]), stride 1,
        padding 1, along L (the descriptors carry height 1)."""
        self._check_dtype(x, "x")
        self._check_dtype(w, "w")
        if x.dim() != 3 or w.dim() != 3 or w.shape[1] != 3 or w.shape[2] != x.shape[2]:
            raise ValueError("x must be [N][L][C] and w [K][3][C]")
        Nn, L, C = x.shape
        K = w.shape[0]
        if y is None:
            y = torch.empty((Nn, L, K), dtype=x.dtype, device=x.device)
        self._check_dtype(y, "y")
        need = self.workspace_bytes_1d(Nn, L, C, K)
        if workspace is None:
            if self._ws is None or self._ws.numel() < need or self._ws.device != x.device:
                self.bind_workspace(torch.empty(need, dtype=torch.uint8, device=x.device))
        else:
            self.bind_workspace(workspace)
        xt = _tensor(x.unsqueeze(1), "x")
        wt = _tensor(w.unsqueeze(1), "w")
        yt = _tensor(y.unsqueeze(1), "y")
        N.check(self._lib.winograd_conv1d(self._h, ctypes.byref(xt), ctypes.byref(wt), ctypes.byref(yt),
                                          _stream_handle(stream)))
        self._keep_for(stream, y)
        return y

    def conv2d_static(self, x, w, y, stream=None):
        """y = conv3x3(x, w) through winograd_conv2d_static: the library's own
        per-GPU device workspace, nothing allocated (y must be given).  Calls
        that overlap in time on one GPU race."""
        self._check_dtype(x, "x")
        self._check_dtype(w, "w")
        self._check_dtype(y, "y")
        xt, wt, yt = _tensor(x, "x"), _tensor(w, "w"), _tensor(y, "y")
        N.check(self._lib.winograd_conv2d_static(self._h, ctypes.byref(xt), ctypes.byref(wt), ctypes.byref(yt),
                                                 _stream_handle(stream)))
        return y

    def bind_call(self, x, w, y, stream=None):
        """Marshal the arguments of one conv2d call once and return a
        zero-argument callable that launches it (for tight loops and graph
        capture).  The tensors and the bound workspace must stay alive."""
        self._check_dtype(x, "x")
        self._check_dtype(w, "w")
        self._check_dtype(y, "y")
        Nn, H, W, C = x.shape
        need = self.workspace_bytes(Nn, H, W, C, w.shape[0])
        if self._ws is None or self._ws.numel() < need:
            self.bind_workspace(torch.empty(need, dtype=torch.uint8, device=x.device))
        xt, wt, yt = _tensor(x, "x"), _tensor(w, "w"), _tensor(y, "y")
        args = (self._h, ctypes.byref(xt), ctypes.byref(wt), ctypes.byref(yt))
        fn = self._lib.winograd_conv2d
        keep = (xt, wt, yt, x, w, y)

        def call(stream_=None):
            st = fn(*args, _stream_handle(stream_ if stream_ is not None else stream))
            if st != N.WG_OK:
                N.check(st)
            return keep[-1]
        return call

    # stage entry points (one kernel each)
    def geometry(self, N_, H, W, C, K):
        th, tw = -(-H // self.m), -(-W // self.m)
        return {"T": N_ * th * tw, "th": th, "tw": tw, "Cp": -(-C // 8) * 8, "Kp": -(-K // 8) * 8}

    def kernel_transform(self, w, stream=None):
        self._check_dtype(w, "w")
        K, _, _, C = w.shape
        Cp = -(-C // 8) * 8
        U = torch.empty((self.alpha * self.alpha, K, Cp), dtype=w.dtype, device=w.device)
        wt = _tensor(w, "w")
        N.check(self._lib.winograd_kernel_transform(self._h, ctypes.byref(wt), ctypes.c_void_p(U.data_ptr()),
                                                    _stream_handle(stream)))
        return U

    def input_transform(self, x, stream=None):
        self._check_dtype(x, "x")
        Nn, H, W, C = x.shape
        g = self.geometry(Nn, H, W, C, 1)
        V = torch.empty((self.alpha * self.alpha, g["T"], g["Cp"]), dtype=x.dtype, device=x.device)
        xt = _tensor(x, "x")
        N.check(self._lib.winograd_input_transform(self._h, ctypes.byref(xt), ctypes.c_void_p(V.data_ptr()),
                                                   _stream_handle(stream)))
        return V

    def kernel_input_transform(self, w, x, stream=None):
        """Both transforms in one launch (conv2d's first kernel): returns (U, V)."""
        self._check_dtype(w, "w")
        self._check_dtype(x, "x")
        K, _, _, C = w.shape
        Nn, H, W, _ = x.shape
        g = self.geometry(Nn, H, W, C, K)
        a2 = self.alpha * self.alpha
        U = torch.empty((a2, K, g["Cp"]), dtype=w.dtype, device=w.device)
        V = torch.empty((a2, g["T"], g["Cp"]), dtype=x.dtype, device=x.device)
        wt, xt = _tensor(w, "w"), _tensor(x, "x")
        N.check(self._lib.winograd_kernel_input_transform(self._h, ctypes.byref(wt), ctypes.byref(xt),
                                                          ctypes.c_void_p(U.data_ptr()), ctypes.c_void_p(V.data_ptr()),
                                                          _stream_handle(stream)))
        return U, V

    def contract(self, V, U, C, stream=None):
        self._check_dtype(V, "V")
        self._check_dtype(U, "U")
        a2, T, Cp = V.shape
        K = U.shape[1]
        if a2 != self.alpha ** 2 or U.shape[0] != a2 or U.shape[2] != Cp or Cp != -(-C // 8) * 8:
            raise ValueError("V must be [alpha'^2][T][Cp] and U [alpha'^2][K][Cp]")
        if not (V.is_contiguous() and U.is_contiguous()):
            raise ValueError("V and U must be contiguous")
        Kp = -(-K // 8) * 8
        M = torch.empty((a2, T, Kp), dtype=torch.float32, device=V.device)
        N.check(self._lib.winograd_contract(self._h, ctypes.c_void_p(V.data_ptr()), ctypes.c_void_p(U.data_ptr()),
                                            ctypes.c_void_p(M.data_ptr()), T, C, K, _stream_handle(stream)))
        return M

    def output_transform(self, M, N_, H, W, K, stream=None):
        g = self.geometry(N_, H, W, 1, K)
        if M.dtype != torch.float32 or tuple(M.shape) != (self.alpha ** 2, g["T"], g["Kp"]):
            raise ValueError("M must be fp32 [alpha'^2][T][Kp]")
        if not M.is_contiguous():
            raise ValueError("M must be contiguous")
        y = torch.empty((N_, H, W, K), dtype=self.torch_dtype, device=M.device)
        yt = _tensor(y, "y")
        N.check(self._lib.winograd_output_transform(self._h, ctypes.c_void_p(M.data_ptr()), ctypes.byref(yt),
                                                    _stream_handle(stream)))
        return y

    def contract_output(self, V, U, C, N_, H, W, stream=None):
        """The fused kernel alone: y [N][H][W][K] from V and U, no M in memory."""
        self._check_dtype(V, "V")
        self._check_dtype(U, "U")
        a2, T, Cp = V.shape
        K = U.shape[1]
        g = self.geometry(N_, H, W, C, K)
        if a2 != self.alpha ** 2 or U.shape[0] != a2 or U.shape[2] != Cp or Cp != g["Cp"] or T != g["T"]:
            raise ValueError("V must be [alpha'^2][T][Cp] and U [alpha'^2][K][Cp]")
        if not (V.is_contiguous() and U.is_contiguous()):
            raise ValueError("V and U must be contiguous")
        y = torch.empty((N_, H, W, K), dtype=self.torch_dtype, device=V.device)
        yt = _tensor(y, "y")
        N.check(self._lib.winograd_contract_output(self._h, ctypes.c_void_p(V.data_ptr()),
                                                   ctypes.c_void_p(U.data_ptr()), C, ctypes.byref(yt),
                                                   _stream_handle(stream)))
        return y

    def input_contract_output(self, x, U, stream=None):
        """The fused kernel with the input transform in its prologue: y [N][H][W][K]
        from x and U, neither V nor M in memory."""
        self._check_dtype(x, "x")
        self._check_dtype(U, "U")
        Nn, H, W, C = x.shape
        a2, K, Cp = U.shape
        if a2 != self.alpha ** 2 or Cp != -(-C // 8) * 8 or not U.is_contiguous():
            raise ValueError("U must be a contiguous [alpha'^2][K][Cp] tensor for x's C")
        y = torch.empty((Nn, H, W, K), dtype=self.torch_dtype, device=x.device)
        xt, yt = _tensor(x, "x"), _tensor(y, "y")
        N.check(self._lib.winograd_input_contract_output(self._h, ctypes.byref(xt), ctypes.c_void_p(U.data_ptr()),
                                                         ctypes.byref(yt), _stream_handle(stream)))
        return y

    # ------------------------------------------------------------ lifetime
    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            self._lib.winograd_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __repr__(self):
        return f"Plan({self.moduli!r}, m={self.m}, dtype={self.dtype!r}, alpha'={self.alpha}, path={self.path!r})"
