"""Thin Python binding of libswsft.so (the C ABI in include/swsft.h).

Argument marshalling only: every step of the transform and the layer runs in
the library's HIP kernels.  Torch tensors supply device memory and the
current stream.  There is no fallback: if the library is not built, or is
called without a GPU, this module raises.

Tensor conventions (see include/swsft.h):
  * f32 plans take complex64 tensors (or float32 with a trailing dim of 2);
  * bf16 plans take bfloat16 tensors with a trailing dim of 2 (re, im);
  * spatial [B, S, C, H, W], coefficients [L*L, B, S, C],
    filters [L, S_out, C_out, S_in, C_in], phase-collapse weights complex64.
"""

from __future__ import annotations

import ctypes
import os
import re

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# SWSFT_LIBRARY may name another build of the same library (e.g. a tuning
# variant); by default the in-tree build is used.
LIB_PATH = os.environ.get("SWSFT_LIBRARY") or os.path.join(_PKG, "libswsft.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "swsft.h")

OK, E_INVALID, E_UNSUPPORTED, E_ALLOC, E_HIP, E_WORKSPACE = range(6)
PLAN_DFT_MATMUL, PLAN_DELTA, PLAN_DELTA_SYM = 1, 2, 4
F32, BF16 = 0, 1
OP_FORWARD, OP_INVERSE, OP_CONV, OP_CONV_BACKWARD, OP_BATCH_NORM = 0, 1, 2, 3, 4
STAGES = ("dft_fwd", "lat_fwd", "mix", "lat_inv", "dft_inv", "phase_collapse", "tables",
          "filter_grad", "filter_adjoint", "batch_norm", "delta_theta", "small_fwd", "small_inv")

_lib = None


class BlockParams(ctypes.Structure):
    """swsft_block_params: device pointers of the residual block's parameters."""
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("K1", "K2", "gamma1", "beta1", "gamma2", "beta2", "pc1_W1", "pc1_W2", "pc1_b",
                 "pc2_W1", "pc2_W2", "pc2_b")] + \
               [("eps", ctypes.c_float), ("var1_out", ctypes.c_void_p),
                ("var2_out", ctypes.c_void_p)]


class SwsftError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libswsft.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2306_05420_amd.build` (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    ip = ctypes.POINTER(ctypes.c_int)
    sigs = {
        "swsft_plan_create": (i, [i, i, i, ip, i, ip, i, i, ctypes.POINTER(vp)]),
        "swsft_plan_create_ex": (i, [i, i, i, ip, i, ip, i, i, ctypes.c_uint,
                                     ctypes.POINTER(vp)]),
        "swsft_plan_destroy": (None, [vp]),
        "swsft_workspace_bytes": (sz, [vp, i, i, i, i]),
        "swsft_forward": (i, [vp, i, i, vp, vp, vp, sz, vp]),
        "swsft_inverse": (i, [vp, i, i, vp, vp, vp, sz, vp]),
        "spin_sph_conv_forward": (i, [vp, i, i, i, vp, vp, vp, vp, sz, vp]),
        "spin_sph_conv_backward": (i, [vp, i, i, i, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "spin_sph_conv_forward_train": (i, [vp, i, i, i, vp, vp, vp, vp, vp, sz, vp]),
        "spin_sph_conv_forward_noalloc": (i, [vp, i, i, i, vp, vp, vp, vp]),
        "spin_sph_phase_collapse": (i, [vp, i, i, vp, vp, vp, vp, vp, vp]),
        "spin_sph_mix": (i, [vp, i, i, i, vp, vp, vp, vp]),
        "spin_sph_spectral_batch_norm": (i, [vp, i, i, vp, vp, vp, ctypes.c_float, vp, vp, vp,
                                             vp, vp, sz, vp]),
        "swsft_block_workspace_bytes": (sz, [vp, vp, i, i]),
        "spin_sph_residual_block_forward": (i, [vp, vp, i, i, vp, ctypes.POINTER(BlockParams),
                                                vp, vp, sz, vp]),
        "swsft_status_string": (ctypes.c_char_p, [i]),
        "swsft_last_error": (ctypes.c_char_p, []),
        "swsft_stage_timing": (i, [vp, i]),
        "swsft_stage_times": (i, [vp, ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(ctypes.c_longlong), i]),
        "swsft_stage_name": (ctypes.c_char_p, [i]),
        "swsft_plan_table": (i, [vp, i, i, vp, sz]),
        "swsft_probe_mfma": (i, [i, i, ctypes.c_longlong, i, vp, ctypes.POINTER(ctypes.c_double),
                                 vp]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def header_functions() -> list:
    """Names of the functions declared in include/swsft.h."""
    text = open(HEADER_PATH).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^[A-Za-z_][\w \*]*?\b(\w+)\s*\(", text, flags=re.M)


def _need(t: torch.Tensor, dtype, shape, name: str):
    if t.dtype != dtype or not t.is_cuda or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be a contiguous {dtype} GPU tensor of shape {tuple(shape)}")


def _check(status: int, what: str):
    if status != OK:
        L = lib()
        detail = L.swsft_last_error().decode()
        raise SwsftError(status, f"{what}: {L.swsft_status_string(status).decode()}: {detail}")


def _stream_handle(stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def probe_mfma(dtype: str, random_operands: bool, iters: int, n_waves: int, out: torch.Tensor,
               stream=None) -> float:
    """Enqueue the register-only MFMA probe (swsft_probe_mfma): n_waves waves
    each run `iters` rounds of four MFMAs of the dtype's shape; `out` is a
    float32 GPU tensor of 64 n_waves checksums.  Returns the flops the kernel
    issues; the caller times it on its stream."""
    _need(out, torch.float32, (64 * n_waves,), "out")
    flops = ctypes.c_double(0.0)
    if dtype not in ("f32", "bf16"):
        raise ValueError("dtype must be 'f32' or 'bf16'")
    _check(lib().swsft_probe_mfma(F32 if dtype == "f32" else BF16, int(bool(random_operands)),
                                  int(iters), int(n_waves), out.data_ptr(), ctypes.byref(flops),
                                  _stream_handle(stream)), "swsft_probe_mfma")
    return flops.value


class Plan:
    """A transform plan: grid H x W, bandlimit L, input/output spins, dtype,
    the longitude stages ("fft": register FFT; "matmul": dense DFT matrix
    products on MFMA, which also take widths that are not powers of two)
    and the latitude stages ("direct": precomputed d^l(theta_j) tables;
    "delta" / "delta_sym": the Wigner-Delta route of eqs. (4)-(6), without /
    with the J and G symmetries).

    Owns the device tables built by swsft_plan_create; workspaces are cached
    per call shape and stream (allocated through torch, i.e. by the caller of
    the C ABI), so calls with the same shape on two streams never share one.
    """

    def __init__(self, H: int, W: int, L: int, spins_in, spins_out, dtype: str = "f32",
                 longitude: str = "fft", latitude: str = "direct"):
        self.H, self.W, self.L = int(H), int(W), int(L)
        self.spins_in = tuple(int(s) for s in spins_in)
        self.spins_out = tuple(int(s) for s in spins_out)
        if dtype not in ("f32", "bf16"):
            raise ValueError("dtype must be 'f32' or 'bf16'")
        self.dtype = dtype
        self._code = F32 if dtype == "f32" else BF16
        si = (ctypes.c_int * len(self.spins_in))(*self.spins_in)
        so = (ctypes.c_int * len(self.spins_out))(*self.spins_out)
        h = ctypes.c_void_p()
        if longitude not in ("fft", "matmul"):
            raise ValueError("longitude must be 'fft' or 'matmul'")
        self.longitude = longitude
        if latitude not in ("direct", "delta", "delta_sym"):
            raise ValueError("latitude must be 'direct', 'delta' or 'delta_sym'")
        self.latitude = latitude
        flags = PLAN_DFT_MATMUL if longitude == "matmul" else 0
        flags |= {"direct": 0, "delta": PLAN_DELTA, "delta_sym": PLAN_DELTA_SYM}[latitude]
        _check(lib().swsft_plan_create_ex(self.H, self.W, self.L, si, len(self.spins_in), so,
                                          len(self.spins_out), self._code, flags,
                                          ctypes.byref(h)),
               "swsft_plan_create_ex")
        self._h = h
        self._ws = {}
        self.device = torch.device("cuda", torch.cuda.current_device())

    # -- lifetime --------------------------------------------------------
    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            torch.cuda.synchronize(self.device)
            lib().swsft_plan_destroy(self._h)
            self._h = ctypes.c_void_p()
        self._ws = {}

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- helpers ---------------------------------------------------------
    def real_view(self, t: torch.Tensor) -> torch.Tensor:
        """Validate a complex tensor of this plan's storage type and return
        its real (..., 2) view."""
        if not t.is_cuda:
            raise ValueError("tensor must be on the GPU")
        if self.dtype == "f32":
            if t.dtype == torch.complex64:
                t = torch.view_as_real(t)
            elif t.dtype != torch.float32 or t.shape[-1] != 2:
                raise ValueError(f"f32 plan needs complex64 tensors, got {t.dtype}")
        else:
            if t.dtype != torch.bfloat16 or t.shape[-1] != 2:
                raise ValueError("bf16 plan needs bfloat16 tensors with a trailing dim of 2")
        if not t.is_contiguous():
            raise ValueError("tensor must be contiguous")
        return t

    def empty(self, *shape) -> torch.Tensor:
        """An uninitialised complex tensor of this plan's storage type."""
        if self.dtype == "f32":
            return torch.empty(*shape, dtype=torch.complex64, device=self.device)
        return torch.empty(*shape, 2, dtype=torch.bfloat16, device=self.device)

    def _shape(self, t, want, name):
        got = tuple(t.shape[:-1])
        if got != tuple(want):
            raise ValueError(f"{name}: shape {got}, expected {tuple(want)}")

    def workspace_bytes(self, op: int, B: int, C_in: int, C_out: int) -> int:
        return int(lib().swsft_workspace_bytes(self._h, op, B, C_in, C_out))

    def workspace(self, op: int, B: int, C_in: int, C_out: int, stream: int = None) -> torch.Tensor:
        """The cached workspace of one call shape on one stream (a stream
        handle as passed to the library; None: the current stream)."""
        if stream is None:
            stream = _stream_handle(None)
        key = (op, B, C_in, C_out, stream)
        ws = self._ws.get(key)
        if ws is None:
            n = self.workspace_bytes(op, B, C_in, C_out)
            if n == 0:
                raise ValueError("invalid workspace request")
            ws = torch.empty(n, dtype=torch.uint8, device=self.device)
            self._ws[key] = ws
        return ws

    # -- the calls ---------------------------------------------------------
    def forward(self, x: torch.Tensor, coef: torch.Tensor = None, stream=None) -> torch.Tensor:
        """Forward transform, eq. (2): x [B, S_in, C, H, W] -> coef [L*L, B, S_in, C]."""
        xr = self.real_view(x)
        B, S, C = xr.shape[:3]
        self._shape(xr, (B, len(self.spins_in), C, self.H, self.W), "x")
        if coef is None:
            coef = self.empty(self.L * self.L, B, S, C)
        cr = self.real_view(coef)
        self._shape(cr, (self.L * self.L, B, S, C), "coef")
        sh = _stream_handle(stream)
        ws = self.workspace(OP_FORWARD, B, C, 1, sh)
        _check(lib().swsft_forward(self._h, B, C, xr.data_ptr(), cr.data_ptr(), ws.data_ptr(),
                                   ws.numel(), sh), "swsft_forward")
        return coef

    def inverse(self, coef: torch.Tensor, y: torch.Tensor = None, stream=None) -> torch.Tensor:
        """Inverse transform, eq. (3): coef [L*L, B, S_out, C] -> y [B, S_out, C, H, W]."""
        cr = self.real_view(coef)
        _, B, S, C = cr.shape[:4]
        self._shape(cr, (self.L * self.L, B, len(self.spins_out), C), "coef")
        if y is None:
            y = self.empty(B, S, C, self.H, self.W)
        yr = self.real_view(y)
        self._shape(yr, (B, S, C, self.H, self.W), "y")
        sh = _stream_handle(stream)
        ws = self.workspace(OP_INVERSE, B, 1, C, sh)
        _check(lib().swsft_inverse(self._h, B, C, cr.data_ptr(), yr.data_ptr(), ws.data_ptr(),
                                   ws.numel(), sh), "swsft_inverse")
        return y

    def conv(self, x: torch.Tensor, filters: torch.Tensor, y: torch.Tensor = None,
             stream=None, coef_x: torch.Tensor = None):
        """The layer: x [B, S_in, C_in, H, W], filters [L, S_out, C_out, S_in, C_in]
        -> y [B, S_out, C_out, H, W].  With coef_x (a [L*L, B, S_in, C_in]
        tensor, or True to allocate one) the input's coefficients are saved
        for the backward pass and (y, coef_x) is returned."""
        xr = self.real_view(x)
        B, S, Cin = xr.shape[:3]
        self._shape(xr, (B, len(self.spins_in), Cin, self.H, self.W), "x")
        kr = self.real_view(filters)
        Cout = kr.shape[2]
        self._shape(kr, (self.L, len(self.spins_out), Cout, len(self.spins_in), Cin), "filters")
        if y is None:
            y = self.empty(B, len(self.spins_out), Cout, self.H, self.W)
        yr = self.real_view(y)
        self._shape(yr, (B, len(self.spins_out), Cout, self.H, self.W), "y")
        sh = _stream_handle(stream)
        ws = self.workspace(OP_CONV, B, Cin, Cout, sh)
        if coef_x is None or coef_x is False:
            _check(lib().spin_sph_conv_forward(self._h, B, Cin, Cout, xr.data_ptr(),
                                               kr.data_ptr(), yr.data_ptr(), ws.data_ptr(),
                                               ws.numel(), sh),
                   "spin_sph_conv_forward")
            return y
        if coef_x is True:
            coef_x = self.empty(self.L * self.L, B, S, Cin)
        cr = self.real_view(coef_x)
        self._shape(cr, (self.L * self.L, B, S, Cin), "coef_x")
        _check(lib().spin_sph_conv_forward_train(self._h, B, Cin, Cout, xr.data_ptr(),
                                                 kr.data_ptr(), yr.data_ptr(), cr.data_ptr(),
                                                 ws.data_ptr(), ws.numel(),
                                                 sh),
               "spin_sph_conv_forward_train")
        return y, coef_x

    def conv_backward(self, x: torch.Tensor, filters: torch.Tensor, grad_y: torch.Tensor,
                      need_x: bool = True, need_filters: bool = True, grad_x: torch.Tensor = None,
                      grad_filters: torch.Tensor = None, stream=None,
                      coef_x: torch.Tensor = None):
        """Gradients of the layer for a real loss with dL = Re sum conj(grad_y) dy:
        returns (grad_x [B, S_in, C_in, H, W] or None,
                 grad_filters [L, S_out, C_out, S_in, C_in] or None).
        coef_x: the input's coefficients saved by conv(..., coef_x=True), so
        that x is not transformed again."""
        if not (need_x or need_filters):
            raise ValueError("request grad_x, grad_filters or both")
        xr = self.real_view(x)
        B, S, Cin = xr.shape[:3]
        self._shape(xr, (B, len(self.spins_in), Cin, self.H, self.W), "x")
        kr = self.real_view(filters)
        Cout = kr.shape[2]
        self._shape(kr, (self.L, len(self.spins_out), Cout, len(self.spins_in), Cin), "filters")
        gr = self.real_view(grad_y)
        self._shape(gr, (B, len(self.spins_out), Cout, self.H, self.W), "grad_y")
        gx_ptr = gk_ptr = None
        if need_x:
            if grad_x is None:
                grad_x = self.empty(B, len(self.spins_in), Cin, self.H, self.W)
            gxr = self.real_view(grad_x)
            self._shape(gxr, tuple(xr.shape[:-1]), "grad_x")
            gx_ptr = gxr.data_ptr()
        else:
            grad_x = None
        if need_filters:
            if grad_filters is None:
                grad_filters = self.empty(*kr.shape[:-1])
            gkr = self.real_view(grad_filters)
            self._shape(gkr, tuple(kr.shape[:-1]), "grad_filters")
            gk_ptr = gkr.data_ptr()
        else:
            grad_filters = None
        cx_ptr = None
        if coef_x is not None:
            cr = self.real_view(coef_x)
            self._shape(cr, (self.L * self.L, B, S, Cin), "coef_x")
            cx_ptr = cr.data_ptr()
        sh = _stream_handle(stream)
        ws = self.workspace(OP_CONV_BACKWARD, B, Cin, Cout, sh)
        _check(lib().spin_sph_conv_backward(self._h, B, Cin, Cout, xr.data_ptr(), cx_ptr,
                                            kr.data_ptr(), gr.data_ptr(), gx_ptr, gk_ptr,
                                            ws.data_ptr(), ws.numel(), sh),
               "spin_sph_conv_backward")
        return grad_x, grad_filters

    def phase_collapse(self, x: torch.Tensor, W1: torch.Tensor, W2: torch.Tensor,
                       bias: torch.Tensor, y: torch.Tensor = None, stream=None) -> torch.Tensor:
        """x0 <- W1 x0 + W2 |x| + b on spins_out (in place if y is x)."""
        xr = self.real_view(x)
        B, S, C = xr.shape[:3]
        self._shape(xr, (B, len(self.spins_out), C, self.H, self.W), "x")
        for t, shp, nm in ((W1, (C, C), "W1"), (W2, (C, S * C), "W2"), (bias, (C,), "bias")):
            if t.dtype != torch.complex64 or not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"{nm} must be a contiguous complex64 GPU tensor")
            if tuple(t.shape) != shp:
                raise ValueError(f"{nm}: shape {tuple(t.shape)}, expected {shp}")
        if y is None:
            y = self.empty(*xr.shape[:-1])
        yr = self.real_view(y)
        self._shape(yr, tuple(xr.shape[:-1]), "y")
        _check(lib().spin_sph_phase_collapse(self._h, B, C, xr.data_ptr(), W1.data_ptr(),
                                             W2.data_ptr(), bias.data_ptr(), yr.data_ptr(),
                                             _stream_handle(stream)), "spin_sph_phase_collapse")
        return y

    def mix(self, coef: torch.Tensor, filters: torch.Tensor, out: torch.Tensor = None,
            stream=None) -> torch.Tensor:
        """Per-degree mixing: coef [L*L, B, S_in, C_in] -> [L*L, B, S_out, C_out]."""
        cr = self.real_view(coef)
        L2, B, S, Cin = cr.shape[:4]
        self._shape(cr, (self.L * self.L, B, len(self.spins_in), Cin), "coef")
        kr = self.real_view(filters)
        Cout = kr.shape[2]
        self._shape(kr, (self.L, len(self.spins_out), Cout, len(self.spins_in), Cin), "filters")
        if out is None:
            out = self.empty(L2, B, len(self.spins_out), Cout)
        orr = self.real_view(out)
        self._shape(orr, (L2, B, len(self.spins_out), Cout), "out")
        _check(lib().spin_sph_mix(self._h, B, Cin, Cout, cr.data_ptr(), kr.data_ptr(),
                                  orr.data_ptr(), _stream_handle(stream)), "spin_sph_mix")
        return out

    def batch_norm(self, coef: torch.Tensor, gamma: torch.Tensor, beta: torch.Tensor = None,
                   eps: float = 1e-5, var: torch.Tensor = None, skip: torch.Tensor = None,
                   out: torch.Tensor = None, stream=None):
        """Spectral batch norm of coefficients [L*L, B, S_out, C] of the output
        spins; gamma float32 [S_out, C], beta complex64 [C] or None, var
        float32 [S_out, C] (given statistics) or None (batch statistics).
        Returns (out, the variance used, float32 [S_out, C])."""
        cr = self.real_view(coef)
        L2, B, S, C = cr.shape[:4]
        self._shape(cr, (self.L * self.L, B, len(self.spins_out), C), "coef")
        _need(gamma, torch.float32, (S, C), "gamma")
        if beta is not None:
            _need(beta, torch.complex64, (C,), "beta")
        if var is not None:
            _need(var, torch.float32, (S, C), "var")
        sk = None
        if skip is not None:
            sk = self.real_view(skip)
            self._shape(sk, tuple(cr.shape[:-1]), "skip")
        if out is None:
            out = self.empty(*cr.shape[:-1])
        orr = self.real_view(out)
        self._shape(orr, tuple(cr.shape[:-1]), "out")
        var_out = torch.empty((S, C), dtype=torch.float32, device=self.device)
        sh = _stream_handle(stream)
        ws = self.workspace(OP_BATCH_NORM, B, 1, C, sh)
        _check(lib().spin_sph_spectral_batch_norm(
            self._h, B, C, cr.data_ptr(), gamma.data_ptr(),
            None if beta is None else beta.data_ptr(), float(eps),
            None if var is None else var.data_ptr(), var_out.data_ptr(),
            None if sk is None else sk.data_ptr(), orr.data_ptr(), ws.data_ptr(), ws.numel(),
            sh), "spin_sph_spectral_batch_norm")
        return out, var_out

    # -- tables and timing -------------------------------------------------
    def table(self, which: int, spin_index: int) -> torch.Tensor:
        """Copy of a plan table on the host (float32 or bfloat16 tensor):
        which 0: [2L-1, L, Hp] forward; which 1: [2L-1, Hp, Lp] inverse;
        which 2: [2L-1, Hp, Lp] backward synthesis (input spins);
        which 3: [2L-1, L, Hp] backward analysis (output spins)."""
        Hp = (self.H + 7) // 8 * 8
        Lp = (self.L + 31) // 32 * 32
        M = 2 * self.L - 1
        shape = (M, self.L, Hp) if which in (0, 3) else (M, Hp, Lp)
        dt = torch.float32 if self.dtype == "f32" else torch.bfloat16
        out = torch.empty(shape, dtype=dt)
        _check(lib().swsft_plan_table(self._h, which, spin_index, out.data_ptr(),
                                      out.numel() * out.element_size()), "swsft_plan_table")
        return out

    def stage_timing(self, enable: bool = True):
        _check(lib().swsft_stage_timing(self._h, 1 if enable else 0), "swsft_stage_timing")

    def stage_times(self) -> dict:
        """{stage: (total ms, launches)} since the last read (synchronizes)."""
        n = len(STAGES)
        ms = (ctypes.c_double * n)()
        cnt = (ctypes.c_longlong * n)()
        lib().swsft_stage_times(self._h, ms, cnt, n)
        return {STAGES[i]: (ms[i], cnt[i]) for i in range(n) if cnt[i]}


class ResidualBlock:
    """The residual block with a Fourier-space skip connection, run by
    spin_sph_residual_block_forward: x on an H_in grid -> y on an H_out grid
    (spectral pooling when H_out < H_in), bandlimit L = H_out / 2 unless given.

    Parameters are device tensors: K1, K2 filters [L, S, C, S, C] in the
    plans' storage type; gamma1, gamma2 float32 [S, C]; beta1, beta2 complex64
    [C] or None; pc1, pc2 = (W1 [C, C], W2 [C, S*C], b [C]) complex64.
    """

    def __init__(self, H_in: int, H_out: int, spins, C: int, dtype: str = "f32", L: int = None):
        self.L = int(L) if L is not None else H_out // 2
        self.C = int(C)
        self.spins = tuple(int(s) for s in spins)
        self.p_in = Plan(H_in, H_in, self.L, self.spins, self.spins, dtype)
        self.p_out = Plan(H_out, H_out, self.L, self.spins, self.spins, dtype)
        self._ws = {}

    def close(self):
        self.p_in.close()
        self.p_out.close()
        self._ws = {}

    def workspace(self, B: int, stream: int = None) -> torch.Tensor:
        """The cached workspace of batch B on one stream (None: the current one)."""
        if stream is None:
            stream = _stream_handle(None)
        key = (B, stream)
        ws = self._ws.get(key)
        if ws is None:
            n = int(lib().swsft_block_workspace_bytes(self.p_in._h, self.p_out._h, B, self.C))
            if n == 0:
                raise ValueError("invalid workspace request")
            ws = torch.empty(n, dtype=torch.uint8, device=self.p_out.device)
            self._ws[key] = ws
        return ws

    def forward(self, x, K1, K2, gamma1, beta1, gamma2, beta2, pc1, pc2, eps: float = 1e-5,
                y: torch.Tensor = None, variances: bool = False, stream=None):
        """y [B, S, C, H_out, H_out]; with variances=True also returns the two
        batch-norm variances (float32 [S, C] each)."""
        po = self.p_out
        xr = self.p_in.real_view(x)
        B = xr.shape[0]
        S, C = len(self.spins), self.C
        self.p_in._shape(xr, (B, S, C, self.p_in.H, self.p_in.W), "x")
        kshape = (self.L, S, C, S, C)
        k1, k2 = po.real_view(K1), po.real_view(K2)
        po._shape(k1, kshape, "K1")
        po._shape(k2, kshape, "K2")
        _need(gamma1, torch.float32, (S, C), "gamma1")
        _need(gamma2, torch.float32, (S, C), "gamma2")
        for b, nm in ((beta1, "beta1"), (beta2, "beta2")):
            if b is not None:
                _need(b, torch.complex64, (C,), nm)
        for (W1, W2, b), nm in ((pc1, "pc1"), (pc2, "pc2")):
            _need(W1, torch.complex64, (C, C), nm + " W1")
            _need(W2, torch.complex64, (C, S * C), nm + " W2")
            _need(b, torch.complex64, (C,), nm + " b")
        if y is None:
            y = po.empty(B, S, C, po.H, po.W)
        yr = po.real_view(y)
        po._shape(yr, (B, S, C, po.H, po.W), "y")
        v1 = torch.empty((S, C), dtype=torch.float32, device=po.device)
        v2 = torch.empty((S, C), dtype=torch.float32, device=po.device)
        ptr = lambda t: None if t is None else t.data_ptr()
        prm = BlockParams(k1.data_ptr(), k2.data_ptr(), gamma1.data_ptr(), ptr(beta1),
                          gamma2.data_ptr(), ptr(beta2), pc1[0].data_ptr(), pc1[1].data_ptr(),
                          pc1[2].data_ptr(), pc2[0].data_ptr(), pc2[1].data_ptr(),
                          pc2[2].data_ptr(), float(eps), v1.data_ptr(), v2.data_ptr())
        sh = _stream_handle(stream)
        ws = self.workspace(B, sh)
        _check(lib().spin_sph_residual_block_forward(self.p_in._h, po._h, B, C, xr.data_ptr(),
                                                     ctypes.byref(prm), yr.data_ptr(),
                                                     ws.data_ptr(), ws.numel(),
                                                     sh),
               "spin_sph_residual_block_forward")
        return (y, v1, v2) if variances else y
