"""ctypes binding for libbakron.so -- argument marshalling only.

Every step of the solver runs in the library's HIP kernels; torch is used only
for device memory (``data_ptr()``) and the current HIP stream.  If the library
has not been built, every call raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbakron.so")

BAKRON_OK, BAKRON_EINVAL, BAKRON_ENOTSPD, BAKRON_ENOMEM, BAKRON_EHIP = range(5)

EXPORTED = ("bakron_factor", "bakron_solve", "bakron_solve_debug", "bakron_factors_free",
            "bakron_status_string", "bakron_factors_error", "bakron_last_error",
            "bakron_factor_export", "bakron_profile_enable", "bakron_profile_read",
            "bakron_solve_check", "bakron_solve_antidiag", "bakron_gram",
            "bakron_sample_weights", "bakron_kron_factors", "bakron_mlp_local_factors",
            "bakron_mse_scales", "bakron_factor_blockdiag", "bakron_quadform_weights",
            "bakron_kron_factors_iter", "bakron_mlp_local_factors_iter", "bakron_solve_noalloc")

ALPHABETS = {"sym": 0, "asym": 1}

BAKRON_KFAC, BAKRON_SHAMPOO = 0, 1
STYLES = {"kfac": BAKRON_KFAC, "shampoo": BAKRON_SHAMPOO}

_lib = None


class BakronError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{status_string(status) if _lib else status}: {msg}")
        self.status = status


class _Quantizer(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("scale", ctypes.c_void_p), ("alphabet", ctypes.c_int32),
                ("group_size", ctypes.c_int32), ("col_scale", ctypes.c_void_p)]


class KernelStat(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double), ("launches", ctypes.c_int64), ("flops", ctypes.c_double),
                ("mfma_flops", ctypes.c_double)]

    def as_dict(self):
        return dict(ms=self.ms, launches=self.launches, flops=self.flops,
                    mfma_flops=self.mfma_flops)


def load(path: str = LIB_PATH):
    """Load libbakron.so (raises if it is missing: there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(path)
    vp = ctypes.c_void_p
    lib.bakron_factor.restype = ctypes.c_int
    lib.bakron_factor.argtypes = [vp, ctypes.c_int64, vp, ctypes.c_int64, ctypes.c_float, vp,
                                  ctypes.POINTER(vp)]
    lib.bakron_solve.restype = ctypes.c_int
    lib.bakron_solve.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, vp, _Quantizer, vp, vp, vp]
    lib.bakron_solve_debug.restype = ctypes.c_int
    lib.bakron_solve_debug.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, vp, _Quantizer, vp, vp,
                                       vp, vp]
    lib.bakron_factors_free.restype = None
    lib.bakron_factors_free.argtypes = [vp]
    lib.bakron_status_string.restype = ctypes.c_char_p
    lib.bakron_status_string.argtypes = [ctypes.c_int]
    lib.bakron_factors_error.restype = ctypes.c_char_p
    lib.bakron_factors_error.argtypes = [vp]
    lib.bakron_last_error.restype = ctypes.c_char_p
    lib.bakron_last_error.argtypes = []
    lib.bakron_factor_export.restype = ctypes.c_int
    lib.bakron_factor_export.argtypes = [vp, ctypes.c_int, vp, vp]
    lib.bakron_profile_enable.restype = ctypes.c_int
    lib.bakron_profile_enable.argtypes = [vp, ctypes.c_int]
    lib.bakron_profile_read.restype = ctypes.c_int
    lib.bakron_profile_read.argtypes = [vp, ctypes.POINTER(KernelStat), ctypes.c_int]
    lib.bakron_solve_antidiag.restype = ctypes.c_int
    lib.bakron_solve_antidiag.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, vp, _Quantizer, vp, vp,
                                          vp, vp]
    lib.bakron_solve_noalloc.restype = ctypes.c_int
    lib.bakron_solve_noalloc.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, vp, _Quantizer, vp, vp,
                                         vp]
    lib.bakron_solve_check.restype = ctypes.c_int
    lib.bakron_solve_check.argtypes = [vp, vp, ctypes.POINTER(ctypes.c_int32)]
    i64, szp = ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)
    lib.bakron_mse_scales.restype = ctypes.c_int
    lib.bakron_mse_scales.argtypes = [vp, i64, i64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_int32, ctypes.c_double, vp, vp]
    lib.bakron_factor_blockdiag.restype = ctypes.c_int
    lib.bakron_factor_blockdiag.argtypes = [vp, i64, vp, i64, i64, ctypes.c_float, vp,
                                            ctypes.POINTER(vp)]
    lib.bakron_gram.restype = ctypes.c_int
    lib.bakron_gram.argtypes = [vp, i64, i64, vp, ctypes.c_float, vp, vp, vp, szp, vp]
    lib.bakron_sample_weights.restype = ctypes.c_int
    lib.bakron_sample_weights.argtypes = [vp, i64, i64, vp, vp, vp]
    lib.bakron_kron_factors.restype = ctypes.c_int
    lib.bakron_kron_factors.argtypes = [vp, vp, i64, i64, i64, ctypes.c_int32, vp, vp, vp, szp, vp]
    lib.bakron_quadform_weights.restype = ctypes.c_int
    lib.bakron_quadform_weights.argtypes = [vp, i64, i64, vp, vp, vp, szp, vp]
    lib.bakron_kron_factors_iter.restype = ctypes.c_int
    lib.bakron_kron_factors_iter.argtypes = [vp, vp, i64, i64, i64, ctypes.c_int32, vp, vp, vp,
                                             szp, vp]
    lib.bakron_mlp_local_factors_iter.restype = ctypes.c_int
    lib.bakron_mlp_local_factors_iter.argtypes = [vp, vp, vp, i64, i64, i64, ctypes.c_int32, vp,
                                                  vp, vp, szp, vp]
    lib.bakron_mlp_local_factors.restype = ctypes.c_int
    lib.bakron_mlp_local_factors.argtypes = [vp, vp, vp, i64, i64, i64, ctypes.c_int32, vp, vp, vp,
                                             szp, vp]
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().bakron_status_string(int(status)).decode()


def _stream(torch, device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check_dev(t, name, dtype):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


class Factors:
    """Owns a bakron_factors handle (normalised L^A, L^B in fp32 on the device)."""

    def __init__(self, handle: int, n: int, m: int | None, device):
        self._h = ctypes.c_void_p(handle)
        self.n = n
        self.m = m
        self.device = device

    @property
    def handle(self):
        return self._h

    def error(self) -> str:
        return load().bakron_factors_error(self._h).decode()

    def export(self, which: str):
        """Dense fp32 copy of L^A ('A') or L^B ('B') for testing."""
        import torch
        d = self.n if which == "A" else (self.m or 0)
        out = torch.empty((max(d, 1), max(d, 1)), dtype=torch.float32, device=self.device)
        st = load().bakron_factor_export(self._h, 0 if which == "A" else 1,
                                         ctypes.c_void_p(out.data_ptr()),
                                         _stream(torch, self.device))
        if st != BAKRON_OK:
            raise BakronError(st, self.error())
        return out

    def profile(self, on: bool = True):
        """Enable/disable per-launch event timing (measurement hook)."""
        st = load().bakron_profile_enable(self._h, 1 if on else 0)
        if st != BAKRON_OK:
            raise BakronError(st, self.error())

    PROFILE_CLASSES = ("prep", "segment", "node")

    def profile_read(self):
        """Per-class stats of the last profiled solve (stream must be synchronised)."""
        arr = (KernelStat * len(self.PROFILE_CLASSES))()
        st = load().bakron_profile_read(self._h, arr, len(self.PROFILE_CLASSES))
        if st != BAKRON_OK:
            raise BakronError(st, self.error())
        return {k: arr[i].as_dict() for i, k in enumerate(self.PROFILE_CLASSES)}

    def check(self) -> bool:
        """True if every solve on this handle since the last check completed
        all of its ordered waits (synchronises the current stream; a give-up
        record is sticky on the device until this call clears it)."""
        import torch
        failed = ctypes.c_int32(0)
        st = load().bakron_solve_check(self._h, _stream(torch, self.device), ctypes.byref(failed))
        if st != BAKRON_OK:
            raise BakronError(st, self.error())
        return failed.value == 0

    def close(self):
        if self._h is not None and self._h.value:
            load().bakron_factors_free(self._h)
            self._h = ctypes.c_void_p(0)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def factor(A, B, damp: float) -> Factors:
    """bakron_factor(A, B, damp) on the current stream.  B=None means I."""
    import torch
    lib = load()
    _check_dev(A, "A", torch.float32)
    n = A.shape[0]
    if A.shape != (n, n):
        raise ValueError("A must be square")
    m = 0
    bptr = None
    if B is not None:
        _check_dev(B, "B", torch.float32)
        m = B.shape[0]
        if B.shape != (m, m):
            raise ValueError("B must be square")
        bptr = ctypes.c_void_p(B.data_ptr())
    h = ctypes.c_void_p(0)
    st = lib.bakron_factor(ctypes.c_void_p(A.data_ptr()), n, bptr, m, float(damp),
                           _stream(torch, A.device), ctypes.byref(h))
    if st != BAKRON_OK:
        raise BakronError(st, lib.bakron_last_error().decode())
    return Factors(h.value, n, m if B is not None else None, A.device)


def _quantizer(bits, scale, m, n, alphabet, group_size, col_scale):
    """bakron_quantizer for per-row (m) or per-(row, group) (m x ceil(n/g))
    scales, optional per-column factors, alphabet "sym" or "asym"."""
    import torch
    _check_dev(scale, "scale", torch.float32)
    g = int(group_size)
    if g < 0:
        raise ValueError("group_size must be >= 0")
    want = m * (-(-n // g)) if g > 0 else m
    if scale.numel() != want:
        raise ValueError(f"scale must have {want} entries")
    cp = None
    if col_scale is not None:
        _check_dev(col_scale, "col_scale", torch.float32)
        if col_scale.numel() != n:
            raise ValueError("col_scale must have n entries")
        cp = col_scale.data_ptr()
    if alphabet not in ALPHABETS:
        raise ValueError(f"alphabet must be one of {sorted(ALPHABETS)}")
    return _Quantizer(int(bits), ctypes.c_void_p(scale.data_ptr()).value, ALPHABETS[alphabet], g,
                      cp)


def solve(W, f: Factors, bits: int, scale, codes=None, V=None, pre=None, debug: bool = False,
          alphabet: str = "sym", group_size: int = 0, col_scale=None):
    """bakron_solve / bakron_solve_debug on the current stream.

    scale: m per-row scales, or m x ceil(n / group_size) with group_size > 0;
    col_scale: None or n per-column factors; alphabet "sym" or "asym".
    Returns (codes int8, V fp32) or (codes, V, pre) when debug=True.
    """
    import torch
    lib = load()
    _check_dev(W, "W", torch.float32)
    m, n = W.shape
    q = _quantizer(bits, scale, m, n, alphabet, group_size, col_scale)
    if codes is None:
        codes = torch.empty((m, n), dtype=torch.int8, device=W.device)
    if V is None:
        V = torch.empty((m, n), dtype=torch.float32, device=W.device)
    _check_dev(codes, "codes", torch.int8)
    _check_dev(V, "V", torch.float32)
    s = _stream(torch, W.device)
    if debug:
        if pre is None:
            pre = torch.empty((m, n), dtype=torch.float32, device=W.device)
        _check_dev(pre, "pre", torch.float32)
        st = lib.bakron_solve_debug(ctypes.c_void_p(W.data_ptr()), m, n, f.handle, q,
                                    ctypes.c_void_p(codes.data_ptr()), ctypes.c_void_p(V.data_ptr()),
                                    ctypes.c_void_p(pre.data_ptr()), s)
    else:
        st = lib.bakron_solve(ctypes.c_void_p(W.data_ptr()), m, n, f.handle, q,
                              ctypes.c_void_p(codes.data_ptr()), ctypes.c_void_p(V.data_ptr()), s)
    if st != BAKRON_OK:
        raise BakronError(st, f.error())
    return (codes, V, pre) if debug else (codes, V)


def solve_noalloc(W, f: Factors, bits: int, scale, codes=None, V=None, alphabet: str = "sym",
                  group_size: int = 0, col_scale=None):
    """bakron_solve_noalloc on the current stream: the solve with its workspace
    in the library's static per-device scratch (no device allocation).
    Quantiser arguments as :func:`solve`; codes and V are allocated here by
    torch only if not given.  Returns (codes int8, V fp32)."""
    import torch
    lib = load()
    _check_dev(W, "W", torch.float32)
    m, n = W.shape
    q = _quantizer(bits, scale, m, n, alphabet, group_size, col_scale)
    if codes is None:
        codes = torch.empty((m, n), dtype=torch.int8, device=W.device)
    if V is None:
        V = torch.empty((m, n), dtype=torch.float32, device=W.device)
    _check_dev(codes, "codes", torch.int8)
    _check_dev(V, "V", torch.float32)
    st = lib.bakron_solve_noalloc(ctypes.c_void_p(W.data_ptr()), m, n, f.handle, q,
                                  ctypes.c_void_p(codes.data_ptr()), ctypes.c_void_p(V.data_ptr()),
                                  _stream(torch, W.device))
    if st != BAKRON_OK:
        raise BakronError(st, f.error())
    return codes, V


def solve_antidiag(W, f: Factors, bits: int, scale, codes=None, V=None, pre=None,
                   alphabet: str = "sym", group_size: int = 0, col_scale=None):
    """bakron_solve_antidiag (BaKron-antidiagonal, Alg. 3) on the current stream.

    Quantiser arguments as :func:`solve`.
    Returns (codes int8, V fp32), or (codes, V, pre) when a pre buffer is given.
    """
    import torch
    lib = load()
    _check_dev(W, "W", torch.float32)
    m, n = W.shape
    q = _quantizer(bits, scale, m, n, alphabet, group_size, col_scale)
    if codes is None:
        codes = torch.empty((m, n), dtype=torch.int8, device=W.device)
    if V is None:
        V = torch.empty((m, n), dtype=torch.float32, device=W.device)
    _check_dev(codes, "codes", torch.int8)
    _check_dev(V, "V", torch.float32)
    if pre is not None:
        _check_dev(pre, "pre", torch.float32)
    st = lib.bakron_solve_antidiag(ctypes.c_void_p(W.data_ptr()), m, n, f.handle, q,
                                   ctypes.c_void_p(codes.data_ptr()), ctypes.c_void_p(V.data_ptr()),
                                   ctypes.c_void_p(pre.data_ptr() if pre is not None else None),
                                   _stream(torch, W.device))
    if st != BAKRON_OK:
        raise BakronError(st, f.error())
    return (codes, V) if pre is None else (codes, V, pre)


def factor_blockdiag(A, B_blocks, damp: float) -> Factors:
    """bakron_factor_blockdiag: B = blockdiag of B_blocks (nblocks x hb x hb)."""
    import torch
    lib = load()
    _check_dev(A, "A", torch.float32)
    _check_dev(B_blocks, "B_blocks", torch.float32)
    n = A.shape[0]
    if A.shape != (n, n) or B_blocks.dim() != 3 or B_blocks.shape[1] != B_blocks.shape[2]:
        raise ValueError("A must be n x n and B_blocks nblocks x hb x hb")
    nb, hb = B_blocks.shape[0], B_blocks.shape[1]
    h = ctypes.c_void_p(0)
    st = lib.bakron_factor_blockdiag(ctypes.c_void_p(A.data_ptr()), n,
                                     ctypes.c_void_p(B_blocks.data_ptr()), nb, hb, float(damp),
                                     _stream(torch, A.device), ctypes.byref(h))
    if st != BAKRON_OK:
        raise BakronError(st, lib.bakron_last_error().decode())
    return Factors(h.value, n, nb * hb, A.device)


def mse_scales(W, bits: int, alphabet: str = "sym", group_size: int = 0, grid: int = 100,
               maxshrink: float = 0.5):
    """bakron_mse_scales on the current stream: m scales, or m x ceil(n/g)."""
    import torch
    lib = load()
    _check_dev(W, "W", torch.float32)
    m, n = W.shape
    g = int(group_size)
    out = torch.empty((m, -(-n // g)) if g > 0 else (m,), dtype=torch.float32, device=W.device)
    st = lib.bakron_mse_scales(ctypes.c_void_p(W.data_ptr()), m, n, int(bits),
                               ALPHABETS[alphabet], g, int(grid), float(maxshrink),
                               ctypes.c_void_p(out.data_ptr()), _stream(torch, W.device))
    if st != BAKRON_OK:
        raise BakronError(st, lib.bakron_last_error().decode())
    return out


# ---------------------------------------------------------------- factor construction
def _ptr(t):
    return ctypes.c_void_p(t.data_ptr() if t is not None else None)


def _raise_last(st):
    if st != BAKRON_OK:
        raise BakronError(st, load().bakron_last_error().decode())


def _with_workspace(call, device):
    """Run a workspace-protocol entry point: query the size, allocate a torch
    buffer (256-byte aligned by the caching allocator), then call."""
    import torch
    need = ctypes.c_size_t(0)
    _raise_last(call(ctypes.c_void_p(None), ctypes.byref(need)))
    work = torch.empty(max(int(need.value), 256), dtype=torch.uint8, device=device)
    if work.data_ptr() % 256:
        raise RuntimeError("workspace is not 256-byte aligned")
    size = ctypes.c_size_t(work.numel())
    _raise_last(call(_ptr(work), ctypes.byref(size)))
    return work


def gram(X, w=None, s: float = 1.0, M=None, C=None, work=None):
    """bakron_gram: C = s * (X^T diag(w) X) (.) M on the current stream.
    X: N x d fp32; w: N or None; M: d x d or None (may be C itself)."""
    import torch
    lib = load()
    _check_dev(X, "X", torch.float32)
    N, d = X.shape
    for t, name, shape in ((w, "w", (N,)), (M, "M", (d, d))):
        if t is not None:
            _check_dev(t, name, torch.float32)
            if tuple(t.shape) != shape:
                raise ValueError(f"{name} must have shape {shape}")
    if C is None:
        C = torch.empty((d, d), dtype=torch.float32, device=X.device)
    _check_dev(C, "C", torch.float32)
    if tuple(C.shape) != (d, d):
        raise ValueError("C must be d x d")
    st = _stream(torch, X.device)

    def call(wk, nbytes):
        return lib.bakron_gram(_ptr(X), N, d, _ptr(w), float(s), _ptr(M), _ptr(C), wk, nbytes, st)
    if work is None:
        _with_workspace(call, X.device)
    else:
        size = ctypes.c_size_t(work.numel() * work.element_size())
        _raise_last(call(_ptr(work), ctypes.byref(size)))
    return C


def gram_workspace_bytes(N: int, d: int) -> int:
    """Workspace bytes bakron_gram needs for an N x d sample matrix on the
    current device."""
    need = ctypes.c_size_t(0)
    _raise_last(load().bakron_gram(None, N, d, None, 1.0, None, None, None, ctypes.byref(need),
                                   None))
    return int(need.value)


def sample_weights(X, c=None, w=None):
    """bakron_sample_weights: w_k = sum_i c_i X_ki^2 on the current stream."""
    import torch
    lib = load()
    _check_dev(X, "X", torch.float32)
    N, d = X.shape
    if c is not None:
        _check_dev(c, "c", torch.float32)
        if c.numel() != d:
            raise ValueError("c must have d entries")
    if w is None:
        w = torch.empty((N,), dtype=torch.float32, device=X.device)
    _check_dev(w, "w", torch.float32)
    _raise_last(lib.bakron_sample_weights(_ptr(X), N, d, _ptr(c), _ptr(w),
                                          _stream(torch, X.device)))
    return w


def quadform_weights(X, M, w=None):
    """bakron_quadform_weights: w_k = x_k^T M x_k (M symmetric) on the current stream."""
    import torch
    lib = load()
    _check_dev(X, "X", torch.float32)
    _check_dev(M, "M", torch.float32)
    N, d = X.shape
    if tuple(M.shape) != (d, d):
        raise ValueError("M must be d x d")
    if w is None:
        w = torch.empty((N,), dtype=torch.float32, device=X.device)
    _check_dev(w, "w", torch.float32)
    st = _stream(torch, X.device)
    _with_workspace(lambda wk, nb: lib.bakron_quadform_weights(_ptr(X), N, d, _ptr(M), _ptr(w), wk,
                                                               nb, st), X.device)
    return w


def kron_factors(a, b, style: str = "kfac", iters: int = 1):
    """bakron_kron_factors (iters = 1) or bakron_kron_factors_iter (Shampoo
    with `iters` power steps): (A, B) of a global Hessian from paired vector
    samples a (N x n) and b (N x m) on the current stream."""
    import torch
    lib = load()
    _check_dev(a, "a", torch.float32)
    _check_dev(b, "b", torch.float32)
    N, n = a.shape
    if b.shape[0] != N:
        raise ValueError("a and b need the same number of samples")
    m = b.shape[1]
    A = torch.empty((n, n), dtype=torch.float32, device=a.device)
    B = torch.empty((m, m), dtype=torch.float32, device=a.device)
    st = _stream(torch, a.device)
    if iters != 1:
        if style != "shampoo":
            raise ValueError("power steps need style='shampoo'")
        _with_workspace(lambda wk, nb: lib.bakron_kron_factors_iter(
            _ptr(a), _ptr(b), N, n, m, int(iters), _ptr(A), _ptr(B), wk, nb, st), a.device)
        return A, B
    _with_workspace(lambda wk, nb: lib.bakron_kron_factors(_ptr(a), _ptr(b), N, n, m, STYLES[style],
                                                           _ptr(A), _ptr(B), wk, nb, st), a.device)
    return A, B


def mlp_local_factors(x, g, D, style: str = "kfac", iters: int = 1):
    """bakron_mlp_local_factors: (A, B) of the MLP-local Hessian from inputs x
    (N x dm), features g or f (N x dff) and W_down D (dm x dff)."""
    import torch
    lib = load()
    for t, name in ((x, "x"), (g, "g"), (D, "D")):
        _check_dev(t, name, torch.float32)
    N, dm = x.shape
    dff = g.shape[1]
    if g.shape[0] != N or tuple(D.shape) != (dm, dff):
        raise ValueError("shapes must be x: N x dm, g: N x dff, D: dm x dff")
    A = torch.empty((dm, dm), dtype=torch.float32, device=x.device)
    B = torch.empty((dff, dff), dtype=torch.float32, device=x.device)
    st = _stream(torch, x.device)
    if iters != 1:
        if style != "shampoo":
            raise ValueError("power steps need style='shampoo'")
        _with_workspace(lambda wk, nb: lib.bakron_mlp_local_factors_iter(
            _ptr(x), _ptr(g), _ptr(D), N, dm, dff, int(iters), _ptr(A), _ptr(B), wk, nb, st),
            x.device)
        return A, B
    _with_workspace(lambda wk, nb: lib.bakron_mlp_local_factors(_ptr(x), _ptr(g), _ptr(D), N, dm,
                                                                dff, STYLES[style], _ptr(A),
                                                                _ptr(B), wk, nb, st), x.device)
    return A, B
