"""Thin ctypes binding of ``libgift.so`` (the C ABI in ``include/gift.h``).

Argument marshalling only: every computation runs in the library's HIP
kernels.  Tensors are torch tensors on the GPU (device memory and streams are
all torch is used for); the wrappers check every tensor's shape against the
sizes the call is given (the library sizes its loops and buffer ranges from
those sizes, so a short tensor would be read or written out of bounds), then
dtype, device and contiguity, pass ``data_ptr()`` and raise
:class:`GiftError` with the library's message when a call fails.  A shape
mismatch raises ``ValueError`` before anything is enqueued.  There is no
fallback: if ``libgift.so`` is missing, importing this module raises.
"""

from __future__ import annotations

import ctypes
import os
import weakref

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libgift.so")

OK, EINVAL, ESHAPE, ENOMEM, EHIP, EUNSUPPORTED = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
SIDE_INPUT, SIDE_OUTPUT, SIDE_BOTH = 1, 2, 3
SCALE_LOCAL, SCALE_SHARED = 0, 1
KERNELS = {
    "amax": 0, "quant": 1, "project": 2, "update_amax": 3, "update_quant": 4,
    "update_store": 5, "reduce": 6, "syrk": 7, "factor": 8, "small": 9,
    "chol": 10, "eig": 11, "decode_project": 12, "chol_transform": 13, "mxfp4": 14,
}

_STATUS = {OK: "GIFT_OK", EINVAL: "GIFT_EINVAL", ESHAPE: "GIFT_ESHAPE", ENOMEM: "GIFT_ENOMEM",
           EHIP: "GIFT_EHIP", EUNSUPPORTED: "GIFT_EUNSUPPORTED"}


class GiftError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


def _load():
    # torch first: its bundled HIP runtime then satisfies libgift.so's
    # libamdhip64 dependency by soname.  Loaded the other way round, the
    # process holds two HIP runtimes and the second one sees no device.
    import torch  # noqa: F401

    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2607_07494_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U64, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float
    PP = ctypes.POINTER(ctypes.c_void_p)
    sigs = {
        "gift_abi_version": ([], I32),
        "gift_last_error": ([], ctypes.c_char_p),
        "gift_ctx_create": ([P, PP], I32),
        "gift_ctx_set_stream": ([P, P], I32),
        "gift_ctx_destroy": ([P], None),
        "gift_ctx_set_statistics_event": ([P, P], I32),
        "gift_ctx_profile_enable": ([P, I32], I32),
        "gift_ctx_profile_select": ([P, ctypes.c_uint32], I32),
        "gift_ctx_profile_read": ([P, I32, ctypes.POINTER(I64), ctypes.POINTER(ctypes.c_double)], I32),
        "gift_ctx_profile_reset": ([P], I32),
        "gift_factor_create": ([P, I64, I64, I32, I32, F, U64, PP], I32),
        "gift_factor_destroy": ([P], None),
        "gift_factor_update": ([P, P, P, P, I64, I32, I32], I32),
        "gift_statistics": ([P, P, I64, I64, I32, P], I32),
        "gift_factor_update_batch": ([P, I32, P, P, P, I64, I32, I32], I32),
        "gift_factor_export": ([P, P, I32, P, P, P, P], I32),
        "gift_factor_import": ([P, P, I32, P, P, P, P], I32),
        "gift_factor_create_chol": ([P, I64, I64, I32, I32, F, PP], I32),
        "gift_factor_export_chol": ([P, P, I32, P, P], I32),
        "gift_factor_import_chol": ([P, P, I32, P, P], I32),
        "gift_encode": ([P, P, P, I32, I64, I64, I32, I32, I32, P, P, P, P], I32),
        "gift_encode_hits": ([P, P, P, I32, I64, I64, I32, I32, I32, P, P, P, P, P], I32),
        "gift_encode_noalloc": ([P, P, P, I32, I64, I64, I32, I32, I32, P, P, P, P], I32),
        "gift_reduce_local": ([P, P, P, I32, I64, I64, I32, I32, P], I32),
        "gift_encode_mxfp4": ([P, P, P, I32, I64, I64, P, P, P, P], I32),
        "gift_reduce_local_mxfp4": ([P, P, P, I32, I64, I64, P], I32),
        "gift_decode": ([P, P, P, I64, I64, P], I32),
        "gift_decode_batch": ([P, I32, P, P, P, I64, I64], I32),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


LIB = _load()


def _check(status: int):
    if status != OK:
        raise GiftError(status, LIB.gift_last_error().decode(errors="replace"))


def exported_symbols():
    """Names declared by include/gift.h that this binding calls."""
    return sorted(n for n in dir(LIB) if n.startswith("gift_"))


def _ptr(t, dtype=None, name="tensor"):
    if t is None:
        return None
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, not {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _expect(t, shape, name):
    """Raise ValueError unless tensor ``t`` (may be None) has exactly ``shape``."""
    if t is None:
        return
    got = tuple(getattr(t, "shape", ()))
    if got != tuple(int(d) for d in shape):
        raise ValueError(f"{name} must have shape {tuple(int(d) for d in shape)}, not {got}")


def _dims(t, k, name):
    """The shape of ``t``, which must be a ``k``-dimensional tensor."""
    shape = tuple(getattr(t, "shape", ()))
    if len(shape) != k:
        raise ValueError(f"{name} must be {k}-dimensional, not of shape {shape}")
    return shape


def scale_grid(m: int, n: int, block_rows: int = 0, block_cols: int = 0):
    """``(nbr, nbc)``: scale-grid shape for allocating the scales output."""
    br = m if block_rows <= 0 else min(block_rows, m)
    bc = n if block_cols <= 0 else min(block_cols, n)
    return -(-m // br), -(-n // bc)


class Context:
    """A library context bound to one HIP stream (default: torch's current)."""

    def __init__(self, stream=None):
        if stream is None:
            import torch
            stream = torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else 0
        self._h = ctypes.c_void_p()
        self._factors = weakref.WeakSet()
        _check(LIB.gift_ctx_create(ctypes.c_void_p(int(stream)), ctypes.byref(self._h)))

    @property
    def handle(self):
        return self._h

    def set_stream(self, stream):
        _check(LIB.gift_ctx_set_stream(self._h, ctypes.c_void_p(int(stream))))

    def set_statistics_event(self, event):
        """Record ``event`` (a torch.cuda.Event, or None) after the statistics
        kernels of every later factor refresh on this context.  The context
        keeps a reference to the event so that it outlives the registration."""
        h = None
        self._stats_event = event
        if event is not None:
            import torch  # noqa: F401
            event.record()          # creates the underlying HIP event
            h = ctypes.c_void_p(event.cuda_event)
        _check(LIB.gift_ctx_set_statistics_event(self._h, h))

    def profile(self, enable: bool = True):
        _check(LIB.gift_ctx_profile_enable(self._h, 1 if enable else 0))

    def profile_select(self, families=None):
        """Time only these kernel families (names or ids; None = all)."""
        if families is None:
            mask = 0xFFFFFFFF
        else:
            mask = 0
            for k in families:
                mask |= 1 << (KERNELS[k] if isinstance(k, str) else int(k))
        _check(LIB.gift_ctx_profile_select(self._h, mask))

    def profile_read(self, kernel):
        k = KERNELS[kernel] if isinstance(kernel, str) else int(kernel)
        n = ctypes.c_int64()
        ms = ctypes.c_double()
        _check(LIB.gift_ctx_profile_read(self._h, k, ctypes.byref(n), ctypes.byref(ms)))
        return n.value, ms.value

    def profile_reset(self):
        _check(LIB.gift_ctx_profile_reset(self._h))

    def close(self):
        """Destroy the context; factors created on it are destroyed first."""
        if self._h:
            for f in list(self._factors):
                f.close()
            LIB.gift_ctx_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Factor:
    """Transform state of one m x n weight matrix (``gift_factor``)."""

    def __init__(self, ctx: Context, m: int, n: int, rank: int, sides: int = SIDE_INPUT,
                 damping: float = 1e-6, seed: int = 0):
        self.ctx, self.m, self.n, self.rank, self.sides = ctx, m, n, rank, sides
        self._h = ctypes.c_void_p()
        if not ctx.handle:
            raise GiftError(EINVAL, "the context is closed")
        _check(LIB.gift_factor_create(ctx.handle, m, n, rank, sides, damping, seed,
                                      ctypes.byref(self._h)))
        ctx._factors.add(self)

    @property
    def handle(self):
        return self._h

    def update(self, acts=None, out_grads=None, iters: int = 4):
        import torch
        x = acts if acts is not None else out_grads
        if x is None:
            raise ValueError("update needs acts and/or out_grads")
        if x.dtype == torch.float32:
            dt = F32
        elif x.dtype == torch.bfloat16:
            dt = BF16
        else:
            raise TypeError("statistics inputs must be float32 or bfloat16")
        T = x.shape[0]
        for t, nm in ((acts, "acts"), (out_grads, "out_grads")):
            if t is not None and (t.dim() != 2 or t.shape[0] != T or t.dtype != x.dtype):
                raise ValueError(f"{nm} must be [T, dim] with the common T and dtype")
        _check_stats_inputs(self, acts, out_grads, T)
        _check(LIB.gift_factor_update(self.ctx.handle, self._h, _ptr(acts, None, "acts"),
                                      _ptr(out_grads, None, "out_grads"), T, dt, iters))

    def export(self, side: int):
        import torch
        dim = self.n if side == SIDE_INPUT else self.m
        dev = torch.device("cuda", torch.cuda.current_device())
        U = torch.empty((dim, self.rank), dtype=torch.float32, device=dev)
        cf = torch.empty(self.rank, dtype=torch.float32, device=dev)
        ci = torch.empty(self.rank, dtype=torch.float32, device=dev)
        s2 = torch.empty(1, dtype=torch.float32, device=dev)
        _check(LIB.gift_factor_export(self.ctx.handle, self._h, side, _ptr(U), _ptr(cf), _ptr(ci),
                                      _ptr(s2)))
        return U, cf, ci, s2

    def import_(self, side: int, U, c_fwd, c_inv, sigma2):
        import torch
        f = torch.float32
        if side not in (SIDE_INPUT, SIDE_OUTPUT):
            raise ValueError("side must be SIDE_INPUT or SIDE_OUTPUT")
        dim = self.n if side == SIDE_INPUT else self.m
        _expect(U, (dim, self.rank), "U")
        _expect(c_fwd, (self.rank,), "c_fwd")
        _expect(c_inv, (self.rank,), "c_inv")
        _expect(sigma2, (1,), "sigma2")
        _check(LIB.gift_factor_import(self.ctx.handle, self._h, side, _ptr(U, f, "U"),
                                      _ptr(c_fwd, f, "c_fwd"), _ptr(c_inv, f, "c_inv"),
                                      _ptr(sigma2, f, "sigma2")))

    def close(self):
        if self._h:
            LIB.gift_factor_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class CholFactor(Factor):
    """Cholesky-form factor (``gift_factor_create_chol``): block 0 = full
    factor, 1 = diagonal, b = b x b diagonal blocks of A + delta I."""

    def __init__(self, ctx: Context, m: int, n: int, block: int = 0, sides: int = SIDE_INPUT,
                 damping: float = 1e-6):
        self.ctx, self.m, self.n, self.block, self.sides = ctx, m, n, block, sides
        self.rank = 0
        self._h = ctypes.c_void_p()
        if not ctx.handle:
            raise GiftError(EINVAL, "the context is closed")
        _check(LIB.gift_factor_create_chol(ctx.handle, m, n, block, sides, damping,
                                           ctypes.byref(self._h)))
        ctx._factors.add(self)

    def block_shape(self, side: int):
        """``(nblk, b_eff)`` of one side's stored blocks."""
        dim = self.n if side == SIDE_INPUT else self.m
        b = dim if self.block <= 0 or self.block >= dim else self.block
        return -(-dim // b), b

    def export(self, side: int):
        import torch
        nblk, b = self.block_shape(side)
        dev = torch.device("cuda", torch.cuda.current_device())
        R = torch.empty((nblk, b, b), dtype=torch.float32, device=dev)
        Ri = torch.empty((nblk, b, b), dtype=torch.float32, device=dev)
        _check(LIB.gift_factor_export_chol(self.ctx.handle, self._h, side, _ptr(R), _ptr(Ri)))
        return R, Ri

    def import_(self, side: int, R, Rinv):
        import torch
        nblk, b = self.block_shape(side)
        for t, nm in ((R, "R"), (Rinv, "Rinv")):
            if tuple(t.shape) != (nblk, b, b):
                raise ValueError(f"{nm} must have shape {(nblk, b, b)}")
        _check(LIB.gift_factor_import_chol(self.ctx.handle, self._h, side,
                                           _ptr(R, torch.float32, "R"),
                                           _ptr(Rinv, torch.float32, "Rinv")))


def _stats_dtype(x):
    import torch
    if x.dtype == torch.float32:
        return F32
    if x.dtype == torch.bfloat16:
        return BF16
    raise TypeError("statistics inputs must be float32 or bfloat16")


def _check_stats_inputs(factor, acts, out_grads, T):
    """acts [T, n] for a factor with the input side, out_grads [T, m] for one
    with the output side (the refresh reads T x dim values of each)."""
    sides = getattr(factor, "sides", 0)
    if sides & SIDE_INPUT:
        if acts is None:
            raise ValueError("acts is required for a factor with the input side")
        _expect(acts, (T, factor.n), "acts")
    if sides & SIDE_OUTPUT:
        if out_grads is None:
            raise ValueError("out_grads is required for a factor with the output side")
        _expect(out_grads, (T, factor.m), "out_grads")


def factor_update_batch(ctx: Context, factors, acts=None, out_grads=None, iters: int = 4):
    """``gift_factor_update_batch``: refresh many factors in one launch sequence.

    ``acts`` / ``out_grads`` are lists (one entry per factor, ``None`` where a
    factor lacks that side) of [T, dim] tensors with a common T and dtype.
    """
    count = len(factors)
    if count == 0:
        return
    acts = list(acts) if acts is not None else [None] * count
    out_grads = list(out_grads) if out_grads is not None else [None] * count
    if len(acts) != count or len(out_grads) != count:
        raise ValueError("acts / out_grads must have one entry per factor")
    tensors = [x for x in acts + out_grads if x is not None]
    if not tensors:
        raise ValueError("factor_update_batch needs statistics inputs")
    T, dt = tensors[0].shape[0], _stats_dtype(tensors[0])
    for x in tensors:
        if x.dim() != 2 or x.shape[0] != T or _stats_dtype(x) != dt:
            raise ValueError("statistics inputs must be [T, dim] with a common T and dtype")
    for f, a, g in zip(factors, acts, out_grads):
        _check_stats_inputs(f, a, g, T)
    arr = ctypes.c_void_p * count
    fa = arr(*[f.handle.value for f in factors])
    aa = arr(*[(_ptr(x).value if x is not None else None) for x in acts])
    ga = arr(*[(_ptr(x).value if x is not None else None) for x in out_grads])
    _check(LIB.gift_factor_update_batch(ctx.handle, count, fa, aa, ga, T, dt, iters))


def statistics(ctx: Context, x, A):
    """``gift_statistics``: x [T, dim] (float32 or bfloat16) -> A [dim, dim] = x^T x / T."""
    import torch
    if x.dim() != 2:
        raise ValueError("x must be [T, dim]")
    T, dim = x.shape
    if tuple(A.shape) != (dim, dim):
        raise ValueError("A must be [dim, dim]")
    _check(LIB.gift_statistics(ctx.handle, _ptr(x, None, "x"), T, dim, _stats_dtype(x),
                               _ptr(A, torch.float32, "A")))


def encode(ctx: Context, factor, grads, codes, scales, block_rows: int = 0, block_cols: int = 0,
           mode: int = SCALE_LOCAL, ef=None, transformed=None, hits=None):
    """``gift_encode``: grads [N, m, n] f32 -> codes [N, m, n] u8, scales [N, nbr, nbc] f32.

    With ``hits`` (an int32 [N, 2] tensor, bit pattern of the uint32 counters)
    this is ``gift_encode_hits``: the per-rank upper / lower boundary hits are
    added to it.
    """
    import torch
    N, m, n = _dims(grads, 3, "grads")
    if factor is not None and (factor.m, factor.n) != (m, n):
        raise ValueError(f"the factor was created for {factor.m} x {factor.n}, not {m} x {n}")
    _expect(codes, (N, m, n), "codes")
    _expect(scales, (N,) + scale_grid(m, n, block_rows, block_cols), "scales")
    _expect(ef, (N, m, n), "ef")
    _expect(transformed, (N, m, n), "transformed")
    _expect(hits, (N, 2), "hits")
    args = [ctx.handle, factor.handle if factor is not None else None,
            _ptr(grads, torch.float32, "grads"), N, m, n, block_rows, block_cols,
            mode, _ptr(ef, torch.float32, "ef"), _ptr(codes, torch.uint8, "codes"),
            _ptr(scales, torch.float32, "scales"), _ptr(transformed, torch.float32, "transformed")]
    if hits is None:
        _check(LIB.gift_encode(*args))
        return
    _check(LIB.gift_encode_hits(*args, _ptr(hits, torch.int32, "hits")))


NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024


def encode_noalloc(ctx: Context, factor, grads, codes, scales, block_rows: int = 0, block_cols: int = 0,
                   mode: int = SCALE_LOCAL, ef=None, transformed=None):
    """``gift_encode_noalloc``: :func:`encode` with its scratch in the library's
    fixed per-device array (no device allocation; calls on one device must
    not overlap)."""
    import torch
    N, m, n = _dims(grads, 3, "grads")
    if factor is not None and (factor.m, factor.n) != (m, n):
        raise ValueError(f"the factor was created for {factor.m} x {factor.n}, not {m} x {n}")
    _expect(codes, (N, m, n), "codes")
    _expect(scales, (N,) + scale_grid(m, n, block_rows, block_cols), "scales")
    _expect(ef, (N, m, n), "ef")
    _expect(transformed, (N, m, n), "transformed")
    _check(LIB.gift_encode_noalloc(ctx.handle, factor.handle if factor is not None else None,
                                   _ptr(grads, torch.float32, "grads"), N, m, n, block_rows, block_cols,
                                   mode, _ptr(ef, torch.float32, "ef"), _ptr(codes, torch.uint8, "codes"),
                                   _ptr(scales, torch.float32, "scales"),
                                   _ptr(transformed, torch.float32, "transformed")))


def reduce_local(ctx: Context, codes, scales, mean, block_rows: int = 0, block_cols: int = 0):
    """``gift_reduce_local``: codes [N, m, n], scales -> mean [m, n] f32."""
    import torch
    N, m, n = _dims(codes, 3, "codes")
    _expect(scales, (N,) + scale_grid(m, n, block_rows, block_cols), "scales")
    _expect(mean, (m, n), "mean")
    _check(LIB.gift_reduce_local(ctx.handle, _ptr(codes, torch.uint8, "codes"),
                                 _ptr(scales, torch.float32, "scales"), N, m, n, block_rows,
                                 block_cols, _ptr(mean, torch.float32, "mean")))


def encode_mxfp4(ctx: Context, factor, grads, codes, scales, ef=None, transformed=None):
    """``gift_encode_mxfp4``: grads [N, m, n] f32 -> codes [N, m, n/2] u8 (packed
    E2M1), scales [N, m, n/32] u8 (E8M0)."""
    import torch
    N, m, n = _dims(grads, 3, "grads")
    if factor is not None and (factor.m, factor.n) != (m, n):
        raise ValueError(f"the factor was created for {factor.m} x {factor.n}, not {m} x {n}")
    if n % 32:
        raise ValueError("MXFP4 needs n to be a multiple of 32")
    _expect(codes, (N, m, n // 2), "codes")
    _expect(scales, (N, m, n // 32), "scales")
    _expect(ef, (N, m, n), "ef")
    _expect(transformed, (N, m, n), "transformed")
    _check(LIB.gift_encode_mxfp4(ctx.handle, factor.handle if factor is not None else None,
                                 _ptr(grads, torch.float32, "grads"), N, m, n, _ptr(ef, torch.float32, "ef"),
                                 _ptr(codes, torch.uint8, "codes"), _ptr(scales, torch.uint8, "scales"),
                                 _ptr(transformed, torch.float32, "transformed")))


def reduce_local_mxfp4(ctx: Context, codes, scales, mean):
    """``gift_reduce_local_mxfp4``: codes [N, m, n/2], scales [N, m, n/32] -> mean [m, n] f32."""
    import torch
    N, m, half = _dims(codes, 3, "codes")
    if (2 * half) % 32:
        raise ValueError("MXFP4 needs n = 2 * codes.shape[2] to be a multiple of 32")
    _expect(scales, (N, m, 2 * half // 32), "scales")
    _expect(mean, (m, 2 * half), "mean")
    _check(LIB.gift_reduce_local_mxfp4(ctx.handle, _ptr(codes, torch.uint8, "codes"),
                                       _ptr(scales, torch.uint8, "scales"), N, m, 2 * half,
                                       _ptr(mean, torch.float32, "mean")))


def decode(ctx: Context, factor, mean, out):
    """``gift_decode``: inverse transform of the rank mean [m, n] f32 into out."""
    import torch
    m, n = _dims(mean, 2, "mean")
    if factor is not None and (factor.m, factor.n) != (m, n):
        raise ValueError(f"the factor was created for {factor.m} x {factor.n}, not {m} x {n}")
    _expect(out, (m, n), "out")
    _check(LIB.gift_decode(ctx.handle, factor.handle if factor is not None else None,
                           _ptr(mean, torch.float32, "mean"), m, n, _ptr(out, torch.float32, "out")))


def decode_batch(ctx: Context, factors, means, outs):
    """``gift_decode_batch``: ``outs[i] = decode(factors[i], means[i])`` for
    matrices of one shape, one launch per pass when the factors allow."""
    import torch
    count = len(means)
    if len(factors) != count or len(outs) != count:
        raise ValueError("factors, means and outs must have one entry per matrix")
    if count == 0:
        return
    m, n = _dims(means[0], 2, "means[0]")
    for i in range(count):
        _expect(means[i], (m, n), f"means[{i}]")
        _expect(outs[i], (m, n), f"outs[{i}]")
        f = factors[i]
        if f is not None and (f.m, f.n) != (m, n):
            raise ValueError(f"factor {i} was created for {f.m} x {f.n}, not {m} x {n}")
    arr = ctypes.c_void_p * count
    fa = arr(*[(f.handle.value if f is not None else None) for f in factors])
    ma = arr(*[_ptr(t, torch.float32, "means").value for t in means])
    oa = arr(*[_ptr(t, torch.float32, "outs").value for t in outs])
    _check(LIB.gift_decode_batch(ctx.handle, count, fa, ma, oa, m, n))
