"""The C ABI library loads and validates arguments on the host (no GPU needed).

Every symbol declared in include/gift.h must be exported by libgift.so.  The
error paths below return before any HIP call, so they run in a CPU-only
container; pointers are fake non-NULL addresses that are never dereferenced.
"""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gift.h")

gift = pytest.importorskip("paper_2607_07494_amd.gift")
LIB = gift.LIB
FAKE = ctypes.c_void_p(0x1000)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gift_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 16
    for name in names:
        assert hasattr(LIB, name), name
    assert LIB.gift_abi_version() == 1


def _err():
    return LIB.gift_last_error().decode()


def test_null_handles_are_einval():
    assert LIB.gift_encode(None, None, FAKE, 1, 4, 4, 0, 0, 0, None, FAKE, FAKE, None) == gift.EINVAL
    assert LIB.gift_reduce_local(None, FAKE, FAKE, 1, 4, 4, 0, 0, FAKE) == gift.EINVAL
    assert LIB.gift_decode(None, None, FAKE, 4, 4, FAKE) == gift.EINVAL
    assert LIB.gift_factor_update(None, None, FAKE, None, 8, 0, 1) == gift.EINVAL
    assert LIB.gift_ctx_create(None, None) == gift.EINVAL
    assert LIB.gift_ctx_set_statistics_event(None, None) == gift.EINVAL
    LIB.gift_ctx_destroy(None)
    LIB.gift_factor_destroy(None)


@pytest.fixture
def ctx():
    c = gift.Context(stream=0)   # creating a context makes no HIP call
    yield c
    c.close()


def test_encode_validation(ctx):
    h = ctx.handle
    enc = LIB.gift_encode
    assert enc(h, None, None, 1, 4, 4, 0, 0, 0, None, FAKE, FAKE, None) == gift.EINVAL
    assert enc(h, None, FAKE, 1, 4, 4, 0, 0, 0, None, None, FAKE, None) == gift.EINVAL
    assert enc(h, None, FAKE, 0, 4, 4, 0, 0, 0, None, FAKE, FAKE, None) == gift.ESHAPE
    assert "N must be" in _err()
    assert enc(h, None, FAKE, -3, 4, 4, 0, 0, 0, None, FAKE, FAKE, None) == gift.ESHAPE
    assert enc(h, None, FAKE, 1, 0, 4, 0, 0, 0, None, FAKE, FAKE, None) == gift.ESHAPE
    assert enc(h, None, FAKE, 1, 4, -1, 0, 0, 0, None, FAKE, FAKE, None) == gift.ESHAPE
    assert enc(h, None, FAKE, 1, 4, 4, -1, 0, 0, None, FAKE, FAKE, None) == gift.ESHAPE
    assert enc(h, None, FAKE, 1, 4, 4, 0, 0, 7, None, FAKE, FAKE, None) == gift.EINVAL
    assert "scale mode" in _err()
    assert enc(h, None, FAKE, 1, 2_000_000, 4, 0, 0, 0, None, FAKE, FAKE, None) == gift.ESHAPE


def test_create_chol_validation(ctx):
    h = ctx.handle
    out = ctypes.c_void_p()
    cr = LIB.gift_factor_create_chol
    assert cr(None, 8, 8, 0, 1, 1e-3, ctypes.byref(out)) == gift.EINVAL
    assert cr(h, 8, 8, 0, 4, 1e-3, ctypes.byref(out)) == gift.EINVAL
    assert cr(h, 8, 8, 0, 1, 0.0, ctypes.byref(out)) == gift.EINVAL
    assert "damping" in _err()
    assert cr(h, 8, 8, 0, 1, float("inf"), ctypes.byref(out)) == gift.EINVAL
    assert cr(h, 8, 8, -2, 1, 1e-3, ctypes.byref(out)) == gift.ESHAPE
    assert cr(h, 8, 9000, 0, 1, 1e-3, ctypes.byref(out)) == gift.ESHAPE   # full factor over 8192
    assert cr(h, 0, 8, 0, 1, 1e-3, ctypes.byref(out)) == gift.ESHAPE
    assert LIB.gift_factor_export_chol(h, None, 1, FAKE, FAKE) == gift.EINVAL
    assert LIB.gift_factor_import_chol(h, None, 1, FAKE, FAKE) == gift.EINVAL


def test_mxfp4_validation(ctx):
    h = ctx.handle
    enc = LIB.gift_encode_mxfp4
    assert enc(None, None, FAKE, 1, 4, 32, None, FAKE, FAKE, None) == gift.EINVAL
    assert enc(h, None, None, 1, 4, 32, None, FAKE, FAKE, None) == gift.EINVAL
    assert enc(h, None, FAKE, 1, 4, 48, None, FAKE, FAKE, None) == gift.ESHAPE
    assert "multiple of 32" in _err()
    assert enc(h, None, FAKE, 0, 4, 32, None, FAKE, FAKE, None) == gift.ESHAPE
    assert enc(h, None, ctypes.c_void_p(0x1004), 1, 4, 32, None, FAKE, FAKE, None) == gift.EINVAL
    red = LIB.gift_reduce_local_mxfp4
    assert red(h, FAKE, FAKE, 1, 4, 40, FAKE) == gift.ESHAPE
    assert red(h, None, FAKE, 1, 4, 32, FAKE) == gift.EINVAL
    assert red(h, FAKE, FAKE, 1, 4, 32, ctypes.c_void_p(0x1008)) == gift.EINVAL


def test_encode_hits_validation(ctx):
    h = ctx.handle
    enc = LIB.gift_encode_hits
    assert enc(h, None, FAKE, 1, 4, 4, 0, 0, 0, None, FAKE, FAKE, None, None) == gift.EINVAL
    assert "hits is NULL" in _err()
    assert enc(h, None, FAKE, 1, 4, 4, 0, 0, 0, None, FAKE, FAKE, None,
               ctypes.c_void_p(0x1002)) == gift.EINVAL
    assert "aligned" in _err()
    # with valid counters the encode's own checks apply
    assert enc(h, None, FAKE, 0, 4, 4, 0, 0, 0, None, FAKE, FAKE, None, FAKE) == gift.ESHAPE
    assert enc(h, None, None, 1, 4, 4, 0, 0, 0, None, FAKE, FAKE, None, FAKE) == gift.EINVAL


def test_reduce_and_decode_validation(ctx):
    h = ctx.handle
    assert LIB.gift_reduce_local(h, FAKE, FAKE, 0, 4, 4, 0, 0, FAKE) == gift.ESHAPE
    assert LIB.gift_reduce_local(h, None, FAKE, 2, 4, 4, 0, 0, FAKE) == gift.EINVAL
    assert LIB.gift_reduce_local(h, FAKE, FAKE, 2, 4, 4, 0, -2, FAKE) == gift.ESHAPE
    assert LIB.gift_decode(h, None, FAKE, 4, 4, FAKE) == gift.EINVAL
    assert "alias" in _err()
    assert LIB.gift_decode(h, None, FAKE, 0, 4, ctypes.c_void_p(0x2000)) == gift.ESHAPE


def test_factor_validation(ctx):
    h = ctx.handle
    out = ctypes.c_void_p()
    mk = LIB.gift_factor_create
    assert mk(h, 8, 8, 2, 0, 0.0, 0, ctypes.byref(out)) == gift.EINVAL       # sides
    assert mk(h, 8, 8, 2, 4, 0.0, 0, ctypes.byref(out)) == gift.EINVAL
    assert mk(h, 8, 8, 2, 1, -1.0, 0, ctypes.byref(out)) == gift.EINVAL      # damping
    assert mk(h, 8, 8, 2, 1, float("inf"), 0, ctypes.byref(out)) == gift.EINVAL
    assert mk(h, 8, 8, 9, 1, 0.0, 0, ctypes.byref(out)) == gift.ESHAPE       # rank > n
    assert mk(h, 4, 8, 5, 2, 0.0, 0, ctypes.byref(out)) == gift.ESHAPE       # rank > m
    assert mk(h, 8, 8, -1, 1, 0.0, 0, ctypes.byref(out)) == gift.ESHAPE
    assert mk(h, 0, 8, 1, 1, 0.0, 0, ctypes.byref(out)) == gift.ESHAPE
    assert mk(h, 8, 8, 1, 1, 0.0, 0, None) == gift.EINVAL


def test_statistics_validation(ctx):
    h = ctx.handle
    st = LIB.gift_statistics
    assert st(None, FAKE, 8, 8, 1, FAKE) == gift.EINVAL
    assert st(h, None, 8, 8, 1, FAKE) == gift.EINVAL
    assert st(h, FAKE, 8, 8, 1, None) == gift.EINVAL
    assert st(h, FAKE, 8, 8, 5, FAKE) == gift.EINVAL        # dtype
    assert st(h, FAKE, 0, 8, 1, FAKE) == gift.ESHAPE
    assert st(h, FAKE, 8, -4, 1, FAKE) == gift.ESHAPE
    assert st(h, FAKE, 8, 2_000_000, 1, FAKE) == gift.ESHAPE


def test_profile_api_host_side(ctx):
    h = ctx.handle
    n = ctypes.c_int64()
    ms = ctypes.c_double()
    assert LIB.gift_ctx_profile_read(h, 99, ctypes.byref(n), ctypes.byref(ms)) == gift.EINVAL
    assert LIB.gift_ctx_profile_select(None, 1) == gift.EINVAL
    assert LIB.gift_ctx_profile_select(h, 1 << 7) == gift.OK
    assert LIB.gift_ctx_profile_enable(h, 1) == gift.OK
    # nothing recorded yet: reading makes no HIP call
    assert LIB.gift_ctx_profile_read(h, 0, ctypes.byref(n), ctypes.byref(ms)) == gift.OK
    assert n.value == 0 and ms.value == 0.0


def test_scale_grid_shapes():
    assert gift.scale_grid(100, 300, 0, 128) == (1, 3)
    assert gift.scale_grid(100, 300, 30, 0) == (4, 1)
    assert gift.scale_grid(5, 7, 100, 100) == (1, 1)


def test_one_hip_runtime_in_the_process():
    """The library must share torch's HIP runtime: with two copies loaded,
    the second one reports no device on a GPU machine."""
    maps = open("/proc/self/maps").read().split("\n")
    hip = {line.split()[-1] for line in maps if "libamdhip64" in line}
    assert len(hip) == 1, hip


# ---------------------------------------------------------------- binding shape checks
# The wrappers check every tensor's shape before any pointer is passed: the
# library sizes its loops and buffer ranges from m, n, N and the factor's
# dims, so a short tensor would be an out-of-bounds device access.  These run
# on CPU tensors (the shape check comes before the device check) and a
# stand-in factor object, so nothing reaches the library.

def _fake_factor(m, n, rank=4, sides=gift.SIDE_INPUT):
    import types
    return types.SimpleNamespace(m=m, n=n, rank=rank, sides=sides, handle=FAKE)


def _z(*shape, dtype=None):
    import torch
    return torch.zeros(shape, dtype=dtype or torch.float32)


def test_binding_encode_shape_checks(ctx):
    import torch
    g = _z(2, 6, 8)
    u8 = torch.uint8
    good = dict(codes=_z(2, 6, 8, dtype=u8), scales=_z(2, 1, 1))
    bad_cases = [
        dict(good, codes=_z(2, 6, 7, dtype=u8)),
        dict(good, codes=_z(1, 6, 8, dtype=u8)),
        dict(good, scales=_z(2, 1, 2)),
        dict(good, ef=_z(2, 6, 4)),
        dict(good, transformed=_z(2, 5, 8)),
    ]
    for kw in bad_cases:
        with pytest.raises(ValueError, match="must have shape"):
            gift.encode(ctx, None, g, **kw)
    with pytest.raises(ValueError, match="must have shape"):   # per-block scale grid
        gift.encode(ctx, None, g, good["codes"], _z(2, 1, 1), 0, 4)
    with pytest.raises(ValueError, match="3-dimensional"):
        gift.encode(ctx, None, _z(6, 8), **good)
    with pytest.raises(ValueError, match="created for"):
        gift.encode(ctx, _fake_factor(6, 9), g, **good)
    with pytest.raises(ValueError, match="must have shape"):
        gift.encode(ctx, None, g, **good, hits=torch.zeros((3, 2), dtype=torch.int32))


def test_binding_reduce_decode_shape_checks(ctx):
    import torch
    codes = _z(3, 6, 8, dtype=torch.uint8)
    with pytest.raises(ValueError, match="scales"):
        gift.reduce_local(ctx, codes, _z(3, 1, 2), _z(6, 8))
    with pytest.raises(ValueError, match="scales"):
        gift.reduce_local(ctx, codes, _z(2, 1, 1), _z(6, 8))
    with pytest.raises(ValueError, match="mean"):
        gift.reduce_local(ctx, codes, _z(3, 1, 1), _z(6, 7))
    with pytest.raises(ValueError, match="out"):
        gift.decode(ctx, None, _z(6, 8), _z(8, 6))
    with pytest.raises(ValueError, match="created for"):
        gift.decode(ctx, _fake_factor(8, 6), _z(6, 8), _z(6, 8))
    with pytest.raises(ValueError, match="2-dimensional"):
        gift.decode(ctx, None, _z(1, 6, 8), _z(6, 8))


def test_binding_mxfp4_shape_checks(ctx):
    import torch
    u8 = torch.uint8
    g = _z(2, 4, 64)
    with pytest.raises(ValueError, match="codes"):
        gift.encode_mxfp4(ctx, None, g, _z(2, 4, 64, dtype=u8), _z(2, 4, 2, dtype=u8))
    with pytest.raises(ValueError, match="scales"):
        gift.encode_mxfp4(ctx, None, g, _z(2, 4, 32, dtype=u8), _z(2, 4, 1, dtype=u8))
    with pytest.raises(ValueError, match="ef"):
        gift.encode_mxfp4(ctx, None, g, _z(2, 4, 32, dtype=u8), _z(2, 4, 2, dtype=u8), ef=_z(2, 4, 32))
    with pytest.raises(ValueError, match="multiple of 32"):
        gift.encode_mxfp4(ctx, None, _z(2, 4, 48), _z(2, 4, 24, dtype=u8), _z(2, 4, 1, dtype=u8))
    with pytest.raises(ValueError, match="scales"):
        gift.reduce_local_mxfp4(ctx, _z(2, 4, 32, dtype=u8), _z(2, 4, 1, dtype=u8), _z(4, 64))
    with pytest.raises(ValueError, match="mean"):
        gift.reduce_local_mxfp4(ctx, _z(2, 4, 32, dtype=u8), _z(2, 4, 2, dtype=u8), _z(4, 32))


def test_binding_factor_input_shape_checks(ctx):
    import torch
    bf = torch.bfloat16
    fi = _fake_factor(6, 8, sides=gift.SIDE_INPUT)
    fb = _fake_factor(6, 8, sides=gift.SIDE_BOTH)
    # acts must be [T, n], out_grads [T, m]
    with pytest.raises(ValueError, match="acts"):
        gift._check_stats_inputs(fi, _z(16, 6, dtype=bf), None, 16)
    with pytest.raises(ValueError, match="out_grads"):
        gift._check_stats_inputs(fb, _z(16, 8, dtype=bf), _z(16, 8, dtype=bf), 16)
    with pytest.raises(ValueError, match="out_grads is required"):
        gift._check_stats_inputs(fb, _z(16, 8, dtype=bf), None, 16)
    gift._check_stats_inputs(fb, _z(16, 8, dtype=bf), _z(16, 6, dtype=bf), 16)   # fine
    with pytest.raises(ValueError, match="acts"):
        gift.factor_update_batch(ctx, [fi, fi], [_z(16, 8, dtype=bf), _z(16, 7, dtype=bf)], None)
    # Factor.update and import_ go through the same checks
    f = gift.Factor.__new__(gift.Factor)
    f.ctx, f.m, f.n, f.rank, f.sides, f._h = ctx, 6, 8, 4, gift.SIDE_BOTH, FAKE
    with pytest.raises(ValueError, match="out_grads"):
        f.update(acts=_z(16, 8, dtype=bf), out_grads=_z(16, 8, dtype=bf))
    with pytest.raises(ValueError, match="U must have shape"):
        f.import_(gift.SIDE_OUTPUT, _z(8, 4), _z(4), _z(4), _z(1))
    with pytest.raises(ValueError, match="c_inv"):
        f.import_(gift.SIDE_INPUT, _z(8, 4), _z(4), _z(3), _z(1))
    f._h = ctypes.c_void_p()   # nothing to destroy


def test_encode_noalloc_host_validation(ctx):
    h = ctx.handle
    enc = LIB.gift_encode_noalloc
    assert enc(h, None, None, 1, 4, 4, 0, 0, 0, None, FAKE, FAKE, None) == gift.EINVAL
    assert enc(h, None, FAKE, 0, 4, 4, 0, 0, 0, None, FAKE, FAKE, None) == gift.ESHAPE
    assert enc(h, None, FAKE, 1, 4, 4, 0, 0, 9, None, FAKE, FAKE, None) == gift.EINVAL
    # 1 x 1 scale blocks on 4 x 300 x 256: 78.6 MB of sub-slots, over the
    # fixed 64 MiB; rejected on the host before any HIP call
    assert enc(h, None, FAKE, 4, 300, 256, 1, 1, 0, None, FAKE, FAKE, None) == gift.ESHAPE
    assert "scratch" in _err() and str(64 * 1024 * 1024) in _err()
