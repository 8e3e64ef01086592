"""C ABI checks that need no GPU: the library loads, exports every function the
header declares, and rejects invalid arguments on the host before launching."""

import ctypes

import pytest

import paper_2410_17243_amd as infcl

# Fake but aligned device addresses: every call below must return before any launch.
A = 1 << 20


@pytest.fixture(scope="module")
def lib():
    return infcl.load_library()


def _single(lib, img=A, txt=A, b=64, d=512, dt=0, scale=A, lr=A, lc=A, aux=A, dloss=A, di=A, dtx=A, ds=A, ws=A,
            wsb=1 << 30):
    return lib.infcl_ablation_bwd_single(img, txt, b, d, dt, scale, lr, lc, aux, dloss, di, dtx, ds, ws, wsb, None)


def test_ablation_header_symbol_exported(lib):
    names = infcl.header_functions(infcl.ABLATION_HEADER_PATH)
    assert names == ["infcl_ablation_bwd_single"]
    assert hasattr(lib, names[0])
    assert _single(lib, img=None) == 1 and _single(lib, dtx=A + 4) == 1 and _single(lib, b=0) == 1
    assert _single(lib, dloss=A + 2) == 1 and _single(lib, ws=A + 16) == 1
    assert _single(lib, dt=2) == 2 and _single(lib, d=768) == 2 and _single(lib, d=128) == 2
    assert _single(lib, wsb=16) == 3


def test_exports_every_declared_function(lib):
    names = infcl.header_functions()
    assert set(names) == {"infcl_workspace_size", "infcl_fwd", "infcl_bwd", "infcl_status_str", "infcl_fwd_shard",
                          "infcl_fwd_shard_finish", "infcl_bwd_shard", "infcl_fwd_noalloc"}
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for st in range(5):
        assert isinstance(infcl.status_str(st), str) and infcl.status_str(st)
    assert infcl.status_str(99) == "unknown status"


def _ws(b, d, dt):
    out = ctypes.c_size_t(0)
    st = infcl.load_library().infcl_workspace_size(b, d, dt, ctypes.byref(out))
    return st, out.value


def test_workspace_size_is_linear_in_b():
    st1, w1 = _ws(1 << 20, 768, infcl.INFCL_BF16)
    st2, w2 = _ws(1 << 21, 768, infcl.INFCL_BF16)
    assert st1 == st2 == infcl.INFCL_OK
    assert 0 < w1 < 1024 * (1 << 20)         # under 1 KiB per sample
    assert abs(w2 - 2 * w1) < 1 << 16        # linear in b (up to alignment)
    assert _ws(1, 128, infcl.INFCL_BF16)[0] == infcl.INFCL_OK


@pytest.mark.parametrize("d,dt,per_sample", [
    # 16-bit inputs, resident-rows forward: 8 row and 32 column partial pairs
    # (8 B each), diagonal, base-2 diagonal reference, 2 base-2 log-sum-exp values
    (512, 0, (8 + 32) * 8 + 4 + 4 + 8), (768, 0, (8 + 32) * 8 + 4 + 4 + 8), (1024, 2, (8 + 32) * 8 + 4 + 4 + 8),
    # fp32 inputs, streamed forward: 32 row and 64 column partial pairs, no reference
    (512, 1, (32 + 64) * 8 + 4 + 8),
])
def test_workspace_bytes_per_sample(d, dt, per_sample):
    """The workspace holds what the launched grid writes, nothing more: the
    per-sample regions above plus per-workgroup partials (under 1 B/sample)."""
    b = 1 << 20
    st, w = _ws(b, d, dt)
    assert st == infcl.INFCL_OK
    assert per_sample * b <= w <= per_sample * b + b


@pytest.mark.parametrize("b,d,dt,expect", [
    (0, 512, 0, infcl.INFCL_ERR_INVALID), (-3, 512, 0, infcl.INFCL_ERR_INVALID), (16, 0, 0, infcl.INFCL_ERR_INVALID),
    (16, 512, 7, infcl.INFCL_ERR_INVALID), (16, 100, 0, infcl.INFCL_ERR_UNSUPPORTED),
    (16, 2048, 0, infcl.INFCL_ERR_UNSUPPORTED), (16, 1024, 1, infcl.INFCL_ERR_UNSUPPORTED),
    (16, 64, 0, infcl.INFCL_OK), (16, 64, 1, infcl.INFCL_OK), ((1 << 30) + 1, 512, 0, infcl.INFCL_ERR_UNSUPPORTED),
    (16, 512, 2, infcl.INFCL_OK), (16, 1024, 2, infcl.INFCL_OK), (16, 64, 2, infcl.INFCL_OK),
    (16, 100, 2, infcl.INFCL_ERR_UNSUPPORTED), (16, 512, 3, infcl.INFCL_ERR_INVALID),
    # 16-bit: any multiple of 8 up to 1024; f32: any multiple of 4 up to 512
    (16, 8, 0, infcl.INFCL_OK), (16, 1000, 0, infcl.INFCL_OK), (16, 1020, 0, infcl.INFCL_ERR_UNSUPPORTED),
    (16, 1032, 0, infcl.INFCL_ERR_UNSUPPORTED), (16, 4, 0, infcl.INFCL_ERR_UNSUPPORTED), (16, 4, 1, infcl.INFCL_OK),
    (16, 36, 1, infcl.INFCL_OK), (16, 514, 1, infcl.INFCL_ERR_UNSUPPORTED), (16, 516, 1, infcl.INFCL_ERR_UNSUPPORTED),
])
def test_workspace_size_validation(b, d, dt, expect):
    assert _ws(b, d, dt)[0] == expect


@pytest.mark.parametrize("d,dt,dk,es", [(8, 0, 128, 2), (72, 0, 128, 2), (200, 2, 256, 2), (1000, 0, 1024, 2),
                                         (4, 1, 64, 4), (100, 1, 128, 4)])
def test_workspace_of_padded_widths(d, dt, dk, es):
    """A width the sweeps are not built for runs at the next multiple of 128
    (16-bit) or 64 (f32): the workspace is that of the padded width plus the
    zero-padded copies of both inputs and the padded fp32 gradients."""
    b = 1 << 16
    st, w = _ws(b, d, dt)
    st_k, w_k = _ws(b, dk, dt)
    assert st == st_k == infcl.INFCL_OK
    extra = 2 * b * dk * es + 2 * b * dk * 4
    assert w_k + extra <= w <= w_k + extra + 1024


def test_workspace_size_null_out(lib):
    assert lib.infcl_workspace_size(16, 512, 0, None) == infcl.INFCL_ERR_INVALID




def _fwd(lib, img=A, txt=A, b=64, d=512, dt=0, scale=A, loss=A, loss64=A, lr=A, lc=A, aux=A, ws=A, wsb=1 << 30):
    return lib.infcl_fwd(img, txt, b, d, dt, scale, loss, loss64, lr, lc, aux, ws, wsb, None)


def _bwd(lib, img=A, txt=A, b=64, d=512, dt=0, scale=A, lr=A, lc=A, aux=A, dloss=A, di=A, dtx=A, gdt=1, ds=A, ws=A,
         wsb=1 << 30):
    return lib.infcl_bwd(img, txt, b, d, dt, scale, lr, lc, aux, dloss, di, dtx, gdt, ds, ws, wsb, None)


@pytest.mark.parametrize("kw,expect", [
    (dict(img=None), infcl.INFCL_ERR_INVALID), (dict(txt=A + 8), infcl.INFCL_ERR_INVALID),
    (dict(scale=None), infcl.INFCL_ERR_INVALID), (dict(loss=None), infcl.INFCL_ERR_INVALID),
    (dict(loss64=A + 4), infcl.INFCL_ERR_INVALID), (dict(lr=A + 4), infcl.INFCL_ERR_INVALID),
    (dict(aux=None), infcl.INFCL_ERR_INVALID), (dict(ws=A + 16), infcl.INFCL_ERR_INVALID),
    (dict(b=0), infcl.INFCL_ERR_INVALID), (dict(d=-1), infcl.INFCL_ERR_INVALID), (dict(dt=3), infcl.INFCL_ERR_INVALID),
    (dict(d=100), infcl.INFCL_ERR_UNSUPPORTED), (dict(wsb=16), infcl.INFCL_ERR_WORKSPACE),
    (dict(d=96, wsb=16), infcl.INFCL_ERR_WORKSPACE),
])
def test_fwd_validation(lib, kw, expect):
    assert _fwd(lib, **kw) == expect


def _fwd_noalloc(lib, img=A, txt=A, b=64, d=512, dt=0, scale=A, loss=A, loss64=A, lr=A, lc=A, aux=A):
    return lib.infcl_fwd_noalloc(img, txt, b, d, dt, scale, loss, loss64, lr, lc, aux, None)


@pytest.mark.parametrize("kw,expect", [
    (dict(img=None), infcl.INFCL_ERR_INVALID), (dict(txt=A + 8), infcl.INFCL_ERR_INVALID),
    (dict(scale=None), infcl.INFCL_ERR_INVALID), (dict(loss=None), infcl.INFCL_ERR_INVALID),
    (dict(loss64=A + 4), infcl.INFCL_ERR_INVALID), (dict(lc=A + 4), infcl.INFCL_ERR_INVALID),
    (dict(b=0), infcl.INFCL_ERR_INVALID), (dict(dt=3), infcl.INFCL_ERR_INVALID),
    (dict(d=100), infcl.INFCL_ERR_UNSUPPORTED),
    # the fixed 32 MiB scratch: 16-bit inputs need 336 B per sample, f32 780 B
    (dict(b=100000), infcl.INFCL_ERR_WORKSPACE), (dict(b=50000, d=256, dt=1), infcl.INFCL_ERR_WORKSPACE),
])
def test_fwd_noalloc_validation(lib, kw, expect):
    assert _fwd_noalloc(lib, **kw) == expect


@pytest.mark.parametrize("kw,expect", [
    (dict(di=None), infcl.INFCL_ERR_INVALID), (dict(dtx=A + 4), infcl.INFCL_ERR_INVALID),
    (dict(ds=None), infcl.INFCL_ERR_INVALID), (dict(dloss=A + 2), infcl.INFCL_ERR_INVALID),
    (dict(lc=None), infcl.INFCL_ERR_INVALID), (dict(b=-5), infcl.INFCL_ERR_INVALID),
    (dict(d=1536), infcl.INFCL_ERR_UNSUPPORTED), (dict(dt=1, d=768), infcl.INFCL_ERR_UNSUPPORTED),
    (dict(wsb=0), infcl.INFCL_ERR_WORKSPACE),
    # gradient types: f32, or the inputs' own 16-bit type
    (dict(gdt=5), infcl.INFCL_ERR_INVALID), (dict(gdt=-1), infcl.INFCL_ERR_INVALID),
    (dict(gdt=2), infcl.INFCL_ERR_UNSUPPORTED), (dict(dt=2, gdt=0), infcl.INFCL_ERR_UNSUPPORTED),
    (dict(dt=1, d=256, gdt=0), infcl.INFCL_ERR_UNSUPPORTED), (dict(dt=1, d=256, gdt=2), infcl.INFCL_ERR_UNSUPPORTED),
    (dict(gdt=0, wsb=0), infcl.INFCL_ERR_WORKSPACE), (dict(dt=2, gdt=2, wsb=0), infcl.INFCL_ERR_WORKSPACE),
])
def test_bwd_validation(lib, kw, expect):
    assert _bwd(lib, **kw) == expect


# ---------------------------------------------------------------- shard calls

def _fwd_shard(lib, b=1000, d=512, dt=0, r0=0, bs=1000, scale=A, cp=A, ws=A, wsb=1 << 30):
    return lib.infcl_fwd_shard(A, A, b, d, dt, r0, bs, scale, cp, ws, wsb, None)


def _finish(lib, b=1000, d=512, dt=0, r0=0, bs=1000, nparts=2, cps=A, scale=A, lr=A, lc=A, aux=A, lp=A, ws=A,
            wsb=1 << 30):
    return lib.infcl_fwd_shard_finish(b, d, dt, r0, bs, nparts, cps, scale, lr, lc, aux, lp, ws, wsb, None)


def _bwd_shard(lib, b=1000, d=512, dt=0, r0=0, bs=1000, ds=A, di=A, gdt=1, wsb=1 << 30):
    return lib.infcl_bwd_shard(A, A, b, d, dt, r0, bs, A, A, A, A, None, di, A, gdt, ds, A, wsb, None)


@pytest.mark.parametrize("kw,expect", [
    (dict(r0=16), infcl.INFCL_ERR_INVALID), (dict(r0=-32), infcl.INFCL_ERR_INVALID), (dict(bs=0), infcl.INFCL_ERR_INVALID),
    (dict(r0=992, bs=9), infcl.INFCL_ERR_INVALID), (dict(cp=A + 4), infcl.INFCL_ERR_INVALID),
    (dict(cp=None), infcl.INFCL_ERR_INVALID), (dict(d=100), infcl.INFCL_ERR_UNSUPPORTED),
    (dict(wsb=16), infcl.INFCL_ERR_WORKSPACE),
])
def test_fwd_shard_validation(lib, kw, expect):
    assert _fwd_shard(lib, **kw) == expect


@pytest.mark.parametrize("kw,expect", [
    (dict(nparts=0), infcl.INFCL_ERR_INVALID), (dict(r0=33), infcl.INFCL_ERR_INVALID), (dict(lp=A + 4), infcl.INFCL_ERR_INVALID),
    (dict(cps=None), infcl.INFCL_ERR_INVALID), (dict(bs=1001), infcl.INFCL_ERR_INVALID),
    (dict(wsb=16), infcl.INFCL_ERR_WORKSPACE),
])
def test_fwd_shard_finish_validation(lib, kw, expect):
    assert _finish(lib, **kw) == expect


@pytest.mark.parametrize("kw,expect", [
    (dict(r0=8), infcl.INFCL_ERR_INVALID), (dict(ds=A + 4), infcl.INFCL_ERR_INVALID), (dict(di=None), infcl.INFCL_ERR_INVALID),
    (dict(r0=960, bs=64), infcl.INFCL_ERR_INVALID), (dict(dt=1, d=1024), infcl.INFCL_ERR_UNSUPPORTED),
    (dict(wsb=16), infcl.INFCL_ERR_WORKSPACE),
])
def test_bwd_shard_validation(lib, kw, expect):
    assert _bwd_shard(lib, **kw) == expect


def test_shard_bounds():
    from paper_2410_17243_amd.shards import shard_bounds
    for b, n in [(1, 1), (100, 3), (1000, 4), (32768, 8), (4097, 7)]:
        bd = shard_bounds(b, n)
        assert bd[0][0] == 0 and sum(bs for _, bs in bd) == b
        assert all(r0 % 32 == 0 and bs >= 1 for r0, bs in bd)
        assert all(bd[k][0] + bd[k][1] == bd[k + 1][0] for k in range(len(bd) - 1))
        assert len(bd) <= n
