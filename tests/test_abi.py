"""C-ABI boundary tests that need no GPU: the library loads, exports every
function include/vcheck.h declares, and rejects every malformed argument on
the host before anything is enqueued (these paths make no HIP call; data
pointers here are never dereferenced)."""
import ctypes
import os
import re

import pytest

from paper_2608_02712_amd import vcheck as vc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vcheck.h")

FAKE = 0x100000  # 16-byte aligned stand-in device address, never touched


@pytest.fixture(scope="module")
def L():
    return vc.lib()


def desc(dtype=vc.VC_F32, shape=(4, 5), data=FAKE):
    d = vc.VcTensor()
    d.data = data
    d.dtype = dtype
    d.ndim = len(shape)
    for i, s in enumerate(shape[:8]):
        d.shape[i] = s
    return d


def tol(atol=1e-5, rtol=1e-5, equal_nan=0):
    t = vc.VcTol()
    t.atol, t.rtol, t.equal_nan = atol, rtol, equal_nan
    return t


def test_exports_every_declared_symbol(L):
    text = open(HEADER).read()
    names = set(re.findall(r"\b(vcheck_\w+)\s*\(", text))
    assert {"vcheck_compare", "vcheck_localize", "vcheck_integrity", "vcheck_sweep",
            "vcheck_workspace_bytes", "vcheck_tile_count", "vcheck_status_str",
            "vcheck_last_error", "vcheck_abi_version"} <= names
    for n in names:
        assert hasattr(L, n), n
    assert L.vcheck_abi_version() == 1


def test_struct_sizes_match_header():
    assert ctypes.sizeof(vc.VcTensor) == 80
    assert ctypes.sizeof(vc.VcTol) == 24
    assert ctypes.sizeof(vc.VcCase) == 176
    assert vc.STATS_DTYPE.itemsize == 128 and vc.INTEG_DTYPE.itemsize == 88


def test_status_strings(L):
    for s in range(-10, 1):
        assert L.vcheck_status_str(s).decode()
    assert L.vcheck_status_str(-99).decode() == "unknown status"


def test_tile_count(L):
    assert L.vcheck_tile_count(ctypes.byref(desc(shape=(1024, 1024))), 32, 32) == 1024
    assert L.vcheck_tile_count(ctypes.byref(desc(shape=(3, 1000003))), 64, 64) == 15626
    assert L.vcheck_tile_count(ctypes.byref(desc(shape=(4, 8192, 8192))), 128, 128) == 16384
    assert L.vcheck_tile_count(ctypes.byref(desc(shape=())), 8, 8) == 1
    assert L.vcheck_tile_count(ctypes.byref(desc(shape=(7,))), 2, 2) == 4
    assert L.vcheck_tile_count(ctypes.byref(desc(shape=(0, 5))), 2, 2) == 0
    assert L.vcheck_tile_count(ctypes.byref(desc(shape=(4, 4))), 0, 2) == -1
    assert L.vcheck_tile_count(None, 2, 2) == -1


def _compare(L, c, r, t, out, ws=FAKE, nbytes=1 << 30):
    return L.vcheck_compare(ctypes.byref(c) if c is not None else None,
                            ctypes.byref(r) if r is not None else None,
                            ctypes.byref(t) if t is not None else None, out, ws, nbytes, None)


def test_compare_argument_errors(L):
    out = (ctypes.c_uint8 * 128)()
    out_p = ctypes.addressof(out)
    c, r, t = desc(), desc(), tol()
    assert _compare(L, None, r, t, out_p) == -1
    assert _compare(L, c, r, None, out_p) == -1
    assert _compare(L, c, r, t, None) == -1
    assert _compare(L, desc(data=None), r, t, out_p) == -1
    assert _compare(L, desc(dtype=7), r, t, out_p) == -2
    assert _compare(L, desc(dtype=vc.VC_F16), r, t, out_p) == -2
    assert _compare(L, desc(shape=(5, 4)), r, t, out_p) == -3
    assert _compare(L, desc(shape=(1,) * 9), desc(shape=(1,) * 9), t, out_p) == -3
    assert _compare(L, desc(shape=(-1, 4)), desc(shape=(-1, 4)), t, out_p) == -3
    assert _compare(L, c, r, tol(atol=-1.0), out_p) == -4
    assert _compare(L, c, r, tol(rtol=float("nan")), out_p) == -4
    assert _compare(L, c, r, tol(atol=float("inf")), out_p) == -4
    assert _compare(L, c, r, tol(equal_nan=2), out_p) == -4
    assert _compare(L, desc(data=FAKE + 2), desc(data=FAKE + 2), t, out_p) == -10
    assert _compare(L, c, r, t, out_p, ws=None) == -7
    assert _compare(L, c, r, t, out_p, nbytes=16) == -7
    assert L.vcheck_last_error().decode()
    assert bytes(out) == bytes(128)  # nothing written on any error


def test_localize_argument_errors(L):
    c, r, t = desc(), desc(), tol()
    tm = FAKE
    fk = FAKE
    def loc(th=2, tw=2, tmap=tm, k=4, fkp=fk, nbytes=1 << 30):
        return L.vcheck_localize(ctypes.byref(c), ctypes.byref(r), ctypes.byref(t), th, tw, tmap,
                                 k, fkp, None, FAKE, nbytes, None)
    assert loc(th=0) == -5
    assert loc(tw=-3) == -5
    assert loc(k=-1) == -6
    assert loc(k=vc.VC_MAX_K + 1) == -6
    assert loc(fkp=None) == -6
    assert loc(tmap=None) == -1
    assert loc(nbytes=100) == -7


def test_integrity_argument_errors(L):
    c, r, t = desc(), desc(), tol()
    out = FAKE
    assert L.vcheck_integrity(ctypes.byref(c), ctypes.byref(r), None, 1, ctypes.byref(t), out,
                              None, FAKE, 1 << 30, None) == -1
    arr = (vc.VcTensor * 9)(*[desc() for _ in range(9)])
    assert L.vcheck_integrity(ctypes.byref(c), ctypes.byref(r), arr, 9, ctypes.byref(t), out,
                              None, FAKE, 1 << 30, None) == -8
    assert L.vcheck_integrity(ctypes.byref(c), ctypes.byref(r), arr, 1, ctypes.byref(t), None,
                              None, FAKE, 1 << 30, None) == -1


def _cases(*pairs):
    arr = (vc.VcCase * len(pairs))()
    for i, (c, r) in enumerate(pairs):
        arr[i].cand, arr[i].ref = c, r
    return arr


def test_sweep_argument_errors(L):
    cases = _cases((desc(), desc()), (desc(shape=(3,)), desc(shape=(3,))))
    tols = (vc.VcTol * 2)(tol(), tol(1e-3, 1e-3))
    out = vc.VcSweepOut(FAKE, None, None, None, None, None, None, None)
    def sw(n_tols=2, opts=None, o=out, cs=cases, n=2, nbytes=1 << 30):
        return L.vcheck_sweep(cs, n, tols, n_tols, ctypes.byref(opts) if opts else None,
                              ctypes.byref(o) if o is not None else None, FAKE, nbytes, None)
    assert sw(n_tols=0) == -8
    assert sw(n_tols=9) == -8
    assert sw(opts=vc.VcSweepOpts(2, 1, 1, 0, 0, 0)) == -4
    assert sw(opts=vc.VcSweepOpts(0, 1, 1, 0, 1, 0)) == -1  # integrity without out->integ
    assert sw(o=None) == -1
    assert sw(o=vc.VcSweepOut(None, None, None, None, None, None, None, None)) == -1
    assert sw(n=-1) == -8
    assert sw(cs=None) == -1
    assert sw(nbytes=8) == -7
    with_tiles = vc.VcSweepOut(FAKE, None, None, None, None, FAKE, None, None)
    assert sw(o=with_tiles, opts=vc.VcSweepOpts(0, 0, 4, 0, 0, 0)) == -5
    with_fk = vc.VcSweepOut(FAKE, None, None, None, None, None, FAKE, None)
    assert sw(o=with_fk, opts=vc.VcSweepOpts(0, 1, 1, vc.VC_MAX_K + 1, 0, 0)) == -6
    bad = _cases((desc(dtype=9), desc(dtype=9)))
    assert sw(cs=bad, n=1) == -2


def test_workspace_bytes(L):
    cases = _cases((desc(shape=(1024, 1024)), desc(shape=(1024, 1024))))
    n = ctypes.c_size_t()
    assert L.vcheck_workspace_bytes(cases, 1, 1, None, ctypes.byref(n)) == 0
    base = n.value
    assert base > 0
    opts = vc.VcSweepOpts(0, 32, 32, 64, 0, 0)
    assert L.vcheck_workspace_bytes(cases, 1, 1, ctypes.byref(opts), ctypes.byref(n)) == 0
    assert n.value > base  # first-k staging
    assert L.vcheck_workspace_bytes(cases, 1, 0, None, ctypes.byref(n)) == -8
    assert L.vcheck_workspace_bytes(cases, 1, 1, None, None) == -1
    # a case with differing shapes is a per-case outcome in a sweep, not an error
    mixed = _cases((desc(shape=(4, 4)), desc(shape=(4, 5))))
    assert L.vcheck_workspace_bytes(mixed, 1, 1, None, ctypes.byref(n)) == 0


ERR_CODES = {v: k for k, v in vc.STATUS_NAMES.items()}
VC_ERR_NULL, VC_ERR_DTYPE = ERR_CODES["VC_ERR_NULL"], ERR_CODES["VC_ERR_DTYPE"]
VC_ERR_WORKSPACE, VC_ERR_LIMIT = ERR_CODES["VC_ERR_WORKSPACE"], ERR_CODES["VC_ERR_LIMIT"]
VC_ERR_ALIGN = ERR_CODES["VC_ERR_ALIGN"]


def test_tensor_stats_host_checks(L):
    """The tensor-statistics probe rejects malformed arguments on the host."""
    size = ctypes.c_size_t(0)
    arr = (vc.VcTensor * 3)(desc(), desc(vc.VC_F16, (7,)), desc(vc.VC_BF16, ()))
    assert L.vcheck_tensor_stats_workspace(arr, 3, ctypes.byref(size)) == 0
    assert size.value > 0
    # workspace grows with the batch
    one = ctypes.c_size_t(0)
    assert L.vcheck_tensor_stats_workspace(arr, 1, ctypes.byref(one)) == 0
    assert one.value <= size.value
    assert L.vcheck_tensor_stats_workspace(arr, -1, ctypes.byref(size)) == VC_ERR_LIMIT
    assert L.vcheck_tensor_stats_workspace(None, 2, ctypes.byref(size)) == VC_ERR_NULL
    assert L.vcheck_tensor_stats_workspace(arr, 3, None) == VC_ERR_NULL
    bad = (vc.VcTensor * 2)(desc(), desc(dtype=7))
    assert L.vcheck_tensor_stats_workspace(bad, 2, ctypes.byref(size)) == VC_ERR_DTYPE
    bad = (vc.VcTensor * 1)(desc(vc.VC_F32, (5,), data=FAKE + 2))
    assert L.vcheck_tensor_stats_workspace(bad, 1, ctypes.byref(size)) == VC_ERR_ALIGN
    bad = (vc.VcTensor * 1)(desc(vc.VC_F32, (5,), data=0))
    assert L.vcheck_tensor_stats_workspace(bad, 1, ctypes.byref(size)) == VC_ERR_NULL
    bad = (vc.VcTensor * 1)(desc(vc.VC_F16, (1 << 16, 1 << 15)))
    assert L.vcheck_tensor_stats_workspace(bad, 1, ctypes.byref(size)) == VC_ERR_LIMIT
    # the entry point itself: argument errors before anything is enqueued
    assert L.vcheck_tensor_stats(arr, 3, None, FAKE, 1 << 30, None) == VC_ERR_NULL
    assert L.vcheck_tensor_stats(arr, 3, FAKE, None, 1 << 30, None) == VC_ERR_WORKSPACE
    assert L.vcheck_tensor_stats(arr, 3, FAKE, FAKE, 16, None) == VC_ERR_WORKSPACE
    assert L.vcheck_tensor_stats(arr, 1 << 21, FAKE, FAKE, 1 << 30, None) == VC_ERR_LIMIT
    # an empty batch enqueues nothing
    assert L.vcheck_tensor_stats(None, 0, None, None, 0, None) == 0
    assert vc.TSTATS_DTYPE.itemsize == 608


def test_nearpass_host_checks(L):
    """The near-pass statistics reject malformed arguments on the host."""
    def case(c, r):
        k = vc.VcCase()
        k.cand, k.ref, k.inputs, k.n_inputs = c, r, None, 0
        return k

    size = ctypes.c_size_t(0)
    ok = (vc.VcCase * 2)(case(desc(), desc()), case(desc(vc.VC_F16, (9,)), desc(vc.VC_F16, (9,))))
    assert L.vcheck_nearpass_workspace(ok, 2, ctypes.byref(size)) == 0 and size.value > 0
    bad = (vc.VcCase * 1)(case(desc(vc.VC_F16, (9,)), desc(vc.VC_BF16, (9,))))
    assert L.vcheck_nearpass_workspace(bad, 1, ctypes.byref(size)) == VC_ERR_DTYPE
    bad = (vc.VcCase * 1)(case(desc(vc.VC_F32, (9,)), desc(vc.VC_F32, (3, 3))))
    assert L.vcheck_nearpass_workspace(bad, 1, ctypes.byref(size)) == ERR_CODES["VC_ERR_SHAPE"]
    bad = (vc.VcCase * 1)(case(desc(vc.VC_F32, (9,), data=FAKE + 1), desc(vc.VC_F32, (9,))))
    assert L.vcheck_nearpass_workspace(bad, 1, ctypes.byref(size)) == VC_ERR_ALIGN
    assert L.vcheck_nearpass_workspace(ok, -1, ctypes.byref(size)) == VC_ERR_LIMIT
    assert L.vcheck_nearpass_workspace(None, 1, ctypes.byref(size)) == VC_ERR_NULL
    t = tol()
    neg = tol(atol=-1.0)
    assert L.vcheck_nearpass(ok, 2, ctypes.byref(neg), FAKE, FAKE, 1 << 30, None) == \
        ERR_CODES["VC_ERR_TOL"]
    assert L.vcheck_nearpass(ok, 2, None, FAKE, FAKE, 1 << 30, None) == VC_ERR_NULL
    assert L.vcheck_nearpass(ok, 2, ctypes.byref(t), None, FAKE, 1 << 30, None) == VC_ERR_NULL
    assert L.vcheck_nearpass(ok, 2, ctypes.byref(t), FAKE, FAKE, 8, None) == VC_ERR_WORKSPACE
    assert L.vcheck_nearpass(None, 0, ctypes.byref(t), None, None, 0, None) == 0
    assert vc.NEARPASS_DTYPE.itemsize == 456


def test_content_hash_host_checks(L):
    size = ctypes.c_size_t(0)
    arr = (vc.VcTensor * 2)(desc(), desc(vc.VC_BF16, (3, 3)))
    assert L.vcheck_content_hash_workspace(arr, 2, ctypes.byref(size)) == 0 and size.value > 0
    assert L.vcheck_content_hash_workspace(arr, -1, ctypes.byref(size)) == VC_ERR_LIMIT
    bad = (vc.VcTensor * 1)(desc(dtype=9))
    assert L.vcheck_content_hash_workspace(bad, 1, ctypes.byref(size)) == VC_ERR_DTYPE
    assert L.vcheck_content_hash(arr, 2, None, FAKE, 1 << 20, None) == VC_ERR_NULL
    assert L.vcheck_content_hash(arr, 2, FAKE, FAKE, 4, None) == VC_ERR_WORKSPACE
    assert L.vcheck_content_hash(None, 0, None, None, 0, None) == 0
