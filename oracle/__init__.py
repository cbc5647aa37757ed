"""CPU oracle for candidate-vs-reference validation (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import this package. The product path (the HIP
library and its Python binding) never imports it, and the two share no code.

The arithmetic lives in ``vcheck_oracle.c`` (plain C, one loop per case, IEEE
binary64, no fused multiply-add); this module only builds that file with gcc
and marshals numpy buffers into it. What the C file computes, and which
passage of the paper each step follows, is stated in its header comment.

Parity status: every output is pinned by ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vcheck_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libvcheck_oracle.so")

F32, F16, BF16 = 0, 1, 2
FLAG_ALL_ZERO, FLAG_CONSTANT, FLAG_INPUT_COPY = 1, 2, 4
FLAG_LOWPREC_BF16, FLAG_LOWPREC_FP16 = 8, 16

GCC_FLAGS = ["-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-shared", "-fPIC"]


def build(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle with gcc into a shared library; returns its path."""
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", *GCC_FLAGS, "-o", tmp, src, "-lm"], check=True)
    os.replace(tmp, out)
    return out


class Stats(ctypes.Structure):
    _fields_ = [
        ("numel", ctypes.c_uint64), ("mismatches", ctypes.c_uint64),
        ("nan_cand", ctypes.c_uint64), ("inf_cand", ctypes.c_uint64),
        ("nan_ref", ctypes.c_uint64), ("inf_ref", ctypes.c_uint64),
        ("n_finite", ctypes.c_uint64), ("n_rel", ctypes.c_uint64),
        ("n_rel_undef", ctypes.c_uint64),
        ("max_abs", ctypes.c_double), ("argmax_abs", ctypes.c_int64),
        ("max_rel", ctypes.c_double), ("argmax_rel", ctypes.c_int64),
        ("sum_abs", ctypes.c_double), ("sum_rel", ctypes.c_double),
    ]


class Integrity(ctypes.Structure):
    _fields_ = [
        ("zero_cand", ctypes.c_uint64), ("zero_ref", ctypes.c_uint64),
        ("eqfirst_cand", ctypes.c_uint64), ("eqfirst_ref", ctypes.c_uint64),
        ("bf16rep_cand", ctypes.c_uint64), ("bf16rep_ref", ctypes.c_uint64),
        ("fp16rep_cand", ctypes.c_uint64), ("fp16rep_ref", ctypes.c_uint64),
        ("flags", ctypes.c_uint32), ("copy_input", ctypes.c_int32),
        ("cand_eq_input_mask", ctypes.c_uint32), ("ref_eq_input_mask", ctypes.c_uint32),
        ("cand_eq_ref", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
    ]


HIST_BINS = 64
HIST_EMIN = -40


class TStats(ctypes.Structure):
    _fields_ = [
        ("numel", ctypes.c_uint64), ("nan", ctypes.c_uint64), ("inf", ctypes.c_uint64),
        ("zero", ctypes.c_uint64), ("n_finite", ctypes.c_uint64),
        ("min", ctypes.c_double), ("max", ctypes.c_double),
        ("argmin", ctypes.c_int64), ("argmax", ctypes.c_int64),
        ("sum", ctypes.c_double), ("sum_sq", ctypes.c_double), ("sum_abs", ctypes.c_double),
        ("hist", ctypes.c_uint64 * HIST_BINS),
    ]


RATIO_BINS = 32
ULP_BINS = 18


class NearPass(ctypes.Structure):
    _fields_ = [
        ("numel", ctypes.c_uint64), ("n_pairs", ctypes.c_uint64), ("n_fail", ctypes.c_uint64),
        ("n_zero_tol", ctypes.c_uint64), ("max_ratio", ctypes.c_double),
        ("argmax_ratio", ctypes.c_int64), ("max_ulp_fail", ctypes.c_uint32),
        ("reserved", ctypes.c_uint32),
        ("ratio_hist", ctypes.c_uint64 * RATIO_BINS), ("ulp_hist", ctypes.c_uint64 * ULP_BINS),
    ]


def _struct_dict(s) -> dict:
    return {name: getattr(s, name) for name, _ in s._fields_ if name != "reserved"}


_P = ctypes.c_void_p


def load(path: str | None = None) -> ctypes.CDLL:
    """Load (building first if absent) the oracle library."""
    path = path or _LIB_PATH
    if path == _LIB_PATH and not os.path.exists(path):
        build()
    lib = ctypes.CDLL(path)
    lib.orc_validate.restype = ctypes.c_int32
    lib.orc_validate.argtypes = [
        ctypes.c_int32, _P, _P, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, _P, _P, _P,
        ctypes.c_int32, _P, ctypes.POINTER(Stats), ctypes.c_int32, ctypes.c_int32, _P,
        ctypes.c_int32, _P, ctypes.c_int32, _P, _P, _P, ctypes.POINTER(Integrity),
    ]
    lib.orc_decode.restype = None
    lib.orc_decode.argtypes = [ctypes.c_int32, _P, ctypes.c_int64, _P]
    lib.orc_suite.restype = None
    lib.orc_suite.argtypes = [ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P, _P]
    lib.orc_nearpass.restype = None
    lib.orc_nearpass.argtypes = [ctypes.c_int32, _P, _P, ctypes.c_int64, ctypes.c_double,
                                 ctypes.c_double, ctypes.POINTER(NearPass)]
    lib.orc_round_binary16.restype = ctypes.c_uint16
    lib.orc_round_binary16.argtypes = [ctypes.c_double]
    lib.orc_content_hash.restype = ctypes.c_uint64
    lib.orc_content_hash.argtypes = [ctypes.c_int32, _P, ctypes.c_int64]
    lib.orc_splitmix_finalize.restype = ctypes.c_uint64
    lib.orc_splitmix_finalize.argtypes = [ctypes.c_uint64]
    lib.orc_tensor_stats.restype = None
    lib.orc_tensor_stats.argtypes = [ctypes.c_int32, _P, ctypes.c_int64, ctypes.POINTER(TStats)]
    return lib


_DEFAULT: ctypes.CDLL | None = None


def default_lib() -> ctypes.CDLL:
    global _DEFAULT
    if _DEFAULT is None:
        _DEFAULT = load()
    return _DEFAULT


def _raw(a: np.ndarray, dtype: int) -> np.ndarray:
    """Contiguous raw-storage view (float32 / 16-bit patterns)."""
    a = np.ascontiguousarray(a)
    want = 4 if dtype == F32 else 2
    if a.dtype.itemsize != want:
        raise ValueError("element size %d does not match dtype code %d" % (a.dtype.itemsize, dtype))
    return a


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


@dataclass
class CaseResult:
    stats: dict
    mismatches: list
    tile_map: np.ndarray | None = None
    first_k: np.ndarray | None = None
    integrity: dict | None = None
    extra: dict = field(default_factory=dict)


def decode(raw: np.ndarray, dtype: int, lib=None) -> np.ndarray:
    lib = lib or default_lib()
    raw = _raw(raw, dtype)
    out = np.empty(raw.size, dtype=np.float64)
    lib.orc_decode(dtype, _ptr(raw), raw.size, _ptr(out))
    return out.reshape(raw.shape)


def view_rows_cols(shape) -> tuple[int, int]:
    """(rows, cols) view of a shape: cols = last dim; 0-d is (1, 1)."""
    shape = tuple(int(s) for s in shape)
    if len(shape) == 0:
        return 1, 1
    cols = shape[-1]
    rows = 1
    for s in shape[:-1]:
        rows *= s
    return rows, cols


def validate_case(cand: np.ndarray, ref: np.ndarray, dtype: int, shape, tols,
                  primary: int = 0, tile=None, k: int | None = None, inputs=None,
                  lib=None) -> CaseResult:
    """Run the oracle on one case.

    cand/ref: raw storage arrays (float32 or 16-bit patterns) of `shape`.
    tols: list of (atol, rtol) or (atol, rtol, equal_nan).
    tile: (tile_h, tile_w) or None. k: first-k length or None.
    inputs: list of (raw array, dtype code) operator inputs, or None to skip
    the degenerate-output detectors.
    """
    lib = lib or default_lib()
    cand = _raw(cand, dtype)
    ref = _raw(ref, dtype)
    rows, cols = view_rows_cols(shape)
    if cand.size != rows * cols or ref.size != rows * cols:
        raise ValueError("buffer size does not match shape")
    tols = [tuple(t) + (0,) * (3 - len(t)) for t in tols]
    atol = np.array([t[0] for t in tols], dtype=np.float64)
    rtol = np.array([t[1] for t in tols], dtype=np.float64)
    eqn = np.array([int(t[2]) for t in tols], dtype=np.int32)
    mism = np.zeros(len(tols), dtype=np.uint64)
    st = Stats()
    tile_map = None
    th = tw = 1
    if tile is not None:
        th, tw = int(tile[0]), int(tile[1])
        tile_map = np.zeros(((rows + th - 1) // th) * ((cols + tw - 1) // tw), dtype=np.uint32)
    fk = np.zeros(k, dtype=np.int64) if k is not None else None
    integ = None
    keep = []
    in_ptrs = in_dt = in_n = None
    n_in = 0
    if inputs is not None:
        integ = Integrity()
        n_in = len(inputs)
        raws = [np.ascontiguousarray(x) for x, _ in inputs]
        keep.extend(raws)
        in_ptrs = (ctypes.c_void_p * max(n_in, 1))(*[_ptr(x) for x in raws])
        in_dt = np.array([d for _, d in inputs] or [0], dtype=np.int32)
        in_n = np.array([x.size for x in raws] or [0], dtype=np.int64)
    rc = lib.orc_validate(
        dtype, _ptr(cand), _ptr(ref), rows, cols, len(tols), _ptr(atol), _ptr(rtol), _ptr(eqn),
        primary, _ptr(mism), ctypes.byref(st), th, tw,
        _ptr(tile_map) if tile_map is not None else None,
        k if k is not None else 0, _ptr(fk) if fk is not None else None,
        n_in, ctypes.cast(in_ptrs, ctypes.c_void_p) if in_ptrs is not None else None,
        _ptr(in_dt) if in_dt is not None else None, _ptr(in_n) if in_n is not None else None,
        ctypes.byref(integ) if integ is not None else None)
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return CaseResult(stats=_struct_dict(st), mismatches=[int(m) for m in mism],
                      tile_map=tile_map, first_k=fk,
                      integrity=_struct_dict(integ) if integ is not None else None)


def suite(mismatches: np.ndarray, status, flags=None, lib=None):
    """Suite verdict: returns (pass[n_cases, n_tols] uint8, rate[n_tols])."""
    lib = lib or default_lib()
    m = np.ascontiguousarray(mismatches, dtype=np.uint64)
    n_cases, n_tols = m.shape
    st = np.ascontiguousarray(status, dtype=np.int32)
    fl = np.ascontiguousarray(flags, dtype=np.uint32) if flags is not None else None
    pas = np.zeros((n_cases, n_tols), dtype=np.uint8)
    rate = np.zeros(n_tols, dtype=np.float64)
    lib.orc_suite(n_cases, n_tols, _ptr(m), _ptr(st), _ptr(fl) if fl is not None else None,
                  _ptr(pas), _ptr(rate))
    return pas, rate


def tensor_stats(raw: np.ndarray, dtype: int, lib=None) -> dict:
    """Tensor-statistics probe of one tensor (raw storage: float32 or 16-bit
    patterns): counts, first-index min/max over finite values, binary64 sums
    in index order and the binary-exponent histogram (see the C header)."""
    lib = lib or default_lib()
    raw = _raw(raw, dtype).reshape(-1)
    st = TStats()
    lib.orc_tensor_stats(dtype, _ptr(raw) if raw.size else None, raw.size, ctypes.byref(st))
    d = _struct_dict(st)
    d["hist"] = [int(v) for v in st.hist]
    return d


def nearpass(cand: np.ndarray, ref: np.ndarray, dtype: int, atol: float, rtol: float,
             lib=None) -> dict:
    """Near-pass statistics of one case at one tolerance pair (raw storage
    arrays; see the C header): violation-ratio maximum and histogram, and
    the distance histogram on the binary16 / bfloat16 grid."""
    lib = lib or default_lib()
    cand = _raw(cand, dtype).reshape(-1)
    ref = _raw(ref, dtype).reshape(-1)
    if cand.size != ref.size:
        raise ValueError("cand and ref sizes differ")
    st = NearPass()
    lib.orc_nearpass(dtype, _ptr(cand) if cand.size else None, _ptr(ref) if ref.size else None,
                     cand.size, float(atol), float(rtol), ctypes.byref(st))
    d = _struct_dict(st)
    d["ratio_hist"] = [int(v) for v in st.ratio_hist]
    d["ulp_hist"] = [int(v) for v in st.ulp_hist]
    return d


def content_hash(raw: np.ndarray, dtype: int, lib=None) -> int:
    """Content hash of one tensor's raw storage (see the C header)."""
    lib = lib or default_lib()
    raw = _raw(raw, dtype).reshape(-1)
    return int(lib.orc_content_hash(dtype, _ptr(raw) if raw.size else None, raw.size))
