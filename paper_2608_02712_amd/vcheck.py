"""Python binding of the gfx950 validation library (include/vcheck.h).

Argument marshalling only: every step of the validation runs in the HIP
kernels of libvcheck.so. PyTorch supplies device memory and streams. The
functions carry the C names (``vcheck_compare``, ``vcheck_localize``,
``vcheck_integrity``, ``vcheck_sweep``, ``vcheck_workspace_bytes``,
``vcheck_tile_count``); each synchronous wrapper allocates outputs and a
workspace with torch, launches on the current stream, waits, and returns the
results as Python values. ``Sweep`` prepares a sweep once
(``vcheck_plan_sweep``: the case table stays in the workspace) and relaunches
it without allocating or uploading anything (``vcheck_plan_launch``), for
repeated validation of one case matrix and for timing loops;
``vcheck_sweep_noalloc`` runs a sweep in the library's own scratch.

There is no fallback: if libvcheck.so is missing or fails to load, every call
raises.
"""
from __future__ import annotations

import ctypes
import hashlib
import hmac
import json
import os

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libvcheck.so")

VC_F32, VC_F16, VC_BF16 = 0, 1, 2
VC_MAX_NDIM, VC_MAX_TOLS, VC_MAX_INPUTS, VC_MAX_K = 8, 8, 8, 1024
FLAG_ALL_ZERO, FLAG_CONSTANT, FLAG_INPUT_COPY = 1, 2, 4
FLAG_LOWPREC_BF16, FLAG_LOWPREC_FP16 = 8, 16

STATUS_NAMES = {0: "VC_OK", -1: "VC_ERR_NULL", -2: "VC_ERR_DTYPE", -3: "VC_ERR_SHAPE",
                -4: "VC_ERR_TOL", -5: "VC_ERR_TILE", -6: "VC_ERR_K", -7: "VC_ERR_WORKSPACE",
                -8: "VC_ERR_LIMIT", -9: "VC_ERR_HIP", -10: "VC_ERR_ALIGN", -11: "VC_ERR_STATE"}
NOALLOC_SCRATCH_BYTES = 64 << 20

_DTYPES = {torch.float32: VC_F32, torch.float16: VC_F16, torch.bfloat16: VC_BF16}


class VcheckError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__("%s (%d): %s" % (STATUS_NAMES.get(status, "?"), status, detail))
        self.status = status


# ---------------------------------------------------------------- C structs
class VcTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * VC_MAX_NDIM)]


class VcTol(ctypes.Structure):
    _fields_ = [("atol", ctypes.c_double), ("rtol", ctypes.c_double),
                ("equal_nan", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class VcCase(ctypes.Structure):
    _fields_ = [("cand", VcTensor), ("ref", VcTensor), ("inputs", ctypes.POINTER(VcTensor)),
                ("n_inputs", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class VcSweepOpts(ctypes.Structure):
    _fields_ = [("primary_tol", ctypes.c_int32), ("tile_h", ctypes.c_int32),
                ("tile_w", ctypes.c_int32), ("k", ctypes.c_int32),
                ("do_integrity", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class VcSweepOut(ctypes.Structure):
    _fields_ = [("stats", ctypes.c_void_p), ("mismatches", ctypes.c_void_p),
                ("pass_", ctypes.c_void_p), ("match_rate", ctypes.c_void_p),
                ("numeric_rate", ctypes.c_void_p), ("tile_maps", ctypes.c_void_p),
                ("first_k", ctypes.c_void_p), ("integ", ctypes.c_void_p)]


# numpy views of the device-resident result structs
STATS_DTYPE = np.dtype([
    ("numel", "<u8"), ("mismatches", "<u8"), ("nan_cand", "<u8"), ("inf_cand", "<u8"),
    ("nan_ref", "<u8"), ("inf_ref", "<u8"), ("n_finite", "<u8"), ("n_rel", "<u8"),
    ("n_rel_undef", "<u8"), ("max_abs", "<f8"), ("argmax_abs", "<i8"), ("max_rel", "<f8"),
    ("argmax_rel", "<i8"), ("sum_abs", "<f8"), ("sum_rel", "<f8"), ("case_status", "<i4"),
    ("pass", "<i4")])
INTEG_DTYPE = np.dtype([
    ("zero_cand", "<u8"), ("zero_ref", "<u8"), ("eqfirst_cand", "<u8"), ("eqfirst_ref", "<u8"),
    ("bf16rep_cand", "<u8"), ("bf16rep_ref", "<u8"), ("fp16rep_cand", "<u8"),
    ("fp16rep_ref", "<u8"), ("flags", "<u4"), ("copy_input", "<i4"),
    ("cand_eq_input_mask", "<u4"), ("ref_eq_input_mask", "<u4"), ("cand_eq_ref", "<u4"),
    ("reserved", "<u4")])
assert STATS_DTYPE.itemsize == 128 and INTEG_DTYPE.itemsize == 88

HIST_BINS = 64
HIST_EMIN = -40
TSTATS_DTYPE = np.dtype([
    ("numel", "<u8"), ("nan", "<u8"), ("inf", "<u8"), ("zero", "<u8"), ("n_finite", "<u8"),
    ("min", "<f8"), ("max", "<f8"), ("argmin", "<i8"), ("argmax", "<i8"),
    ("sum", "<f8"), ("sum_sq", "<f8"), ("sum_abs", "<f8"), ("hist", "<u8", (HIST_BINS,)),
])
assert TSTATS_DTYPE.itemsize == 608

RATIO_BINS, ULP_BINS = 32, 18
NEARPASS_DTYPE = np.dtype([
    ("numel", "<u8"), ("n_pairs", "<u8"), ("n_fail", "<u8"), ("n_zero_tol", "<u8"),
    ("max_ratio", "<f8"), ("argmax_ratio", "<i8"), ("max_ulp_fail", "<u4"), ("reserved", "<u4"),
    ("ratio_hist", "<u8", (RATIO_BINS,)), ("ulp_hist", "<u8", (ULP_BINS,)),
])
assert NEARPASS_DTYPE.itemsize == 456

_LIB = None


def lib() -> ctypes.CDLL:
    """The loaded libvcheck.so (raises if it is missing)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libvcheck.so is not built (run python -m paper_2608_02712_amd.build)")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    L.vcheck_compare.argtypes = [ctypes.POINTER(VcTensor), ctypes.POINTER(VcTensor),
                                 ctypes.POINTER(VcTol), P, P, ctypes.c_size_t, P]
    L.vcheck_localize.argtypes = [ctypes.POINTER(VcTensor), ctypes.POINTER(VcTensor),
                                  ctypes.POINTER(VcTol), ctypes.c_int32, ctypes.c_int32, P,
                                  ctypes.c_int32, P, P, P, ctypes.c_size_t, P]
    L.vcheck_integrity.argtypes = [ctypes.POINTER(VcTensor), ctypes.POINTER(VcTensor),
                                   ctypes.POINTER(VcTensor), ctypes.c_int32,
                                   ctypes.POINTER(VcTol), P, P, P, ctypes.c_size_t, P]
    L.vcheck_sweep.argtypes = [ctypes.POINTER(VcCase), ctypes.c_int32, ctypes.POINTER(VcTol),
                               ctypes.c_int32, ctypes.POINTER(VcSweepOpts),
                               ctypes.POINTER(VcSweepOut), P, ctypes.c_size_t, P]
    L.vcheck_workspace_bytes.argtypes = [ctypes.POINTER(VcCase), ctypes.c_int32, ctypes.c_int32,
                                         ctypes.POINTER(VcSweepOpts),
                                         ctypes.POINTER(ctypes.c_size_t)]
    L.vcheck_tile_count.argtypes = [ctypes.POINTER(VcTensor), ctypes.c_int32, ctypes.c_int32]
    L.vcheck_tile_count.restype = ctypes.c_int64
    L.vcheck_status_str.argtypes = [ctypes.c_int32]
    L.vcheck_status_str.restype = ctypes.c_char_p
    L.vcheck_last_error.argtypes = []
    L.vcheck_last_error.restype = ctypes.c_char_p
    L.vcheck_profile_events.argtypes = [P, P]
    L.vcheck_profile_events.restype = ctypes.c_int32
    L.vcheck_abi_version.argtypes = []
    L.vcheck_abi_version.restype = ctypes.c_int32
    L.vcheck_tensor_stats.argtypes = [ctypes.POINTER(VcTensor), ctypes.c_int32, P, P,
                                      ctypes.c_size_t, P]
    L.vcheck_tensor_stats_workspace.argtypes = [ctypes.POINTER(VcTensor), ctypes.c_int32,
                                                ctypes.POINTER(ctypes.c_size_t)]
    L.vcheck_content_hash.argtypes = [ctypes.POINTER(VcTensor), ctypes.c_int32, P, P,
                                      ctypes.c_size_t, P]
    L.vcheck_content_hash_workspace.argtypes = [ctypes.POINTER(VcTensor), ctypes.c_int32,
                                                ctypes.POINTER(ctypes.c_size_t)]
    L.vcheck_nearpass.argtypes = [ctypes.POINTER(VcCase), ctypes.c_int32, ctypes.POINTER(VcTol),
                                  P, P, ctypes.c_size_t, P]
    L.vcheck_nearpass_workspace.argtypes = [ctypes.POINTER(VcCase), ctypes.c_int32,
                                            ctypes.POINTER(ctypes.c_size_t)]
    L.vcheck_plan_sweep.argtypes = [ctypes.POINTER(VcCase), ctypes.c_int32, ctypes.POINTER(VcTol),
                                    ctypes.c_int32, ctypes.POINTER(VcSweepOpts),
                                    ctypes.POINTER(VcSweepOut), P, ctypes.c_size_t, P,
                                    ctypes.POINTER(ctypes.c_void_p)]
    L.vcheck_plan_launch.argtypes = [P, P]
    L.vcheck_plan_free.argtypes = [P]
    L.vcheck_init.argtypes = []
    L.vcheck_sweep_noalloc.argtypes = [ctypes.POINTER(VcCase), ctypes.c_int32,
                                       ctypes.POINTER(VcTol), ctypes.c_int32,
                                       ctypes.POINTER(VcSweepOpts), ctypes.POINTER(VcSweepOut), P]
    for name in ("vcheck_compare", "vcheck_localize", "vcheck_integrity", "vcheck_sweep",
                 "vcheck_workspace_bytes", "vcheck_tensor_stats",
                 "vcheck_tensor_stats_workspace", "vcheck_nearpass",
                 "vcheck_nearpass_workspace", "vcheck_content_hash",
                 "vcheck_content_hash_workspace", "vcheck_plan_sweep", "vcheck_plan_launch",
                 "vcheck_plan_free", "vcheck_init", "vcheck_sweep_noalloc"):
        getattr(L, name).restype = ctypes.c_int32
    if L.vcheck_abi_version() != 1:
        raise RuntimeError("libvcheck.so ABI version mismatch")
    _LIB = L
    return L


def _check(status: int) -> None:
    if status != 0:
        raise VcheckError(status, lib().vcheck_last_error().decode())


# ------------------------------------------------------------ marshalling
def tensor_desc(t: torch.Tensor | None, dtype: int | None = None, shape=None) -> VcTensor:
    """vc_tensor for a contiguous torch tensor (or a raw description)."""
    d = VcTensor()
    if t is not None:
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
        if t.dtype not in _DTYPES:
            raise TypeError("unsupported dtype %s" % t.dtype)
        d.data = t.data_ptr() if t.numel() > 0 else (t.data_ptr() or None)
        d.dtype = _DTYPES[t.dtype]
        shape = tuple(t.shape)
    else:
        d.dtype = dtype
    if len(shape) > VC_MAX_NDIM:
        raise ValueError("at most %d dimensions" % VC_MAX_NDIM)
    d.ndim = len(shape)
    for i, s in enumerate(shape):
        d.shape[i] = int(s)
    return d


def _tols(tols) -> tuple:
    arr = (VcTol * len(tols))()
    for i, t in enumerate(tols):
        t = tuple(t)
        arr[i].atol = float(t[0])
        arr[i].rtol = float(t[1])
        arr[i].equal_nan = int(t[2]) if len(t) > 2 else 0
    return arr


def _stream_ptr(stream) -> int | None:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream or None


def _ws(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def parse_stats(buf: torch.Tensor) -> list[dict]:
    arr = np.frombuffer(buf.cpu().numpy().tobytes(), dtype=STATS_DTYPE)
    return [{k: arr[k][i].item() for k in STATS_DTYPE.names} for i in range(arr.size)]


def parse_integrity(buf: torch.Tensor) -> list[dict]:
    arr = np.frombuffer(buf.cpu().numpy().tobytes(), dtype=INTEG_DTYPE)
    return [{k: arr[k][i].item() for k in INTEG_DTYPE.names if k != "reserved"}
            for i in range(arr.size)]


def vcheck_workspace_bytes(cases_desc, n_tols: int, opts: VcSweepOpts | None = None) -> int:
    """Workspace bytes for an array of VcCase (see vcheck_sweep)."""
    n = ctypes.c_size_t(0)
    arr = cases_desc
    _check(lib().vcheck_workspace_bytes(arr, len(arr), n_tols,
                                        ctypes.byref(opts) if opts is not None else None,
                                        ctypes.byref(n)))
    return n.value


def vcheck_profile_events(begin: "torch.cuda.Event | None", end: "torch.cuda.Event | None") -> None:
    """Arm the profiling hook for the next call on this thread (see vcheck.h).
    The events must already exist (record them once before arming)."""
    _check(lib().vcheck_profile_events(begin.cuda_event if begin is not None else None,
                                       end.cuda_event if end is not None else None))


def vcheck_tile_count(t: torch.Tensor, tile_h: int, tile_w: int) -> int:
    d = tensor_desc(t)
    return int(lib().vcheck_tile_count(ctypes.byref(d), tile_h, tile_w))


def _single_case(cand, ref, inputs=()) -> tuple:
    keep = []
    case = (VcCase * 1)()
    case[0].cand = tensor_desc(cand)
    case[0].ref = tensor_desc(ref)
    if inputs:
        arr = (VcTensor * len(inputs))(*[tensor_desc(x) for x in inputs])
        keep.append(arr)
        case[0].inputs = ctypes.cast(arr, ctypes.POINTER(VcTensor))
        case[0].n_inputs = len(inputs)
    return case, keep


def vcheck_compare(cand: torch.Tensor, ref: torch.Tensor, atol: float, rtol: float,
                   equal_nan: bool = False, stream=None) -> dict:
    """Validate cand against ref (one tolerance pair); returns vc_stats."""
    case, _keep = _single_case(cand, ref)
    tol = _tols([(atol, rtol, int(equal_nan))])
    nbytes = vcheck_workspace_bytes(case, 1)
    ws = _ws(nbytes, ref.device)
    out = torch.zeros(128, dtype=torch.uint8, device=ref.device)
    _check(lib().vcheck_compare(ctypes.byref(case[0].cand), ctypes.byref(case[0].ref), tol,
                                out.data_ptr(), ws.data_ptr(), ws.numel(), _stream_ptr(stream)))
    torch.cuda.synchronize(ref.device)
    return parse_stats(out)[0]


def vcheck_localize(cand: torch.Tensor, ref: torch.Tensor, atol: float, rtol: float,
                    tile_h: int, tile_w: int, k: int, equal_nan: bool = False,
                    stream=None) -> dict:
    """vcheck_compare plus tile map and first-k; returns stats, tile_map, first_k."""
    case, _keep = _single_case(cand, ref)
    tol = _tols([(atol, rtol, int(equal_nan))])
    opts = VcSweepOpts(0, tile_h, tile_w, k, 0, 0)
    nbytes = vcheck_workspace_bytes(case, 1, opts)
    ws = _ws(nbytes, ref.device)
    n_tiles = max(vcheck_tile_count(ref, tile_h, tile_w), 0)
    tmap = torch.empty(max(n_tiles, 1), dtype=torch.int32, device=ref.device)
    fk = torch.empty(max(k, 1), dtype=torch.int64, device=ref.device)
    out = torch.zeros(128, dtype=torch.uint8, device=ref.device)
    _check(lib().vcheck_localize(ctypes.byref(case[0].cand), ctypes.byref(case[0].ref), tol,
                                 tile_h, tile_w, tmap.data_ptr(), k, fk.data_ptr(),
                                 out.data_ptr(), ws.data_ptr(), ws.numel(), _stream_ptr(stream)))
    torch.cuda.synchronize(ref.device)
    return {"stats": parse_stats(out)[0],
            "tile_map": tmap[:n_tiles].cpu().numpy().view(np.uint32).copy(),
            "first_k": fk[:k].cpu().numpy().copy()}


def vcheck_integrity(cand: torch.Tensor, ref: torch.Tensor, inputs, atol: float, rtol: float,
                     equal_nan: bool = False, stream=None) -> dict:
    """Degenerate-output detectors (+ stats) in one pass; inputs: operator inputs."""
    inputs = list(inputs)
    case, keep = _single_case(cand, ref, inputs)
    tol = _tols([(atol, rtol, int(equal_nan))])
    opts = VcSweepOpts(0, 0, 0, 0, 1, 0)
    nbytes = vcheck_workspace_bytes(case, 1, opts)
    ws = _ws(nbytes, ref.device)
    out = torch.zeros(88, dtype=torch.uint8, device=ref.device)
    st = torch.zeros(128, dtype=torch.uint8, device=ref.device)
    in_arr = keep[0] if keep else None
    _check(lib().vcheck_integrity(ctypes.byref(case[0].cand), ctypes.byref(case[0].ref),
                                  in_arr, len(inputs), tol, out.data_ptr(), st.data_ptr(),
                                  ws.data_ptr(), ws.numel(), _stream_ptr(stream)))
    torch.cuda.synchronize(ref.device)
    return {"integrity": parse_integrity(out)[0], "stats": parse_stats(st)[0]}


class Sweep:
    """A vcheck_sweep call over a fixed case matrix.

    cases: list of (cand, ref) or (cand, ref, [inputs]) torch tensors.
    tols: list of (atol, rtol[, equal_nan]). tile: (tile_h, tile_w) or None;
    k: first-k length or 0; integrity: run the detectors.
    mode: "prepared" (default): the sweep is prepared once
    (vcheck_plan_sweep) and each ``launch()`` runs vcheck_plan_launch;
    "oneshot": each ``launch()`` is a full vcheck_sweep call; "noalloc": each
    ``launch()`` is a vcheck_sweep_noalloc call (no workspace is allocated;
    vcheck_init runs first). ``launch()`` enqueues on a stream without
    allocating; ``results()`` synchronises and returns the outputs.
    """

    def __init__(self, cases, tols, primary: int = 0, tile=None, k: int = 0,
                 integrity: bool = False, rates: bool = True, device=None, mode="prepared",
                 stream=None):
        if mode not in ("prepared", "oneshot", "noalloc"):
            raise ValueError("unknown mode %r" % (mode,))
        self.mode = mode
        self._plan = None
        self.n_cases = len(cases)
        self.n_tols = len(tols)
        self.k = int(k)
        self.tile = tile
        self.integrity = bool(integrity)
        self._keep = []
        self.cases = (VcCase * max(self.n_cases, 1))()
        dev = device
        for i, c in enumerate(cases):
            cand, ref = c[0], c[1]
            inputs = list(c[2]) if len(c) > 2 and c[2] is not None else []
            dev = dev or ref.device
            self.cases[i].cand = tensor_desc(cand)
            self.cases[i].ref = tensor_desc(ref)
            if inputs:
                arr = (VcTensor * len(inputs))(*[tensor_desc(x) for x in inputs])
                self._keep.append(arr)
                self.cases[i].inputs = ctypes.cast(arr, ctypes.POINTER(VcTensor))
                self.cases[i].n_inputs = len(inputs)
            self._keep.append((cand, ref, inputs))
        dev = torch.device(dev if dev is not None else "cuda")
        self.device = dev
        self.tols = _tols(tols)
        th, tw = tile if tile is not None else (0, 0)
        self.opts = VcSweepOpts(primary, th, tw, self.k, int(self.integrity), 0)
        if mode == "noalloc":
            self.ws_bytes = 0
            self.ws = None
        else:
            self.ws_bytes = vcheck_workspace_bytes(self.cases, self.n_tols, self.opts) \
                if self.n_cases else 4096
            self.ws = _ws(self.ws_bytes, dev)
        self.stats = torch.zeros(max(self.n_cases, 1) * 128, dtype=torch.uint8, device=dev)
        self.mism = torch.zeros(max(self.n_cases * self.n_tols, 1), dtype=torch.int64, device=dev)
        self.pass_ = torch.zeros(max(self.n_cases * self.n_tols, 1), dtype=torch.uint8, device=dev)
        self.rate = torch.zeros(self.n_tols, dtype=torch.float64, device=dev)
        self.nrate = torch.zeros(self.n_tols, dtype=torch.float64, device=dev)
        self.tile_counts = []
        self.tmaps = None
        if tile is not None:
            self.tile_counts = [max(vcheck_tile_count(c[1], th, tw), 0) for c in cases]
            self.tmaps = torch.zeros(max(sum(self.tile_counts), 1), dtype=torch.int32, device=dev)
        self.fk = torch.zeros(max(self.n_cases * self.k, 1), dtype=torch.int64, device=dev) \
            if self.k > 0 else None
        self.integ = torch.zeros(max(self.n_cases, 1) * 88, dtype=torch.uint8, device=dev) \
            if self.integrity else None
        self.out = VcSweepOut(
            self.stats.data_ptr(), self.mism.data_ptr(), self.pass_.data_ptr(),
            self.rate.data_ptr() if rates else None, self.nrate.data_ptr() if rates else None,
            self.tmaps.data_ptr() if self.tmaps is not None else None,
            self.fk.data_ptr() if self.fk is not None else None,
            self.integ.data_ptr() if self.integ is not None else None)
        if mode == "prepared":
            plan = ctypes.c_void_p()
            with torch.cuda.device(dev):
                _check(lib().vcheck_plan_sweep(self.cases, self.n_cases, self.tols, self.n_tols,
                                               ctypes.byref(self.opts), ctypes.byref(self.out),
                                               self.ws.data_ptr(), self.ws.numel(),
                                               _stream_ptr(stream), ctypes.byref(plan)))
            self._plan = plan
        elif mode == "noalloc":
            with torch.cuda.device(dev):
                _check(lib().vcheck_init())

    def launch(self, stream=None) -> None:
        if self.mode == "prepared":
            _check(lib().vcheck_plan_launch(self._plan, _stream_ptr(stream)))
        elif self.mode == "oneshot":
            _check(lib().vcheck_sweep(self.cases, self.n_cases, self.tols, self.n_tols,
                                      ctypes.byref(self.opts), ctypes.byref(self.out),
                                      self.ws.data_ptr(), self.ws.numel(), _stream_ptr(stream)))
        else:
            _check(lib().vcheck_sweep_noalloc(self.cases, self.n_cases, self.tols, self.n_tols,
                                              ctypes.byref(self.opts), ctypes.byref(self.out),
                                              _stream_ptr(stream)))

    def close(self) -> None:
        """Frees the prepared plan (after the launches in flight are done)."""
        if self._plan is not None:
            torch.cuda.synchronize(self.device)
            lib().vcheck_plan_free(self._plan)
            self._plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:  # interpreter shutdown
            pass

    def results(self) -> dict:
        torch.cuda.synchronize(self.device)
        n, nt = self.n_cases, self.n_tols
        res = {
            "stats": parse_stats(self.stats[:n * 128]) if n else [],
            "mismatches": self.mism[:n * nt].cpu().numpy().reshape(n, nt).astype(np.uint64),
            "pass": self.pass_[:n * nt].cpu().numpy().reshape(n, nt).copy(),
            "match_rate": self.rate.cpu().numpy().copy(),
            "numeric_rate": self.nrate.cpu().numpy().copy(),
        }
        if self.tmaps is not None:
            flat = self.tmaps.cpu().numpy().view(np.uint32)
            maps, off = [], 0
            for c in self.tile_counts:
                maps.append(flat[off:off + c].copy())
                off += c
            res["tile_maps"] = maps
        if self.fk is not None:
            res["first_k"] = self.fk[:n * self.k].cpu().numpy().reshape(n, self.k).copy()
        if self.integ is not None:
            res["integrity"] = parse_integrity(self.integ[:n * 88]) if n else []
        return res


def vcheck_sweep(cases, tols, primary: int = 0, tile=None, k: int = 0, integrity: bool = False,
                 stream=None) -> dict:
    """Validate a whole case matrix in one vcheck_sweep call; returns per-case
    results and per-pair suite match rates."""
    sw = Sweep(cases, tols, primary=primary, tile=tile, k=k, integrity=integrity, mode="oneshot")
    sw.launch(stream)
    return sw.results()


def vcheck_sweep_noalloc(cases, tols, primary: int = 0, tile=None, k: int = 0,
                         integrity: bool = False, stream=None) -> dict:
    """vcheck_sweep in the library's scratch (vcheck_sweep_noalloc)."""
    sw = Sweep(cases, tols, primary=primary, tile=tile, k=k, integrity=integrity, mode="noalloc")
    sw.launch(stream)
    return sw.results()


compare = vcheck_compare
localize = vcheck_localize
integrity = vcheck_integrity
sweep = vcheck_sweep


class TensorStats:
    """A prepared tensor-statistics probe over a fixed batch of device tensors
    (descriptors, output and workspace allocated once); launch() enqueues
    vcheck_tensor_stats, results() reads the statistics back."""

    def __init__(self, tensors):
        self.tensors = list(tensors)
        n = len(self.tensors)
        self.desc = (VcTensor * max(n, 1))(*[tensor_desc(t) for t in self.tensors])
        size = ctypes.c_size_t(0)
        _check(lib().vcheck_tensor_stats_workspace(self.desc, n, ctypes.byref(size)))
        dev = self.tensors[0].device if n else torch.device("cuda")
        self.ws = _ws(size.value, dev)
        self.out = torch.zeros(max(n, 1) * TSTATS_DTYPE.itemsize, dtype=torch.uint8, device=dev)

    def launch(self, stream=None) -> None:
        _check(lib().vcheck_tensor_stats(self.desc, len(self.tensors), self.out.data_ptr(),
                                         self.ws.data_ptr(), self.ws.numel(),
                                         _stream_ptr(stream)))

    def results(self) -> list[dict]:
        torch.cuda.synchronize(self.out.device)
        arr = np.frombuffer(self.out.cpu().numpy().tobytes(), dtype=TSTATS_DTYPE)
        res = []
        for i in range(len(self.tensors)):
            d = {k: arr[k][i].item() for k in TSTATS_DTYPE.names if k != "hist"}
            d["hist"] = [int(v) for v in arr["hist"][i]]
            # derived: mean and mean magnitude. (No spread statistic: the
            # one the sums give, sum_sq / n - mean^2, cancels catastrophically
            # when |mean| is large against the spread.)
            nf = d["n_finite"]
            d["mean"] = d["sum"] / nf if nf else 0.0
            d["abs_mean"] = d["sum_abs"] / nf if nf else 0.0
            res.append(d)
        return res


def vcheck_tensor_stats(tensors, stream=None) -> list[dict]:
    """Tensor-statistics probe of a batch of device tensors (one pass); one
    dict per tensor: counts, min/max with first index, binary64 sums, the
    binary-exponent histogram and the derived mean / abs_mean."""
    ts = TensorStats(tensors)
    if ts.tensors:
        ts.launch(stream)
    return ts.results()


class NearPass:
    """Prepared near-pass statistics over a fixed list of (cand, ref) device
    tensor pairs at one tolerance pair; launch() enqueues vcheck_nearpass,
    results() reads one dict per case (plus the derived fp16_ceiling: the
    case fails, and only within one grid step)."""

    def __init__(self, cases, atol: float, rtol: float):
        self.cases = [(c, r) for c, r, *_ in cases]
        n = len(self.cases)
        self._keep = []
        arr = (VcCase * max(n, 1))()
        for i, (c, r) in enumerate(self.cases):
            arr[i].cand = tensor_desc(c)
            arr[i].ref = tensor_desc(r)
            arr[i].inputs = None
            arr[i].n_inputs = 0
        self.desc = arr
        self.tol = _tols([(atol, rtol, 0)])
        size = ctypes.c_size_t(0)
        _check(lib().vcheck_nearpass_workspace(self.desc, n, ctypes.byref(size)))
        dev = self.cases[0][1].device if n else torch.device("cuda")
        self.ws = _ws(size.value, dev)
        self.out = torch.zeros(max(n, 1) * NEARPASS_DTYPE.itemsize, dtype=torch.uint8,
                               device=dev)

    def launch(self, stream=None) -> None:
        _check(lib().vcheck_nearpass(self.desc, len(self.cases), self.tol, self.out.data_ptr(),
                                     self.ws.data_ptr(), self.ws.numel(), _stream_ptr(stream)))

    def results(self) -> list[dict]:
        torch.cuda.synchronize(self.out.device)
        arr = np.frombuffer(self.out.cpu().numpy().tobytes(), dtype=NEARPASS_DTYPE)
        res = []
        for i in range(len(self.cases)):
            d = {k: arr[k][i].item() for k in NEARPASS_DTYPE.names
                 if k not in ("ratio_hist", "ulp_hist", "reserved")}
            d["ratio_hist"] = [int(v) for v in arr["ratio_hist"][i]]
            d["ulp_hist"] = [int(v) for v in arr["ulp_hist"][i]]
            d["fp16_ceiling"] = d["n_fail"] > 0 and d["max_ulp_fail"] <= 1
            res.append(d)
        return res


def vcheck_nearpass(cases, atol: float, rtol: float, stream=None) -> list[dict]:
    """Near-pass statistics of (cand, ref) device tensor pairs at one
    tolerance pair (violation ratios and grid distances; see vcheck.h)."""
    np_ = NearPass(cases, atol, rtol)
    if np_.cases:
        np_.launch(stream)
    return np_.results()


class ContentHash:
    """Prepared content hashes of a fixed list of device tensors (see
    vcheck.h): launch() enqueues vcheck_content_hash, results() returns one
    64-bit integer per tensor."""

    def __init__(self, tensors):
        self.tensors = list(tensors)
        n = len(self.tensors)
        self.desc = (VcTensor * max(n, 1))(*[tensor_desc(t) for t in self.tensors])
        size = ctypes.c_size_t(0)
        _check(lib().vcheck_content_hash_workspace(self.desc, n, ctypes.byref(size)))
        dev = self.tensors[0].device if n else torch.device("cuda")
        self.ws = _ws(size.value, dev)
        self.out = torch.zeros(max(n, 1), dtype=torch.int64, device=dev)

    def launch(self, stream=None) -> None:
        _check(lib().vcheck_content_hash(self.desc, len(self.tensors), self.out.data_ptr(),
                                         self.ws.data_ptr(), self.ws.numel(),
                                         _stream_ptr(stream)))

    def results(self) -> list[int]:
        torch.cuda.synchronize(self.out.device)
        return [int(v) for v in self.out.cpu().numpy()[:len(self.tensors)].view(np.uint64)]


def vcheck_content_hash(tensors, stream=None) -> list[int]:
    """Content hashes of device tensors (one pass; see vcheck.h)."""
    h = ContentHash(tensors)
    if h.tensors:
        h.launch(stream)
    return h.results()


# The engine's signing key for evidence records: drawn once per process, so
# only this engine can produce a record that verifies (callers that keep
# records across processes pass their own key to escalate / verify_evidence).
_EVIDENCE_KEY = os.urandom(32)


def _evidence_mac(record: dict, key: bytes | None = None) -> str:
    body = json.dumps(record, sort_keys=True, separators=(",", ":")).encode()
    return hmac.new(key if key is not None else _EVIDENCE_KEY, body, hashlib.sha256).hexdigest()


def escalate(compact, extended, tols, primary: int = 0, gate: float = 1.0, tile=None,
             k: int = 0, integrity: bool = True, evidence_path: str | None = None,
             key: bytes | None = None) -> dict:
    """Two-stage validation with full-coverage evidence (Sec. 4.3, the
    validation-escalation panel of the mechanisms figure; Sec. S2.2).

    The compact case set runs first; only when its certified match rate at
    the primary pair reaches `gate` does the extended set (the full coverage:
    every shape and dtype) run, as one vcheck_sweep. Acceptance requires the
    extended set to certify every case (numerically passing at the primary
    pair, no detector flag) with the detectors run (`integrity`, on by
    default). The evidence record holds, per stage and case, the pass bits,
    mismatch counts, detector flags, shape, storage type and the content
    hashes of cand and ref, the stage's match rates, whether the detectors
    ran, and a hash of its case set. The record is signed with an HMAC-SHA256
    under the engine's key (`key`, else a per-process secret): an edited
    record, or one re-signed without the key, fails verify_evidence. Written
    as JSON to `evidence_path` when given.

    compact / extended: lists of (cand, ref) or (cand, ref, inputs)."""

    def stage(cases):
        res = vcheck_sweep(cases, tols, primary=primary, tile=tile, k=k, integrity=integrity)
        tensors = [t for c in cases for t in (c[0], c[1])]
        hashes = vcheck_content_hash(tensors)
        rows = []
        for i in range(len(cases)):
            flags = res["integrity"][i]["flags"] if res.get("integrity") else 0
            ref = cases[i][1]
            rows.append({
                "pass": [int(x) for x in res["pass"][i]],
                "mismatches": [int(x) for x in res["mismatches"][i]],
                "flags": int(flags),
                "shape": [int(x) for x in ref.shape],
                "dtype": str(ref.dtype).replace("torch.", ""),
                "cand_hash": "%016x" % hashes[2 * i],
                "ref_hash": "%016x" % hashes[2 * i + 1],
            })
        set_digest = hashlib.sha256("".join(
            "%s%s%s%s" % (r["cand_hash"], r["ref_hash"], r["dtype"], r["shape"])
            for r in rows).encode()).hexdigest()
        return {"n_cases": len(cases), "match_rate": [float(x) for x in res["match_rate"]],
                "numeric_rate": [float(x) for x in res["numeric_rate"]],
                "detectors_ran": bool(integrity),
                "case_set_hash": set_digest, "cases": rows}

    record = {"tols": [list(map(float, t[:2])) for t in tols], "primary": primary,
              "gate": gate, "compact": stage(compact), "extended": None}
    if record["compact"]["match_rate"][primary] >= gate:
        record["extended"] = stage(extended)
    ext = record["extended"]
    record["accepted"] = bool(ext is not None and ext["n_cases"] > 0 and
                              ext["detectors_ran"] and ext["match_rate"][primary] == 1.0)
    record["mac"] = _evidence_mac(record, key)
    if evidence_path is not None:
        with open(evidence_path, "w") as f:
            json.dump(record, f, indent=1, sort_keys=True)
    return record


def verify_evidence(record: dict, key: bytes | None = None) -> bool:
    """Whether an evidence record carries a valid signature under the
    engine's key (`key`, else this process's secret)."""
    body = {k: v for k, v in record.items() if k != "mac"}
    mac = record.get("mac")
    return isinstance(mac, str) and hmac.compare_digest(_evidence_mac(body, key), mac)


class BestCandidate:
    """State-continuous repair bookkeeping (Sec. 4.4; the mechanisms figure's
    state-continuous panel): the engine keeps the highest-scoring candidate,
    and after `patience` (two) consecutive attempts that do not improve on
    it, it rolls back to that candidate.

    record(name, score) takes an attempt's score, the certified match rate
    at the primary pair of its full-coverage evaluation (vcheck_sweep's
    match_rate, or an evidence record's), and returns "promote" (a new best:
    strictly higher score, or the first attempt), "continue" (not better,
    fewer than `patience` such attempts in a row) or "rollback" (the
    patience-th non-improving attempt in a row: continue from `best`; the
    count restarts)."""

    def __init__(self, patience: int = 2):
        if patience < 1:
            raise ValueError("patience must be at least 1")
        self.patience = patience
        self.best = None
        self.best_score = None
        self.stale = 0
        self.history = []

    def record(self, name, score: float) -> str:
        score = float(score)
        if self.best_score is None or score > self.best_score:
            self.best, self.best_score, self.stale = name, score, 0
            decision = "promote"
        else:
            self.stale += 1
            decision = "continue"
            if self.stale >= self.patience:
                decision = "rollback"
                self.stale = 0
        self.history.append((name, score, decision))
        return decision

    def record_evidence(self, name, record: dict, key: bytes | None = None) -> str:
        """record() with the score of an escalate() evidence record: the
        extended set's certified match rate at the primary pair, or 0 when
        the compact set stopped the escalation or the record does not verify
        (edited, or signed without the engine's key)."""
        if not verify_evidence(record, key) or record.get("extended") is None:
            return self.record(name, 0.0)
        return self.record(name, record["extended"]["match_rate"][record["primary"]])

