"""Shared helpers of the GPU parity tests: move seeded raw inputs to the
device, run the CPU oracle on the same bytes, and compare field by field."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import workloads as wl

EXACT_STATS = ("numel", "mismatches", "nan_cand", "inf_cand", "nan_ref", "inf_ref", "n_finite",
               "n_rel", "n_rel_undef", "max_abs", "argmax_abs", "max_rel", "argmax_rel")
SUM_RTOL = 1e-6  # binary64 error sums: relative agreement bar
INTEG_FIELDS = ("zero_cand", "zero_ref", "eqfirst_cand", "eqfirst_ref", "bf16rep_cand",
                "bf16rep_ref", "fp16rep_cand", "fp16rep_ref", "flags", "copy_input",
                "cand_eq_input_mask", "ref_eq_input_mask", "cand_eq_ref")

TORCH_OF = {oracle.F32: torch.float32, oracle.F16: torch.float16, oracle.BF16: torch.bfloat16}


def to_device(raw: np.ndarray, dtype: int, shape, device="cuda") -> torch.Tensor:
    """Device tensor holding exactly the given raw storage."""
    raw = np.ascontiguousarray(raw)
    if dtype == oracle.F32:
        t = torch.from_numpy(raw.view(np.float32).copy())
    else:
        t = torch.from_numpy(raw.view(np.int16).copy()).view(TORCH_OF[dtype])
    return t.reshape(shape).to(device)


def oracle_case(cand: torch.Tensor, ref: torch.Tensor, tols, primary=0, tile=None, k=None,
                inputs=None) -> oracle.CaseResult:
    dtype = wl.dtype_code(ref.dtype)
    ins = None
    if inputs is not None:
        ins = [(wl.raw_numpy(x).reshape(-1), wl.dtype_code(x.dtype)) for x in inputs]
    return oracle.validate_case(wl.raw_numpy(cand).reshape(-1), wl.raw_numpy(ref).reshape(-1),
                                dtype, tuple(ref.shape), tols, primary=primary, tile=tile, k=k,
                                inputs=ins)


def assert_stats(gpu: dict, orc: dict, tag: str = "") -> None:
    for key in EXACT_STATS:
        g, o = gpu[key], orc[key]
        assert g == o or (isinstance(o, float) and np.isnan(o) and np.isnan(g)), \
            "%s %s: gpu %r oracle %r" % (tag, key, g, o)
    for key in ("sum_abs", "sum_rel"):
        g, o = gpu[key], orc[key]
        assert abs(g - o) <= SUM_RTOL * abs(o), "%s %s: gpu %r oracle %r" % (tag, key, g, o)


def assert_integrity(gpu: dict, orc: dict, tag: str = "") -> None:
    for key in INTEG_FIELDS:
        assert gpu[key] == orc[key], "%s %s: gpu %r oracle %r" % (tag, key, gpu[key], orc[key])
