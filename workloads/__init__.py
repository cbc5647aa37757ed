"""Seeded synthetic validation workloads (inputs only; no validation arithmetic).

Both sides use these generators: the CPU oracle (in tests and in the
benchmark's CPU-baseline leg) and the HIP library. The module produces
candidate / reference / operator-input tensors and the positions of the faults
it injected; it never evaluates the tolerance gate or any metric.

Five workloads, stand-ins for the paper's full-coverage operator case matrix
(Sec. 4.3 full-coverage evaluation; Sec. S6.1 reports 5 to 58 cases per
operator):

1. fp32 single case 1024x1024 with a zeroed 24x64 corner block.
2. fp16 batch of 64 cases 2048x2048, one shifted 64x64 tile and 3 NaNs each.
3. bf16 single case 4x8192x8192 with sparse x1.1 faults and a +Inf burst.
4. fp32 sweep of 500 odd-shaped cases (1x1 .. 2^24 elements), 4 tolerance
   pairs, faults in the last (partial) tile.
5. fp32 integrity batch of 256 cases 4096x4096 mixing correct, input-copy,
   all-zero, constant-fill and bf16-computed candidates.

Every size argument defaults to the full workload; the tests pass smaller
sizes with the same structure. Bulk values come from a torch generator on the
target device seeded with ``seed + case``; fault positions and class
assignments come from numpy's PCG64 on the host, so the injected sets are
known independently of any device.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

BASE_SEED = 2608


def config_seed(s: int) -> int:
    return BASE_SEED * 1000 + s


@dataclass
class Case:
    cand: torch.Tensor
    ref: torch.Tensor
    inputs: list = field(default_factory=list)


@dataclass
class Workload:
    name: str
    dtype: torch.dtype
    cases: list
    tols: list  # [(atol, rtol, equal_nan)]
    primary: int = 0
    tile: tuple | None = None
    k: int | None = None
    integrity: bool = False
    meta: dict = field(default_factory=dict)

    @property
    def numel(self) -> int:
        return sum(c.ref.numel() for c in self.cases)

    @property
    def ref_cand_bytes(self) -> int:
        return sum(c.ref.numel() * c.ref.element_size() * 2 for c in self.cases)


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _distinct(rng: np.random.Generator, n: int, count: int, reject=None) -> np.ndarray:
    """`count` distinct integers in [0, n) (ascending), avoiding `reject(i)`."""
    chosen: set[int] = set()
    while len(chosen) < count:
        i = int(rng.integers(0, n))
        if i in chosen or (reject is not None and reject(i)):
            continue
        chosen.add(i)
    return np.array(sorted(chosen), dtype=np.int64)


# --------------------------------------------------------------------------- 1
def fp32_single(device="cuda", rows: int = 1024, cols: int = 1024, seed: int | None = None) -> Workload:
    """fp32 single case; ref ~ N(0,1), cand = ref + 1e-7 N(0,1); the last 24
    rows x last 64 cols of cand are set to 0.0 (rows 1000-1023, cols 960-1023
    at full size). atol = rtol = 1e-5, 32x32 tiles, first-k = 64."""
    seed = config_seed(1) if seed is None else seed
    g = _gen(device, seed)
    ref = torch.randn(rows, cols, generator=g, device=device, dtype=torch.float32)
    cand = ref + 1e-7 * torch.randn(rows, cols, generator=g, device=device, dtype=torch.float32)
    r0, c0 = rows - 24, cols - 64
    cand[r0:, c0:] = 0.0
    return Workload("fp32 1x1024x1024", torch.float32, [Case(cand, ref)], [(1e-5, 1e-5, 0)],
                    tile=(32, 32), k=64,
                    meta={"fault_rows": (r0, rows), "fault_cols": (c0, cols)})


# --------------------------------------------------------------------------- 2
def fp16_batch(device="cuda", n_cases: int = 64, rows: int = 2048, cols: int = 2048,
            tile: int = 64, seed: int | None = None) -> Workload:
    """fp16 batch. Per case: r32 ~ N(0,1), ref = fp16(r32), cand =
    fp16(r32 + 1e-4 N(0,1)); one seeded tile-aligned 64x64 block gets
    cand = fp16(cand + 0.5); 3 NaNs at seeded distinct positions outside it.
    atol = rtol = 1e-3, 64x64 tiles, first-k = 64."""
    seed = config_seed(2) if seed is None else seed
    ref_all = torch.empty(n_cases, rows, cols, device=device, dtype=torch.float16)
    cand_all = torch.empty_like(ref_all)
    faults = []
    for i in range(n_cases):
        g = _gen(device, seed + i)
        rng = _rng(seed + i)
        r32 = torch.randn(rows, cols, generator=g, device=device, dtype=torch.float32)
        ref_all[i] = r32.half()
        cand = (r32 + 1e-4 * torch.randn(rows, cols, generator=g, device=device,
                                         dtype=torch.float32)).half()
        ti = int(rng.integers(0, rows // tile))
        tj = int(rng.integers(0, cols // tile))
        blk = cand[ti * tile:(ti + 1) * tile, tj * tile:(tj + 1) * tile]
        cand[ti * tile:(ti + 1) * tile, tj * tile:(tj + 1) * tile] = (blk.float() + 0.5).half()

        def in_tile(f, ti=ti, tj=tj):
            return (f // cols) // tile == ti and (f % cols) // tile == tj

        nans = _distinct(rng, rows * cols, 3, reject=in_tile)
        cand.view(-1)[torch.as_tensor(nans, device=device)] = float("nan")
        cand_all[i] = cand
        faults.append({"tile": (ti, tj), "nans": nans})
        del r32, cand
    cases = [Case(cand_all[i], ref_all[i]) for i in range(n_cases)]
    return Workload("fp16 64x2048x2048", torch.float16, cases, [(1e-3, 1e-3, 0)],
                    tile=(tile, tile), k=64, meta={"faults": faults, "tile_size": tile})


# --------------------------------------------------------------------------- 3
def bf16_bursts(device="cuda", shape=(4, 8192, 8192), burst: int = 512, seed: int | None = None,
            fault_fraction: float = 1e-6) -> Workload:
    """bf16 single large case. ref = bf16(U(-4,4)); cand = bf16(fp32(ref)),
    bit-identical to ref; floor(1e-6 n) seeded positions get
    cand = bf16(1.1 * fp32(ref)); a seeded burst of 512 contiguous elements,
    disjoint from those, is set to +Inf. atol = 1e-2, rtol = 1.6e-2,
    128x128 tiles, first-k = 64."""
    seed = config_seed(3) if seed is None else seed
    g = _gen(device, seed)
    rng = _rng(seed)
    n = math.prod(shape)
    ref = (torch.rand(shape, generator=g, device=device, dtype=torch.float32) * 8.0 - 4.0
           ).to(torch.bfloat16)
    cand = ref.float().to(torch.bfloat16)
    n_scaled = int(math.floor(fault_fraction * n))
    scaled = _distinct(rng, n, n_scaled)
    idx = torch.as_tensor(scaled, device=device)
    flat = cand.view(-1)
    flat[idx] = (ref.view(-1)[idx].float() * 1.1).to(torch.bfloat16)
    scaled_set = set(scaled.tolist())
    while True:
        s = int(rng.integers(0, n - burst + 1))
        if not any(p in scaled_set for p in range(s, s + burst)):
            break
    flat[s:s + burst] = float("inf")
    return Workload("bf16 4x8192x8192", torch.bfloat16, [Case(cand, ref)], [(1e-2, 1.6e-2, 0)],
                    tile=(128, 128), k=64,
                    meta={"scaled": scaled, "burst": (s, s + burst)})


# --------------------------------------------------------------------------- 4
CONFIG4_FIXED_SHAPES = [(1, 7), (3, 1000003), (257, 513), (1, 1), (1, 16777216)]
CONFIG4_TOLS = [(1e-6, 1e-6, 0), (1e-5, 1e-5, 0), (1e-4, 1e-4, 0), (1e-3, 1e-3, 0)]


def fp32_sweep_shapes(n_cases: int = 500, max_log2: int = 24, seed: int | None = None,
                   fixed=CONFIG4_FIXED_SHAPES):
    """Seeded odd shapes: log2(numel) ~ U(0, max_log2), R = 2^U(0, log2 numel),
    C = ceil(numel / R) forced odd, R*C <= 2^max_log2. The fixed shapes come
    first."""
    seed = config_seed(4) if seed is None else seed
    rng = _rng(seed)
    cap = 1 << max_log2
    shapes = [s for s in fixed if s[0] * s[1] <= cap][:n_cases]
    while len(shapes) < n_cases:
        u = rng.uniform(0.0, max_log2)
        numel = max(1, int(2.0 ** u))
        v = rng.uniform(0.0, math.log2(numel)) if numel > 1 else 0.0
        r = max(1, int(2.0 ** v))
        c = -(-numel // r)
        if c % 2 == 0:
            c += 1
        while r * c > cap and c > 1:
            c -= 2
        shapes.append((r, c))
    return shapes


def _aligned_offsets(sizes, align_elems: int):
    offs, cur = [], 0
    for n in sizes:
        offs.append(cur)
        cur += -(-n // align_elems) * align_elems if n else align_elems
    return offs, cur


def fp32_sweep(device="cuda", n_cases: int = 500, max_log2: int = 24, tile: int = 64,
            n_cauchy: int = 50, n_faulted: int = 250, seed: int | None = None,
            fixed=CONFIG4_FIXED_SHAPES) -> Workload:
    """fp32 coverage sweep. ref ~ N(0,1) except n_cauchy seeded cases with
    ref = clip(Cauchy(0,1), +-1e4); cand = ref + 1e-5 N(0,1); n_faulted
    seeded cases get m = min(U{1..4}, elements in the last tile) faults at
    distinct seeded positions of the last (bottom-right, usually partial) tile:
    cand = ref + 0.5 (1 + |ref|). Four tolerance pairs 1e-6 .. 1e-3, primary
    pair (1e-3, 1e-3), 64x64 tiles, first-k = 64. Cases are packed into one
    buffer at 256-byte aligned offsets."""
    seed = config_seed(4) if seed is None else seed
    shapes = fp32_sweep_shapes(n_cases, max_log2, seed, fixed)
    rng = _rng(seed + 100000)
    cauchy = set(rng.choice(n_cases, size=min(n_cauchy, n_cases), replace=False).tolist())
    faulted = set(rng.choice(n_cases, size=min(n_faulted, n_cases), replace=False).tolist())
    sizes = [r * c for r, c in shapes]
    offs, total = _aligned_offsets(sizes, 64)
    ref_buf = torch.empty(total, device=device, dtype=torch.float32)
    cand_buf = torch.empty(total, device=device, dtype=torch.float32)
    cases, faults = [], []
    for i, (r, c) in enumerate(shapes):
        n = r * c
        g = _gen(device, seed + i)
        ref = ref_buf[offs[i]:offs[i] + n].view(r, c)
        cand = cand_buf[offs[i]:offs[i] + n].view(r, c)
        if i in cauchy:
            ref.cauchy_(generator=g).clamp_(-1e4, 1e4)
        else:
            ref.normal_(generator=g)
        cand.copy_(ref + 1e-5 * torch.randn(r, c, generator=g, device=device, dtype=torch.float32))
        pos = np.zeros(0, dtype=np.int64)
        if i in faulted:
            frng = _rng(seed + 200000 + i)
            r0 = ((r - 1) // tile) * tile
            c0 = ((c - 1) // tile) * tile
            th, tw = r - r0, c - c0
            m = min(int(frng.integers(1, 5)), th * tw)
            local = _distinct(frng, th * tw, m)
            pos = np.array(sorted((r0 + l // tw) * c + (c0 + l % tw) for l in local), dtype=np.int64)
            idx = torch.as_tensor(pos, device=device)
            rv = ref.view(-1)[idx]
            cand.view(-1)[idx] = rv + 0.5 * (1.0 + rv.abs())
        cases.append(Case(cand, ref))
        faults.append(pos)
    return Workload("fp32 sweep 500 odd shapes", torch.float32, cases, list(CONFIG4_TOLS),
                    primary=3, tile=(tile, tile), k=64,
                    meta={"faults": faults, "cauchy": sorted(cauchy), "faulted": sorted(faulted),
                          "shapes": shapes})


# --------------------------------------------------------------------------- 5
CLASS_CORRECT, CLASS_COPY, CLASS_ZERO, CLASS_CONSTANT, CLASS_BF16 = range(5)
CLASS_NAMES = ["correct", "input_copy", "all_zero", "constant", "bf16_computed"]


def fp32_integrity_classes(n_cases: int = 256, seed: int | None = None) -> np.ndarray:
    """Seeded shuffle of n slots assigning class (slot mod 5)."""
    seed = config_seed(5) if seed is None else seed
    classes = np.arange(n_cases) % 5
    _rng(seed + 100000).shuffle(classes)
    return classes


def fp32_integrity(device="cuda", n_cases: int = 256, rows: int = 4096, cols: int = 4096,
            seed: int | None = None) -> Workload:
    """fp32 integrity batch. Per case: x ~ N(0,1), ref = x*0.5 + 1 (fp32);
    cand by class: correct = ref + 1e-7 N(0,1); input copy = x; all-zero;
    constant fill 1.0; bf16-computed = fp32(bf16(bf16(bf16(x)*0.5) + 1)).
    atol = rtol = 1e-5; the detectors get x as operator input 0."""
    seed = config_seed(5) if seed is None else seed
    classes = fp32_integrity_classes(n_cases, seed)
    x_all = torch.empty(n_cases, rows, cols, device=device, dtype=torch.float32)
    ref_all = torch.empty_like(x_all)
    cand_all = torch.empty_like(x_all)
    for i in range(n_cases):
        g = _gen(device, seed + i)
        x = x_all[i]
        x.normal_(generator=g)
        ref_all[i] = x * 0.5 + 1.0
        k = int(classes[i])
        if k == CLASS_CORRECT:
            cand_all[i] = ref_all[i] + 1e-7 * torch.randn(rows, cols, generator=g, device=device,
                                                          dtype=torch.float32)
        elif k == CLASS_COPY:
            cand_all[i] = x
        elif k == CLASS_ZERO:
            cand_all[i].zero_()
        elif k == CLASS_CONSTANT:
            cand_all[i].fill_(1.0)
        else:
            cand_all[i] = ((x.to(torch.bfloat16) * 0.5).to(torch.bfloat16) + 1.0
                           ).to(torch.bfloat16).float()
    cases = [Case(cand_all[i], ref_all[i], [x_all[i]]) for i in range(n_cases)]
    return Workload("fp32 integrity 256x4096x4096", torch.float32, cases, [(1e-5, 1e-5, 0)],
                    integrity=True, meta={"classes": classes})


WORKLOADS = {1: fp32_single, 2: fp16_batch, 3: bf16_bursts, 4: fp32_sweep, 5: fp32_integrity}


def raw_numpy(t: torch.Tensor) -> np.ndarray:
    """Host copy of a tensor's raw storage: float32, or uint16 bit patterns."""
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.float32:
        return t.numpy()
    if t.dtype in (torch.float16, torch.bfloat16):
        return t.view(torch.int16).numpy().view(np.uint16)
    raise TypeError("unsupported dtype %s" % t.dtype)


def dtype_code(dt: torch.dtype) -> int:
    return {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}[dt]
