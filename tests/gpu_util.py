"""Helpers for the GPU parity tests: seeded inputs -> device tensors, calls through the
C ABI (paper_2601_20595_amd), results -> fp64 numpy for comparison with the oracle."""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

import oracle
import paper_2601_20595_amd as csg
import seeded_inputs as si

DEV = "cuda:0"
BF16_NAN = np.uint16(0x7FC0)


def to_dev(arr: np.ndarray) -> torch.Tensor:
    if arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16).copy()).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(arr).copy()).to(DEV)


def out_to_f64(t: torch.Tensor, dtype: str) -> np.ndarray:
    a = t.cpu().numpy()
    if dtype == "bf16":
        return si.bf16_bits_to_f32(a.view(np.uint16)).astype(np.float64)
    return a.astype(np.float64)


def bf16_rne_of_f64(x: np.ndarray) -> np.ndarray:
    """Round exactly-representable-in-fp32 values to bf16 (RNE), returned as fp64."""
    return si.bf16_bits_to_f32(si.f32_to_bf16_bits(x.astype(np.float32))).astype(np.float64)


def empty_out(M: int, N: int, dtype: str) -> torch.Tensor:
    return torch.empty((M, N), dtype=torch.int16 if dtype == "bf16" else torch.float32, device=DEV)


def nan_fill_(t: torch.Tensor) -> None:
    if t.dtype == torch.int16:
        t.fill_(int(BF16_NAN))
    else:
        t.fill_(float("nan"))


@dataclass
class Streams:
    compute: torch.cuda.Stream
    copy: torch.cuda.Stream


def streams() -> Streams:
    return Streams(torch.cuda.Stream(device=DEV), torch.cuda.Stream(device=DEV))


def sample_rows(chunks, extra: int, seed: int, M: int):
    """First and last row of every chunk plus `extra` random rows."""
    rows = set()
    for c in chunks:
        rows.add(c.row_begin)
        rows.add(c.row_end - 1)
    rng = np.random.default_rng(seed)
    rows.update(int(r) for r in rng.integers(0, M, size=extra))
    return sorted(rows)


def run_ag(plan: csg.Plan, chunks, A: si.Matrix, B: si.Matrix, out_dtype: str, mode: str = "overlap",
           poison_remote: bool = False, touch_remote: bool = False, st: Optional[Streams] = None,
           repeats: int = 1):
    """AllGather + GEMM (or grouped) through the C ABI. landing holds the local rows,
    staging the whole A; returns (C tensor, landing tensor)."""
    M, K = A.values.shape
    N = B.values.shape[-2]
    st = st or streams()
    a_full = to_dev(A.device_array)
    landing = a_full.clone()
    for c in chunks:
        # compute-only moves nothing: the landing buffer must already hold every row
        if not c.is_local and mode != "compute_only":
            if poison_remote:
                nan_fill_(landing[c.row_begin:c.row_end])
            else:
                landing[c.row_begin:c.row_end].zero_()
    if touch_remote:
        # read the poisoned rows so their lines sit in the caches before the call
        _ = landing.float().sum().item() if landing.dtype != torch.int16 else landing.sum().item()
    b = to_dev(B.device_array)
    c = empty_out(M, N, out_dtype)
    nan_fill_(c)
    torch.cuda.synchronize()
    for _ in range(repeats):
        if plan.op == "grouped":
            plan.grouped_gemm(landing, a_full, b, c, mode, st.compute, st.copy)
        else:
            plan.ag_gemm(landing, a_full, b, c, mode, st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    return c, landing


def run_rs(plan: csg.Plan, A: si.Matrix, B: si.Matrix, out_dtype: str, mode: str = "overlap",
           st: Optional[Streams] = None, repeats: int = 1):
    M, K = A.values.shape
    N = B.values.shape[0]
    st = st or streams()
    a = to_dev(A.device_array)
    b = to_dev(B.device_array)
    c = empty_out(M, N, out_dtype)
    nan_fill_(c)
    out = empty_out(M, N, out_dtype)
    out.zero_()
    torch.cuda.synchronize()
    for _ in range(repeats):
        plan.gemm_rs(a, b, c, out, mode, st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    return c, out


def tol_for(out_dtype: str, in_dtype: str) -> float:
    # bound on oracle.max_rel_error: 2e-2 when bf16 is involved, 1e-4 for fp32 end to end
    return 2e-2 if (out_dtype == "bf16" or in_dtype == "bf16") else 1e-4


def assert_close(G: np.ndarray, R: np.ndarray, tol: float, what: str = ""):
    assert not np.isnan(G).any(), "NaN in GPU result " + what
    err = oracle.max_rel_error(G, R)
    assert err <= tol, "%s: max rel error %.3g > %.3g" % (what, err, tol)
    return err
