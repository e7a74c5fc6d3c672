"""Parity margins recorded by the GPU tests (shared with conftest's summary).

One entry per (case, tensor): the worst per-slice relative errors and the
tolerance they were held to.  conftest prints them in the terminal summary,
so a `pytest -q` log carries them, and writes parity_margins.json into the
results folder it names, when that folder exists.
"""
from __future__ import annotations

import numpy as np

MARGINS: list[dict] = []


def slice_errors(got, ref) -> tuple[float, float]:
    """(max|got - ref| / max|ref|, rms(got - ref) / rms(ref)) of one slice."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    diff = got - ref
    mx = float(np.abs(diff).max() / max(np.abs(ref).max(), 1e-30)) if diff.size else 0.0
    rms = float(np.sqrt((diff ** 2).mean()) / max(np.sqrt((ref ** 2).mean()), 1e-30)) if diff.size else 0.0
    return mx, rms


def record(case: str, tensor: str, max_rel: float, rms_rel: float, tol: float, slices: int) -> None:
    MARGINS.append(dict(case=case, tensor=tensor, max_rel=float(max_rel), rms_rel=float(rms_rel),
                        tol=float(tol), slices=int(slices)))
