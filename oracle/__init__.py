"""CPU oracle for the Fast Multipole Attention forward pass (test infrastructure).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  Nothing here imports the product
package and the product never imports this package.

The arithmetic lives in ``fma_oracle.c`` (plain C, double precision, OpenMP),
written from Section 3 of the paper (Eq. agg1d, Eq. fma1d, Eq. agg2d,
Eq. fma2d and the set-builder definitions of the near and far fields).  This
module only marshals numpy arrays in and out of it.  ``brute.py`` holds a
second, independent formulation (per-row sets in pure Python and a dense
masked softmax over augmented keys) used to pin this one.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fma_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle_fma.so")
_lib = None

NORM_JOINT = 0      # one softmax over near tokens and far groups together
NORM_PER_SET = 1    # printed form: alpha over N(i), beta^l over G_l(i)


def build_oracle(force: bool = True) -> str:
    """Compile the C oracle with gcc (OpenMP).  Returns the library path."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fopenmp", "-shared",
             "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or (
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
        build_oracle(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    i64, i32, dp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
    lib.fmao_num_levels.argtypes = [i64]
    lib.fmao_num_levels.restype = ctypes.c_int
    lib.fmao_coarse_rows_1d.argtypes = [i64, i64]
    lib.fmao_coarse_rows_1d.restype = i64
    lib.fmao_coarse_rows_2d.argtypes = [i64, i64]
    lib.fmao_coarse_rows_2d.restype = i64
    lib.fmao_lists_1d.argtypes = [i64, i64, i32, dp, dp, dp]
    lib.fmao_lists_1d.restype = ctypes.c_int
    lib.fmao_lists_2d.argtypes = [i64, i64, i32, dp]
    lib.fmao_lists_2d.restype = ctypes.c_int
    lib.fmao_labels_1d.argtypes = [i64, i64, i64, dp]
    lib.fmao_labels_1d.restype = ctypes.c_int
    lib.fmao_labels_2d.argtypes = [i64, i64, i64, dp]
    lib.fmao_labels_2d.restype = ctypes.c_int
    lib.fmao_coarsen_1d.argtypes = [dp, i64, i64, i64, i64, dp, dp]
    lib.fmao_coarsen_1d.restype = ctypes.c_int
    lib.fmao_coarsen_2d.argtypes = [dp, i64, i64, i64, i64, dp, dp]
    lib.fmao_coarsen_2d.restype = ctypes.c_int
    lib.fmao_forward_1d.argtypes = [dp, dp, dp, i64, i64, i64, i64, ctypes.c_int, i64,
                                    dp, dp, dp, i64, ctypes.c_double, ctypes.c_int, dp, dp]
    lib.fmao_forward_1d.restype = ctypes.c_int
    lib.fmao_forward_2d.argtypes = [dp, dp, dp, i64, i64, i64, i64, i64,
                                    dp, dp, dp, i64, ctypes.c_double, ctypes.c_int, dp, dp]
    lib.fmao_backward_1d.argtypes = [dp, dp, dp, i64, i64, i64, i64, ctypes.c_int, i64, dp, dp, i64,
                                     ctypes.c_double, ctypes.c_int, dp, dp, dp, dp, dp, dp]
    lib.fmao_backward_1d.restype = ctypes.c_int
    lib.fmao_backward_2d.argtypes = [dp, dp, dp, i64, i64, i64, i64, i64, dp, dp, i64,
                                     ctypes.c_double, ctypes.c_int, dp, dp, dp, dp, dp, dp]
    lib.fmao_backward_2d.restype = ctypes.c_int
    lib.fmao_backward_linear_1d.argtypes = [dp, dp, dp, i64, i64, i64, i64, dp, dp, dp, i64, ctypes.c_double,
                                            dp, dp, dp, dp, dp, dp, dp]
    lib.fmao_backward_linear_1d.restype = ctypes.c_int
    lib.fmao_backward_linear_2d.argtypes = [dp, dp, dp, i64, i64, i64, i64, dp, dp, dp, i64, ctypes.c_double,
                                            dp, dp, dp, dp, dp, dp, dp]
    lib.fmao_backward_linear_2d.restype = ctypes.c_int
    lib.fmao_forward_2d.restype = ctypes.c_int
    # 2D maps of H rows and W columns
    lib.fmao_coarse_rows_2d_hw.argtypes = [i64, i64, i64]
    lib.fmao_coarse_rows_2d_hw.restype = i64
    lib.fmao_lists_2d_hw.argtypes = [i64, i64, i64, i32, dp]
    lib.fmao_lists_2d_hw.restype = ctypes.c_int
    lib.fmao_labels_2d_hw.argtypes = [i64, i64, i64, i64, dp]
    lib.fmao_labels_2d_hw.restype = ctypes.c_int
    lib.fmao_coarsen_2d_hw.argtypes = [dp, i64, i64, i64, i64, i64, dp, dp]
    lib.fmao_coarsen_2d_hw.restype = ctypes.c_int
    lib.fmao_forward_2d_hw.argtypes = [dp, dp, dp, i64, i64, i64, i64, i64, i64,
                                       dp, dp, dp, i64, ctypes.c_double, ctypes.c_int, dp, dp]
    lib.fmao_forward_2d_hw.restype = ctypes.c_int
    lib.fmao_backward_2d_hw.argtypes = [dp, dp, dp, i64, i64, i64, i64, i64, i64, dp, dp, i64,
                                        ctypes.c_double, ctypes.c_int, dp, dp, dp, dp, dp, dp]
    lib.fmao_backward_2d_hw.restype = ctypes.c_int
    lib.fmao_backward_linear_2d_hw.argtypes = [dp, dp, dp, i64, i64, i64, i64, i64, dp, dp, dp, i64,
                                               ctypes.c_double, dp, dp, dp, dp, dp, dp, dp]
    lib.fmao_backward_linear_2d_hw.restype = ctypes.c_int
    _lib = lib
    return lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str) -> None:
    if rc != 0:
        names = {1: "bad argument", 2: "near/far sets do not cover the sequence",
                 3: "host allocation failed"}
        raise RuntimeError("oracle %s failed: %s" % (what, names.get(rc, rc)))


# ----------------------------------------------------------------- geometry
def num_levels(ratio: int) -> int:
    """L = ceil(log2(ratio)), 0 for ratio <= 1 (Sec. 3)."""
    return _load().fmao_num_levels(int(ratio))


def coarse_rows_1d(n: int, r: int) -> int:
    return int(_load().fmao_coarse_rows_1d(n, r))


def coarse_rows_2d(W: int, r: int, H: int | None = None) -> int:
    """Coarse rows of a map of H rows (default W) and W columns."""
    return int(_load().fmao_coarse_rows_2d_hw(W if H is None else H, W, r))


def levels_2d(W: int, r: int, H: int | None = None) -> int:
    """L of an H x W map: the longer side sets the depth (reading R19)."""
    H = W if H is None else H
    return num_levels(max(H, W) // r)


# --------------------------------------------------------------- index sets
def lists_1d(n: int, r: int, kcap: int = 3):
    """Per base block b: int32 [nb][L-1][kcap] ascending group indices of
    G_l(i) (padded with -1), plus the near-field token range [lo, hi)."""
    nb = n // r
    L = num_levels(nb)
    out = np.full((nb, max(L - 1, 0), kcap), -1, dtype=np.int32)
    lo = np.zeros(nb, dtype=np.int64)
    hi = np.zeros(nb, dtype=np.int64)
    _check(_load().fmao_lists_1d(n, r, kcap, _ptr(out), _ptr(lo), _ptr(hi)), "lists_1d")
    return out, lo, hi


def lists_2d(W: int, r: int, kcap: int = 27, H: int | None = None):
    """Per base cell (row-major cell index, H/r rows of W/r cells): int32
    [ncell][L-1][kcap] ascending square indices u*My_l+v of Q_l(i), padded
    with -1 (My_l = squares per map row)."""
    H = W if H is None else H
    L = levels_2d(W, r, H)
    out = np.full(((H // r) * (W // r), max(L - 1, 0), kcap), -1, dtype=np.int32)
    _check(_load().fmao_lists_2d_hw(H, W, r, kcap, _ptr(out)), "lists_2d")
    return out


def labels_1d(n: int, r: int, i: int) -> np.ndarray:
    lab = np.zeros(n, dtype=np.int8)
    _check(_load().fmao_labels_1d(n, r, i, _ptr(lab)), "labels_1d")
    return lab


def labels_2d(W: int, r: int, i: int, H: int | None = None) -> np.ndarray:
    H = W if H is None else H
    lab = np.zeros(H * W, dtype=np.int8)
    _check(_load().fmao_labels_2d_hw(H, W, r, i, _ptr(lab)), "labels_2d")
    return lab


# --------------------------------------------------------------- coarsening
def coarsen_1d(x, r: int, pi, rank: int = 1) -> np.ndarray:
    """x [n, d], pi (concatenated per level, rank bases per level) ->
    [rank*R, d] (Eq. agg1d; rows level, basis, group)."""
    x = _f64(x)
    pi = _f64(pi)
    n, d = x.shape
    _check_wlen(pi, weight_len_1d(n, r, rank), "coarsen_1d")
    out = np.zeros((max(rank * coarse_rows_1d(n, r), 0), d))
    _check(_load().fmao_coarsen_1d(_ptr(x), n, d, r, rank, _ptr(pi), _ptr(out)), "coarsen_1d")
    return out


def coarsen_2d(x, W: int, r: int, pi, rank: int = 1, H: int | None = None) -> np.ndarray:
    """x [H*W, d] (H defaults to W), pi (per level and basis [pi_x | pi_y])
    -> [rank*R, d] (Eq. agg2d; rows level, basis, square)."""
    H = W if H is None else H
    x = _f64(x)
    pi = _f64(pi)
    d = x.shape[1]
    _check_wlen(pi, weight_len_2d(W, r, rank, H), "coarsen_2d")
    out = np.zeros((max(rank * coarse_rows_2d(W, r, H), 0), d))
    _check(_load().fmao_coarsen_2d_hw(_ptr(x), H, W, d, r, rank, _ptr(pi), _ptr(out)), "coarsen_2d")
    return out


# ------------------------------------------------------------------ forward
def _slices(q, k, v):
    q, k, v = _f64(q), _f64(k), _f64(v)
    if q.shape != k.shape or q.shape != v.shape:
        raise ValueError("q, k, v must have one shape")
    lead = q.shape[:-2]
    n, d = q.shape[-2:]
    S = int(np.prod(lead)) if lead else 1
    return q.reshape(S, n, d), k.reshape(S, n, d), v.reshape(S, n, d), lead, S, n, d


def _weights(w, S, lead, heads_axis):
    """Weights are [H, wlen] (per head) or [wlen] (shared).  Returns an
    array indexed by slice with a stride (0 when shared)."""
    w = _f64(w)
    if w.ndim == 1:
        return w, 0
    # per-head weights: broadcast over the batch axis
    H = w.shape[0]
    if not lead or lead[-1] != H:
        raise ValueError("per-head weights need the head axis last before (n, d)")
    reps = S // H
    full = np.ascontiguousarray(np.broadcast_to(w[None], (reps, H, w.shape[1])).reshape(S, -1))
    return full, full.shape[1]


def weight_len_1d(n: int, r: int, rank: int = 1) -> int:
    """Length of one head's 1D weights: rank * sum_l s_l."""
    L = num_levels(n // r)
    return rank * r * (2 ** (L - 1) - 1) if L > 1 else 0


def weight_len_2d(W: int, r: int, rank: int = 1, H: int | None = None) -> int:
    """Length of one head's 2D weights: rank * sum_l 2 s_l."""
    L = levels_2d(W, r, H)
    return rank * 2 * r * (2 ** (L - 1) - 1) if L > 1 else 0


def _check_wlen(w, want, what):
    if w.shape[-1] != want:
        raise ValueError(f"{what}: weights of length {w.shape[-1]}, need {want}")


def forward_1d(q, k, v, r: int, pik=None, piv=None, causal: bool = False,
               scale: float | None = None, norm: int = NORM_JOINT,
               return_counts: bool = False, rank: int = 1, piq=None):
    """FMA 1D forward (Eq. fma1d) in float64.  q, k, v: [..., n, d];
    rank = p basis vectors per level (Sec. 3, coarse level rank p);
    piq: query aggregation weights (FMA-linear, laid out like pik)."""
    qs, ks, vs, lead, S, n, d = _slices(q, k, v)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    L = num_levels(n // r) if n % r == 0 else 0
    wk = wv = wq = None
    stride = 0
    if L > 1:
        wk, stride = _weights(pik, S, lead, -1)
        wv, stride_v = _weights(piv, S, lead, -1)
        assert stride == stride_v
        _check_wlen(wk, weight_len_1d(n, r, rank), "forward_1d")
        _check_wlen(wv, weight_len_1d(n, r, rank), "forward_1d")
        if piq is not None:
            wq, stride_q = _weights(piq, S, lead, -1)
            assert stride_q == stride
            _check_wlen(wq, weight_len_1d(n, r, rank), "forward_1d")
    o = np.zeros_like(qs)
    counts = np.zeros((S, n), dtype=np.int64)
    _check(_load().fmao_forward_1d(_ptr(qs), _ptr(ks), _ptr(vs), S, n, d, r, int(bool(causal)), int(rank),
                                   _ptr(wk), _ptr(wv), _ptr(wq), stride, float(scale), int(norm),
                                   _ptr(o), _ptr(counts)), "forward_1d")
    o = o.reshape(*lead, n, d) if lead else o.reshape(n, d)
    if return_counts:
        return o, counts.reshape(*lead, n) if lead else counts.reshape(n)
    return o


def forward_2d(q, k, v, W: int, r: int, pik=None, piv=None,
               scale: float | None = None, norm: int = NORM_JOINT,
               return_counts: bool = False, rank: int = 1, piq=None, H: int | None = None):
    """FMA 2D forward (Eq. fma2d) in float64.  q, k, v: [..., H*W, d] (a
    map of H rows, default W, and W columns; token x*W + y);
    rank = p basis pairs per level (Sec. 3, coarse level rank p);
    piq: query aggregation weights (FMA-linear, laid out like pik)."""
    H = W if H is None else H
    qs, ks, vs, lead, S, n, d = _slices(q, k, v)
    if n != H * W:
        raise ValueError("2D inputs need n == H*W")
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    L = levels_2d(W, r, H) if W % r == 0 and H % r == 0 else 0
    wk = wv = wq = None
    stride = 0
    if L > 1:
        wk, stride = _weights(pik, S, lead, -1)
        wv, _ = _weights(piv, S, lead, -1)
        _check_wlen(wk, weight_len_2d(W, r, rank, H), "forward_2d")
        _check_wlen(wv, weight_len_2d(W, r, rank, H), "forward_2d")
        if piq is not None:
            wq, _ = _weights(piq, S, lead, -1)
            _check_wlen(wq, weight_len_2d(W, r, rank, H), "forward_2d")
    o = np.zeros_like(qs)
    counts = np.zeros((S, n), dtype=np.int64)
    _check(_load().fmao_forward_2d_hw(_ptr(qs), _ptr(ks), _ptr(vs), S, H, W, d, r, int(rank),
                                   _ptr(wk), _ptr(wv), _ptr(wq), stride, float(scale), int(norm),
                                   _ptr(o), _ptr(counts)), "forward_2d")
    o = o.reshape(*lead, n, d) if lead else o.reshape(n, d)
    if return_counts:
        return o, counts.reshape(*lead, n) if lead else counts.reshape(n)
    return o


# ----------------------------------------------------------------- backward
def _weight_grads(dw_slices, w, S, lead):
    """Per-slice weight gradients [S, wlen] -> the shape of the weights given
    to the forward: per head [H, wlen] (summed over the batch) or shared
    [wlen] (summed over every slice)."""
    w = _f64(w)
    if w.ndim == 1:
        return dw_slices.sum(axis=0)
    H = w.shape[0]
    return dw_slices.reshape(S // H, H, -1).sum(axis=0)


def backward_1d(q, k, v, r: int, pik, piv, dout, causal: bool = False, scale: float | None = None,
                norm: int = NORM_JOINT, rank: int = 1, piq=None):
    """Gradients of sum(dout * forward_1d(...)) in float64: (dq, dk, dv,
    dpik, dpiv), weights shaped like pik / piv (None when L <= 1).  With piq
    (FMA-linear, reading R18: bidirectional, rank 1, joint normalisation) a
    sixth entry, dpiq, follows."""
    qs, ks, vs, lead, S, n, d = _slices(q, k, v)
    dos = _f64(dout).reshape(S, n, d).copy()
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    L = num_levels(n // r) if n % r == 0 else 0
    wk = wv = None
    stride = 0
    wl = weight_len_1d(n, r, rank) if L > 1 else 0
    if L > 1:
        wk, stride = _weights(pik, S, lead, -1)
        wv, _ = _weights(piv, S, lead, -1)
        _check_wlen(wk, wl, "backward_1d")
        _check_wlen(wv, wl, "backward_1d")
    dq, dk, dv = np.zeros_like(qs), np.zeros_like(qs), np.zeros_like(qs)
    dwk = np.zeros((S, max(wl, 1)))
    dwv = np.zeros((S, max(wl, 1)))
    dwq = np.zeros((S, max(wl, 1)))
    if piq is not None:
        if causal or rank != 1 or norm != NORM_JOINT:
            raise ValueError("FMA-linear is bidirectional, rank 1, joint normalisation")
        wq = None
        if L > 1:
            wq, _ = _weights(piq, S, lead, -1)
            _check_wlen(wq, wl, "backward_1d")
        else:
            wq = np.zeros((1, 1))
        _check(_load().fmao_backward_linear_1d(_ptr(qs), _ptr(ks), _ptr(vs), S, n, d, r, _ptr(wk), _ptr(wv),
                                               _ptr(wq), stride, float(scale), _ptr(dos), _ptr(dq), _ptr(dk),
                                               _ptr(dv), _ptr(dwk), _ptr(dwv), _ptr(dwq)), "backward_1d")
    else:
        _check(_load().fmao_backward_1d(_ptr(qs), _ptr(ks), _ptr(vs), S, n, d, r, int(bool(causal)), int(rank),
                                        _ptr(wk), _ptr(wv), stride, float(scale), int(norm), _ptr(dos),
                                        _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dwk), _ptr(dwv)), "backward_1d")
    shp = (*lead, n, d) if lead else (n, d)
    out = [dq.reshape(shp), dk.reshape(shp), dv.reshape(shp)]
    if L > 1:
        out += [_weight_grads(dwk[:, :wl], pik, S, lead), _weight_grads(dwv[:, :wl], piv, S, lead)]
        if piq is not None:
            out.append(_weight_grads(dwq[:, :wl], piq, S, lead))
    else:
        out += [None, None] + ([None] if piq is not None else [])
    return tuple(out)


def backward_2d(q, k, v, W: int, r: int, pik, piv, dout, scale: float | None = None,
                norm: int = NORM_JOINT, rank: int = 1, piq=None, H: int | None = None):
    """2D analogue of backward_1d (piq: FMA-linear, a sixth entry dpiq; H:
    map rows, default W)."""
    H = W if H is None else H
    qs, ks, vs, lead, S, n, d = _slices(q, k, v)
    if n != H * W:
        raise ValueError("2D inputs need n == H*W")
    dos = _f64(dout).reshape(S, n, d).copy()
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    L = levels_2d(W, r, H) if W % r == 0 and H % r == 0 else 0
    wk = wv = None
    stride = 0
    wl = weight_len_2d(W, r, rank, H) if L > 1 else 0
    if L > 1:
        wk, stride = _weights(pik, S, lead, -1)
        wv, _ = _weights(piv, S, lead, -1)
        _check_wlen(wk, wl, "backward_2d")
        _check_wlen(wv, wl, "backward_2d")
    dq, dk, dv = np.zeros_like(qs), np.zeros_like(qs), np.zeros_like(qs)
    dwk = np.zeros((S, max(wl, 1)))
    dwv = np.zeros((S, max(wl, 1)))
    dwq = np.zeros((S, max(wl, 1)))
    if piq is not None:
        if rank != 1 or norm != NORM_JOINT:
            raise ValueError("FMA-linear is rank 1, joint normalisation")
        if L > 1:
            wq, _ = _weights(piq, S, lead, -1)
            _check_wlen(wq, wl, "backward_2d")
        else:
            wq = np.zeros((1, 1))
        _check(_load().fmao_backward_linear_2d_hw(_ptr(qs), _ptr(ks), _ptr(vs), S, H, W, d, r, _ptr(wk), _ptr(wv),
                                               _ptr(wq), stride, float(scale), _ptr(dos), _ptr(dq), _ptr(dk),
                                               _ptr(dv), _ptr(dwk), _ptr(dwv), _ptr(dwq)), "backward_2d")
    else:
        _check(_load().fmao_backward_2d_hw(_ptr(qs), _ptr(ks), _ptr(vs), S, H, W, d, r, int(rank),
                                        _ptr(wk), _ptr(wv), stride, float(scale), int(norm), _ptr(dos),
                                        _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dwk), _ptr(dwv)), "backward_2d")
    shp = (*lead, n, d) if lead else (n, d)
    out = [dq.reshape(shp), dk.reshape(shp), dv.reshape(shp)]
    if L > 1:
        out += [_weight_grads(dwk[:, :wl], pik, S, lead), _weight_grads(dwv[:, :wl], piv, S, lead)]
        if piq is not None:
            out.append(_weight_grads(dwq[:, :wl], piq, S, lead))
    else:
        out += [None, None] + ([None] if piq is not None else [])
    return tuple(out)
