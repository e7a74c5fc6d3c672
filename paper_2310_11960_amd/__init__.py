"""MI355X (gfx950) Fast Multipole Attention forward pass.

Thin ctypes binding of the C ABI in include/fma.h (libfma_mi355x.so, built by
``paper_2310_11960_amd.build``).  The functions ``fma_*`` below carry the C
names and only marshal arguments: every step of the computation runs in the
library's HIP kernels.  PyTorch supplies device memory and the current
stream.  There is no CPU fallback: without the built library every call
raises.

High-level use::

    op = FMA(ndim=1, batch=B, heads=H, seq_len=n, block=128, causal=True,
             dtype=torch.bfloat16)
    out = op.forward(q, k, v, wk, wv)        # q, k, v: [B, H, n, d] on cuda
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfma_mi355x.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "fma.h")

FMA_OK = 0
FMA_ERR_NULL = 1
FMA_ERR_SHAPE = 2
FMA_ERR_UNSUPPORTED = 3
FMA_ERR_WORKSPACE = 4
FMA_ERR_HIP = 5
FMA_ERR_HOST_ALLOC = 6
FMA_ERR_ALIGN = 7
FMA_ERR_ARG = 8
FMA_F32 = 0
FMA_BF16 = 1
FMA_NORM_JOINT = 0
FMA_NORM_PER_LEVEL = 1

HEAD_DIM = 64


class FmaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("FMA status %d: %s" % (status, message))
        self.status = status


class fma_desc_t(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_int32),
        ("ndim", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("heads", ctypes.c_int32),
        ("seq_len", ctypes.c_int64),
        ("side", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block", ctypes.c_int32),
        ("num_levels", ctypes.c_int32),
        ("causal", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("weights_per_head", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("rank", ctypes.c_int32),
        ("norm", ctypes.c_int32),
        ("query_downsample", ctypes.c_int32),
    ]


_lib = None


def library() -> ctypes.CDLL:
    """Load the built HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libfma_mi355x.so is not built; run `python -m paper_2310_11960_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, st, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int32, ctypes.c_int64
    lib.fma_plan.argtypes = [ctypes.POINTER(fma_desc_t), ctypes.POINTER(vp)]
    lib.fma_destroy.argtypes = [vp]
    lib.fma_workspace_size.argtypes = [vp, ctypes.POINTER(ctypes.c_size_t)]
    lib.fma_weights_len.argtypes = [vp, ctypes.POINTER(i64)]
    lib.fma_coarse_rows.argtypes = [vp, ctypes.POINTER(i64)]
    lib.fma_num_levels.argtypes = [vp, ctypes.POINTER(i32)]
    for name in ("fma_forward_1d", "fma_forward_2d"):
        getattr(lib, name).argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.fma_coarsen.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.fma_attend.argtypes = [vp, vp, vp, vp, vp, ctypes.c_size_t, vp, vp]
    lib.fma_interaction_lists.argtypes = [vp, vp, vp]
    lib.fma_dense_reference.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.fma_backward_workspace_size.argtypes = [vp, ctypes.POINTER(ctypes.c_size_t)]
    lib.fma_forward_linear.argtypes = [vp] * 9 + [ctypes.c_size_t, vp]
    lib.fma_backward.argtypes = [vp] + [vp] * 12 + [vp, ctypes.c_size_t, vp]
    lib.fma_backward_linear.argtypes = [vp] + [vp] * 14 + [vp, ctypes.c_size_t, vp]
    lib.fma_forward_static.argtypes = [vp] * 8
    lib.fma_stream_reference.argtypes = [vp, ctypes.c_size_t, vp, ctypes.c_size_t, i32, vp]
    lib.fma_plan_params.argtypes = [vp, ctypes.POINTER(i64), i32, ctypes.POINTER(i32)]
    for name in ("fma_plan", "fma_destroy", "fma_workspace_size", "fma_weights_len", "fma_coarse_rows",
                 "fma_num_levels", "fma_forward_1d", "fma_forward_2d", "fma_coarsen", "fma_attend",
                 "fma_interaction_lists", "fma_dense_reference", "fma_backward_workspace_size",
                 "fma_backward", "fma_backward_linear", "fma_forward_linear", "fma_forward_static",
                 "fma_stream_reference", "fma_plan_params"):
        getattr(lib, name).restype = st
    lib.fma_last_error.argtypes = []
    lib.fma_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def header_functions() -> list[str]:
    """Names of the functions include/fma.h declares."""
    text = open(HEADER_PATH).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fma_[a-z0-9_]+)\s*\(", text)))


def _check(status: int) -> None:
    if status != FMA_OK:
        raise FmaError(status, library().fma_last_error().decode())


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---------------------------------------------------------------- C names
def fma_plan(desc: fma_desc_t) -> int:
    h = ctypes.c_void_p()
    _check(library().fma_plan(ctypes.byref(desc), ctypes.byref(h)))
    return h.value


def fma_destroy(plan: int) -> None:
    _check(library().fma_destroy(plan))


def fma_workspace_size(plan: int) -> int:
    x = ctypes.c_size_t()
    _check(library().fma_workspace_size(plan, ctypes.byref(x)))
    return x.value


def fma_weights_len(plan: int) -> int:
    x = ctypes.c_int64()
    _check(library().fma_weights_len(plan, ctypes.byref(x)))
    return x.value


def fma_coarse_rows(plan: int) -> int:
    x = ctypes.c_int64()
    _check(library().fma_coarse_rows(plan, ctypes.byref(x)))
    return x.value


def fma_num_levels(plan: int) -> int:
    x = ctypes.c_int32()
    _check(library().fma_num_levels(plan, ctypes.byref(x)))
    return x.value


def fma_forward_1d(plan, q, k, v, wk, wv, out, workspace, workspace_bytes, stream=None):
    _check(library().fma_forward_1d(plan, _ptr(q), _ptr(k), _ptr(v), _ptr(wk), _ptr(wv), _ptr(out),
                                    _ptr(workspace), workspace_bytes, _stream(stream)))


def fma_forward_2d(plan, q, k, v, wk, wv, out, workspace, workspace_bytes, stream=None):
    _check(library().fma_forward_2d(plan, _ptr(q), _ptr(k), _ptr(v), _ptr(wk), _ptr(wv), _ptr(out),
                                    _ptr(workspace), workspace_bytes, _stream(stream)))


def fma_coarsen(plan, k, v, wk, wv, workspace, workspace_bytes, stream=None):
    _check(library().fma_coarsen(plan, _ptr(k), _ptr(v), _ptr(wk), _ptr(wv), _ptr(workspace),
                                 workspace_bytes, _stream(stream)))


def fma_attend(plan, q, k, v, workspace, workspace_bytes, out, stream=None):
    _check(library().fma_attend(plan, _ptr(q), _ptr(k), _ptr(v), _ptr(workspace), workspace_bytes,
                                _ptr(out), _stream(stream)))


def fma_interaction_lists(plan, dev_out, stream=None):
    _check(library().fma_interaction_lists(plan, _ptr(dev_out), _stream(stream)))


def fma_dense_reference(plan, q, k, v, out, stream=None):
    _check(library().fma_dense_reference(plan, _ptr(q), _ptr(k), _ptr(v), _ptr(out), _stream(stream)))


def fma_forward_linear(plan, q, k, v, wq, wk, wv, out, workspace, workspace_bytes, stream=None):
    _check(library().fma_forward_linear(plan, _ptr(q), _ptr(k), _ptr(v), _ptr(wq), _ptr(wk), _ptr(wv), _ptr(out),
                                        _ptr(workspace), workspace_bytes, _stream(stream)))


def fma_forward_static(plan, q, k, v, wk, wv, out, stream=None):
    _check(library().fma_forward_static(plan, _ptr(q), _ptr(k), _ptr(v), _ptr(wk), _ptr(wv), _ptr(out),
                                        _stream(stream)))


def fma_stream_reference(src, src_bytes, dst, dst_bytes, write_every, stream=None):
    _check(library().fma_stream_reference(_ptr(src), src_bytes, _ptr(dst), dst_bytes, write_every, _stream(stream)))


PLAN_PARAM_NAMES = [
    "n", "side", "block", "nbx", "qtile", "tiles_per_slice", "nslice", "R", "causal", "nslot", "slot_group",
    "rank", "norm_level", "ndim", "esize", "heads", "w_stride", "wlen", "nsets", "chunk", "run", "nchunk",
    "tiles_y", "first_partial", "npartial", "part_span", "part_count", "depth", "wave_lds",
    "coarsen_smem", "part_offset", "coarse_bytes", "ws_bytes", "linear", "heads_w", "dtype", "pair2d",
    "height", "nby", "tiles_x", "head_dim"]
SET_PARAM_NAMES = ("off", "M", "My", "size", "woff", "lvl")


def fma_plan_params(plan: int) -> dict:
    """The plan's launch parameters (fma_plan_params) as a dict; per-set
    tables under "sets" (dicts of off, M, My, size, woff, lvl)."""
    nb, ns = len(PLAN_PARAM_NAMES), len(SET_PARAM_NAMES)
    cap = nb + ns * 64
    buf = (ctypes.c_int64 * cap)()
    cnt = ctypes.c_int32()
    _check(library().fma_plan_params(plan, buf, cap, ctypes.byref(cnt)))
    vals = list(buf[:cnt.value])
    d = dict(zip(PLAN_PARAM_NAMES, vals[:nb]))
    d["sets"] = [dict(zip(SET_PARAM_NAMES, vals[nb + ns * e:nb + ns * (e + 1)])) for e in range(d["nsets"])]
    return d


def fma_backward_workspace_size(plan: int) -> int:
    x = ctypes.c_size_t()
    _check(library().fma_backward_workspace_size(plan, ctypes.byref(x)))
    return x.value


def fma_backward(plan, q, k, v, wk, wv, out, dout, dq, dk, dv, dwk, dwv, workspace, workspace_bytes,
                 stream=None):
    _check(library().fma_backward(plan, _ptr(q), _ptr(k), _ptr(v), _ptr(wk), _ptr(wv), _ptr(out), _ptr(dout),
                                  _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dwk), _ptr(dwv), _ptr(workspace),
                                  workspace_bytes, _stream(stream)))


def fma_backward_linear(plan, q, k, v, wk, wv, wq, out, dout, dq, dk, dv, dwk, dwv, dwq, workspace,
                        workspace_bytes, stream=None):
    _check(library().fma_backward_linear(plan, _ptr(q), _ptr(k), _ptr(v), _ptr(wk), _ptr(wv), _ptr(wq),
                                         _ptr(out), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dwk),
                                         _ptr(dwv), _ptr(dwq), _ptr(workspace), workspace_bytes, _stream(stream)))


def fma_last_error() -> str:
    return library().fma_last_error().decode()


# ---------------------------------------------------------------- object API
_DTYPES = {torch.float32: FMA_F32, torch.bfloat16: FMA_BF16}


def make_desc(ndim=1, batch=1, heads=1, seq_len=0, block=64, causal=False, dtype=torch.bfloat16,
              side=0, head_dim=HEAD_DIM, num_levels=-1, weights_per_head=True, softmax_scale=0.0,
              rank=1, norm=FMA_NORM_JOINT, linear=False):
    d = fma_desc_t()
    d.struct_size = ctypes.sizeof(fma_desc_t)
    d.ndim = ndim
    d.batch = batch
    d.heads = heads
    d.seq_len = seq_len
    d.side = side
    d.head_dim = head_dim
    d.block = block
    d.num_levels = num_levels
    d.causal = int(bool(causal))
    d.dtype = _DTYPES[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    d.weights_per_head = int(bool(weights_per_head))
    d.softmax_scale = softmax_scale
    d.rank = rank
    d.norm = norm
    d.query_downsample = int(bool(linear))
    return d


class FMA:
    """One plan (shape + options) and the calls that use it."""

    def __init__(self, ndim=1, batch=1, heads=1, seq_len=0, block=64, causal=False,
                 dtype=torch.bfloat16, side=0, weights_per_head=True, softmax_scale=0.0,
                 num_levels=-1, head_dim=HEAD_DIM, rank=1, norm=FMA_NORM_JOINT, linear=False):
        if ndim == 2 and side == 0:
            side = int(round(seq_len ** 0.5))
        self.desc = make_desc(ndim, batch, heads, seq_len, block, causal, dtype, side, head_dim,
                              num_levels, weights_per_head, softmax_scale, rank, norm, linear)
        self.rank, self.norm, self.linear = rank, norm, linear
        self.ndim, self.batch, self.heads, self.n = ndim, batch, heads, seq_len
        self.side, self.block, self.causal, self.dtype = side, block, causal, dtype
        self.head_dim = head_dim
        self.handle = fma_plan(self.desc)
        self.workspace_bytes = fma_workspace_size(self.handle)
        self.weights_len = fma_weights_len(self.handle)
        self.coarse_rows = fma_coarse_rows(self.handle)
        self.levels = fma_num_levels(self.handle)
        self.backward_workspace_bytes = fma_backward_workspace_size(self.handle)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                library().fma_destroy(h)
            except Exception:
                pass
            self.handle = None

    # ---------------------------------------------------------- helpers
    def new_workspace(self, device) -> torch.Tensor:
        return torch.empty(max(self.workspace_bytes, 16), dtype=torch.uint8, device=device)

    def coarse_views(self, workspace: torch.Tensor):
        """(K_bar, V_bar) views [B, H, R, d] of a workspace filled by coarsen()."""
        R = self.coarse_rows
        numel = self.batch * self.heads * R * self.head_dim
        flat = workspace[: 2 * numel * (2 if self.dtype == torch.bfloat16 else 4)].view(self.dtype)
        kb = flat[:numel].view(self.batch, self.heads, R, self.head_dim)
        vb = flat[numel:2 * numel].view(self.batch, self.heads, R, self.head_dim)
        return kb, vb

    # ---------------------------------------------------------- calls
    def forward(self, q, k, v, wk=None, wv=None, out=None, workspace=None, stream=None):
        if out is None:
            out = torch.empty_like(q)
        if workspace is None:
            workspace = self.new_workspace(q.device)
        fn = fma_forward_1d if self.ndim == 1 else fma_forward_2d
        fn(self.handle, q, k, v, wk, wv, out, workspace, workspace.numel(), stream)
        return out

    def forward_static(self, q, k, v, wk=None, wv=None, out=None, stream=None):
        """The forward pass with the library's static per-GPU workspace
        (fma_forward_static): no workspace argument, nothing allocated."""
        if out is None:
            out = torch.empty_like(q)
        fma_forward_static(self.handle, q, k, v, wk, wv, out, stream)
        return out

    def forward_linear(self, q, k, v, wq, wk, wv, out=None, workspace=None, stream=None):
        """FMA-linear (plan made with linear=True): wq aggregates the queries."""
        if out is None:
            out = torch.empty_like(q)
        if workspace is None:
            workspace = self.new_workspace(q.device)
        fma_forward_linear(self.handle, q, k, v, wq, wk, wv, out, workspace, workspace.numel(), stream)
        return out

    def coarsen(self, k, v, wk, wv, workspace=None, stream=None):
        if workspace is None:
            workspace = self.new_workspace(k.device)
        fma_coarsen(self.handle, k, v, wk, wv, workspace, workspace.numel(), stream)
        return workspace

    def attend(self, q, k, v, workspace, out=None, stream=None):
        if out is None:
            out = torch.empty_like(q)
        fma_attend(self.handle, q, k, v, workspace, workspace.numel(), out, stream)
        return out

    def backward(self, q, k, v, wk, wv, out, dout, workspace=None, stream=None):
        """Gradients (dq, dk, dv, dwk, dwv) of sum(dout * out) for out =
        forward(q, k, v, wk, wv); dwk, dwv shaped like wk, wv (None when the
        plan has no coarse level)."""
        dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
        dwk = torch.empty_like(wk) if wk is not None and wk.numel() else None
        dwv = torch.empty_like(wv) if wv is not None and wv.numel() else None
        if workspace is None:
            workspace = torch.empty(max(self.backward_workspace_bytes, 16), dtype=torch.uint8, device=q.device)
        fma_backward(self.handle, q, k, v, wk if dwk is not None else None, wv if dwv is not None else None,
                     out, dout, dq, dk, dv, dwk, dwv, workspace, workspace.numel(), stream)
        return dq, dk, dv, dwk, dwv

    def backward_linear(self, q, k, v, wk, wv, wq, out, dout, workspace=None, stream=None):
        """FMA-linear plans: gradients (dq, dk, dv, dwk, dwv, dwq) of
        sum(dout * out) for out = forward_linear(q, k, v, wk, wv, wq)."""
        dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
        has_w = wk is not None and wk.numel() > 0
        dwk = torch.empty_like(wk) if has_w else None
        dwv = torch.empty_like(wv) if has_w else None
        dwq = torch.empty_like(wq) if has_w else None
        if workspace is None:
            workspace = torch.empty(max(self.backward_workspace_bytes, 16), dtype=torch.uint8, device=q.device)
        fma_backward_linear(self.handle, q, k, v, wk if has_w else None, wv if has_w else None,
                            wq if has_w else None, out, dout, dq, dk, dv, dwk, dwv, dwq, workspace,
                            workspace.numel(), stream)
        return dq, dk, dv, dwk, dwv, dwq

    def interaction_lists(self, device, stream=None) -> torch.Tensor:
        K = 3 if self.ndim == 1 else 27
        nb = self.n // self.block if self.ndim == 1 else (self.side // self.block) * (self.n // self.side // self.block)
        out = torch.empty((nb, max(self.levels - 1, 0), K), dtype=torch.int32, device=device)
        if out.numel():
            fma_interaction_lists(self.handle, out, stream)
        return out

    def dense_reference(self, q, k, v, out=None, stream=None):
        if out is None:
            out = torch.empty_like(q)
        fma_dense_reference(self.handle, q, k, v, out, stream)
        return out
