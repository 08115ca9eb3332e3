"""tpdq: TP-aware dequantization (arXiv 2402.04925) on AMD MI355X.

Thin Python binding of libtpdq (include/tpdq.h). Every function here only
marshals torch tensors (device memory and the current stream) into the C ABI;
all computation runs in the library's HIP kernels. If the library is not
built, calls raise: there is no fallback.
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import Optional

from . import _abi
from ._abi import (BF16, FP16, LAYOUT_GPTQ, LAYOUT_TILED, OP_GATED_MLP, OP_GEMM, OP_MLP, OP_REORDER,
                   PATH_ACTORDER, PATH_ACTORDER_GLOBAL, PATH_ORDERED, TpdqError)

__all__ = [
    "QuantWeight", "reorder", "pack_tiled", "w4a16_gemm", "mlp_shard", "mlp_shard_noalloc",
    "gated_mlp_shard",
    "workspace_bytes", "Workspace",
    "LAYOUT_GPTQ", "LAYOUT_TILED", "tiled_ld",
    "TpdqError", "PATH_ACTORDER", "PATH_ORDERED", "PATH_ACTORDER_GLOBAL", "FP16", "BF16", "version",
]


def _torch():
    import torch
    return torch


def version() -> str:
    return _abi.lib().tpdq_version().decode()


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_handle(device) -> int:
    torch = _torch()
    return torch.cuda.current_stream(device).cuda_stream


def _dtype_code(dt) -> int:
    torch = _torch()
    if dt == torch.float16:
        return FP16
    if dt == torch.bfloat16:
        return BF16
    raise TypeError(f"activations and scales must be float16 or bfloat16, got {dt}")


def _check_args(device, scales_dtype=None, **tensors):
    """Every tensor argument is on `device`, a GPU, so that the library only
    ever receives device pointers; int32 index tensors are contiguous; the
    activations' element type is the scales' (the C ABI takes one type)."""
    torch = _torch()
    if device.type != "cuda":
        raise ValueError(f"the weights must be on a GPU, got {device}")
    for name, t in tensors.items():
        if t is None:
            continue
        if t.device != device:
            raise ValueError(f"{name} is on {t.device}, the weights on {device}")
        if name in ("x_perm", "P1") and (t.dtype != torch.int32 or not t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous int32 tensor")
    X = tensors.get("X")
    if X is not None and scales_dtype is not None and X.dtype != scales_dtype:
        raise TypeError(f"X is {X.dtype} but the scales are {scales_dtype}: one element type per call")


def _check_layers(X, *layers):
    """The layers share X's device and element type (their scales')."""
    for i, w in enumerate(layers):
        if w.device != X.device:
            raise ValueError(f"layer {i} is on {w.device}, X on {X.device}")
        if w.scales.dtype != X.dtype:
            raise TypeError(f"layer {i} has {w.scales.dtype} scales, X is {X.dtype}")


def _check_out(name, t, M, N, dtype):
    if t is not None and (tuple(t.shape) != (M, N) or t.stride(1) != 1 or t.dtype != dtype):
        raise ValueError(f"{name} must be [{M}][{N}] of {dtype} with unit column stride")


def tiled_ld(K: int) -> int:
    """Words per 16-column tile of a dense tiled qweight with K rows."""
    return (K + 127) // 128 * 256


@dataclasses.dataclass
class QuantWeight:
    """A quantized layer (or a shard of one as views) in device memory.

    qweight int32: GPTQ layout [K/8][>=N], or tiled layout
    [ceil(N/16)][>=tiled_ld(K)] (see include/tpdq.h); scales fp16
    [num_groups][>=N]; qzeros int32 [num_groups][>=N/8]; g_idx int32 [K] or
    None. G = 0: groups of unequal sizes given by g_idx alone. zero_offset
    (0 or 1) is added to every stored zero code.
    """
    qweight: object
    scales: object
    qzeros: object
    g_idx: object
    K: int
    N: int
    G: int
    num_groups: int
    layout: int = LAYOUT_GPTQ
    zero_offset: int = 0

    @classmethod
    def from_tensors(cls, qweight, scales, qzeros, g_idx, G: int, num_groups: Optional[int] = None,
                     zero_offset: int = 0):
        """A GPTQ-layout layer: K and N follow from qweight's shape."""
        K = qweight.shape[0] * 8
        N = qweight.shape[1]
        ng = scales.shape[0] if num_groups is None else num_groups
        return cls(qweight, scales, qzeros, g_idx, K, N, G, ng, LAYOUT_GPTQ, zero_offset)

    def c_struct(self) -> _abi.W4:
        torch = _torch()
        for name in ("qweight", "scales", "qzeros", "g_idx"):
            t = getattr(self, name)
            if t is None:
                continue
            if t.device != self.qweight.device:
                raise ValueError(f"{name} is on {t.device}, qweight on {self.qweight.device}")
            want = (torch.float16, torch.bfloat16) if name == "scales" else (torch.int32,)
            if t.dtype not in want:
                raise TypeError(f"{name} must be {' or '.join(str(d) for d in want)}, got {t.dtype}")
        for name in ("qweight", "scales", "qzeros"):
            t = getattr(self, name)
            if t.stride(1) != 1:
                raise ValueError(f"{name} must have unit column stride")
        if self.g_idx is not None and not self.g_idx.is_contiguous():
            raise ValueError("g_idx must be contiguous")
        return _abi.W4(
            qweight=_ptr(self.qweight), ld_q=self.qweight.stride(0),
            scales=_ptr(self.scales), ld_s=self.scales.stride(0),
            qzeros=_ptr(self.qzeros), ld_z=self.qzeros.stride(0),
            g_idx=_ptr(self.g_idx), K=self.K, N=self.N, group_size=self.G,
            num_groups=self.num_groups, layout=self.layout, zero_offset=self.zero_offset)

    @property
    def device(self):
        return self.qweight.device

    def column_shard(self, rank: int, tp: int) -> "QuantWeight":
        """Megatron column-parallel shard (views): columns [rank*N/tp, ...)."""
        n = self.N // tp
        c0 = rank * n
        if self.layout == LAYOUT_TILED:
            if c0 % 16 or n % 16:
                raise ValueError("a tiled column shard must start and end on 16-column tiles")
            qw = self.qweight[c0 // 16:(c0 + n) // 16]
        else:
            qw = self.qweight[:, c0:c0 + n]
        return QuantWeight(qw, self.scales[:, c0:c0 + n], self.qzeros[:, c0 // 8:(c0 + n) // 8],
                           self.g_idx, self.K, n, self.G, self.num_groups, self.layout, self.zero_offset)

    def row_shard(self, rank: int, tp: int, sorted_rows: bool) -> "QuantWeight":
        """Megatron row-parallel shard (views): rows [rank*K/tp, ...).

        Sorted rows keep only their own consecutive groups (the shard must
        start on a group boundary; the last may end in a partial group);
        act-order rows, and sorted rows in groups of unequal sizes (G = 0),
        keep the global g_idx values of their rows and all the metadata."""
        k = self.K // tp
        r0 = rank * k
        if self.layout == LAYOUT_TILED:
            if r0 % 128:
                raise ValueError("a tiled row shard must start on a 128-row block")
            c0 = (r0 // 128) * 256
            qw = self.qweight[:, c0:min(c0 + tiled_ld(k), self.qweight.shape[1])]
        else:
            qw = self.qweight[r0 // 8:(r0 + k) // 8]
        g = None if self.g_idx is None else self.g_idx[r0:r0 + k]
        if sorted_rows and self.G > 0:
            if r0 % self.G:
                raise ValueError("a sorted row shard must start on a group boundary")
            g0, ng = r0 // self.G, -(-k // self.G)
            return QuantWeight(qw, self.scales[g0:g0 + ng], self.qzeros[g0:g0 + ng], g, k, self.N,
                               self.G, ng, self.layout, self.zero_offset)
        return QuantWeight(qw, self.scales, self.qzeros, g, k, self.N, self.G, self.num_groups,
                           self.layout, self.zero_offset)


class Workspace:
    """Device scratch for the library calls, grown on demand. One workspace
    serves any number of calls issued one after another on one stream."""

    def __init__(self, device=None):
        self.device = device
        self.buf = None

    def get(self, nbytes: int):
        torch = _torch()
        if self.buf is None or self.buf.numel() < nbytes:
            n = max(nbytes, 1 << 20)
            self.buf = torch.empty(n, dtype=torch.uint8, device=self.device)
        return self.buf


_default_ws = {}


def _workspace(device, nbytes, ws: Optional[Workspace]):
    if ws is None:
        key = (str(device), _stream_handle(device))
        ws = _default_ws.get(key)
        if ws is None:
            ws = _default_ws[key] = Workspace(device)
    return ws.get(nbytes)


def workspace_bytes(op: int, M: int, a: QuantWeight, b: Optional[QuantWeight] = None) -> int:
    ca = a.c_struct()
    cb = b.c_struct() if b is not None else None
    return _abi.lib().tpdq_workspace_bytes(op, M, ctypes.byref(ca),
                                          ctypes.byref(cb) if cb is not None else None)


def reorder(w1: QuantWeight, w2: Optional[QuantWeight] = None, workspace: Optional[Workspace] = None,
            layout: int = LAYOUT_TILED):
    """Alg. 1 on w1 (and w2) plus the TP-aware fold W1[P1, P2], W2[P2].

    Returns (P1, g1_sorted, P2, g2_sorted, w1_out, w2_out); P2, g2_sorted and
    w2_out are None without w2. w1_out/w2_out are sorted-row QuantWeights in
    `layout` (their g_idx is the sorted g_idx)."""
    torch = _torch()
    dev = w1.device
    i32 = dict(dtype=torch.int32, device=dev)

    def qbuf(K, N):
        if layout == LAYOUT_TILED:
            return torch.empty((N + 15) // 16, tiled_ld(K), **i32)
        return torch.empty(K // 8, N, **i32)

    P1 = torch.empty(w1.K, **i32)
    g1 = torch.empty(w1.K, **i32)
    q1 = qbuf(w1.K, w1.N)
    s1 = torch.empty(w1.num_groups, w1.N, dtype=w1.scales.dtype, device=dev)
    z1 = torch.empty(w1.num_groups, w1.N // 8, **i32)
    P2 = g2 = q2 = None
    if w2 is not None:
        P2 = torch.empty(w2.K, **i32)
        g2 = torch.empty(w2.K, **i32)
        q2 = qbuf(w2.K, w2.N)
    c1 = w1.c_struct()
    c2 = w2.c_struct() if w2 is not None else None
    lib = _abi.lib()
    nbytes = lib.tpdq_workspace_bytes(OP_REORDER, 0, ctypes.byref(c1),
                                      ctypes.byref(c2) if c2 is not None else None)
    buf = _workspace(dev, nbytes, workspace)
    _abi.check(lib.tpdq_reorder(
        ctypes.byref(c1), ctypes.byref(c2) if c2 is not None else None,
        _ptr(P1), _ptr(g1), _ptr(P2), _ptr(g2), _ptr(q1), _ptr(s1), _ptr(z1), _ptr(q2),
        _dtype_code(w1.scales.dtype), layout, _ptr(buf), buf.numel(), _stream_handle(dev)))
    w1o = QuantWeight(q1, s1, z1, g1, w1.K, w1.N, w1.G, w1.num_groups, layout, w1.zero_offset)
    w2o = None
    if w2 is not None:
        w2o = QuantWeight(q2, w2.scales, w2.qzeros, g2, w2.K, w2.N, w2.G, w2.num_groups, layout,
                          w2.zero_offset)
    return P1, g1, P2, g2, w1o, w2o


def pack_tiled(w: QuantWeight) -> QuantWeight:
    """The same layer with qweight in the tiled layout (metadata shared)."""
    torch = _torch()
    out = torch.empty((w.N + 15) // 16, tiled_ld(w.K), dtype=torch.int32, device=w.device)
    c = w.c_struct()
    _abi.check(_abi.lib().tpdq_pack_tiled(ctypes.byref(c), _ptr(out), _stream_handle(w.device)))
    return QuantWeight(out, w.scales, w.qzeros, w.g_idx, w.K, w.N, w.G, w.num_groups, LAYOUT_TILED,
                       w.zero_offset)


def w4a16_gemm(X, w: QuantWeight, path: int, x_perm=None, out=None,
               workspace: Optional[Workspace] = None):
    """Y = X' @ deq(w) with X' = X or X[:, x_perm]; fp32 accumulation."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D with unit column stride")
    _check_args(w.device, w.scales.dtype, X=X, x_perm=x_perm, out=out)
    M = X.shape[0]
    _check_out("out", out, M, w.N, X.dtype)
    if out is None:
        out = torch.empty(M, w.N, dtype=X.dtype, device=X.device)
    cw = w.c_struct()
    lib = _abi.lib()
    nbytes = lib.tpdq_workspace_bytes(OP_GEMM, M, ctypes.byref(cw), None)
    buf = _workspace(X.device, nbytes, workspace)
    _abi.check(lib.tpdq_w4a16_gemm(
        _ptr(X), X.stride(0), M, _ptr(x_perm), ctypes.byref(cw), path, _dtype_code(X.dtype),
        _ptr(out), out.stride(0), _ptr(buf), buf.numel(), _stream_handle(X.device)))
    return out


def mlp_shard(X, w1: QuantWeight, w2: QuantWeight, path: int, P1=None, y1=None, y2=None,
              workspace: Optional[Workspace] = None):
    """One rank's Alg. 3 (ordered) or act-order MLP share, up to the AllReduce.
    Returns (Y1, Y2_partial)."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D with unit column stride")
    _check_args(w1.device, w1.scales.dtype, X=X, P1=P1, y1=y1, y2=y2)
    _check_layers(X, w1, w2)
    M = X.shape[0]
    _check_out("y1", y1, M, w1.N, X.dtype)
    _check_out("y2", y2, M, w2.N, X.dtype)
    if y1 is None:
        y1 = torch.empty(M, w1.N, dtype=X.dtype, device=X.device)
    if y2 is None:
        y2 = torch.empty(M, w2.N, dtype=X.dtype, device=X.device)
    c1, c2 = w1.c_struct(), w2.c_struct()
    lib = _abi.lib()
    nbytes = lib.tpdq_workspace_bytes(OP_MLP, M, ctypes.byref(c1), ctypes.byref(c2))
    buf = _workspace(X.device, nbytes, workspace)
    _abi.check(lib.tpdq_mlp_shard(
        _ptr(X), X.stride(0), M, _ptr(P1), ctypes.byref(c1), ctypes.byref(c2), path,
        _dtype_code(X.dtype), _ptr(y1), _ptr(y2), _ptr(buf), buf.numel(),
        _stream_handle(X.device)))
    return y1, y2


def mlp_shard_noalloc(X, w1: QuantWeight, w2: QuantWeight, path: int, P1=None, y1=None, y2=None):
    """mlp_shard through tpdq_mlp_shard_noalloc: the library's static scratch
    instead of a workspace, so the call itself allocates no device memory
    when y1 and y2 are given. Returns (Y1, Y2_partial)."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D with unit column stride")
    _check_args(w1.device, w1.scales.dtype, X=X, P1=P1, y1=y1, y2=y2)
    _check_layers(X, w1, w2)
    M = X.shape[0]
    _check_out("y1", y1, M, w1.N, X.dtype)
    _check_out("y2", y2, M, w2.N, X.dtype)
    if y1 is None:
        y1 = torch.empty(M, w1.N, dtype=X.dtype, device=X.device)
    if y2 is None:
        y2 = torch.empty(M, w2.N, dtype=X.dtype, device=X.device)
    c1, c2 = w1.c_struct(), w2.c_struct()
    _abi.check(_abi.lib().tpdq_mlp_shard_noalloc(
        _ptr(X), X.stride(0), M, _ptr(P1), ctypes.byref(c1), ctypes.byref(c2), path,
        _dtype_code(X.dtype), _ptr(y1), _ptr(y2), _stream_handle(X.device)))
    return y1, y2


def gated_mlp_shard(X, w_gate: QuantWeight, w_up: QuantWeight, w_down: QuantWeight, path: int, P1=None,
                    y1=None, y2=None, workspace: Optional[Workspace] = None):
    """One rank's gated MLP share up to the AllReduce: Y1 = silu(X' W_gate) *
    (X' W_up), Y2_partial = Y1 @ W_down (X' = X[:, P1] on the ordered path,
    where gate and up are column shards of W[P1, P2] and down a row shard of
    W_down[P2]). Returns (Y1, Y2_partial)."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D with unit column stride")
    _check_args(w_gate.device, w_gate.scales.dtype, X=X, P1=P1, y1=y1, y2=y2)
    _check_layers(X, w_gate, w_up, w_down)
    M = X.shape[0]
    _check_out("y1", y1, M, w_gate.N, X.dtype)
    _check_out("y2", y2, M, w_down.N, X.dtype)
    if y1 is None:
        y1 = torch.empty(M, w_gate.N, dtype=X.dtype, device=X.device)
    if y2 is None:
        y2 = torch.empty(M, w_down.N, dtype=X.dtype, device=X.device)
    cg, cu, cd = w_gate.c_struct(), w_up.c_struct(), w_down.c_struct()
    lib = _abi.lib()
    nbytes = lib.tpdq_workspace_bytes(OP_GATED_MLP, M, ctypes.byref(cg), ctypes.byref(cd))
    buf = _workspace(X.device, nbytes, workspace)
    _abi.check(lib.tpdq_gated_mlp_shard(
        _ptr(X), X.stride(0), M, _ptr(P1), ctypes.byref(cg), ctypes.byref(cu), ctypes.byref(cd), path,
        _dtype_code(X.dtype), _ptr(y1), _ptr(y2), _ptr(buf), buf.numel(), _stream_handle(X.device)))
    return y1, y2
