"""Token-condensation MoE layer (Luffy, arXiv 2411.15419) on one MI355X.

Thin ctypes binding of ``libluffy.so`` (the HIP kernels behind the C ABI in
``include/luffy.h``).  Every function passes device pointers, sizes and the
current HIP stream through; every step of the layer runs in the library's
kernels.  torch supplies device memory and streams only.  There is no
fallback: without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

__all__ = [
    "LuffyError", "load_library", "LUFFY_F32", "LUFFY_BF16", "LUFFY_ACT_GELU",
    "LUFFY_ACT_SILU", "luffy_route", "luffy_route_noalloc", "luffy_condense", "luffy_expert_ffn",
    "luffy_combine", "route_workspace_size", "condense_workspace_size",
    "expert_ffn_workspace_size", "capacity", "MoELayer", "LIB_PATH", "profile_kernel",
    "profile_read", "KERNELS", "adaptive_threshold", "AdaptiveThreshold",
    "luffy_combine_backward", "combine_backward_workspace_size", "luffy_expert_ffn_backward",
    "expert_ffn_backward_workspace_size", "luffy_condense_history", "history_size",
    "condense_history_workspace_size", "MoEStack", "CondensationDriver",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libluffy.so")

LUFFY_F32, LUFFY_BF16 = 0, 1
LUFFY_ACT_GELU, LUFFY_ACT_SILU = 0, 1
_ACTS = {"gelu": LUFFY_ACT_GELU, "silu": LUFFY_ACT_SILU}

_c_int, _c_float, _c_size, _vp = ctypes.c_int, ctypes.c_float, ctypes.c_size_t, ctypes.c_void_p

_SIGS = {
    "luffy_abi_version": (_c_int, []),
    "luffy_status_string": (ctypes.c_char_p, [_c_int]),
    "luffy_last_error": (ctypes.c_char_p, []),
    "luffy_route_workspace_size": (_c_size, [_c_int, _c_int, _c_int]),
    "luffy_capacity": (_c_int, [_c_int, _c_int, _c_int, ctypes.c_double]),
    "luffy_route": (_c_int, [_vp, _c_int, _c_int, _c_int, _vp, _vp, _c_int, _c_int, ctypes.c_double,
                             _vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_size, _vp]),
    "luffy_route_noalloc_max_bytes": (_c_size, []),
    "luffy_route_noalloc": (_c_int, [_vp, _c_int, _c_int, _c_int, _vp, _vp, _c_int, _c_int, ctypes.c_double,
                                     _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "luffy_condense_workspace_size": (_c_size, [_c_int, _c_int, _c_int, _c_int, _c_int]),
    "luffy_condense": (_c_int, [_vp, _c_int, _c_int, _c_int, _vp, _vp, _c_int, _c_int, _c_int,
                                _c_float, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_size, _vp]),
    "luffy_set_similarity_screen": (_c_int, [_c_int]),
    "luffy_similarity_screen_applies": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int]),
    "luffy_history_size": (_c_size, [_c_int, _c_int, _c_int, _c_int]),
    "luffy_condense_history_workspace_size": (_c_size, [_c_int, _c_int, _c_int, _c_int, _c_int]),
    "luffy_condense_history": (_c_int, [_vp, _c_int, _c_int, _c_int, _vp, _vp, _vp, _c_int, _c_int, _c_int,
                                        _c_float, _vp, _vp, _c_float, _c_float, _vp, _vp, _vp, _vp, _vp, _vp,
                                        _vp, _vp, _vp, _c_size, _vp]),
    "luffy_expert_ffn_workspace_size": (_c_size, [_c_int, _c_int, _c_int, _c_int]),
    "luffy_expert_ffn": (_c_int, [_vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _vp, _vp,
                                  _c_int, _c_int, _vp, _vp, _c_size, _vp]),
    "luffy_combine": (_c_int, [_vp, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _vp, _vp]),
    "luffy_combine_backward_workspace_size": (_c_size, [_c_int, _c_int, _c_int]),
    "luffy_combine_backward": (_c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _c_int,
                                        _c_int, _c_int, _c_int, _vp, _vp, _vp, _c_size, _vp]),
    "luffy_expert_ffn_backward_workspace_size": (_c_size, [_c_int, _c_int, _c_int, _c_int, _c_int]),
    "luffy_expert_ffn_backward": (_c_int, [_vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _c_int,
                                           _c_int, _vp, _vp, _vp, _vp, _c_int, _vp, _c_size, _vp]),
    "luffy_adaptive_threshold": (_c_int, [ctypes.c_double, ctypes.c_double, ctypes.POINTER(ctypes.c_double)]),
    "luffy_profile_kernel": (_c_int, [ctypes.c_char_p]),
    "luffy_profile_read": (_c_int, [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_c_int)]),
}

_LIB = None


class LuffyError(RuntimeError):
    pass


def load_library(path: str = LIB_PATH):
    """Loads libluffy.so once and declares the C signatures."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise LuffyError(f"{path} is not built; run `python -m paper_2411_15419_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def _check(status: int, what: str):
    if status != 0:
        lib = load_library()
        msg = lib.luffy_last_error().decode()
        raise LuffyError(f"{what}: {lib.luffy_status_string(status).decode()} ({status}): {msg}")


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return LUFFY_F32
    if t.dtype == torch.bfloat16:
        return LUFFY_BF16
    raise LuffyError(f"unsupported dtype {t.dtype}")


def _p(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise LuffyError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise LuffyError("tensor must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def capacity(T: int, k: int, E: int, cf: float) -> int:
    """Per-expert capacity of luffy_route (luffy_capacity; 0 = unlimited)."""
    return int(load_library().luffy_capacity(int(T), int(k), int(E), float(cf)))


def route_workspace_size(T: int, E: int, k: int) -> int:
    return load_library().luffy_route_workspace_size(T, E, k)


def condense_workspace_size(T: int, d: int, E: int, k: int, max_bucket: int) -> int:
    return load_library().luffy_condense_workspace_size(T, d, E, k, max_bucket)


def set_similarity_screen(on: bool) -> bool:
    """Enables or disables the fp8 similarity screen of luffy_condense
    (luffy_set_similarity_screen); returns the previous setting."""
    return bool(load_library().luffy_set_similarity_screen(1 if on else 0))


def similarity_screen_applies(T: int, d: int, E: int, k: int, dtype: int = LUFFY_BF16) -> bool:
    """Whether a condense call of this shape takes the fp8 screen now."""
    return bool(load_library().luffy_similarity_screen_applies(int(T), int(d), int(E), int(k), int(dtype)))


def expert_ffn_workspace_size(max_rows: int, E: int, d_ff: int, dtype: int) -> int:
    return load_library().luffy_expert_ffn_workspace_size(max_rows, E, d_ff, dtype)


def luffy_route(x, w_gate, b_gate, k, capacity_factor, topk_idx, topk_gate, slot_pos,
                perm_token, offsets, workspace, stream=None, inv_norm=None):
    T, d = x.shape
    E = w_gate.shape[0]
    lib = load_library()
    _check(lib.luffy_route(_p(x), T, d, _dtype_code(x), _p(w_gate), _p(b_gate), E, k,
                           float(capacity_factor), _p(topk_idx), _p(topk_gate), _p(slot_pos),
                           _p(perm_token), _p(offsets), _p(inv_norm), _p(workspace),
                           workspace.numel(), _stream(stream)), "luffy_route")


def luffy_route_noalloc(x, w_gate, b_gate, k, capacity_factor, topk_idx, topk_gate, slot_pos,
                        perm_token, offsets, stream=None, inv_norm=None):
    """luffy_route without a workspace (the library's own scratch array;
    calls that may overlap on one GPU must be ordered by the caller)."""
    T, d = x.shape
    E = w_gate.shape[0]
    lib = load_library()
    _check(lib.luffy_route_noalloc(_p(x), T, d, _dtype_code(x), _p(w_gate), _p(b_gate), E, k,
                                   float(capacity_factor), _p(topk_idx), _p(topk_gate), _p(slot_pos),
                                   _p(perm_token), _p(offsets), _p(inv_norm), _stream(stream)),
           "luffy_route_noalloc")


def luffy_condense(x, perm_token, offsets, k, max_bucket, threshold, rep_of_pos, rep_row,
                   rep_offsets, rep_token, x_rep, degree, workspace, stream=None, inv_norm=None):
    T, d = x.shape
    E = offsets.numel() - 1
    lib = load_library()
    _check(lib.luffy_condense(_p(x), T, d, _dtype_code(x), _p(perm_token), _p(offsets), E, k,
                              max_bucket, float(threshold), _p(rep_of_pos), _p(rep_row),
                              _p(rep_offsets), _p(rep_token), _p(x_rep), _p(degree),
                              _p(inv_norm), _p(workspace), workspace.numel(), _stream(stream)),
           "luffy_condense")


def history_size(T: int, E: int, k: int, max_bucket: int) -> int:
    return int(load_library().luffy_history_size(T, E, k, max_bucket))


def condense_history_workspace_size(T: int, d: int, E: int, k: int, max_bucket: int) -> int:
    return int(load_library().luffy_condense_history_workspace_size(T, d, E, k, max_bucket))


def luffy_condense_history(x, perm_token, offsets, slot_pos, k, max_bucket, threshold, hist_in, hist_out, S1, S2,
                           rep_of_pos, rep_row, rep_offsets, rep_token, x_rep, degree, stats, workspace,
                           stream=None, inv_norm=None):
    """luffy_condense with the historical similarity of Sec. 5.1 step 2:
    hist_in is the previous block's record (or None), hist_out receives this
    block's (or None); stats (4 int64 or None) receives undecided pairs,
    decided pairs, tiles computed and tiles skipped."""
    T, d = x.shape
    E = offsets.numel() - 1
    _check(load_library().luffy_condense_history(
        _p(x), T, d, _dtype_code(x), _p(perm_token), _p(offsets), _p(slot_pos), E, k, max_bucket,
        float(threshold), _p(hist_in), _p(hist_out), float(S1), float(S2), _p(rep_of_pos), _p(rep_row),
        _p(rep_offsets), _p(rep_token), _p(x_rep), _p(degree), _p(inv_norm), _p(stats), _p(workspace),
        workspace.numel(), _stream(stream)), "luffy_condense_history")


def luffy_expert_ffn(x, row_index, rep_offsets, w1, w2, act, max_rows, y_rep, workspace,
                     stream=None):
    E, d_ff, d = w1.shape
    lib = load_library()
    act_code = _ACTS[act] if isinstance(act, str) else int(act)
    _check(lib.luffy_expert_ffn(_p(x), _p(row_index), _p(rep_offsets), E, d, d_ff,
                                _dtype_code(x), _p(w1), _p(w2), act_code, max_rows, _p(y_rep),
                                _p(workspace), workspace.numel(), _stream(stream)),
           "luffy_expert_ffn")


def luffy_combine(y_rep, rep_row, slot_pos, topk_gate, y, stream=None):
    T, k = slot_pos.shape
    d = y.shape[1]
    lib = load_library()
    _check(lib.luffy_combine(_p(y_rep), _p(rep_row), _p(slot_pos), _p(topk_gate), T, k, d,
                             _dtype_code(y), _p(y), _stream(stream)), "luffy_combine")


def combine_backward_workspace_size(T: int, k: int, max_rows: int) -> int:
    return int(load_library().luffy_combine_backward_workspace_size(T, k, max_rows))


def luffy_combine_backward(dy, y_rep, rep_row, perm_token, slot_pos, topk_gate, offsets, rep_offsets,
                           dy_rep, dgate, workspace, stream=None):
    """Transpose of luffy_combine: dy_rep (the representatives' rows) and
    dgate [T, k] from dy [T, d]."""
    T, d = dy.shape
    k = slot_pos.shape[1]
    max_rows = y_rep.shape[0]
    if dy_rep.shape != y_rep.shape or dy_rep.dtype != y_rep.dtype or dy.dtype != y_rep.dtype:
        raise LuffyError("dy, y_rep and dy_rep must share dtype; dy_rep must have y_rep's shape")
    E = rep_offsets.numel() - 1
    _check(load_library().luffy_combine_backward(
        _p(dy), _p(y_rep), _p(rep_row), _p(perm_token), _p(slot_pos), _p(topk_gate), _p(offsets),
        _p(rep_offsets), E, T, k, d, _dtype_code(dy), max_rows, _p(dy_rep), _p(dgate), _p(workspace),
        workspace.numel(), _stream(stream)),
        "luffy_combine_backward")


def expert_ffn_backward_workspace_size(max_rows: int, E: int, d: int, d_ff: int, dtype: int) -> int:
    return int(load_library().luffy_expert_ffn_backward_workspace_size(max_rows, E, d, d_ff, dtype))


def luffy_expert_ffn_backward(x, row_index, rep_offsets, w1, w2, act, max_rows, dy_rep, dx_rep, dw1, dw2,
                              workspace, stream=None):
    """Gradients of luffy_expert_ffn: dx_rep [max_rows, d] (bf16), dw1
    [E, d_ff, d] and dw2 [E, d, d_ff] (float32 or bf16, both the same) from
    dy_rep."""
    E, d_ff, d = w1.shape
    if dw1.dtype != dw2.dtype:
        raise LuffyError("luffy_expert_ffn_backward: dw1 and dw2 must have the same dtype")
    _check(load_library().luffy_expert_ffn_backward(
        _p(x), _p(row_index), _p(rep_offsets), E, d, d_ff, _dtype_code(x), _p(w1), _p(w2), _ACTS[act],
        max_rows, _p(dy_rep), _p(dx_rep), _p(dw1), _p(dw2), _dtype_code(dw1), _p(workspace), workspace.numel(),
        _stream(stream)), "luffy_expert_ffn_backward")


def adaptive_threshold(l_ini: float, l_prev: float) -> float:
    """h_t of Sec. 5.2 Eq. 2 from the first and the previous loss
    (luffy_adaptive_threshold)."""
    h = ctypes.c_double()
    _check(load_library().luffy_adaptive_threshold(float(l_ini), float(l_prev), ctypes.byref(h)),
           "luffy_adaptive_threshold")
    return h.value


class AdaptiveThreshold:
    """The threshold schedule of Sec. 5.2 over a training run: threshold()
    gives h_t for the coming iteration, record(loss) takes that iteration's
    loss.  The first recorded loss is l_ini; before any loss, and for the
    iteration after the first, h_t = 1/2."""

    def __init__(self):
        self.l_ini: Optional[float] = None
        self.l_prev: Optional[float] = None

    def threshold(self) -> float:
        if self.l_ini is None:
            return 0.5
        return adaptive_threshold(self.l_ini, self.l_prev)

    def record(self, loss: float) -> None:
        if self.l_ini is None:
            self.l_ini = float(loss)
        self.l_prev = float(loss)


def profile_kernel(name: Optional[str]) -> None:
    """Selects the kernel whose launches are bracketed by HIP events (None: off)."""
    _check(load_library().luffy_profile_kernel(name.encode() if name else None),
           "luffy_profile_kernel")


def profile_read():
    """(summed milliseconds, launches) of the selected kernel since the last read."""
    ms, n = ctypes.c_double(), _c_int()
    _check(load_library().luffy_profile_read(ctypes.byref(ms), ctypes.byref(n)),
           "luffy_profile_read")
    return ms.value, n.value


KERNELS = ("gate", "slot_scan", "slot_scatter", "norm", "gram", "gram_recheck", "greedy_round",
           "greedy_more", "greedy_finish", "rep_local", "rep_finalize", "gather", "ffn_queue", "ffn1", "ffn2",
           "ffn2_reduce", "combine")


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator hands out 512-byte aligned blocks
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


@dataclass
class LayerBuffers:
    topk_idx: torch.Tensor
    topk_gate: torch.Tensor
    slot_pos: torch.Tensor
    perm_token: torch.Tensor
    offsets: torch.Tensor
    rep_of_pos: torch.Tensor
    rep_row: torch.Tensor
    rep_offsets: torch.Tensor
    rep_token: torch.Tensor
    degree: Optional[torch.Tensor]
    x_rep: Optional[torch.Tensor]
    y_rep: torch.Tensor
    y: torch.Tensor
    inv_norm: torch.Tensor
    ws_route: torch.Tensor
    ws_condense: torch.Tensor
    ws_ffn: torch.Tensor


class MoELayer:
    """Holds the weights and every buffer of one condensed MoE layer and runs
    the four library calls in order on the current stream.

    gather_x_rep=False (default) lets the FFN read representative rows of x
    through rep_token instead of materialising x_rep.
    """

    def __init__(self, w_gate, b_gate, w1, w2, *, k: int, act: str, threshold: float,
                 capacity_factor: float = 0.0, T: int, keep_degree: bool = True,
                 gather_x_rep: bool = False, norms_from_route: bool = True,
                 history: Optional[tuple] = None):
        self.w_gate, self.b_gate, self.w1, self.w2 = w_gate, b_gate, w1, w2
        self.k, self.act, self.h, self.cf = k, act, threshold, capacity_factor
        self.E, self.d_ff, self.d = w1.shape
        self.T = T
        self.norms_from_route = norms_from_route
        self.dtype = w1.dtype
        dev = w1.device
        S = T * k
        C = capacity(T, k, self.E, capacity_factor)
        self.max_bucket = min(T, C) if C > 0 else T
        # history = (S1, S2): condense with the historical similarity of the
        # previous block's record and leave this block's in self.record
        self.history = history
        i32 = dict(dtype=torch.int32, device=dev)
        self.buf = LayerBuffers(
            topk_idx=torch.empty(T, k, **i32),
            topk_gate=torch.empty(T, k, dtype=torch.float32, device=dev),
            slot_pos=torch.empty(T, k, **i32),
            perm_token=torch.empty(S, **i32),
            offsets=torch.empty(self.E + 1, **i32),
            rep_of_pos=torch.empty(S, **i32),
            rep_row=torch.empty(S, **i32),
            rep_offsets=torch.empty(self.E + 1, **i32),
            rep_token=torch.empty(S, **i32),
            degree=torch.empty(S, **i32) if keep_degree else None,
            x_rep=torch.empty(S, self.d, dtype=self.dtype, device=dev) if gather_x_rep else None,
            y_rep=torch.empty(S, self.d, dtype=self.dtype, device=dev),
            y=torch.empty(T, self.d, dtype=self.dtype, device=dev),
            inv_norm=torch.empty(T, dtype=torch.float32, device=dev),
            ws_route=_workspace(route_workspace_size(T, self.E, k), dev),
            ws_condense=_workspace((condense_history_workspace_size if history else condense_workspace_size)(
                T, self.d, self.E, k, self.max_bucket), dev),
            ws_ffn=_workspace(expert_ffn_workspace_size(
                S, self.E, self.d_ff, LUFFY_BF16 if self.dtype == torch.bfloat16 else LUFFY_F32),
                dev),
        )
        if history:
            self.record = _workspace(history_size(T, self.E, k, self.max_bucket), dev)
            self.hist_stats = torch.zeros(4, dtype=torch.int64, device=dev)

    def route(self, x, stream=None):
        b = self.buf
        luffy_route(x, self.w_gate, self.b_gate, self.k, self.cf, b.topk_idx, b.topk_gate,
                    b.slot_pos, b.perm_token, b.offsets, b.ws_route, stream, inv_norm=b.inv_norm)

    def condense(self, x, stream=None, threshold=None, hist_in=None):
        b = self.buf
        h = self.h if threshold is None else threshold
        inv = b.inv_norm if self.norms_from_route else None
        if self.history:
            S1, S2 = self.history
            luffy_condense_history(x, b.perm_token, b.offsets, b.slot_pos, self.k, self.max_bucket, h, hist_in,
                                   self.record, S1, S2, b.rep_of_pos, b.rep_row, b.rep_offsets, b.rep_token,
                                   b.x_rep, b.degree, self.hist_stats, b.ws_condense, stream, inv_norm=inv)
        else:
            if hist_in is not None:
                raise LuffyError("MoELayer: hist_in needs a layer built with history=(S1, S2)")
            luffy_condense(x, b.perm_token, b.offsets, self.k, self.max_bucket, h, b.rep_of_pos,
                           b.rep_row, b.rep_offsets, b.rep_token, b.x_rep, b.degree, b.ws_condense,
                           stream, inv_norm=inv)

    def expert_ffn(self, x, stream=None):
        b = self.buf
        if b.x_rep is not None:
            src, idx = b.x_rep, None
        else:
            src, idx = x, b.rep_token
        luffy_expert_ffn(src, idx, b.rep_offsets, self.w1, self.w2, self.act, self.T * self.k,
                         b.y_rep, b.ws_ffn, stream)

    def combine(self, stream=None):
        b = self.buf
        luffy_combine(b.y_rep, b.rep_row, b.slot_pos, b.topk_gate, b.y, stream)

    def backward(self, x, dy, stream=None, dw_dtype=torch.float32):
        """Gradients of the last call's output for dy = dL/dy [T, d], with its
        condensation held fixed (bf16 layers): returns (dgate [T, k] float32,
        dx_rep [T*k, d] with rows 0..R-1 the representatives' input
        gradients, in the order of rep_token, dw1, dw2 of dw_dtype: float32,
        or bfloat16 as the gradient of a bf16 parameter).  Buffers are
        allocated on the first call and reused."""
        b = self.buf
        if self.dtype != torch.bfloat16:
            raise LuffyError("MoELayer.backward: the expert FFN backward is bf16 only")
        S = self.T * self.k
        dev = dy.device
        if getattr(self, "_bwd", None) is None or self._bwd["dw1"].dtype != dw_dtype:
            E, dff, d = self.w1.shape
            self._bwd = dict(
                dy_rep=torch.empty_like(b.y_rep),
                dgate=torch.empty(self.T, self.k, dtype=torch.float32, device=dev),
                dx_rep=torch.empty(S, d, dtype=self.dtype, device=dev),
                dw1=torch.empty(E, dff, d, dtype=dw_dtype, device=dev),
                dw2=torch.empty(E, d, dff, dtype=dw_dtype, device=dev),
                ws_c=_workspace(combine_backward_workspace_size(self.T, self.k, S), dev),
                ws_f=_workspace(expert_ffn_backward_workspace_size(S, E, d, dff, LUFFY_BF16), dev),
            )
        g = self._bwd
        luffy_combine_backward(dy, b.y_rep, b.rep_row, b.perm_token, b.slot_pos, b.topk_gate, b.offsets,
                               b.rep_offsets, g["dy_rep"], g["dgate"], g["ws_c"], stream)
        if b.x_rep is not None:
            src, idx = b.x_rep, None
        else:
            src, idx = x, b.rep_token
        luffy_expert_ffn_backward(src, idx, b.rep_offsets, self.w1, self.w2, self.act, S, g["dy_rep"],
                                  g["dx_rep"], g["dw1"], g["dw2"], g["ws_f"], stream)
        return g["dgate"], g["dx_rep"], g["dw1"], g["dw2"]

    def __call__(self, x, stream=None, threshold=None, hist_in=None):
        if x.shape != (self.T, self.d) or x.dtype != self.dtype:
            raise LuffyError(f"x must be [{self.T}, {self.d}] {self.dtype}")
        self.route(x, stream)
        self.condense(x, stream, threshold, hist_in)
        self.expert_ffn(x, stream)
        self.combine(stream)
        return self.buf.y


class MoEStack:
    """Consecutive MoE blocks over the same tokens, each condensing with the
    historical similarity of the block before it (Sec. 5.1 step 2): block b
    reads block b-1's record (block 0 computes every pair) and leaves its
    own.  Each block takes its own input (the caller's model computes block
    b's input from block b-1's output)."""

    def __init__(self, layers):
        if not layers or any(not L.history for L in layers):
            raise LuffyError("MoEStack: every layer needs history=(S1, S2)")
        self.layers = list(layers)

    def __call__(self, xs, stream=None, threshold=None, ffn=True):
        """Runs every block on its input xs[b]; returns the blocks' outputs
        (with ffn=False only route and condense run, and nothing is
        returned)."""
        prev = None
        outs = []
        for layer, x in zip(self.layers, xs):
            layer.route(x, stream)
            layer.condense(x, stream, threshold, prev)
            if ffn:
                layer.expert_ffn(x, stream)
                layer.combine(stream)
                outs.append(layer.buf.y)
            prev = layer.record
        return outs if ffn else None


class CondensationDriver:
    """Training iterations over a stack of condensed MoE blocks with the
    adaptive threshold of Sec. 5.2 (Eq. 2): before an iteration, h_t comes
    from the first and the previous iteration's loss (AdaptiveThreshold; 1/2
    until a loss is recorded, as Eq. 2 gives for an unmoved loss); every
    block of the iteration condenses at h_t, each with the historical
    similarity of the block before it (Sec. 5.1 step 2); after it, the
    iteration's loss is recorded.  Eq. 2 as printed keeps h_t in
    (1/(1+e), 1/2] while the loss falls.

    stack: an MoEStack (or a single MoELayer, run alone)."""

    def __init__(self, stack, schedule: Optional[AdaptiveThreshold] = None):
        self.stack = stack
        self.schedule = schedule if schedule is not None else AdaptiveThreshold()
        self.thresholds = []
        self.losses = []

    def step(self, xs, loss, stream=None, ffn=True):
        """One iteration on the blocks' inputs xs (a list, one per block, or
        one tensor for a single layer).  loss: a number, or a callable that
        takes the outputs and returns this iteration's loss.  Returns
        (h_t, outputs)."""
        h = self.schedule.threshold()
        if isinstance(self.stack, MoEStack):
            outs = self.stack(xs, stream, threshold=h, ffn=ffn)
        else:
            outs = self.stack(xs, stream, threshold=h)
        value = float(loss(outs) if callable(loss) else loss)
        self.schedule.record(value)
        self.thresholds.append(h)
        self.losses.append(value)
        return h, outs
