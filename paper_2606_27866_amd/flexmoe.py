"""ctypes binding of libflexmoe.so (include/flexmoe.h).

Argument marshalling only: every step of the layer runs in the HIP library.
Functions keep the C names; device buffers are passed as torch CUDA tensors
(their data pointers), the stream defaults to torch's current stream.  There
is no fallback: if the library is missing or a call fails, an exception is
raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

from .build import LIB

FLEXMOE_F32 = 0
FLEXMOE_BF16 = 1

ERRORS = {
    -1: "FLEXMOE_EINVAL",
    -2: "FLEXMOE_ESHAPE",
    -3: "FLEXMOE_EKEEP",
    -4: "FLEXMOE_EWORKSPACE",
    -5: "FLEXMOE_EDTYPE",
    -6: "FLEXMOE_EHIP",
}

EXPORTED = ("flexmoe_workspace_bytes", "flexmoe_rank_reorder", "flexmoe_set_budget",
            "flexmoe_layer_forward", "flexmoe_keep_from_ratio", "flexmoe_last_error",
            "flexmoe_timing_enable", "flexmoe_timing_read", "flexmoe_clipped_channels",
            "flexmoe_export_clipped", "flexmoe_layer_forward_clipped",
            "flexmoe_layer_forward_bucketed", "flexmoe_saliency_workspace_bytes",
            "flexmoe_channel_saliency", "flexmoe_transpose_weights", "flexmoe_sample_actions",
            "flexmoe_train_workspace_bytes", "flexmoe_train_forward", "flexmoe_train_backward",
            "flexmoe_action_grad", "flexmoe_layer_forward_noalloc")

# kernel indices of flexmoe_kernel_times
KERNELS = ("route", "dispatch_scan", "dispatch_scatter", "gate_up", "down", "combine",
           "gate_up_shared", "down_shared", "sal_transpose", "sal_prep", "sal_dgrad", "sal_wgrad",
           "sal_reduce", "act_dgrad", "act_dx", "act_other")
MAX_ACTIONS = 16


class FlexMoEError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("%s (%d): %s" % (ERRORS.get(code, "?"), code, msg))
        self.code = code


class flexmoe_layer_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("d", "E", "I", "top_k", "I_shared", "dtype", "norm_topk", "max_tokens")]


class flexmoe_kernel_times(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * len(KERNELS)), ("launches", ctypes.c_int64 * len(KERNELS))]


class flexmoe_action_set(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("ratio", ctypes.c_double * MAX_ACTIONS)]


def make_actions(ratios) -> flexmoe_action_set:
    a = flexmoe_action_set()
    a.K = len(ratios)
    for i, r in enumerate(ratios):
        a.ratio[i] = float(r)
    return a


class flexmoe_route_out(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("topk_idx", "topk_w", "counts", "offsets", "perm", "pos")]


_lib = None


def lib():
    """Load libflexmoe.so (built in-tree by build.py); raise if it is absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise RuntimeError("libflexmoe.so is not built (%s); run "
                               "`python -m paper_2606_27866_amd.build`" % LIB)
        # torch ships its own HIP runtime (soname libamdhip64.so.7).  Loading
        # torch first makes the library's libamdhip64.so.7 dependency resolve
        # to that same runtime, so device pointers and streams are shared; a
        # second runtime in the process would not see the GPU.
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        D = ctypes.POINTER(flexmoe_layer_desc)
        L.flexmoe_workspace_bytes.argtypes = [D, i32]
        L.flexmoe_workspace_bytes.restype = sz
        L.flexmoe_rank_reorder.argtypes = [D] + [vp] * 9
        L.flexmoe_rank_reorder.restype = ctypes.c_int
        L.flexmoe_set_budget.argtypes = [D, vp, vp, vp]
        L.flexmoe_set_budget.restype = ctypes.c_int
        L.flexmoe_layer_forward.argtypes = [D, i32] + [vp] * 11 + [sz, ctypes.POINTER(flexmoe_route_out), vp]
        L.flexmoe_layer_forward.restype = ctypes.c_int
        L.flexmoe_layer_forward_noalloc.argtypes = [D, i32] + [vp] * 10 + [ctypes.POINTER(flexmoe_route_out), vp]
        L.flexmoe_layer_forward_noalloc.restype = ctypes.c_int
        L.flexmoe_clipped_channels.argtypes = [D, vp]
        L.flexmoe_clipped_channels.restype = ctypes.c_int64
        L.flexmoe_export_clipped.argtypes = [D] + [vp] * 8
        L.flexmoe_export_clipped.restype = ctypes.c_int
        L.flexmoe_layer_forward_clipped.argtypes = ([D, i32] + [vp] * 6 + [ctypes.c_int64] + [vp] * 5
                                                    + [sz, ctypes.POINTER(flexmoe_route_out), vp])
        L.flexmoe_layer_forward_clipped.restype = ctypes.c_int
        L.flexmoe_layer_forward_bucketed.argtypes = ([D, i32] + [vp] * 6 + [i32] + [vp] * 5
                                                     + [sz, ctypes.POINTER(flexmoe_route_out), vp])
        L.flexmoe_layer_forward_bucketed.restype = ctypes.c_int
        L.flexmoe_saliency_workspace_bytes.argtypes = [D, i32]
        L.flexmoe_saliency_workspace_bytes.restype = sz
        L.flexmoe_channel_saliency.argtypes = ([D, i32] + [vp] * 10 + [ctypes.c_float] + [vp] * 2
                                               + [sz, vp])
        L.flexmoe_channel_saliency.restype = ctypes.c_int
        AS = ctypes.POINTER(flexmoe_action_set)
        f32 = ctypes.c_float
        L.flexmoe_transpose_weights.argtypes = [D] + [vp] * 13
        L.flexmoe_transpose_weights.restype = ctypes.c_int
        L.flexmoe_sample_actions.argtypes = [D, AS] + [vp] * 5
        L.flexmoe_sample_actions.restype = ctypes.c_int
        L.flexmoe_train_workspace_bytes.argtypes = [D, i32]
        L.flexmoe_train_workspace_bytes.restype = sz
        L.flexmoe_train_forward.argtypes = [D, i32] + [vp] * 11 + [sz, vp]
        L.flexmoe_train_forward.restype = ctypes.c_int
        L.flexmoe_train_backward.argtypes = [D, i32] + [vp] * 12 + [sz, vp]
        L.flexmoe_train_backward.restype = ctypes.c_int
        L.flexmoe_action_grad.argtypes = [D, i32, AS, vp, vp, f32, f32, f32, vp, vp, vp, vp, sz, vp]
        L.flexmoe_action_grad.restype = ctypes.c_int
        L.flexmoe_keep_from_ratio.argtypes = [ctypes.c_double, i32]
        L.flexmoe_keep_from_ratio.restype = ctypes.c_int
        L.flexmoe_timing_enable.argtypes = [ctypes.c_int]
        L.flexmoe_timing_enable.restype = ctypes.c_int
        L.flexmoe_timing_read.argtypes = [ctypes.POINTER(flexmoe_kernel_times)]
        L.flexmoe_timing_read.restype = ctypes.c_int
        L.flexmoe_last_error.argtypes = []
        L.flexmoe_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(rc: int):
    if rc != 0:
        raise FlexMoEError(rc, lib().flexmoe_last_error().decode())


def _p(t) -> Optional[int]:
    """Device pointer of a tensor (or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def make_desc(d, E, I, top_k, I_shared=0, dtype=FLEXMOE_BF16, norm_topk=1, max_tokens=0):
    return flexmoe_layer_desc(d, E, I, top_k, I_shared, dtype, norm_topk, max_tokens)


def flexmoe_last_error() -> str:
    return lib().flexmoe_last_error().decode()


def flexmoe_timing_enable(on: bool):
    _check(lib().flexmoe_timing_enable(1 if on else 0))


def flexmoe_timing_read():
    """{kernel name: (total ms, launches)} since the last enable/read."""
    t = flexmoe_kernel_times()
    _check(lib().flexmoe_timing_read(ctypes.byref(t)))
    return {n: (t.ms[i], int(t.launches[i])) for i, n in enumerate(KERNELS)}


def flexmoe_keep_from_ratio(r: float, I: int) -> int:
    return int(lib().flexmoe_keep_from_ratio(float(r), int(I)))


def flexmoe_workspace_bytes(desc: flexmoe_layer_desc, T: int) -> int:
    n = lib().flexmoe_workspace_bytes(ctypes.byref(desc), int(T))
    if n == 0:
        raise FlexMoEError(-2, flexmoe_last_error())
    return int(n)


def flexmoe_set_budget(desc, keep_dev, keep_host: Sequence[int], stream=None):
    kh = np.ascontiguousarray(np.asarray(keep_host, dtype=np.int32))
    _check(lib().flexmoe_set_budget(ctypes.byref(desc), _p(keep_dev),
                                    kh.ctypes.data_as(ctypes.c_void_p), _stream(stream)))


def flexmoe_rank_reorder(desc, scores, w_gate, w_up, w_down, w_gate_r, w_up_r, w_down_r, perm,
                         stream=None):
    _check(lib().flexmoe_rank_reorder(ctypes.byref(desc), _p(scores), _p(w_gate), _p(w_up),
                                      _p(w_down), _p(w_gate_r), _p(w_up_r), _p(w_down_r), _p(perm),
                                      _stream(stream)))


def flexmoe_layer_forward(desc, T, x, logits, w_gate_r, w_up_r, w_down_r, keep_dev, ws_gate,
                          ws_up, ws_down, y, workspace, workspace_bytes=None, dbg=None,
                          stream=None):
    """dbg: optional dict with any of topk_idx, topk_w, counts, offsets, perm, pos tensors."""
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size()
    ro = None
    if dbg:
        ro = flexmoe_route_out(*[_p(dbg.get(n)) for n, _ in flexmoe_route_out._fields_])
    _check(lib().flexmoe_layer_forward(
        ctypes.byref(desc), int(T), _p(x), _p(logits), _p(w_gate_r), _p(w_up_r), _p(w_down_r),
        _p(keep_dev), _p(ws_gate), _p(ws_up), _p(ws_down), _p(y), _p(workspace),
        int(workspace_bytes), ctypes.byref(ro) if ro is not None else None, _stream(stream)))


def flexmoe_layer_forward_noalloc(desc, T, x, logits, w_gate_r, w_up_r, w_down_r, keep_dev, ws_gate,
                                  ws_up, ws_down, y, dbg=None, stream=None):
    """flexmoe_layer_forward without a workspace (the library's static scratch)."""
    ro = None
    if dbg:
        ro = flexmoe_route_out(*[_p(dbg.get(n)) for n, _ in flexmoe_route_out._fields_])
    _check(lib().flexmoe_layer_forward_noalloc(
        ctypes.byref(desc), int(T), _p(x), _p(logits), _p(w_gate_r), _p(w_up_r), _p(w_down_r),
        _p(keep_dev), _p(ws_gate), _p(ws_up), _p(ws_down), _p(y),
        ctypes.byref(ro) if ro is not None else None, _stream(stream)))


def flexmoe_clipped_channels(desc, keep_host: Sequence[int]) -> int:
    kh = np.ascontiguousarray(np.asarray(keep_host, dtype=np.int32))
    n = int(lib().flexmoe_clipped_channels(ctypes.byref(desc), kh.ctypes.data_as(ctypes.c_void_p)))
    if n < 0:
        raise FlexMoEError(n, flexmoe_last_error())
    return n


def flexmoe_export_clipped(desc, keep_host, w_gate_r, w_up_r, w_down_r, w_gate_c, w_up_c, w_down_c,
                           stream=None):
    kh = np.ascontiguousarray(np.asarray(keep_host, dtype=np.int32))
    _check(lib().flexmoe_export_clipped(ctypes.byref(desc), kh.ctypes.data_as(ctypes.c_void_p),
                                        _p(w_gate_r), _p(w_up_r), _p(w_down_r), _p(w_gate_c),
                                        _p(w_up_c), _p(w_down_c), _stream(stream)))


def flexmoe_layer_forward_clipped(desc, T, x, logits, w_gate_c, w_up_c, w_down_c, keep_dev,
                                  packed_channels, ws_gate, ws_up, ws_down, y, workspace,
                                  workspace_bytes=None, dbg=None, stream=None):
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size()
    ro = None
    if dbg:
        ro = flexmoe_route_out(*[_p(dbg.get(n)) for n, _ in flexmoe_route_out._fields_])
    _check(lib().flexmoe_layer_forward_clipped(
        ctypes.byref(desc), int(T), _p(x), _p(logits), _p(w_gate_c), _p(w_up_c), _p(w_down_c),
        _p(keep_dev), int(packed_channels), _p(ws_gate), _p(ws_up), _p(ws_down), _p(y),
        _p(workspace), int(workspace_bytes), ctypes.byref(ro) if ro is not None else None,
        _stream(stream)))


def flexmoe_layer_forward_bucketed(desc, T, x, logits, w_gate_r, w_up_r, w_down_r, keep_host, k_align,
                                   ws_gate, ws_up, ws_down, y, workspace, workspace_bytes=None,
                                   dbg=None, stream=None):
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size()
    kh = np.ascontiguousarray(np.asarray(keep_host, dtype=np.int32))
    ro = None
    if dbg:
        ro = flexmoe_route_out(*[_p(dbg.get(n)) for n, _ in flexmoe_route_out._fields_])
    _check(lib().flexmoe_layer_forward_bucketed(
        ctypes.byref(desc), int(T), _p(x), _p(logits), _p(w_gate_r), _p(w_up_r), _p(w_down_r),
        kh.ctypes.data_as(ctypes.c_void_p), int(k_align), _p(ws_gate), _p(ws_up), _p(ws_down), _p(y),
        _p(workspace), int(workspace_bytes), ctypes.byref(ro) if ro is not None else None,
        _stream(stream)))


def flexmoe_saliency_workspace_bytes(desc: flexmoe_layer_desc, T: int) -> int:
    n = lib().flexmoe_saliency_workspace_bytes(ctypes.byref(desc), int(T))
    if n == 0:
        raise FlexMoEError(-2, lib().flexmoe_last_error().decode())
    return n


def flexmoe_channel_saliency(desc, T, x, logits, w_gate, w_up, w_down, w_down_t, ws_gate, ws_up, ws_down,
                             y_target, scale, scores, workspace, workspace_bytes=None, stream=None):
    nbytes = workspace.numel() * workspace.element_size() if workspace_bytes is None else workspace_bytes
    _check(lib().flexmoe_channel_saliency(ctypes.byref(desc), int(T), _p(x), _p(logits), _p(w_gate),
                                          _p(w_up), _p(w_down), _p(w_down_t), _p(ws_gate), _p(ws_up),
                                          _p(ws_down), _p(y_target), float(scale), _p(scores), _p(workspace),
                                          nbytes, _stream(stream)))


def _nbytes(t, given):
    return t.numel() * t.element_size() if given is None else given


def flexmoe_transpose_weights(desc, w_gate, w_up, w_down, ws_gate, ws_up, ws_down, w_gate_t, w_up_t, w_down_t,
                              ws_gate_t, ws_up_t, ws_down_t, stream=None):
    _check(lib().flexmoe_transpose_weights(ctypes.byref(desc), *[_p(t) for t in (
        w_gate, w_up, w_down, ws_gate, ws_up, ws_down, w_gate_t, w_up_t, w_down_t, ws_gate_t, ws_up_t,
        ws_down_t)], _stream(stream)))


def flexmoe_sample_actions(desc, actions, alpha, gumbel, keep_dev, action_dev=None, stream=None):
    _check(lib().flexmoe_sample_actions(ctypes.byref(desc), ctypes.byref(actions), _p(alpha), _p(gumbel),
                                        _p(keep_dev), _p(action_dev), _stream(stream)))


def flexmoe_train_workspace_bytes(desc, T: int) -> int:
    n = lib().flexmoe_train_workspace_bytes(ctypes.byref(desc), int(T))
    if n == 0:
        raise FlexMoEError(-2, lib().flexmoe_last_error().decode())
    return n


def flexmoe_train_forward(desc, T, x, logits, w_gate, w_up, w_down, keep_dev, ws_gate, ws_up, ws_down, y,
                          workspace, workspace_bytes=None, stream=None):
    _check(lib().flexmoe_train_forward(ctypes.byref(desc), int(T), _p(x), _p(logits), _p(w_gate), _p(w_up),
                                       _p(w_down), _p(keep_dev), _p(ws_gate), _p(ws_up), _p(ws_down), _p(y),
                                       _p(workspace), _nbytes(workspace, workspace_bytes), _stream(stream)))


def flexmoe_train_backward(desc, T, logits, dy, w_gate_t, w_up_t, w_down_t, ws_gate_t, ws_up_t, ws_down_t, dx,
                           dlogits, dmask, workspace, workspace_bytes=None, stream=None):
    _check(lib().flexmoe_train_backward(ctypes.byref(desc), int(T), _p(logits), _p(dy), _p(w_gate_t),
                                        _p(w_up_t), _p(w_down_t), _p(ws_gate_t), _p(ws_up_t), _p(ws_down_t),
                                        _p(dx), _p(dlogits), _p(dmask), _p(workspace),
                                        _nbytes(workspace, workspace_bytes), _stream(stream)))


def flexmoe_action_grad(desc, T, actions, alpha, gumbel, tau, lambda_cost, beta, dmask, dalpha, stats,
                        workspace, workspace_bytes=None, stream=None):
    _check(lib().flexmoe_action_grad(ctypes.byref(desc), int(T), ctypes.byref(actions), _p(alpha), _p(gumbel),
                                     float(tau), float(lambda_cost), float(beta), _p(dmask), _p(dalpha),
                                     _p(stats), _p(workspace), _nbytes(workspace, workspace_bytes),
                                     _stream(stream)))


class ClippedWeights:
    """The packed weights of one exported budget (offline clipping) and its
    device keep table."""

    def __init__(self, keep_host, w_gate_c, w_up_c, w_down_c, packed_channels, keep_dev):
        self.keep_host = np.asarray(keep_host, dtype=np.int32).copy()
        self.w_gate_c, self.w_up_c, self.w_down_c = w_gate_c, w_up_c, w_down_c
        self.packed_channels = packed_channels
        self.keep_dev = keep_dev


class Layer:
    """Device-resident masked MoE layer: weights, keep table, workspace.

    A thin holder around the C calls (no arithmetic): it allocates torch
    buffers once and forwards with the library.
    """

    def __init__(self, d, E, I, top_k, I_shared=0, dtype=FLEXMOE_BF16, norm_topk=1,
                 max_tokens=1, device="cuda"):
        import torch
        self.desc = make_desc(d, E, I, top_k, I_shared, dtype, norm_topk, max_tokens)
        self.tdtype = torch.bfloat16 if dtype == FLEXMOE_BF16 else torch.float32
        self.device = device
        self.keep = torch.full((E,), I, dtype=torch.int32, device=device)
        nbytes = flexmoe_workspace_bytes(self.desc, max_tokens)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.w_gate = self.w_up = self.w_down = None
        self.ws_gate = self.ws_up = self.ws_down = None

    def set_weights(self, w_gate, w_up, w_down, ws_gate=None, ws_up=None, ws_down=None):
        self.w_gate, self.w_up, self.w_down = w_gate, w_up, w_down
        self.ws_gate, self.ws_up, self.ws_down = ws_gate, ws_up, ws_down

    def set_budget(self, keep_host, stream=None):
        flexmoe_set_budget(self.desc, self.keep, keep_host, stream)

    def export_clipped(self, keep_host, stream=None) -> ClippedWeights:
        """Pack the current ranked weights for the budget keep_host."""
        import torch
        P = flexmoe_clipped_channels(self.desc, keep_host)
        bufs = [torch.empty((max(P, 1) * self.desc.d,), dtype=self.tdtype, device=self.device)
                for _ in range(3)]
        flexmoe_export_clipped(self.desc, keep_host, self.w_gate, self.w_up, self.w_down, *bufs,
                               stream=stream)
        keep_dev = torch.from_numpy(np.asarray(keep_host, dtype=np.int32).copy()).to(self.device)
        return ClippedWeights(keep_host, *bufs, P, keep_dev)

    def forward(self, x, logits, y=None, keep=None, dbg=None, stream=None, clipped=None,
                bucketed=None):
        """clipped: a ClippedWeights of this layer -> the offline-clipped path;
        bucketed: (keep_host, k_align) -> the bucketed ablation."""
        import torch
        T = x.shape[0]
        if y is None:
            y = torch.empty((T, self.desc.d), dtype=self.tdtype, device=self.device)
        if bucketed is not None:
            flexmoe_layer_forward_bucketed(self.desc, T, x, logits, self.w_gate, self.w_up, self.w_down,
                                           bucketed[0], bucketed[1], self.ws_gate, self.ws_up,
                                           self.ws_down, y, self.workspace, dbg=dbg, stream=stream)
            return y
        if clipped is not None:
            flexmoe_layer_forward_clipped(self.desc, T, x, logits, clipped.w_gate_c, clipped.w_up_c,
                                          clipped.w_down_c, clipped.keep_dev if keep is None else keep,
                                          clipped.packed_channels, self.ws_gate, self.ws_up,
                                          self.ws_down, y, self.workspace, dbg=dbg, stream=stream)
            return y
        flexmoe_layer_forward(self.desc, T, x, logits, self.w_gate, self.w_up, self.w_down,
                              self.keep if keep is None else keep, self.ws_gate, self.ws_up,
                              self.ws_down, y, self.workspace, dbg=dbg, stream=stream)
        return y


class Saliency:
    """Channel ranking on the device (Sec. 3.1): the running Eq. 2 scores of
    one layer over calibration batches, then the reorder of Eq. 3.

    Holds the score table and a saliency workspace for up to max_tokens
    tokens per batch; the weights are those of `layer` (original order).
    """

    def __init__(self, layer: "Layer", max_tokens: int, transpose_once: bool = True):
        import torch
        self.layer = layer
        D = layer.desc
        self.desc = make_desc(D.d, D.E, D.I, D.top_k, D.I_shared, D.dtype, D.norm_topk, max_tokens)
        nbytes = flexmoe_saliency_workspace_bytes(self.desc, max_tokens)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=layer.device)
        self.scores = torch.zeros((D.E, D.I), dtype=torch.float32, device=layer.device)
        self.w_down_t = None
        if transpose_once:   # W_down^T made once for the whole ranking set
            self.w_down_t = torch.empty((D.E, D.I, D.d), dtype=layer.tdtype, device=layer.device)
            flexmoe_transpose_weights(self.desc, None, None, layer.w_down, None, None, None,
                                      None, None, self.w_down_t, None, None, None)

    def add_batch(self, x, logits, y_target, scale=1.0, stream=None):
        L = self.layer
        flexmoe_channel_saliency(self.desc, x.shape[0], x, logits, L.w_gate, L.w_up, L.w_down, self.w_down_t,
                                 L.ws_gate, L.ws_up, L.ws_down, y_target, scale, self.scores, self.workspace,
                                 stream=stream)

    def rank_reorder(self, stream=None):
        """Ranked copies of the layer's weights and the permutation (Eq. 3)."""
        import torch
        L = self.layer
        out = [torch.empty_like(w) for w in (L.w_gate, L.w_up, L.w_down)]
        perm = torch.empty((L.desc.E, L.desc.I), dtype=torch.int32, device=L.device)
        flexmoe_rank_reorder(L.desc, self.scores, L.w_gate, L.w_up, L.w_down, *out, perm, stream=stream)
        return (*out, perm)


class ActionLearner:
    """One layer's action-learning step on the device (Sec. 3.2): sample the
    per-expert widths (Eq. 5), run the sampled subnet forward, backward for
    an upstream gradient, and the action-logit gradient (Eqs. 6-8).

    Holds the transposed weight copies (made once: the weights are frozen),
    the sampled keep table and a training workspace for up to max_tokens.
    """

    def __init__(self, layer: "Layer", max_tokens: int, ratios):
        import torch
        self.layer = layer
        D = layer.desc
        self.desc = make_desc(D.d, D.E, D.I, D.top_k, D.I_shared, D.dtype, D.norm_topk, max_tokens)
        self.actions = make_actions(ratios)
        dev = layer.device
        nbytes = flexmoe_train_workspace_bytes(self.desc, max_tokens)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        bf = layer.tdtype
        self.wt = [torch.empty((D.E, D.d, D.I), dtype=bf, device=dev),
                   torch.empty((D.E, D.d, D.I), dtype=bf, device=dev),
                   torch.empty((D.E, D.I, D.d), dtype=bf, device=dev)]
        if D.I_shared:
            self.wst = [torch.empty((D.d, D.I_shared), dtype=bf, device=dev),
                        torch.empty((D.d, D.I_shared), dtype=bf, device=dev),
                        torch.empty((D.I_shared, D.d), dtype=bf, device=dev)]
        else:
            self.wst = [None, None, None]
        self.keep = torch.zeros((D.E,), dtype=torch.int32, device=dev)
        self.action = torch.zeros((D.E,), dtype=torch.int32, device=dev)
        self.T = 0

    def transpose_weights(self, stream=None):
        L = self.layer
        flexmoe_transpose_weights(self.desc, L.w_gate, L.w_up, L.w_down, L.ws_gate, L.ws_up, L.ws_down,
                                  *self.wt, *self.wst, stream=stream)

    def sample(self, alpha, gumbel, stream=None):
        flexmoe_sample_actions(self.desc, self.actions, alpha, gumbel, self.keep, self.action, stream=stream)

    def forward(self, x, logits, y=None, keep=None, stream=None):
        import torch
        L = self.layer
        self.T = x.shape[0]
        if y is None:
            y = torch.empty((self.T, self.desc.d), dtype=L.tdtype, device=L.device)
        flexmoe_train_forward(self.desc, self.T, x, logits, L.w_gate, L.w_up, L.w_down,
                              self.keep if keep is None else keep, L.ws_gate, L.ws_up, L.ws_down, y,
                              self.workspace, stream=stream)
        return y

    def backward(self, logits, dy, stream=None):
        import torch
        D, dev = self.desc, self.layer.device
        dx = torch.empty((self.T, D.d), dtype=torch.float32, device=dev)
        dl = torch.empty((self.T, D.E), dtype=torch.float32, device=dev)
        dm = torch.empty((D.E, D.I), dtype=torch.float32, device=dev)
        flexmoe_train_backward(D, self.T, logits, dy, *self.wt, *self.wst, dx, dl, dm, self.workspace,
                               stream=stream)
        return dx, dl, dm

    def action_grad(self, alpha, gumbel, tau, lambda_cost, beta, dmask, stream=None):
        import torch
        dalpha = torch.empty_like(alpha)
        stats = torch.empty((2,), dtype=torch.float32, device=alpha.device)
        flexmoe_action_grad(self.desc, self.T, self.actions, alpha, gumbel, tau, lambda_cost, beta, dmask, dalpha,
                            stats, self.workspace, stream=stream)
        return dalpha, stats


def to_device(a: np.ndarray, device="cuda"):
    """NumPy array (fp32, int32, or uint16 bf16 bits) -> torch CUDA tensor."""
    import torch
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def to_host(t) -> np.ndarray:
    """torch tensor -> NumPy (bf16 becomes uint16 bits)."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()
