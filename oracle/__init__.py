"""Python access to the CPU oracle of the masked MoE layer (fp64).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg use this package; the product package never imports it.
The arithmetic lives in ``flexmoe_oracle.c`` (plain C, fp64 accumulation);
this module only marshals NumPy arrays.  See that file's header for what is
computed and which passages of the paper each function follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "flexmoe_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# A test that checks the pins against deliberately broken copies of the
# oracle points this at such a copy (built in a temporary directory).
_LIB_OVERRIDE = os.environ.get("FLEXMOE_ORACLE_LIB")

F32 = 0
BF16 = 1


# The timing build of the CPU baseline: the same source with fp32
# accumulators in the forward's dot products, -O3 -march=native.  The parity
# checks use the fp64 build only.
_LIB_F32ACC = os.path.join(_HERE, "liboracle_f32acc.so")
_FLAGS = {"fp64": (_LIB, ["-O2"]),
          "f32acc": (_LIB_F32ACC, ["-O3", "-march=native", "-DORACLE_ACC_F32"])}


def build(force: bool = False, variant: str = "fp64") -> str:
    """Compile the oracle with gcc (OpenMP over independent tokens/rows)."""
    path, flags = _FLAGS[variant]
    if force or not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
        tmp = path + ".tmp%d" % os.getpid()
        cmd = ["gcc", *flags, "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, path)
    return path


_libs = {}


def lib(variant: str = "fp64"):
    if variant not in _libs:
        if _LIB_OVERRIDE and variant == "fp64":
            L = ctypes.CDLL(_LIB_OVERRIDE)
        else:
            path = _FLAGS[variant][0]
            if not os.path.exists(path):
                build(variant=variant)
            L = ctypes.CDLL(path)
        p = ctypes.c_void_p
        i = ctypes.c_int
        L.oracle_route.argtypes = [i, i, i, p, i, p, p]
        L.oracle_dispatch.argtypes = [i, i, i, p, p, p, p, p, p]
        L.oracle_layer_forward.argtypes = [i] * 8 + [p] * 16
        L.oracle_rank_reorder.argtypes = [i, i, i, i] + [p] * 8
        L.oracle_keep_from_ratio.argtypes = [ctypes.c_double, i]
        L.oracle_num_threads.argtypes = []
        L.oracle_layer_grads.argtypes = [i] * 8 + [p] * 14
        L.oracle_channel_saliency.argtypes = [i] * 4 + [p] * 7
        L.oracle_sample_actions.argtypes = [i, i, p, i, p, p, ctypes.c_double, p, p, p]
        L.oracle_masked_backward.argtypes = [i] * 8 + [p] * 13
        L.oracle_action_grad.argtypes = [i, i, p, i, p, p, ctypes.c_double, p, p, ctypes.c_longlong,
                                         ctypes.c_double, ctypes.c_double, p, p, p]
        fns = [L.oracle_sample_actions, L.oracle_masked_backward, L.oracle_action_grad, L.oracle_route,
               L.oracle_dispatch, L.oracle_layer_forward, L.oracle_rank_reorder, L.oracle_keep_from_ratio,
               L.oracle_num_threads, L.oracle_layer_grads, L.oracle_channel_saliency]
        if hasattr(L, "oracle_set_threads"):  # absent from older mutant copies
            L.oracle_set_threads.argtypes = [i]
            L.oracle_acc_f32.argtypes = []
            fns += [L.oracle_set_threads, L.oracle_acc_f32]
        for f in fns:
            f.restype = ctypes.c_int
        _libs[variant] = L
    return _libs[variant]


def set_threads(n: int, variant: str = "fp64") -> int:
    """OpenMP threads of the oracle's loops (for CPU-baseline timing)."""
    return int(lib(variant).oracle_set_threads(int(n)))


def _ptr(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _dtype_of(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError("x / weights must be float32 or uint16 (bf16 bits), got %s" % a.dtype)


def route(logits: np.ndarray, k: int, norm_topk: int):
    """Top-k expert ids [T][k] (int32) and router weights [T][k] (fp64)."""
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    T, E = logits.shape
    idx = np.empty((T, k), dtype=np.int32)
    w = np.empty((T, k), dtype=np.float64)
    rc = lib().oracle_route(T, E, k, _ptr(logits), int(norm_topk), _ptr(idx), _ptr(w))
    if rc != 0:
        raise ValueError("oracle_route failed (%d)" % rc)
    return idx, w


def dispatch(idx: np.ndarray, keep: np.ndarray, E: int):
    """counts [E], offsets [E+1], perm [P], pos [T*k]."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    keep = np.ascontiguousarray(keep, dtype=np.int32)
    T, k = idx.shape
    counts = np.empty(E, dtype=np.int32)
    offsets = np.empty(E + 1, dtype=np.int32)
    perm = np.empty(T * k, dtype=np.int32)
    pos = np.empty(T * k, dtype=np.int32)
    P = lib().oracle_dispatch(T, E, k, _ptr(idx), _ptr(keep), _ptr(counts), _ptr(offsets),
                              _ptr(perm), _ptr(pos))
    if P < 0:
        raise ValueError("oracle_dispatch failed")
    return counts, offsets, perm[:P].copy(), pos


def layer_forward(x, logits, w_gate, w_up, w_down, keep, top_k, norm_topk,
                  ws_gate=None, ws_up=None, ws_down=None, want_route=False, variant="fp64"):
    """Masked MoE layer: y [T][d] fp64 (unrounded).

    x [T][d]; logits [T][E] fp32; w_gate/w_up [E][I][d]; w_down [E][d][I];
    keep [E] int32; shared weights [I_s][d], [I_s][d], [d][I_s] or None.
    x and weights are float32 or uint16 bf16 bits (all the same type).
    """
    x = np.ascontiguousarray(x)
    dtype = _dtype_of(x)
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    T, d = x.shape
    E, I, d2 = w_gate.shape
    assert d2 == d and logits.shape == (T, E)
    for a in (w_gate, w_up, w_down):
        assert _dtype_of(a) == dtype
    assert w_down.shape == (E, d, I)
    I_s = 0
    if ws_gate is not None:
        I_s = ws_gate.shape[0]
        assert ws_up.shape == (I_s, d) and ws_down.shape == (d, I_s)
    keep = np.ascontiguousarray(keep, dtype=np.int32)
    y = np.empty((T, d), dtype=np.float64)
    A = T * top_k
    idx = np.empty((T, top_k), dtype=np.int32)
    w = np.empty((T, top_k), dtype=np.float64)
    counts = np.empty(E, dtype=np.int32)
    offsets = np.empty(E + 1, dtype=np.int32)
    perm = np.empty(max(A, 1), dtype=np.int32)
    pos = np.empty(max(A, 1), dtype=np.int32)
    rc = lib(variant).oracle_layer_forward(
        T, d, E, I, top_k, I_s, dtype, int(norm_topk), _ptr(x), _ptr(logits),
        _ptr(np.ascontiguousarray(w_gate)), _ptr(np.ascontiguousarray(w_up)),
        _ptr(np.ascontiguousarray(w_down)), _ptr(keep),
        _ptr(None if ws_gate is None else np.ascontiguousarray(ws_gate)),
        _ptr(None if ws_up is None else np.ascontiguousarray(ws_up)),
        _ptr(None if ws_down is None else np.ascontiguousarray(ws_down)),
        _ptr(y), _ptr(idx), _ptr(w), _ptr(counts), _ptr(offsets), _ptr(perm), _ptr(pos))
    if rc != 0:
        raise ValueError("oracle_layer_forward failed (%d)" % rc)
    if not want_route:
        return y
    P = int(offsets[E]) if T > 0 else 0
    return y, dict(idx=idx, w=w, counts=counts, offsets=offsets, perm=perm[:P].copy(),
                   pos=pos[:A].copy())


def rank_reorder(scores, w_gate, w_up, w_down):
    """Eq. 3 reorder: returns (w_gate_r, w_up_r, w_down_r, perm [E][I])."""
    scores = np.ascontiguousarray(scores, dtype=np.float32)
    E, I = scores.shape
    dtype = _dtype_of(w_gate)
    d = w_gate.shape[2]
    wg_r = np.empty(w_gate.shape, dtype=w_gate.dtype)
    wu_r = np.empty(w_up.shape, dtype=w_up.dtype)
    wd_r = np.empty(w_down.shape, dtype=w_down.dtype)
    perm = np.empty((E, I), dtype=np.int32)
    rc = lib().oracle_rank_reorder(E, I, d, dtype, _ptr(scores), _ptr(np.ascontiguousarray(w_gate)),
                                   _ptr(np.ascontiguousarray(w_up)), _ptr(np.ascontiguousarray(w_down)),
                                   _ptr(wg_r), _ptr(wu_r), _ptr(wd_r), _ptr(perm))
    if rc != 0:
        raise ValueError("oracle_rank_reorder failed (%d)" % rc)
    return wg_r, wu_r, wd_r, perm


def layer_grads(x, logits, w_gate, w_up, w_down, keep, top_k, norm_topk, y_target,
                ws_gate=None, ws_up=None, ws_down=None):
    """Gradients of L = 1/2 sum_t ||y_t - y_target_t||^2 of the masked layer
    with respect to the routed expert weights (the g of Eq. 2).

    Returns (L, g_gate [E][I][d], g_up [E][I][d], g_down [E][d][I]), fp64.
    Same argument conventions as layer_forward; y_target [T][d] fp32.
    """
    x = np.ascontiguousarray(x)
    dtype = _dtype_of(x)
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    T, d = x.shape
    E, I, _ = w_gate.shape
    I_s = 0 if ws_gate is None else ws_gate.shape[0]
    y_target = np.ascontiguousarray(y_target, dtype=np.float32)
    assert y_target.shape == (T, d)
    keep = np.ascontiguousarray(keep, dtype=np.int32)
    gg = np.empty((E, I, d), dtype=np.float64)
    gu = np.empty((E, I, d), dtype=np.float64)
    gd = np.empty((E, d, I), dtype=np.float64)
    loss = np.zeros(1, dtype=np.float64)
    rc = lib().oracle_layer_grads(
        T, d, E, I, top_k, I_s, dtype, int(norm_topk), _ptr(x), _ptr(logits),
        _ptr(np.ascontiguousarray(w_gate)), _ptr(np.ascontiguousarray(w_up)),
        _ptr(np.ascontiguousarray(w_down)), _ptr(keep),
        _ptr(None if ws_gate is None else np.ascontiguousarray(ws_gate)),
        _ptr(None if ws_up is None else np.ascontiguousarray(ws_up)),
        _ptr(None if ws_down is None else np.ascontiguousarray(ws_down)),
        _ptr(y_target), _ptr(loss), _ptr(gg), _ptr(gu), _ptr(gd))
    if rc != 0:
        raise ValueError("oracle_layer_grads failed (%d)" % rc)
    return float(loss[0]), gg, gu, gd


def channel_saliency_from_grads(w_gate, w_up, w_down, g_gate, g_up, g_down):
    """Eq. 2 for one batch: s[e][j] = sum over channel j's group of (theta * g)^2."""
    dtype = _dtype_of(w_gate)
    E, I, d = w_gate.shape
    s = np.empty((E, I), dtype=np.float64)
    rc = lib().oracle_channel_saliency(
        d, E, I, dtype, _ptr(np.ascontiguousarray(w_gate)), _ptr(np.ascontiguousarray(w_up)),
        _ptr(np.ascontiguousarray(w_down)), _ptr(np.ascontiguousarray(g_gate, dtype=np.float64)),
        _ptr(np.ascontiguousarray(g_up, dtype=np.float64)),
        _ptr(np.ascontiguousarray(g_down, dtype=np.float64)), _ptr(s))
    if rc != 0:
        raise ValueError("oracle_channel_saliency failed (%d)" % rc)
    return s


def channel_saliency(batches, w_gate, w_up, w_down, top_k, norm_topk,
                     ws_gate=None, ws_up=None, ws_down=None):
    """Eq. 2 over a ranking set: the mean over batches of the per-batch
    saliency of the unpruned layer (every k_e = I).

    batches: sequence of (x, logits, y_target).  Returns s [E][I] fp64.
    """
    E, I, _ = w_gate.shape
    keep = np.full(E, I, dtype=np.int32)
    total = np.zeros((E, I), dtype=np.float64)
    for x, logits, y_target in batches:
        _, gg, gu, gd = layer_grads(x, logits, w_gate, w_up, w_down, keep, top_k, norm_topk,
                                    y_target, ws_gate, ws_up, ws_down)
        total += channel_saliency_from_grads(w_gate, w_up, w_down, gg, gu, gd)
    return total / max(len(batches), 1)


def sample_actions(ratios, I, alpha, gumbel, tau):
    """Eq. 5: (keep [E] int32, action [E] int32, z_soft [E][K] fp64)."""
    alpha = np.ascontiguousarray(alpha, dtype=np.float32)
    gumbel = np.ascontiguousarray(gumbel, dtype=np.float32)
    E, K = alpha.shape
    r = np.ascontiguousarray(ratios, dtype=np.float64)
    keep = np.empty(E, np.int32)
    act = np.empty(E, np.int32)
    zs = np.empty((E, K), np.float64)
    rc = lib().oracle_sample_actions(E, K, _ptr(r), int(I), _ptr(alpha), _ptr(gumbel), float(tau),
                                     _ptr(keep), _ptr(zs), _ptr(act))
    if rc != 0:
        raise ValueError("oracle_sample_actions failed (%d)" % rc)
    return keep, act, zs


def masked_backward(x, logits, w_gate, w_up, w_down, keep, top_k, norm_topk, dy,
                    ws_gate=None, ws_up=None, ws_down=None):
    """Backward of the masked layer for the upstream gradient dy [T][d] fp32:
    (dx [T][d], dlogits [T][E], dmask [E][I]), fp64."""
    x = np.ascontiguousarray(x)
    dtype = _dtype_of(x)
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    T, d = x.shape
    E, I, _ = w_gate.shape
    I_s = 0 if ws_gate is None else ws_gate.shape[0]
    dy = np.ascontiguousarray(dy, dtype=np.float32)
    keep = np.ascontiguousarray(keep, dtype=np.int32)
    dx = np.empty((T, d), np.float64)
    dl = np.empty((T, E), np.float64)
    dm = np.empty((E, I), np.float64)
    rc = lib().oracle_masked_backward(
        T, d, E, I, top_k, I_s, dtype, int(norm_topk), _ptr(x), _ptr(logits),
        _ptr(np.ascontiguousarray(w_gate)), _ptr(np.ascontiguousarray(w_up)),
        _ptr(np.ascontiguousarray(w_down)), _ptr(keep),
        _ptr(None if ws_gate is None else np.ascontiguousarray(ws_gate)),
        _ptr(None if ws_up is None else np.ascontiguousarray(ws_up)),
        _ptr(None if ws_down is None else np.ascontiguousarray(ws_down)),
        _ptr(dy), _ptr(dx), _ptr(dl), _ptr(dm))
    if rc != 0:
        raise ValueError("oracle_masked_backward failed (%d)" % rc)
    return dx, dl, dm


def action_grad(ratios, I, alpha, gumbel, tau, dmask, counts, assignments, lambda_cost, beta):
    """Eqs. 5-8: (dalpha [E][K] fp64, cost C, entropy H)."""
    alpha = np.ascontiguousarray(alpha, dtype=np.float32)
    gumbel = np.ascontiguousarray(gumbel, dtype=np.float32)
    E, K = alpha.shape
    r = np.ascontiguousarray(ratios, dtype=np.float64)
    dm = np.ascontiguousarray(dmask, dtype=np.float64)
    cnt = np.ascontiguousarray(counts, dtype=np.int32)
    da = np.empty((E, K), np.float64)
    c = np.zeros(1, np.float64)
    h = np.zeros(1, np.float64)
    rc = lib().oracle_action_grad(E, K, _ptr(r), int(I), _ptr(alpha), _ptr(gumbel), float(tau), _ptr(dm),
                                  _ptr(cnt), int(assignments), float(lambda_cost), float(beta), _ptr(da),
                                  _ptr(c), _ptr(h))
    if rc != 0:
        raise ValueError("oracle_action_grad failed (%d)" % rc)
    return da, float(c[0]), float(h[0])


def packed_width(k: int) -> int:
    """Channels an expert occupies in the clipped layout: k rounded up to 8."""
    return (int(k) + 7) // 8 * 8


def export_clipped(keep, w_gate_r, w_up_r, w_down_r):
    """Offline clipping (Sec. 4.4, Table 2): the subnetwork of budget `keep`
    as standalone compact weights, by the definition of the clipped layout.

    Expert e keeps its first k_e ranked channels, padded with zeros to
    kp_e = ceil8(k_e): a gate/up block [kp_e][d] (rows = channels) and a down
    block [d][kp_e] (columns = channels), the experts' blocks in expert
    order.  Returns the three packed buffers as flat arrays of P*d elements
    (P = sum_e kp_e) -- a pure rearrangement of the ranked weights, no
    arithmetic.
    """
    keep = np.asarray(keep, dtype=np.int64)
    E, I, d = w_gate_r.shape
    g_blocks, u_blocks, d_blocks = [], [], []
    for e in range(E):
        k, kp = int(keep[e]), packed_width(keep[e])
        g = np.zeros((kp, d), dtype=w_gate_r.dtype)
        u = np.zeros((kp, d), dtype=w_up_r.dtype)
        dn = np.zeros((d, kp), dtype=w_down_r.dtype)
        g[:k] = w_gate_r[e, :k]
        u[:k] = w_up_r[e, :k]
        dn[:, :k] = w_down_r[e, :, :k]
        g_blocks.append(g.reshape(-1))
        u_blocks.append(u.reshape(-1))
        d_blocks.append(dn.reshape(-1))
    cat = lambda bl, dt: np.concatenate(bl) if bl else np.zeros(0, dtype=dt)
    return (cat(g_blocks, w_gate_r.dtype), cat(u_blocks, w_up_r.dtype), cat(d_blocks, w_down_r.dtype))


def keep_from_ratio(r: float, I: int) -> int:
    return int(lib().oracle_keep_from_ratio(float(r), int(I)))


def num_threads(variant: str = "fp64") -> int:
    return int(lib(variant).oracle_num_threads())
