"""Independent dense brute force of the masked MoE layer (NumPy, fp64).

Used only to pin the oracle.  It is written in a different form from the
oracle on purpose: it evaluates EVERY expert on EVERY token with full
matrices, applies the prefix mask m(r) of Eq. 4 by multiplication, and mixes
the experts through a dense [T][E] gate matrix that is zero off the top-k.
Routing uses a full lexicographic sort and SciPy's softmax.
"""
import numpy as np
from scipy.special import softmax

from paper_2606_27866_amd.synth import bf16_bits_to_f32


def f64(a):
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return bf16_bits_to_f32(a).astype(np.float64)
    return a.astype(np.float64)


def topk_by_sort(logits, k):
    """Expert ids ordered by (logit desc, id asc) via a full lexsort; NaN last."""
    logits = np.asarray(logits, dtype=np.float32)
    T, E = logits.shape
    ids = np.broadcast_to(np.arange(E), (T, E))
    nan = np.isnan(logits)
    key = np.where(nan, 0.0, -logits.astype(np.float64))
    order = np.lexsort((ids, key, nan), axis=-1)
    return order[:, :k].astype(np.int32)


def router_weights(logits, idx, norm_topk):
    p = softmax(np.asarray(logits, dtype=np.float64), axis=1)
    w = np.take_along_axis(p, idx.astype(np.int64), axis=1)
    if norm_topk:
        w = w / w.sum(axis=1, keepdims=True)
    return w


def silu(v):
    return v / (1.0 + np.exp(-v))


def dense_layer(x, logits, w_gate, w_up, w_down, keep, top_k, norm_topk,
                ws_gate=None, ws_up=None, ws_down=None):
    X = f64(x)
    T, d = X.shape
    Wg, Wu, Wd = f64(w_gate), f64(w_up), f64(w_down)
    E, I, _ = Wg.shape
    idx = topk_by_sort(logits, top_k)
    w = router_weights(logits, idx, norm_topk)
    G = np.zeros((T, E))
    rows = np.repeat(np.arange(T), top_k)
    G[rows, idx.reshape(-1)] = w.reshape(-1)
    Y = np.zeros((T, d))
    chan = np.arange(I)
    for e in range(E):
        m = (chan < keep[e]).astype(np.float64)
        H = silu(X @ Wg[e].T) * (X @ Wu[e].T) * m[None, :]
        Y += G[:, e:e + 1] * (H @ Wd[e].T)
    if ws_gate is not None:
        Sg, Su, Sd = f64(ws_gate), f64(ws_up), f64(ws_down)
        Y += (silu(X @ Sg.T) * (X @ Su.T)) @ Sd.T
    return Y


def random_layer(rng, T, d, E, I, k, I_s=0, bf16=False):
    """Small random layer (fp32 or bf16 bits) for brute-force comparisons."""
    from paper_2606_27866_amd.synth import f32_to_bf16_bits

    def mk(*shape, std=1.0):
        a = (rng.standard_normal(shape) * std).astype(np.float32)
        return f32_to_bf16_bits(a) if bf16 else a

    x = mk(T, d)
    logits = rng.standard_normal((T, E)).astype(np.float32)
    wg, wu = mk(E, I, d, std=0.3), mk(E, I, d, std=0.3)
    wd = mk(E, d, I, std=0.3)
    shared = (None, None, None)
    if I_s:
        shared = (mk(I_s, d, std=0.3), mk(I_s, d, std=0.3), mk(d, I_s, std=0.3))
    return x, logits, wg, wu, wd, shared
