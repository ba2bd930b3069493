"""Seeded synthetic inputs for the masked MoE layer.

This module only draws random numbers and builds keep-count tables.  It holds
none of the layer's arithmetic (no routing weights, no FFN, no combine), so
both the GPU path and the CPU checker can take their inputs from it.

Every tensor is drawn from NumPy's PCG64 with seed = 1000*config_id +
tensor_id.  bf16 tensors are produced by round-to-nearest-even from the fp32
draw, so the exact same bytes reach every consumer.

Shapes follow the models the paper evaluates (Sec. 4.1 and Table A1): a
Mixtral-8x7B-shaped layer (8 experts, top-2), a Qwen2-57B-A14B-shaped layer
(64 routed experts, top-8, plus a shared expert) and a Qwen1.5-MoE-A2.7B-shaped
layer.  Keep counts are integers k_e in [0, I]; the paper's retention ratio r
maps to k = ceil(r*I) (Sec. 3.1, text after Eq. 3).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

F32 = 0
BF16 = 1

# tensor ids inside one config's seed space
_TID_X = 1
_TID_LOGITS = 2
_TID_BIAS = 3
_TID_WGATE = 4
_TID_WUP = 5
_TID_WDOWN = 6
_TID_SGATE = 7
_TID_SUP = 8
_TID_SDOWN = 9
_TID_SCORES = 10
_TID_KEEP = 11
_TID_NESTED = 12
_TID_CALIB = 13
_TID_ZIPF_PERM = 14
_TID_POOL = 100  # decode batches use 100 + batch index

_CHUNK = 1 << 24  # elements per generation chunk (fixed: part of the recipe)


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    config_id: int
    T: int
    d: int
    E: int
    I: int
    top_k: int
    I_shared: int
    dtype: int
    norm_topk: int
    bias_std: float = 0.0      # per-expert router bias std (0 = none)
    zipf_s: float = 0.0        # >0: calibrate biases for Zipf(s) expert load
    x_std: float = 1.0
    w_std: float = 0.02
    logit_std: float = 1.0

    @property
    def max_tokens(self) -> int:
        return self.T


# The five workloads.  T of the decode config is its largest batch (64).
CONFIGS: Dict[str, LayerConfig] = {
    "tiny_fp32": LayerConfig("tiny_fp32", 1, T=64, d=256, E=8, I=512, top_k=2,
                             I_shared=0, dtype=F32, norm_topk=1),
    "qwen15_moe_a27b": LayerConfig("qwen15_moe_a27b", 2, T=4096, d=2048, E=60, I=1408,
                                   top_k=4, I_shared=5632, dtype=BF16, norm_topk=0,
                                   bias_std=0.5),
    "qwen2_57b_a14b_prefill": LayerConfig("qwen2_57b_a14b_prefill", 3, T=8192, d=3584,
                                          E=64, I=2560, top_k=8, I_shared=20480,
                                          dtype=BF16, norm_topk=0, bias_std=0.5),
    "qwen2_57b_a14b_decode": LayerConfig("qwen2_57b_a14b_decode", 4, T=64, d=3584, E=64,
                                         I=2560, top_k=8, I_shared=20480, dtype=BF16,
                                         norm_topk=0, bias_std=0.5),
    "mixtral_8x7b": LayerConfig("mixtral_8x7b", 5, T=16384, d=4096, E=8, I=14336,
                                top_k=2, I_shared=0, dtype=BF16, norm_topk=1,
                                zipf_s=1.2),
}

NESTED_FRACTIONS = (1.0, 0.8, 0.6, 0.4, 0.2)


def rng_for(config_id: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(1000 * config_id + tensor_id))


# ----------------------------------------------------------------------------
# bf16 bit conversions (round to nearest even; NaN -> canonical quiet NaN)
# ----------------------------------------------------------------------------
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, dtype=np.uint16)
    flat_in = a.reshape(-1)
    flat_out = out.reshape(-1)
    for s in range(0, flat_in.size, _CHUNK):
        u = flat_in[s:s + _CHUNK].view(np.uint32)
        r = ((u >> 16) & 1) + np.uint32(0x7FFF)
        b = ((u + r) >> 16).astype(np.uint16)
        nan = np.isnan(flat_in[s:s + _CHUNK])
        if nan.any():
            b[nan] = 0x7FC0
        flat_out[s:s + _CHUNK] = b
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def _normal(config_id: int, tensor_id: int, n: int, std: float) -> np.ndarray:
    g = rng_for(config_id, tensor_id)
    out = np.empty(n, dtype=np.float32)
    for s in range(0, n, _CHUNK):
        m = min(_CHUNK, n - s)
        out[s:s + m] = g.standard_normal(m, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def _as_dtype(a: np.ndarray, dtype: int) -> np.ndarray:
    return a if dtype == F32 else f32_to_bf16_bits(a)


# ----------------------------------------------------------------------------
# router logits
# ----------------------------------------------------------------------------
def zipf_shares(E: int, s: float) -> np.ndarray:
    r = np.arange(1, E + 1, dtype=np.float64)
    p = r ** (-s)
    return p / p.sum()


def _top_k_membership_counts(logits: np.ndarray, k: int) -> np.ndarray:
    """How often each expert lands among a token's k largest logits.

    Used only to calibrate the synthetic router biases of the skewed-load
    workload; it is not part of the layer computation.
    """
    part = np.argpartition(-logits, k - 1, axis=1)[:, :k]
    return np.bincount(part.reshape(-1), minlength=logits.shape[1]).astype(np.float64)


def calibrate_zipf_bias(cfg: LayerConfig, n_calib: int = 65536, iters: int = 200) -> np.ndarray:
    """Per-expert logit bias giving a Zipf(s) share of routed assignments.

    Deterministic fixed-point iteration on a seeded calibration sample of
    N(0,1) logits: b <- b + 0.5*(log target - log realized).  The rank -> expert
    id map is a seeded permutation.
    """
    target_rank = zipf_shares(cfg.E, cfg.zipf_s)
    perm = rng_for(cfg.config_id, _TID_ZIPF_PERM).permutation(cfg.E)
    target = np.empty(cfg.E)
    target[perm] = target_rank
    calib = _normal(cfg.config_id, _TID_CALIB, n_calib * cfg.E, cfg.logit_std).reshape(n_calib, cfg.E)
    calib = calib.astype(np.float64)
    b = np.log(target) - np.log(target).mean()
    for _ in range(iters):
        share = _top_k_membership_counts(calib + b, cfg.top_k)
        share = np.maximum(share, 1.0) / (n_calib * cfg.top_k)
        step = 0.5 * (np.log(target) - np.log(share))
        b = b + step
        b -= b.mean()
        if np.max(np.abs(share - target)) < 2e-3:
            break
    return b.astype(np.float32)


def router_bias(cfg: LayerConfig) -> np.ndarray:
    if cfg.zipf_s > 0:
        return calibrate_zipf_bias(cfg)
    if cfg.bias_std > 0:
        return _normal(cfg.config_id, _TID_BIAS, cfg.E, cfg.bias_std)
    return np.zeros(cfg.E, dtype=np.float32)


def make_tokens(cfg: LayerConfig, T: Optional[int] = None, batch: int = -1,
                bias: Optional[np.ndarray] = None):
    """x [T][d] (fp32 or bf16 bits) and logits [T][E] fp32.

    batch < 0: the config's main batch; batch >= 0: one of the decode pool's
    independent batches.
    """
    T = cfg.T if T is None else T
    if bias is None:
        bias = router_bias(cfg)
    if batch < 0:
        x = _normal(cfg.config_id, _TID_X, T * cfg.d, cfg.x_std).reshape(T, cfg.d)
        lg = _normal(cfg.config_id, _TID_LOGITS, T * cfg.E, cfg.logit_std).reshape(T, cfg.E)
    else:
        g = rng_for(cfg.config_id, _TID_POOL + batch)
        x = g.standard_normal(T * cfg.d, dtype=np.float32).reshape(T, cfg.d) * np.float32(cfg.x_std)
        lg = g.standard_normal(T * cfg.E, dtype=np.float32).reshape(T, cfg.E) * np.float32(cfg.logit_std)
    lg = (lg + bias[None, :]).astype(np.float32)
    return _as_dtype(x, cfg.dtype), np.ascontiguousarray(lg)


_TID_TARGET = 16
_TID_CALIB_BATCH = 200  # calibration batch b of the saliency uses 200 + 2b and 201 + 2b


def make_target(cfg: LayerConfig, T: Optional[int] = None, std: float = 0.05, batch: int = -1):
    """Target [T][d] fp32 of the layer-level loss L = 1/2 sum_t ||Y_t - target_t||^2
    the channel saliency is measured with: seeded Gaussian noise of the given std.
    batch >= 0: the target of calibration batch `batch`."""
    T = cfg.T if T is None else T
    tid = _TID_TARGET if batch < 0 else _TID_CALIB_BATCH + 2 * batch + 1
    return _normal(cfg.config_id, tid, T * cfg.d, std).reshape(T, cfg.d)


_TID_ALPHA = 17
_TID_GUMBEL = 18


def make_action_inputs(cfg: LayerConfig, K: int, step: int = 0, alpha_std: float = 1.0):
    """Action logits alpha [E][K] (Gaussian) and the Gumbel(0, 1) draws of one
    sampling step [E][K] (-log(-log U), U uniform in (0, 1)), both fp32."""
    alpha = _normal(cfg.config_id, _TID_ALPHA, cfg.E * K, alpha_std).reshape(cfg.E, K)
    g = rng_for(cfg.config_id, _TID_GUMBEL + 1000 * step)
    u = g.random(cfg.E * K, dtype=np.float64)
    u = np.clip(u, 1e-12, 1.0 - 1e-12)
    gumbel = (-np.log(-np.log(u))).astype(np.float32).reshape(cfg.E, K)
    return alpha, gumbel


def make_calibration_batch(cfg: LayerConfig, batch: int, T: Optional[int] = None,
                           bias: Optional[np.ndarray] = None):
    """Tokens x [T][d] and logits [T][E] of calibration batch `batch` (same
    distributions as make_tokens, independent draws)."""
    T = cfg.T if T is None else T
    if bias is None:
        bias = router_bias(cfg)
    g = rng_for(cfg.config_id, _TID_CALIB_BATCH + 2 * batch)
    x = g.standard_normal(T * cfg.d, dtype=np.float32).reshape(T, cfg.d) * np.float32(cfg.x_std)
    lg = g.standard_normal(T * cfg.E, dtype=np.float32).reshape(T, cfg.E) * np.float32(cfg.logit_std)
    lg = (lg + bias[None, :]).astype(np.float32)
    return _as_dtype(x, cfg.dtype), np.ascontiguousarray(lg)


def _draw_all(specs):
    """Draw several tensors at once, one thread each.

    Each tensor has its own generator (its own seed), and NumPy's generators
    and array arithmetic release the interpreter lock while they fill large
    arrays, so the bytes are exactly those of drawing the tensors one after
    another; only the wall time shrinks.  specs: (tensor_id, n, shape, dtype,
    std) per tensor.
    """
    from concurrent.futures import ThreadPoolExecutor

    def one(spec):
        tid, n, shape, dtype, std, cid = spec
        return _as_dtype(_normal(cid, tid, n, std).reshape(shape), dtype)

    if len(specs) == 1:
        return [one(specs[0])]
    with ThreadPoolExecutor(len(specs)) as ex:
        return list(ex.map(one, specs))


def _expert_specs(cfg: LayerConfig):
    E, I, d = cfg.E, cfg.I, cfg.d
    return [(_TID_WGATE, E * I * d, (E, I, d), cfg.dtype, cfg.w_std, cfg.config_id),
            (_TID_WUP, E * I * d, (E, I, d), cfg.dtype, cfg.w_std, cfg.config_id),
            (_TID_WDOWN, E * d * I, (E, d, I), cfg.dtype, cfg.w_std, cfg.config_id)]


def _shared_specs(cfg: LayerConfig):
    Is, d = cfg.I_shared, cfg.d
    return [(_TID_SGATE, Is * d, (Is, d), cfg.dtype, cfg.w_std, cfg.config_id),
            (_TID_SUP, Is * d, (Is, d), cfg.dtype, cfg.w_std, cfg.config_id),
            (_TID_SDOWN, d * Is, (d, Is), cfg.dtype, cfg.w_std, cfg.config_id)]


def make_expert_weights(cfg: LayerConfig):
    """w_gate, w_up [E][I][d]; w_down [E][d][I] (output rows, channel columns).

    Random weights are exchangeable across channels, so they serve directly as
    an importance-ranked layer for the forward benchmarks.
    """
    return tuple(_draw_all(_expert_specs(cfg)))


def make_shared_weights(cfg: LayerConfig):
    """ws_gate, ws_up [I_s][d]; ws_down [d][I_s]; None if the layer has none."""
    if cfg.I_shared == 0:
        return None, None, None
    return tuple(_draw_all(_shared_specs(cfg)))


def make_layer_weights(cfg: LayerConfig):
    """(w_gate, w_up, w_down), (ws_gate, ws_up, ws_down): the same tensors as
    make_expert_weights and make_shared_weights, all six drawn at once."""
    specs = _expert_specs(cfg) + (_shared_specs(cfg) if cfg.I_shared else [])
    out = _draw_all(specs)
    shared = tuple(out[3:]) if cfg.I_shared else (None, None, None)
    return tuple(out[:3]), shared


def make_scores(cfg: LayerConfig, tie_every: int = 0) -> np.ndarray:
    """Synthetic channel saliency scores [E][I] fp32 (non-negative).

    Eq. 2 scores are sums of squares, hence >= 0.  tie_every > 0 quantises the
    scores coarsely so that ties occur.
    """
    s = np.abs(_normal(cfg.config_id, _TID_SCORES, cfg.E * cfg.I, 1.0)).reshape(cfg.E, cfg.I)
    if tie_every > 0:
        s = np.round(s * tie_every) / tie_every
    return s.astype(np.float32)


# ----------------------------------------------------------------------------
# keep-count tables
# ----------------------------------------------------------------------------
def nested_keep_family(E: int, I: int, seed: int, grid: int = 64,
                       fractions=NESTED_FRACTIONS) -> List[np.ndarray]:
    """Nested keep tables: k^1 >= k^2 >= ... elementwise.

    Start with every k_e = I; to reach kept fraction f, repeatedly remove one
    grid step from a seeded-uniform expert with k_e > 0 until
    sum(k) = round(f*E*I/grid)*grid.  Monotone by construction.
    """
    assert I % grid == 0
    g = np.random.Generator(np.random.PCG64(seed))
    k = np.full(E, I, dtype=np.int64)
    total_units = E * I // grid
    out = []
    for f in fractions:
        target = int(round(f * total_units)) * grid
        while k.sum() > target:
            live = np.nonzero(k > 0)[0]
            e = live[g.integers(0, live.size)]
            k[e] -= grid
        out.append(k.astype(np.int32).copy())
    return out


def grid_keep_table(E: int, I: int, seed: int, kept_fraction: float, grid: int = 64) -> np.ndarray:
    """Keep table on a grid with one expert at 0, one at I, sum exactly f*E*I."""
    assert I % grid == 0
    g = np.random.Generator(np.random.PCG64(seed))
    units = I // grid
    k = g.integers(0, units + 1, size=E).astype(np.int64)
    lo, hi = g.choice(E, size=2, replace=False)
    k[lo] = 0
    k[hi] = units
    target = int(round(kept_fraction * E * units))
    free = np.array([e for e in range(E) if e not in (lo, hi)])
    while k.sum() != target:
        e = free[g.integers(0, free.size)]
        if k.sum() < target and k[e] < units:
            k[e] += 1
        elif k.sum() > target and k[e] > 0:
            k[e] -= 1
    return (k * grid).astype(np.int32)


def quarter_keep_table(E: int, I: int, seed: int, mean_quarters: int = 2) -> np.ndarray:
    """k_e in {25,50,75,100}% of I (I % 4 == 0) with mean exactly 50%."""
    assert I % 4 == 0
    g = np.random.Generator(np.random.PCG64(seed))
    q = g.integers(1, 5, size=E).astype(np.int64)
    target = mean_quarters * E
    while q.sum() != target:
        e = g.integers(0, E)
        if q.sum() < target and q[e] < 4:
            q[e] += 1
        elif q.sum() > target and q[e] > 1:
            q[e] -= 1
    return (q * (I // 4)).astype(np.int32)


# The paper's discrete action set of retention ratios (Sec. 4.1).
ACTION_RATIOS = (0.1, 0.4, 0.7, 1.0)
_TID_ACTION = 15


def action_keep_table(E: int, levels, seed: int, kept_fraction: float) -> np.ndarray:
    """Keep table whose widths come from a discrete action set.

    `levels` are the channel counts of the actions, ascending (the caller
    maps the ratios to widths).  Every expert starts at the widest action;
    seeded-uniform experts above the narrowest action step down one action
    at a time until the kept fraction sum(k) / (E * max(levels)) is at most
    `kept_fraction` (or every expert is at the narrowest action).
    """
    levels = [int(v) for v in levels]
    g = np.random.Generator(np.random.PCG64(seed))
    a = np.full(E, len(levels) - 1, dtype=np.int64)
    full = E * levels[-1]

    def kept():
        return sum(levels[i] for i in a) / full

    while kept() > kept_fraction and (a > 0).any():
        live = np.nonzero(a > 0)[0]
        a[live[g.integers(0, live.size)]] -= 1
    return np.array([levels[i] for i in a], dtype=np.int32)


def tiny_keep_table(E: int, I: int, seed: int) -> np.ndarray:
    """Arbitrary integers in [0, I] that include 0, I and non-tile multiples."""
    g = np.random.Generator(np.random.PCG64(seed))
    k = g.integers(0, I + 1, size=E).astype(np.int32)
    forced = [0, I, 1, 17, 100, I - 1, 63, 65]
    order = g.permutation(E)
    for i, v in zip(order, forced):
        k[i] = min(max(v, 0), I)
    return k


def config_keep_tables(cfg: LayerConfig) -> Dict[str, np.ndarray]:
    """Named keep tables for a config: the nested family plus its own table."""
    seed = 1000 * cfg.config_id + _TID_NESTED
    fam = nested_keep_family(cfg.E, cfg.I, seed) if cfg.I % 64 == 0 else []
    tables = {f"kept{int(round(f * 100))}": t for f, t in zip(NESTED_FRACTIONS, fam)}
    own_seed = 1000 * cfg.config_id + _TID_KEEP
    if cfg.name == "tiny_fp32":
        tables["own"] = tiny_keep_table(cfg.E, cfg.I, own_seed)
    elif cfg.name == "qwen15_moe_a27b":
        tables["own"] = grid_keep_table(cfg.E, cfg.I, own_seed, 0.5)
    elif cfg.name == "mixtral_8x7b":
        tables["own"] = quarter_keep_table(cfg.E, cfg.I, own_seed)
    return tables


def keep_fraction(keep: np.ndarray, I: int) -> float:
    return float(np.asarray(keep, dtype=np.int64).sum()) / (len(keep) * I)


def small_config(name: str, T: int, d: int, E: int, I: int, top_k: int, I_shared: int = 0,
                 dtype: int = BF16, norm_topk: int = 1, config_id: int = 50,
                 bias_std: float = 0.0) -> LayerConfig:
    """A reduced layer used by parity tests (several tiles plus ragged tails)."""
    return LayerConfig(name, config_id, T=T, d=d, E=E, I=I, top_k=top_k, I_shared=I_shared,
                       dtype=dtype, norm_topk=norm_topk, bias_std=bias_std)


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)

