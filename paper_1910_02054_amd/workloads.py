"""Seeded synthetic shard workloads.

This module only describes workloads and draws their random inputs.  It holds
none of the step's arithmetic: no layout, no statistics, no update.  Both the
GPU path's tests/benchmark and the CPU oracle consume the very bytes it
produces, so parity never depends on the generator.

Each workload is one data-parallel rank's shard of a model shaped like those
trained in ZeRO (arXiv 1910.02054), Sec. 10 and its appendix tables: GPT-2
1.5B, the 13B data-parallel-only point, the 100B model at 16-way model
parallelism x 25-way data parallelism, and a 1T model at MP 16 x N_d 1024.
The model-parallel slice Psi/N_m is what the ZeRO-DP layout partitions.

Inputs, all seeded from numpy PCG64 streams keyed by
(seed, workload id, tensor id, step, chunk), one stream per 2^22-element chunk
so that chunks can be drawn in parallel threads:

* master parameters ~ N(0, 0.02) in fp32 (the second argument of N is a
  standard deviation);
* momentum and variance: zero (cold start) or N(0, 1e-4) and |N(0, 1e-6)|
  (warm start);
* per step, fp16 gradients = binary16(N(0, sigma) * loss_scale), with the loss
  scale current at that step;
* for the overflow-stress workload, at chosen 1-based steps, a fraction of
  the gradient positions (drawn without replacement) is set to +inf or NaN
  with probability 1/2 each;
* the fp16 parameter output buffer starts as a sentinel pattern so that an
  untouched buffer is detectable.
"""
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Tuple

import numpy as np

F16_POS_INF = 0x7C00
F16_QNAN = 0x7E00
P16_SENTINEL = 0x5A5A  # binary16 pattern not produced by N(0, 0.02) parameters

_TENSOR_IDS = {"master": 1, "m": 2, "v": 3, "grad": 4, "inject": 5, "inject_kind": 6}


@dataclass(frozen=True)
class ShardWorkload:
    key: str
    wid: int               # workload id, part of every seed
    description: str
    psi: int               # elements partitioned by ZeRO-DP (the MP slice)
    nd: int                # data-parallel degree
    rank: int              # rank whose shard is run
    steps: int
    loss_scale: float      # starting loss scale
    grad_std: float
    warm_start: bool       # m, v drawn (True) or zero (False)
    lr: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.0
    clip: float = 1.0
    master_std: float = 0.02
    m_std: float = 1e-4
    v_std: float = 1e-6
    inject_steps: Tuple[int, ...] = field(default_factory=tuple)  # 1-based steps
    inject_frac: float = 0.0
    seed: int = 0

    def hyper(self):
        return dict(lr=self.lr, beta1=self.beta1, beta2=self.beta2, eps=self.eps,
                    weight_decay=self.weight_decay, clip=self.clip)


WORKLOADS = {
    w.key: w for w in (
        ShardWorkload("tiny", 0, "tiny shard: Psi=4,194,304 over N_d=4, rank 1",
                      psi=4_194_304, nd=4, rank=1, steps=3, loss_scale=2.0 ** 16, grad_std=1e-3,
                      warm_start=False),
        ShardWorkload("gpt2_1p5b", 1, "GPT-2 1.5B over N_d=16, rank 0",
                      psi=1_500_000_000, nd=16, rank=0, steps=10, loss_scale=2.0 ** 16, grad_std=1e-3,
                      warm_start=True),
        ShardWorkload("dp_13b", 2, "13B pure data parallel over N_d=64, rank 0",
                      psi=13_000_000_000, nd=64, rank=0, steps=10, loss_scale=2.0 ** 15, grad_std=1e-2,
                      warm_start=True),
        ShardWorkload("mp16_dp25_100b", 3, "100B at MP 16 x N_d 25: 6.25B slice, rank 0",
                      psi=6_250_000_000, nd=25, rank=0, steps=10, loss_scale=2.0 ** 16, grad_std=1e-3,
                      warm_start=True),
        ShardWorkload("ragged_1t", 4, "1T at MP 16 x N_d 1024: 62.5B slice, last rank (padded), "
                      "inf/NaN injected at steps 3 and 7",
                      psi=62_500_000_000, nd=1024, rank=1023, steps=12, loss_scale=2.0 ** 16, grad_std=1e-3,
                      warm_start=True, inject_steps=(3, 7), inject_frac=1e-5),
    )
}


CHUNK = 1 << 22
_POOL = None


def _pool():
    global _POOL
    if _POOL is None:
        try:
            k = len(os.sched_getaffinity(0))
        except AttributeError:
            k = 4
        _POOL = ThreadPoolExecutor(max_workers=max(1, min(16, k)))
    return _POOL


def _rng(w: ShardWorkload, tensor: str, step: int = 0, chunk: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [w.seed, w.wid, _TENSOR_IDS[tensor], step, chunk])))


def _normal(w: ShardWorkload, tensor: str, step: int, n: int, std: float, absolute: bool = False,
            out_dtype=np.float32) -> np.ndarray:
    """n draws of N(0, std) (|N(0, std)| if absolute) in fp32, cast to out_dtype."""
    out = np.empty(n, out_dtype)

    def fill(c):
        a, b = c * CHUNK, min(n, (c + 1) * CHUNK)
        z = _rng(w, tensor, step, c).standard_normal(b - a, dtype=np.float32)
        if absolute:
            np.abs(z, out=z)
        z *= np.float32(std)
        out[a:b] = z  # fp32 -> out_dtype, round to nearest even
    list(_pool().map(fill, range((n + CHUNK - 1) // CHUNK)))
    return out


def initial_state(w: ShardWorkload, n: int):
    """(master fp32, m fp32, v fp32) for an n-element shard."""
    master = _normal(w, "master", 0, n, w.master_std)
    if w.warm_start:
        m = _normal(w, "m", 0, n, w.m_std)
        v = _normal(w, "v", 0, n, w.v_std, absolute=True)
    else:
        m = np.zeros(n, np.float32)
        v = np.zeros(n, np.float32)
    return master, m, v


def gradients(w: ShardWorkload, n: int, step: int, loss_scale: float) -> np.ndarray:
    """Loss-scaled fp16 gradients for 1-based `step`, as uint16 bit patterns."""
    g16 = _normal(w, "grad", step, n, w.grad_std * loss_scale, out_dtype=np.float16).view(np.uint16)
    if step in w.inject_steps and n > 0:
        k = max(1, int(round(w.inject_frac * n)))
        pos = _rng(w, "inject", step).choice(n, size=min(k, n), replace=False)
        kind = _rng(w, "inject_kind", step).integers(0, 2, size=pos.size)
        g16[pos] = np.where(kind == 0, F16_POS_INF, F16_QNAN).astype(np.uint16)
    return g16


def injected_positions(w: ShardWorkload, n: int, step: int) -> np.ndarray:
    """Positions that `gradients` overwrites with inf/NaN at `step` (empty if none)."""
    if step not in w.inject_steps or n <= 0:
        return np.empty(0, np.int64)
    k = max(1, int(round(w.inject_frac * n)))
    return np.sort(_rng(w, "inject", step).choice(n, size=min(k, n), replace=False))


def p16_sentinel(n: int) -> np.ndarray:
    return np.full(n, P16_SENTINEL, np.uint16)


def random_case(seed: int, n: int, grad_std: float = 1e-3, loss_scale: float = 2.0 ** 16,
                warm: bool = True):
    """A free-form seeded case (g16, master, m, v) for edge-case tests."""
    r = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 99, n])))
    master = (r.standard_normal(n, dtype=np.float32) * np.float32(0.02)).astype(np.float32)
    if warm:
        m = (r.standard_normal(n, dtype=np.float32) * np.float32(1e-4)).astype(np.float32)
        v = (np.abs(r.standard_normal(n, dtype=np.float32)) * np.float32(1e-6)).astype(np.float32)
    else:
        m = np.zeros(n, np.float32)
        v = np.zeros(n, np.float32)
    z = r.standard_normal(n, dtype=np.float32) * np.float32(grad_std * loss_scale)
    with np.errstate(over="ignore"):  # a scale too large for fp16 gives inf, as in training
        g16 = z.astype(np.float16).view(np.uint16).copy()
    return g16, master, m, v


# ---------------------------------------------------------------------------
# Layer structure (for the per-layer trust ratio of LAMB)
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class ModelShape:
    """A GPT-2-like transformer as in ZeRO's evaluation (Sec. 10 and its
    appendix tables), sliced for mp-way model parallelism the Megatron way:
    the QKV and first MLP projections split by columns (weights and biases),
    the attention output and second MLP projections by rows (weights split,
    biases replicated), layer norms replicated, the token embedding split by
    vocabulary rows."""
    hidden: int
    mp: int = 1
    vocab: int = 50257
    positions: int = 1024


MODEL_SHAPES = {
    "tiny": ModelShape(hidden=128, vocab=2048, positions=256),
    "gpt2_1p5b": ModelShape(hidden=1600),             # 48 layers, HD 1600, MP 1
    "dp_13b": ModelShape(hidden=4096),                # the 10B-13B points: HD 4096, MP 1
    "mp16_dp25_100b": ModelShape(hidden=8192, mp=16),  # 125 layers, HD 8192, MP 16
    "ragged_1t": ModelShape(hidden=25600, mp=16),     # no shape in the paper: HD 25600 gives ~1T
}


def _layer_tensors(s: ModelShape):
    h, mp = s.hidden, s.mp
    return [h, h,                         # attention layer norm
            h * (3 * h // mp), 3 * h // mp,  # QKV (column-parallel)
            (h // mp) * h, h,             # attention output (row-parallel; bias replicated)
            h, h,                         # MLP layer norm
            h * (4 * h // mp), 4 * h // mp,  # MLP up (column-parallel)
            (4 * h // mp) * h, h]         # MLP down (row-parallel; bias replicated)


def model_tensor_sizes(shape: ModelShape, psi: int):
    """Sizes of the model slice's tensors in flat order (token and position
    embeddings, then transformer layers as many as needed), the last one cut
    so that the sizes add up to exactly psi."""
    sizes = []
    total = 0
    emb = [-(-shape.vocab // shape.mp) * shape.hidden, shape.positions * shape.hidden]
    layer = _layer_tensors(shape)
    k = 0
    while total < psi:
        t = emb[k] if k < len(emb) else layer[(k - len(emb)) % len(layer)]
        t = min(t, psi - total)
        sizes.append(t)
        total += t
        k += 1
    return sizes


def layer_offsets_in(sizes, start: int, stop: int) -> np.ndarray:
    """The layer table of the flat range [start, stop): offsets relative to
    start of the pieces of every tensor that meets the range (n_seg + 1
    entries, from 0 to stop - start).  Bookkeeping only."""
    bounds = np.concatenate([[0], np.cumsum(np.asarray(sizes, dtype=np.int64))])
    inner = bounds[(bounds > start) & (bounds < stop)]
    return np.concatenate([[start], inner, [stop]]).astype(np.int64) - start


def layer_ids_in(sizes, start: int, stop: int) -> np.ndarray:
    """Global tensor index of each layer of layer_offsets_in(sizes, start, stop)."""
    bounds = np.concatenate([[0], np.cumsum(np.asarray(sizes, dtype=np.int64))])
    first = int(np.searchsorted(bounds, start, side="right")) - 1
    n_seg = layer_offsets_in(sizes, start, stop).size - 1
    return np.arange(first, first + n_seg, dtype=np.int64)
