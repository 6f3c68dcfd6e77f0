"""Seeded synthetic inputs for the SDM sparse recurrence.

This module only draws random numbers and shapes them into the input
distributions of the five workloads; it contains none of the layer's own
arithmetic (no scoring, no selection, no recurrence).  Both the CPU oracle
(``oracle/``) and the HIP path consume what it produces, bit for bit.

Recipe (every stream is generated independently, so any (b, h) stream can be
regenerated alone for sampled checks):

* one ``numpy.random.Generator(PCG64)`` per (workload seed, tensor id, b, h),
  built from ``SeedSequence(seed, spawn_key=(tensor_id, b, h))``;
  per-head tensors (codebooks, cluster centres, shared initial memory) use
  ``b = 0``.
* q, k: i.i.d. N(0, 1) in fp64, L2-normalised per token over d_k.
* clustered keys (long-context workload): 4096 unit-norm centres per head,
  a centre drawn uniformly per token, key = normalise(centre + 0.1 * N(0, I)).
* v: N(0, 1).
* beta = sigmoid(z), alpha = exp(-softplus(z)) with z ~ N(0, 1), so both gates
  have median 0.5 (the gate shapes of the paper's Sec. 3.1, step 2).
* sub-key codebooks [H, 2, sqrt(N), d_k/2]: N(0, 1) rows, L2-normalised.
* learned initial memory [H, N, d_v]: N(0, 0.02^2), shared across the batch.
* upstream output gradient dy: N(0, 1), fp32.
* inputs of the steps either side of the recurrence (``LayerInputs``): gate
  pre-activations a, b ~ N(0, 1) [B, H, T]; output gate g ~ N(0, 1)
  [B, H, T, d_v]; per head A ~ U(0, 16) and b_dt = inverse softplus of
  U(0.001, 0.1) (the paper's Sec. 4 initialisation); norm scale
  gamma ~ U(0.5, 1.5) [d_v]; upstream gradient of the epilogue's output
  N(0, 1), fp32.
* low-precision workloads round fp64 -> fp32 -> bf16 (round to nearest even);
  fp32 workloads round fp64 -> fp32.  Both sides read the same bits.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace
from typing import Iterable, Sequence

import numpy as np

# tensor ids used in the seed spawn key
_Q, _K, _V, _BETA, _ALPHA, _CB, _M0, _CENTRES, _ASSIGN, _DY, _DMT, _MNOISE = range(12)
_APRE, _BPRE, _GATE_OUT, _GATE_PARAM, _GAMMA, _DOUT = range(12, 18)


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    T: int
    d_k: int
    d_v: int
    N: int
    topk: int
    dtype: str = "bf16"          # input dtype of q/k/v/gates/codebooks: "f32" | "bf16"
    seed: int = 0
    clustered_keys: bool = False
    n_clusters: int = 4096
    cluster_sigma: float = 0.1
    m0: str = "zero"             # "zero" | "shared" (N(0, m0_std^2) per head, shared over b)
    m0_std: float = 0.02
    train: bool = False
    chunk: int = 64
    codebook: bool = True        # False: direct mode, d_k == 2*sqrt(N)
    extra: dict = field(default_factory=dict)

    @property
    def sqrtN(self) -> int:
        s = math.isqrt(self.N)
        assert s * s == self.N
        return s

    @property
    def W(self) -> int:
        return self.topk

    @property
    def R(self) -> int:
        return self.topk

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five workloads, by the shapes and distributions they are specified with.
WORKLOADS = {
    0: Workload("tiny-f32", B=1, H=2, T=256, d_k=32, d_v=32, N=1024, topk=8, dtype="f32", seed=0),
    1: Workload("sdm-1.4b-fwd", B=8, H=16, T=4096, d_k=128, d_v=128, N=65536, topk=32, seed=1),
    2: Workload("long-context-fwd", B=1, H=16, T=65536, d_k=128, d_v=128, N=262144, topk=32,
                seed=2, clustered_keys=True),
    3: Workload("big-learned-m0-fwd", B=4, H=8, T=8192, d_k=128, d_v=128, N=1048576, topk=32,
                seed=3, m0="shared"),
    4: Workload("train-fwd-bwd", B=4, H=16, T=4096, d_k=128, d_v=128, N=65536, topk=32,
                seed=4, train=True, chunk=64),
}


def _rng(w: Workload, tensor: int, b: int, h: int) -> np.random.Generator:
    ss = np.random.SeedSequence(w.seed, spawn_key=(tensor, b, h))
    return np.random.Generator(np.random.PCG64(ss))


# ---------------------------------------------------------------- rounding
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = np.right_shift(u, np.uint32(16))
    np.bitwise_and(r, np.uint32(1), out=r)
    np.add(r, np.uint32(0x7FFF), out=r)
    np.add(r, u, out=r)
    np.right_shift(r, np.uint32(16), out=r)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


class Stored:
    """An input tensor in its storage dtype plus its exact value.

    ``f32`` holds the exact value of every element (bf16 values widen to fp32
    exactly); ``bits`` holds the bf16 bit patterns for bf16 storage."""

    def __init__(self, shape, dtype: str):
        if dtype not in ("f32", "bf16"):
            raise ValueError(dtype)
        self.dtype = dtype
        self.f32 = np.empty(shape, np.float32)
        self.bits = np.empty(shape, np.uint16) if dtype == "bf16" else None

    @classmethod
    def from_f64(cls, arr64: np.ndarray, dtype: str) -> "Stored":
        st = cls(arr64.shape, dtype)
        st.put(slice(None), arr64)
        return st

    def put(self, index, arr64: np.ndarray):
        """Round fp64 values to the storage dtype and store them at ``index``."""
        f32 = np.asarray(arr64, dtype=np.float32)
        if self.dtype == "bf16":
            bits = f32_to_bf16_bits(f32).reshape(f32.shape)
            self.bits[index] = bits
            self.f32[index] = bf16_bits_to_f32(bits).reshape(f32.shape)
        else:
            self.f32[index] = f32

    @property
    def f64(self) -> np.ndarray:
        return self.f32.astype(np.float64)

    @property
    def storage(self) -> np.ndarray:
        """Array in storage layout: uint16 for bf16, float32 for f32."""
        return self.bits if self.dtype == "bf16" else self.f32


# ---------------------------------------------------------------- draws
def _normalise(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _softplus(z):
    return np.logaddexp(0.0, z)


def codebook_head(w: Workload, h: int) -> np.ndarray:
    """fp64 sub-key codebook of one head, [2, sqrt(N), d_k/2], rows unit-norm."""
    cb = _rng(w, _CB, 0, h).standard_normal((2, w.sqrtN, w.d_k // 2))
    return _normalise(cb)


def centres_head(w: Workload, h: int) -> np.ndarray:
    return _normalise(_rng(w, _CENTRES, 0, h).standard_normal((w.n_clusters, w.d_k)))


def m0_head(w: Workload, h: int) -> np.ndarray:
    """Shared initial memory of one head, fp32 [N, d_v]."""
    g = _rng(w, _M0, 0, h)
    return (g.standard_normal((w.N, w.d_v), dtype=np.float32) * np.float32(w.m0_std))


def stream_inputs(w: Workload, b: int, h: int, centres: np.ndarray | None = None) -> dict:
    """fp64 draws for one (b, h) stream: q, k [T,d_k], v [T,d_v], alpha, beta [T]."""
    T = w.T
    q = _normalise(_rng(w, _Q, b, h).standard_normal((T, w.d_k)))
    if w.clustered_keys:
        cen = centres if centres is not None else centres_head(w, h)
        ga = _rng(w, _ASSIGN, b, h)
        assign = ga.integers(0, w.n_clusters, size=T)
        k = _normalise(cen[assign] + w.cluster_sigma * _rng(w, _K, b, h).standard_normal((T, w.d_k)))
    else:
        k = _normalise(_rng(w, _K, b, h).standard_normal((T, w.d_k)))
    v = _rng(w, _V, b, h).standard_normal((T, w.d_v))
    beta = 1.0 / (1.0 + np.exp(-_rng(w, _BETA, b, h).standard_normal(T)))
    alpha = np.exp(-_softplus(_rng(w, _ALPHA, b, h).standard_normal(T)))
    return dict(q=q, k=k, v=v, alpha=alpha, beta=beta)


def stream_dy(w: Workload, b: int, h: int) -> np.ndarray:
    return _rng(w, _DY, b, h).standard_normal((w.T, w.d_v), dtype=np.float32)


class Inputs:
    """All inputs of a workload (or of a subset of its streams).

    Arrays are laid out [B, H, T, ...] for the full workload.  With
    ``streams=[(b, h), ...]`` they are laid out [S, 1, T, ...]: each sampled
    stream becomes its own batch row with one head.  ``heads[s]`` is the head
    of flat stream s (its codebook and initial memory) in either layout.
    Streams are drawn in parallel threads; each from its own generator, so
    the values do not depend on the thread count.
    """

    def __init__(self, w: Workload, streams: Sequence[tuple] | None = None, threads: int = 8):
        self.w = w
        if streams is None:
            self.streams = [(b, h) for b in range(w.B) for h in range(w.H)]
            self.shape_bh = (w.B, w.H)
        else:
            self.streams = list(streams)
            self.shape_bh = (len(self.streams), 1)
        S, T = len(self.streams), w.T
        self.heads = [h for _, h in self.streams]
        self.q = Stored((S, T, w.d_k), w.dtype)
        self.k = Stored((S, T, w.d_k), w.dtype)
        self.v = Stored((S, T, w.d_v), w.dtype)
        self.alpha = Stored((S, T), w.dtype)
        self.beta = Stored((S, T), w.dtype)
        self._centres = {}
        if w.clustered_keys:
            for h in sorted(set(self.heads)):
                self._centres[h] = centres_head(w, h)

        def one(s):
            b, h = self.streams[s]
            d = stream_inputs(w, b, h, centres=self._centres.get(h))
            for name in ("q", "k", "v", "alpha", "beta"):
                getattr(self, name).put(s, d[name])

        if S:
            with ThreadPoolExecutor(max(1, min(threads, S))) as ex:
                list(ex.map(one, range(S)))
        bh = self.shape_bh
        for name, last in (("q", (T, w.d_k)), ("k", (T, w.d_k)), ("v", (T, w.d_v)),
                           ("alpha", (T,)), ("beta", (T,))):
            st = getattr(self, name)
            st.f32 = st.f32.reshape(bh + last)
            if st.bits is not None:
                st.bits = st.bits.reshape(bh + last)
        if w.codebook:
            heads = list(range(w.H)) if streams is None else self.heads
            cbs = {h: codebook_head(w, h) for h in set(heads)}
            self.codebook = Stored.from_f64(np.stack([cbs[h] for h in heads]), w.dtype)
        else:
            self.codebook = None
        self._m0_cache = {}

    # initial memory ------------------------------------------------------
    def m0_head(self, h: int) -> np.ndarray | None:
        """fp32 [N, d_v] initial memory of head h (None when it is zero)."""
        if self.w.m0 == "zero":
            return None
        if h not in self._m0_cache:
            self._m0_cache[h] = m0_head(self.w, h)
        return self._m0_cache[h]

    def dy(self) -> np.ndarray:
        w = self.w
        out = np.empty((len(self.streams), w.T, w.d_v), np.float32)
        for s, (b, h) in enumerate(self.streams):
            out[s] = stream_dy(w, b, h)
        return out.reshape(self.shape_bh + (w.T, w.d_v))


def tiny(**kw) -> Workload:
    """A small workload for unit tests (defaults: 2 streams, sqrt(N)=8)."""
    base = dict(name="tiny", B=1, H=2, T=16, d_k=8, d_v=8, N=64, topk=4, dtype="f32", seed=123)
    base.update(kw)
    return Workload(**base)


class LayerInputs:
    """The inputs of the gate producers and the output epilogue for a
    workload's streams, drawn as the recipe above states: gate
    pre-activations ``a_pre``, ``b_pre`` [B, H, T] and the output gate ``g``
    [B, H, T, d_v] in the workload's dtype; per-head ``A`` and ``b_dt`` [H],
    the norm scale ``gamma`` [d_v] and ``dout`` [B, H, T, d_v] in fp32."""

    def __init__(self, w: Workload):
        self.w = w
        B, H, T, dv = w.B, w.H, w.T, w.d_v
        a = np.stack([np.stack([_rng(w, _APRE, b, h).standard_normal(T) for h in range(H)]) for b in range(B)])
        bb = np.stack([np.stack([_rng(w, _BPRE, b, h).standard_normal(T) for h in range(H)]) for b in range(B)])
        g = np.stack([np.stack([_rng(w, _GATE_OUT, b, h).standard_normal((T, dv)) for h in range(H)])
                      for b in range(B)])
        self.a_pre = Stored.from_f64(a.reshape(B, H, T), w.dtype)
        self.b_pre = Stored.from_f64(bb.reshape(B, H, T), w.dtype)
        self.g = Stored.from_f64(g.reshape(B, H, T, dv), w.dtype)
        gp = _rng(w, _GATE_PARAM, 0, 0)
        self.A = gp.uniform(0.0, 16.0, H).astype(np.float32)
        dt = gp.uniform(0.001, 0.1, H)
        self.b_dt = np.log(np.expm1(dt)).astype(np.float32)
        self.gamma = _rng(w, _GAMMA, 0, 0).uniform(0.5, 1.5, dv).astype(np.float32)
        self.dout = np.stack([np.stack([_rng(w, _DOUT, b, h).standard_normal((T, dv), dtype=np.float32)
                                        for h in range(H)]) for b in range(B)]).reshape(B, H, T, dv)
