"""Seeded synthetic inputs for the LaCT fast-weight layer forward.

This module is shared by the tests, the benchmark and the oracle checks. It
holds no arithmetic of the method itself: it only draws random tensors, puts
them in the shapes of the paper's workloads and rounds them to the I/O
precision. Both the HIP path and the oracle consume exactly the arrays it
returns.

Recipe (one (seed, config) -> one set of host arrays):

* independent sub-streams for q, k, v, eta, W1, W2, W3 (and beta) from
  ``numpy.random.SeedSequence(seed).spawn(8)``;
* q, k, v ~ N(0, 1), L2-normalised per token per head (the layer normalises q
  and k before the fast-weight path, Alg. 1; v is normalised too so that all
  three share one scale), then rounded to bfloat16 (round-to-nearest-even)
  for bf16 workloads;
* eta = 0.01 * softplus(N(0, 1)) per token per head, float32 (a per-token
  learning rate, eq. of the chunk gradient; the 0.01 scale is the paper's
  constant learning-rate bias magnitude);
* W1, W3 in R^{h x d}, W2 in R^{d x h} ~ N(0, 1/d), then every row (the input
  dimension of that matrix) scaled to unit L2 norm, float32, one copy per
  head repeated over the batch (Alg. 1 repeats the per-head initial fast
  weight over the batch);
* per-matrix-rate workloads: eta = 0.01 * softplus(N(0, 1)) drawn as
  [B*H, n_kv, 3] (lr1, lr2, lr3) from the same sub-stream;
* momentum workloads only: beta = sigmoid(N(0, 1)) per token per head,
  float32, from an eighth sub-stream (the factor is the sigmoid of a linear
  projection of the token, App. A; a unit-variance logit stands in for the
  projection), so the other seven draws are the same with or without it.

Cotangents for the backward (``make_cotangents``), from their own two
sub-streams of ``SeedSequence([seed, 1])``: dO ~ N(0, 1/d) per element in the
shape of q (rounded to bfloat16 for bf16 workloads) and the cotangents of the
final fast weights ~ N(0, 1/d) per element, float32 (one d x d matrix for the
linear fast weight, else W1, W2, W3 in that order from the second stream).
"""
from __future__ import annotations

import dataclasses
import numpy as np

__all__ = ["LactConfig", "CONFIGS", "make_inputs", "make_cotangents", "make_schedule", "round_to_bf16",
           "bf16_bits"]


@dataclasses.dataclass(frozen=True)
class LactConfig:
    name: str
    B: int
    H: int
    d: int
    h: int
    n_kv: int
    n_q: int
    chunk: int
    order: int            # 0 = apply-then-update, 1 = update-then-apply
    use_muon: int
    ns_steps: int
    io: str               # "bf16" or "fp32"
    momentum: int = 0     # 1: momentum test-time optimizer (inputs carry beta)
    lr3: int = 0          # 1: per-matrix learning rates, eta [B*H, n_kv, 3]
    schedule: str = ""    # "": uniform chunks in `order`; else a make_schedule() recipe
    layer_io: int = 0     # 1: the step also runs the prologue and the output norm
    linear: int = 0       # 1: linear fast weight f_W(x) = W1 x (h == d; W1 is the state)

    @property
    def BH(self) -> int:
        return self.B * self.H

    @property
    def n_chunks(self) -> int:
        return (self.n_kv + self.chunk - 1) // self.chunk

    def with_(self, **kw) -> "LactConfig":
        return dataclasses.replace(self, **kw)


# The paper's workload shapes (language model, novel-view synthesis, video).
CONFIGS = {
    "tiny_fp32": LactConfig("tiny_fp32", 1, 2, 64, 64, 1024, 1024, 256, 0, 0, 0, "fp32"),
    "lm32k": LactConfig("lm32k", 4, 4, 512, 512, 32768, 32768, 2048, 0, 0, 0, "bf16"),
    "lm32k_muon": LactConfig("lm32k_muon", 4, 4, 512, 512, 32768, 32768, 2048, 0, 1, 5, "bf16"),
    "nvs256k": LactConfig("nvs256k", 1, 1, 768, 1536, 262144, 262144 + 4096, 262144, 1, 0, 0, "bf16"),
    "nvs1m": LactConfig("nvs1m", 1, 1, 768, 1536, 1048576, 1048576 + 4096, 1048576, 1, 0, 0, "bf16"),
    "video": LactConfig("video", 1, 40, 128, 256, 56160, 56160, 3120, 0, 1, 5, "bf16"),
    "lm32k_mom": LactConfig("lm32k_mom", 4, 4, 512, 512, 32768, 32768, 2048, 0, 0, 0, "bf16", 1),
    "lm32k_muon_mom": LactConfig("lm32k_muon_mom", 4, 4, 512, 512, 32768, 32768, 2048, 0, 1, 5, "bf16", 1),
    "lm32k_layer": LactConfig("lm32k_layer", 4, 4, 512, 512, 32768, 32768, 2048, 0, 0, 0, "bf16", layer_io=1),
    # linear fast weight at the NVS shape (a state of d^2 per head)
    "nvs256k_linear": LactConfig("nvs256k_linear", 1, 1, 768, 768, 262144, 262144 + 4096, 262144, 1, 0, 0, "bf16",
                                 linear=1),
    "lm32k_lr3": LactConfig("lm32k_lr3", 4, 4, 512, 512, 32768, 32768, 2048, 0, 0, 0, "bf16", lr3=1),
    # linear fast weight at the LM shape (the workload of its backward)
    "lm32k_linear": LactConfig("lm32k_linear", 4, 4, 512, 512, 32768, 32768, 2048, 0, 0, 0, "bf16", linear=1),
    "lm32k_linear_mom": LactConfig("lm32k_linear_mom", 4, 4, 512, 512, 32768, 32768, 2048, 0, 0, 0, "bf16", 1,
                                   linear=1),
    # video teacher forcing: 18 clean chunks of 3120 tokens interleaved with 19
    # noisy ones, [X1n, X1, ..., X18, X19n] (115440 tokens in all)
    "video_tf": LactConfig("video_tf", 1, 40, 128, 256, 37 * 3120, 37 * 3120, 3120, 0, 1, 5, "bf16",
                           schedule="video_tf"),
}


def make_schedule(cfg: LactConfig):
    """Segments (mode, begin, end) of a scheduled workload.

    "video_tf": the strided mask of teacher-forced video diffusion: noisy
    chunks of `chunk` tokens are applied only, clean ones update then apply,
    alternating and starting and ending with a noisy chunk.
    """
    if cfg.schedule == "video_tf":
        C = cfg.chunk
        assert cfg.n_kv % (2 * C) == C, "odd number of chunks"
        return [("apply_only" if (t // C) % 2 == 0 else "update_then_apply", t, t + C)
                for t in range(0, cfg.n_kv, C)]
    raise ValueError(f"unknown schedule {cfg.schedule!r}")


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 array -> uint16 bfloat16 bit patterns, round-to-nearest-even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    nan = np.isnan(x)
    if nan.any():
        r = np.where(nan, np.uint32(0x7FC0), r)
    return r.astype(np.uint16)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """float32 array rounded (RNE) to the nearest bfloat16, returned as float32."""
    return (bf16_bits(x).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _unit_rows(x: np.ndarray) -> np.ndarray:
    n = np.sqrt(np.sum(x.astype(np.float64) ** 2, axis=-1, keepdims=True))
    return (x / n).astype(np.float32)


def make_inputs(cfg: LactConfig, seed: int = 0, heads: list | None = None):
    """Draw the inputs of one workload.

    Returns a dict of float32 numpy arrays (bf16 workloads hold values that are
    exactly representable in bfloat16):
      q [B*H, n_q, d], k, v [B*H, n_kv, d], eta [B*H, n_kv] (or [B*H, n_kv, 3]),
      W1, W3 [B*H, h, d], W2 [B*H, d, h], and beta [B*H, n_kv] for momentum
      workloads.
    ``heads`` restricts the draw to a subset of the flattened (b, h) instances;
    the values of each kept instance are the same as in the full draw only for
    the weights (token tensors are drawn for the kept instances only).
    """
    ss = np.random.SeedSequence(seed).spawn(8)
    rq, rk, rv, re, r1, r2, r3, rb = (np.random.default_rng(s) for s in ss)
    BH = cfg.BH
    inst = list(range(BH)) if heads is None else list(heads)
    n = len(inst)

    def tok(rng, ntok):
        x = rng.standard_normal((n, ntok, cfg.d), dtype=np.float32)
        x /= np.sqrt(np.sum(np.square(x, dtype=np.float32), axis=-1, keepdims=True))
        return round_to_bf16(x) if cfg.io == "bf16" else x

    q = tok(rq, cfg.n_q)
    k = tok(rk, cfg.n_kv)
    v = tok(rv, cfg.n_kv)
    z = re.standard_normal((n, cfg.n_kv, 3) if cfg.lr3 else (n, cfg.n_kv), dtype=np.float32).astype(np.float64)
    eta = (0.01 * np.logaddexp(0.0, z)).astype(np.float32)

    std = 1.0 / np.sqrt(cfg.d)
    w1 = _unit_rows(r1.standard_normal((cfg.H, cfg.h, cfg.d), dtype=np.float32) * std)
    w2 = _unit_rows(r2.standard_normal((cfg.H, cfg.d, cfg.h), dtype=np.float32) * std)
    w3 = _unit_rows(r3.standard_normal((cfg.H, cfg.h, cfg.d), dtype=np.float32) * std)
    head_of = [i % cfg.H for i in inst]
    W1 = np.ascontiguousarray(w1[head_of])
    W2 = np.ascontiguousarray(w2[head_of])
    W3 = np.ascontiguousarray(w3[head_of])
    out = dict(q=q, k=k, v=v, eta=eta, W1=W1, W2=W2, W3=W3)
    if cfg.momentum:
        zb = rb.standard_normal((n, cfg.n_kv), dtype=np.float32).astype(np.float64)
        out["beta"] = (1.0 / (1.0 + np.exp(-zb))).astype(np.float32)
    return out


def make_cotangents(cfg: LactConfig, seed: int = 0, heads: list | None = None):
    """Seeded cotangents of the layer's outputs: dict with ``do`` [n, n_q, d]
    (the I/O precision's values, float32 arrays) and the final fast weights'
    cotangents, float32: ``dW`` [n, d, d] for the linear fast weight, else
    ``dW1``, ``dW3`` [n, h, d] and ``dW2`` [n, d, h] (drawn in that order);
    n = the number of kept instances."""
    rd, rw, rm = (np.random.default_rng(s) for s in np.random.SeedSequence([seed, 1]).spawn(3))
    n = cfg.BH if heads is None else len(heads)
    std = 1.0 / np.sqrt(cfg.d)
    do = rd.standard_normal((n, cfg.n_q, cfg.d), dtype=np.float32) * np.float32(std)
    if cfg.io == "bf16":
        do = round_to_bf16(do)
    if cfg.linear:
        dW = rw.standard_normal((n, cfg.d, cfg.d), dtype=np.float32) * np.float32(std)
        out = dict(do=do, dW=dW)
        if cfg.momentum:   # the final momentum's cotangent, dM [n, d, d]
            out["dM"] = rm.standard_normal((n, cfg.d, cfg.d), dtype=np.float32) * np.float32(std)
        return out
    dW1 = rw.standard_normal((n, cfg.h, cfg.d), dtype=np.float32) * np.float32(std)
    dW2 = rw.standard_normal((n, cfg.d, cfg.h), dtype=np.float32) * np.float32(std)
    dW3 = rw.standard_normal((n, cfg.h, cfg.d), dtype=np.float32) * np.float32(std)
    out = dict(do=do, dW1=dW1, dW2=dW2, dW3=dW3)
    if cfg.momentum:   # the final momentum's cotangents dM1, dM2, dM3 (shapes of the weights)
        for name, shape in (("dM1", (n, cfg.h, cfg.d)), ("dM2", (n, cfg.d, cfg.h)), ("dM3", (n, cfg.h, cfg.d))):
            out[name] = rm.standard_normal(shape, dtype=np.float32) * np.float32(std)
    return out


def make_momentum_state(cfg: LactConfig, seed: int = 0, heads: list | None = None):
    """A seeded momentum state to start from, float32: ``M`` [n, d, d] for the
    linear fast weight, else ``M1``, ``M3`` [n, h, d] and ``M2`` [n, d, h].
    Entries are N(0, 1) times 1e-3 / sqrt(d): a few chunk gradients' worth at
    the rates of make_inputs (a chunk gradient's entries are ~1e-3 of the
    weights' own, which are ~1 / sqrt(d))."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 2]))
    n = cfg.BH if heads is None else len(heads)
    sc = np.float32(1e-3 / np.sqrt(cfg.d))
    if cfg.linear:
        return dict(M=rng.standard_normal((n, cfg.d, cfg.d), dtype=np.float32) * sc)
    return {name: rng.standard_normal(shape, dtype=np.float32) * sc
            for name, shape in (("M1", (n, cfg.h, cfg.d)), ("M2", (n, cfg.d, cfg.h)), ("M3", (n, cfg.h, cfg.d)))}
