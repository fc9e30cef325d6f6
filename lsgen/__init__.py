"""Seeded synthetic inputs for the sparse-FFN decode step.

This package is the only code shared by the CPU oracle's tests and the GPU
path's tests and benchmark.  It draws random numbers and rounds them to a
storage type; it holds none of the method's arithmetic (no projection, no
activation, no selection).

Workloads (``CONFIGS``) are synthetic stand-ins shaped like the FFN stacks of
Llama-2-7B/13B/70B and Mistral-7B; the paper's own models and datasets are not
used.  Tensor ids of the element streams: gate 1, up 2, down 3, P1 5, P2 6,
decode tokens 7, calibration tokens 8.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, field, replace
from statistics import NormalDist

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lsgen.c")
_LIB = os.path.join(_HERE, "liblsgen.so")

BASE_SEED = 20260903
DT_F32, DT_F16, DT_BF16 = 0, 1, 2
DTYPE_NAMES = {DT_F32: "f32", DT_F16: "f16", DT_BF16: "bf16"}
ACT_REGLU, ACT_SWIGLU_THRESH = 0, 1

TID_GATE, TID_UP, TID_DOWN, TID_P1, TID_P2, TID_TOKEN, TID_CALIB, TID_SPREAD = 1, 2, 3, 5, 6, 7, 8, 9
TID_HASH_W1, TID_HASH_WBIN, TID_HASH_TABLES, TID_HASH_HEAD = 10, 11, 12, 13


def build(force: bool = True) -> str:
    """Compile the generator with gcc into ``lsgen/liblsgen.so``."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm", "-lpthread"],
                       check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.lsgen_normal.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                                     ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double,
                                     ctypes.c_double, ctypes.c_int, ctypes.c_void_p, ctypes.c_int]
        lib.lsgen_normal.restype = ctypes.c_int
        lib.lsgen_const.argtypes = [ctypes.c_double, ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p]
        lib.lsgen_const.restype = ctypes.c_int
        lib.lsgen_splitmix64.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        lib.lsgen_splitmix64.restype = ctypes.c_uint64
        _lib = lib
    return _lib


def np_dtype(dtype: int):
    """numpy container for a storage type: float32, float16, or uint16 bits for bf16."""
    return {DT_F32: np.float32, DT_F16: np.float16, DT_BF16: np.uint16}[dtype]


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def normal(shape, *, seed: int, tensor_id: int, layer: int, std: float, mean: float = 0.0,
           dtype: int = DT_F32, offset: int = 0, out: np.ndarray | None = None) -> np.ndarray:
    """Elements ``offset .. offset+prod(shape)`` of stream (seed, tensor_id, layer)."""
    n = int(np.prod(shape)) if len(shape) else 1
    if out is None:
        out = np.empty(shape, dtype=np_dtype(dtype))
    assert out.flags.c_contiguous and out.size == n and out.dtype == np_dtype(dtype)
    rc = _load().lsgen_normal(seed, tensor_id, layer, offset, n, mean, std, dtype,
                              out.ctypes.data, _threads())
    if rc != 0:
        raise ValueError("lsgen_normal rejected its arguments")
    return out


def const(shape, value: float, dtype: int) -> np.ndarray:
    out = np.empty(shape, dtype=np_dtype(dtype))
    if _load().lsgen_const(value, out.size, dtype, out.ctypes.data) != 0:
        raise ValueError("lsgen_const rejected its arguments")
    return out


def to_storage(a: np.ndarray, dtype: int) -> np.ndarray:
    """fp32 values rounded to nearest-even in a storage type (finite inputs)."""
    a = np.ascontiguousarray(a, np.float32)
    if dtype == DT_F32:
        return a
    if dtype == DT_F16:
        return a.astype(np.float16)
    bits = a.view(np.uint32).astype(np.uint64)
    return ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16).astype(np.uint16)


def splitmix64(seed: int, n: int) -> int:
    return int(_load().lsgen_splitmix64(seed, n))


def decode_bits(a: np.ndarray, dtype: int) -> np.ndarray:
    """Exact float64 values of a stored array (bf16 bits widened to binary32)."""
    if dtype == DT_BF16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# --------------------------------------------------------------------------------------
# Workloads
# --------------------------------------------------------------------------------------

@dataclass(frozen=True)
class Config:
    """One synthetic FFN-stack workload."""
    name: str
    n_layers: int
    d_model: int
    d_ff: int
    dtype: int
    act: int
    block: int
    rank: int
    keep_pct: int            # block keep fraction, in percent
    gate_bias: float | None  # constant gate bias (None: no bias)
    prenorm: bool            # RMS prenorm of the residual before the FFN
    steps: int               # decode steps of the workload
    batches: tuple = (1,)
    sparsity_target: float = 0.0  # SwiGLU-threshold neuron sparsity (fraction dropped)
    swiglu_threshold: float = 0.0  # per-layer |SiLU(g)| threshold (same for every layer)
    calib_tokens: int = 64
    host_resident: bool = False
    hbm_cache_bytes: int = 0
    seed: int = BASE_SEED
    note: str = ""
    # "random": predictor factors independent of the FFN weights.  "planted": the gate rows of
    # block b share a direction C_b (rows (C_b + spread_i) B / sqrt(r) + noise), and the
    # predictor is P1 = B, P2 = C / sqrt(r): its block score is the shared part of the block's
    # gate pre-activations, so it ranks blocks by expected activity (a trained predictor's role).
    predictor: str = "random"
    down_gain: float = 1.0   # down-projection std = down_gain / sqrt(d_model)

    @property
    def n_blk(self) -> int:
        return self.d_ff // self.block

    @property
    def k(self) -> int:
        """Blocks kept per token: ceil(keep * n_blk) in integer arithmetic."""
        return (self.keep_pct * self.n_blk + 99) // 100

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == DT_F32 else 2

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


def _probit(p: float) -> float:
    return NormalDist().inv_cdf(p)


CONFIGS = {
    # Single ReGLU layer, fp32: the small case the oracle finishes in seconds.
    "c1_reglu_512": Config("c1_reglu_512", 1, 512, 1536, DT_F32, ACT_REGLU, 32, 64, 20,
                           -0.5, False, 64),
    # Llama-2-7B-shaped FFN stack, fp16, ~10% active neurons.
    "llama2_7b_ffn": Config("llama2_7b_ffn", 32, 4096, 11008, DT_F16, ACT_REGLU, 64, 1024, 12,
                            -_probit(0.90), True, 256),
    # Mistral-7B-shaped FFN stack, bf16, SwiGLU with a per-layer magnitude threshold (50%).
    # The threshold is the median of |SiLU(Z)| for Z ~ N(0, 1) (the gate pre-activation
    # law under the RMS prenorm and N(0, 1/d) rows), found by quadrature: 0.2543196702.
    "mistral_7b_ffn": Config("mistral_7b_ffn", 32, 4096, 14336, DT_BF16, ACT_SWIGLU_THRESH, 128,
                             1024, 50, None, True, 256, batches=(1, 4), sparsity_target=0.5,
                             swiglu_threshold=0.25431967022723184),
    # Llama-2-13B-shaped FFN stack, fp16, ~10% active, batched decode with a block union.
    "llama2_13b_ffn": Config("llama2_13b_ffn", 40, 5120, 13824, DT_F16, ACT_REGLU, 64, 1280, 12,
                             -_probit(0.90), True, 256, batches=(1, 2, 4, 8)),
    # Llama-2-7B-shaped FFN stack with a planted predictor (gate rows of a block share a
    # direction the predictor knows), for the quality of refined next-layer predictions.
    "llama2_7b_planted": Config("llama2_7b_planted", 32, 4096, 11008, DT_F16, ACT_REGLU, 64, 1024, 12,
                                -_probit(0.90), True, 64, predictor="planted"),
    # Llama-2-70B-shaped FFN stack, weights in pinned host memory, 16 GiB HBM block cache.
    "llama2_70b_stream": Config("llama2_70b_stream", 80, 8192, 28672, DT_F16, ACT_REGLU, 128, 2048,
                                10, -_probit(0.92), True, 64, host_resident=True,
                                hbm_cache_bytes=16 << 30),
}


# planted predictor: per-neuron spread of the shared block direction, and the gate noise (both
# relative to the unit shared part)
PLANT_SPREAD = 0.5
PLANT_NOISE = 0.5


@dataclass
class LayerWeights:
    """One layer's weights in storage type, in nn.Linear layouts.

    gate, up: [d_ff, d_model]; down: [d_model, d_ff]; bias: [d_ff] or None;
    p1: [rank, d_model]; p2: [n_blk, rank]; threshold: float (SwiGLU-threshold only).
    """
    gate: np.ndarray
    up: np.ndarray
    down: np.ndarray
    bias: np.ndarray | None
    p1: np.ndarray
    p2: np.ndarray
    threshold: float = 0.0
    extra: dict = field(default_factory=dict)


def layer_weights(cfg: Config, layer: int, threshold: float | None = None) -> LayerWeights:
    """Weights of one layer.  FFN weights ~ N(0, 1/d_model); P1 ~ N(0, 1/d_model);
    P2 ~ N(0, 1/rank); constant gate bias when the config has one."""
    d, F, r, nb, dt, s = cfg.d_model, cfg.d_ff, cfg.rank, cfg.n_blk, cfg.dtype, cfg.seed
    sd = 1.0 / math.sqrt(d)
    up = normal((F, d), seed=s, tensor_id=TID_UP, layer=layer, std=sd, dtype=dt)
    down = normal((d, F), seed=s, tensor_id=TID_DOWN, layer=layer, std=cfg.down_gain * sd, dtype=dt)
    bias = const((F,), cfg.gate_bias, dt) if cfg.gate_bias is not None else None
    if cfg.predictor == "planted":
        B = normal((r, d), seed=s, tensor_id=TID_P1, layer=layer, std=sd, dtype=DT_F32)
        C = normal((nb, r), seed=s, tensor_id=TID_P2, layer=layer, std=1.0, dtype=DT_F32)
        A = normal((F, r), seed=s, tensor_id=TID_SPREAD, layer=layer, std=PLANT_SPREAD, dtype=DT_F32)
        A += np.repeat(C, cfg.block, axis=0)
        A *= np.float32(1.0 / math.sqrt(r))
        G = normal((F, d), seed=s, tensor_id=TID_GATE, layer=layer, std=PLANT_NOISE * sd, dtype=DT_F32)
        G += A @ B
        gate = to_storage(G, dt)
        p1 = to_storage(B, dt)
        p2 = to_storage(C * np.float32(1.0 / math.sqrt(r)), dt)
    else:
        gate = normal((F, d), seed=s, tensor_id=TID_GATE, layer=layer, std=sd, dtype=dt)
        p1 = normal((r, d), seed=s, tensor_id=TID_P1, layer=layer, std=sd, dtype=dt)
        p2 = normal((nb, r), seed=s, tensor_id=TID_P2, layer=layer, std=1.0 / math.sqrt(r), dtype=dt)
    t = cfg.swiglu_threshold if threshold is None else threshold
    return LayerWeights(gate, up, down, bias, p1, p2, t)


def tokens(cfg: Config, step0: int, n_steps: int, batch: int, max_batch: int | None = None
           ) -> np.ndarray:
    """Decode-step inputs x ~ N(0,1), fp32, shape [n_steps, batch, d_model].

    Token t of batch lane b is the element stream of tensor id 7 at offset
    (t * max_batch + b) * d_model."""
    mb = max_batch or batch
    d = cfg.d_model
    out = np.empty((n_steps, batch, d), dtype=np.float32)
    for t in range(n_steps):
        for b in range(batch):
            normal((d,), seed=cfg.seed, tensor_id=TID_TOKEN, layer=0, std=1.0, dtype=DT_F32,
                   offset=((step0 + t) * mb + b) * d, out=out[t, b])
    return out


def calib_tokens(cfg: Config, layer: int) -> np.ndarray:
    """Calibration inputs of one layer, fp32 [calib_tokens, d_model], x ~ N(0,1)."""
    return normal((cfg.calib_tokens, cfg.d_model), seed=cfg.seed, tensor_id=TID_CALIB,
                  layer=layer, std=1.0, dtype=DT_F32)


def adversarial_scores(rng: np.random.Generator, B: int, n_blk: int, kind: str) -> np.ndarray:
    """Host-made score arrays for selection tests: heavy ties, signed zeros, NaN, +-inf."""
    if kind == "ties":
        s = rng.choice(np.array([-1.0, 0.0, 1.0], np.float32), size=(B, n_blk))
    elif kind == "zeros":
        s = rng.choice(np.array([-0.0, 0.0, 1.0, -1.0], np.float32), size=(B, n_blk))
    elif kind == "special":
        s = rng.choice(np.array([np.nan, np.inf, -np.inf, 0.0, -0.0, 1.0, -1.0, 2.0], np.float32),
                       size=(B, n_blk))
    elif kind == "normal":
        s = rng.standard_normal((B, n_blk)).astype(np.float32)
    else:
        raise ValueError(kind)
    return np.ascontiguousarray(s, dtype=np.float32)


@dataclass
class HashWeights:
    """A stacked hashing predictor (5 layers, 8 hash bits, 256-wide binary features).

    w1: fp32 [d_model, 8] real hyperplanes of the first layer; w_bin: uint32 [4, 8, 8] binary
    hyperplanes of layers 2..5 (hash bit b's 256 signs, bit-packed, 1 = +1); tables: uint32
    [4, 256, 8] feature tables T_1..T_4 (bucket i's 256 signs, bit-packed); head: uint8
    [256, n_blk] block-priority levels of the final bucket."""
    w1: np.ndarray
    w_bin: np.ndarray
    tables: np.ndarray
    head: np.ndarray


def _sign_bits(shape_words, *, seed, tensor_id, layer) -> np.ndarray:
    """Random {-1,+1} vectors, bit-packed: bit j of word m is set iff element 32m + j of the
    stream is >= 0 (a fair coin per element)."""
    n_words = int(np.prod(shape_words))
    z = normal((n_words * 32,), seed=seed, tensor_id=tensor_id, layer=layer, std=1.0, dtype=DT_F32)
    bits = (z >= 0).reshape(n_words, 32).astype(np.uint64)
    words = (bits << np.arange(32, dtype=np.uint64)[None, :]).sum(axis=1).astype(np.uint32)
    return words.reshape(shape_words)


def hash_weights(cfg: Config, layer: int) -> HashWeights:
    """Random (untrained) weights of the hashing predictor of one layer: N(0, 1) first-layer
    hyperplanes, fair-coin signs elsewhere, and head levels uniform on 0..255 (8-bit
    equal-probability quantisation of an N(0, 1) draw)."""
    s = cfg.seed
    w1 = normal((cfg.d_model, 8), seed=s, tensor_id=TID_HASH_W1, layer=layer, std=1.0, dtype=DT_F32)
    w_bin = _sign_bits((4, 8, 8), seed=s, tensor_id=TID_HASH_WBIN, layer=layer)
    tables = _sign_bits((4, 256, 8), seed=s, tensor_id=TID_HASH_TABLES, layer=layer)
    z = normal((256, cfg.n_blk), seed=s, tensor_id=TID_HASH_HEAD, layer=layer, std=1.0, dtype=DT_F32)
    u = 0.5 * (1.0 + np.vectorize(math.erf)(z.astype(np.float64) / math.sqrt(2.0)))
    head = np.minimum(np.floor(u * 256.0), 255).astype(np.uint8)
    return HashWeights(w1, w_bin, tables, head)
