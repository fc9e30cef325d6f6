"""CPU oracle for one decode step of the activation-sparse gated FFN.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by ``__graft_entry__.smoke()``
and by the CPU-baseline leg of ``bench.py``; never by the GPU library or its
binding.  The arithmetic lives in ``ls_oracle.c`` (plain loops, fp64); this
module marshals numpy arrays and composes the C steps in the order the paper
gives them:

* Eq. 1 (Sec. 2.1): a stage's partial FFN output from its gate/up/down slices.
* Eq. 2 (Sec. 2.1): the refined prediction feature after the first j stages.
* Sec. 3.2.2: the FFN output as a sum over hidden neurons, in any order.
* Sec. 3.3.3: predictor = a linear input projection (PCA role), here followed
  by a linear head that scores neuron blocks (a reading, see the design notes).
* Sec. 3.3.1: stacked learnable hashing at inference (Eq. hash_layer,
  Eq. hashfunc_layer), as an alternative block scorer.

Every function here is pinned by a ``-m "not gpu"`` test; none is "parity
unpinned".
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ls_oracle.c")
_LIB = os.path.join(_HERE, "liblsoracle.so")

F32, F16, BF16 = 0, 1, 2
ACT_REGLU, ACT_SWIGLU_THRESH = 0, 1
SEL_TOPK, SEL_THRESHOLD = 0, 1


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, plain C, no intrinsics)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm", "-lpthread"],
                       check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int
_D = ctypes.c_double
_F = ctypes.c_float


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.orc_decode.argtypes = [_P, _I, ctypes.c_size_t]
        lib.orc_decode.restype = _D
        lib.orc_mlp_input.argtypes = [_I, _P, _I, _P]
        lib.orc_mlp_input.restype = None
        lib.orc_predict.argtypes = [_I, _I, _I, _P, _P, _I, _P, _P, _P]
        lib.orc_predict.restype = None
        lib.orc_select.argtypes = [_P, _I, _I, _I, _I, _F, _I, _I, _P, _P]
        lib.orc_select.restype = _I
        lib.orc_activations.argtypes = [_I, _I, _P, _P, _P, _I, _I, _D, _P, _I, _P, _P, _P, _P]
        lib.orc_activations.restype = None
        lib.orc_down.argtypes = [_I, _I, _P, _I, _I, _P, _P, _P]
        lib.orc_down.restype = None
        lib.orc_ffn_masked_dense.argtypes = [_I, _I, _P, _P, _P, _P, _I, _I, _D, _P, _P, _P]
        lib.orc_ffn_masked_dense.restype = None
        lib.orc_layer_step.argtypes = [_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _I, _D, _I,
                                       _I, _P, _P, _P, _P, _P]
        lib.orc_layer_step.restype = _I
        lib.orc_layer_step_mt.argtypes = [_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _I, _D, _I,
                                          _I, _P, _P, _P, _P, _P, _I]
        lib.orc_layer_step_mt.restype = _I
        lib.orc_hash_predict.argtypes = [_I, _I, _P, _P, _P, _P, _P, _I, _P, _P, _P]
        lib.orc_hash_predict.restype = None
        _lib = lib
    return _lib


def _c(a: np.ndarray, dtype=None) -> np.ndarray:
    if dtype is not None:
        a = np.asarray(a, dtype=dtype)
    return np.ascontiguousarray(a)


def _ptr(a):
    return None if a is None else a.ctypes.data


def storage_code(a: np.ndarray) -> int:
    """Storage type of a weight array: float32, float16, or uint16 holding bfloat16 bits."""
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.float16:
        return F16
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"unsupported weight container {a.dtype}")


def decode(a: np.ndarray) -> np.ndarray:
    """Exact float64 values of a stored weight array, decoded by the C oracle."""
    a = _c(a)
    code = storage_code(a)
    lib = _load()
    flat = a.reshape(-1)
    return np.array([lib.orc_decode(flat.ctypes.data, code, i) for i in range(flat.size)],
                    dtype=np.float64).reshape(a.shape)


def mlp_input(x: np.ndarray, rms: bool) -> np.ndarray:
    """h from the residual x (one token, fp32 [d])."""
    x = _c(x, np.float32)
    h = np.empty(x.shape[0], np.float64)
    _load().orc_mlp_input(x.shape[0], x.ctypes.data, int(rms), h.ctypes.data)
    return h


def predict(p1: np.ndarray, p2: np.ndarray, h: np.ndarray, return_z: bool = False):
    """Scores s = P2 (P1 h), rounded to fp32 (one token)."""
    p1, p2, h = _c(p1), _c(p2), _c(h, np.float64)
    r, d = p1.shape
    nblk = p2.shape[0]
    assert p2.shape[1] == r and h.shape[0] == d and storage_code(p1) == storage_code(p2)
    z = np.empty(r, np.float64)
    s = np.empty(nblk, np.float32)
    _load().orc_predict(d, r, nblk, p1.ctypes.data, p2.ctypes.data, storage_code(p1),
                        h.ctypes.data, z.ctypes.data, s.ctypes.data)
    return (s, z) if return_z else s


def select(scores: np.ndarray, mode: int = SEL_TOPK, k: int = 1, tau: float = 0.0,
           union_batch: bool = False, cap: int | None = None):
    """Block selection over fp32 scores [B, n_blk] (or [n_blk]).

    Returns (idx, count): per token ([B, cap], [B]) or, for a union, ([cap], [1])."""
    s = _c(scores, np.float32)
    if s.ndim == 1:
        s = s[None, :]
    B, nblk = s.shape
    if cap is None:
        cap = nblk
    if union_batch and B > 1:
        idx = np.full(cap, -1, np.int32)
        cnt = np.zeros(1, np.int32)
    else:
        idx = np.full((B, cap), -1, np.int32)
        cnt = np.zeros(B, np.int32)
    rc = _load().orc_select(s.ctypes.data, B, nblk, mode, k, np.float32(tau), int(union_batch),
                            cap, idx.ctypes.data, cnt.ctypes.data)
    if rc != 0:
        raise ValueError("selection does not fit in cap")
    return idx, cnt


def neurons_of_blocks(blocks, block: int) -> np.ndarray:
    """Neuron ids of a block list, expanded in list order."""
    blocks = np.asarray(blocks, np.int64)
    return (blocks[:, None] * block + np.arange(block)[None, :]).reshape(-1).astype(np.int32)


def activations(w, h: np.ndarray, neurons, act: int, thresh: float = 0.0):
    """(g, u, a) of the listed neurons for one token.  ``w`` has .gate .up .bias."""
    gate, up = _c(w.gate), _c(w.up)
    bias = None if w.bias is None else _c(w.bias)
    F, d = gate.shape
    neurons = _c(neurons, np.int32)
    n = neurons.shape[0]
    g = np.empty(n, np.float64)
    u = np.empty(n, np.float64)
    a = np.empty(n, np.float64)
    _load().orc_activations(d, F, gate.ctypes.data, up.ctypes.data, _ptr(bias), storage_code(gate),
                            act, thresh, _c(h, np.float64).ctypes.data, n, neurons.ctypes.data,
                            g.ctypes.data, u.ctypes.data, a.ctypes.data)
    return g, u, a


def down(w, neurons, a: np.ndarray) -> np.ndarray:
    """y = sum over the listed neurons of a_t * Wd[:, neuron_t] (Wd is [d, F])."""
    wd = _c(w.down)
    d, F = wd.shape
    neurons = _c(neurons, np.int32)
    y = np.empty(d, np.float64)
    _load().orc_down(d, F, wd.ctypes.data, storage_code(wd), neurons.shape[0], neurons.ctypes.data,
                     _c(a, np.float64).ctypes.data, y.ctypes.data)
    return y


def ffn_masked_dense(w, h: np.ndarray, act: int, thresh: float = 0.0, mask=None) -> np.ndarray:
    """Dense FFN output, with a_j := 0 wherever mask[j] is 0 (mask None: dense)."""
    gate, up, wd = _c(w.gate), _c(w.up), _c(w.down)
    bias = None if w.bias is None else _c(w.bias)
    F, d = gate.shape
    m = None if mask is None else _c(mask, np.uint8)
    y = np.empty(d, np.float64)
    _load().orc_ffn_masked_dense(d, F, gate.ctypes.data, up.ctypes.data, wd.ctypes.data, _ptr(bias),
                                 storage_code(gate), act, thresh, _c(h, np.float64).ctypes.data,
                                 _ptr(m), y.ctypes.data)
    return y


def sparse_ffn(w, h: np.ndarray, blocks, block: int, act: int, thresh: float = 0.0,
               return_a: bool = False):
    """FFN output over the selected blocks, in list order (Eq. 1 for one stage)."""
    neurons = neurons_of_blocks(blocks, block)
    _, _, a = activations(w, h, neurons, act, thresh)
    y = down(w, neurons, a)
    return (y, a) if return_a else y


def stage_bounds(U: int, K: int):
    """Stage s of K covers entries [floor(s U / K), floor((s+1) U / K)) of the list."""
    return [((s * U) // K, ((s + 1) * U) // K) for s in range(K)]


def staged_ffn(w, x: np.ndarray, h: np.ndarray, blocks, block: int, K: int, act: int,
               thresh: float = 0.0):
    """Eq. 1 and Eq. 2: partial outputs dm[s] of K stages over the priority list, and
    the refined features x_tilde[j] = x + sum_{s <= j} dm[s]."""
    blocks = np.asarray(blocks)
    dms, xt = [], []
    acc = np.asarray(x, np.float64).copy()
    for lo, hi in stage_bounds(len(blocks), K):
        dm = sparse_ffn(w, h, blocks[lo:hi], block, act, thresh) if hi > lo else \
            np.zeros_like(acc)
        dms.append(dm)
        acc = acc + dm
        xt.append(acc.copy())
    return dms, xt


def layer_step(w, cfg, x: np.ndarray, k: int | None = None, n_threads: int = 0):
    """One layer for one token via the C composition: returns (scores, idx, y, x_out).
    n_threads > 0: the same composition with its output loops split over that many threads
    (identical results)."""
    d, F, r, blk = cfg.d_model, cfg.d_ff, cfg.rank, cfg.block
    k = cfg.k if k is None else k
    nblk = F // blk
    gate, up, wd, p1, p2 = (_c(t) for t in (w.gate, w.up, w.down, w.p1, w.p2))
    bias = None if w.bias is None else _c(w.bias)
    x = _c(x, np.float32)
    scores = np.empty(nblk, np.float32)
    idx = np.empty(k, np.int32)
    y = np.empty(d, np.float64)
    x_out = np.empty(d, np.float32)
    args = (d, F, r, blk, gate.ctypes.data, up.ctypes.data, wd.ctypes.data, _ptr(bias),
            p1.ctypes.data, p2.ctypes.data, storage_code(gate), cfg.act, float(w.threshold),
            int(cfg.prenorm), k, x.ctypes.data, scores.ctypes.data, idx.ctypes.data, y.ctypes.data,
            x_out.ctypes.data)
    if n_threads > 0:
        n = _load().orc_layer_step_mt(*args, int(n_threads))
    else:
        n = _load().orc_layer_step(*args)
    if n < 0:
        raise RuntimeError("orc_layer_step failed")
    return scores, idx[:n], y, x_out


def calibrate_threshold(w, cfg, calib_x: np.ndarray, target: float) -> float:
    """Per-layer SwiGLU-threshold t_l: the ceil(target * N)-th smallest |SiLU(g)| over the
    calibration tokens x all d_ff neurons (N = tokens * d_ff).  The gate projection of all
    tokens is one float64 library matmul over exactly decoded weights."""
    H = np.stack([mlp_input(x, cfg.prenorm) for x in calib_x])          # [T, d]
    Wg = _decoded_matrix(w.gate)                                         # [F, d]
    G = H @ Wg.T
    if w.bias is not None:
        G = G + _decoded_matrix(w.bias)[None, :]
    mag = np.abs(G / (1.0 + np.exp(-G))).reshape(-1)
    kth = math.ceil(target * mag.size)
    return float(np.partition(mag, kth - 1)[kth - 1])


def _decoded_matrix(a: np.ndarray) -> np.ndarray:
    """Vectorised exact decode (float16/float32 widen exactly; bf16 bits widen to binary32)."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# ---- quality of the refined next-layer prediction (Sec. 6, the refinement-step validation) ----
#
# The paper measures, after each of K priority-ordered stages of a layer, how well the next
# layer's prediction on the refined feature x~^(j) (Eq. 2) captures that layer's important
# blocks: the importance ratio (importance captured by the predicted set, normalised by the
# most a set of the same size can capture) and the top-10% recall.  Block importance is read
# here as the size of the blocks' contribution to the output: sum over its neurons of
# |a_j| * ||Wd[:, j]||_2 on the layer's complete input.

def block_importance(w, h: np.ndarray, block: int, act: int, thresh: float = 0.0) -> np.ndarray:
    """Importance of every block of a layer on input h (float64 [n_blk])."""
    F = w.gate.shape[0]
    _, _, a = activations(w, h, np.arange(F, dtype=np.int32), act, thresh)
    wd = _decoded_matrix(_c(w.down))
    col = np.sqrt((wd * wd).sum(axis=0))
    return (np.abs(a) * col).reshape(F // block, block).sum(axis=1)


def importance_ratio(imp: np.ndarray, predicted) -> float:
    """Importance of the predicted blocks over the largest importance of as many blocks."""
    predicted = np.asarray(predicted, np.int64)
    best = np.sort(np.asarray(imp, np.float64))[::-1][:predicted.size].sum()
    return float(imp[predicted].sum() / best) if best > 0 else 1.0


def top_fraction_recall(imp: np.ndarray, predicted, frac: float = 0.1) -> float:
    """Share of the ceil(frac * n_blk) most important blocks (ties to the smaller index) that
    the predicted set holds."""
    n = imp.shape[0]
    m = max(1, math.ceil(frac * n))
    top = np.lexsort((np.arange(n), -np.asarray(imp, np.float64)))[:m]
    return float(np.isin(top, np.asarray(predicted)).sum() / m)


def refinement_quality(w_n, w_next, cfg, x: np.ndarray, K: int, order=None, k: int | None = None):
    """Per stage j = 0..K of layer n (j = 0: the one-shot prediction from x), the next layer's
    top-k on the refined feature x~^(j) (Eq. 2) and its (importance ratio, top-10% recall)
    against the next layer's block importance on the complete output x~^(K).  The stages run
    over layer n's priority list, or over list[order] for another order of the same blocks.

    Returns (metrics [(ratio, recall)] * (K+1), predicted sets, refined features)."""
    k = cfg.k if k is None else k
    h = mlp_input(x, cfg.prenorm)
    s = predict(w_n.p1, w_n.p2, h)
    idx = select(s, k=k, cap=k)[0][0]
    lst = idx if order is None else idx[np.asarray(order)]
    _, xt = staged_ffn(w_n, x, h, lst, cfg.block, K, cfg.act, w_n.threshold)
    feats = [np.asarray(x, np.float32)] + [f.astype(np.float32) for f in xt]
    imp = block_importance(w_next, mlp_input(feats[-1], cfg.prenorm), cfg.block, cfg.act,
                           w_next.threshold)
    out, sets = [], []
    for f in feats:
        sc = predict(w_next.p1, w_next.p2, mlp_input(f, cfg.prenorm))
        P = select(sc, k=k, cap=k)[0][0]
        sets.append(P)
        out.append((importance_ratio(imp, P), top_fraction_recall(imp, P)))
    return out, sets, feats


# ---- stacked learnable hashing (Sec. 3.3.1) ----

HASH_TAU, HASH_DH, HASH_LAYERS = 8, 256, 5


def hash_predict(hw, x: np.ndarray, n_blk: int, code0: int | None = None):
    """Block scores of the stacked hashing predictor for one token (fp32 [n_blk]), the five
    bucket indices and the first layer's real products x . W_1[:, b] (float64 [8]).  The first
    bucket is phi(sign(x W_1)) from those float64 products, or ``code0`` when given (the later
    layers are then evaluated from it).  ``hw`` has .w1 (fp32 [d, 8]), .w_bin (uint32 [4, 8, 8]),
    .tables (uint32 [4, 256, 8]), .head (uint8 [256, n_blk])."""
    x = _c(x, np.float32)
    w1, wb, tb, hd = _c(hw.w1, np.float32), _c(hw.w_bin, np.uint32), _c(hw.tables, np.uint32), \
        _c(hw.head, np.uint8)
    d = x.shape[0]
    assert w1.shape == (d, HASH_TAU) and wb.shape == (4, HASH_TAU, HASH_DH // 32)
    assert tb.shape == (4, HASH_DH, HASH_DH // 32) and hd.shape == (HASH_DH, n_blk)
    assert code0 is None or 0 <= code0 < 256
    codes = np.zeros(HASH_LAYERS, np.int32)
    prods = np.zeros(HASH_TAU, np.float64)
    scores = np.empty(n_blk, np.float32)
    _load().orc_hash_predict(d, n_blk, x.ctypes.data, w1.ctypes.data, wb.ctypes.data, tb.ctypes.data,
                             hd.ctypes.data, -1 if code0 is None else int(code0), prods.ctypes.data,
                             codes.ctypes.data, scores.ctypes.data)
    return scores, codes, prods
