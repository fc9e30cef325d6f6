"""Python binding of the gfx950 sparse-FFN decode library (``liblsffn.so``).

Argument marshalling only: every step of the decode path runs in the HIP
kernels behind the C ABI of ``include/ls_ffn.h``.  Function names mirror the C
entry points.  PyTorch supplies device memory and the stream.

The library is loaded from this package directory.  There is no fallback: if
it has not been built, every call raises ``RuntimeError``.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import weakref

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblsffn.so")

LS_OK, LS_E_INVAL, LS_E_NOMEM, LS_E_DEVICE, LS_E_STATE, LS_E_UNSUPPORTED, LS_E_CAPACITY = range(7)
STATUS_NAMES = {0: "LS_OK", 1: "LS_E_INVAL", 2: "LS_E_NOMEM", 3: "LS_E_DEVICE", 4: "LS_E_STATE",
                5: "LS_E_UNSUPPORTED", 6: "LS_E_CAPACITY"}
LS_F32, LS_F16, LS_BF16 = 0, 1, 2
LS_ACT_REGLU, LS_ACT_SWIGLU_THRESH = 0, 1
LS_WEIGHTS_HBM, LS_WEIGHTS_HOST = 0, 1
LS_SEL_TOPK, LS_SEL_THRESHOLD = 0, 1
LS_PREFETCH_NONE, LS_PREFETCH_ONESHOT, LS_PREFETCH_REFINE = 0, 1, 2

EXPORTS = ("ls_ffn_create", "ls_ffn_set_layer", "ls_ffn_destroy", "ls_predict", "ls_select_blocks",
           "ls_sparse_ffn_step", "ls_sparse_ffn_step_static", "ls_stream_weights", "ls_decode_step_streamed", "ls_decode_step",
           "ls_set_hash_predictor", "ls_hash_predict",
           "ls_debug_last_activations", "ls_set_kernel_timing", "ls_kernel_timing",
           "ls_configure", "ls_ffn_sync", "ls_debug_decode_trace", "ls_debug_phase_trace",
           "ls_debug_stages_done", "ls_measure_read_bandwidth", "ls_build_digest", "ls_last_error")
(LS_CFG_DECODE_PATH, LS_CFG_SPEC_BLOCKS, LS_CFG_TRACE_WG, LS_CFG_COOPERATIVE, LS_CFG_BATCH_MFMA, LS_CFG_ZERO_SKIP,
 LS_CFG_STREAM_SYNC, LS_CFG_STAGE_WAIT_US) = range(8)
LS_SYNC_EVENTS, LS_SYNC_FLAGS, LS_SYNC_HOST = range(3)
PHASES = ("layer_start", "input_ready", "scores_published", "all_scores", "acts_gathered",
          "exact_ranked", "slot_map", "misses_done", "partials_ready", "output_published",
          "prefetch_issued", "partials_done", "next_list_ranked", "early_gateup_done",
          "worker_start", "worker_acts_seen")
(LS_K_PRENORM, LS_K_PRED_P1, LS_K_PRED_P2, LS_K_SELECT, LS_K_GATEUP, LS_K_DOWN, LS_K_DECODE,
 LS_K_HASH, LS_K_STAGE) = range(9)


class LsFfnDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("d_ff", ctypes.c_int32), ("block", ctypes.c_int32), ("rank", ctypes.c_int32),
                ("max_batch", ctypes.c_int32), ("dtype", ctypes.c_int), ("act", ctypes.c_int),
                ("residency", ctypes.c_int), ("prenorm_rms", ctypes.c_int32),
                ("hbm_cache_bytes", ctypes.c_uint64), ("stream", ctypes.c_void_p),
                ("debug_flags", ctypes.c_uint32)]


class LsLayerWeights(ctypes.Structure):
    _fields_ = [("w_gate", ctypes.c_void_p), ("w_up", ctypes.c_void_p),
                ("w_down", ctypes.c_void_p), ("b_gate", ctypes.c_void_p),
                ("p1", ctypes.c_void_p), ("p2", ctypes.c_void_p), ("threshold", ctypes.c_float)]


class LsStreamStats(ctypes.Structure):
    _fields_ = [("hits", ctypes.c_int64), ("misses", ctypes.c_int64), ("bytes", ctypes.c_int64),
                ("evictions", ctypes.c_int64)]


class LsHashWeights(ctypes.Structure):
    _fields_ = [("w1", ctypes.c_void_p), ("w_bin", ctypes.c_void_p), ("tables", ctypes.c_void_p),
                ("head", ctypes.c_void_p)]


class LsStreamReport(ctypes.Structure):
    _fields_ = [("final_bytes", ctypes.c_int64), ("copied_bytes", ctypes.c_int64),
                ("late_bytes", ctypes.c_int64), ("spec_bytes", ctypes.c_int64),
                ("wasted_bytes", ctypes.c_int64)]


class LsError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_lib = None


def load():
    """Load ``liblsffn.so`` (no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library not built: {LIB_PATH} is missing (run __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    from . import build as _build
    lib.ls_build_digest.argtypes = []
    lib.ls_build_digest.restype = ctypes.c_char_p
    built = lib.ls_build_digest().decode()
    want = _build.source_digest()
    if built != want:
        raise RuntimeError(f"{LIB_PATH} was built from other sources (digest {built[:12]}, sources "
                           f"{want[:12]}): rebuild it (__graft_entry__.build())")
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.ls_ffn_create.argtypes = [ctypes.POINTER(LsFfnDesc), ctypes.POINTER(ctypes.c_void_p)]
    lib.ls_ffn_set_layer.argtypes = [P, I32, ctypes.POINTER(LsLayerWeights)]
    lib.ls_ffn_destroy.argtypes = [P]
    lib.ls_predict.argtypes = [P, I32, P, I32, P]
    lib.ls_select_blocks.argtypes = [P, P, I32, ctypes.c_int, I32, ctypes.c_float, I32, I32, P, P]
    lib.ls_sparse_ffn_step.argtypes = [P, I32, P, I32, P, P, I32, I32, P]
    lib.ls_sparse_ffn_step_static.argtypes = [P, I32, P, I32, P, P, I32, I32, P]
    lib.ls_stream_weights.argtypes = [P, I32, P, I32, I32, ctypes.POINTER(LsStreamStats)]
    lib.ls_decode_step.argtypes = [P, P, I32, I32]
    lib.ls_decode_step_streamed.argtypes = [P, P, I32, I32, I32, I32, ctypes.POINTER(LsStreamReport)]
    lib.ls_set_hash_predictor.argtypes = [P, I32, ctypes.POINTER(LsHashWeights)]
    lib.ls_hash_predict.argtypes = [P, I32, P, I32, P]
    lib.ls_debug_last_activations.argtypes = [P, P, I64, ctypes.POINTER(I64)]
    lib.ls_set_kernel_timing.argtypes = [P, I32]
    lib.ls_kernel_timing.argtypes = [P, I32, I32, ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(I64)]
    lib.ls_configure.argtypes = [P, I32, I64]
    lib.ls_ffn_sync.argtypes = [P]
    lib.ls_debug_decode_trace.argtypes = [P, I32, P, P]
    lib.ls_debug_phase_trace.argtypes = [P, P, I64, ctypes.POINTER(I64)]
    lib.ls_measure_read_bandwidth.argtypes = [P, P, I64, I32, ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(ctypes.c_double)]
    lib.ls_last_error.argtypes = [P]
    lib.ls_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name not in ("ls_last_error", "ls_build_digest"):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(lib, ctx, status: int):
    if status != LS_OK:
        msg = lib.ls_last_error(ctx)
        raise LsError(status, msg.decode() if msg else "")


def _ptr(t) -> int | None:
    """Device pointer of a torch tensor (or None)."""
    return None if t is None else t.data_ptr()


def _host_ptr(a):
    return None if a is None else np.ascontiguousarray(a).ctypes.data


_live = weakref.WeakSet()


@atexit.register
def _close_all():
    """Destroy every context still open at interpreter exit, while the HIP runtime is alive:
    objects left to the garbage collector would otherwise be released during interpreter
    teardown, after the runtime's own exit handlers may have run."""
    for f in list(_live):
        try:
            f.close()
        except Exception:
            pass


class Ffn:
    """One library context.  Methods mirror the C entry points one to one."""

    def __init__(self, *, n_layers, d_model, d_ff, block, rank, max_batch=1, dtype=LS_F16,
                 act=LS_ACT_REGLU, residency=LS_WEIGHTS_HBM, prenorm_rms=1, hbm_cache_bytes=0,
                 stream=None):
        self.lib = load()
        import torch
        if stream is None:
            stream = torch.cuda.current_stream()
        self.torch_stream = stream
        desc = LsFfnDesc(n_layers, d_model, d_ff, block, rank, max_batch, dtype, act, residency,
                         prenorm_rms, hbm_cache_bytes, ctypes.c_void_p(stream.cuda_stream), 0)
        h = ctypes.c_void_p()
        st = self.lib.ls_ffn_create(ctypes.byref(desc), ctypes.byref(h))
        _check(self.lib, None, st)
        self.ctx = h
        self.n_layers, self.d_model, self.d_ff, self.block, self.rank = (n_layers, d_model, d_ff,
                                                                          block, rank)
        self.n_blk = d_ff // block
        self.max_batch = max_batch
        _live.add(self)

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.ls_ffn_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def ls_ffn_set_layer(self, layer: int, w) -> None:
        """w: object with gate, up, down, bias, p1, p2 (host arrays in storage type), threshold."""
        arrs = [np.ascontiguousarray(a) if a is not None else None
                for a in (w.gate, w.up, w.down, w.bias, w.p1, w.p2)]
        lw = LsLayerWeights(*[_host_ptr(a) for a in arrs], float(getattr(w, "threshold", 0.0)))
        _check(self.lib, self.ctx, self.lib.ls_ffn_set_layer(self.ctx, layer, ctypes.byref(lw)))

    def ls_predict(self, layer: int, x, B: int, scores) -> None:
        _check(self.lib, self.ctx, self.lib.ls_predict(self.ctx, layer, _ptr(x), B, _ptr(scores)))

    def ls_select_blocks(self, scores, B: int, mode: int, k: int, tau: float, union_batch: int,
                         cap: int, idx, count) -> None:
        _check(self.lib, self.ctx, self.lib.ls_select_blocks(self.ctx, _ptr(scores), B, mode, k, tau,
                                                             union_batch, cap, _ptr(idx),
                                                             _ptr(count)))

    def ls_sparse_ffn_step(self, layer: int, x_in, B: int, idx, count, begin: int, end: int,
                           x_acc) -> None:
        _check(self.lib, self.ctx, self.lib.ls_sparse_ffn_step(self.ctx, layer, _ptr(x_in), B,
                                                               _ptr(idx), _ptr(count), begin, end,
                                                               _ptr(x_acc)))

    def ls_sparse_ffn_step_static(self, layer: int, x_in, B: int, idx, count, begin: int, end: int,
                                  x_acc) -> None:
        _check(self.lib, self.ctx, self.lib.ls_sparse_ffn_step_static(self.ctx, layer, _ptr(x_in), B,
                                                                      _ptr(idx), _ptr(count), begin, end,
                                                                      _ptr(x_acc)))

    def ls_stream_weights(self, layer: int, idx_host, n_stages: int = 1) -> LsStreamStats:
        a = np.ascontiguousarray(idx_host, dtype=np.int32)
        stats = LsStreamStats()
        _check(self.lib, self.ctx, self.lib.ls_stream_weights(self.ctx, layer, a.ctypes.data,
                                                              int(a.size), n_stages,
                                                              ctypes.byref(stats)))
        return stats

    def ls_set_hash_predictor(self, layer: int, hw) -> None:
        """hw: .w1 fp32 [d, 8], .w_bin uint32 [4, 8, 8], .tables uint32 [4, 256, 8], .head uint8 [256, n_blk]"""
        arrs = [np.ascontiguousarray(hw.w1, np.float32), np.ascontiguousarray(hw.w_bin, np.uint32),
                np.ascontiguousarray(hw.tables, np.uint32), np.ascontiguousarray(hw.head, np.uint8)]
        if arrs[0].shape != (self.d_model, 8) or arrs[1].shape != (4, 8, 8) or \
                arrs[2].shape != (4, 256, 8) or arrs[3].shape != (256, self.d_ff // self.block):
            raise ValueError("hashing predictor arrays have the wrong shapes")
        w = LsHashWeights(*[a.ctypes.data for a in arrs])
        _check(self.lib, self.ctx, self.lib.ls_set_hash_predictor(self.ctx, layer, ctypes.byref(w)))

    def ls_hash_predict(self, layer: int, x, B: int, scores) -> None:
        _check(self.lib, self.ctx, self.lib.ls_hash_predict(self.ctx, layer, _ptr(x), B, _ptr(scores)))

    def ls_decode_step_streamed(self, x, k: int, n_stages: int, mode: int, k_spec: int = 0
                                ) -> LsStreamReport:
        rep = LsStreamReport()
        _check(self.lib, self.ctx, self.lib.ls_decode_step_streamed(self.ctx, _ptr(x), k, n_stages,
                                                                    mode, k_spec, ctypes.byref(rep)))
        return rep

    def ls_decode_step(self, x, B: int, k: int) -> None:
        _check(self.lib, self.ctx, self.lib.ls_decode_step(self.ctx, _ptr(x), B, k))

    def ls_configure(self, key: int, value: int) -> None:
        _check(self.lib, self.ctx, self.lib.ls_configure(self.ctx, key, int(value)))

    def ls_debug_decode_trace(self, layer: int, x_in=None, scores=None) -> None:
        _check(self.lib, self.ctx, self.lib.ls_debug_decode_trace(self.ctx, layer, _ptr(x_in),
                                                                  _ptr(scores)))

    def ls_debug_phase_trace(self):
        """Phase timestamps [n_layers, 16] (100 MHz ticks) of the traced workgroup (see PHASES)."""
        out = np.zeros((self.n_layers, len(PHASES)), np.int64)
        n = ctypes.c_int64()
        _check(self.lib, self.ctx, self.lib.ls_debug_phase_trace(self.ctx, out.ctypes.data, out.size,
                                                                 ctypes.byref(n)))
        return out

    def ls_debug_stages_done(self, layer: int) -> int:
        """Stages of the layer's latest flagged request whose done word carries its tag."""
        n = ctypes.c_int32()
        _check(self.lib, self.ctx, self.lib.ls_debug_stages_done(self.ctx, layer, ctypes.byref(n)))
        return n.value

    def ls_ffn_sync(self) -> None:
        _check(self.lib, self.ctx, self.lib.ls_ffn_sync(self.ctx))

    def ls_set_kernel_timing(self, enable: bool, kernels=None) -> None:
        """enable: bracket launches with HIP events; kernels: the LS_K_* ids to bracket
        (default: every kernel)."""
        mask = 0
        if enable:
            mask = 1 if kernels is None else sum(1 << int(k) for k in set(kernels) if int(k) != LS_K_PRENORM)
            if mask == 0:
                raise ValueError("no launching kernel id given")
        _check(self.lib, self.ctx, self.lib.ls_set_kernel_timing(self.ctx, mask))

    def ls_kernel_timing(self, kernel: int, reset: bool = False):
        """(total milliseconds, launches) of one kernel id since the last reset."""
        ms, n = ctypes.c_double(), ctypes.c_int64()
        _check(self.lib, self.ctx, self.lib.ls_kernel_timing(self.ctx, kernel, int(reset),
                                                             ctypes.byref(ms), ctypes.byref(n)))
        return ms.value, n.value

    def ls_measure_read_bandwidth(self, buf, reps: int = 10):
        """(best, median) GB/s of a streaming-read kernel over the device tensor buf."""
        best, med = ctypes.c_double(), ctypes.c_double()
        nbytes = buf.numel() * buf.element_size()
        _check(self.lib, self.ctx, self.lib.ls_measure_read_bandwidth(self.ctx, _ptr(buf), nbytes, reps,
                                                                      ctypes.byref(best), ctypes.byref(med)))
        return best.value, med.value

    def ls_debug_last_activations(self, dst) -> int:
        n = ctypes.c_int64()
        _check(self.lib, self.ctx, self.lib.ls_debug_last_activations(self.ctx, _ptr(dst),
                                                                      dst.numel(), ctypes.byref(n)))
        return n.value
