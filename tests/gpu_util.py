"""Helpers shared by the GPU tests: build a library context from a workload and
compare it against the oracle.  Imported only by tests marked ``gpu``."""
from __future__ import annotations

import numpy as np
import torch

import lsgen
import paper_2609_03079_amd as lsffn

DEV = "cuda:0"

# tolerance on the FFN output y = x_out - x_in, relative L2 (fp32 weights: 1e-5; 16-bit: 2e-3)
Y_TOL = {lsgen.DT_F32: 1e-5, lsgen.DT_F16: 2e-3, lsgen.DT_BF16: 2e-3}
SCORE_TOL = 1e-5


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    if nb == 0:
        return 0.0 if np.all(a == 0) else float("inf")
    return float(np.linalg.norm(a - b) / nb)


def y_err(a, b) -> float:
    """Error of an FFN output a against the reference b: the larger of the relative L2 error
    and the largest element error over the largest reference element, so one wrong output
    column cannot hide in the vector norm.  Both are held to the same tolerance."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    mb = np.max(np.abs(b)) if b.size else 0.0
    if mb == 0:
        return 0.0 if np.all(a == 0) else float("inf")
    return max(rel_l2(a, b), float(np.max(np.abs(a - b)) / mb))


def make_ffn(cfg: lsgen.Config, n_layers: int | None = None, max_batch: int = 1,
             residency: int = lsffn.LS_WEIGHTS_HBM, hbm_cache_bytes: int = 0, weights=None):
    """Context for cfg (optionally fewer layers) and the host weights it was given."""
    L = cfg.n_layers if n_layers is None else n_layers
    f = lsffn.Ffn(n_layers=L, d_model=cfg.d_model, d_ff=cfg.d_ff, block=cfg.block, rank=cfg.rank,
                  max_batch=max_batch, dtype=cfg.dtype, act=cfg.act, residency=residency,
                  prenorm_rms=int(cfg.prenorm), hbm_cache_bytes=hbm_cache_bytes)
    ws = []
    for l in range(L):
        w = weights[l] if weights is not None else lsgen.layer_weights(cfg, l)
        f.ls_ffn_set_layer(l, w)
        ws.append(w)
    return f, ws


def dev_f32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(DEV)


def empty_f32(*shape) -> torch.Tensor:
    return torch.empty(*shape, dtype=torch.float32, device=DEV)


def empty_i32(*shape) -> torch.Tensor:
    return torch.full(shape, -7, dtype=torch.int32, device=DEV)


def host(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.cpu().numpy()
