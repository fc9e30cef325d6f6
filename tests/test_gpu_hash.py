"""GPU parity of the stacked hashing predictor (Sec. 3.3.1): block scores bit-exact against the
oracle for several widths, ragged block counts and batch sizes, plus the edge cases the
definition fixes.

The oracle takes the first layer's eight real products in float64 (the definition sign(x W_1));
the kernel sums them in binary32.  A decision is held to the oracle's sign unless its product
lies within the worst-case binary32 summation error of zero, gamma_d * sum_j |x_j W_1[j, b]|
with gamma_n = n u / (1 - n u), u = 2^-24, which bounds any order of d fused multiply-adds.
For a decision inside that band either sign is correct: the GPU's scores must then equal the
oracle's for one of the in-band sign choices, the later (integer) layers re-derived from it."""
import itertools

import numpy as np
import pytest

import lsgen
import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_03079_amd as lsffn  # noqa: E402
from gpu_util import dev_f32, empty_f32, empty_i32, host  # noqa: E402

CASES = {
    "d1024_nb32": lsgen.CONFIGS["llama2_7b_ffn"].with_(n_layers=2, d_model=1024, d_ff=4096, block=128, rank=256),
    "d4096_nb172": lsgen.CONFIGS["llama2_7b_ffn"].with_(n_layers=2),
    "d512_nb300": lsgen.CONFIGS["c1_reglu_512"].with_(n_layers=1, d_ff=9600, block=32),
}


def _ctx(cfg, B):
    f = lsffn.Ffn(n_layers=cfg.n_layers, d_model=cfg.d_model, d_ff=cfg.d_ff, block=cfg.block,
                  rank=cfg.rank, max_batch=B, dtype=cfg.dtype, act=cfg.act)
    hws = []
    for l in range(cfg.n_layers):
        hw = lsgen.hash_weights(cfg, l)
        f.ls_set_hash_predictor(l, hw)
        hws.append(hw)
    return f, hws


def _gamma(n: int) -> float:
    u = 2.0 ** -24
    return n * u / (1.0 - n * u)


def _check_token(hw, x, nb, got):
    """GPU scores ``got`` of one token against the oracle under the guard band; returns the
    number of in-band first-layer decisions."""
    ref, codes, prods = oracle.hash_predict(hw, x, nb)
    absum = np.abs(x.astype(np.float64)[:, None] * hw.w1.astype(np.float64)).sum(axis=0)
    band = np.abs(prods) <= _gamma(x.shape[0]) * absum
    band &= absum > 0          # an exactly zero product (x = 0) is exact in any precision
    if not band.any():
        assert np.array_equal(got, ref)
        return 0
    inband = [b for b in range(8) if band[b]]
    fixed = int(codes[0])
    for choice in itertools.product([0, 1], repeat=len(inband)):
        c0 = fixed
        for bit, v in zip(inband, choice):
            c0 = (c0 & ~(1 << (7 - bit))) | (v << (7 - bit))
        alt, _, _ = oracle.hash_predict(hw, x, nb, code0=c0)
        if np.array_equal(got, alt):
            return len(inband)
    raise AssertionError(f"scores match no sign choice of the in-band bits {inband}")


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("B", [1, 3, 8])
def test_hash_scores_bit_exact(name, B):
    cfg = CASES[name]
    f, hws = _ctx(cfg, B)
    nb = cfg.n_blk
    x = lsgen.tokens(cfg, 7, 1, B, max_batch=B)[0]          # [B, d]
    scores = empty_f32(B, nb)
    for l in range(cfg.n_layers):
        f.ls_hash_predict(l, dev_f32(x), B, scores)
        got = host(scores)
        for b in range(B):
            _check_token(hws[l], x[b], nb, got[b])
        # ranking those scores: ties are the rule here (256 levels), broken by index
        k = min(cfg.k, nb)
        idx, cnt = empty_i32(B, k), empty_i32(B)
        f.ls_select_blocks(scores, B, lsffn.LS_SEL_TOPK, k, 0.0, 0, k, idx, cnt)
        ref_idx, _ = oracle.select(got, k=k, cap=k)
        assert np.array_equal(host(idx), ref_idx)
    f.ls_ffn_sync()


def test_hash_many_tokens_guard_band():
    """64 tokens on the 4096-wide shape: every decision outside the band equals the oracle's."""
    cfg = CASES["d4096_nb172"]
    f, hws = _ctx(cfg, 8)
    nb = cfg.n_blk
    scores = empty_f32(8, nb)
    inband = 0
    for t in range(8):
        x = lsgen.tokens(cfg, 100 + t, 1, 8, max_batch=8)[0]
        f.ls_hash_predict(0, dev_f32(x), 8, scores)
        got = host(scores)
        for b in range(8):
            inband += _check_token(hws[0], x[b], nb, got[b])
    f.ls_ffn_sync()
    assert inband < 64 * 8 // 4    # the band is a small part of the decisions


def test_hash_edge_cases():
    cfg = CASES["d1024_nb32"]
    f, hws = _ctx(cfg, 4)
    nb = cfg.n_blk
    x = lsgen.tokens(cfg, 3, 1, 4, max_batch=4)[0]
    x[0] = 0.0                         # every product 0: sign(0) = +1, first bucket 255
    x[2] = x[1] * np.float32(1024.0)   # a power-of-two scale changes no rounding: same codes
    x[3, :] = np.float32(-1e-30)       # tiny values still decide by sign
    scores = empty_f32(4, nb)
    f.ls_hash_predict(0, dev_f32(x), 4, scores)
    got = host(scores)
    for b in range(4):
        _check_token(hws[0], x[b], nb, got[b])
    ref0, codes0, prods0 = oracle.hash_predict(hws[0], x[0], nb)
    assert codes0[0] == 255 and np.all(prods0 == 0) and np.array_equal(got[0], ref0)
    assert np.array_equal(got[1], got[2])
    with pytest.raises(lsffn.LsError) as e:
        f.ls_hash_predict(1, dev_f32(x), 5, scores)   # B above max_batch
    assert e.value.status == lsffn.LS_E_INVAL
    g = lsffn.Ffn(n_layers=1, d_model=cfg.d_model, d_ff=cfg.d_ff, block=cfg.block, rank=cfg.rank,
                  max_batch=1, dtype=cfg.dtype, act=cfg.act)
    with pytest.raises(lsffn.LsError) as e:
        g.ls_hash_predict(0, dev_f32(x[:1]), 1, scores)
    assert e.value.status == lsffn.LS_E_STATE
    f.ls_ffn_sync()
