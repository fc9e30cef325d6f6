"""GPU: row-level zero skip within the selected blocks (LS_CFG_ZERO_SKIP).

A neuron whose gate output is zero contributes nothing to Eq. 1, so reading its up row and
its down vector can be skipped without changing any sum.  The library's zero-skip kernels
must therefore give outputs EQUAL to the block path's (torch.equal) on the same inputs, and
the block path is itself checked against the oracle; ReGLU shapes are also checked against
the oracle directly.  Cases: several tiles with ragged tails, batches 1-3 and 8 (skip only
when every token's gate output is zero), stages over the list (Eq. 1 partial outputs),
dead blocks, host-resident blocks through the cache's slot table, the per-kernel decode
step, and full-size 7B and Mistral-7B layers in the launch configuration the benchmark
times.
"""
import numpy as np
import pytest

import lsgen
import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_03079_amd as lsffn  # noqa: E402
from gpu_util import Y_TOL, dev_f32, empty_f32, empty_i32, host, make_ffn, y_err  # noqa: E402

C = lsgen.CONFIGS

SMALL = {
    "c1": C["c1_reglu_512"],
    "f16_ragged": C["llama2_7b_ffn"].with_(n_layers=2, d_model=576, d_ff=1200, block=24, rank=192,
                                           keep_pct=30),
    "bf16_swiglu": C["mistral_7b_ffn"].with_(n_layers=2, d_model=512, d_ff=2048, block=128,
                                             rank=128, keep_pct=50),
    "f32_stack": C["c1_reglu_512"].with_(n_layers=3, prenorm=True, d_model=320, d_ff=960,
                                         block=40, rank=64),
    "f16_b64": C["llama2_7b_ffn"].with_(n_layers=2, d_model=640, d_ff=1728, block=64, rank=192,
                                        keep_pct=30),
    # fp32 blocks of 520 neurons: 33 16-byte chunks per lane and column tile, past the 32 whose
    # activity the down kernel tracks
    "f32_wide": C["c1_reglu_512"].with_(n_layers=1, d_model=64, d_ff=2080, block=520, rank=64,
                                        keep_pct=50),
}


def _both(f, layer, x_in, B, idx, cnt, begin, end, d, F):
    """(outputs, activations) of one sparse step with zero skip off, then on."""
    outs, acts = [], []
    for zs in (0, 1):
        f.ls_configure(lsffn.LS_CFG_ZERO_SKIP, zs)
        out = empty_f32(B, d)
        f.ls_sparse_ffn_step(layer, x_in, B, idx, cnt, begin, end, out)
        a = empty_f32(B * F)
        n = f.ls_debug_last_activations(a)
        outs.append(host(out))
        acts.append(host(a)[:B * n])
    f.ls_configure(lsffn.LS_CFG_ZERO_SKIP, 0)
    return outs, acts


@pytest.mark.parametrize("name", list(SMALL))
@pytest.mark.parametrize("B", [1, 2, 3, 8])
def test_zero_skip_equals_block_path(name, B):
    cfg = SMALL[name]
    f, ws = make_ffn(cfg, max_batch=B)
    f.ls_configure(lsffn.LS_CFG_BATCH_MFMA, 0)  # zero skip runs the vector-ALU kernels at every B
    xs = lsgen.tokens(cfg, 7, 1, B)[0]
    x_in = dev_f32(xs)
    scores = empty_f32(B, cfg.n_blk)
    cap = min(cfg.n_blk, B * cfg.k)
    idx, cnt = empty_i32(cap), empty_i32(1)
    skipped = 0
    for l in range(cfg.n_layers):
        f.ls_predict(l, x_in, B, scores)
        f.ls_select_blocks(scores, B, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 1, cap, idx, cnt)
        (y0, y1), (a0, a1) = _both(f, l, x_in, B, idx, cnt, 0, cap, cfg.d_model, cfg.d_ff)
        assert np.array_equal(y0, y1), (name, B, l)
        # the union list has U <= cap entries: positions past it are not written by either step
        U = int(host(cnt)[0])
        a = a1.reshape(B, -1)[:, :U * cfg.block]
        assert np.array_equal(a0.reshape(B, -1)[:, :U * cfg.block], a), (name, B, l)
        skipped += int((~(a != 0).any(axis=0)).sum())
        if cfg.act == lsgen.ACT_REGLU:
            blocks = host(idx)[:U]
            xi = host(x_in)
            for b in range(B):
                y_ref = oracle.sparse_ffn(ws[l], oracle.mlp_input(xi[b], cfg.prenorm), blocks, cfg.block,
                                          cfg.act, ws[l].threshold)
                assert y_err(y1[b].astype(np.float64) - xi[b], y_ref) <= Y_TOL[cfg.dtype], (name, B, l, b)
        x_in = dev_f32(y1)
    assert skipped > 0  # the case exercises the skip


@pytest.mark.parametrize("name", ["c1", "f16_ragged", "bf16_swiglu"])
def test_zero_skip_stages(name):
    """Eq. 1 partial outputs over stages of the list: every stage's accumulated output equal."""
    cfg = SMALL[name]
    f, _ = make_ffn(cfg, n_layers=1)
    x_in = dev_f32(lsgen.tokens(cfg, 2, 1, 1)[0])
    scores = empty_f32(1, cfg.n_blk)
    idx, cnt = empty_i32(cfg.k), empty_i32(1)
    f.ls_predict(0, x_in, 1, scores)
    f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 0, cfg.k, idx, cnt)
    K = 3
    accs = []
    for zs in (0, 1):
        f.ls_configure(lsffn.LS_CFG_ZERO_SKIP, zs)
        acc = empty_f32(1, cfg.d_model)
        stages = []
        for s in range(K):
            f.ls_sparse_ffn_step(0, x_in, 1, idx, cnt, s * cfg.k // K, (s + 1) * cfg.k // K, acc)
            stages.append(host(acc).copy())
        accs.append(stages)
    for s in range(K):
        assert np.array_equal(accs[0][s], accs[1][s]), (name, s)


def test_zero_skip_dead_blocks():
    """Blocks whose every gate output is zero: only gate rows are read, output equal."""
    cfg = SMALL["f16_ragged"].with_(n_layers=1)
    w = lsgen.layer_weights(cfg, 0)
    dead = [2, 5, 11]
    b = w.bias.copy()
    for blk in dead:
        b[blk * cfg.block:(blk + 1) * cfg.block] = np.float16(-1e4)
    w.bias = b
    f, _ = make_ffn(cfg, n_layers=1, weights=[w])
    x = lsgen.tokens(cfg, 3, 1, 1)[0]
    order = np.array([0, 2, 3, 5, 7, 11], np.int32)
    (y0, y1), (a0, a1) = _both(f, 0, dev_f32(x), 1, dev_f32(order).int(), dev_f32([6]).int(), 0, 6,
                               cfg.d_model, cfg.d_ff)
    assert np.array_equal(y0, y1) and np.array_equal(a0, a1)
    a = a1[:6 * cfg.block].reshape(6, cfg.block)
    for pos, blk in enumerate(order):
        if blk in dead:
            assert np.all(a[pos] == 0.0)
    y_ref = oracle.sparse_ffn(w, oracle.mlp_input(x[0], cfg.prenorm), [0, 3, 7], cfg.block, cfg.act,
                              w.threshold)
    assert y_err(y1[0].astype(np.float64) - x[0], y_ref) <= Y_TOL[cfg.dtype]
    # every block dead: the output is the input
    all_dead = np.array(dead, np.int32)
    (z0, z1), _ = _both(f, 0, dev_f32(x), 1, dev_f32(all_dead).int(), dev_f32([3]).int(), 0, 3,
                        cfg.d_model, cfg.d_ff)
    assert np.array_equal(z1[0], x[0]) and np.array_equal(z0, z1)


def test_zero_skip_host_resident_blocks():
    """Blocks in the HBM cache (slot table): equal outputs with and without the skip."""
    cfg = C["llama2_70b_stream"].with_(n_layers=2, d_model=1024, d_ff=4096, block=128, rank=256)
    slots = 12
    bb = 3 * cfg.block * cfg.d_model * cfg.elem_bytes
    ws = [lsgen.layer_weights(cfg, l) for l in range(cfg.n_layers)]
    fh, _ = make_ffn(cfg, weights=ws, residency=lsffn.LS_WEIGHTS_HOST, hbm_cache_bytes=slots * bb)
    x = dev_f32(lsgen.tokens(cfg, 4, 1, 1)[0])
    n = 8
    scores = empty_f32(1, cfg.n_blk)
    idx, cnt = empty_i32(n), empty_i32(1)
    for l in range(cfg.n_layers):
        fh.ls_predict(l, x, 1, scores)
        fh.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, n, 0.0, 0, n, idx, cnt)
        fh.ls_stream_weights(l, host(idx), n_stages=2)
        (y0, y1), _ = _both(fh, l, x, 1, idx, cnt, 0, n, cfg.d_model, cfg.d_ff)
        assert np.array_equal(y0, y1), l
        y_ref = oracle.sparse_ffn(ws[l], oracle.mlp_input(host(x)[0], cfg.prenorm), host(idx), cfg.block,
                                  cfg.act, ws[l].threshold)
        assert y_err(y1[0].astype(np.float64) - host(x)[0], y_ref) <= Y_TOL[cfg.dtype]
        x = dev_f32(y1)
    fh.ls_ffn_sync()


@pytest.mark.parametrize("B", [1, 3])
def test_zero_skip_decode_step(B):
    """The per-kernel decode step through every layer: equal with and without the skip."""
    cfg = SMALL["f32_stack"]
    f, _ = make_ffn(cfg, max_batch=B)
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, 1)
    x0 = lsgen.tokens(cfg, 9, 1, B)[0]
    got = []
    for zs in (0, 1):
        f.ls_configure(lsffn.LS_CFG_ZERO_SKIP, zs)
        x = dev_f32(x0)
        f.ls_decode_step(x, B, cfg.k)
        got.append(host(x))
    assert np.array_equal(got[0], got[1])
    with pytest.raises(lsffn.LsError):
        f.ls_configure(lsffn.LS_CFG_ZERO_SKIP, 2)


@pytest.mark.parametrize("cfg_name", ["llama2_7b_ffn", "mistral_7b_ffn"])
def test_zero_skip_full_size_layer(cfg_name):
    """One full-size layer of the benchmark's workloads (the launch configuration the zero-skip
    benchmark times): outputs and activations equal, a sample of outputs against the oracle."""
    cfg = C[cfg_name].with_(n_layers=1)
    f, ws = make_ffn(cfg)
    x = lsgen.tokens(cfg, 1, 1, 1)[0]
    x_in = dev_f32(x)
    scores = empty_f32(1, cfg.n_blk)
    idx, cnt = empty_i32(cfg.k), empty_i32(1)
    f.ls_predict(0, x_in, 1, scores)
    f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 0, cfg.k, idx, cnt)
    (y0, y1), (a0, a1) = _both(f, 0, x_in, 1, idx, cnt, 0, cfg.k, cfg.d_model, cfg.d_ff)
    assert np.array_equal(y0, y1) and np.array_equal(a0, a1)
    if cfg.act == lsgen.ACT_REGLU:
        blocks = host(idx)[:cfg.k]
        y_ref = oracle.sparse_ffn(ws[0], oracle.mlp_input(x[0], cfg.prenorm), blocks, cfg.block, cfg.act,
                                  ws[0].threshold)
        assert y_err(y1[0].astype(np.float64) - x[0], y_ref) <= Y_TOL[cfg.dtype]
