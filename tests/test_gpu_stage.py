"""GPU: device-side arrival flags for the streamed step (LS_CFG_STREAM_SYNC).

The copy stream writes an arrival word after each stage's copies; one persistent kernel per
layer consumes the stages as they land (Sec. 3.2.1, Alg. 1).  It runs the per-call kernels'
own per-neuron and per-tile code, so the streamed step must give the same x BITWISE with
device flags, with per-stage events and with a host synchronisation after every stage, and
the same as the staged computation on HBM-resident weights (itself checked against the
oracle in the streaming tests).  Cases: evictions (a cache of 12 slots for 3 layers of
lists), stage counts that leave stages empty, one-shot prefetch, plain and cooperative
launches, two tokens in a row (the kernel's counters reset between calls), every done word
written, a full-size 70B-shaped layer pair, and the refused combinations.
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

CFG = lsgen.CONFIGS["llama2_70b_stream"].with_(n_layers=3, d_model=1024, d_ff=4096, block=128,
                                                 rank=256)  # k = 4 of 32 blocks
SLOTS = 12


def _block_bytes(cfg):
    return 3 * cfg.block * cfg.d_model * cfg.elem_bytes


def _host_ctx(cfg, ws, slots):
    f, _ = make_ffn(cfg, weights=ws, residency=lsffn.LS_WEIGHTS_HOST, hbm_cache_bytes=slots * _block_bytes(cfg))
    return f


def _replay_resident(fr, cfg, x0, k, K):
    """The same staged computation through the per-layer calls on HBM-resident weights."""
    cur = dev_f32(x0)
    scores = empty_f32(1, cfg.n_blk)
    idx, cnt = empty_i32(k), empty_i32(1)
    for l in range(cfg.n_layers):
        fr.ls_predict(l, cur, 1, scores)
        fr.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, k, 0.0, 0, k, idx, cnt)
        out = empty_f32(1, cfg.d_model)
        for s in range(K):
            fr.ls_sparse_ffn_step(l, cur, 1, idx, cnt, s * k // K, (s + 1) * k // K, out)
        cur = out
    return host(cur)


@pytest.mark.parametrize("K", [1, 3, 8])
@pytest.mark.parametrize("mode", ["none", "oneshot"])
@pytest.mark.parametrize("coop", [1, 0])
def test_flags_events_and_host_sync_bitwise_equal(K, mode, coop):
    ws = [lsgen.layer_weights(CFG, l) for l in range(CFG.n_layers)]
    fr, _ = make_ffn(CFG, weights=ws)
    k = CFG.k
    m = {"none": lsffn.LS_PREFETCH_NONE, "oneshot": lsffn.LS_PREFETCH_ONESHOT}[mode]
    hosts = {}
    for sync in (lsffn.LS_SYNC_EVENTS, lsffn.LS_SYNC_FLAGS, lsffn.LS_SYNC_HOST):
        f = _host_ctx(CFG, ws, SLOTS)
        f.ls_configure(lsffn.LS_CFG_STREAM_SYNC, sync)
        f.ls_configure(lsffn.LS_CFG_COOPERATIVE, coop)
        hosts[sync] = f
    for t in range(2):
        x0 = lsgen.tokens(CFG, 30 + t, 1, 1)[0]
        ref = _replay_resident(fr, CFG, x0, k, K)
        got = {}
        for sync, f in hosts.items():
            x = dev_f32(x0)
            rep = f.ls_decode_step_streamed(x, k, K, m, k)
            f.ls_ffn_sync()
            got[sync] = host(x)
            assert rep.final_bytes == CFG.n_layers * k * _block_bytes(CFG)
        for sync in hosts:
            assert np.array_equal(got[sync], ref), (t, sync, K, mode, coop)
        f = hosts[lsffn.LS_SYNC_FLAGS]
        for l in range(CFG.n_layers):
            assert f.ls_debug_stages_done(l) == K, (t, l)


def test_flags_with_empty_stages_and_more_stages_than_blocks():
    """k = 2 blocks in 5 stages: three stages are empty and still signal done."""
    cfg = CFG.with_(n_layers=2, keep_pct=6)
    ws = [lsgen.layer_weights(cfg, l) for l in range(cfg.n_layers)]
    fr, _ = make_ffn(cfg, weights=ws)
    k = cfg.k
    assert k == 2
    f = _host_ctx(cfg, ws, 8)
    f.ls_configure(lsffn.LS_CFG_STREAM_SYNC, lsffn.LS_SYNC_FLAGS)
    x0 = lsgen.tokens(cfg, 4, 1, 1)[0]
    x = dev_f32(x0)
    f.ls_decode_step_streamed(x, k, 5, lsffn.LS_PREFETCH_NONE, k)
    f.ls_ffn_sync()
    assert np.array_equal(host(x), _replay_resident(fr, cfg, x0, k, 5))
    assert f.ls_debug_stages_done(0) == 5 and f.ls_debug_stages_done(1) == 5


def test_flags_refused_combinations():
    ws = [lsgen.layer_weights(CFG, l) for l in range(CFG.n_layers)]
    f = _host_ctx(CFG, ws, SLOTS)
    with pytest.raises(lsffn.LsError):
        f.ls_debug_stages_done(0)  # no flagged step yet
    f.ls_configure(lsffn.LS_CFG_STREAM_SYNC, lsffn.LS_SYNC_FLAGS)
    x = dev_f32(lsgen.tokens(CFG, 1, 1, 1)[0])
    with pytest.raises(lsffn.LsError):
        f.ls_decode_step_streamed(x, CFG.k, 4, lsffn.LS_PREFETCH_REFINE, CFG.k)
    with pytest.raises(lsffn.LsError):
        f.ls_decode_step_streamed(x, CFG.k, 65, lsffn.LS_PREFETCH_NONE, CFG.k)
    with pytest.raises(lsffn.LsError):
        f.ls_configure(lsffn.LS_CFG_STREAM_SYNC, 3)
    # the context still works after refused calls
    f.ls_decode_step_streamed(x, CFG.k, 2, lsffn.LS_PREFETCH_NONE, CFG.k)
    f.ls_ffn_sync()


def test_flags_full_size_70b_layers_and_oracle():
    """Two full-size 70B-shaped layers (d 8192, d_ff 28672, block 128, k 23 of 224) streamed
    from host memory in 8 stages: device flags equal events bitwise; the first layer's output
    against the oracle on the GPU's list."""
    cfg = lsgen.CONFIGS["llama2_70b_stream"].with_(n_layers=2)
    ws = [lsgen.layer_weights(cfg, l) for l in range(cfg.n_layers)]
    k = cfg.k
    outs = {}
    for sync in (lsffn.LS_SYNC_EVENTS, lsffn.LS_SYNC_FLAGS):
        f = _host_ctx(cfg, ws, 2 * k)
        f.ls_configure(lsffn.LS_CFG_STREAM_SYNC, sync)
        x0 = lsgen.tokens(cfg, 2, 1, 1)[0]
        x = dev_f32(x0)
        f.ls_decode_step_streamed(x, k, 8, lsffn.LS_PREFETCH_NONE, k)
        f.ls_ffn_sync()
        outs[sync] = host(x)
        if sync == lsffn.LS_SYNC_FLAGS:
            assert f.ls_debug_stages_done(0) == 8 and f.ls_debug_stages_done(1) == 8
            # layer 0 on its own: one flagged layer, then the oracle on the same list
            f1 = _host_ctx(cfg.with_(n_layers=1), ws[:1], k)
            f1.ls_configure(lsffn.LS_CFG_STREAM_SYNC, sync)
            x1 = dev_f32(x0)
            f1.ls_decode_step_streamed(x1, k, 8, lsffn.LS_PREFETCH_NONE, k)
            f1.ls_ffn_sync()
            scores = empty_f32(1, cfg.n_blk)
            idx, cnt = empty_i32(k), empty_i32(1)
            f1.ls_predict(0, dev_f32(x0), 1, scores)
            f1.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, k, 0.0, 0, k, idx, cnt)
            y_ref = oracle.sparse_ffn(ws[0], oracle.mlp_input(x0[0], cfg.prenorm), host(idx), cfg.block,
                                      cfg.act, ws[0].threshold)
            assert y_err(host(x1)[0].astype(np.float64) - x0[0], y_ref) <= Y_TOL[cfg.dtype]
    assert np.array_equal(outs[lsffn.LS_SYNC_EVENTS], outs[lsffn.LS_SYNC_FLAGS])


def test_flags_wait_timeout_fails_the_call_instead_of_hanging():
    """A 1 us wait limit against a cold cache: the first stage's copies cannot land in time, so
    the kernel's bounded arrival wait runs out, the kernel ends, and the call (or the sync)
    reports a device error; the context stays failed and can still be destroyed."""
    ws = [lsgen.layer_weights(CFG, l) for l in range(CFG.n_layers)]
    f = _host_ctx(CFG, ws, SLOTS)
    f.ls_configure(lsffn.LS_CFG_STREAM_SYNC, lsffn.LS_SYNC_FLAGS)
    with pytest.raises(lsffn.LsError):
        f.ls_configure(lsffn.LS_CFG_STAGE_WAIT_US, 0)
    f.ls_configure(lsffn.LS_CFG_STAGE_WAIT_US, 1)
    x = dev_f32(lsgen.tokens(CFG, 5, 1, 1)[0])
    with pytest.raises(lsffn.LsError) as err:
        f.ls_decode_step_streamed(x, CFG.k, 4, lsffn.LS_PREFETCH_NONE, CFG.k)
        f.ls_ffn_sync()
    assert "timed out" in str(err.value)
    with pytest.raises(lsffn.LsError):
        f.ls_ffn_sync()  # the failure is sticky
    f.close()
