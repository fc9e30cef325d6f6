"""GPU parity of the fused decode-step kernel (one persistent launch per token).

Teacher-forced per layer against the CPU oracle, using the per-layer inputs and
scores the fused kernel exchanged (read back through ls_debug_decode_trace):
scores rel-L2 <= 1e-5; block list = the oracle's selection on those scores;
y_l = x_{l+1} - x_l within 1e-5 (fp32) / 2e-3 (fp16, bf16) of the oracle.
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
from gpu_util import SCORE_TOL, Y_TOL, dev_f32, empty_f32, host, make_ffn, rel_l2, y_err  # noqa: E402

C = lsgen.CONFIGS

FUSED = {
    "c1": C["c1_reglu_512"],
    "f32_stack": C["c1_reglu_512"].with_(n_layers=3, prenorm=True),
    "f16_d1024": C["llama2_7b_ffn"].with_(n_layers=3, d_model=1024, d_ff=2816, block=32, rank=256),
    "llama2_7b_4l": C["llama2_7b_ffn"].with_(n_layers=4),
    "bf16_swiglu_d4096": C["mistral_7b_ffn"].with_(n_layers=3, d_ff=8192, block=64, keep_pct=12),
}


def _fused_ffn(cfg, n_layers=None):
    f, ws = make_ffn(cfg, n_layers=n_layers)
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, 2)  # fused kernel only
    return f, ws


def _check_layers(f, ws, cfg, x0, x_final):
    L = len(ws)
    scores = empty_f32(cfg.n_blk)
    xin = empty_f32(cfg.d_model)
    x_l = x0.astype(np.float32)
    for l in range(L):
        if l > 0:
            f.ls_debug_decode_trace(l, x_in=xin)
            x_l = host(xin).copy()
        f.ls_debug_decode_trace(l, scores=scores)
        s_gpu = host(scores).copy()
        s_ref = oracle.predict(ws[l].p1, ws[l].p2, oracle.mlp_input(x_l, cfg.prenorm))
        assert rel_l2(s_gpu, s_ref) <= SCORE_TOL, (l, rel_l2(s_gpu, s_ref))
        idx, _ = oracle.select(s_gpu, k=cfg.k, cap=cfg.k)
        blocks = idx[0]
        if l + 1 < L:
            f.ls_debug_decode_trace(l + 1, x_in=xin)
            x_next = host(xin).copy()
        else:
            x_next = x_final
        y_gpu = x_next.astype(np.float64) - x_l.astype(np.float64)
        h = oracle.mlp_input(x_l, cfg.prenorm)
        y_ref = oracle.sparse_ffn(ws[l], h, blocks, cfg.block, cfg.act, ws[l].threshold)
        assert y_err(y_gpu, y_ref) <= Y_TOL[cfg.dtype], (l, y_err(y_gpu, y_ref))


@pytest.mark.parametrize("name", list(FUSED))
def test_fused_teacher_forced_per_layer(name):
    cfg = FUSED[name]
    f, ws = _fused_ffn(cfg)
    for t in range(2):  # two launches: the epoch tags advance between them
        x0 = lsgen.tokens(cfg, t, 1, 1)[0, 0]
        x = dev_f32(x0[None, :])
        f.ls_decode_step(x, 1, cfg.k)
        f.ls_ffn_sync()
        _check_layers(f, ws, cfg, x0, host(x)[0].copy())


@pytest.mark.parametrize("name", ["c1", "f16_d1024", "llama2_7b_4l"])
def test_fused_matches_per_kernel_path_and_is_deterministic(name):
    cfg = FUSED[name]
    f, ws = _fused_ffn(cfg)
    xs = lsgen.tokens(cfg, 3, 4, 1)
    outs = []
    for rep in range(2):
        o = []
        for t in range(4):
            x = dev_f32(xs[t])
            f.ls_decode_step(x, 1, cfg.k)
            o.append(host(x)[0].copy())
        outs.append(np.stack(o))
    f.ls_ffn_sync()
    assert np.array_equal(outs[0], outs[1])  # bitwise reproducible
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, 1)
    for t in range(4):
        x = dev_f32(xs[t])
        f.ls_decode_step(x, 1, cfg.k)
        ref = host(x)[0]
        y_f = outs[0][t].astype(np.float64) - xs[t, 0]
        y_k = ref.astype(np.float64) - xs[t, 0]
        assert y_err(y_f, y_k) <= Y_TOL[cfg.dtype]


def test_fused_speculative_width_does_not_change_results():
    cfg = FUSED["llama2_7b_4l"]
    f, ws = _fused_ffn(cfg)
    x0 = lsgen.tokens(cfg, 9, 1, 1)[0]
    res = []
    for kp in (cfg.k, cfg.k + 1, 0):  # no spare slots, one spare, automatic
        f.ls_configure(lsffn.LS_CFG_SPEC_BLOCKS, kp)
        x = dev_f32(x0)
        f.ls_decode_step(x, 1, cfg.k)
        res.append(host(x)[0].astype(np.float64) - x0[0])
    f.ls_ffn_sync()
    for r in res[1:]:
        assert y_err(r, res[0]) <= Y_TOL[cfg.dtype]


def test_fused_width_changes_between_launches():
    """Launches alternate between two halves of the bare-word exchange rows, each launch emptying
    the other half for the next one; widening or narrowing the speculative list between launches
    must not expose words of an older launch.  Every launch is checked against the per-kernel
    path on the same token."""
    cfg = FUSED["llama2_7b_4l"]
    f, ws = _fused_ffn(cfg)
    widths = (cfg.k + 6, cfg.k, cfg.k + 3, 0, cfg.k + 1, cfg.k + 6, cfg.k)
    xs = lsgen.tokens(cfg, 21, len(widths), 1)
    fused = []
    for t, kp in enumerate(widths):
        f.ls_configure(lsffn.LS_CFG_SPEC_BLOCKS, kp)
        x = dev_f32(xs[t])
        f.ls_decode_step(x, 1, cfg.k)
        fused.append(host(x)[0].astype(np.float64) - xs[t, 0])
    f.ls_ffn_sync()
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, 1)
    for t in range(len(widths)):
        x = dev_f32(xs[t])
        f.ls_decode_step(x, 1, cfg.k)
        ref = host(x)[0].astype(np.float64) - xs[t, 0]
        assert y_err(fused[t], ref) <= Y_TOL[cfg.dtype], (t, widths[t], y_err(fused[t], ref))


def test_fused_unsupported_shape_reports_and_auto_falls_back():
    cfg = C["llama2_7b_ffn"].with_(n_layers=2, d_model=576, d_ff=1200, block=24, rank=192)
    f, _ = make_ffn(cfg)
    x = dev_f32(lsgen.tokens(cfg, 0, 1, 1)[0])
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, 2)
    with pytest.raises(lsffn.LsError) as e:
        f.ls_decode_step(x, 1, cfg.k)
    assert e.value.status == lsffn.LS_E_UNSUPPORTED
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, 0)
    f.ls_decode_step(x, 1, cfg.k)  # per-kernel path
    f.ls_ffn_sync()
    with pytest.raises(lsffn.LsError) as e:
        f.ls_debug_decode_trace(1, scores=empty_f32(cfg.n_blk))
    assert e.value.status == lsffn.LS_E_STATE


def test_plain_launch_matches_cooperative_bitwise():
    cfg = FUSED["llama2_7b_4l"]
    f, ws = _fused_ffn(cfg)
    xs = lsgen.tokens(cfg, 5, 3, 1)
    outs = []
    for coop in (1, 0):
        f.ls_configure(lsffn.LS_CFG_COOPERATIVE, coop)
        o = []
        for t in range(3):
            x = dev_f32(xs[t])
            f.ls_decode_step(x, 1, cfg.k)
            o.append(host(x)[0].copy())
        f.ls_ffn_sync()
        outs.append(np.stack(o))
    assert np.array_equal(outs[0], outs[1])
    with pytest.raises(lsffn.LsError) as e:
        f.ls_configure(lsffn.LS_CFG_COOPERATIVE, 2)
    assert e.value.status == lsffn.LS_E_INVAL


def test_fused_headline_stack_all_layers_plain_launch():
    """The full Llama-2-7B-shaped stack (32 layers, d 4096, d_ff 11008, fp16, k = 21 of 172) in
    the benchmark's configuration (plain launch of the persistent grid, default speculative
    width), two fresh tokens, every layer teacher-forced against the oracle."""
    cfg = C["llama2_7b_ffn"]
    f, ws = _fused_ffn(cfg)
    f.ls_configure(lsffn.LS_CFG_COOPERATIVE, 0)
    f.ls_configure(lsffn.LS_CFG_SPEC_BLOCKS, 0)
    for t in range(2):
        x0 = lsgen.tokens(cfg, 40 + t, 1, 1)[0, 0]
        x = dev_f32(x0[None, :])
        f.ls_decode_step(x, 1, cfg.k)
        f.ls_ffn_sync()
        _check_layers(f, ws, cfg, x0, host(x)[0].copy())
