"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Per step: scores (rel-L2 <= 1e-5), block ids (bit-exact on identical fp32
scores), FFN output y = x_out - x_in teacher-forced with the GPU's input and
block list (rel-L2 <= 1e-5 fp32, <= 2e-3 fp16/bf16).
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
from gpu_util import (DEV, SCORE_TOL, Y_TOL, dev_f32, empty_f32, empty_i32, host, make_ffn,  # noqa: E402
                      rel_l2, y_err)

C = lsgen.CONFIGS

# Shapes spanning several tiles with ragged tails, small enough for the oracle.
SMALL = {
    "c1": C["c1_reglu_512"],
    "f16_ragged": C["llama2_7b_ffn"].with_(n_layers=2, d_model=576, d_ff=1200, block=24, rank=192,
                                           keep_pct=30),
    "bf16_swiglu": C["mistral_7b_ffn"].with_(n_layers=2, d_model=512, d_ff=2048, block=128,
                                             rank=128, keep_pct=50),
    "f32_stack": C["c1_reglu_512"].with_(n_layers=3, prenorm=True, d_model=320, d_ff=960,
                                         block=40, rank=64),
    # 16-bit weights, block a multiple of 32: batches of 4+ run on the matrix cores
    "f16_b64": C["llama2_7b_ffn"].with_(n_layers=2, d_model=640, d_ff=1728, block=64, rank=192,
                                        keep_pct=30),
    # many small blocks and a narrow rank: the fp32 product P2 P1 (512 x 256) would be larger
    # than the two fp16 factors, so the library keeps P1 then P2
    "f16_factored": C["llama2_7b_ffn"].with_(n_layers=2, d_model=256, d_ff=4096, block=8, rank=64,
                                             keep_pct=5),
}


def _folded(cfg) -> bool:
    """Whether the library stores the predictor as the fp32 product P2 P1 (no larger than the
    two factors in their storage type)."""
    return 4 * cfg.n_blk * cfg.d_model <= cfg.elem_bytes * (cfg.rank * cfg.d_model + cfg.n_blk * cfg.rank)


GUARD = 1e-4  # |SiLU(g)| this close to the threshold may be decided either way


def _oracle_y(w, cfg, x, blocks):
    h = oracle.mlp_input(x, cfg.prenorm)
    return oracle.sparse_ffn(w, h, blocks, cfg.block, cfg.act, w.threshold)


def _check_y(f, ws_l, cfg, xin, yg, blocks, tol, tag):
    """y of every token against the oracle.  SwiGLU-threshold: the GPU's keep/drop decisions
    (from its activation dump) must equal the oracle's outside a guard band around the
    threshold; the oracle then recomputes y with the GPU's decisions."""
    B = xin.shape[0]
    neurons = oracle.neurons_of_blocks(blocks, cfg.block)
    a_gpu = None
    if cfg.act == lsgen.ACT_SWIGLU_THRESH:
        buf = empty_f32(B * max(1, cfg.d_ff))
        n = f.ls_debug_last_activations(buf)
        a_gpu = host(buf)[:B * n].reshape(B, n)[:, :len(neurons)]
    for b in range(B):
        if a_gpu is None:
            y_ref = _oracle_y(ws_l, cfg, xin[b], blocks)
        else:
            h = oracle.mlp_input(xin[b], cfg.prenorm)
            g, _, a_t = oracle.activations(ws_l, h, neurons, cfg.act, ws_l.threshold)
            _, _, a_all = oracle.activations(ws_l, h, neurons, cfg.act, -1.0)
            sig = np.abs(g / (1.0 + np.exp(-g)))
            keep_gpu = a_gpu[b] != 0
            keep_ref = a_t != 0
            flips = keep_gpu != keep_ref
            assert np.all(np.abs(sig[flips] - ws_l.threshold) <= GUARD), (tag, b, int(flips.sum()))
            y_ref = oracle.down(ws_l, neurons, np.where(keep_gpu, a_all, 0.0))
        assert y_err(yg[b], y_ref) <= tol, (tag, b, y_err(yg[b], y_ref))


@pytest.mark.parametrize("B", [1, 4, 7, 8])
@pytest.mark.parametrize("name", list(SMALL))
def test_predict_parity(name, B):
    """Batches of 4+ compute four predictor rows per workgroup; the shapes include row counts
    that are not a multiple of four (50 and 27 blocks) and both the folded form (P2 P1 in fp32)
    and the factored one (P1, then P2: f16_factored)."""
    cfg = SMALL[name]
    assert _folded(cfg) == (name != "f16_factored")
    f, ws = make_ffn(cfg, max_batch=B)
    xs = lsgen.tokens(cfg, 0, 1, B)[0]
    scores = empty_f32(B, cfg.n_blk)
    for l in range(cfg.n_layers):
        f.ls_predict(l, dev_f32(xs), B, scores)
        got = host(scores)
        for b in range(B):
            ref = oracle.predict(ws[l].p1, ws[l].p2, oracle.mlp_input(xs[b], cfg.prenorm))
            assert rel_l2(got[b], ref) <= SCORE_TOL, (name, l, b)


@pytest.mark.parametrize("B", [1, 2, 3, 8])
@pytest.mark.parametrize("kind", ["normal", "ties", "zeros", "special"])
@pytest.mark.parametrize("n_blk", [1, 48, 172, 224, 2048])
def test_select_bit_exact(B, kind, n_blk):
    cfg = C["c1_reglu_512"].with_(d_ff=8 * n_blk, block=8, d_model=64, rank=64)
    f, _ = make_ffn(cfg, max_batch=8)
    rng = np.random.default_rng(1000 * B + n_blk)
    S = lsgen.adversarial_scores(rng, B, n_blk, kind)
    s_dev = dev_f32(S)
    for k in sorted({1, max(1, n_blk // 7), n_blk}):
        for uni in ([0, 1] if B > 1 else [0]):
            cap = min(n_blk, B * k) if uni else k
            idx = empty_i32(cap if uni else B * cap)
            cnt = empty_i32(1 if uni else B)
            f.ls_select_blocks(s_dev, B, lsffn.LS_SEL_TOPK, k, 0.0, uni, cap, idx, cnt)
            ref_idx, ref_cnt = oracle.select(S, k=k, union_batch=bool(uni), cap=cap)
            gi, gc = host(idx), host(cnt)
            assert np.array_equal(gc, ref_cnt)
            if uni:
                assert np.array_equal(gi[:gc[0]], ref_idx[:ref_cnt[0]])
            else:
                gi = gi.reshape(B, cap)
                for b in range(B):
                    assert np.array_equal(gi[b, :gc[b]], ref_idx[b, :ref_cnt[b]])
    for tau in (0.0, -0.5, 1.0):
        for uni in ([0, 1] if B > 1 else [0]):
            idx = empty_i32(n_blk if uni else B * n_blk)
            cnt = empty_i32(1 if uni else B)
            f.ls_select_blocks(s_dev, B, lsffn.LS_SEL_THRESHOLD, 1, tau, uni, n_blk, idx, cnt)
            ref_idx, ref_cnt = oracle.select(S, mode=oracle.SEL_THRESHOLD, tau=tau,
                                             union_batch=bool(uni), cap=n_blk)
            gi, gc = host(idx), host(cnt)
            assert np.array_equal(gc, ref_cnt)
            if uni:
                assert np.array_equal(gi[:gc[0]], ref_idx[:ref_cnt[0]])
            else:
                gi = gi.reshape(B, n_blk)
                for b in range(B):
                    assert np.array_equal(gi[b, :gc[b]], ref_idx[b, :ref_cnt[b]])


@pytest.mark.parametrize("name", list(SMALL))
@pytest.mark.parametrize("B", [1, 3, 4, 8])
def test_sparse_step_teacher_forced(name, B):
    cfg = SMALL[name]
    f, ws = make_ffn(cfg, max_batch=B)
    tol = Y_TOL[cfg.dtype]
    xs = lsgen.tokens(cfg, 5, 1, B)[0]
    x_in = dev_f32(xs)
    scores = empty_f32(B, cfg.n_blk)
    cap = min(cfg.n_blk, B * cfg.k)
    idx, cnt = empty_i32(cap), empty_i32(1)
    x_out = empty_f32(B, cfg.d_model)
    for l in range(cfg.n_layers):
        f.ls_predict(l, x_in, B, scores)
        f.ls_select_blocks(scores, B, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 1, cap, idx, cnt)
        f.ls_sparse_ffn_step(l, x_in, B, idx, cnt, 0, cap, x_out)
        gi, gc = host(idx), host(cnt)
        blocks = gi[:gc[0]]
        # the GPU's block list is the oracle's selection on the GPU's scores
        ref_idx, ref_cnt = oracle.select(host(scores), k=cfg.k, union_batch=True, cap=cap)
        assert np.array_equal(blocks, (ref_idx if B > 1 else ref_idx[0])[:gc[0]])
        xin_h, xout_h = host(x_in), host(x_out)
        yg = xout_h.astype(np.float64) - xin_h.astype(np.float64)
        _check_y(f, ws[l], cfg, xin_h, yg, blocks, tol, (name, l))
        x_in, x_out = x_out, x_in


@pytest.mark.parametrize("name", ["c1", "f16_ragged", "f32_stack"])
def test_stages_eq1_eq2(name):
    """Stages over the priority list: x_acc after the last stage equals the single-shot output
    (Eq. 1-2); each intermediate x_acc matches the oracle's refined feature x_tilde^(j)."""
    cfg = SMALL[name]
    f, ws = make_ffn(cfg, n_layers=1)
    tol = Y_TOL[cfg.dtype]
    x = lsgen.tokens(cfg, 7, 1, 1)[0]
    x_in = dev_f32(x)
    scores = empty_f32(1, cfg.n_blk)
    k = max(cfg.k, 5)
    idx, cnt = empty_i32(k), empty_i32(1)
    f.ls_predict(0, x_in, 1, scores)
    f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, k, 0.0, 0, k, idx, cnt)
    blocks = host(idx)[:k]
    single = empty_f32(1, cfg.d_model)
    f.ls_sparse_ffn_step(0, x_in, 1, idx, cnt, 0, k, single)
    for K in (2, 3, k):
        acc = empty_f32(1, cfg.d_model)
        h = oracle.mlp_input(x[0], cfg.prenorm)
        _, xt = oracle.staged_ffn(ws[0], x[0], h, blocks, cfg.block, K, cfg.act, ws[0].threshold)
        for j, (lo, hi) in enumerate(oracle.stage_bounds(k, K)):
            f.ls_sparse_ffn_step(0, x_in, 1, idx, cnt, lo, hi, acc)
            got = host(acc)[0].astype(np.float64)
            assert y_err(got - x[0], xt[j] - x[0]) <= tol, (K, j)
        assert y_err(host(acc)[0] - x[0], host(single)[0] - x[0]) <= tol


@pytest.mark.parametrize("name", ["c1", "f16_ragged"])
def test_permutation_invariance(name):
    cfg = SMALL[name]
    f, ws = make_ffn(cfg, n_layers=1)
    tol = Y_TOL[cfg.dtype]
    x = lsgen.tokens(cfg, 9, 1, 1)[0]
    x_in = dev_f32(x)
    rng = np.random.default_rng(2)
    blocks = rng.choice(cfg.n_blk, size=min(cfg.n_blk, 11), replace=False).astype(np.int32)
    outs = []
    for perm in range(3):
        order = blocks if perm == 0 else rng.permutation(blocks)
        out = empty_f32(1, cfg.d_model)
        f.ls_sparse_ffn_step(0, x_in, 1, dev_f32(order).int(), dev_f32([len(order)]).int(), 0,
                             len(order), out)
        outs.append(host(out)[0].astype(np.float64) - x[0])
    y_ref = _oracle_y(ws[0], cfg, x[0], blocks)
    for y in outs:
        assert y_err(y, y_ref) <= tol
        assert y_err(y, outs[0]) <= tol


def test_relu_dead_blocks_exact_zero():
    cfg = SMALL["f16_ragged"].with_(n_layers=1)
    w = lsgen.layer_weights(cfg, 0)
    dead = [2, 5, 11]
    b = w.bias.copy()
    for blk in dead:
        b[blk * cfg.block:(blk + 1) * cfg.block] = np.float16(-1e4)
    w.bias = b
    f, _ = make_ffn(cfg, n_layers=1, weights=[w])
    x = lsgen.tokens(cfg, 3, 1, 1)[0]
    x_in = dev_f32(x)
    live = [0, 3, 7]
    order = np.array([0, 2, 3, 5, 7, 11], np.int32)
    out = empty_f32(1, cfg.d_model)
    f.ls_sparse_ffn_step(0, x_in, 1, dev_f32(order).int(), dev_f32([6]).int(), 0, 6, out)
    a = empty_f32(6 * cfg.block)
    n = f.ls_debug_last_activations(a)
    assert n == 6 * cfg.block
    a = host(a).reshape(6, cfg.block)
    for pos, blk in enumerate(order):
        if blk in dead:
            assert np.all(a[pos] == 0.0)
    y = host(out)[0].astype(np.float64) - x[0]
    y_ref = _oracle_y(w, cfg, x[0], live)
    assert y_err(y, y_ref) <= Y_TOL[cfg.dtype]


def test_empty_and_clamped_ranges():
    cfg = SMALL["c1"]
    f, ws = make_ffn(cfg)
    x = lsgen.tokens(cfg, 1, 1, 1)[0]
    x_in = dev_f32(x)
    idx = dev_f32([3, 1, 4, 1, 5]).int()
    cnt = dev_f32([3]).int()
    out = empty_f32(1, cfg.d_model)
    f.ls_sparse_ffn_step(0, x_in, 1, idx, cnt, 0, 0, out)   # empty: x_acc = x_in
    assert np.array_equal(host(out)[0], x[0])
    f.ls_sparse_ffn_step(0, x_in, 1, idx, cnt, 0, 5, out)   # clamped to count = 3
    y = host(out)[0].astype(np.float64) - x[0]
    assert y_err(y, _oracle_y(ws[0], cfg, x[0], [3, 1, 4])) <= Y_TOL[cfg.dtype]
    zero = dev_f32([0]).int()
    f.ls_sparse_ffn_step(0, x_in, 1, idx, zero, 0, 5, out)  # count 0
    assert np.array_equal(host(out)[0], x[0])


def test_decode_step_equals_composition_and_is_deterministic():
    cfg = SMALL["f16_ragged"].with_(n_layers=3)
    for B in (1, 4):
        f, ws = make_ffn(cfg, max_batch=B)
        x0 = lsgen.tokens(cfg, 11, 1, B)[0]
        xd = dev_f32(x0)
        f.ls_decode_step(xd, B, cfg.k)
        got = host(xd)
        xd2 = dev_f32(x0)
        f.ls_decode_step(xd2, B, cfg.k)
        assert np.array_equal(host(xd2), got)
        # composition of the per-layer calls, teacher-forced oracle check at every layer
        cap = min(cfg.n_blk, B * cfg.k)
        x_in = dev_f32(x0)
        x_out = empty_f32(B, cfg.d_model)
        scores = empty_f32(B, cfg.n_blk)
        idx, cnt = empty_i32(cap), empty_i32(1)
        for l in range(cfg.n_layers):
            f.ls_predict(l, x_in, B, scores)
            f.ls_select_blocks(scores, B, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 1, cap, idx, cnt)
            f.ls_sparse_ffn_step(l, x_in, B, idx, cnt, 0, cap, x_out)
            blocks = host(idx)[:host(cnt)[0]]
            xi, xo = host(x_in), host(x_out)
            _check_y(f, ws[l], cfg, xi, xo.astype(np.float64) - xi, blocks, Y_TOL[cfg.dtype], l)
            x_in, x_out = x_out, x_in
        assert y_err(host(x_in) - x0, got - x0) <= Y_TOL[cfg.dtype]


def test_invalid_arguments_return_codes():
    cfg = SMALL["c1"]
    f, _ = make_ffn(cfg, max_batch=2)
    x = empty_f32(2, cfg.d_model)
    s = empty_f32(2, cfg.n_blk)
    idx, cnt = empty_i32(cfg.n_blk), empty_i32(2)
    bad = [
        lambda: f.ls_predict(1, x, 1, s),                      # layer out of range
        lambda: f.ls_predict(0, x, 3, s),                      # B > max_batch
        lambda: f.ls_predict(0, None, 1, s),                   # null
        lambda: f.ls_select_blocks(s, 1, 0, 0, 0.0, 0, 5, idx, cnt),           # k = 0
        lambda: f.ls_select_blocks(s, 1, 0, cfg.n_blk + 1, 0.0, 0, 99, idx, cnt),
        lambda: f.ls_select_blocks(s, 1, 0, 5, 0.0, 0, 4, idx, cnt),           # cap < k
        lambda: f.ls_select_blocks(s, 2, 0, 30, 0.0, 1, 47, idx, cnt),         # union cap
        lambda: f.ls_select_blocks(s, 1, 1, 1, 0.0, 0, 10, idx, cnt),          # threshold cap
        lambda: f.ls_sparse_ffn_step(0, x, 1, idx, cnt, 0, 3, x),              # aliasing
        lambda: f.ls_sparse_ffn_step(0, x, 1, idx, cnt, 4, 3, s),              # begin > end
        lambda: f.ls_decode_step(x, 1, 0),
    ]
    for i, call in enumerate(bad):
        with pytest.raises(lsffn.LsError) as e:
            call()
        assert e.value.status == lsffn.LS_E_INVAL, i
    g = lsffn.Ffn(n_layers=2, d_model=64, d_ff=64, block=8, rank=64, dtype=lsffn.LS_F32)
    with pytest.raises(lsffn.LsError) as e:
        g.ls_predict(1, x, 1, s)                                # layer never set
    assert e.value.status == lsffn.LS_E_STATE
    with pytest.raises(lsffn.LsError) as e:
        lsffn.Ffn(n_layers=1, d_model=100, d_ff=64, block=8, rank=64)
    assert e.value.status == lsffn.LS_E_INVAL


WIDE = {
    "llama2_7b_2l": C["llama2_7b_ffn"].with_(n_layers=2),
    "llama2_13b_2l": C["llama2_13b_ffn"].with_(n_layers=2),
    # 300 blocks: the selection inside the gate/up launch takes its 8-keys-per-lane form
    "f16_nb300": C["llama2_7b_ffn"].with_(n_layers=2, d_model=512, d_ff=4800, block=16, rank=64, keep_pct=10),
}


@pytest.mark.parametrize("name", ["f16_b64", "bf16_swiglu", "f32_stack", "llama2_7b_2l", "llama2_13b_2l", "f16_nb300"])
def test_decode_step_per_kernel_equals_entry_points(name):
    """ls_decode_step on the per-kernel path at B = 1, where the selection runs inside the
    gate/up launch, gives the same bits as ls_predict, ls_select_blocks and
    ls_sparse_ffn_step called layer by layer."""
    cfg = SMALL[name] if name in SMALL else WIDE[name]
    f, ws = make_ffn(cfg)
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, 1)
    for t in range(2):
        x0 = lsgen.tokens(cfg, 21 + t, 1, 1)[0]
        x = dev_f32(x0)
        f.ls_decode_step(x, 1, cfg.k)
        got = host(x)
        xin, xout = dev_f32(x0), empty_f32(1, cfg.d_model)
        scores = empty_f32(1, cfg.n_blk)
        idx, cnt = empty_i32(cfg.k), empty_i32(1)
        for l in range(cfg.n_layers):
            f.ls_predict(l, xin, 1, scores)
            f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 0, cfg.k, idx, cnt)
            f.ls_sparse_ffn_step(l, xin, 1, idx, cnt, 0, cfg.k, xout)
            xin, xout = xout, xin
        assert np.array_equal(got, host(xin)), (name, t)
    f.ls_ffn_sync()


@pytest.mark.parametrize("cfg_name", ["llama2_13b_ffn", "mistral_7b_ffn"])
def test_every_block_selected_equals_dense(cfg_name):
    """One full-size layer with every block in the list at B = 1: the activations no longer fit
    the down kernel's LDS copy (13B shape: 216 x 64 floats), so it reads them from memory; with
    d = 5120 it also runs two workgroups per CU.  The result is the dense FFN (oracle)."""
    cfg = C[cfg_name].with_(n_layers=1)
    f, ws = make_ffn(cfg)
    x = lsgen.tokens(cfg, 3, 1, 1)[0]
    x_in = dev_f32(x)
    x_out = empty_f32(1, cfg.d_model)
    idx = torch.arange(cfg.n_blk, dtype=torch.int32, device=DEV)
    cnt = torch.full((1,), cfg.n_blk, dtype=torch.int32, device=DEV)
    f.ls_sparse_ffn_step(0, x_in, 1, idx, cnt, 0, cfg.n_blk, x_out)
    y = host(x_out).astype(np.float64) - x.astype(np.float64)
    _check_y(f, ws[0], cfg, x, y, np.arange(cfg.n_blk), Y_TOL[cfg.dtype], cfg_name)
    f.ls_ffn_sync()


@pytest.mark.parametrize("cfg_name", ["llama2_7b_ffn", "llama2_13b_ffn", "mistral_7b_ffn"])
def test_full_size_layers_sampled(cfg_name):
    """Full-size layer shapes (2 layers of each stack), B=1, teacher-forced per layer."""
    cfg = C[cfg_name].with_(n_layers=2)
    f, ws = make_ffn(cfg)
    x = lsgen.tokens(cfg, 0, 1, 1)[0]
    x_in = dev_f32(x)
    x_out = empty_f32(1, cfg.d_model)
    scores = empty_f32(1, cfg.n_blk)
    idx, cnt = empty_i32(cfg.k), empty_i32(1)
    for l in range(cfg.n_layers):
        f.ls_predict(l, x_in, 1, scores)
        xi = host(x_in)[0]
        ref_s = oracle.predict(ws[l].p1, ws[l].p2, oracle.mlp_input(xi, cfg.prenorm))
        assert rel_l2(host(scores)[0], ref_s) <= SCORE_TOL
        f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 0, cfg.k, idx, cnt)
        blocks = host(idx)
        ref_idx, _ = oracle.select(host(scores), k=cfg.k, cap=cfg.k)
        assert np.array_equal(blocks, ref_idx[0])
        f.ls_sparse_ffn_step(l, x_in, 1, idx, cnt, 0, cfg.k, x_out)
        y = host(x_out).astype(np.float64) - xi[None, :]
        _check_y(f, ws[l], cfg, xi[None, :], y, blocks, Y_TOL[cfg.dtype], (cfg_name, l))
        x_in, x_out = x_out, x_in


def test_mistral_full_width_batch4_matrix_cores():
    """Two full Mistral-7B-shaped layers (d 4096, d_ff 14336, bf16, thresholded SiLU, 128-neuron
    blocks, k = 56) at B = 4 on the matrix-core kernels (the union list, eight 512-value chunks
    per row, bf16 hi + lo activations), teacher-forced per layer against the oracle with the
    threshold guard band."""
    cfg = C["mistral_7b_ffn"].with_(n_layers=2)
    B = 4
    f, ws = make_ffn(cfg, max_batch=B)
    f.ls_configure(lsffn.LS_CFG_BATCH_MFMA, 1)
    xs = lsgen.tokens(cfg, 13, 1, B)[0]
    x_in = dev_f32(xs)
    x_out = empty_f32(B, cfg.d_model)
    scores = empty_f32(B, cfg.n_blk)
    cap = min(cfg.n_blk, B * cfg.k)
    idx, cnt = empty_i32(cap), empty_i32(1)
    for l in range(cfg.n_layers):
        f.ls_predict(l, x_in, B, scores)
        f.ls_select_blocks(scores, B, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 1, cap, idx, cnt)
        f.ls_sparse_ffn_step(l, x_in, B, idx, cnt, 0, cap, x_out)
        xi, xo, sc = host(x_in), host(x_out), host(scores)
        for b in range(B):
            ref_s = oracle.predict(ws[l].p1, ws[l].p2, oracle.mlp_input(xi[b], cfg.prenorm))
            assert rel_l2(sc[b], ref_s) <= SCORE_TOL, (l, b)
        blocks = host(idx)[:host(cnt)[0]]
        ref_idx, ref_cnt = oracle.select(sc, k=cfg.k, union_batch=True, cap=cap)
        assert np.array_equal(blocks, ref_idx[:ref_cnt[0]])
        assert blocks.size > cfg.k       # a real union of four lists
        _check_y(f, ws[l], cfg, xi, xo.astype(np.float64) - xi, blocks, Y_TOL[cfg.dtype], l)
        x_in, x_out = x_out, x_in


# ReGLU shapes: with thresholded SiLU, two fp32-accurate paths may decide neurons within
# rounding of the threshold differently (the oracle tests cover that with a guard band).
MFMA_CMP = {
    "f16_b64": SMALL["f16_b64"],
    "bf16_reglu": C["mistral_7b_ffn"].with_(n_layers=1, d_model=512, d_ff=2048, block=128, rank=128,
                                            keep_pct=50, act=lsgen.ACT_REGLU),
    # 256 column tiles: below B = 8 the down projection runs unsplit with 16-column tiles, at
    # B = 8 with 32-column tiles and the list in 2 parts (the two above: 32-column tiles, 8 parts)
    "f16_d4096": C["llama2_7b_ffn"].with_(n_layers=1, d_model=4096, d_ff=2048, block=64, rank=128,
                                          keep_pct=30),
}


@pytest.mark.parametrize("name", list(MFMA_CMP))
@pytest.mark.parametrize("B", [4, 6, 8])
def test_batch_matrix_core_path_matches_vector_path(name, B):
    """The matrix-core kernels (B >= 4) against the vector-ALU kernels on the same union list:
    both accumulate in fp32, the activations enter the matrix cores as hi + lo 16-bit parts
    (about 22 significant bits for fp16 operands, 16 for bf16)."""
    cfg = MFMA_CMP[name]
    f, ws = make_ffn(cfg, max_batch=B)
    xs = lsgen.tokens(cfg, 11, 1, B)[0]
    x_in = dev_f32(xs)
    scores = empty_f32(B, cfg.n_blk)
    cap = min(cfg.n_blk, B * cfg.k)
    idx, cnt = empty_i32(cap), empty_i32(1)
    f.ls_predict(0, x_in, B, scores)
    f.ls_select_blocks(scores, B, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 1, cap, idx, cnt)
    ys = []
    for mfma in (1, 0):
        f.ls_configure(lsffn.LS_CFG_BATCH_MFMA, mfma)
        x_out = empty_f32(B, cfg.d_model)
        f.ls_sparse_ffn_step(0, x_in, B, idx, cnt, 0, cap, x_out)
        ys.append(host(x_out).astype(np.float64) - xs.astype(np.float64))
    # the same list in three ranges: the first range adds the residual, the others accumulate
    n = int(host(cnt)[0])
    cuts = [0, n // 3, (2 * n) // 3, cap]
    for mfma in (1, 0):
        f.ls_configure(lsffn.LS_CFG_BATCH_MFMA, mfma)
        x_out = empty_f32(B, cfg.d_model)
        for r in range(3):
            f.ls_sparse_ffn_step(0, x_in, B, idx, cnt, cuts[r], cuts[r + 1], x_out)
        ys.append(host(x_out).astype(np.float64) - xs.astype(np.float64))
    tol = 1e-5 if cfg.dtype == lsgen.DT_F16 else 1e-4
    for b in range(B):
        for y in ys[1:]:
            assert y_err(ys[0][b], y[b]) <= tol, (name, B, b, y_err(ys[0][b], y[b]))
    with pytest.raises(lsffn.LsError):
        f.ls_configure(lsffn.LS_CFG_BATCH_MFMA, 2)


def test_kernel_timing_mask():
    """ls_set_kernel_timing with a kernel-id mask brackets only those kernels' launches; the
    default brackets every launch; a mask of only the prenorm id (which launches nothing) is
    refused by the binding."""
    cfg = SMALL["f16_b64"]
    f, _ = make_ffn(cfg, max_batch=4)
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, 1)
    xs = lsgen.tokens(cfg, 2, 2, 4)
    launched = (lsffn.LS_K_PRED_P1, lsffn.LS_K_SELECT, lsffn.LS_K_GATEUP, lsffn.LS_K_DOWN)
    f.ls_set_kernel_timing(True, kernels=[lsffn.LS_K_GATEUP])
    f.ls_kernel_timing(0, reset=True)
    f.ls_decode_step(dev_f32(xs[0]), 4, cfg.k)
    ms, n = f.ls_kernel_timing(lsffn.LS_K_GATEUP)
    assert n == cfg.n_layers and ms > 0
    for kid in launched:
        if kid != lsffn.LS_K_GATEUP:
            assert f.ls_kernel_timing(kid)[1] == 0, kid
    f.ls_set_kernel_timing(True)
    f.ls_kernel_timing(0, reset=True)
    f.ls_decode_step(dev_f32(xs[1]), 4, cfg.k)
    for kid in launched:
        assert f.ls_kernel_timing(kid)[1] == cfg.n_layers, kid
    f.ls_set_kernel_timing(False)
    with pytest.raises(ValueError):
        f.ls_set_kernel_timing(True, kernels=[lsffn.LS_K_PRENORM])
