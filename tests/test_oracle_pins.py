"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: hand-derived
values (tests/golden/tiny_ffn.json), closed forms, float64 library routines on
the same exactly-decoded weights, brute force on tiny inputs, and invariants
that the paper states (Eq. 1-2 staging, Sec. 3.2.2 permutation invariance).
"""
import itertools
import json
import math
import os
from types import SimpleNamespace

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import lsgen
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def _small_layer(d=96, F=256, blk=16, r=24, dtype=lsgen.DT_F32, bias=-0.3, seed=7, layer=0):
    cfg = lsgen.Config("t", 1, d, F, dtype, lsgen.ACT_REGLU, blk, r, 25, bias, True, 1, seed=seed)
    return cfg, lsgen.layer_weights(cfg, layer)


def _dec(a):
    return lsgen.decode_bits(a, oracle.storage_code(a))


# ----------------------------------------------------------------------------- decoding

def test_decode_f16_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(bits.view(np.float16))
    ref = bits.view(np.float16).astype(np.float64)  # numpy's own binary16 widening
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_decode_bf16_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(bits)
    ref = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


# ----------------------------------------------------------------------------- golden example

def _golden():
    with open(os.path.join(GOLDEN, "tiny_ffn.json")) as f:
        g = json.load(f)
    w = SimpleNamespace(gate=np.array(g["w_gate"], np.float32), up=np.array(g["w_up"], np.float32),
                        down=np.array(g["w_down"], np.float32),
                        bias=np.array(g["b_gate"], np.float32),
                        p1=np.array(g["p1"], np.float32), p2=np.array(g["p2"], np.float32))
    return g, w


def test_golden_reglu_by_hand():
    g, w = _golden()
    h = oracle.mlp_input(np.array(g["x"], np.float32), rms=False)
    gg, uu, aa = oracle.activations(w, h, np.arange(4, dtype=np.int32), oracle.ACT_REGLU)
    assert gg.tolist() == g["reglu"]["g"]
    assert uu.tolist() == g["reglu"]["u"]
    assert aa.tolist() == g["reglu"]["a"]
    y = oracle.down(w, np.arange(4, dtype=np.int32), aa)
    assert y.tolist() == g["reglu"]["y"]
    assert oracle.ffn_masked_dense(w, h, oracle.ACT_REGLU).tolist() == g["reglu"]["y"]
    # the all-zero block contributes nothing: block 0 alone gives the full output
    assert oracle.sparse_ffn(w, h, [0], 2, oracle.ACT_REGLU).tolist() == g["reglu"]["y"]
    assert oracle.sparse_ffn(w, h, [1], 2, oracle.ACT_REGLU).tolist() == [0.0, 0.0]


def test_golden_predictor_and_selection_by_hand():
    g, w = _golden()
    h = oracle.mlp_input(np.array(g["x"], np.float32), rms=False)
    s, z = oracle.predict(w.p1, w.p2, h, return_z=True)
    assert z.tolist() == [3.0, -1.0]
    assert s.tolist() == g["scores"]
    idx, cnt = oracle.select(s, k=1, cap=1)
    assert idx[0, :cnt[0]].tolist() == g["top1"]
    idx, cnt = oracle.select(s, k=2, cap=2)
    assert idx[0, :cnt[0]].tolist() == g["top2"]


def test_golden_swiglu_threshold_by_hand():
    g, w = _golden()
    s1, t1 = g["silu_pos1"], g["silu_neg1"]
    assert s1 == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), abs=1e-16)
    h = oracle.mlp_input(np.array(g["x"], np.float32), rms=False)
    y = oracle.ffn_masked_dense(w, h, oracle.ACT_SWIGLU_THRESH, 0.5)
    assert y == pytest.approx([8 * s1, -3 * s1], rel=1e-15)
    y = oracle.ffn_masked_dense(w, h, oracle.ACT_SWIGLU_THRESH, 0.25)
    assert y == pytest.approx([8 * s1 + 29 * t1, -3 * s1 + 34 * t1], rel=1e-14)
    # strictly above: a threshold equal to |SiLU(1)| drops neurons 0 and 1 as well
    _, _, a = oracle.activations(w, h, np.arange(4, dtype=np.int32), oracle.ACT_SWIGLU_THRESH, s1)
    assert a.tolist() == [0.0, 0.0, 0.0, 0.0]


# ----------------------------------------------------------------------------- MLP input

def test_mlp_input_closed_form():
    h = oracle.mlp_input(np.array([3.0, 4.0], np.float32), rms=True)
    assert h.tolist() == pytest.approx([3 / math.sqrt(12.5 + 1e-6), 4 / math.sqrt(12.5 + 1e-6)],
                                       rel=1e-15)
    x = np.random.default_rng(0).standard_normal(4096).astype(np.float32) * 3.0
    h = oracle.mlp_input(x, rms=True)
    assert np.mean(h * h) == pytest.approx(1.0, rel=1e-6)
    assert np.array_equal(oracle.mlp_input(x, rms=False), x.astype(np.float64))


# ----------------------------------------------------------------------------- library routines

@pytest.mark.parametrize("dtype", [lsgen.DT_F32, lsgen.DT_F16, lsgen.DT_BF16])
def test_predict_matches_float64_matmul(dtype):
    cfg, w = _small_layer(dtype=dtype)
    x = lsgen.tokens(cfg, 0, 1, 1)[0, 0]
    h = oracle.mlp_input(x, rms=True)
    s, z = oracle.predict(w.p1, w.p2, h, return_z=True)
    z_ref = _dec(w.p1) @ h
    s_ref = _dec(w.p2) @ z_ref
    assert np.allclose(z, z_ref, rtol=1e-12, atol=1e-14)
    ulps = np.abs(s.view(np.int32).astype(np.int64) - s_ref.astype(np.float32).view(np.int32))
    assert ulps.max() <= 1


@pytest.mark.parametrize("dtype", [lsgen.DT_F32, lsgen.DT_F16, lsgen.DT_BF16])
@pytest.mark.parametrize("act", [oracle.ACT_REGLU, oracle.ACT_SWIGLU_THRESH])
def test_dense_ffn_matches_float64_matmul(dtype, act):
    cfg, w = _small_layer(dtype=dtype)
    x = lsgen.tokens(cfg, 3, 1, 1)[0, 0]
    h = oracle.mlp_input(x, rms=True)
    t = 0.1
    y = oracle.ffn_masked_dense(w, h, act, t)
    g = _dec(w.gate) @ h + _dec(w.bias)
    u = _dec(w.up) @ h
    if act == oracle.ACT_REGLU:
        a = np.maximum(g, 0.0) * u
    else:
        sig = g * (1.0 / (1.0 + np.exp(-g)))
        a = np.where(np.abs(sig) > t, sig * u, 0.0)
    y_ref = _dec(w.down) @ a
    assert _rel(y, y_ref) < 1e-12
    # the list-driven path over every neuron gives the same result
    y2 = oracle.sparse_ffn(w, h, np.arange(cfg.n_blk), cfg.block, act, t)
    assert _rel(y2, y_ref) < 1e-12


# ----------------------------------------------------------------------------- masking identities

def test_masked_equals_sparse_and_all_blocks_equal_dense():
    cfg, w = _small_layer()
    rng = np.random.default_rng(1)
    x = lsgen.tokens(cfg, 1, 1, 1)[0, 0]
    h = oracle.mlp_input(x, rms=True)
    for trial in range(4):
        blocks = rng.choice(cfg.n_blk, size=rng.integers(1, cfg.n_blk), replace=False)
        mask = np.zeros(cfg.d_ff, np.uint8)
        mask[oracle.neurons_of_blocks(blocks, cfg.block)] = 1
        y_sparse = oracle.sparse_ffn(w, h, blocks, cfg.block, oracle.ACT_REGLU)
        y_mask = oracle.ffn_masked_dense(w, h, oracle.ACT_REGLU, mask=mask)
        assert _rel(y_sparse, y_mask) < 1e-12
    y_all = oracle.sparse_ffn(w, h, np.arange(cfg.n_blk), cfg.block, oracle.ACT_REGLU)
    y_dense = oracle.ffn_masked_dense(w, h, oracle.ACT_REGLU)
    assert _rel(y_all, y_dense) < 1e-12


def test_relu_zero_blocks_contribute_exactly_nothing():
    cfg, w = _small_layer(bias=0.0)
    dead = [1, 4, 9]
    bias = w.bias.copy()
    for b in dead:
        bias[b * cfg.block:(b + 1) * cfg.block] = -1e4
    w.bias = bias
    x = lsgen.tokens(cfg, 2, 1, 1)[0, 0]
    h = oracle.mlp_input(x, rms=True)
    live = [0, 2, 3, 5, 7]
    with_dead = [0, 1, 2, 4, 3, 5, 9, 7]  # same relative order of the live blocks
    _, a = oracle.sparse_ffn(w, h, dead, cfg.block, oracle.ACT_REGLU, return_a=True)
    assert np.all(a == 0.0)
    y1 = oracle.sparse_ffn(w, h, live, cfg.block, oracle.ACT_REGLU)
    y2 = oracle.sparse_ffn(w, h, with_dead, cfg.block, oracle.ACT_REGLU)
    assert np.array_equal(y1, y2)


# ----------------------------------------------------------------------------- Eq. 1-2 and Sec. 3.2.2

@pytest.mark.parametrize("K", [1, 2, 3, 8])
def test_stages_sum_to_single_shot(K):
    cfg, w = _small_layer()
    x = lsgen.tokens(cfg, 4, 1, 1)[0, 0]
    h = oracle.mlp_input(x, rms=True)
    s = oracle.predict(w.p1, w.p2, h)
    idx, cnt = oracle.select(s, k=7)
    blocks = idx[0, :cnt[0]]
    y = oracle.sparse_ffn(w, h, blocks, cfg.block, oracle.ACT_REGLU)
    dms, xt = oracle.staged_ffn(w, x, h, blocks, cfg.block, K, oracle.ACT_REGLU)
    assert len(dms) == K
    assert _rel(np.sum(dms, axis=0), y) < 1e-13
    assert _rel(xt[-1], x.astype(np.float64) + y) < 1e-13
    bounds = oracle.stage_bounds(7, K)
    assert bounds[0][0] == 0 and bounds[-1][1] == 7
    assert all(bounds[i][1] == bounds[i + 1][0] for i in range(K - 1))


def test_permutation_invariance():
    cfg, w = _small_layer()
    x = lsgen.tokens(cfg, 5, 1, 1)[0, 0]
    h = oracle.mlp_input(x, rms=True)
    rng = np.random.default_rng(3)
    blocks = rng.choice(cfg.n_blk, size=9, replace=False)
    y = oracle.sparse_ffn(w, h, blocks, cfg.block, oracle.ACT_REGLU)
    for _ in range(3):
        perm = rng.permutation(blocks)
        assert _rel(oracle.sparse_ffn(w, h, perm, cfg.block, oracle.ACT_REGLU), y) < 1e-13
    # neuron-level permutation as well (the sum over hidden neurons in any order)
    neurons = oracle.neurons_of_blocks(blocks, cfg.block)
    perm_n = rng.permutation(neurons).astype(np.int32)
    _, _, a = oracle.activations(w, h, perm_n, oracle.ACT_REGLU)
    assert _rel(oracle.down(w, perm_n, a), y) < 1e-13


def test_layer_step_composition():
    cfg, w = _small_layer()
    x = lsgen.tokens(cfg, 6, 1, 1)[0, 0]
    scores, idx, y, x_out = oracle.layer_step(w, cfg, x)
    h = oracle.mlp_input(x, rms=True)
    assert np.array_equal(scores, oracle.predict(w.p1, w.p2, h))
    ref_idx, _ = oracle.select(scores, k=cfg.k)
    assert np.array_equal(idx, ref_idx[0, :cfg.k])
    assert np.array_equal(y, oracle.sparse_ffn(w, h, idx, cfg.block, oracle.ACT_REGLU))
    assert np.array_equal(x_out, (x.astype(np.float64) + y).astype(np.float32))


# ----------------------------------------------------------------------------- selection

def _key(v):
    """Sort key of a float32 score: NaN below everything, -0 == +0, else IEEE order."""
    v = float(v)
    return (0, 0.0) if math.isnan(v) else (1, v + 0.0)


def _ref_order(s):
    return sorted(range(len(s)), key=lambda i: (tuple(-c for c in _key(s[i])), i))


def _ref_topk(s, k):
    return _ref_order(s)[:k]


def _ref_threshold(s, tau):
    tau = float(np.float32(tau))
    return [i for i in _ref_order(s) if not math.isnan(float(s[i])) and float(s[i]) > tau]


def _ref_union(S, sel_sets):
    members = set().union(*[set(x) for x in sel_sets])
    best = {i: max((_key(S[b][i]) for b in range(len(S)))) for i in members}
    return sorted(members, key=lambda i: (tuple(-c for c in best[i]), i))


def test_topk_brute_force_small():
    rng = np.random.default_rng(11)
    for n in range(1, 9):
        for trial in range(6):
            s = lsgen.adversarial_scores(rng, 1, n, ["ties", "zeros", "special", "normal"][trial % 4])[0]
            for k in range(1, n + 1):
                # brute force: the subset whose sorted (key, -index) vector is largest
                def vec(sub):
                    return sorted(((_key(s[i]), -i) for i in sub), reverse=True)
                best = max(itertools.combinations(range(n), k), key=vec)
                best_sorted = [i for _, i in ((None, -t[1]) for t in vec(best))]
                idx, cnt = oracle.select(s, k=k)
                assert cnt[0] == k
                assert idx[0, :k].tolist() == best_sorted


@settings(max_examples=200, deadline=None)
@given(st.lists(st.sampled_from([np.nan, np.inf, -np.inf, 0.0, -0.0, 1.0, -1.0, 0.5, 2.0]),
                min_size=1, max_size=40),
       st.integers(min_value=1, max_value=40))
def test_topk_matches_stable_sort(vals, k):
    s = np.array(vals, np.float32)
    k = min(k, len(vals))
    idx, cnt = oracle.select(s, k=k)
    assert cnt[0] == k
    assert idx[0, :k].tolist() == _ref_topk(s, k)


@settings(max_examples=150, deadline=None)
@given(st.lists(st.sampled_from([np.nan, np.inf, -np.inf, 0.0, -0.0, 1.0, -1.0, 0.5, 2.0]),
                min_size=1, max_size=40),
       st.sampled_from([0.0, -0.0, 0.5, -1.0, 1.0, np.inf, -np.inf]))
def test_threshold_matches_filter(vals, tau):
    s = np.array(vals, np.float32)
    idx, cnt = oracle.select(s, mode=oracle.SEL_THRESHOLD, tau=tau)
    ref = _ref_threshold(s, tau)
    assert cnt[0] == len(ref)
    assert idx[0, :cnt[0]].tolist() == ref


@settings(max_examples=120, deadline=None)
@given(st.integers(min_value=2, max_value=8), st.integers(min_value=1, max_value=30),
       st.integers(min_value=1, max_value=30), st.integers(min_value=0, max_value=10_000))
def test_union_properties(B, n, k, seed):
    k = min(k, n)
    rng = np.random.default_rng(seed)
    S = lsgen.adversarial_scores(rng, B, n, ["ties", "zeros", "special", "normal"][seed % 4])
    idx, cnt = oracle.select(S, k=k, union_batch=True, cap=min(n, B * k))
    per_tok = [_ref_topk(S[b], k) for b in range(B)]
    got = idx[:cnt[0]].tolist()
    assert got == _ref_union(S, per_tok)
    for b in range(B):
        assert set(per_tok[b]) <= set(got)
    assert len(got) <= min(n, B * k)
    assert len(set(got)) == len(got)


def test_per_token_batch_selection_and_cap():
    rng = np.random.default_rng(5)
    S = lsgen.adversarial_scores(rng, 3, 20, "normal")
    idx, cnt = oracle.select(S, k=4, cap=4)
    for b in range(3):
        assert idx[b].tolist() == _ref_topk(S[b], 4)
    with pytest.raises(ValueError):
        oracle.select(S, k=4, union_batch=True, cap=3)


# ----------------------------------------------------------------------------- generator & workload

def _splitmix_ref(seed, n):
    """SplitMix64 (Steele, Lea & Flood 2014): n-th output = mix(seed + n * gamma)."""
    M = (1 << 64) - 1
    z = (seed + n * 0x9E3779B97F4A7C15) & M
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
    return z ^ (z >> 31)


def test_generator_splitmix_definition():
    for seed in (0, 1, 1234567, 2**63 + 5):
        for n in (1, 2, 3, 1000):
            assert lsgen.splitmix64(seed, n) == _splitmix_ref(seed, n)
    # published first outputs of SplitMix64 seeded with 1234567
    assert [lsgen.splitmix64(1234567, n) for n in range(1, 6)] == [
        6457827717110365317, 3203168211198807973, 9817491932198370423,
        4593380528125082431, 16408922859458223821]


def test_generator_normal_statistics_and_determinism():
    a = lsgen.normal((400_000,), seed=3, tensor_id=1, layer=2, std=0.25, dtype=lsgen.DT_F32)
    assert abs(a.mean()) < 4 * 0.25 / math.sqrt(a.size)
    assert a.std() == pytest.approx(0.25, rel=4 * math.sqrt(2.0 / a.size))
    b = lsgen.normal((1000,), seed=3, tensor_id=1, layer=2, std=0.25, dtype=lsgen.DT_F32,
                     offset=123_000)
    assert np.array_equal(a[123_000:124_000], b)
    c = lsgen.normal((400_000,), seed=3, tensor_id=1, layer=3, std=0.25, dtype=lsgen.DT_F32)
    assert not np.array_equal(a, c)


def _bf16_rne_bruteforce(v64):
    """Nearest bf16 by search over all finite bf16 values, ties to the even pattern."""
    bits = np.arange(65536, dtype=np.uint32)
    vals = (bits << 16).view(np.float32).astype(np.float64)
    fin = np.isfinite(vals) & ~((vals == 0) & (bits >= 0x8000))
    vals, bits = vals[fin], bits[fin]
    order = np.argsort(vals, kind="stable")
    vals, bits = vals[order], bits[order]
    out = np.empty(v64.shape, np.uint16)
    pos = np.searchsorted(vals, v64)
    for i, (v, p) in enumerate(zip(v64, pos)):
        cands = [q for q in (p - 1, p) if 0 <= q < len(vals)]
        dist = [abs(vals[q] - v) for q in cands]
        m = min(dist)
        best = [q for q, dd in zip(cands, dist) if dd == m]
        q = best[0] if len(best) == 1 else [q for q in best if bits[q] % 2 == 0][0]
        out[i] = bits[q] if not (vals[q] == 0 and v < 0) else 0x8000
    return out


def test_generator_rounding_to_storage_types():
    a64 = lsgen.normal((20_000,), seed=9, tensor_id=2, layer=0, std=0.02, dtype=lsgen.DT_F32)
    # f16: same stream, compare with numpy's own double -> binary16 rounding of the fp64 value
    src = np.array([lsgen.splitmix64(0, 1)], dtype=np.uint64)  # noqa: F841 (touch the lib)
    f16 = lsgen.normal((20_000,), seed=9, tensor_id=2, layer=0, std=0.02, dtype=lsgen.DT_F16)
    f32 = a64  # binary32 rounding of the same fp64 values
    # binary16 has 11 significant bits < 24, so rounding the binary32 value is exact except at
    # double-rounding ties; require agreement on all but a tiny fraction and within 1 ulp
    diff = np.abs(f16.view(np.int16).astype(np.int32) - f32.astype(np.float16).view(np.int16))
    assert diff.max() <= 1 and (diff > 0).mean() < 1e-3
    bf = lsgen.normal((3000,), seed=9, tensor_id=2, layer=0, std=0.02, dtype=lsgen.DT_BF16)
    ref = _bf16_rne_bruteforce(f32[:3000].astype(np.float64))
    d = np.abs(bf.astype(np.int32) - ref.astype(np.int32))
    assert d.max() <= 1 and (d > 0).mean() < 1e-2
    assert lsgen.const((2,), -1.2815515655446004, lsgen.DT_F16).tolist() == [-1.28125, -1.28125]


def test_workload_constants():
    cfgs = lsgen.CONFIGS
    assert [c.k for c in cfgs.values()] == [10, 21, 56, 26, 21, 23]
    assert [c.n_blk for c in cfgs.values()] == [48, 172, 112, 216, 172, 224]
    from statistics import NormalDist
    assert NormalDist().cdf(cfgs["llama2_7b_ffn"].gate_bias) == pytest.approx(0.10, abs=1e-12)
    assert NormalDist().cdf(cfgs["llama2_70b_stream"].gate_bias) == pytest.approx(0.08, abs=1e-12)


def test_swiglu_threshold_constant_by_quadrature():
    """P(|SiLU(Z)| > t) = 1/2 for Z ~ N(0,1), integrated numerically (scipy)."""
    from scipy import integrate, stats
    t = lsgen.CONFIGS["mistral_7b_ffn"].swiglu_threshold

    def silu(z):
        return z / (1.0 + math.exp(-z))
    p = integrate.quad(lambda z: stats.norm.pdf(z) * (abs(silu(z)) > t), -12, 12, limit=500,
                       points=[-3.0, -1.2785, -0.5, 0.0, 0.5])[0]
    assert p == pytest.approx(0.5, abs=2e-6)


def test_active_fraction_matches_closed_form():
    """ReGLU gate bias b gives P(g > 0) = Phi(b) under the RMS prenorm (C2/C4 shape)."""
    cfg = lsgen.CONFIGS["llama2_7b_ffn"].with_(d_ff=1024, n_layers=1)
    w = lsgen.layer_weights(cfg, 0)
    xs = lsgen.tokens(cfg, 0, 8, 1)[:, 0]
    act = 0
    for x in xs:
        h = oracle.mlp_input(x, rms=True)
        g, _, _ = oracle.activations(w, h, np.arange(cfg.d_ff, dtype=np.int32), oracle.ACT_REGLU)
        act += int((g > 0).sum())
    n = cfg.d_ff * len(xs)
    p = 0.10
    assert abs(act / n - p) < 4 * math.sqrt(p * (1 - p) / n) + 0.01


def test_swiglu_threshold_gives_half_sparsity():
    cfg = lsgen.CONFIGS["mistral_7b_ffn"].with_(d_ff=1024, calib_tokens=16)
    w = lsgen.layer_weights(cfg, 0)
    t_emp = oracle.calibrate_threshold(w, cfg, lsgen.calib_tokens(cfg, 0), 0.5)
    assert t_emp == pytest.approx(cfg.swiglu_threshold, rel=0.05)


# ------------------------------------------------------ refinement quality (Sec. 6 validation)

def test_importance_ratio_brute_force_small():
    rng = np.random.default_rng(3)
    for _ in range(50):
        n = int(rng.integers(2, 8))
        imp = rng.random(n) * rng.integers(0, 2, n)  # some zero importances
        m = int(rng.integers(1, n + 1))
        P = rng.choice(n, m, replace=False)
        best = max(sum(imp[list(c)]) for c in itertools.combinations(range(n), m))
        expect = imp[P].sum() / best if best > 0 else 1.0
        assert math.isclose(oracle.importance_ratio(imp, P), expect, rel_tol=1e-12)
    imp = np.array([3.0, 1.0, 2.0])
    assert oracle.importance_ratio(imp, [0, 2]) == 1.0  # the best set of two


def test_top_fraction_recall_definition():
    imp = np.array([5.0, 1.0, 5.0, 0.0, 2.0, 9.0, 0.5, 0.5, 0.5, 7.0, 4.0])  # n = 11: top 2
    # top two by importance: 5 (9.0), 9 (7.0)
    assert oracle.top_fraction_recall(imp, [5, 9, 0]) == 1.0
    assert oracle.top_fraction_recall(imp, [5, 1]) == 0.5
    assert oracle.top_fraction_recall(imp, [1, 2]) == 0.0
    # ties go to the smaller index: top 3 of [1,1,1,1] at frac 0.75 is {0,1,2}
    assert oracle.top_fraction_recall(np.ones(4), [0, 1, 2], frac=0.75) == 1.0
    assert oracle.top_fraction_recall(np.ones(4), [3], frac=0.75) == 0.0


def test_block_importance_invariants():
    cfg, w = _small_layer(bias=-0.2)
    x = lsgen.tokens(cfg, 0, 1, 1)[0, 0]
    h = oracle.mlp_input(x, cfg.prenorm)
    imp = oracle.block_importance(w, h, cfg.block, cfg.act)
    assert imp.shape == (cfg.n_blk,) and np.all(imp >= 0)
    # scaling the down projection by c scales every importance by |c| (c = -2: exact in fp32)
    w2 = SimpleNamespace(**{**w.__dict__, "down": (w.down * np.float32(-2.0)).astype(w.down.dtype)})
    assert np.allclose(oracle.block_importance(w2, h, cfg.block, cfg.act), 2 * imp, rtol=1e-12)
    # permuting the neurons within a block (gate, up rows, down columns, bias together) keeps
    # the block's importance (Sec. 3.2.2)
    perm = np.arange(cfg.d_ff).reshape(cfg.n_blk, cfg.block)[:, ::-1].reshape(-1)
    w3 = SimpleNamespace(gate=w.gate[perm], up=w.up[perm], down=np.ascontiguousarray(w.down[:, perm]),
                         bias=None if w.bias is None else w.bias[perm], threshold=w.threshold)
    assert np.allclose(oracle.block_importance(w3, h, cfg.block, cfg.act), imp, rtol=1e-12)
    # a block whose neurons are all inactive has no importance: ReLU(g) = 0 for g + b <= 0
    _, _, a = oracle.activations(w, h, np.arange(cfg.d_ff, dtype=np.int32), cfg.act)
    dead = np.all(a.reshape(cfg.n_blk, cfg.block) == 0, axis=1)
    assert np.all(imp[dead] == 0) and np.all(imp[~dead] > 0)


def test_threaded_layer_step_is_identical():
    """The oracle's thread-split layer step (used to time it on every host core) gives the very
    same scores, list and outputs as the single-thread one, for any thread count."""
    cfg = lsgen.CONFIGS["llama2_7b_ffn"].with_(n_layers=1, d_model=256, d_ff=1024, block=32, rank=64)
    w = lsgen.layer_weights(cfg, 0)
    x = lsgen.tokens(cfg, 2, 1, 1)[0, 0]
    ref = oracle.layer_step(w, cfg, x)
    for nt in (1, 3, 8, 64):
        got = oracle.layer_step(w, cfg, x, n_threads=nt)
        for a, b in zip(got, ref):
            assert np.array_equal(a, b), nt


def test_block_importance_hand_computed_value():
    # d = 2, F = 4, two blocks of 2 neurons, ReGLU, no bias, h = (1, 2):
    #   g = (1, 2, 3, -1), u = (2, 2, 1, 6), a = max(g, 0) * u = (2, 4, 3, 0)
    #   W_down columns (3,4), (0,1), (1,1), (5,12) have L2 norms 5, 1, sqrt(2), 13
    #   block 0: |2|*5 + |4|*1 = 14; block 1: |3|*sqrt(2) + 0*13 = 3*sqrt(2)
    # An L1 column norm would give 18 and 6; the norm of the block's summed contribution
    # 2*(3,4) + 4*(0,1) = (6,12) would give sqrt(180) for block 0.
    f32 = np.float32
    w = SimpleNamespace(gate=np.array([[1, 0], [0, 1], [1, 1], [-1, 0]], f32),
                        up=np.array([[2, 0], [0, 1], [1, 0], [0, 3]], f32),
                        down=np.array([[3, 0, 1, 5], [4, 1, 1, 12]], f32),
                        bias=None, threshold=0.0)
    imp = oracle.block_importance(w, np.array([1.0, 2.0]), 2, lsgen.ACT_REGLU)
    assert np.allclose(imp, [14.0, 3.0 * math.sqrt(2.0)], rtol=1e-14, atol=0)


def test_refinement_last_stage_is_the_complete_output_prediction():
    cfg = lsgen.CONFIGS["llama2_7b_ffn"].with_(n_layers=2, d_model=256, d_ff=1024, block=32, rank=64,
                                               dtype=lsgen.DT_F32, predictor="planted")
    ws = [lsgen.layer_weights(cfg, l) for l in range(2)]
    x = lsgen.tokens(cfg, 0, 1, 1)[0, 0]
    q1, s1, f1 = oracle.refinement_quality(ws[0], ws[1], cfg, x, 1)
    q4, s4, f4 = oracle.refinement_quality(ws[0], ws[1], cfg, x, 4)
    # stage 0 is the one-shot prediction from x in both; the last stage sees the whole output
    # (Eq. 2 with j = K equals the complete layer), whatever the number of stages
    assert np.array_equal(s1[0], s4[0]) and np.array_equal(f1[0], f4[0])
    assert _rel(f1[-1], f4[-1]) < 1e-6
    h = oracle.mlp_input(x, cfg.prenorm)
    idx = oracle.select(oracle.predict(ws[0].p1, ws[0].p2, h), k=cfg.k, cap=cfg.k)[0][0]
    full = x.astype(np.float64) + oracle.sparse_ffn(ws[0], h, idx, cfg.block, cfg.act)
    assert _rel(f4[-1], full) < 1e-6
    # the prediction on the complete output scored against the importance on that same output
    # is what a stage-K refinement reports; a random predictor order is not pinned here
    assert all(0.0 <= r <= 1.0 and 0.0 <= c <= 1.0 for r, c in q4)
    # the reverse order visits the same blocks: same complete output
    q4r, s4r, f4r = oracle.refinement_quality(ws[0], ws[1], cfg, x, 4, order=np.arange(cfg.k)[::-1])
    assert _rel(f4r[-1], f4[-1]) < 1e-6 and np.array_equal(s4r[-1], s4[-1])


# ------------------------------------------------------ stacked learnable hashing (Sec. 3.3.1)

def _unpack_signs(words):
    """bit-packed {-1,+1} vectors (uint32, last axis words) -> int64 arrays of +-1"""
    w = np.asarray(words, np.uint64)
    bits = (w[..., None] >> np.arange(32, dtype=np.uint64)) & 1
    return (2 * bits.reshape(*w.shape[:-1], -1).astype(np.int64) - 1)


def _Z(tau=8):
    """The paper's sign-pattern matrix: row i enumerates the patterns in the order of its
    example, (-1,...,-1), (-1,...,-1,+1), ..., (+1,...,+1) (Eq. hashfunc_mod)."""
    return np.array(list(itertools.product([-1, 1], repeat=tau)), np.int64)


def _hash_ref(hw, x, n_blk):
    """Independent reading: fp64 first layer, +-1 integer products after it, and the index
    as argmax_i Z[i] . code (Eq. hashfunc_mod) instead of a bit packing."""
    Z = _Z()
    dots = np.asarray(x, np.float64) @ hw.w1.astype(np.float64)
    code = np.where(dots >= 0, 1, -1)
    idx = [int(np.argmax(Z @ code))]
    T, W = _unpack_signs(hw.tables), _unpack_signs(hw.w_bin)     # [4,256,256], [4,8,256]
    for k in range(4):
        y = T[k, idx[-1]]
        code = np.where(W[k] @ y >= 0, 1, -1)
        idx.append(int(np.argmax(Z @ code)))
    return hw.head[idx[-1]].astype(np.float32), np.array(idx), dots


def test_hash_index_is_the_papers_sign_pattern_enumeration():
    # tau = 3 example of the paper: row 1 of Z is (-1, -1, +1), row 6 is (+1, +1, -1)
    Z3 = _Z(3)
    assert Z3[1].tolist() == [-1, -1, 1] and Z3[6].tolist() == [1, 1, -1]
    cfg = lsgen.CONFIGS["llama2_7b_ffn"].with_(d_model=256, d_ff=1024, block=64)
    hw = lsgen.hash_weights(cfg, 0)
    Z = _Z()
    for j in range(0, 256, 37):  # one-hot inputs: layer 1's code is the sign pattern of W1[j]
        x = np.zeros(256, np.float32)
        x[j] = 1.0
        _, codes, _ = oracle.hash_predict(hw, x, cfg.n_blk)
        code = np.where(hw.w1[j] >= 0, 1, -1)
        assert codes[0] == int(np.argmax(Z @ code))
    # x = 0: every product is 0 and sign(0) = +1, the all-plus bucket
    _, codes, _ = oracle.hash_predict(hw, np.zeros(256, np.float32), cfg.n_blk)
    assert codes[0] == 255


def test_hash_stack_matches_integer_products_and_argmax_reading():
    cfg = lsgen.CONFIGS["llama2_7b_ffn"].with_(d_model=1024, d_ff=4096, block=64)
    rng = np.random.default_rng(11)
    for layer in range(3):
        hw = lsgen.hash_weights(cfg, layer)
        for _ in range(20):
            x = rng.standard_normal(1024).astype(np.float32)
            s, codes, prods = oracle.hash_predict(hw, x, cfg.n_blk)
            s_ref, idx_ref, dots = _hash_ref(hw, x, cfg.n_blk)
            # both sides take the first layer in float64 (library matmul against the oracle's
            # plain loop); only a product within float64 rounding of zero could differ
            assert np.min(np.abs(dots)) > 1e-9
            assert np.allclose(prods, dots, rtol=1e-12, atol=1e-12)
            assert codes.tolist() == idx_ref.tolist()
            assert np.array_equal(s, s_ref)
            assert np.array_equal(s, hw.head[codes[-1]].astype(np.float32))


def test_hash_imposed_first_bucket_drives_the_later_layers():
    cfg = lsgen.CONFIGS["llama2_7b_ffn"].with_(d_model=256, d_ff=1024, block=64)
    hw = lsgen.hash_weights(cfg, 1)
    x = np.random.default_rng(3).standard_normal(256).astype(np.float32)
    s, codes, prods = oracle.hash_predict(hw, x, cfg.n_blk)
    # imposing the bucket the products give changes nothing
    s2, codes2, prods2 = oracle.hash_predict(hw, x, cfg.n_blk, code0=int(codes[0]))
    assert np.array_equal(s, s2) and codes.tolist() == codes2.tolist()
    assert np.array_equal(prods, prods2)
    # flipping one first-layer bit re-derives layers 2-5 from the flipped code (integer
    # products of the table row it selects, Eq. hashfunc_layer)
    T, W = _unpack_signs(hw.tables), _unpack_signs(hw.w_bin)
    Z = _Z()
    for bit in range(8):
        c0 = int(codes[0]) ^ (1 << (7 - bit))
        s3, codes3, _ = oracle.hash_predict(hw, x, cfg.n_blk, code0=c0)
        idx = [c0]
        for k in range(4):
            code = np.where(W[k] @ T[k, idx[-1]] >= 0, 1, -1)
            idx.append(int(np.argmax(Z @ code)))
        assert codes3.tolist() == idx
        assert np.array_equal(s3, hw.head[idx[-1]].astype(np.float32))


def test_hash_xnor_popcount_equals_signed_product():
    rng = np.random.default_rng(5)
    a = rng.integers(0, 2**32, size=(50, 8), dtype=np.uint64).astype(np.uint32)
    b = rng.integers(0, 2**32, size=(50, 8), dtype=np.uint64).astype(np.uint32)
    pa, pb = _unpack_signs(a), _unpack_signs(b)
    mism = np.array([sum(bin(int(x) ^ int(y)).count("1") for x, y in zip(ra, rb)) for ra, rb in zip(a, b)])
    assert np.array_equal((pa * pb).sum(axis=1), 256 - 2 * mism)
