"""The no-allocation sparse step (ls_sparse_ffn_step_static): the same results as
ls_sparse_ffn_step, bit for bit, with its scratch in the library's fixed device array.
Two calls in a row, the second with fewer tokens and a shorter list (the array keeps the
first call's contents), on a shape whose batch runs the matrix-core kernels with the down
projection split in parts (both scratch regions in use), then on a vector-ALU shape; each
output also against the oracle, teacher-forced.  A request larger than the array is refused."""
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

SHAPES = {
    # 16-bit weights, 64-neuron blocks, 40 column tiles: B >= 4 runs the matrix-core kernels
    # and cuts the down projection's list in parts
    "f16_mfma_split": C["llama2_7b_ffn"].with_(n_layers=1, d_model=640, d_ff=1728, block=64, rank=192,
                                               keep_pct=30),
    "f32_valu": C["c1_reglu_512"].with_(n_layers=1, d_model=320, d_ff=960, block=40, rank=64,
                                        keep_pct=40),
}


def _run_both(f, cfg, xs, B, k):
    x_in = dev_f32(xs[:B])
    scores = empty_f32(B, cfg.n_blk)
    cap = min(cfg.n_blk, B * k)
    idx, cnt = empty_i32(cap), empty_i32(1)
    f.ls_predict(0, x_in, B, scores)
    f.ls_select_blocks(scores, B, lsffn.LS_SEL_TOPK, k, 0.0, 1, cap, idx, cnt)
    out_ref = empty_f32(B, cfg.d_model)
    out_st = empty_f32(B, cfg.d_model)
    out_st.fill_(float("nan"))
    f.ls_sparse_ffn_step(0, x_in, B, idx, cnt, 0, cap, out_ref)
    f.ls_sparse_ffn_step_static(0, x_in, B, idx, cnt, 0, cap, out_st)
    f.ls_ffn_sync()
    return host(out_ref), host(out_st), host(idx)[:host(cnt)[0]]


@pytest.mark.parametrize("name", list(SHAPES))
def test_static_scratch_step_equals_the_allocating_step(name):
    cfg = SHAPES[name]
    f, ws = make_ffn(cfg, max_batch=8)
    xs = lsgen.tokens(cfg, 21, 1, 8, max_batch=8)[0]
    for B, k in ((8, cfg.k), (2, max(1, cfg.k // 2))):   # the second call is smaller
        ref, got, blocks = _run_both(f, cfg, xs, B, k)
        assert np.array_equal(got, ref), (name, B)
        for b in range(B):
            h = oracle.mlp_input(xs[b], cfg.prenorm)
            y_ref = oracle.sparse_ffn(ws[0], h, blocks, cfg.block, cfg.act, ws[0].threshold)
            assert y_err(got[b].astype(np.float64) - xs[b], y_ref) <= Y_TOL[cfg.dtype], (name, B, b)
    f.close()


def test_static_scratch_refuses_an_oversized_request():
    # B * (d_ff + 8 d_model) = 4 * (262144 + 512) floats > the 4 MiB array
    f = lsffn.Ffn(n_layers=1, d_model=64, d_ff=262144, block=128, rank=64, max_batch=4,
                  dtype=lsffn.LS_F16)
    x = empty_f32(4, 64)
    out = empty_f32(4, 64)
    idx, cnt = empty_i32(4), empty_i32(1)
    with pytest.raises(lsffn.LsError) as e:
        f.ls_sparse_ffn_step_static(0, x, 4, idx, cnt, 0, 4, out)
    assert e.value.status == lsffn.LS_E_CAPACITY
    f.close()
