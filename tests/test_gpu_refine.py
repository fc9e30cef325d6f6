"""GPU parity of refined next-layer prediction (Sec. 2.1, Eq. 2; the refinement-step validation).

Layer n runs in K staged sparse steps over its priority list; after each stage the
library scores layer n+1 on the partial result x~^(j).  Checked per stage against the
oracle: x~^(j) - x within the FFN output tolerance, the scores teacher-forced on the
GPU's x~^(j) within 1e-5, and the next layer's selection on those scores bit-exact.
The workload has a planted predictor (lsgen "planted"), so the quality numbers the
bench reports are meaningful; their arithmetic is pinned on the CPU.
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
from gpu_util import SCORE_TOL, Y_TOL, dev_f32, empty_f32, empty_i32, host, make_ffn, rel_l2, y_err  # noqa: E402

CFG = lsgen.CONFIGS["llama2_7b_planted"].with_(n_layers=2, d_model=1024, d_ff=4096, block=64, rank=256)


@pytest.mark.parametrize("K,reverse", [(4, False), (8, False), (4, True)])
def test_refined_prediction_per_stage(K, reverse):
    f, ws = make_ffn(CFG)
    k = CFG.k
    scores = empty_f32(1, CFG.n_blk)
    idx, cnt = empty_i32(k), empty_i32(1)
    nidx, ncnt = empty_i32(k), empty_i32(1)
    for t in range(2):
        x0 = lsgen.tokens(CFG, 40 + t, 1, 1)[0]
        x = dev_f32(x0)
        f.ls_predict(0, x, 1, scores)
        f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, k, 0.0, 0, k, idx, cnt)
        order = np.arange(k)[::-1].copy() if reverse else None
        lst = host(idx) if order is None else host(idx)[order]
        lst_d = torch.from_numpy(np.ascontiguousarray(lst)).to(x.device)
        _, sets_ref, feats_ref = oracle.refinement_quality(ws[0], ws[1], CFG, x0[0], K, order=order)
        acc = empty_f32(1, CFG.d_model)
        x_np = x0[0].astype(np.float64)
        for j in range(K):
            lo, hi = j * k // K, (j + 1) * k // K
            f.ls_sparse_ffn_step(0, x, 1, lst_d, cnt, lo, hi, acc)  # acc = x + stages 0..j
            xt = host(acc)[0]
            assert y_err(xt - x_np, feats_ref[j + 1] - x_np) <= Y_TOL[CFG.dtype], (t, j)
            f.ls_predict(1, acc, 1, scores)
            s_gpu = host(scores)[0]
            s_ref = oracle.predict(ws[1].p1, ws[1].p2, oracle.mlp_input(xt, CFG.prenorm))
            assert rel_l2(s_gpu, s_ref) <= SCORE_TOL, (t, j)
            f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, k, 0.0, 0, k, nidx, ncnt)
            sel_ref = oracle.select(s_gpu, k=k, cap=k)[0][0]
            assert np.array_equal(host(nidx), sel_ref), (t, j)
    f.ls_ffn_sync()
