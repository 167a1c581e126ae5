"""GPU parity of the direct attention-score collector (Sec. 3.1 Eqs.
score-partial, score-global-weight, attention-score; Sec. 4.2) against the
oracle: paged_attn_decode_scores (decode outputs within 1e-3, as every decode)
and kv_page_scores_update (normalized page masses q~, head means r and the
EWMA scores a).

Tolerance of the masses: a page's mass is a sum of softmax weights exp(s_i -
lse); the decode's scores carry an absolute error of order 1e-5 (its outputs
are within 1e-5 - 8e-5 of the oracle), so each mass has a relative error of
that order.  The test allows 2e-3 relative plus 1e-7 absolute, and the masses
of each head must sum to 1 within 1e-5.
"""
import dataclasses

import numpy as np
import pytest

import mkv_workloads as wl
from _harness import max_abs

pytestmark = pytest.mark.gpu

TOL = 1e-3
REL, ABS = 2e-3, 1e-7


def _close(got, want):
    return np.abs(got - want) <= REL * np.abs(want) + ABS


def _scores_case(w, lens, recent, layer=0, beta=0.8, seed=0, n_layers=1):
    import torch
    import paper_2608_23834_amd as mk
    from _harness import Twin
    print(f"\n[scores] {w.name} lens={lens[:4]} W={recent}", flush=True)
    tw = Twin(w, n_layers=n_layers, lens=lens, recent=recent)
    tw.fill()
    tw.migrate()
    n_req, Hq, d, mp = len(lens), w.n_q_heads, w.head_dim, tw.max_pages
    q = wl.q_decode(w, layer)
    q = np.ascontiguousarray(np.resize(q, (n_req,) + q.shape[1:]))
    sl = np.array(tw.cur, np.int32)
    rng = np.random.default_rng(seed)
    head_mask = (rng.random(Hq) < 0.5).astype(np.uint8)
    head_mask[0] = 1
    a0 = rng.random((n_req, mp)).astype(np.float32)
    out = torch.full((n_req, Hq, d), float("nan"), device="cuda")
    lse = torch.full((n_req, Hq), float("nan"), device="cuda")
    pm = torch.full((n_req, mp, Hq, 2), float("nan"), device="cuda")
    ws = mk.workspace(tw.gpu, n_req, mp)
    slg = torch.from_numpy(sl).cuda()
    mk.paged_attn_decode_scores(tw.gpu, layer, torch.from_numpy(q.view(np.int16)).cuda(), tw.bt,
                                tw.tags, slg, out, lse, ws, pm)
    a_g = torch.from_numpy(a0).cuda()
    r_g = torch.full((n_req, mp), float("nan"), device="cuda")
    qn_g = torch.full((n_req, mp, Hq), float("nan"), device="cuda")
    mk.kv_page_scores_update(tw.gpu, slg, lse, pm, torch.from_numpy(head_mask).cuda(), beta, a_g,
                             r_g, qn_g)
    torch.cuda.synchronize()
    assert mk.kv_pool_check_errors(tw.gpu) == 0
    ref_o, ref_l = tw.orc.decode(layer, q, tw.obt, tw.otags, sl)
    err = max(max_abs(out.cpu().numpy(), ref_o), max_abs(lse.cpu().numpy(), ref_l))
    a_ref = a0.astype(np.float64).copy()
    qn_ref, r_ref = tw.orc.page_scores(layer, q, tw.obt, tw.otags, sl, head_mask, beta, a_ref)
    qn, r, a = qn_g.cpu().numpy(), r_g.cpu().numpy(), a_g.cpu().numpy()
    worst = 0.0
    for i, L in enumerate(lens):
        npg = (L + 15) // 16
        assert np.all(_close(qn[i, :npg], qn_ref[i, :npg])), i
        assert np.all(_close(r[i, :npg], r_ref[i, :npg])), i
        assert np.all(_close(a[i, :npg], a_ref[i, :npg])), i
        assert np.all(np.abs(qn[i, :npg].sum(axis=0) - 1.0) <= 1e-5), i
        assert np.array_equal(a[i, npg:], a0[i, npg:]), i  # pages past the end untouched
        worst = max(worst, float(np.max(np.abs(qn[i, :npg] - qn_ref[i, :npg]) /
                                        (np.abs(qn_ref[i, :npg]) + 1e-7))))
    print(f"  decode max|dO|, max|dlse| {err:.2e}; masses max rel err {worst:.2e}; "
          f"TQ3 pages {int((tw.otags == 2).sum())}", flush=True)
    assert err <= TOL
    return tw


def test_scores_ragged_d256_group6():
    _scores_case(wl.workload(2), [1, 17, 700, 3000], recent=64)


def test_scores_d128_group8_and_group12():
    _scores_case(wl.workload(1), [2048, 300], recent=256, seed=1)
    _scores_case(dataclasses.replace(wl.workload(2), n_kv_heads=2, name="group12"), [1500, 40],
                 recent=64, seed=2)


def test_scores_long_pair_full_size():
    """The long pair at full size (2 x 59,008 tokens), one layer."""
    w = wl.workload(3)
    _scores_case(w, list(w.ctx), recent=None, seed=3)
