"""Pins for the oracle's attention-score collector (Sec. 3.1, Eqs.
score-partial, score-global-weight, attention-score).

* With lossless FP8 pages the normalized page mass q~_{h,p} equals scipy's
  softmax over the original data summed per page.
* The paper's partition form w_j rho_p^{(j)}, computed here from scipy scores
  for random partitions of the pages, gives the same masses.
* Closed forms: one token carries all the mass; identical keys spread it as
  (valid tokens of the page) / seq_len; the masses of a head sum to 1.
* The EWMA a_T = beta^T a_0 + (1 - beta^T) r for a repeated input, and r is the
  mean over the sampled heads only.
"""
import numpy as np
import pytest
from scipy.special import softmax

import mkv_workloads as wl

PAGE = 16


def _lossless_state(orc, d, hq, hkv, lens, seed):
    rng = np.random.default_rng(seed)
    sigma = np.where(rng.integers(0, 2, d) == 1, 1, -1).astype(np.int8)
    n_pg = sum((L + PAGE - 1) // PAGE for L in lens) + 4
    P = orc.Pool(1, hq, hkv, d, n_pg, n_pg, 10 ** 6, sigma, rng.permutation(n_pg), None)
    kv = []
    for L in lens:
        vals = orc.e4m3_to_f64(rng.integers(0, 0x7E, size=(2, L, hkv, d)).astype(np.uint8))
        vals *= rng.choice([-1, 1], size=vals.shape)
        vals[:, ::16, :, 0] = 448.0
        vals *= 2.0 ** -5
        kv.append(vals.astype(np.float32))
    k = wl.bf16_round(np.concatenate([x[0] for x in kv]))
    v = wl.bf16_round(np.concatenate([x[1] for x in kv]))
    mp = max((L + PAGE - 1) // PAGE for L in lens)
    bt = np.full((len(lens), mp), -1, np.int32)
    tags = np.full((len(lens), mp), orc.TAG_NONE, np.uint8)
    cu = np.r_[0, np.cumsum(lens)].astype(np.int32)
    assert P.append(-1, bt, tags, np.zeros(len(lens), np.int32), cu, k[None], v[None]) == 0
    q = wl.bf16_round(rng.standard_normal((len(lens), hq, d)).astype(np.float32))
    return P, kv, q, bt, tags


@pytest.mark.parametrize("d", (128, 256))
def test_page_mass_equals_softmax_per_page(orc, d):
    hq, hkv, lens = 4, 2, [100, 33, 16]
    P, kv, q, bt, tags = _lossless_state(orc, d, hq, hkv, lens, 20 + d)
    a = np.zeros(bt.shape)
    qn, r = P.page_scores(0, q, bt, tags, np.array(lens, np.int32), np.ones(hq, np.uint8), 0.0, a)
    qf = wl.bf16_to_f32(q).astype(np.float64)
    for ri, L in enumerate(lens):
        np_ = (L + PAGE - 1) // PAGE
        for h in range(hq):
            s = kv[ri][0][:, h // (hq // hkv)].astype(np.float64) @ qf[ri, h] / np.sqrt(d)
            pi = softmax(s)
            want = np.array([pi[p * PAGE:(p + 1) * PAGE].sum() for p in range(np_)])
            assert np.allclose(qn[ri, :np_, h], want, rtol=0, atol=1e-13)
            assert abs(qn[ri, :np_, h].sum() - 1.0) < 1e-13
        assert np.allclose(r[ri, :np_], qn[ri, :np_].mean(axis=1), atol=1e-15)
        assert np.allclose(a[ri, :np_], r[ri, :np_], atol=1e-15)  # beta = 0


def test_partition_form_equals_page_mass(orc):
    """Eq. score-global-weight: q_p = w_j rho_p^{(j)} for any partition of the
    pages, computed from the per-partition (m_j, l_j) of Eq. score-partial."""
    d, hq, hkv, L = 128, 2, 1, 300
    P, kv, q, bt, tags = _lossless_state(orc, d, hq, hkv, [L], 3)
    a = np.zeros(bt.shape)
    qn, _ = P.page_scores(0, q, bt, tags, np.array([L], np.int32), np.ones(hq, np.uint8), 0.5, a)
    s_all = kv[0][0][:, 0].astype(np.float64) @ wl.bf16_to_f32(q[0, 1]).astype(np.float64) / np.sqrt(d)
    np_ = (L + PAGE - 1) // PAGE
    rng = np.random.default_rng(8)
    for _ in range(10):
        cuts = np.sort(rng.choice(np.arange(1, np_), size=rng.integers(1, 6), replace=False))
        parts = np.split(np.arange(np_), cuts)
        m = np.array([s_all[p[0] * PAGE:min(L, (p[-1] + 1) * PAGE)].max() for p in parts])
        l = np.array([np.exp(s_all[p[0] * PAGE:min(L, (p[-1] + 1) * PAGE)] - m[j]).sum()
                      for j, p in enumerate(parts)])
        M = m.max()
        ell = (np.exp(m - M) * l).sum()
        for j, pages in enumerate(parts):
            w = np.exp(m[j] - M) * l[j] / ell
            for p in pages:
                rho = np.exp(s_all[p * PAGE:min(L, (p + 1) * PAGE)] - m[j]).sum() / l[j]
                assert abs(w * rho - qn[0, p, 1]) < 1e-13


def test_closed_forms_and_ewma(orc):
    d, hq, hkv = 128, 3, 1
    rng = np.random.default_rng(2)
    sigma = np.ones(d, np.int8)
    P = orc.Pool(1, hq, hkv, d, 16, 16, 10 ** 6, sigma)
    k = wl.bf16_round(np.broadcast_to(rng.standard_normal((1, 1, d)), (71, 1, d)).astype(np.float32))
    v = wl.bf16_round(rng.standard_normal((71, 1, d)).astype(np.float32))
    bt = np.full((2, 5), -1, np.int32)
    tags = np.full((2, 5), orc.TAG_NONE, np.uint8)
    # request 0: 70 identical keys; request 1: a single token
    assert P.append(-1, bt, tags, np.zeros(2, np.int32), np.array([0, 70, 71], np.int32),
                    k[None], v[None]) == 0
    q = wl.bf16_round(rng.standard_normal((2, hq, d)).astype(np.float32))
    a0 = rng.random((2, 5))
    a = a0.copy()
    sl = np.array([70, 1], np.int32)
    beta, T = 0.9, 5
    mask = np.array([1, 0, 1], np.uint8)
    for _ in range(T):
        qn, r = P.page_scores(0, q, bt, tags, sl, mask, beta, a)
    # identical keys: mass = valid tokens / seq_len; one token: all the mass
    want = np.array([16, 16, 16, 16, 6]) / 70.0
    for h in range(hq):
        assert np.allclose(qn[0, :5, h], want, atol=1e-13)
    assert np.allclose(qn[1, 0], 1.0, atol=1e-15)
    assert np.allclose(r[0, :5], want, atol=1e-13)
    assert np.allclose(a[0], beta ** T * a0[0] + (1 - beta ** T) * want, atol=1e-13)
    # request 1 has one page: the rest of its row is left as it was
    assert np.allclose(a[1, 0], beta ** T * a0[1, 0] + (1 - beta ** T) * 1.0, atol=1e-13)
    assert np.array_equal(a[1, 1:], a0[1, 1:])
    # r averages the sampled heads only
    q2 = q.copy()
    q2[0, 1] = wl.bf16_round(100 * rng.standard_normal(d).astype(np.float32))  # unsampled head
    _, r2 = P.page_scores(0, q2, bt, tags, sl, mask, beta, a.copy())
    assert np.allclose(r2[0, :5], r[0, :5], atol=1e-15)
