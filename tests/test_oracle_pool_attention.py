"""Pins for the oracle's pool state machine (Alg. 1 Append/Retier, Sec. 3.1 tier
rule, Sec. 4.1 compact lists) and its reference attention (Sec. 3.3).

Attention is pinned against scipy's softmax on the original data when every
page is FP8 and the data is exactly representable (lossless case), plus the
closed forms seq_len = 1 and identical keys; the merge (Eq. softmax-merge) is
pinned by split invariance; the state machine by the tiny workload's closed-form
tier map, allocation order and physical-id permutation invariance.
"""
import numpy as np
import pytest
from scipy.special import softmax

import mkv_workloads as wl


def _pool(orc, d=128, hq=8, hkv=1, n_fp8=256, n_tq3=256, W=256, layers=1, seed=0,
          orders=True):
    rng = np.random.default_rng(seed)
    sigma = np.where(rng.integers(0, 2, d) == 1, 1, -1).astype(np.int8)
    o8 = rng.permutation(n_fp8) if orders else None
    o3 = rng.permutation(n_tq3) if orders else None
    return orc.Pool(layers, hq, hkv, d, n_fp8, n_tq3, W, sigma, o8, o3)


def _fill(orc, P, lens, k, v, max_pages):
    n_req = len(lens)
    bt = np.full((n_req, max_pages), -1, np.int32)
    tags = np.full((n_req, max_pages), orc.TAG_NONE, np.uint8)
    cu = np.r_[0, np.cumsum(lens)].astype(np.int32)
    rc = P.append(-1, bt, tags, np.zeros(n_req, np.int32), cu, k, v)
    assert rc == 0
    return bt, tags


def test_tiny_workload_tier_map_closed_form(orc):
    """Config 1: pages 0-3 Anchor, 4-111 Stale, 112-127 Recent."""
    w = wl.workload(1)
    P = orc.Pool(1, w.n_q_heads, w.n_kv_heads, w.head_dim, 128, 128, w.recent, wl.rot_signs(w),
                 wl.free_order(w, 128, "fp8"), wl.free_order(w, 128, "tq3"))
    k, v = wl.kv_layer(w, 0, 2048)
    bt, tags = _fill(orc, P, [2048], k[None], v[None], 128)
    assert np.all(tags == orc.TAG_R)
    am = wl.anchor_mask(w, 128)
    n = P.migrate(bt, tags, am, np.array([2048], np.int32))
    assert n == 108
    want = np.full(128, orc.TAG_S, np.uint8)
    want[:4] = orc.TAG_A
    want[112:] = orc.TAG_R
    assert np.array_equal(tags[0], want)
    # TQ3 ids handed out in the pool's order, in ascending logical page order
    assert np.array_equal(bt[0, 4:112], wl.free_order(w, 128, "tq3")[:108])
    # released FP8 ids pushed in the same order: the stack top is the last one
    assert P.fp8_top[0] == 108
    assert np.array_equal(P.fp8_stack[:108], bt_fp8_ids_of(orc, w)[4:112])


def bt_fp8_ids_of(orc, w):
    return wl.free_order(w, 128, "fp8")[:128]


def test_partition_is_stable_and_complete(orc):
    rng = np.random.default_rng(1)
    n_req, mp = 5, 70
    tags = rng.choice([orc.TAG_R, orc.TAG_A, orc.TAG_S], size=(n_req, mp)).astype(np.uint8)
    bt = rng.integers(0, 1000, size=(n_req, mp)).astype(np.int32)
    lens = rng.integers(1, mp * 16 + 1, size=n_req).astype(np.int32)
    o8, o3, cnt = orc.partition(bt, tags, lens)
    for r in range(n_req):
        npg = (lens[r] + 15) // 16
        pages = list(range(npg))
        want8 = [(p, bt[r, p]) for p in pages if tags[r, p] != orc.TAG_S]
        want3 = [(p, bt[r, p]) for p in pages if tags[r, p] == orc.TAG_S]
        assert cnt[r, 0] == len(want8) and cnt[r, 1] == len(want3)
        assert [tuple(x) for x in o8[r, :cnt[r, 0]]] == want8
        assert [tuple(x) for x in o3[r, :cnt[r, 1]]] == want3


@pytest.mark.parametrize("d", (128, 256))
def test_lossless_fp8_attention_equals_dense_softmax(orc, d):
    """All pages FP8 and every value exactly E4M3 with power-of-two page
    scales: the oracle's paged attention must equal dense softmax on the data."""
    rng = np.random.default_rng(d)
    hq, hkv, L = 4, 2, 200
    P = _pool(orc, d=d, hq=hq, hkv=hkv, W=10 ** 6)
    # values: e4m3 grid values times 2^-3; every 16-token page-head contains 448
    vals = orc.e4m3_to_f64(rng.integers(0, 0x7E, size=(2, L, hkv, d)).astype(np.uint8))
    vals *= rng.choice([-1, 1], size=vals.shape)
    vals[:, ::16, :, 0] = 448.0
    vals *= 2.0 ** -3
    kv = vals.astype(np.float32)
    kb = wl.bf16_round(kv[0])
    vb = wl.bf16_round(kv[1])
    assert np.array_equal(wl.bf16_to_f32(kb), kv[0])
    bt, tags = _fill(orc, P, [L], kb[None], vb[None], 32)
    q = wl.bf16_round(rng.standard_normal((1, hq, d)).astype(np.float32))
    out, lse = P.decode(0, q, bt, tags, np.array([L], np.int32))
    qf = wl.bf16_to_f32(q).astype(np.float64)
    for h in range(hq):
        kh = kv[0][:, h // (hq // hkv)].astype(np.float64)
        vh = kv[1][:, h // (hq // hkv)].astype(np.float64)
        s = kh @ qf[0, h] / np.sqrt(d)
        ref = softmax(s) @ vh
        assert np.allclose(out[0, h], ref, rtol=0, atol=1e-12)
        assert np.isclose(lse[0, h], np.log(np.sum(np.exp(s - s.max()))) + s.max(), atol=1e-12)


def test_seq_len_one_and_identical_keys(orc):
    d = 128
    P = _pool(orc, d=d, hq=2, hkv=1, W=10 ** 6)
    rng = np.random.default_rng(2)
    k = wl.bf16_round(rng.standard_normal((40, 1, d)).astype(np.float32))
    v = wl.bf16_round(rng.standard_normal((40, 1, d)).astype(np.float32))
    k[:] = k[0]  # identical keys
    bt, tags = _fill(orc, P, [40], k[None], v[None], 8)
    q = wl.bf16_round(rng.standard_normal((1, 2, d)).astype(np.float32))
    out1, _ = P.decode(0, q, bt, tags, np.array([1], np.int32))
    _, vh = P.reconstruct(0, 0, 0, bt, tags, 40)
    assert np.allclose(out1[0, 0], vh[0], atol=1e-15)
    out, _ = P.decode(0, q, bt, tags, np.array([40], np.int32))
    # every page-head shares one K scale only if amax matches: compare to the
    # mean of the reconstructed values weighted by softmax of reconstructed keys
    kh, vh = P.reconstruct(0, 0, 0, bt, tags, 40)
    if np.all(kh == kh[0]):
        assert np.allclose(out[0, 0], vh.mean(0), atol=1e-12)
    s = kh @ wl.bf16_to_f32(q[0, 0]).astype(np.float64) / np.sqrt(d)
    assert np.allclose(out[0, 0], softmax(s) @ vh, atol=1e-12)


def test_merge_split_invariance(orc):
    rng = np.random.default_rng(4)
    d, n = 64, 300
    s = rng.standard_normal(n) * 3
    v = rng.standard_normal((n, d))
    ref = softmax(s) @ v
    for _ in range(20):
        cuts = np.sort(rng.choice(np.arange(1, n), size=rng.integers(1, 12), replace=False))
        parts = np.split(np.arange(n), cuts)
        parts.append(np.arange(0))  # an empty split is skipped
        m = np.array([s[p].max() if p.size else -np.inf for p in parts])
        l = np.array([np.exp(s[p] - s[p].max()).sum() if p.size else 0.0 for p in parts])
        ob = np.array([(np.exp(s[p] - s[p].max()) @ v[p]) / l[i] if p.size else np.zeros(d)
                       for i, p in enumerate(parts)])
        out, lse = orc.merge(m, l, ob)
        assert np.allclose(out, ref, atol=1e-12)
        assert np.isclose(lse, np.log(np.exp(s - s.max()).sum()) + s.max())


def test_mixed_attention_invariant_to_physical_ids(orc):
    """Same logical cache under two different free-list orders -> same outputs."""
    w = wl.scaled(wl.workload(2), (700,), n_layers=1)
    w = wl.Workload(**{**w.__dict__, "recent": 128})
    k, v = wl.kv_layer(w, 0, 700)
    q = wl.q_decode(w, 0)
    outs = []
    for seed in (0, 1):
        P = _pool(orc, d=256, hq=24, hkv=4, n_fp8=64, n_tq3=64, W=128, seed=seed)
        P.sigma[:] = wl.rot_signs(w)
        bt, tags = _fill(orc, P, [700], k[None], v[None], 44)
        am = wl.anchor_mask(w, 44)
        P.migrate(bt, tags, am, np.array([700], np.int32))
        assert (tags == orc.TAG_S).sum() > 20
        outs.append(P.decode(0, q, bt, tags, np.array([700], np.int32))[0])
    assert np.array_equal(outs[0], outs[1])


def test_append_partial_pages_and_rescale(orc):
    """Partial-page append: scales only grow; a later append that does not
    exceed the page's range keeps earlier codes; requantisation is used only
    when the new amax exceeds 448 * s_old."""
    d = 128
    P = _pool(orc, d=d, hq=1, hkv=1, W=10 ** 6, orders=False)
    rng = np.random.default_rng(12)
    bt = np.full((1, 4), -1, np.int32)
    tags = np.full((1, 4), orc.TAG_NONE, np.uint8)
    x1 = wl.bf16_round(rng.standard_normal((5, 1, d)).astype(np.float32))
    assert P.append(-1, bt, tags, np.array([0], np.int32), np.array([0, 5], np.int32),
                    x1[None], x1[None]) == 0
    id0 = bt[0, 0]
    s1 = P.fp8_scale[0, id0, 0, 0]
    codes1 = P.fp8[0, id0, 0, :5 * d].copy()
    x2 = wl.bf16_round(0.5 * rng.standard_normal((3, 1, d)).astype(np.float32))
    x2[0, 0, 0] = 0.0
    assert P.append(-1, bt, tags, np.array([5], np.int32), np.array([0, 3], np.int32),
                    x2[None], x2[None]) == 0
    if np.abs(wl.bf16_to_f32(x2)).max() <= 448 * s1:
        assert P.fp8_scale[0, id0, 0, 0] == s1
        assert np.array_equal(P.fp8[0, id0, 0, :5 * d], codes1)
    x3 = wl.bf16_round(10 * rng.standard_normal((20, 1, d)).astype(np.float32))
    assert P.append(-1, bt, tags, np.array([8], np.int32), np.array([0, 20], np.int32),
                    x3[None], x3[None]) == 0
    s3 = P.fp8_scale[0, id0, 0, 0]
    assert s3 > s1
    assert bt[0, 1] >= 0 and tags[0, 1] == orc.TAG_R
    # requantised old codes equal E4M3(dequant(code) * s_old / s_new) in fp32
    old = orc.e4m3_to_f64(codes1[:d]).astype(np.float32) * np.float32(s1)
    want = orc.e4m3_from_f32((old / np.float32(s3)).astype(np.float32))
    assert np.array_equal(P.fp8[0, id0, 0, :d], want)
    # all-zero tokens -> scale 0 and zero codes
    P2 = _pool(orc, d=d, hq=1, hkv=1, W=10 ** 6, orders=False)
    bt2 = np.full((1, 2), -1, np.int32)
    tg2 = np.full((1, 2), orc.TAG_NONE, np.uint8)
    z = np.zeros((1, 3, 1, d), np.uint16)
    assert P2.append(-1, bt2, tg2, np.array([0], np.int32), np.array([0, 3], np.int32), z, z) == 0
    assert P2.fp8_scale[0, bt2[0, 0], 0, 0] == 0.0


def test_append_and_migrate_fail_closed(orc):
    d = 128
    P = _pool(orc, d=d, hq=1, hkv=1, n_fp8=2, n_tq3=1, W=16, orders=False)
    bt = np.full((1, 8), -1, np.int32)
    tags = np.full((1, 8), orc.TAG_NONE, np.uint8)
    x = np.zeros((1, 48, 1, d), np.uint16)
    before = (bt.copy(), tags.copy(), P.fp8_top.copy())
    assert P.append(-1, bt, tags, np.array([0], np.int32), np.array([0, 48], np.int32), x, x) == 1
    assert np.array_equal(bt, before[0]) and np.array_equal(tags, before[1])
    assert P.fp8_top[0] == before[2][0]
    x = np.zeros((1, 32, 1, d), np.uint16)
    assert P.append(-1, bt, tags, np.array([0], np.int32), np.array([0, 32], np.int32), x, x) == 0
    # window of 16 tokens: page 0 leaves it once seq_len >= 32; TQ3 pool holds 1 page
    assert P.migrate(bt, tags, None, np.array([32], np.int32)) == 1
    assert tags[0, 0] == orc.TAG_S and tags[0, 1] == orc.TAG_R
