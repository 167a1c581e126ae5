"""Pins for the oracle's Promote transition (Alg. 1 Promote; Sec. 3.1, a Stale
page that re-enters the protected budget is materialized into FP8).

* A key that is a basis vector comes back as that basis vector, with the norm
  of the original key up to the binary16 rounding of the norm correction.
* The fp32 reconstruction agrees with tq3_dequant (one fp32 rounding) and
  keeps every key's norm (to binary16 precision).
* The new FP8 page follows the scale rule of a fresh page: s = amax / 448 in
  fp32, code = E4M3(x / s), recomputed here with numpy.
* Pool state: tag Anchor, FP8 ids popped and TQ3 ids pushed in ascending
  (request, page) order, non-Stale and out-of-range pages untouched, and a
  call the FP8 free list cannot serve changes nothing.
"""
import numpy as np
import pytest

import mkv_workloads as wl

PAGE = 16


def _pool(orc, d, hq, hkv, n_fp8, n_tq3, W, seed=0):
    rng = np.random.default_rng(seed)
    sigma = np.where(rng.integers(0, 2, d) == 1, 1, -1).astype(np.int8)
    return orc.Pool(1, hq, hkv, d, n_fp8, n_tq3, W, sigma, rng.permutation(n_fp8),
                    rng.permutation(n_tq3))


def _fill(orc, P, lens, k, v):
    mp = max((L + PAGE - 1) // PAGE for L in lens)
    bt = np.full((len(lens), mp), -1, np.int32)
    tags = np.full((len(lens), mp), orc.TAG_NONE, np.uint8)
    cu = np.r_[0, np.cumsum(lens)].astype(np.int32)
    assert P.append(-1, bt, tags, np.zeros(len(lens), np.int32), cu, k[None], v[None]) == 0
    return bt, tags


def _fp8_page(orc, P, pid, h, d):
    """(K values, V values) [16][d] in fp64 of an FP8 page-head, read through
    the layout functions."""
    reg = P.fp8[0, pid, h]
    sK, sV = P.fp8_scale[0, pid, h]
    kq = np.array([[reg[orc.fp8_k_off(d, t, c)] for c in range(d)] for t in range(PAGE)], np.uint8)
    vq = np.array([[reg[orc.fp8_v_off(d, t, c)] for c in range(d)] for t in range(PAGE)], np.uint8)
    return kq, vq, np.float32(sK), np.float32(sV)


def _rule(orc, x32):
    """FP8 scale rule of a fresh page-head on fp32 values."""
    amax = np.float32(np.abs(x32).max())
    s = np.float32(amax / np.float32(448.0))
    if s == 0:
        return s, np.zeros(x32.shape, np.uint8)
    return s, orc.e4m3_from_f32((x32 / s).astype(np.float32))


@pytest.mark.parametrize("d", (128, 256))
def test_promote_basis_vector_round_trip(orc, d):
    """Every token's key is +-56 e_j (channel j and sign drawn per token, 56 =
    448 / 8 so the FP8 scale is 1/8 and the key exact).  After Retier and
    Promote each key is the same basis vector with magnitude 56 up to the
    binary16 rounding of gamma; the page holds +-448 codes there and zeros
    elsewhere.  Values constant per channel come back through the binary16
    rounding of their FP8 values."""
    hkv, W = 1, 16
    rng = np.random.default_rng(d)
    P = _pool(orc, d, 2, hkv, 8, 8, W, seed=d)
    L = 2 * PAGE
    j = rng.integers(0, d, L)
    sgn = rng.choice([-1.0, 1.0], L)
    k = np.zeros((L, hkv, d), np.float32)
    k[np.arange(L), 0, j] = 56.0 * sgn
    vc = (rng.integers(-128, 128, d) / 16.0).astype(np.float32)  # bf16-exact
    v = np.broadcast_to(vc, (L, hkv, d)).astype(np.float32)
    bt, tags = _fill(orc, P, [L], wl.bf16_round(k), wl.bf16_round(v))
    sl = np.array([L], np.int32)
    assert P.migrate(bt, tags, None, sl) == 1 and tags[0, 0] == orc.TAG_S
    mask = np.ones_like(tags)
    assert P.promote(bt, tags, mask, sl) == 1
    assert tags[0, 0] == orc.TAG_A and tags[0, 1] == orc.TAG_R
    kq, vq, sK, sV = _fp8_page(orc, P, bt[0, 0], 0, d)
    kval = orc.e4m3_to_f64(kq) * np.float64(sK)
    for t in range(PAGE):
        want = np.zeros(d)
        want[j[t]] = 56.0 * sgn[t]
        assert kq[t, j[t]] == (0x7E if sgn[t] > 0 else 0xFE)
        assert np.count_nonzero(kval[t]) == 1  # the other channels are +-0
        assert abs(kval[t, j[t]] - want[j[t]]) <= 56.0 * (2.0 ** -11 + 2.0 ** -22)
    # values: each channel is constant, so its TQ3 scale is 0 and its zero is
    # the binary16 rounding (numpy's) of the FP8 value the page held; the
    # promoted page is the scale rule applied to those zeros
    s0, c0 = _rule(orc, np.broadcast_to(vc, (PAGE, d)).astype(np.float32))
    v8 = orc.e4m3_to_f64(c0) * np.float64(s0)
    zero = v8.astype(np.float16).astype(np.float32)
    s_v, codes = _rule(orc, zero)
    assert sV == s_v and np.array_equal(vq, codes)


@pytest.mark.parametrize("d", (128, 256))
def test_promote_reconstruction_norm_and_scale_rule(orc, d):
    """Random pages (log-normal channel scales): for every promoted page-head
    the fp32 reconstruction equals tq3_dequant to one fp32 rounding, keeps
    each key's norm (that of the FP8 key it was encoded from) to binary16
    precision, and the new FP8 page is the scale rule applied to it."""
    hkv, W = 2, 32
    rng = np.random.default_rng(10 + d)
    lens = [120, 75]
    n = sum(lens)
    P = _pool(orc, d, 4, hkv, 64, 64, W, seed=3 * d)
    k = (rng.standard_normal((n, hkv, d)) * np.exp(0.5 * rng.standard_normal(d))).astype(np.float32)
    v = rng.standard_normal((n, hkv, d)).astype(np.float32)
    bt, tags = _fill(orc, P, lens, wl.bf16_round(k), wl.bf16_round(v))
    sl = np.array(lens, np.int32)
    # FP8 keys of every page before migration
    fp8_before = {}
    for r, Lr in enumerate(lens):
        for p in range((Lr + PAGE - 1) // PAGE):
            for h in range(hkv):
                fp8_before[(r, p, h)] = _fp8_page(orc, P, bt[r, p], h, d)
    assert P.migrate(bt, tags, None, sl) > 0
    stale = np.argwhere(tags == orc.TAG_S)
    tq3_before = {(r, p, h): P.tq3[0, bt[r, p], h].copy() for r, p in stale for h in range(hkv)}
    mask = np.zeros_like(tags)
    for r, p in stale[::2]:
        mask[r, p] = 1
    n_pro = P.promote(bt, tags, mask, sl)
    assert n_pro == len(stale[::2])
    for r, p in stale[::2]:
        assert tags[r, p] == orc.TAG_A
        for h in range(hkv):
            enc = orc.tq3_unpack(d, tq3_before[(r, p, h)])
            k32, v32 = orc.tq3_reconstruct_f32(d, enc, P.sigma)
            kh, vh = orc.tq3_dequant(d, enc, P.sigma)
            assert np.all(np.abs(k32 - kh) <= 2.0 ** -23 * np.abs(kh) + 1e-30)
            assert np.all(np.abs(v32 - vh) <= 2.0 ** -24 * np.abs(vh))
            kq0, _, sK0, _ = fp8_before[(r, p, h)]
            n_orig = np.linalg.norm(orc.e4m3_to_f64(kq0) * np.float64(sK0), axis=1)
            n_rec = np.linalg.norm(k32.astype(np.float64), axis=1)
            assert np.all(np.abs(n_rec - n_orig) <= 2.0 ** -10 * n_orig)
            kq, vq, sK, sV = _fp8_page(orc, P, bt[r, p], h, d)
            s_k, ck = _rule(orc, k32)
            s_v, cv = _rule(orc, v32)
            assert sK == s_k and np.array_equal(kq, ck)
            assert sV == s_v and np.array_equal(vq, cv)


def test_promote_state_machine_and_fail_closed(orc):
    d, hkv, W = 128, 1, 16
    rng = np.random.default_rng(1)
    lens = [100, 70]
    n = sum(lens)
    P = _pool(orc, d, 2, hkv, 16, 16, W, seed=5)
    k = rng.standard_normal((n, hkv, d)).astype(np.float32)
    bt, tags = _fill(orc, P, lens, wl.bf16_round(k), wl.bf16_round(k))
    sl = np.array(lens, np.int32)
    anchor = np.zeros_like(tags)
    anchor[1, 0] = 1
    assert P.migrate(bt, tags, anchor, sl) == 5 + 2
    assert P.fp8_top[0] == 16 - 12 + 7
    # request 0: pages 0-4 Stale, 5-6 Recent; request 1: 0 Anchor, 1-2 Stale, 3-4 Recent
    mask = np.zeros_like(tags)
    mask[0, [1, 4, 6]] = 1   # page 6 is Recent: untouched
    mask[1, [0, 2]] = 1      # page 0 is an Anchor already: untouched
    bt0, tags0 = bt.copy(), tags.copy()
    top8, top3 = P.fp8_top[0], P.tq3_top[0]
    stack8 = P.fp8_stack[:top8].copy()
    assert P.promote(bt, tags, mask, sl) == 3
    promoted = [(0, 1), (0, 4), (1, 2)]
    for i, (r, p) in enumerate(promoted):
        assert tags[r, p] == orc.TAG_A
        assert bt[r, p] == stack8[top8 - 1 - i]
        assert P.tq3_stack[top3 + i] == bt0[r, p]
    changed = (bt != bt0) | (tags != tags0)
    assert changed.sum() == 3
    assert P.fp8_top[0] == top8 - 3 and P.tq3_top[0] == top3 + 3
    # a later Retier leaves the promoted (Anchor) pages alone
    assert P.migrate(bt, tags, anchor, sl) == 0
    # the FP8 free list cannot hold the request: nothing changes
    mask[:] = 0
    mask[tags == orc.TAG_S] = 1
    P.fp8_top[0] = 1
    bt1, tags1 = bt.copy(), tags.copy()
    assert P.promote(bt, tags, mask, sl) == -1
    assert np.array_equal(bt, bt1) and np.array_equal(tags, tags1) and P.fp8_top[0] == 1
