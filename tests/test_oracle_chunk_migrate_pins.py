"""Pins for the oracle's causal chunk attention (Sec. 3.3 causal mask), its
FP8 -> TQ3 migration (Alg. 1 Retier, Sec. 4.3 normalize-rotate-pack) and its
mixed-format decode (Sec. 3.3, Eq. softmax-merge), each checked against
something other than the oracle's own pool code:

* chunk attention with lossless FP8 pages equals scipy's dense causal softmax
  on the original data, for ragged requests and chunks;
* a migrated page-head's TQ3 region equals tq3_pack(tq3_encode(...)) of the
  page's logical FP8 codes recomputed here from the bf16 input and the scale
  rule (s = amax / 448, code = E4M3(x / s)), whatever the request order;
* mixed decode equals numpy's softmax over keys and values rebuilt here from
  tq3_dequant (Stale pages) and code * scale (FP8 pages).
"""
import numpy as np
import pytest
from scipy.special import softmax

import mkv_workloads as wl

PAGE = 16


def _pool(orc, d, hq, hkv, n_fp8, n_tq3, W, seed=0, layers=1):
    rng = np.random.default_rng(seed)
    sigma = np.where(rng.integers(0, 2, d) == 1, 1, -1).astype(np.int8)
    return orc.Pool(layers, hq, hkv, d, n_fp8, n_tq3, W, sigma, rng.permutation(n_fp8),
                    rng.permutation(n_tq3))


def _lossless_kv(orc, rng, n_tok, hkv, d):
    """bf16-exact values on the E4M3 grid times 2^-3, every 16-token page-head
    holding 448 * 2^-3: the FP8 scale is 2^-3 and storage is lossless."""
    vals = orc.e4m3_to_f64(rng.integers(0, 0x7E, size=(2, n_tok, hkv, d)).astype(np.uint8))
    vals *= rng.choice([-1, 1], size=vals.shape)
    vals[:, ::16, :, 0] = 448.0
    vals *= 2.0 ** -3
    kv = vals.astype(np.float32)
    kb, vb = wl.bf16_round(kv[0]), wl.bf16_round(kv[1])
    assert np.array_equal(wl.bf16_to_f32(kb), kv[0]) and np.array_equal(wl.bf16_to_f32(vb), kv[1])
    return kv, kb, vb


@pytest.mark.parametrize("d", (128, 256))
def test_chunk_lossless_equals_dense_causal_softmax(orc, d):
    """Ragged requests and chunks (1, 5, 16 and 37 queries; lengths inside and
    at page boundaries): every chunk row equals dense causal softmax, query i
    of a chunk of n at position L - n + i seeing keys 0 .. L - n + i."""
    rng = np.random.default_rng(100 + d)
    hq, hkv = 4, 2
    lens, nq = [37, 80, 129, 16], [5, 16, 37, 1]
    mp = max((L + PAGE - 1) // PAGE for L in lens)
    n_pg = sum((L + PAGE - 1) // PAGE for L in lens) + 4
    P = _pool(orc, d, hq, hkv, n_pg, n_pg, 10 ** 6, seed=d)
    kvs = [_lossless_kv(orc, rng, L, hkv, d) for L in lens]
    kb = np.concatenate([x[1] for x in kvs])
    vb = np.concatenate([x[2] for x in kvs])
    bt = np.full((len(lens), mp), -1, np.int32)
    tags = np.full((len(lens), mp), orc.TAG_NONE, np.uint8)
    cu = np.r_[0, np.cumsum(lens)].astype(np.int32)
    assert P.append(-1, bt, tags, np.zeros(len(lens), np.int32), cu, kb[None], vb[None]) == 0
    q = wl.bf16_round(rng.standard_normal((sum(nq), hq, d)).astype(np.float32))
    cq = np.r_[0, np.cumsum(nq)].astype(np.int32)
    out = P.chunk(0, q, cq, bt, tags, np.array(lens, np.int32))
    qf = wl.bf16_to_f32(q).astype(np.float64)
    G = hq // hkv
    for r, (L, n) in enumerate(zip(lens, nq)):
        kv = kvs[r][0].astype(np.float64)
        for i in range(n):
            pos = L - n + i
            for h in range(hq):
                s = kv[0][: pos + 1, h // G] @ qf[cq[r] + i, h] / np.sqrt(d)
                ref = softmax(s) @ kv[1][: pos + 1, h // G]
                assert np.allclose(out[cq[r] + i, h], ref, rtol=0, atol=1e-12), (r, i, h)


def _mixed_pool(orc, d, hq, hkv, lens, W, seed):
    mp = max((L + PAGE - 1) // PAGE for L in lens)
    n_pg = sum((L + PAGE - 1) // PAGE for L in lens) + 4
    P = _pool(orc, d, hq, hkv, n_pg, n_pg, W, seed=seed)
    rng = np.random.default_rng(seed)
    k = wl.bf16_round((rng.standard_normal((sum(lens), hkv, d)) *
                       np.exp(0.5 * rng.standard_normal(d))).astype(np.float32))
    v = wl.bf16_round(rng.standard_normal((sum(lens), hkv, d)).astype(np.float32))
    bt = np.full((len(lens), mp), -1, np.int32)
    tags = np.full((len(lens), mp), orc.TAG_NONE, np.uint8)
    cu = np.r_[0, np.cumsum(lens)].astype(np.int32)
    assert P.append(-1, bt, tags, np.zeros(len(lens), np.int32), cu, k[None], v[None]) == 0
    return P, k, v, bt, tags, cu


def _logical_fp8(orc, x_bf16):
    """FP8 scale and codes of one full page-head of K or V by the scale rule:
    s = amax / 448 in fp32, code = E4M3(x / s) with one fp32 division."""
    x = wl.bf16_to_f32(x_bf16)
    amax = np.float32(np.abs(x).max())
    s = np.float32(amax / np.float32(448.0))
    codes = orc.e4m3_from_f32((x / s).astype(np.float32)) if s > 0 else np.zeros(x.shape, np.uint8)
    return s, codes


@pytest.mark.parametrize("d", (128, 256))
def test_migrate_equals_direct_encode(orc, d):
    """C-16 / Alg. 1 Retier: every migrated page-head's TQ3 region equals the
    direct encoding of that page's FP8 codes (K codes with the K scale, V codes
    with the V scale), recomputed here from the input; the result does not
    depend on the order of the requests in the call."""
    hq, hkv, W = 4, 2, 32
    lens = [100, 64, 161]
    P, k, v, bt, tags, cu = _mixed_pool(orc, d, hq, hkv, lens, W, seed=7 + d)
    anchor = np.zeros_like(tags)
    anchor[0, 1] = 1
    P2 = _pool(orc, d, hq, hkv, P.n_fp8, P.n_tq3, W, seed=99)
    P2.sigma[:] = P.sigma
    # second pool: same requests in reverse order
    order = [2, 1, 0]
    lens2 = [lens[r] for r in order]
    k2 = np.concatenate([k[cu[r]:cu[r + 1]] for r in order])
    v2 = np.concatenate([v[cu[r]:cu[r + 1]] for r in order])
    bt2 = np.full_like(bt, -1)
    tags2 = np.full_like(tags, orc.TAG_NONE)
    cu2 = np.r_[0, np.cumsum(lens2)].astype(np.int32)
    assert P2.append(-1, bt2, tags2, np.zeros(3, np.int32), cu2, k2[None], v2[None]) == 0
    sl = np.array(lens, np.int32)
    n = P.migrate(bt, tags, anchor, sl)
    n2 = P2.migrate(bt2, tags2, anchor[order], sl[order])
    assert n == n2 > 0
    assert tags[0, 1] == orc.TAG_A
    checked = 0
    for r, L in enumerate(lens):
        r2 = order.index(r)
        for p in range((L + PAGE - 1) // PAGE):
            if tags[r, p] != orc.TAG_S:
                continue
            assert (p + 1) * PAGE <= L - W and tags2[r2, p] == orc.TAG_S
            for h in range(hkv):
                rows = slice(cu[r] + PAGE * p, cu[r] + PAGE * (p + 1))
                sK, k8 = _logical_fp8(orc, k[rows, h])
                sV, v8 = _logical_fp8(orc, v[rows, h])
                enc = orc.tq3_encode(d, k8, sK, v8, sV, P.sigma)
                want = orc.tq3_pack(d, enc)
                assert np.array_equal(P.tq3[0, bt[r, p], h], want), (r, p, h)
                assert np.array_equal(P2.tq3[0, bt2[r2, p], h], want), (r, p, h)
                checked += 1
    assert checked == n * hkv


@pytest.mark.parametrize("d", (128, 256))
def test_mixed_decode_equals_softmax_over_dequantized_pages(orc, d):
    """Decode over FP8 and TQ3 pages equals softmax attention over keys and
    values rebuilt page by page: tq3_dequant(tq3_encode(codes)) for Stale
    pages, E4M3 code * scale for Recent/Anchor pages."""
    hq, hkv, W = 4, 2, 48
    lens = [161, 70]
    P, k, v, bt, tags, cu = _mixed_pool(orc, d, hq, hkv, lens, W, seed=3 + d)
    anchor = np.zeros_like(tags)
    anchor[1, 0] = 1
    sl = np.array(lens, np.int32)
    assert P.migrate(bt, tags, anchor, sl) > 0
    rng = np.random.default_rng(5)
    q = wl.bf16_round(rng.standard_normal((len(lens), hq, d)).astype(np.float32))
    out, lse = P.decode(0, q, bt, tags, sl)
    G = hq // hkv
    for r, L in enumerate(lens):
        for h in range(hkv):
            kh = np.zeros((L, d))
            vh = np.zeros((L, d))
            for p in range((L + PAGE - 1) // PAGE):
                t0, t1 = PAGE * p, min(L, PAGE * (p + 1))
                rows = slice(cu[r] + t0, cu[r] + t1)
                sK, k8 = _logical_fp8(orc, k[rows, h])
                sV, v8 = _logical_fp8(orc, v[rows, h])
                if tags[r, p] == orc.TAG_S:
                    enc = orc.tq3_encode(d, k8, sK, v8, sV, P.sigma)
                    a, b = orc.tq3_dequant(d, enc, P.sigma)
                else:
                    a = orc.e4m3_to_f64(k8) * np.float64(sK)
                    b = orc.e4m3_to_f64(v8) * np.float64(sV)
                kh[t0:t1], vh[t0:t1] = a[: t1 - t0], b[: t1 - t0]
            for j in range(G):
                hh = h * G + j
                s = kh @ wl.bf16_to_f32(q[r, hh]).astype(np.float64) / np.sqrt(d)
                assert np.allclose(out[r, hh], softmax(s) @ vh, rtol=0, atol=1e-12)
                assert np.isclose(lse[r, hh], s.max() + np.log(np.exp(s - s.max()).sum()),
                                  rtol=0, atol=1e-12)
    assert (tags == orc.TAG_S).sum() >= 5


def test_chunk_single_query_equals_decode_on_mixed_pages(orc):
    """A chunk of one query per request (Stale TQ3 pages included) equals
    decode for that query: the chunk's last query sees the whole context."""
    d, hq, hkv, W = 256, 6, 1, 32
    lens = [150, 47]
    P, k, v, bt, tags, cu = _mixed_pool(orc, d, hq, hkv, lens, W, seed=11)
    sl = np.array(lens, np.int32)
    assert P.migrate(bt, tags, None, sl) > 0
    rng = np.random.default_rng(6)
    q = wl.bf16_round(rng.standard_normal((len(lens), hq, d)).astype(np.float32))
    oc = P.chunk(0, q, np.arange(len(lens) + 1, dtype=np.int32), bt, tags, sl)
    od, _ = P.decode(0, q, bt, tags, sl)
    assert np.array_equal(oc, od)
