"""Pins for the oracle's reference-counted pools and shared prefixes (Alg. 1
SealPrefix and Finish; Sec. 4.4 prefix reuse).

* Conservation: after every call, each page's count equals its block-table
  references plus the cache references the test holds, and the free lists
  hold exactly the pages with count 0, each once.
* A request attached to a sealed prefix attends to the shared pages in place:
  its decode equals, bit for bit, the decode of a request that appended the
  same tokens itself.
* Shared pages are immutable: Retier and Promote leave them alone until the
  cache's reference is dropped.
* Release order: a page returns to its free list when its last listed
  reference goes; over-release and acquiring a free page change nothing.
"""
import numpy as np

import mkv_workloads as wl

PAGE = 16


def _check_conservation(orc, P, tables, cache):
    """tables: list of (bt, tags); cache: list of (id, tag) references held."""
    want8 = np.zeros(P.n_fp8, np.int64)
    want3 = np.zeros(P.n_tq3, np.int64)
    for bt, tags in tables:
        m = bt >= 0
        for i, t in zip(bt[m], tags[m]):
            (want3 if t == orc.TAG_S else want8)[i] += 1
    for i, t in cache:
        (want3 if t == orc.TAG_S else want8)[i] += 1
    assert np.array_equal(P.rc8[:P.n_fp8], want8)
    assert np.array_equal(P.rc3[:P.n_tq3], want3)
    f8 = P.fp8_stack[:P.fp8_top[0]]
    f3 = P.tq3_stack[:P.tq3_top[0]]
    assert len(set(f8.tolist())) == len(f8) and set(f8.tolist()) == set(np.flatnonzero(want8 == 0))
    assert len(set(f3.tolist())) == len(f3) and set(f3.tolist()) == set(np.flatnonzero(want3 == 0))


def test_prefix_share_seal_finish_lifecycle(orc):
    w = wl.scaled(wl.workload(2), (300,), n_layers=2)
    d, hq, hkv, W = w.head_dim, w.n_q_heads, w.n_kv_heads, 64
    mp = 40
    P = orc.Pool(2, hq, hkv, d, 80, 80, W, wl.rot_signs(w), wl.free_order(w, 80, "fp8"),
                 wl.free_order(w, 80, "tq3"))
    # request A: 300 tokens (18 full pages + 12 tokens)
    kA, vA = zip(*(wl.kv_layer(w, l, 300) for l in range(2)))
    kA, vA = np.stack(kA), np.stack(vA)
    btA = np.full((1, mp), -1, np.int32)
    tgA = np.full((1, mp), orc.TAG_NONE, np.uint8)
    assert P.append(-1, btA, tgA, np.array([0], np.int32), np.array([0, 300], np.int32), kA, vA) == 0
    _check_conservation(orc, P, [(btA, tgA)], [])
    # SealPrefix: the cache takes a reference on A's 16 first (full) pages
    cache = [(int(btA[0, p]), int(tgA[0, p])) for p in range(16)]
    assert P.acquire([c[0] for c in cache], [c[1] for c in cache]) == 0
    _check_conservation(orc, P, [(btA, tgA)], cache)
    # Retier of A leaves the shared pages alone (every page still Recent FP8)
    assert P.migrate(btA, tgA, None, np.array([300], np.int32)) == 0
    assert (tgA[0, :19] == orc.TAG_R).all()
    # Finish(A): its 19 references go; the 3 unshared pages return to the list
    top8 = P.fp8_top[0]
    priv = btA[0, 16:19].copy()
    assert P.finish([0], btA, tgA) == 3
    assert (btA == -1).all() and (tgA == orc.TAG_NONE).all()
    assert np.array_equal(P.fp8_stack[top8:top8 + 3], priv)  # ascending page order
    _check_conservation(orc, P, [(btA, tgA)], cache)
    # request B hits the cached prefix: installs the 16 pages, acquires them,
    # then appends its own 100 tokens after position 256
    btB = np.full((1, mp), -1, np.int32)
    tgB = np.full((1, mp), orc.TAG_NONE, np.uint8)
    btB[0, :16] = [c[0] for c in cache]
    tgB[0, :16] = orc.TAG_R
    assert P.acquire(btB[0, :16], tgB[0, :16]) == 0
    kB, vB = zip(*(wl.kv_layer(w, l, 100, token_offset=5000) for l in range(2)))
    kB, vB = np.stack(kB), np.stack(vB)
    assert P.append(-1, btB, tgB, np.array([256], np.int32), np.array([0, 100], np.int32), kB, vB) == 0
    _check_conservation(orc, P, [(btB, tgB)], cache)
    # the same tokens appended by a request of its own in a fresh pool
    Q = orc.Pool(2, hq, hkv, d, 80, 80, W, wl.rot_signs(w))
    btC = np.full((1, mp), -1, np.int32)
    tgC = np.full((1, mp), orc.TAG_NONE, np.uint8)
    assert Q.append(-1, btC, tgC, np.array([0], np.int32), np.array([0, 256], np.int32),
                    kA[:, :256], vA[:, :256]) == 0
    assert Q.append(-1, btC, tgC, np.array([256], np.int32), np.array([0, 100], np.int32), kB, vB) == 0
    q = wl.q_decode(w, 1)
    oB, lB = P.decode(1, q, btB, tgB, np.array([356], np.int32))
    oC, lC = Q.decode(1, q, btC, tgC, np.array([356], np.int32))
    assert np.array_equal(oB, oC) and np.array_equal(lB, lC)
    # Retier of B: the shared prefix stays FP8; B's own old pages are encoded
    assert P.migrate(btB, tgB, None, np.array([356], np.int32)) == 2  # pages 16, 17
    assert (tgB[0, :16] == orc.TAG_R).all() and (tgB[0, 16:18] == orc.TAG_S).all()
    # Promote does not touch shared pages either
    mask = np.ones_like(tgB)
    assert P.promote(btB, tgB, mask, np.array([356], np.int32)) == 2
    assert (tgB[0, 16:18] == orc.TAG_A).all()
    _check_conservation(orc, P, [(btB, tgB)], cache)
    # prefix eviction: the cache drops its references; B owns the pages alone,
    # so the next Retier encodes the old ones
    assert P.release([c[0] for c in cache], [c[1] for c in cache]) == 0
    cache = []
    _check_conservation(orc, P, [(btB, tgB)], cache)
    assert P.migrate(btB, tgB, None, np.array([356], np.int32)) == 16
    assert (tgB[0, :16] == orc.TAG_S).all()
    _check_conservation(orc, P, [(btB, tgB)], cache)
    # Finish(B): everything returns
    assert P.finish([0], btB, tgB) == 16 + 2 + 5
    assert P.fp8_top[0] == 80 and P.tq3_top[0] == 80
    _check_conservation(orc, P, [(btB, tgB)], cache)


def test_release_order_and_fail_closed(orc):
    d = 128
    P = orc.Pool(1, 2, 1, d, 8, 4, 10 ** 6, np.ones(d, np.int8))
    bt = np.full((2, 4), -1, np.int32)
    tags = np.full((2, 4), orc.TAG_NONE, np.uint8)
    x = np.zeros((1, 32, 1, d), np.uint16)
    assert P.append(-1, bt, tags, np.zeros(2, np.int32), np.array([0, 32, 32], np.int32), x, x) == 0
    a, b = int(bt[0, 0]), int(bt[0, 1])
    # request 1 shares request 0's two pages
    bt[1, :2] = bt[0, :2]
    tags[1, :2] = orc.TAG_R
    assert P.acquire([a, b], [orc.TAG_R, orc.TAG_R]) == 0
    assert P.rc8[a] == 2 and P.rc8[b] == 2
    # acquiring a free page, or with a bad tag / id: nothing changes
    free_id = int(P.fp8_stack[0])
    assert P.acquire([a, free_id], [orc.TAG_R, orc.TAG_R]) == -1 and P.rc8[a] == 2
    assert P.acquire([a], [0x7]) == -1 and P.acquire([99], [orc.TAG_R]) == -1
    # over-release: nothing changes
    top = P.fp8_top[0]
    assert P.release([a, a, a], [orc.TAG_R] * 3) == -1
    assert P.rc8[a] == 2 and P.fp8_top[0] == top
    # both requests finish together: each page goes at its second entry, in
    # ascending (request, page) order: a (request 1 page 0), then b
    assert P.finish([0, 1], bt, tags) == 2
    assert list(P.fp8_stack[top:top + 2]) == [a, b]
    assert P.fp8_top[0] == 8 and (P.rc8 == 0).all()
