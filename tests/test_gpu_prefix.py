"""GPU parity of reference-counted pools and shared prefixes (Alg. 1
SealPrefix and Finish; Sec. 4.4 prefix reuse) against the oracle: block
tables, tags, free lists, reference counts and pages bit for bit after every
call, decode over shared pages within 1e-3."""
import numpy as np
import pytest

import mkv_workloads as wl
from _harness import max_abs

pytestmark = pytest.mark.gpu

TOL = 1e-3


def _check(tw, what, decode_reqs=None):
    tw.check_tables()
    tw.check_refcounts()
    tw.check_pages()
    if decode_reqs:
        res = tw.decode(layer=1)
        err = max(max_abs(res["out"][decode_reqs], res["ref_out"][decode_reqs]),
                  max_abs(res["lse"][decode_reqs], res["ref_lse"][decode_reqs]))
        print(f"  {what}: decode max|dO|, max|dlse| {err:.2e}", flush=True)
        assert np.all(np.isfinite(res["out"][decode_reqs])) and err <= TOL
        # rows of finished requests (length 0) are decoded too and flag a range error
        import paper_2608_23834_amd as mk
        e = mk.kv_pool_check_errors(tw.gpu, clear=True)
        assert e in (0, mk.DEVERR["RANGE"]), e


def test_prefix_lifecycle_matches_oracle():
    from _harness import Twin
    w = wl.workload(2)
    print(f"\n[prefix] {w.name}", flush=True)
    tw = Twin(w, n_layers=2, lens=[300, 400, 400], recent=64, n_fp8=120, n_tq3=120)
    tw.fill_to([300, 0, 0])
    _check(tw, "A appended")
    cache_ids = tw.obt[0, :16].copy()
    cache_tags = np.full(16, 0, np.uint8)
    tw.acquire(cache_ids, cache_tags)                     # SealPrefix
    tw.migrate()                                          # shared pages stay
    _check(tw, "sealed, Retier")
    assert (tw.otags[0, :16] < 2).all()  # FP8: Recent, or Anchor (first four pages)
    tw.finish([0])                                        # Finish(A)
    _check(tw, "A finished")
    for r, extra in ((1, 100), (2, 50)):                  # two requests hit the prefix
        tw.set_rows(r, np.arange(16), cache_ids, cache_tags)
        tw.acquire(cache_ids, cache_tags)
        tw.cur[r] = 256
    tw.append([0, 100, 50])
    _check(tw, "B and C attached and appended", decode_reqs=[1, 2])
    tw.migrate()
    _check(tw, "Retier with a shared prefix", decode_reqs=[1, 2])
    assert (tw.otags[1, :16] < 2).all() and (tw.otags[1, 16:18] == 2).all()
    n = tw.promote((tw.otags == 2).astype(np.uint8))
    assert n == 2
    _check(tw, "Promote", decode_reqs=[1, 2])
    assert tw.release(cache_ids, cache_tags) == 0         # prefix eviction: B and C still hold
    tw.migrate()
    _check(tw, "evicted; Retier with two sharers", decode_reqs=[1, 2])
    assert (tw.otags[1:, :16] < 2).all()
    tw.finish([2])                                        # C done: B is the only owner
    tw.migrate()
    _check(tw, "C finished; Retier encodes B's prefix", decode_reqs=[1])
    assert (tw.otags[1, :4] == 1).all() and (tw.otags[1, 4:16] == 2).all()
    tw.finish([1])
    _check(tw, "B finished")
    assert tw.orc.fp8_top[0] == 120 and tw.orc.tq3_top[0] == 120


def test_joint_finish_with_shared_pages_and_fail_closed():
    """Two requests that share pages finish in one call: each shared page
    returns at its second reference; over-release and stale acquires change
    nothing and set the error word."""
    import torch
    import paper_2608_23834_amd as mk
    from _harness import Twin
    w = wl.workload(1)
    tw = Twin(w, lens=[64, 80], recent=10 ** 6, n_fp8=16, n_tq3=4)
    tw.fill_to([64, 0])
    ids, tg = tw.obt[0, :3].copy(), np.zeros(3, np.uint8)
    tw.set_rows(1, np.arange(3), ids, tg)
    tw.acquire(ids, tg)
    tw.cur[1] = 48
    tw.append([0, 20])
    _check(tw, "two sharers")
    before = (tw.bt.cpu().numpy().copy(), mk.kv_pool_read_free_lists(tw.gpu),
              mk.kv_pool_read_refcounts(tw.gpu))
    bad_ids = torch.tensor([ids[0]] * 3, dtype=torch.int32, device="cuda")
    mk.kv_pages_release(tw.gpu, bad_ids, torch.zeros(3, dtype=torch.uint8, device="cuda"))
    free_id = int(before[1][0][0])
    mk.kv_pages_acquire(tw.gpu, torch.tensor([free_id], dtype=torch.int32, device="cuda"),
                        torch.zeros(1, dtype=torch.uint8, device="cuda"))
    assert mk.kv_pool_check_errors(tw.gpu, clear=True) == mk.DEVERR["REFCOUNT"]
    assert np.array_equal(tw.bt.cpu().numpy(), before[0])
    assert all(np.array_equal(a, b) for a, b in zip(mk.kv_pool_read_free_lists(tw.gpu), before[1]))
    assert all(np.array_equal(a, b) for a, b in zip(mk.kv_pool_read_refcounts(tw.gpu), before[2]))
    tw.finish([0, 1])
    _check(tw, "joint finish")
    assert tw.orc.fp8_top[0] == 16 and (tw.orc.rc8 == 0).all()
