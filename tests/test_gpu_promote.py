"""GPU parity of kv_promote_to_fp8 (Alg. 1 Promote) against the oracle, through
the C ABI: block tables, tags, free lists, and the new FP8 pages (codes and
scales) bit for bit; decode after promotion within 1e-3."""
import numpy as np
import pytest

import mkv_workloads as wl
from _harness import max_abs

pytestmark = pytest.mark.gpu

TOL = 1e-3


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_23834_amd as mk
    mk.lib()
    return torch


def _mask_every(tags, k, offset=0):
    m = np.zeros(tags.shape, np.uint8)
    st = np.argwhere(tags == 2)
    for r, p in st[offset::k]:
        m[r, p] = 1
    return m


def _check_decode(tw, what):
    res = tw.decode()
    err = max(max_abs(res["out"], res["ref_out"]), max_abs(res["lse"], res["ref_lse"]))
    print(f"  {what}: max|dO|, max|dlse| {err:.3e}", flush=True)
    assert np.all(np.isfinite(res["out"]))
    assert err <= TOL


def test_promote_ragged_d256_then_steps(torch_cuda):
    """Ragged lengths (1, 17, 700, 3000, 90), d = 256, six query heads per KV
    head, two layers: every third Stale page promoted (mask also set on
    Recent, unmapped and past-the-end entries, which stay as they are), then
    decode, then decode steps with appends and Retier around the promoted
    Anchor pages, and a second promotion."""
    from _harness import Twin
    w = wl.workload(2)
    lens = [1, 17, 700, 3000, 90]
    print(f"\n[promote] {w.name} lens={lens}", flush=True)
    tw = Twin(w, n_layers=2, lens=lens, recent=64, headroom=48)
    tw.fill()
    tw.migrate()
    tw.check_tables()
    mask = _mask_every(tw.otags, 3)
    mask[tw.otags == 0] = 1          # Recent pages: not Stale, untouched
    mask[:, -1] = 1                  # past every request's end
    n = tw.promote(mask)
    print(f"  promoted {n} pages", flush=True)
    assert n > 50
    tw.check_tables()
    tw.check_pages()
    _check_decode(tw, "after promotion")
    for step in range(8):
        tw.append([3] * len(lens))
        tw.migrate()
        tw.check_tables()
    tw.check_pages()
    _check_decode(tw, "after 8 append + Retier steps")
    n2 = tw.promote(_mask_every(tw.otags, 5, offset=1))
    print(f"  promoted {n2} more pages", flush=True)
    tw.check_tables()
    tw.check_pages()
    _check_decode(tw, "after the second promotion")


def test_promote_d128_all_stale_pages(torch_cuda):
    """The tiny workload (d = 128, eight query heads per KV head, outlier key
    channels): every Stale page promoted back to FP8."""
    from _harness import Twin
    w = wl.workload(1)
    tw = Twin(w, lens=list(w.ctx))
    tw.fill()
    tw.migrate()
    mask = (tw.otags == 2).astype(np.uint8)
    assert tw.promote(mask) == 108
    tw.check_tables()
    n8, n3 = tw.check_pages()
    assert n3 == 0 and n8 == 128
    _check_decode(tw, "all pages FP8 after promotion")


def test_promote_16k_single_request(torch_cuda):
    """Config 2's single 16K request (one layer): 10 % of its Stale pages,
    scattered, promoted."""
    from _harness import Twin
    w = wl.workload(2)
    tw = Twin(w, lens=list(w.ctx))
    tw.fill()
    tw.migrate()
    assert tw.promote(_mask_every(tw.otags, 10, offset=3)) >= 90
    tw.check_tables()
    tw.check_pages()
    _check_decode(tw, "16K after promotion")


def test_promote_fails_closed(torch_cuda):
    """FP8 free list too short for the request: no state changes, the error
    word says so; a later call that fits succeeds."""
    import paper_2608_23834_amd as mk
    from _harness import Twin
    torch = torch_cuda
    w = wl.workload(1)
    tw = Twin(w, lens=[600], recent=32, n_fp8=40, n_tq3=40, with_oracle=False, headroom=96)
    tw.fill()
    tw.migrate()
    tw.append([96])  # six more Recent pages take FP8 ids (no Retier after it)
    tags = tw.tags.cpu().numpy()
    n_stale = int((tags == 2).sum())
    f8, f3 = mk.kv_pool_free_counts(tw.gpu)
    assert n_stale > f8
    before = (tw.bt.cpu().numpy().copy(), tags.copy(), mk.kv_pool_read_free_lists(tw.gpu))
    mask = (tags == 2).astype(np.uint8)
    sl = torch.tensor(tw.cur, dtype=torch.int32, device="cuda")
    mk.kv_promote_to_fp8(tw.gpu, tw.bt, tw.tags, torch.from_numpy(mask).cuda(), sl)
    assert mk.kv_pool_check_errors(tw.gpu, clear=True) & mk.DEVERR["FP8_EXHAUSTED"]
    assert np.array_equal(tw.bt.cpu().numpy(), before[0])
    assert np.array_equal(tw.tags.cpu().numpy(), before[1])
    after = mk.kv_pool_read_free_lists(tw.gpu)
    assert all(np.array_equal(a, b) for a, b in zip(after, before[2]))
    mask2 = np.zeros_like(mask)
    st = np.argwhere(tags == 2)[:f8]
    mask2[st[:, 0], st[:, 1]] = 1
    mk.kv_promote_to_fp8(tw.gpu, tw.bt, tw.tags, torch.from_numpy(mask2).cuda(), sl)
    assert mk.kv_pool_check_errors(tw.gpu) == 0
    assert mk.kv_pool_free_counts(tw.gpu) == (0, f3 + f8)
    assert int((tw.tags.cpu().numpy() == 1).sum()) == int((tags == 1).sum()) + f8
