"""paged_attn_decode_noalloc (the decode for callers that cannot allocate) against
paged_attn_decode with a caller workspace and against the oracle, through the
C ABI: two calls in a row on the library's fixed device scratch, the second on
a smaller batch, then a shape whose partials exceed the scratch (rejected on
the host with MKV_ENOMEM)."""
import numpy as np
import pytest

import mkv_workloads as wl

pytestmark = pytest.mark.gpu

TOL = 1e-3


def test_decode_noalloc_matches_workspace_decode():
    import torch
    import paper_2608_23834_amd as mk
    from _harness import Twin, max_abs
    assert torch.cuda.is_available()
    w = wl.workload(2)
    lens = [3000, 100, 5000, 17]
    print(f"\n[noalloc] {w.name} lens={lens}", flush=True)
    tw = Twin(w, lens=lens, recent=64)
    tw.fill()
    tw.migrate()
    tw.check_tables()
    q_all = wl.q_decode(w, 0)
    q_all = np.resize(q_all, (len(lens),) + q_all.shape[1:])
    for n in (4, 2):  # the second call on a smaller batch
        bt, tags = tw.bt[:n].contiguous(), tw.tags[:n].contiguous()
        sl = np.array(tw.cur[:n], np.int32)
        q = torch.from_numpy(np.ascontiguousarray(q_all[:n]).view(np.int16)).cuda()
        slg = torch.from_numpy(sl).cuda()
        out_n = torch.full((n, w.n_q_heads, w.head_dim), float("nan"), device="cuda")
        lse_n = torch.full((n, w.n_q_heads), float("nan"), device="cuda")
        mk.paged_attn_decode_noalloc(tw.gpu, 0, q, bt, tags, slg, out_n, lse_n)
        out_w = torch.full_like(out_n, float("nan"))
        lse_w = torch.full_like(lse_n, float("nan"))
        ws = mk.workspace(tw.gpu, n, tw.max_pages)
        mk.paged_attn_decode(tw.gpu, 0, q, bt, tags, slg, out_w, lse_w, ws)
        torch.cuda.synchronize()
        assert mk.kv_pool_check_errors(tw.gpu) == 0
        o_n, o_w = out_n.cpu().numpy(), out_w.cpu().numpy()
        l_n, l_w = lse_n.cpu().numpy(), lse_w.cpu().numpy()
        ref_o, ref_l = tw.orc.decode(0, q_all[:n], tw.obt[:n], tw.otags[:n], sl)
        d_w = max(max_abs(o_n, o_w), max_abs(l_n, l_w))
        d_r = max(max_abs(o_n, ref_o), max_abs(l_n, ref_l))
        print(f"  n_req {n}: max|noalloc - workspace| {d_w:.3e}  max|noalloc - oracle| {d_r:.3e}",
              flush=True)
        assert np.all(np.isfinite(o_n)) and np.all(np.isfinite(l_n))
        assert d_w <= TOL and d_r <= TOL
    # a batch whose partials exceed the fixed scratch is refused before any launch
    n_big, mp_big = 200, 4096
    assert mk.paged_attn_workspace_bytes(tw.gpu, n_big, mp_big) > mk.DECODE_SCRATCH_BYTES
    bt = torch.full((n_big, mp_big), -1, dtype=torch.int32, device="cuda")
    tags = torch.full((n_big, mp_big), 0xFF, dtype=torch.uint8, device="cuda")
    q = torch.zeros((n_big, w.n_q_heads, w.head_dim), dtype=torch.int16, device="cuda")
    out = torch.zeros((n_big, w.n_q_heads, w.head_dim), device="cuda")
    with pytest.raises(mk.MkvError) as e:
        mk.paged_attn_decode_noalloc(tw.gpu, 0, q, bt, tags,
                                     torch.ones(n_big, dtype=torch.int32, device="cuda"), out, None)
    assert e.value.code == 3  # MKV_ENOMEM
