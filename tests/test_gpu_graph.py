"""Decode steps captured into a HIP graph and replayed, with cohort gating
(Sec. 4.1: the graph path is gated on a homogeneous physical-cache cohort and
anything else fails closed to the generic path).

Two pools are built identically; one runs every decode step eagerly (and is
checked against the oracle), the other replays one captured step -- per
layer paged_attn_decode_append, then kv_migrate_to_tq3 -- with the step's
inputs copied into fixed buffers between replays (eager work and
synchronizations in between).  Every replay must leave the same block table,
tags, free lists and pages as the eager run, bit for bit, and the same
outputs up to fp32 summation order.
"""
import numpy as np
import pytest

import mkv_workloads as wl
from _harness import max_abs

pytestmark = pytest.mark.gpu

TOL = 1e-3


def test_decode_step_graph_replays_match_eager():
    import torch
    import paper_2608_23834_amd as mk
    from _harness import Twin
    assert torch.cuda.is_available()
    w = wl.workload(2)
    lens, L, n_steps = [700, 1500, 33], 2, 12
    print(f"\n[graph] {w.name} lens={lens} layers={L} steps={n_steps}", flush=True)
    ta = Twin(w, n_layers=L, lens=lens, recent=64, headroom=n_steps + 16)
    tb = Twin(w, n_layers=L, lens=lens, recent=64, headroom=n_steps + 16, with_oracle=False)
    for t in (ta, tb):
        t.fill()
        t.migrate()
    n_req, Hq, Hkv, d = len(lens), w.n_q_heads, w.n_kv_heads, w.head_dim
    dev = "cuda"
    bufs = {
        "q": torch.zeros((L, n_req, Hq, d), dtype=torch.int16, device=dev),
        "k_new": torch.zeros((L, n_req, Hkv, d), dtype=torch.int16, device=dev),
        "v_new": torch.zeros((L, n_req, Hkv, d), dtype=torch.int16, device=dev),
        "seq_before": torch.zeros(n_req, dtype=torch.int32, device=dev),
        "seq_after": torch.zeros(n_req, dtype=torch.int32, device=dev),
        "anchor": torch.from_numpy(tb.anchor()).cuda(),
    }
    out = torch.zeros((L, n_req, Hq, d), device=dev)
    lse = torch.zeros((L, n_req, Hq), device=dev)
    ws = mk.workspace(tb.gpu, n_req, tb.max_pages)
    g = mk.DecodeStepGraph(tb.gpu, tb.bt, tb.tags, bufs, out, lse, ws)
    key = mk.paged_attn_decode_cohort_key(tb.gpu, n_req, tb.max_pages)
    assert key == g.key
    rng = np.random.default_rng(9)
    # the last step is of another cohort (its key is that of a batch with one
    # request fewer): it must fail closed to the direct calls
    other = mk.paged_attn_decode_cohort_key(tb.gpu, n_req - 1, tb.max_pages)
    assert other != g.key
    for step in range(n_steps + 1):
        # eager pool (and oracle): append + decode per layer, then Retier
        qs, worst = [], 0.0
        for layer in range(L):
            q = wl.bf16_round(rng.standard_normal((n_req, Hq, d)).astype(np.float32))
            qs.append(q)
            res = ta.decode_append(layer, q=q)
            worst = max(worst, max_abs(res["out"], res["ref_out"]), max_abs(res["lse"], res["ref_lse"]))
            if layer == 0:
                eager = [res]
            else:
                eager.append(res)
        assert worst <= TOL, (step, worst)
        ta.advance()
        ta.migrate()
        # graph pool: refill the fixed inputs, then replay (captured before step 0)
        for layer in range(L):
            bufs["q"][layer].copy_(torch.from_numpy(qs[layer].view(np.int16)))
            kk, vv = zip(*(wl.kv_layer(w, layer, 1, token_offset=r * 1_000_000 + tb.cur[r])
                           for r in range(n_req)))
            bufs["k_new"][layer].copy_(torch.from_numpy(np.concatenate(kk).view(np.int16)))
            bufs["v_new"][layer].copy_(torch.from_numpy(np.concatenate(vv).view(np.int16)))
        bufs["seq_before"].copy_(torch.tensor(tb.cur, dtype=torch.int32))
        bufs["seq_after"].copy_(torch.tensor([c + 1 for c in tb.cur], dtype=torch.int32))
        if g.graph is None:
            g.capture()
        torch.cuda.synchronize()
        g.run(mk.paged_attn_decode_cohort_key(tb.gpu, n_req, tb.max_pages) if step < n_steps
              else other)
        torch.cuda.synchronize()
        tb.advance()
        diff = max(max(max_abs(out[l].cpu().numpy(), eager[l]["out"]),
                       max_abs(lse[l].cpu().numpy(), eager[l]["lse"])) for l in range(L))
        print(f"  step {step}: eager vs oracle {worst:.2e}, replay vs eager {diff:.2e}", flush=True)
        assert diff <= 1e-5, (step, diff)
        assert np.array_equal(tb.bt.cpu().numpy(), ta.bt.cpu().numpy()), step
        assert np.array_equal(tb.tags.cpu().numpy(), ta.tags.cpu().numpy()), step
        fa, fb = mk.kv_pool_read_free_lists(ta.gpu), mk.kv_pool_read_free_lists(tb.gpu)
        assert all(np.array_equal(x, y) for x, y in zip(fa, fb)), step
        if step % 4 == 3 or step >= n_steps - 1:
            assert torch.equal(ta.gpu.fp8, tb.gpu.fp8) and torch.equal(ta.gpu.tq3, tb.gpu.tq3)
            assert torch.equal(ta.gpu.fp8_scales, tb.gpu.fp8_scales)
            ta.check_tables()
            ta.check_pages()
    assert g.replays == n_steps and g.direct == 1
    assert (ta.otags == 2).sum() > 0 and mk.kv_pool_check_errors(tb.gpu) == 0


def test_cohort_key_properties():
    """The key changes with everything a capture bakes in and refuses pools
    that are not a compressed cohort or have kernel timing on."""
    import torch
    import paper_2608_23834_amd as mk
    assert torch.cuda.is_available()
    d = 128
    p1 = mk.Pool(2, 8, 1, d, 64, 64, 256, np.ones(d, np.int8))
    p2 = mk.Pool(2, 8, 1, d, 64, 64, 256, np.ones(d, np.int8))
    k = mk.paged_attn_decode_cohort_key
    base = k(p1, 3, 40)
    assert base == k(p1, 3, 40)
    variants = [k(p2, 3, 40), k(p1, 4, 40), k(p1, 3, 41), k(p1, 3, 40, fused_append=False),
                k(p1, 3, 40, scoring=True)]
    assert len({base, *variants}) == 1 + len(variants)
    no_tq3 = mk.Pool(1, 8, 1, d, 16, 0, 256, np.ones(d, np.int8))
    with pytest.raises(mk.MkvError) as e:
        k(no_tq3, 1, 4)
    assert e.value.code == 5  # MKV_ESTATE: not a compressed cohort
    mk.paged_attn_set_timing(p1, True)
    with pytest.raises(mk.MkvError) as e:
        k(p1, 3, 40)
    assert e.value.code == 5
    mk.paged_attn_set_timing(p1, False)
    assert k(p1, 3, 40) == base
