"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bit-exact: block tables, tags, free lists, FP8 codes and scales, TQ3 packed
regions (codes, gamma, V scale/zero).  Attention output: max-abs <= 1e-3
(fp32 accumulation), the bound the decode path must meet; lse likewise.
"""
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


def _run_decode_case(w, lens, recent=None, n_layers=1, chunk=None):
    from _harness import Twin, max_abs
    print(f"\n[case] {w.name} lens={lens[:6]}{'...' if len(lens) > 6 else ''} W={recent}", flush=True)
    tw = Twin(w, n_layers=n_layers, lens=lens, recent=recent)
    tw.fill(chunk=chunk)
    tw.check_tables()
    tw.migrate()
    tw.check_tables()
    n8, n3 = tw.check_pages()
    for layer in range(n_layers):
        res = tw.decode(layer=layer)
        err = max_abs(res["out"], res["ref_out"])
        lerr = max_abs(res["lse"], res["ref_lse"])
        print(f"  layer {layer}: live fp8 {n8} tq3 {n3}  max|dO| {err:.3e}  max|dlse| {lerr:.3e}",
              flush=True)
        assert np.all(np.isfinite(res["out"]))
        assert err <= TOL, err
        assert lerr <= TOL, lerr
    return tw


def test_tiny_config_full(torch_cuda):
    """Config 1 at full size: d=128, GQA 8, 2048 tokens, anchors 0-63, W=256."""
    w = wl.workload(1)
    tw = _run_decode_case(w, list(w.ctx))
    tags = tw.tags.cpu().numpy()[0]
    assert (tags == 1).sum() == 4 and (tags == 2).sum() == 108 and (tags == 0).sum() == 16


def test_ragged_multi_request_d256(torch_cuda):
    """Several requests with ragged lengths (1, page-aligned, partial pages),
    GQA 6, d=256, a short Recent window so most pages are TQ3."""
    w = wl.workload(2)
    lens = [1, 15, 16, 17, 333, 1024, 2049, 4000]
    _run_decode_case(w, lens, recent=64)


def test_two_layers_chunked_fill(torch_cuda):
    w = wl.workload(2)
    _run_decode_case(w, [900, 1700], recent=128, n_layers=2, chunk=250)


def test_single_request_16k_config(torch_cuda):
    """Config 2 at full size: one 16K request, anchors 4 + 2 %, all 16
    layers appended, migrated and decoded."""
    w = wl.workload(2)
    assert w.n_layers == 16
    _run_decode_case(w, list(w.ctx), n_layers=16)


def test_long_pair_full_size(torch_cuda):
    """Config 3 at full size (2 x 59,008 tokens) on one layer: the launch
    configuration the benchmark times."""
    w = wl.workload(3)
    tw = _run_decode_case(w, list(w.ctx))
    tags = tw.tags.cpu().numpy()
    for r in range(2):
        assert (tags[r] == 0).sum() == 128
        assert (tags[r] == 1).sum() == 8 + 36
        assert (tags[r] == 2).sum() == 3516


def test_batch64_config_full_size(torch_cuda):
    """Config 4 at full size: 64 requests with lengths drawn from U[4096,
    65536], pages of every request interleaved in one pool through shuffled
    free stacks, one layer, in the launch configuration of the benchmark's
    decode call.  The GPU holds all 64 requests; the oracle models 16 of
    them (the shortest, the longest and 14 others, most with a partly filled
    last page) from the same K/V bytes, copied back from the device.  Physical ids differ between the two
    pools (the oracle does not see the other requests), so pages are
    compared bit for bit through each side's block table."""
    import oracle
    import paper_2608_23834_amd as mk
    torch = torch_cuda
    w = wl.workload(4)
    lens = list(w.ctx)
    n_req, H, d = len(lens), w.n_kv_heads, w.head_dim
    mp = max((L + 15) // 16 for L in lens)
    tot = sum((L + 15) // 16 for L in lens) + 8
    print(f"\n[case] {w.name}: {n_req} requests, {sum(lens)} tokens, {tot} pages", flush=True)
    gp = mk.Pool(1, w.n_q_heads, H, d, tot, tot, w.recent, wl.rot_signs(w),
                 wl.free_order(w, tot, "fp8"), wl.free_order(w, tot, "tq3"))
    bt = torch.full((n_req, mp), -1, dtype=torch.int32, device="cuda")
    tags = torch.full((n_req, mp), 0xFF, dtype=torch.uint8, device="cuda")
    K, V = wl.kv_layer_device(w, 0, sum(lens))
    cu = np.r_[0, np.cumsum(lens)].astype(np.int32)
    sl = np.array(lens, np.int32)
    mk.kv_append_fp8(gp, 0, bt, tags, torch.zeros(n_req, dtype=torch.int32, device="cuda"),
                     torch.from_numpy(cu).cuda(), K, V)
    am = wl.anchor_mask(w, mp)
    mk.kv_migrate_to_tq3(gp, bt, tags, torch.from_numpy(am).cuda(), torch.from_numpy(sl).cuda())
    q = wl.q_decode(w, 0)
    out = torch.full((n_req, w.n_q_heads, d), float("nan"), device="cuda")
    ws = mk.workspace(gp, n_req, mp)
    mk.paged_attn_decode(gp, 0, torch.from_numpy(q.view(np.int16)).cuda(), bt, tags,
                         torch.from_numpy(sl).cuda(), out, None, ws)
    torch.cuda.synchronize()
    assert mk.kv_pool_check_errors(gp) == 0
    out = out.cpu().numpy()
    assert np.all(np.isfinite(out))
    g_bt, g_tags = bt.cpu().numpy(), tags.cpu().numpy()
    rng = np.random.default_rng(4)
    rest = [r for r in range(n_req) if r not in (int(np.argmin(lens)), int(np.argmax(lens)))]
    sample = sorted({int(np.argmin(lens)), int(np.argmax(lens)), *rng.choice(rest, 14, replace=False).tolist()})
    assert len(sample) == 16
    assert sum(lens[r] % 16 != 0 for r in sample) >= 8  # partly filled last pages
    s_lens = [lens[r] for r in sample]
    s_mp = max((L + 15) // 16 for L in s_lens)
    s_tot = sum((L + 15) // 16 for L in s_lens) + 8
    print(f"  oracle sample {sample} lens {s_lens}", flush=True)
    orc = oracle.Pool(1, w.n_q_heads, H, d, s_tot, s_tot, w.recent, wl.rot_signs(w),
                      wl.free_order(w, s_tot, "fp8"), wl.free_order(w, s_tot, "tq3"))
    o_bt = np.full((len(sample), s_mp), -1, np.int32)
    o_tags = np.full((len(sample), s_mp), 0xFF, np.uint8)
    ks = np.concatenate([K[cu[r]:cu[r + 1]].cpu().numpy() for r in sample]).view(np.uint16)
    vs = np.concatenate([V[cu[r]:cu[r + 1]].cpu().numpy() for r in sample]).view(np.uint16)
    s_cu = np.r_[0, np.cumsum(s_lens)].astype(np.int32)
    assert orc.append(0, o_bt, o_tags, np.zeros(len(sample), np.int32), s_cu, ks[None], vs[None]) == 0
    assert orc.migrate(o_bt, o_tags, am[sample][:, :s_mp], np.array(s_lens, np.int32)) >= 0
    g8, gs, g3 = gp.fp8_view(), gp.fp8_scales_view(), gp.tq3_view()
    for i, r in enumerate(sample):
        npg = (lens[r] + 15) // 16
        assert np.array_equal(g_tags[r, :npg], o_tags[i, :npg]), f"tags of request {r}"
        for fmt, pick in (("fp8", g_tags[r, :npg] < 2), ("tq3", g_tags[r, :npg] == 2)):
            gid = torch.from_numpy(g_bt[r, :npg][pick].astype(np.int64)).cuda()
            oid = o_bt[i, :npg][pick]
            if fmt == "fp8":
                assert np.array_equal(g8[0, gid].cpu().numpy(), orc.fp8[0, oid]), f"fp8 pages of {r}"
                assert np.array_equal(gs[0, gid].cpu().numpy().view(np.uint32),
                                      orc.fp8_scale[0, oid].view(np.uint32)), f"fp8 scales of {r}"
            else:
                assert np.array_equal(g3[0, gid].cpu().numpy(), orc.tq3[0, oid]), f"tq3 pages of {r}"
    ref, _ = orc.decode(0, q[sample], o_bt, o_tags, np.array(s_lens, np.int32))
    err = max_abs(out[sample], ref)
    print(f"  sampled requests: max|dO| {err:.3e}", flush=True)
    assert err <= TOL, err


def test_group12_decode(torch_cuda):
    """Twelve query heads per KV head (the kernel instance without the page
    pair layout): ragged lengths, short Recent window."""
    import dataclasses
    w = dataclasses.replace(wl.workload(2), n_kv_heads=2, name="group12")
    _run_decode_case(w, [3000, 777, 1], recent=64)


def test_stream_probe_reads_every_word(torch_cuda):
    """The streaming-read probe folds every 32-bit word of the buffer once:
    the XOR of its per-workgroup words equals the XOR of the buffer."""
    import paper_2608_23834_amd as mk
    torch = torch_cuda
    rng = np.random.default_rng(7)
    for n_words in (4, 4 * 1000 + 4, 1 << 22):
        x = rng.integers(0, 2 ** 31, size=n_words, dtype=np.int64).astype(np.int32)
        buf = torch.from_numpy(x).cuda()
        sink = torch.zeros(mk.STREAM_PROBE_WORKGROUPS, dtype=torch.int32, device="cuda")
        mk.mkv_stream_read(buf, sink)
        torch.cuda.synchronize()
        want = np.bitwise_xor.reduce(x.view(np.uint32))
        got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
        assert got == want, (n_words, got, want)


def test_decode_steps_with_appends(torch_cuda):
    """Token-by-token decode: append one token per request, migrate, decode;
    pages are partly filled and rescaled along the way."""
    from _harness import Twin, max_abs
    w = wl.workload(2)
    tw = Twin(w, n_layers=1, lens=[200, 47], recent=32, headroom=32)
    tw.fill()
    tw.migrate()
    for step in range(20):
        tw.append([1, 1])
        tw.migrate()
        tw.check_tables()
        if step % 5 == 4:
            tw.check_pages()
            res = tw.decode()
            assert max_abs(res["out"], res["ref_out"]) <= TOL


def _fused_steps(w, lens, n_layers, n_steps, recent, check_every=4, headroom=None):
    """Decode steps through the fused call (append one token per request and
    decode, per layer), then migration; the oracle runs append, decode and
    migrate as separate calls.  Tables, tags and free lists bit-exact after
    every step, page bytes every few steps, outputs within TOL."""
    from _harness import Twin, max_abs
    print(f"\n[fused steps] {w.name} lens={lens} layers={n_layers} W={recent}", flush=True)
    tw = Twin(w, n_layers=n_layers, lens=lens, recent=recent,
              headroom=n_steps + 16 if headroom is None else headroom)
    tw.fill()
    tw.migrate()
    worst = 0.0
    for step in range(n_steps):
        for layer in range(n_layers):
            res = tw.decode_append(layer)
            err = max(max_abs(res["out"], res["ref_out"]), max_abs(res["lse"], res["ref_lse"]))
            worst = max(worst, err)
            assert np.all(np.isfinite(res["out"]))
            assert err <= TOL, (step, layer, err)
        tw.advance()
        tw.migrate()
        tw.check_tables()
        if step % check_every == check_every - 1 or step == n_steps - 1:
            tw.check_pages()
    print(f"  {n_steps} steps, max|dO|, max|dlse| {worst:.3e}", flush=True)
    return tw


def test_decode_append_fused_steps_d256(torch_cuda):
    """Fused decode steps, d = 256, six query heads per KV head, two layers:
    lengths 0, 1, 47, 64 and 200 cross page boundaries, so layer 0's call
    opens fresh pages that layer 1's call then writes; partly filled pages
    grow their FP8 scales; pages leave the short Recent window as TQ3."""
    w = wl.workload(2)
    _fused_steps(w, [200, 47, 64, 1, 0], n_layers=2, n_steps=36, recent=32)


def test_decode_append_fused_steps_d128_group12(torch_cuda):
    """Fused decode steps for the other kernel instances: d = 128 with eight
    query heads per KV head (page pairs), and twelve query heads per KV
    head (no pairs)."""
    import dataclasses
    _fused_steps(wl.workload(1), [1000, 15, 33], n_layers=1, n_steps=20, recent=48)
    w = dataclasses.replace(wl.workload(2), n_kv_heads=2, name="group12")
    _fused_steps(w, [700, 16, 5], n_layers=1, n_steps=20, recent=64)


def test_decode_append_fused_full_size(torch_cuda):
    """The long pair at full size (2 x 59,008 tokens, one layer) with the
    table width of the benchmark's default run (3,693 pages): three fused
    steps (the first opens a fresh page in each request), bit-exact state and
    outputs against the oracle's append + decode."""
    w = wl.workload(3)
    tw = _fused_steps(w, list(w.ctx), n_layers=1, n_steps=3, recent=None, check_every=3,
                      headroom=3 + 3 * 20 + 16)
    assert tw.max_pages == 3693
    assert (tw.otags == 0).sum() == 2 * 129


def test_decode_append_many_requests(torch_cuda):
    """The fused decode step with many requests: 24 ragged requests (d = 256,
    two layers; fresh pages opened for several requests in one launch)
    against the oracle's separate append and decode, bit-exact state; and the
    fail-closed contract (zero outputs, lse -inf, no state change) for 20
    requests when the free list cannot hold their fresh pages."""
    import paper_2608_23834_amd as mk
    torch = torch_cuda
    rng = np.random.default_rng(24)
    lens = [int(x) for x in rng.integers(0, 900, 24)]
    lens[:3] = [0, 1, 16]
    tw = _fused_steps(wl.workload(2), lens, n_layers=2, n_steps=6, recent=64, check_every=3)
    assert tw.n_req > 16
    # free list too short for the fresh pages of one step: nothing changes
    d, Hq, n = 128, 2, 20
    gp = mk.Pool(1, Hq, 1, d, 8, 2, 16, np.ones(d, np.int8))
    bt = torch.full((n, 4), -1, dtype=torch.int32, device="cuda")
    tg = torch.full((n, 4), 0xFF, dtype=torch.uint8, device="cuda")
    ws = mk.workspace(gp, n, 4)
    q = torch.from_numpy(rng.integers(0x3c00, 0x3f00, (n, Hq, d)).astype(np.int16)).cuda()
    kv = torch.from_numpy(rng.integers(0x3c00, 0x3f00, (n, 1, d)).astype(np.int16)).cuda()
    out = torch.full((n, Hq, d), 7.0, device="cuda")
    lse = torch.full((n, Hq), 7.0, device="cuda")
    mk.paged_attn_decode_append(gp, 0, q, kv, kv, bt, tg, torch.zeros(n, dtype=torch.int32,
                                                                      device="cuda"), out, lse, ws)
    torch.cuda.synchronize()
    assert mk.kv_pool_check_errors(gp, clear=True) & mk.DEVERR["FP8_EXHAUSTED"]
    assert (out.cpu().numpy() == 0).all() and np.isneginf(lse.cpu().numpy()).all()
    assert (bt.cpu().numpy() == -1).all() and mk.kv_pool_free_counts(gp) == (8, 2)


def test_decode_append_fails_closed(torch_cuda):
    """A fused step that cannot append as a whole (free list exhausted, a
    length out of range, a page that is not Recent) changes no state, sets
    the error word and writes zero outputs (lse -inf) for every request."""
    import paper_2608_23834_amd as mk
    torch = torch_cuda
    d, Hq = 128, 2
    gp = mk.Pool(1, Hq, 1, d, 1, 2, 16, np.ones(d, np.int8))
    bt = torch.full((2, 4), -1, dtype=torch.int32, device="cuda")
    tg = torch.full((2, 4), 0xFF, dtype=torch.uint8, device="cuda")
    ws = mk.workspace(gp, 2, 4)
    rng = np.random.default_rng(7)
    q = torch.from_numpy(rng.integers(0x3c00, 0x3f00, (2, Hq, d)).astype(np.int16)).cuda()
    kv = torch.from_numpy(rng.integers(0x3c00, 0x3f00, (2, 1, d)).astype(np.int16)).cuda()

    def call(sl, n=2):
        out = torch.full((n, Hq, d), 7.0, device="cuda")
        lse = torch.full((n, Hq), 7.0, device="cuda")
        mk.paged_attn_decode_append(gp, 0, q[:n], kv[:n], kv[:n], bt[:n], tg[:n],
                                    torch.tensor(sl, dtype=torch.int32, device="cuda"), out, lse, ws)
        torch.cuda.synchronize()
        return out.cpu().numpy(), lse.cpu().numpy()

    def unchanged():
        assert (bt.cpu().numpy() == -1).all() and (tg.cpu().numpy() == 0xFF).all()
        assert mk.kv_pool_free_counts(gp) == (1, 2)

    # two fresh pages wanted, one free
    out, lse = call([0, 0])
    assert mk.kv_pool_check_errors(gp, clear=True) & mk.DEVERR["FP8_EXHAUSTED"]
    assert (out == 0).all() and np.isneginf(lse).all()
    unchanged()
    # a length past the table
    out, lse = call([0, 64])
    assert mk.kv_pool_check_errors(gp, clear=True) & mk.DEVERR["RANGE"]
    assert (out == 0).all() and np.isneginf(lse).all()
    unchanged()
    # one request: the page is opened, the output is the token's V (one key)
    out, lse = call([0], n=1)
    assert mk.kv_pool_check_errors(gp, clear=True) == 0
    assert bt.cpu().numpy()[0, 0] >= 0 and tg.cpu().numpy()[0, 0] == mk.TAG_R
    assert mk.kv_pool_free_counts(gp) == (0, 2)
    v = (kv[0, 0].cpu().numpy().astype(np.uint32) << 16).view(np.float32)
    assert np.abs(out[0] - v[None]).max() <= 0.07 * np.abs(v).max()  # one E4M3 rounding
    # the opened page tagged Stale: appending to it is refused
    tg[0, 0] = mk.TAG_S
    bt_before = bt.cpu().numpy().copy()
    out, lse = call([1], n=1)
    assert mk.kv_pool_check_errors(gp, clear=True) & mk.DEVERR["NOT_RECENT"]
    assert (out == 0).all() and np.array_equal(bt.cpu().numpy(), bt_before)


def test_partition_pages_matches_oracle(torch_cuda):
    import oracle
    import paper_2608_23834_amd as mk
    torch = torch_cuda
    rng = np.random.default_rng(3)
    n_req, mp = 7, 300
    tags = rng.choice([0, 1, 2], size=(n_req, mp)).astype(np.uint8)
    bt = rng.integers(0, 10 ** 6, size=(n_req, mp)).astype(np.int32)
    lens = np.array([1, 16, 17, 4799, 4800, 2000, 333], np.int32)
    o8, o3, cnt = oracle.partition(bt, tags, lens)
    g8 = torch.full((n_req, mp, 2), -1, dtype=torch.int32, device="cuda")
    g3 = torch.full((n_req, mp, 2), -1, dtype=torch.int32, device="cuda")
    gc = torch.zeros((n_req, 2), dtype=torch.int32, device="cuda")
    mk.kv_partition_pages(torch.from_numpy(bt).cuda(), torch.from_numpy(tags).cuda(),
                          torch.from_numpy(lens).cuda(), g8, g3, gc)
    assert np.array_equal(gc.cpu().numpy(), cnt)
    assert np.array_equal(g8.cpu().numpy(), o8)
    assert np.array_equal(g3.cpu().numpy(), o3)


def test_e4m3_encode_all_bf16_inputs(torch_cuda):
    """Every bf16 value in [-448, 448] through the append path with page scale
    exactly 1 (each page-head's amax is 448): codes must equal the oracle's
    E4M3 rounding of the same value."""
    import oracle
    import paper_2608_23834_amd as mk
    torch = torch_cuda
    d = 128
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = wl.bf16_to_f32(bits)
    keep = np.isfinite(vals) & (np.abs(vals) <= 448.0)
    bits = bits[keep]
    per_tok = d - 1
    n_tok = -(-bits.size // per_tok)
    n_tok = -(-n_tok // 16) * 16
    x = np.zeros((n_tok, d), np.uint16)
    flat = np.zeros(n_tok * per_tok, np.uint16)
    flat[: bits.size] = bits
    x[:, 1:] = flat.reshape(n_tok, per_tok)
    x[:, 0] = wl.bf16_round(np.float32(448.0))
    K = x.reshape(1, n_tok, 1, d)
    pages = n_tok // 16
    gp = mk.Pool(1, 1, 1, d, pages, 1, 10 ** 6, np.ones(d, np.int8))
    bt = torch.full((1, pages), -1, dtype=torch.int32, device="cuda")
    tg = torch.full((1, pages), 0xFF, dtype=torch.uint8, device="cuda")
    kk = torch.from_numpy(K.view(np.int16)).cuda()
    mk.kv_append_fp8(gp, -1, bt, tg, torch.zeros(1, dtype=torch.int32, device="cuda"),
                     torch.tensor([0, n_tok], dtype=torch.int32, device="cuda"), kk, kk)
    torch.cuda.synchronize()
    assert np.all(gp.fp8_scales_view().cpu().numpy() == 1.0)
    ids = bt.cpu().numpy()[0]
    codes = gp.fp8_view()[0, torch.from_numpy(ids).long().cuda(), 0, : 16 * d].cpu().numpy()
    codes = codes.reshape(n_tok, d)
    want = oracle.e4m3_from_f32(wl.bf16_to_f32(x))
    assert np.array_equal(codes, want)


def test_workspace_reuse_and_repeat(torch_cuda):
    """Repeated calls on one workspace agree (up to fp32 summation order)."""
    import paper_2608_23834_amd as mk
    from _harness import Twin
    torch = torch_cuda
    w = wl.workload(2)
    tw = Twin(w, lens=[3000, 100, 5000], recent=64, with_oracle=False)
    tw.fill()
    tw.migrate()
    q = torch.from_numpy(wl.q_decode(w, 0)[:1].repeat(3, 0).view(np.int16)).cuda()
    sl = torch.tensor(tw.cur, dtype=torch.int32, device="cuda")
    ws = mk.workspace(tw.gpu, 3, tw.max_pages)
    outs = []
    for _ in range(4):
        out = torch.zeros((3, w.n_q_heads, w.head_dim), device="cuda")
        mk.paged_attn_decode(tw.gpu, 0, q, tw.bt, tw.tags, sl, out, None, ws)
        outs.append(out.cpu().numpy())
    # the waves claim pages at run time: repeats agree up to fp32 summation order
    for o in outs[1:]:
        assert np.abs(o - outs[0]).max() <= 1e-6
    c = mk.kv_pool_counters(tw.gpu)
    assert c["decode_routes"] == 4 and c["fallbacks"] == 0 and c["dense_shadow_bytes"] == 0
    # the optional kernel timing leaves results unchanged
    with pytest.raises(mk.MkvError):
        mk.paged_attn_last_times(tw.gpu)  # timing off: no timed call
    mk.paged_attn_set_timing(tw.gpu, True)
    out = torch.zeros((3, w.n_q_heads, w.head_dim), device="cuda")
    mk.paged_attn_decode(tw.gpu, 0, q, tw.bt, tw.tags, sl, out, None, ws)
    scan_us, merge_us = mk.paged_attn_last_times(tw.gpu)
    mk.paged_attn_set_timing(tw.gpu, False)
    assert scan_us > 0.0 and merge_us > 0.0
    assert np.abs(out.cpu().numpy() - outs[0]).max() <= 1e-6


def test_workspace_contents_do_not_matter(torch_cuda):
    """The workspace needs no initialisation: filled with NaN bits (and with
    +inf) before every call, decode and the fused decode step still match
    the oracle on ragged lengths, where many chunk slots of the split are
    empty or past a request's end (their O rows are never written)."""
    from _harness import Twin, max_abs
    w = wl.workload(2)
    tw = Twin(w, lens=[1, 17, 700, 3000, 90], recent=64, headroom=40)
    tw.fill()
    tw.migrate()
    for fill in (float("nan"), float("inf")):
        res = tw.decode(ws_fill=fill)
        assert np.all(np.isfinite(res["out"])) and np.all(np.isfinite(res["lse"]))
        assert max_abs(res["out"], res["ref_out"]) <= TOL
        assert max_abs(res["lse"], res["ref_lse"]) <= TOL
    for step in range(3):
        res = tw.decode_append(ws_fill=float("nan"))
        assert np.all(np.isfinite(res["out"])), step
        assert max_abs(res["out"], res["ref_out"]) <= TOL
        assert max_abs(res["lse"], res["ref_lse"]) <= TOL
        tw.advance()
        tw.migrate()
        tw.check_tables()
    tw.check_pages()


def test_device_errors_fail_closed(torch_cuda):
    """Free lists too short: the call changes nothing and sets the error word."""
    import paper_2608_23834_amd as mk
    torch = torch_cuda
    d = 128
    gp = mk.Pool(1, 2, 1, d, 3, 1, 16, np.ones(d, np.int8))
    bt = torch.full((1, 8), -1, dtype=torch.int32, device="cuda")
    tg = torch.full((1, 8), 0xFF, dtype=torch.uint8, device="cuda")
    x = torch.zeros((1, 64, 1, d), dtype=torch.int16, device="cuda")
    mk.kv_append_fp8(gp, -1, bt, tg, torch.zeros(1, dtype=torch.int32, device="cuda"),
                     torch.tensor([0, 64], dtype=torch.int32, device="cuda"), x, x)
    assert mk.kv_pool_check_errors(gp, clear=True) & mk.DEVERR["FP8_EXHAUSTED"]
    assert (bt.cpu().numpy() == -1).all() and mk.kv_pool_free_counts(gp) == (3, 1)
    x = x[:, :48].contiguous()
    mk.kv_append_fp8(gp, -1, bt, tg, torch.zeros(1, dtype=torch.int32, device="cuda"),
                     torch.tensor([0, 48], dtype=torch.int32, device="cuda"), x, x)
    assert mk.kv_pool_check_errors(gp) == 0
    # window 16 tokens, 48 tokens live: pages 0 and 1 leave it, TQ3 pool holds 1 page
    before = (bt.cpu().numpy().copy(), tg.cpu().numpy().copy())
    mk.kv_migrate_to_tq3(gp, bt, tg, None, torch.tensor([48], dtype=torch.int32, device="cuda"))
    assert mk.kv_pool_check_errors(gp, clear=True) & mk.DEVERR["TQ3_EXHAUSTED"]
    assert np.array_equal(bt.cpu().numpy(), before[0]) and np.array_equal(tg.cpu().numpy(), before[1])
    # an invalid sequence length gives zero output and the RANGE bit
    ws = mk.workspace(gp, 1, 8)
    out = torch.full((1, 2, d), 7.0, device="cuda")
    q = torch.zeros((1, 2, d), dtype=torch.int16, device="cuda")
    mk.paged_attn_decode(gp, 0, q, bt, tg, torch.tensor([0], dtype=torch.int32, device="cuda"),
                         out, None, ws)
    assert (out.cpu().numpy() == 0).all()
    assert mk.kv_pool_check_errors(gp, clear=True) & mk.DEVERR["RANGE"]


def _run_chunk_case(w, lens, n_q, recent=None, sample_stride=1, migrate_after=False):
    """Context of each request appended and migrated, then its chunk of n_q[r]
    tokens appended as FP8; chunk attention of those queries vs the oracle;
    optionally the pages that left the Recent window with the chunk are then
    re-encoded FP8 -> TQ3 and compared bit for bit."""
    from _harness import Twin, max_abs
    print(f"\n[chunk case] {w.name} lens={lens[:6]} n_q={n_q[:6]} W={recent}", flush=True)
    tw = Twin(w, lens=lens, recent=recent)
    tw.fill_to([l - n for l, n in zip(lens, n_q)])
    tw.migrate()
    tw.append(list(n_q))
    tw.check_tables()
    tw.check_pages()  # multi-token appends into partly filled pages, bit-exact
    res = tw.chunk(n_q, sample_stride=sample_stride)
    ref = res["ref_out"]
    rows = ~np.isnan(ref[:, 0, 0])
    err = max_abs(res["out"][rows], ref[rows])
    print(f"  rows compared {int(rows.sum())} of {rows.size}  max|dO| {err:.3e}", flush=True)
    assert np.all(np.isfinite(res["out"]))
    assert err <= TOL, err
    import paper_2608_23834_amd as mk
    assert mk.kv_pool_check_errors(tw.gpu) == 0
    if migrate_after:
        before = (tw.otags == 2).sum()
        tw.migrate()
        tw.check_tables()
        n8, n3 = tw.check_pages()
        print(f"  after the chunk: {int((tw.otags == 2).sum() - before)} pages re-encoded to TQ3, "
              f"live fp8 {n8} tq3 {n3}", flush=True)
    return tw, res


def test_chunk_tiny_d128(torch_cuda):
    """d = 128, GQA 8: a 64-query chunk at the end of 2,048 tokens, every query."""
    w = wl.workload(1)
    _run_chunk_case(w, [2048], [64])


def test_chunk_ragged_d256(torch_cuda):
    """d = 256, GQA 6: ragged chunks (100, 33, 1 and a whole short request)
    over mixed pages with a short Recent window, every query."""
    w = wl.scaled(wl.workload(5), (3000, 1500, 700, 40), n_layers=1, name="chunk-ragged")
    _run_chunk_case(w, list(w.ctx), [100, 33, 1, 40], recent=64)


def test_chunk_group12_d256(torch_cuda):
    """Twelve query heads per KV head: chunk rows (query, head) cross the
    32-row tiles at other boundaries; a chunk of 70 queries after 1,930
    tokens and one of 21 after 600, short Recent window, every query."""
    import dataclasses
    w = dataclasses.replace(wl.scaled(wl.workload(5), (2000, 621), n_layers=1, name="chunk-g12"),
                            n_kv_heads=2)
    _run_chunk_case(w, list(w.ctx), [70, 21], recent=48)


def test_chunk_over_tq3_chunk_pages(torch_cuda):
    """The chunk's own pages already re-encoded to TQ3 (the migration ran
    after the chunk was appended, with a 32-token Recent window): TQ3 pairs
    now hold tokens past some queries, so the causal mask applies to TQ3
    pages too (the masked score passes, including the pass that finishes the
    last pair), every query row against the oracle."""
    from _harness import Twin, max_abs
    w = wl.scaled(wl.workload(5), (900, 467), n_layers=1, name="chunk-tq3-masked")
    n_q = [200, 150]
    print(f"\n[chunk case] {w.name} lens={list(w.ctx)} n_q={n_q} W=32, migrated after the append",
          flush=True)
    tw = Twin(w, lens=list(w.ctx), recent=32)
    tw.fill_to([l - n for l, n in zip(w.ctx, n_q)])
    tw.append(n_q)
    tw.migrate()
    tw.check_tables()
    tw.check_pages()
    tags = tw.otags
    for r, (L, n) in enumerate(zip(w.ctx, n_q)):
        first, last = (L - n) // 16, (L - 1) // 16
        assert (tags[r, first:last + 1] == 2).sum() >= (last - first + 1) // 2  # mostly TQ3
    res = tw.chunk(n_q)
    err = max_abs(res["out"], res["ref_out"])
    print(f"  every row: max|dO| {err:.3e}", flush=True)
    assert np.all(np.isfinite(res["out"]))
    assert err <= TOL, err


def test_chunk_invalid_requests(torch_cuda):
    """Error paths of the chunk call.  A request whose length is shorter than
    its chunk gets zero rows and the range bit, while the other requests'
    rows equal those of the valid call bit for bit (each 128-row block is
    computed on its own).  Query ranges that overlap so that their row blocks
    exceed the launch set the range bit and leave the output untouched."""
    from _harness import Twin
    import paper_2608_23834_amd as mk
    torch = torch_cuda
    w = wl.scaled(wl.workload(5), (700, 300, 500), n_layers=1, name="chunk-errors")
    n_q = [40, 21, 33]
    tw = Twin(w, lens=list(w.ctx), with_oracle=False, recent=64)
    tw.fill_to([l - n for l, n in zip(w.ctx, n_q)])
    tw.migrate()
    tw.append(n_q)
    res = tw.chunk(n_q)
    assert mk.kv_pool_check_errors(tw.gpu, clear=True) == 0
    good, cu = res["out"], res["cu"]
    q = torch.from_numpy(res["q"].view(np.int16)).cuda()
    ws = mk.workspace(tw.gpu, tw.n_req, tw.max_pages, res["q"].shape[0])

    def call(cu_np, sl_np, n_rows):
        out = torch.full((n_rows, w.n_q_heads, w.head_dim), float("nan"), device="cuda")
        mk.paged_attn_chunk(tw.gpu, 0, q[:n_rows].contiguous(), torch.from_numpy(cu_np).cuda(), tw.bt,
                            tw.tags, torch.from_numpy(sl_np).cuda(), out, ws)
        torch.cuda.synchronize()
        return out.cpu().numpy()

    sl = res["seq_lens"].copy()
    sl[1] = 10  # below its 21 queries
    o = call(cu, sl, res["q"].shape[0])
    assert mk.kv_pool_check_errors(tw.gpu, clear=True) & mk.DEVERR["RANGE"]
    assert np.all(o[cu[1]:cu[2]] == 0.0)
    assert np.array_equal(o[:cu[1]], good[:cu[1]]) and np.array_equal(o[cu[2]:], good[cu[2]:])
    # requests 0 and 2 both claim queries 0..93 (request 1's range is
    # reversed): 5 + 1 + 5 row blocks against a launch of ceil(94 * 6 / 128)
    # + 3 = 8
    o = call(np.array([0, 94, 0, 94], np.int32), res["seq_lens"], 94)
    assert mk.kv_pool_check_errors(tw.gpu, clear=True) & mk.DEVERR["RANGE"]
    assert np.all(np.isnan(o))
    print("\n  invalid length: zero rows, others bit-identical; overlap: untouched", flush=True)


@pytest.mark.parametrize("n_q_heads,n_kv_heads", [(4, 4), (32, 2)])
def test_chunk_group_extremes(torch_cuda, n_q_heads, n_kv_heads):
    """The smallest and the largest GQA group (1 and 16 query heads per KV
    head): a 128-row block then holds 128 or 8 queries, so the row-block
    table and the row -> (query, head) mapping meet their edge cases; three
    requests with chunks of 129, 8 and 1 queries, every row."""
    import dataclasses
    w = dataclasses.replace(wl.scaled(wl.workload(5), (1100, 500, 260), n_layers=1,
                                      name=f"chunk-g{n_q_heads // n_kv_heads}"),
                            n_q_heads=n_q_heads, n_kv_heads=n_kv_heads)
    _run_chunk_case(w, list(w.ctx), [129, 8, 1], recent=48)


def test_pool_random_lifecycles(torch_cuda):
    """Seeded random sequences of pool calls on two layers — appends of up
    to 200 tokens per request, Retier with random anchor masks, Promote of a
    random third of the Stale pages, fused decode steps, Finish of random
    requests (which later append from zero again) — with tables, tags, free
    lists, reference counts and every page compared bit for bit after each
    call, decode outputs within 1e-3, and no error bits."""
    import dataclasses
    from _harness import Twin, max_abs
    import paper_2608_23834_amd as mk
    rng = np.random.default_rng(16)
    for sq in range(4):
        d = int(rng.choice([128, 256]))
        H, G = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 6, 8]))
        n_req = int(rng.integers(1, 5))
        cap = [int(rng.integers(64, 1500)) for _ in range(n_req)]
        recent = int(rng.choice([16, 32, 64, 256]))
        w = dataclasses.replace(wl.scaled(wl.workload(1 if d == 128 else 5), tuple(cap), n_layers=2,
                                          name=f"lifecycle-{sq}"), n_q_heads=H * G, n_kv_heads=H)
        print(f"\n[lifecycle {sq}] d {d} H {H} G {G} capacity {cap} W {recent}", flush=True)
        tw = Twin(w, n_layers=2, lens=cap, recent=recent, headroom=64)
        done = []
        for step in range(12):
            op = str(rng.choice(["append", "migrate", "promote", "step", "finish"],
                                p=[0.35, 0.25, 0.15, 0.15, 0.10]))
            if op == "append":
                cnt = [int(max(0, min(rng.integers(0, 200), c - cur))) for c, cur in zip(cap, tw.cur)]
                if sum(cnt) == 0:
                    continue
                tw.append(cnt)
            elif op == "migrate":
                tw.migrate(anchor=(rng.random((n_req, tw.max_pages)) < 0.1).astype(np.uint8))
            elif op == "promote":
                tw.promote(((tw.otags == 2) & (rng.random(tw.otags.shape) < 0.3)).astype(np.uint8))
            elif op == "step":
                if min(tw.cur) < 1 or any(c >= cp + 32 for c, cp in zip(tw.cur, cap)):
                    continue
                res = tw.decode_append(layer=int(rng.integers(0, 2)))
                tw.advance()
                err = max(max_abs(res["out"], res["ref_out"]), max_abs(res["lse"], res["ref_lse"]))
                assert err <= TOL, (sq, step, err)
            else:
                tw.finish(sorted(set(int(x) for x in rng.integers(0, n_req, size=int(rng.integers(1, n_req + 1))))))
            tw.check_tables()
            tw.check_refcounts()
            tw.check_pages()
            assert mk.kv_pool_check_errors(tw.gpu, clear=True) == 0, (sq, step, op)
            done.append(op)
        print(f"  bit-exact after: {' '.join(done)}", flush=True)


def test_decode_random_shapes(torch_cuda):
    """Seeded random decode calls: head dim 128 or 256, 1-8 KV heads, GQA
    groups 1-16, 1-8 requests of 0-3,000 tokens (empty ones included),
    Recent windows of 16-1,024 tokens, the stage schedule deterministic or
    claimed at run time; a plain decode, then a fused decode step, each
    against the oracle (outputs and lse), tables bit-exact, no error bits."""
    import dataclasses
    from _harness import Twin, max_abs
    import paper_2608_23834_amd as mk
    rng = np.random.default_rng(59008)
    for c in range(6):
        d = int(rng.choice([128, 256]))
        H, G = int(rng.choice([1, 2, 4, 8])), int(rng.choice([1, 2, 3, 4, 6, 8, 12, 16]))
        lens = [int(rng.integers(0, 3000)) for _ in range(int(rng.integers(1, 9)))]
        lens[0] = max(lens[0], 1)
        recent = int(rng.choice([16, 32, 64, 256, 1024]))
        det = bool(rng.integers(0, 2))
        w = dataclasses.replace(wl.scaled(wl.workload(1 if d == 128 else 5), tuple(max(L, 1) for L in lens),
                                          n_layers=1, name=f"decode-random-{c}"),
                                n_q_heads=H * G, n_kv_heads=H)
        print(f"\n[case] d {d} H {H} G {G} lens {lens} W {recent} deterministic {det}", flush=True)
        tw = Twin(w, lens=[max(L, 1) for L in lens], recent=recent, headroom=16)
        tw.fill_to(lens)
        tw.migrate()
        mk.paged_attn_set_deterministic(tw.gpu, det)
        r1 = tw.decode()
        e1 = max(max_abs(r1["out"], r1["ref_out"]), max_abs(r1["lse"], r1["ref_lse"]))
        r2 = tw.decode_append()
        tw.advance()
        e2 = max(max_abs(r2["out"], r2["ref_out"]), max_abs(r2["lse"], r2["ref_lse"]))
        tw.check_tables()
        print(f"  decode max|d| {e1:.3e}, fused step {e2:.3e}", flush=True)
        assert np.all(np.isfinite(r1["out"])) and np.all(np.isfinite(r2["out"]))
        assert e1 <= TOL and e2 <= TOL, (c, e1, e2)
        assert mk.kv_pool_check_errors(tw.gpu) == 0


def test_chunk_random_shapes(torch_cuda):
    """Seeded random chunk calls: head dim 128 or 256, 1-4 KV heads, GQA
    groups 1-16, 1-4 requests of up to 2,500 tokens with chunks of 1-300
    queries, Recent windows of 16-256 tokens, the migration before or after
    the chunk's append (so TQ3 pairs with masked tokens appear); every row
    against the oracle, no error bits."""
    import dataclasses
    from _harness import Twin, max_abs
    import paper_2608_23834_amd as mk
    rng = np.random.default_rng(2608)
    for c in range(6):
        d = int(rng.choice([128, 256]))
        H, G = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 3, 4, 6, 8, 12, 16]))
        lens = [int(rng.integers(1, 2500)) for _ in range(int(rng.integers(1, 5)))]
        n_q = [int(rng.integers(1, min(L, 300) + 1)) for L in lens]
        recent = int(rng.choice([16, 32, 48, 64, 256]))
        after = bool(rng.integers(0, 2))
        w = dataclasses.replace(wl.scaled(wl.workload(1 if d == 128 else 5), tuple(lens), n_layers=1,
                                          name=f"chunk-random-{c}"), n_q_heads=H * G, n_kv_heads=H)
        print(f"\n[chunk case] d {d} H {H} G {G} lens {lens} n_q {n_q} W {recent} "
              f"migrated {'after' if after else 'before'} the append", flush=True)
        tw = Twin(w, lens=lens, recent=recent)
        tw.fill_to([L - n for L, n in zip(lens, n_q)])
        if not after:
            tw.migrate()
        tw.append(n_q)
        if after:
            tw.migrate()
        res = tw.chunk(n_q)
        err = max_abs(res["out"], res["ref_out"])
        print(f"  every row: max|dO| {err:.3e}", flush=True)
        assert np.all(np.isfinite(res["out"]))
        assert err <= TOL, (c, err)
        assert mk.kv_pool_check_errors(tw.gpu) == 0


def test_chunk_last_query_matches_decode(torch_cuda):
    """Property that holds at any size, checked without the oracle: the last
    query of each request's chunk sees the whole context, so the chunk kernel's
    output for it equals the decode kernel's for the same query (two kernels,
    two tilings, one definition)."""
    from _harness import Twin, max_abs
    w = wl.scaled(wl.workload(5), (9000, 4100, 1500), n_layers=1, name="chunk-vs-decode")
    n_q = [128, 40, 7]
    tw = Twin(w, lens=list(w.ctx), with_oracle=False, recent=256)
    tw.fill_to([l - n for l, n in zip(w.ctx, n_q)])
    tw.migrate()
    tw.append(n_q)
    res = tw.chunk(n_q)
    last = res["cu"][1:] - 1
    dec = tw.decode(q=res["q"][last])
    err = max_abs(res["out"][last], dec["out"])
    print(f"\n  chunk vs decode, last query of each request: max|dO| {err:.3e}", flush=True)
    assert err <= TOL, err


@pytest.mark.timeout(900)
def test_chunk_config5_full_size(torch_cuda):
    """Config 5 at full size: 8 requests, a 512-query chunk each against a
    65,536-token context of mixed pages (every query row of requests 0 and 1,
    every 8th and the last of the others), then the migration of the pages
    the chunk pushed out of the Recent window, bit-exact."""
    w = wl.workload(5)
    assert all(L == 65536 + 512 for L in w.ctx)
    tw, res = _run_chunk_case(w, list(w.ctx), [512] * 8, sample_stride=[1, 1] + [8] * 6,
                              migrate_after=True)
    assert np.all(np.isfinite(res["out"]))
    # 512 new tokens push 32 pages per request out of the 1,024-token window;
    # anchors among them stay FP8
    tags = tw.otags
    for r in range(8):
        assert (tags[r] == 0).sum() == 1024 // 16
