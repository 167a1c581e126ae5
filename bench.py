#!/usr/bin/env python3
"""Benchmark of the Minima-KV mixed FP8/TQ3 decode path on one MI355X.

Workload: the long-context pair (2 requests x 59,008 tokens, 16 full-attention
layers, 24 query / 4 KV heads, head dim 256, 16-token pages, Recent window
2,048 tokens, anchors = first 8 pages + 1 % of the rest), synthetic seeded
data with the distributions of mkv_workloads.

One step is one decode step of the whole path: for each of the 16 layers,
paged_attn_decode_append (the new token of each request appended inside the
decode launch, then attention over the grown context); after the last layer
kv_migrate_to_tq3 (pages leaving the Recent window).  The same steps with the
append as its own call (kv_append_fp8, then paged_attn_decode) are timed too,
for comparison, and the same KV held all-FP8 and all-bf16 is timed as dense
controls (decode-only sweeps of every layer on the three caches).  All inputs
are resident in HBM before the timed region.  The headline value is the step
time per layer (us/layer, lower is better); the decode kernel's own time, its
effective KV bandwidth and its fraction of the 8 TB/s HBM peak are reported
next to it, measured with HIP events on the stream the kernels run on.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3]
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import mkv_workloads as wl  # noqa: E402

HBM_PEAK = 8.0e12  # MI355X HBM3E, bytes/s
MFMA_FP8_PEAK = 5.0e15  # dense fp8 MFMA, MI355X
MFMA_F16_PEAK = 2.5e15  # MI355X dense f16 MFMA, flop/s
PAGE = 16


def kv_bytes_of(tags_row: np.ndarray, seq_len: int, d: int, n_kv_heads: int) -> int:
    """Algorithmic KV bytes one decode reads for one request: per attended
    page-head, FP8 = 2*B*d codes + 8 B scales, TQ3 = 2*B*3d/8 codes + 2*B gamma
    + 4*d V scale/zero (B = valid tokens of the page)."""
    tot = 0
    npg = (seq_len + PAGE - 1) // PAGE
    for p in range(npg):
        b = min(PAGE, seq_len - p * PAGE)
        if tags_row[p] == 2:
            tot += 2 * b * 3 * d // 8 + 2 * b + 4 * d
        else:
            tot += 2 * b * d + 8
    return tot * n_kv_heads


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_kernel_long_pair_2x59008_hbm_traffic.txt")
DECODE_SOURCES = [os.path.join(ROOT, "paper_2608_23834_amd", "csrc", f)
                  for f in ("mkv_decode.hip", "mkv_append.h", "mkv_attn.h", "mkv_device.h")]


def decode_source_hash() -> str:
    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload_name: str):
    """HBM bytes per decode launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary (copy-calibrated), or None when that summary was taken
    on other decode sources or another workload."""
    try:
        with open(TRAFFIC_FILE) as fh:
            kv = dict(line.split(":", 1) for line in fh if ":" in line and not line.startswith(" "))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("decode_sources_sha256") != decode_source_hash() or kv.get("workload") != workload_name:
        return None
    return int(kv["hbm_bytes_per_launch"])


def build_state(w, n_layers, extra_tokens, mk, torch, also=None):
    """Pool for `n_layers` layers filled with the workload's context, migrated.
    `also(layer, k, v, cu)`, if given, receives each layer's K/V (device bf16
    bits) too, for the dense controls."""
    lens = list(w.ctx)
    n_req = len(lens)
    max_pages = (max(lens) + extra_tokens + PAGE - 1) // PAGE
    tot_pages = sum((l + extra_tokens + PAGE - 1) // PAGE for l in lens)
    pool = mk.Pool(n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, tot_pages + 16, tot_pages + 16,
                   w.recent, wl.rot_signs(w), wl.free_order(w, tot_pages + 16, "fp8"),
                   wl.free_order(w, tot_pages + 16, "tq3"))
    bt = torch.full((n_req, max_pages), -1, dtype=torch.int32, device="cuda")
    tags = torch.full((n_req, max_pages), 0xFF, dtype=torch.uint8, device="cuda")
    sb = torch.zeros(n_req, dtype=torch.int32, device="cuda")
    cu = torch.tensor(np.r_[0, np.cumsum(lens)], dtype=torch.int32, device="cuda")

    def gen(layer):
        ks, vs = [], []
        for r, L in enumerate(lens):
            k, v = wl.kv_layer(w, layer, L, token_offset=r * 1_000_000)
            ks.append(k)
            vs.append(v)
        return np.concatenate(ks), np.concatenate(vs)

    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        futs = [ex.submit(gen, l) for l in range(n_layers)]
        for l, f in enumerate(futs):
            k, v = f.result()
            kt = torch.from_numpy(k.view(np.int16)).cuda()
            vt = torch.from_numpy(v.view(np.int16)).cuda()
            mk.kv_append_fp8(pool, l, bt, tags, sb, cu, kt, vt)
            if also is not None:
                also(l, kt, vt, cu)
            torch.cuda.synchronize()
            del kt, vt
    am = torch.from_numpy(wl.anchor_mask(w, max_pages)).cuda()
    sl = torch.tensor(lens, dtype=torch.int32, device="cuda")
    mk.kv_migrate_to_tq3(pool, bt, tags, am, sl)
    torch.cuda.synchronize()
    err = mk.kv_pool_check_errors(pool)
    if err:
        raise RuntimeError(f"device error word {err:#x} while building the state")
    return pool, bt, tags, am, max_pages


def cpu_baseline(w, budget_s=25.0, max_req=4):
    """The CPU oracle, as it stands, on a bounded sample of the same workload:
    one layer (all heads) of every request, or of max_req of them (the
    shortest, the longest and two between) when there are more, with the same
    K/V bytes as the GPU state; the state is built by the oracle's own append
    + migrate (not timed), the oracle's decode is timed and, for a sample of
    requests, scaled by total tokens / sampled tokens."""
    import oracle
    lens_all = list(w.ctx)
    pick = list(range(len(lens_all)))
    if len(pick) > max_req:
        order = np.argsort(lens_all, kind="stable")
        n = len(order)
        pick = sorted({int(order[0]), int(order[n // 3]), int(order[2 * n // 3]), int(order[-1])})
    lens = [lens_all[i] for i in pick]
    n_req = len(lens)
    max_pages = (max(lens_all) + PAGE - 1) // PAGE
    tot = sum((l + PAGE - 1) // PAGE for l in lens) + 16
    P = oracle.Pool(1, w.n_q_heads, w.n_kv_heads, w.head_dim, tot, tot, w.recent, wl.rot_signs(w),
                    wl.free_order(w, tot, "fp8"), wl.free_order(w, tot, "tq3"))
    bt = np.full((n_req, max_pages), -1, np.int32)
    tags = np.full((n_req, max_pages), 0xFF, np.uint8)
    ks, vs = zip(*(wl.kv_layer(w, 0, L, token_offset=i * 1_000_000) for i, L in zip(pick, lens)))
    k = np.concatenate(ks)[None]
    v = np.concatenate(vs)[None]
    assert P.append(-1, bt, tags, np.zeros(n_req, np.int32),
                    np.r_[0, np.cumsum(lens)].astype(np.int32), k, v) == 0
    del ks, vs, k, v
    P.migrate(bt, tags, np.ascontiguousarray(wl.anchor_mask(w, max_pages)[pick]),
              np.array(lens, np.int32))
    q = np.ascontiguousarray(wl.q_decode(w, 0)[pick])
    sl = np.array(lens, np.int32)
    times = []
    t_end = time.perf_counter() + budget_s
    while True:
        t0 = time.perf_counter()
        P.decode(0, q, bt, tags, sl)
        times.append(time.perf_counter() - t0)
        if time.perf_counter() + times[-1] > t_end or len(times) >= 5:
            break
    kvb = sum(kv_bytes_of(tags[r], lens[r], w.head_dim, w.n_kv_heads) for r in range(n_req))
    med = float(np.median(times))
    scale = sum(lens_all) / sum(lens)
    what = (f"all {n_req} requests" if n_req == len(lens_all) else
            f"{n_req} of {len(lens_all)} requests (lengths {lens}), time x {scale:.2f} = total / "
            f"sampled tokens")
    return {"value": med * scale * 1e6, "unit": "us/layer", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"one layer of {w.name}, {what}, all {w.n_q_heads}/{w.n_kv_heads} heads, "
                      f"fp64 decode over the reconstructed cache, median of {len(times)} runs",
            "kv_gb_per_s": kvb / med / 1e9,
            "cpu": _cpu_model()}


def chunk_bench(mk, torch, reps=5):
    """Chunked prefill (paged_attn_chunk) on the chunk workload at full size:
    8 requests, each with a 512-query chunk appended after 65,536 context
    tokens (mixed FP8/TQ3 pages), one layer.  HIP events on the current
    stream around `reps` calls; MFMA share = algorithmic causal-attention
    flops (4 d flops per query-key pair and head) / time / dense f16 peak."""
    w = wl.workload(5)
    lens = list(w.ctx)
    n_req, nq = len(lens), 512
    w0 = wl.scaled(w, tuple(L - nq for L in lens), n_layers=1, name=w.name + "-context")
    pool, bt, tags, am, mp = build_state(w0, 1, nq + 16, mk, torch)
    ks, vs = zip(*(wl.kv_layer(w, 0, nq, token_offset=r * 1_000_000 + L - nq)
                   for r, L in enumerate(lens)))
    sb = torch.tensor([L - nq for L in lens], dtype=torch.int32, device="cuda")
    cu = torch.tensor(np.r_[0, np.cumsum([nq] * n_req)], dtype=torch.int32, device="cuda")
    mk.kv_append_fp8(pool, 0, bt, tags, sb, cu,
                     torch.from_numpy(np.concatenate(ks).view(np.int16)).cuda(),
                     torch.from_numpy(np.concatenate(vs).view(np.int16)).cuda())
    q = torch.from_numpy(wl.q_chunk(w, 0, nq).view(np.int16)).cuda()
    sl = torch.tensor(lens, dtype=torch.int32, device="cuda")
    out = torch.empty((n_req * nq, w.n_q_heads, w.head_dim), device="cuda")
    ws = mk.workspace(pool, n_req, mp, n_req * nq)
    mk.paged_attn_chunk(pool, 0, q, cu, bt, tags, sl, out, ws)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        mk.paged_attn_chunk(pool, 0, q, cu, bt, tags, sl, out, ws)
    e1.record(stream)
    torch.cuda.synchronize()
    err = mk.kv_pool_check_errors(pool)
    if err:
        raise RuntimeError(f"device error word {err:#x} in the chunk benchmark")
    us = e0.elapsed_time(e1) / reps * 1e3
    pairs = sum(nq * (L - nq) + nq * (nq + 1) // 2 for L in lens)  # causal (query, key) pairs
    flops = 4.0 * pairs * w.n_q_heads * w.head_dim
    tf = flops / (us * 1e-6) / 1e12
    del pool
    return {"workload": f"{w.name}: {n_req} requests x {nq}-query chunk after "
                        f"{lens[0] - nq} context tokens, 1 layer, {w.n_q_heads}/{w.n_kv_heads} "
                        f"heads, d {w.head_dim}",
            "us_per_call": round(us, 1), "algorithmic_tflop": round(flops / 1e12, 3),
            "tflop_per_s": round(tf, 1), "mfma_peak_tflop_per_s": MFMA_F16_PEAK / 1e12,
            "mfma_frac": round(tf * 1e12 / MFMA_F16_PEAK, 4),
            "mfma_frac_of_fp8_peak": round(tf * 1e12 / MFMA_FP8_PEAK, 4),
            "mfma_dtypes": "TQ3 scores on fp8 MFMA (3-term E4M3 query), PV and FP8-page scores "
                           "on f16 MFMA (hi + lo operands), fp32 accumulate",
            "kernel": "chunk_kernel<256> (+ partition_kernel, chunk_stages_kernel, chunk_rows_kernel)"}


class DenseControls:
    """The same KV as the mixed pool held all-FP8 (a pool with no Retier: every
    page stays FP8) and all-bf16 (the library's control pages), filled layer
    by layer from the K/V build_state generates (the dense controls of the
    paper's fused-decode canary, Sec. 6.3)."""

    def __init__(self, w, n_layers, mk, torch):
        lens = list(w.ctx)
        self.w, self.lens, self.n_layers = w, lens, n_layers
        self.mp = (max(lens) + PAGE - 1) // PAGE
        n_pg = sum((L + PAGE - 1) // PAGE for L in lens)
        self.fp8 = mk.Pool(n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, n_pg + 16, 1,
                           w.recent, wl.rot_signs(w), wl.free_order(w, n_pg + 16, "fp8"), None)
        self.bt8 = torch.full((len(lens), self.mp), -1, dtype=torch.int32, device="cuda")
        self.tags8 = torch.full((len(lens), self.mp), 0xFF, dtype=torch.uint8, device="cuda")
        self.bf16 = mk.ControlBf16(n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, n_pg)
        ids = np.random.default_rng(w.seed).permutation(n_pg).astype(np.int32)
        bt = np.full((len(lens), self.mp), -1, np.int32)
        k0 = 0
        for r, L in enumerate(lens):
            npg = (L + PAGE - 1) // PAGE
            bt[r, :npg] = ids[k0:k0 + npg]
            k0 += npg
        self.bt16 = torch.from_numpy(bt).cuda()
        self.sb = torch.zeros(len(lens), dtype=torch.int32, device="cuda")
        self.sl = torch.tensor(lens, dtype=torch.int32, device="cuda")
        self.mk = mk

    def add_layer(self, layer, k, v, cu):
        self.mk.kv_append_fp8(self.fp8, layer, self.bt8, self.tags8, self.sb, cu, k, v)
        self.bf16.write(layer, self.bt16, self.sb, cu, k, v)

    def time(self, torch, q_all, mixed, reps):
        """Decode-only sweeps of every layer (no append, no Retier) on the
        mixed pool as it stands and on both controls; HIP events around
        `reps` sweeps; us/layer, KV bytes per layer and GB/s for each."""
        mk, w, n_layers = self.mk, self.w, self.n_layers
        n_req, d, H = len(self.lens), w.head_dim, w.n_kv_heads
        out = torch.zeros((n_req, w.n_q_heads, d), device="cuda")
        stream = torch.cuda.current_stream()

        def sweep_time(fn):
            for _ in range(2):
                for l in range(n_layers):
                    fn(l)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                for l in range(n_layers):
                    fn(l)
            e1.record(stream)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) * 1e3 / (reps * n_layers)

        pool, bt, tags, sl = mixed
        ws_m = mk.workspace(pool, n_req, bt.shape[1])
        t_mixed = sweep_time(lambda l: mk.paged_attn_decode(pool, l, q_all[l], bt, tags, sl, out,
                                                            None, ws_m))
        tg = tags.cpu().numpy()
        sl_h = sl.cpu().numpy()
        b_mixed = sum(kv_bytes_of(tg[r], int(sl_h[r]), d, H) for r in range(n_req))
        ws8 = mk.workspace(self.fp8, n_req, self.mp)
        t_fp8 = sweep_time(lambda l: mk.paged_attn_decode(self.fp8, l, q_all[l], self.bt8,
                                                          self.tags8, self.sl, out, None, ws8))
        tg8 = self.tags8.cpu().numpy()
        assert (tg8[tg8 != 0xFF] == 0).all()
        b_fp8 = sum(kv_bytes_of(tg8[r], L, d, H) for r, L in enumerate(self.lens))
        ws16 = self.bf16.workspace(n_req, self.mp)
        t_bf16 = sweep_time(lambda l: self.bf16.decode(l, q_all[l], self.bt16, self.sl, out, None,
                                                       ws16))
        b_bf16 = sum(2 * L * d * 2 for L in self.lens) * H
        for pool_ in (pool, self.fp8):
            if mk.kv_pool_check_errors(pool_):
                raise RuntimeError("device error word set in the dense-control sweeps")

        def row(t, b):
            return {"us_per_layer": round(t, 3), "kv_bytes_per_layer": int(b),
                    "kv_gb_per_s": round(b / (t * 1e-6) / 1e9, 1),
                    "frac_of_hbm_peak": round(b / (t * 1e-6) / HBM_PEAK, 4)}

        return {
            "timing": f"decode only (decode + merge per layer, no append, no Retier), "
                      f"{reps} sweeps of {n_layers} layers between two HIP events",
            "mixed": {**row(t_mixed, b_mixed), "seq_len": int(sl_h[0]),
                      "kernel": "decode_kernel<256, true, true, false, false> + decode_merge_kernel"},
            "all_fp8": {**row(t_fp8, b_fp8), "seq_len": self.lens[0],
                        "kernel": "the same kernels, every page FP8"},
            "all_bf16": {**row(t_bf16, b_bf16), "seq_len": self.lens[0],
                         "kernel": "bf16_decode_kernel<256, 8> + bf16_merge_kernel (control)"},
            "mixed_vs_fp8_throughput": round(t_fp8 / t_mixed, 4),
            "mixed_vs_bf16_throughput": round(t_bf16 / t_mixed, 4),
            "fp8_over_mixed_kv_bytes": round(b_fp8 / b_mixed, 4),
            "bf16_over_mixed_kv_bytes": round(b_bf16 / b_mixed, 4),
            "paper_context": "the paper's canary on its Blackwell GPU: 0.9821x the dense FP8 "
                             "route's throughput for the whole serving step while reading "
                             "3.625x fewer KV bytes than its BF16-priced cache (Sec. 6.3)",
        }


def score_overhead(mk, torch, pool, bt, tags, sl, q_all, n_layers, w, reps=5, det_after=False):
    """Cost of the direct attention-score collector (Sec. 3.1 / 4.2) on the
    mixed cache: decode-only sweeps of every layer with paged_attn_decode, then
    with paged_attn_decode_scores plus kv_page_scores_update (all query heads
    sampled), HIP events around `reps` sweeps."""
    n_req, mp = bt.shape
    d, Hq = w.head_dim, w.n_q_heads
    out = torch.zeros((n_req, Hq, d), device="cuda")
    lse = torch.zeros((n_req, Hq), device="cuda")
    ws = mk.workspace(pool, n_req, mp)
    pm = torch.zeros((n_req, mp, Hq, 2), device="cuda")
    scores = torch.zeros((n_req, mp), device="cuda")
    hm = torch.ones(Hq, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    mk.paged_attn_set_deterministic(pool, False)

    def sweep(fn):
        for l in range(n_layers):
            fn(l)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            for l in range(n_layers):
                fn(l)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / (reps * n_layers)

    t_plain = sweep(lambda l: mk.paged_attn_decode(pool, l, q_all[l], bt, tags, sl, out, lse, ws))

    def scored(l):
        mk.paged_attn_decode_scores(pool, l, q_all[l], bt, tags, sl, out, lse, ws, pm)
        mk.kv_page_scores_update(pool, sl, lse, pm, hm, 0.9, scores)

    t_score = sweep(scored)
    # the same plain sweeps with the fixed (deterministic) stage schedule
    mk.paged_attn_set_deterministic(pool, True)
    try:
        t_det = sweep(lambda l: mk.paged_attn_decode(pool, l, q_all[l], bt, tags, sl, out, lse, ws))
    finally:
        mk.paged_attn_set_deterministic(pool, det_after)
    if mk.kv_pool_check_errors(pool):
        raise RuntimeError("device error word set in the score-collector sweeps")
    return {"decode_us_per_layer": round(t_plain, 3),
            "decode_with_scores_us_per_layer": round(t_score, 3),
            "overhead_frac": round(t_score / t_plain - 1.0, 4),
            "deterministic_decode_us_per_layer": round(t_det, 3),
            "what": "paged_attn_decode_scores + kv_page_scores_update (every query head "
                    "sampled, EWMA beta 0.9) against paged_attn_decode, decode-only sweeps of "
                    f"all {n_layers} layers, {reps} sweeps between two HIP events; and "
                    "paged_attn_decode with paged_attn_set_deterministic on"}


def stream_probe(mk, torch, nbytes, achieved, reps=20):
    """A plain streaming read of `nbytes` (the library's probe kernel, 16-byte
    loads, each byte once), cycling through 16 buffers so no read is served
    from the 256 MB last-level cache, timed with HIP events around each call:
    a measured bandwidth ceiling for a kernel that reads that many bytes."""
    n = nbytes // 16 * 16
    bufs = [torch.ones(n // 4, dtype=torch.float32, device="cuda") for _ in range(16)]
    sink = torch.zeros(mk.STREAM_PROBE_WORKGROUPS, dtype=torch.int32, device="cuda")
    for b in bufs:
        mk.mkv_stream_read(b, sink)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ts = []
    for i in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        mk.mkv_stream_read(bufs[i % 16], sink)
        e1.record(stream)
        ts.append((e0, e1))
    torch.cuda.synchronize()
    us = float(np.mean([a.elapsed_time(b) for a, b in ts[2:]]) * 1e3)
    bw = n / (us * 1e-6)
    del bufs
    return {"bytes": n, "us": round(us, 2), "gb_per_s": round(bw / 1e9, 1),
            "frac_of_peak": round(bw / HBM_PEAK, 4),
            "decode_frac_of_stream": round(achieved / bw, 4),
            "kernel": "stream_read_kernel (mkv_stream_read), HIP events around each call "
                      "(these also span the launch; the decode scan is timed by its dispatch, "
                      "so decode_frac_of_stream reads a few % high)"}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    # the headline pass runs first: enough warm-up steps that its working set
    # (TLBs, caches) is as warm as the later passes' (3 steps left the 64-request
    # batch's first pass 12 % slow)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--cfg", type=int, default=3)
    ap.add_argument("--layers", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true",
                    help="skip the comparison pass with the append as its own call")
    ap.add_argument("--no-chunk", action="store_true",
                    help="skip the chunked-prefill measurement")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run one 1 GiB device-to-device copy (calibrates HBM byte counters)")
    ap.add_argument("--no-stream-probe", action="store_true",
                    help="skip the streaming-read probe (a kernel that reads the decode's byte "
                         "count once, over cycled buffers: the measured bandwidth ceiling)")
    ap.add_argument("--no-scores", action="store_true",
                    help="skip timing the attention-score collector")
    ap.add_argument("--no-controls", action="store_true",
                    help="skip the dense controls (the same KV all-FP8 and all-bf16)")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the pass that replays the same steps as captured HIP graphs")
    ap.add_argument("--deterministic", action="store_true",
                    help="decode with the fixed stage schedule (bit-identical outputs call to call)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the decode path would shard by request or KV head with no exchange between "
              "GPUs)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_23834_amd as mk
    mk.lib()
    torch.cuda.init()
    w = wl.workload(args.cfg)
    n_layers = args.layers or w.n_layers
    n_pass = 2 + (not args.no_unfused) + (not args.no_graph)
    n_steps = args.warmup + n_pass * args.steps  # warmup, pass A, pass B (, pass C) (, pass D)
    t_setup = time.perf_counter()
    ctl = None if args.no_controls or args.cfg not in (2, 3) else DenseControls(w, n_layers, mk, torch)
    pool, bt, tags, am, max_pages = build_state(w, n_layers, n_steps + 16, mk, torch,
                                                None if ctl is None else ctl.add_layer)
    lens = list(w.ctx)
    n_req = len(lens)
    Hkv, d = w.n_kv_heads, w.head_dim

    # per-step inputs, resident before timing
    q_all = torch.from_numpy(np.stack([wl.q_decode(w, l) for l in range(n_layers)]).view(np.int16)).cuda()
    new_k = np.zeros((n_layers, n_steps, n_req, Hkv, d), np.uint16)
    new_v = np.zeros_like(new_k)
    for l in range(n_layers):
        for r in range(n_req):
            k, v = wl.kv_layer(w, l, n_steps, token_offset=r * 1_000_000 + lens[r])
            new_k[l, :, r] = k
            new_v[l, :, r] = v
    nk = torch.from_numpy(new_k.view(np.int16)).cuda()
    nv = torch.from_numpy(new_v.view(np.int16)).cuda()
    seq_before = torch.tensor([[L + s for L in lens] for s in range(n_steps)], dtype=torch.int32,
                              device="cuda")
    seq_after = seq_before + 1
    cu1 = torch.arange(n_req + 1, dtype=torch.int32, device="cuda")
    out = torch.zeros((n_req, w.n_q_heads, d), device="cuda")
    ws = mk.workspace(pool, n_req, max_pages)
    if args.deterministic:
        mk.paged_attn_set_deterministic(pool, True)
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup
    print(f"[bench] {w.name}: state built in {setup_s:.1f} s", file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    n_ev = args.steps * n_layers
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n_ev)]

    def step(s):
        for l in range(n_layers):
            mk.paged_attn_decode_append(pool, l, q_all[l], nk[l, s], nv[l, s], bt, tags,
                                        seq_before[s], out, None, ws)
        mk.kv_migrate_to_tq3(pool, bt, tags, am, seq_after[s])

    def step_unfused(s):
        for l in range(n_layers):
            mk.kv_append_fp8(pool, l, bt, tags, seq_before[s], cu1, nk[l, s], nv[l, s])
            mk.paged_attn_decode(pool, l, q_all[l], bt, tags, seq_after[s], out, None, ws)
        mk.kv_migrate_to_tq3(pool, bt, tags, am, seq_after[s])

    for s in range(args.warmup):
        step(s)
    torch.cuda.synchronize()
    # pass A (headline): whole decode steps, events only around the timed region
    tags_start = tags.cpu().numpy()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for s in range(args.warmup, args.warmup + args.steps):
        step(s)
    t1.record(stream)
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    tags_mid = tags.cpu().numpy()
    # pass B: the same steps again with HIP events around every decode call;
    # the library's own events (same stream) time the split-scan and merge
    # kernels of each step's last decode call, read once the step is queued
    mk.paged_attn_set_timing(pool, True)
    scan_us, merge_us = [], []
    for i, s in enumerate(range(args.warmup + args.steps, args.warmup + 2 * args.steps)):
        evs = ev[i * n_layers:(i + 1) * n_layers]
        for l in range(n_layers):
            evs[l][0].record(stream)
            mk.paged_attn_decode_append(pool, l, q_all[l], nk[l, s], nv[l, s], bt, tags,
                                        seq_before[s], out, None, ws)
            evs[l][1].record(stream)
        a_us, m_us = mk.paged_attn_last_times(pool)
        scan_us.append(a_us)
        merge_us.append(m_us)
        mk.kv_migrate_to_tq3(pool, bt, tags, am, seq_after[s])
    torch.cuda.synchronize()
    mk.paged_attn_set_timing(pool, False)
    dec_ms = np.array([a.elapsed_time(b) for a, b in ev])
    scan_us = np.array(scan_us)
    merge_us = np.array(merge_us)
    err = mk.kv_pool_check_errors(pool)
    if err:
        raise RuntimeError(f"device error word {err:#x} during the benchmark")
    tags_end = tags.cpu().numpy()
    # pass C: the append as its own call (two launches per layer), whole steps
    unfused_ms = None
    if not args.no_unfused:
        c0 = torch.cuda.Event(enable_timing=True)
        c1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        c0.record(stream)
        for s in range(args.warmup + 2 * args.steps, args.warmup + 3 * args.steps):
            step_unfused(s)
        c1.record(stream)
        torch.cuda.synchronize()
        unfused_ms = c0.elapsed_time(c1) / args.steps
        err = mk.kv_pool_check_errors(pool)
        if err:
            raise RuntimeError(f"device error word {err:#x} during the benchmark")
    # pass D: the same whole steps (fused append, decode, Retier) captured once
    # each into a HIP graph -- the serving loop's graph path (Sec. 4.1) -- and
    # replayed in order; the same kernels, without the per-launch host gaps
    graph_ms = None
    if not args.no_graph:
        s_first = args.warmup + (3 if not args.no_unfused else 2) * args.steps
        graphs = []
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        for s in range(s_first, s_first + args.steps):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=cap):
                step(s)
            graphs.append(g)
        stream.wait_stream(cap)
        torch.cuda.synchronize()
        g0 = torch.cuda.Event(enable_timing=True)
        g1 = torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for g in graphs:
            g.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        graph_ms = g0.elapsed_time(g1) / args.steps
        err = mk.kv_pool_check_errors(pool)
        if err:
            raise RuntimeError(f"device error word {err:#x} in the graph pass")
        del graphs
    sl0 = [L + args.warmup + args.steps + 1 for L in lens]
    sl1 = [L + args.warmup + 2 * args.steps for L in lens]
    kvb0 = sum(kv_bytes_of(tags_mid[r], sl0[r], d, Hkv) for r in range(n_req))
    kvb1 = sum(kv_bytes_of(tags_end[r], sl1[r], d, Hkv) for r in range(n_req))
    kv_bytes = 0.5 * (kvb0 + kvb1)
    dec_us = float(dec_ms.mean() * 1e3)
    scan_mean = float(scan_us.mean())
    achieved = kv_bytes / (scan_mean * 1e-6)
    traffic = measured_traffic(w.name)
    ms_per_step = total_ms / args.steps
    counters = mk.kv_pool_counters(pool)

    res = {
        "metric": "mixed FP8/TQ3 decode attn: us/layer, effective KV GB/s, % of HBM roofline",
        "value": round(ms_per_step * 1e3 / n_layers, 3),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8/f16 MFMA, fp32 accumulate",
        "dtype_detail": "TQ3 scores on the fp8 MFMA (E4M3 codebook keys, rotated query as three "
                        "E4M3 terms); FP8-page scores and all PV products on the f16 MFMA with "
                        "hi + lo fp16 operands; softmax, scales and merge in fp32",
        "data": "synthetic",
        "config": {"workload": w.name, "n_req": n_req, "seq_len": lens[0], "layers": n_layers,
                   "q_heads": w.n_q_heads, "kv_heads": Hkv, "head_dim": d, "page_tokens": PAGE,
                   "recent_tokens": w.recent, "kv_formats": "fp8-e4m3 (R,A) + tq3 (S)",
                   "step": "per layer: decode with the append of 1 token/request fused "
                           "(paged_attn_decode_append); then migrate",
                   "stage_schedule": "fixed (deterministic)" if args.deterministic else "run-time"},
        "decode_attn_us_per_layer": round(dec_us, 3),
        "decode_scan_us": round(scan_mean, 3),
        "decode_merge_us": round(float(merge_us.mean()), 3),
        "decode_timing": "second pass of the same steps: HIP events around each "
                         "paged_attn_decode_append call; the library's events (same stream) "
                         "around the split-scan (with the fused append) and merge kernels of "
                         "each step's last call",
        "unfused_us_per_layer": None if unfused_ms is None else round(unfused_ms * 1e3 / n_layers, 3),
        "graph_us_per_layer": None if graph_ms is None else round(graph_ms * 1e3 / n_layers, 3),
        "graph_step": "last pass: the same whole steps, each captured into a HIP graph and replayed in order",
        "unfused_step": "third pass: the same steps with kv_append_fp8 and paged_attn_decode "
                        "as separate calls",
        "kv_bytes_per_layer": int(kv_bytes),
        "effective_kv_gb_per_s": round(kv_bytes / (ms_per_step * 1e-3 / n_layers) / 1e9, 1),
        "effective_kv_note": "algorithmic KV bytes per layer / the headline step time per layer "
                             "(decode, fused append, merge and the step's Retier share)",
        "roofline": {"bound": "hbm", "achieved": round(achieved / 1e9, 1), "peak": HBM_PEAK / 1e9,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK, 4), "traffic": traffic,
                     "kernel": "decode_kernel<256, true, true, true, false> (split scan with "
                               "the fused append, one launch per layer)"},
        "counters": {k: int(v) for k, v in counters.items()},
        "setup_s": round(setup_s, 1),
    }
    if ctl is not None:
        print("[bench] dense controls", file=sys.stderr, flush=True)
        res["dense_controls"] = ctl.time(torch, q_all, (pool, bt, tags, seq_after[n_steps - 1]), 5)
        del ctl
        torch.cuda.empty_cache()
    if not args.no_scores:
        res["score_collector"] = score_overhead(mk, torch, pool, bt, tags, seq_after[n_steps - 1],
                                                q_all, n_layers, w, det_after=args.deterministic)
    if not args.no_stream_probe:
        res["stream_probe"] = stream_probe(mk, torch, int(kv_bytes), achieved)
    if args.copy_probe:
        a_ = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        b_ = torch.empty_like(a_)
        torch.cuda.synchronize()
        b_.copy_(a_)
        torch.cuda.synchronize()
        res["copy_probe_bytes"] = 1 << 30
        del a_, b_
    print(f"[bench] decode passes done ({ms_per_step * 1e3 / n_layers:.2f} us/layer)",
          file=sys.stderr, flush=True)
    if not args.no_chunk:
        del pool
        torch.cuda.empty_cache()
        res["chunk"] = chunk_bench(mk, torch)
    if not args.no_cpu_baseline and args.cfg != 5:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
