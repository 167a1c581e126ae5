"""Builds the same Minima-KV state on the GPU (through the C ABI) and in the CPU
oracle from one seeded workload, and compares them."""
from __future__ import annotations

import numpy as np

import mkv_workloads as wl

PAGE = 16


def _torch():
    import torch
    return torch


class Twin:
    """GPU pool + oracle pool fed with identical calls."""

    def __init__(self, w, n_layers=1, lens=None, n_fp8=None, n_tq3=None, with_oracle=True,
                 recent=None, headroom=0):
        import oracle
        import paper_2608_23834_amd as mk
        torch = _torch()
        self.w = w
        self.lens = list(w.ctx if lens is None else lens)
        self.n_req = len(self.lens)
        self.L = n_layers
        self.W = w.recent if recent is None else recent
        self.max_pages = max(1, max((l + headroom + PAGE - 1) // PAGE for l in self.lens))
        tot_pages = sum((l + headroom + PAGE - 1) // PAGE for l in self.lens)
        self.n_fp8 = n_fp8 if n_fp8 is not None else tot_pages + 8
        self.n_tq3 = n_tq3 if n_tq3 is not None else tot_pages + 8
        self.sigma = wl.rot_signs(w)
        self.o8 = wl.free_order(w, self.n_fp8, "fp8")
        self.o3 = wl.free_order(w, self.n_tq3, "tq3")
        self.gpu = mk.Pool(n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, self.n_fp8, self.n_tq3,
                           self.W, self.sigma, self.o8, self.o3)
        self.bt = torch.full((self.n_req, self.max_pages), -1, dtype=torch.int32, device="cuda")
        self.tags = torch.full((self.n_req, self.max_pages), 0xFF, dtype=torch.uint8, device="cuda")
        self.orc = None
        if with_oracle:
            self.orc = oracle.Pool(n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, self.n_fp8,
                                   self.n_tq3, self.W, self.sigma, self.o8, self.o3)
            self.obt = np.full((self.n_req, self.max_pages), -1, np.int32)
            self.otags = np.full((self.n_req, self.max_pages), 0xFF, np.uint8)
        self.cur = [0] * self.n_req

    # -- calls -------------------------------------------------------------
    def append(self, new_counts, layer_kv=None, layer=-1):
        """Append new_counts[r] tokens to request r (K/V drawn from the workload)."""
        import paper_2608_23834_amd as mk
        torch = _torch()
        sb = np.array(self.cur, np.int32)
        cu = np.r_[0, np.cumsum(new_counts)].astype(np.int32)
        if layer_kv is None:
            ks, vs = [], []
            for l in range(self.L) if layer < 0 else [layer]:
                kk, vv = [], []
                for r, n in enumerate(new_counts):
                    k, v = wl.kv_layer(self.w, l, n, token_offset=r * 1_000_000 + self.cur[r])
                    kk.append(k)
                    vv.append(v)
                ks.append(np.concatenate(kk) if kk else np.zeros((0, self.w.n_kv_heads, self.w.head_dim), np.uint16))
                vs.append(np.concatenate(vv) if vv else np.zeros((0, self.w.n_kv_heads, self.w.head_dim), np.uint16))
            K = np.stack(ks) if layer < 0 else ks[0]
            V = np.stack(vs) if layer < 0 else vs[0]
        else:
            K, V = layer_kv
        mk.kv_append_fp8(self.gpu, layer, self.bt, self.tags,
                         torch.from_numpy(sb).cuda(), torch.from_numpy(cu).cuda(),
                         torch.from_numpy(K.view(np.int16)).cuda(),
                         torch.from_numpy(V.view(np.int16)).cuda())
        if self.orc is not None:
            Ko = K if layer < 0 else K[None]
            Vo = V if layer < 0 else V[None]
            rc = self.orc.append(layer, self.obt, self.otags, sb, cu, Ko, Vo)
            assert rc == 0, rc
        for r, n in enumerate(new_counts):
            self.cur[r] += n
        return K, V

    def fill(self, chunk=None):
        """Append every request's full context (in chunks of `chunk` tokens)."""
        target = list(self.lens)
        while any(c < t for c, t in zip(self.cur, target)):
            step = [min(t - c, chunk or (t - c)) for c, t in zip(self.cur, target)]
            self.append(step)

    def fill_to(self, targets, chunk=None):
        """Append until request r holds targets[r] tokens."""
        while any(c < t for c, t in zip(self.cur, targets)):
            step = [max(0, min(t - c, chunk or (t - c))) for c, t in zip(self.cur, targets)]
            self.append(step)

    def anchor(self):
        return wl.anchor_mask(self.w, self.max_pages, self.lens)

    def migrate(self, anchor=None):
        import paper_2608_23834_amd as mk
        torch = _torch()
        am = self.anchor() if anchor is None else anchor
        sl = np.array(self.cur, np.int32)
        mk.kv_migrate_to_tq3(self.gpu, self.bt, self.tags, torch.from_numpy(am).cuda(),
                             torch.from_numpy(sl).cuda())
        if self.orc is not None:
            n = self.orc.migrate(self.obt, self.otags, am, sl)
            assert n >= 0

    def promote(self, mask):
        """Alg. 1 Promote of the Stale pages whose mask entry is set."""
        import paper_2608_23834_amd as mk
        torch = _torch()
        sl = np.array(self.cur, np.int32)
        mk.kv_promote_to_fp8(self.gpu, self.bt, self.tags, torch.from_numpy(mask).cuda(),
                             torch.from_numpy(sl).cuda())
        if self.orc is not None:
            n = self.orc.promote(self.obt, self.otags, mask, sl)
            assert n >= 0
            return n

    # -- reference counts and shared prefixes (Alg. 1 SealPrefix / Finish) --
    def acquire(self, ids, tags):
        import paper_2608_23834_amd as mk
        torch = _torch()
        ids = np.ascontiguousarray(ids, np.int32)
        tags = np.ascontiguousarray(tags, np.uint8)
        mk.kv_pages_acquire(self.gpu, torch.from_numpy(ids).cuda(), torch.from_numpy(tags).cuda())
        if self.orc is not None:
            assert self.orc.acquire(ids, tags) == 0

    def release(self, ids, tags):
        import paper_2608_23834_amd as mk
        torch = _torch()
        ids = np.ascontiguousarray(ids, np.int32)
        tags = np.ascontiguousarray(tags, np.uint8)
        mk.kv_pages_release(self.gpu, torch.from_numpy(ids).cuda(), torch.from_numpy(tags).cuda())
        if self.orc is not None:
            return self.orc.release(ids, tags)

    def finish(self, reqs):
        import paper_2608_23834_amd as mk
        torch = _torch()
        rq = np.ascontiguousarray(reqs, np.int32)
        mk.kv_request_finish(self.gpu, torch.from_numpy(rq).cuda(), self.bt, self.tags)
        if self.orc is not None:
            n = self.orc.finish(rq, self.obt, self.otags)
            assert n >= 0
        for r in reqs:
            self.cur[r] = 0

    def set_rows(self, r, pages, ids, tags):
        """Write block-table entries of request r (both sides), e.g. a cached prefix."""
        torch = _torch()
        self.bt[r, pages] = torch.tensor(np.asarray(ids, np.int32), device="cuda")
        self.tags[r, pages] = torch.tensor(np.asarray(tags, np.uint8), device="cuda")
        if self.orc is not None:
            self.obt[r, pages] = ids
            self.otags[r, pages] = tags

    def check_refcounts(self):
        import paper_2608_23834_amd as mk
        r8, r3 = mk.kv_pool_read_refcounts(self.gpu)
        assert np.array_equal(r8, self.orc.rc8[: self.n_fp8]), "fp8 reference counts"
        assert np.array_equal(r3, self.orc.rc3[: self.n_tq3]), "tq3 reference counts"
        return r8, r3

    def _ws(self, ws_fill):
        import paper_2608_23834_amd as mk
        ws = mk.workspace(self.gpu, self.n_req, self.max_pages)
        if ws_fill is not None:  # e.g. NaN bits: the calls must not depend on the contents
            ws.view(_torch().float32)[: ws.numel() // 4].fill_(ws_fill)
        return ws

    def decode(self, layer=0, q=None, seq_lens=None, ws_fill=None):
        import paper_2608_23834_amd as mk
        torch = _torch()
        w = self.w
        q = wl.q_decode(w, layer) if q is None else q
        if q.shape[0] != self.n_req:
            q = np.resize(q, (self.n_req,) + q.shape[1:])
        sl = np.array(self.cur if seq_lens is None else seq_lens, np.int32)
        out = torch.full((self.n_req, w.n_q_heads, w.head_dim), float("nan"), device="cuda")
        lse = torch.full((self.n_req, w.n_q_heads), float("nan"), device="cuda")
        ws = self._ws(ws_fill)
        mk.paged_attn_decode(self.gpu, layer, torch.from_numpy(q.view(np.int16)).cuda(), self.bt,
                             self.tags, torch.from_numpy(sl).cuda(), out, lse, ws)
        torch.cuda.synchronize()
        res = dict(out=out.cpu().numpy(), lse=lse.cpu().numpy(), q=q, seq_lens=sl, ws=ws)
        if self.orc is not None:
            o, l = self.orc.decode(layer, q, self.obt, self.otags, sl)
            res["ref_out"], res["ref_lse"] = o, l
        return res

    def decode_append(self, layer=0, q=None, ws_fill=None):
        """One fused decode step on `layer`: append one token per request at
        its current length, then decode over length + 1.  The oracle runs the
        append and the decode as two calls.  Lengths advance with advance()."""
        import paper_2608_23834_amd as mk
        torch = _torch()
        w = self.w
        kk, vv = [], []
        for r in range(self.n_req):
            k, v = wl.kv_layer(w, layer, 1, token_offset=r * 1_000_000 + self.cur[r])
            kk.append(k)
            vv.append(v)
        K, V = np.concatenate(kk), np.concatenate(vv)  # [n_req][H][d]
        q = wl.q_decode(w, layer) if q is None else q
        if q.shape[0] != self.n_req:
            q = np.resize(q, (self.n_req,) + q.shape[1:])
        sb = np.array(self.cur, np.int32)
        out = torch.full((self.n_req, w.n_q_heads, w.head_dim), float("nan"), device="cuda")
        lse = torch.full((self.n_req, w.n_q_heads), float("nan"), device="cuda")
        ws = self._ws(ws_fill)
        mk.paged_attn_decode_append(
            self.gpu, layer, torch.from_numpy(q.view(np.int16)).cuda(),
            torch.from_numpy(K.view(np.int16)).cuda(), torch.from_numpy(V.view(np.int16)).cuda(),
            self.bt, self.tags, torch.from_numpy(sb).cuda(), out, lse, ws)
        torch.cuda.synchronize()
        res = dict(out=out.cpu().numpy(), lse=lse.cpu().numpy(), q=q, seq_lens=sb + 1)
        if self.orc is not None:
            cu = np.arange(self.n_req + 1, dtype=np.int32)
            rc = self.orc.append(layer, self.obt, self.otags, sb, cu, K[None], V[None])
            assert rc == 0, rc
            o, l = self.orc.decode(layer, q, self.obt, self.otags, sb + 1)
            res["ref_out"], res["ref_lse"] = o, l
        return res

    def advance(self, n=1):
        self.cur = [c + n for c in self.cur]

    def chunk(self, n_q, layer=0, sample_stride=1):
        """Chunk attention for the last n_q[r] tokens of each request (already
        appended).  The oracle computes every sample_stride-th query of each
        request and its last one; the other rows of ref_out stay NaN."""
        import paper_2608_23834_amd as mk
        torch = _torch()
        w = self.w
        n_q = [int(x) for x in n_q]
        mx = max(n_q)
        qa = wl.q_chunk(w, layer, mx)
        q = np.concatenate([qa[r * mx: r * mx + n_q[r]] for r in range(self.n_req)])
        cu = np.r_[0, np.cumsum(n_q)].astype(np.int32)
        sl = np.array(self.cur, np.int32)
        out = torch.full((q.shape[0], w.n_q_heads, w.head_dim), float("nan"), device="cuda")
        ws = mk.workspace(self.gpu, self.n_req, self.max_pages, q.shape[0])
        mk.paged_attn_chunk(self.gpu, layer, torch.from_numpy(q.view(np.int16)).cuda(),
                            torch.from_numpy(cu).cuda(), self.bt, self.tags,
                            torch.from_numpy(sl).cuda(), out, ws)
        torch.cuda.synchronize()
        res = dict(out=out.cpu().numpy(), q=q, cu=cu, seq_lens=sl)
        if self.orc is not None:
            if np.ndim(sample_stride) == 0:
                res["ref_out"] = self.orc.chunk(layer, q, cu, self.obt, self.otags, sl, sample_stride)
            else:  # per-request strides, one request per oracle call (progress lines)
                ref = np.full(res["out"].shape, np.nan)
                for r in range(self.n_req):
                    st = np.full(self.n_req, 1 << 30, np.int32)
                    st[r] = sample_stride[r]
                    o = self.orc.chunk(layer, q, cu, self.obt, self.otags, sl, st)
                    ref[cu[r]:cu[r + 1]] = o[cu[r]:cu[r + 1]]
                    print(f"  oracle chunk rows of request {r} done (stride {sample_stride[r]})",
                          flush=True)
                res["ref_out"] = ref
        return res

    # -- comparisons -------------------------------------------------------
    def check_tables(self):
        torch = _torch()
        import paper_2608_23834_amd as mk
        assert np.array_equal(self.bt.cpu().numpy(), self.obt), "block table"
        assert np.array_equal(self.tags.cpu().numpy(), self.otags), "tags"
        f8, f3 = mk.kv_pool_read_free_lists(self.gpu)
        assert np.array_equal(f8, self.orc.fp8_stack[: self.orc.fp8_top[0]]), "fp8 free list"
        assert np.array_equal(f3, self.orc.tq3_stack[: self.orc.tq3_top[0]]), "tq3 free list"
        assert mk.kv_pool_check_errors(self.gpu) == 0

    def check_pages(self):
        """Bit-exact FP8 codes/scales and TQ3 regions of every live page."""
        tags = self.otags
        bt = self.obt
        live8 = sorted(set(bt[(tags == 0) | (tags == 1)].tolist()))
        live3 = sorted(set(bt[tags == 2].tolist()))
        g8 = self.gpu.fp8_view()
        gs = self.gpu.fp8_scales_view()
        g3 = self.gpu.tq3_view()
        if live8:
            idx = _torch().tensor(live8, device="cuda", dtype=_torch().long)
            a = g8[:, idx].cpu().numpy()
            b = self.orc.fp8[:, live8]
            bad = np.argwhere(a != b)
            assert bad.size == 0, f"fp8 codes differ at {bad[:5]} ({a[tuple(bad[0])]} vs {b[tuple(bad[0])]})"
            sa = gs[:, idx].cpu().numpy()
            sb = self.orc.fp8_scale[:, live8]
            assert np.array_equal(sa.view(np.uint32), sb.view(np.uint32)), "fp8 scales"
        if live3:
            idx = _torch().tensor(live3, device="cuda", dtype=_torch().long)
            a = g3[:, idx].cpu().numpy()
            b = self.orc.tq3[:, live3]
            bad = np.argwhere(a != b)
            assert bad.size == 0, f"tq3 bytes differ at {bad[:5]}"
        return len(live8), len(live3)


def max_abs(a, b):
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))
