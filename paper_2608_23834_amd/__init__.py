"""Python binding of libminimakv (MI355X / gfx950 Minima-KV hot path).

Argument marshalling only: every step of the path runs in the HIP kernels of
``libminimakv.so``.  torch supplies device memory and streams.  The functions
keep the C ABI's names (include/minima_kv.h).  There is no CPU fallback: if the
built library is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libminimakv.so")

MKV_ALL_LAYERS = -1
PAGE = 16
TAG_R, TAG_A, TAG_S, TAG_NONE = 0, 1, 2, 0xFF
STATUS = {0: "MKV_OK", 1: "MKV_EINVAL", 2: "MKV_EUNSUP", 3: "MKV_ENOMEM", 4: "MKV_ERANGE",
          5: "MKV_ESTATE", 6: "MKV_EHIP"}
DEVERR = {"FP8_EXHAUSTED": 0x1, "TQ3_EXHAUSTED": 0x2, "NOT_RECENT": 0x4, "RANGE": 0x8,
          "BAD_TAG": 0x10, "REFCOUNT": 0x20}
EXPORTS = ["kv_pool_bytes", "kv_pool_create", "kv_pool_destroy", "kv_append_fp8",
           "kv_migrate_to_tq3", "kv_promote_to_fp8", "kv_pages_acquire", "kv_pages_release",
           "kv_request_finish", "kv_pool_read_refcounts", "paged_attn_workspace_bytes", "paged_attn_workspace_init",
           "paged_attn_decode", "paged_attn_decode_append", "paged_attn_chunk",
           "kv_partition_pages", "kv_pool_free_counts",
           "kv_pool_read_free_lists", "kv_pool_counters", "kv_pool_check_errors",
           "paged_attn_set_timing", "paged_attn_set_deterministic", "paged_attn_last_times",
           "mkv_stream_read",
           "paged_attn_decode_noalloc", "mkv_fp64_probe", "mkv_control_bf16_write",
           "mkv_control_bf16_workspace_bytes", "mkv_control_bf16_decode",
           "paged_attn_decode_cohort_key", "paged_attn_decode_scores", "kv_page_scores_update",
           "mkv_status_string"]

_lib = None


class MkvError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} failed: {STATUS.get(code, code)}")
        self.code = code


class PoolDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("n_fp8_pages", ctypes.c_int32),
                ("n_tq3_pages", ctypes.c_int32), ("recent_tokens", ctypes.c_int32),
                ("rot_signs", ctypes.c_void_p), ("fp8_order", ctypes.c_void_p),
                ("tq3_order", ctypes.c_void_p),
                ("fp8_data", ctypes.c_void_p), ("fp8_data_bytes", ctypes.c_size_t),
                ("fp8_scales", ctypes.c_void_p), ("fp8_scales_bytes", ctypes.c_size_t),
                ("tq3_data", ctypes.c_void_p), ("tq3_data_bytes", ctypes.c_size_t),
                ("ctrl", ctypes.c_void_p), ("ctrl_bytes", ctypes.c_size_t)]


class Counters(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in (
        "decode_routes", "chunk_routes", "fallbacks", "dense_shadow_bytes", "fp8_pages_live",
        "tq3_pages_live", "fp8_bytes_live", "tq3_bytes_live")]


def lib() -> ctypes.CDLL:
    """Load the built library (build it with ``python -m paper_2608_23834_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libminimakv.so is not built ({LIB_PATH}); run "
                               "`python -m paper_2608_23834_amd.build` first")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        for name in EXPORTS:
            getattr(L, name).restype = ctypes.c_int
        L.mkv_status_string.restype = ctypes.c_char_p
        L.kv_pool_bytes.argtypes = [vp, vp, vp, vp, vp]
        L.kv_pool_create.argtypes = [vp, vp]
        L.kv_pool_destroy.argtypes = [vp]
        L.kv_append_fp8.argtypes = [vp, i32, i32, vp, vp, i32, vp, vp, i32, vp, vp, vp]
        L.kv_migrate_to_tq3.argtypes = [vp, i32, vp, vp, i32, vp, vp, vp]
        L.kv_promote_to_fp8.argtypes = [vp, i32, vp, vp, i32, vp, vp, vp]
        L.kv_pages_acquire.argtypes = [vp, i32, vp, vp, vp]
        L.kv_pages_release.argtypes = [vp, i32, vp, vp, vp]
        L.kv_request_finish.argtypes = [vp, i32, vp, i32, vp, vp, i32, vp]
        L.kv_pool_read_refcounts.argtypes = [vp, vp, vp]
        L.paged_attn_workspace_bytes.argtypes = [vp, i32, i32, i32, vp]
        L.paged_attn_workspace_init.argtypes = [vp, sz, vp]
        L.paged_attn_decode.argtypes = [vp, i32, i32, vp, vp, vp, i32, vp, vp, vp, vp, sz, vp]
        L.paged_attn_decode_noalloc.argtypes = [vp, i32, i32, vp, vp, vp, i32, vp, vp, vp, vp]
        L.paged_attn_decode_append.argtypes = [vp, i32, i32, vp, vp, vp, vp, vp, i32, vp, vp, vp,
                                               vp, sz, vp]
        L.paged_attn_chunk.argtypes = [vp, i32, i32, vp, vp, i32, vp, vp, i32, vp, vp, vp, sz, vp]
        L.kv_partition_pages.argtypes = [i32, vp, vp, i32, vp, vp, vp, vp, vp]
        L.kv_pool_free_counts.argtypes = [vp, vp, vp]
        L.kv_pool_read_free_lists.argtypes = [vp, vp, vp, vp, vp]
        L.kv_pool_counters.argtypes = [vp, vp]
        L.kv_pool_check_errors.argtypes = [vp, vp, i32]
        L.paged_attn_set_timing.argtypes = [vp, i32]
        L.paged_attn_set_deterministic.argtypes = [vp, i32]
        L.paged_attn_last_times.argtypes = [vp, vp, vp]
        L.mkv_stream_read.argtypes = [vp, sz, vp, vp]
        L.mkv_fp64_probe.argtypes = [vp, vp, ctypes.c_int64, vp, vp, vp, vp]
        L.paged_attn_decode_cohort_key.argtypes = [vp, i32, i32, i32, i32, vp]
        L.paged_attn_decode_scores.argtypes = [vp, i32, i32, vp, vp, vp, i32, vp, vp, vp, vp, sz,
                                               vp, vp]
        L.kv_page_scores_update.argtypes = [vp, i32, i32, vp, vp, vp, vp, ctypes.c_float, vp, vp,
                                            vp, vp]
        L.mkv_control_bf16_write.argtypes = [vp, i32, i32, i32, i32, i32, i32, vp, i32, vp, vp, i32,
                                             vp, vp, vp]
        L.mkv_control_bf16_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, vp]
        L.mkv_control_bf16_decode.argtypes = [vp, i32, i32, i32, i32, i32, i32, i32, vp, vp, i32,
                                              vp, vp, vp, vp, sz, vp]
        L.mkv_status_string.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


def _check(fn, code):
    if code != 0:
        raise MkvError(fn, code)


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def pool_bytes(n_layers, n_q_heads, n_kv_heads, head_dim, n_fp8_pages, n_tq3_pages, recent_tokens):
    d = PoolDesc(n_layers, n_q_heads, n_kv_heads, head_dim, PAGE, n_fp8_pages, n_tq3_pages,
                 recent_tokens)
    out = (ctypes.c_size_t * 4)()
    _check("kv_pool_bytes", lib().kv_pool_bytes(ctypes.byref(d), ctypes.byref(out, 0),
                                                ctypes.byref(out, 8), ctypes.byref(out, 16),
                                                ctypes.byref(out, 24)))
    return tuple(out)


class Pool:
    """A pool over torch-allocated device buffers (the caller owns memory)."""

    def __init__(self, n_layers, n_q_heads, n_kv_heads, head_dim, n_fp8_pages, n_tq3_pages,
                 recent_tokens, rot_signs, fp8_order=None, tq3_order=None, device="cuda"):
        import torch
        self.n_layers, self.n_q_heads, self.n_kv_heads, self.d = n_layers, n_q_heads, n_kv_heads, head_dim
        self.n_fp8, self.n_tq3, self.recent = n_fp8_pages, n_tq3_pages, recent_tokens
        b8, bs, b3, bc = pool_bytes(n_layers, n_q_heads, n_kv_heads, head_dim, n_fp8_pages,
                                    n_tq3_pages, recent_tokens)
        self.fp8 = torch.zeros(b8, dtype=torch.uint8, device=device)
        self.fp8_scales = torch.zeros(bs // 4, dtype=torch.float32, device=device)
        self.tq3 = torch.zeros(max(b3, 16), dtype=torch.uint8, device=device)
        self.ctrl = torch.zeros(bc // 4, dtype=torch.int32, device=device)
        sig = np.ascontiguousarray(rot_signs, dtype=np.int8)
        o8 = None if fp8_order is None else np.ascontiguousarray(fp8_order, dtype=np.int32)
        o3 = None if tq3_order is None else np.ascontiguousarray(tq3_order, dtype=np.int32)
        desc = PoolDesc(n_layers, n_q_heads, n_kv_heads, head_dim, PAGE, n_fp8_pages, n_tq3_pages,
                        recent_tokens, sig.ctypes.data,
                        None if o8 is None else o8.ctypes.data,
                        None if o3 is None else o3.ctypes.data,
                        self.fp8.data_ptr(), b8, self.fp8_scales.data_ptr(), bs,
                        self.tq3.data_ptr(), b3, self.ctrl.data_ptr(), bc)
        h = ctypes.c_void_p()
        torch.cuda.synchronize()
        _check("kv_pool_create", lib().kv_pool_create(ctypes.byref(desc), ctypes.byref(h)))
        self.handle = h

    # views in the documented layouts
    def fp8_view(self):
        return self.fp8.view(self.n_layers, self.n_fp8, self.n_kv_heads, 2 * PAGE * self.d)

    def fp8_scales_view(self):
        return self.fp8_scales.view(self.n_layers, self.n_fp8, self.n_kv_heads, 2)

    def tq3_view(self):
        return self.tq3[: self.n_layers * self.n_tq3 * self.n_kv_heads * (16 * self.d + 32)].view(
            self.n_layers, self.n_tq3, self.n_kv_heads, 16 * self.d + 32)

    def close(self):
        if getattr(self, "handle", None):
            lib().kv_pool_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def kv_append_fp8(pool: Pool, layer, block_table, tags, seq_lens_before, cu_new_tokens, k, v,
                  stream=None):
    n_req, max_pages = block_table.shape
    n_new = int(k.shape[-3]) if k is not None else 0
    _check("kv_append_fp8", lib().kv_append_fp8(
        pool.handle, layer, n_req, _ptr(block_table), _ptr(tags), max_pages, _ptr(seq_lens_before),
        _ptr(cu_new_tokens), n_new, _ptr(k), _ptr(v), _stream(stream)))


def kv_migrate_to_tq3(pool: Pool, block_table, tags, anchor_mask, seq_lens, stream=None):
    n_req, max_pages = block_table.shape
    _check("kv_migrate_to_tq3", lib().kv_migrate_to_tq3(
        pool.handle, n_req, _ptr(block_table), _ptr(tags), max_pages, _ptr(anchor_mask),
        _ptr(seq_lens), _stream(stream)))


def kv_promote_to_fp8(pool: Pool, block_table, tags, promote_mask, seq_lens, stream=None):
    n_req, max_pages = block_table.shape
    _check("kv_promote_to_fp8", lib().kv_promote_to_fp8(
        pool.handle, n_req, _ptr(block_table), _ptr(tags), max_pages, _ptr(promote_mask),
        _ptr(seq_lens), _stream(stream)))


def kv_pages_acquire(pool: Pool, ids, tags, stream=None):
    """SealPrefix / prefix attach: one more reference per listed page (device tensors)."""
    _check("kv_pages_acquire", lib().kv_pages_acquire(pool.handle, int(ids.numel()), _ptr(ids),
                                                      _ptr(tags), _stream(stream)))


def kv_pages_release(pool: Pool, ids, tags, stream=None):
    """Prefix eviction: one reference fewer per listed page (device tensors)."""
    _check("kv_pages_release", lib().kv_pages_release(pool.handle, int(ids.numel()), _ptr(ids),
                                                      _ptr(tags), _stream(stream)))


def kv_request_finish(pool: Pool, reqs, block_table, tags, stream=None):
    """Finish(q) of the requests in `reqs` (device int32, ascending)."""
    n_req, max_pages = block_table.shape
    _check("kv_request_finish", lib().kv_request_finish(
        pool.handle, int(reqs.numel()), _ptr(reqs), n_req, _ptr(block_table), _ptr(tags),
        max_pages, _stream(stream)))


def kv_pool_read_refcounts(pool: Pool):
    r8 = np.zeros(pool.n_fp8, np.int32)
    r3 = np.zeros(max(pool.n_tq3, 1), np.int32)
    _check("kv_pool_read_refcounts", lib().kv_pool_read_refcounts(pool.handle, r8.ctypes.data,
                                                                  r3.ctypes.data))
    return r8, r3[: pool.n_tq3]


def paged_attn_workspace_bytes(pool: Pool, n_req, max_pages, n_q_total=0):
    out = ctypes.c_size_t()
    _check("paged_attn_workspace_bytes", lib().paged_attn_workspace_bytes(
        pool.handle, n_req, max_pages, n_q_total, ctypes.byref(out)))
    return out.value


def workspace(pool: Pool, n_req, max_pages, n_q_total=0, device="cuda"):
    import torch
    return torch.zeros(paged_attn_workspace_bytes(pool, n_req, max_pages, n_q_total),
                       dtype=torch.uint8, device=device)


def paged_attn_workspace_init(ws, stream=None):
    _check("paged_attn_workspace_init", lib().paged_attn_workspace_init(
        _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def paged_attn_decode(pool: Pool, layer, q, block_table, tags, seq_lens, out, lse, ws,
                      stream=None):
    n_req, max_pages = block_table.shape
    _check("paged_attn_decode", lib().paged_attn_decode(
        pool.handle, layer, n_req, _ptr(q), _ptr(block_table), _ptr(tags), max_pages,
        _ptr(seq_lens), _ptr(out), _ptr(lse), _ptr(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def paged_attn_decode_scores(pool: Pool, layer, q, block_table, tags, seq_lens, out, lse, ws,
                             page_mass, stream=None):
    """paged_attn_decode that also writes each page's local mass and reference
    exponent (page_mass: device float32 [n_req][max_pages][n_q_heads][2])."""
    n_req, max_pages = block_table.shape
    _check("paged_attn_decode_scores", lib().paged_attn_decode_scores(
        pool.handle, layer, n_req, _ptr(q), _ptr(block_table), _ptr(tags), max_pages,
        _ptr(seq_lens), _ptr(out), _ptr(lse), _ptr(ws), ws.numel() * ws.element_size(),
        _ptr(page_mass), _stream(stream)))


def kv_page_scores_update(pool: Pool, seq_lens, lse, page_mass, head_mask, beta, scores,
                          r_out=None, qn_out=None, stream=None):
    n_req, max_pages = scores.shape
    _check("kv_page_scores_update", lib().kv_page_scores_update(
        pool.handle, n_req, max_pages, _ptr(seq_lens), _ptr(lse), _ptr(page_mass),
        _ptr(head_mask), float(beta), _ptr(scores), _ptr(r_out), _ptr(qn_out), _stream(stream)))


DECODE_SCRATCH_BYTES = 32 * 1024 * 1024


def paged_attn_decode_noalloc(pool: Pool, layer, q, block_table, tags, seq_lens, out, lse,
                              stream=None):
    """paged_attn_decode with the split partials in the library's fixed device
    scratch (no workspace argument; the call allocates nothing)."""
    n_req, max_pages = block_table.shape
    _check("paged_attn_decode_noalloc", lib().paged_attn_decode_noalloc(
        pool.handle, layer, n_req, _ptr(q), _ptr(block_table), _ptr(tags), max_pages,
        _ptr(seq_lens), _ptr(out), _ptr(lse), _stream(stream)))


def paged_attn_decode_append(pool: Pool, layer, q, k_new, v_new, block_table, tags,
                             seq_lens_before, out, lse, ws, stream=None):
    n_req, max_pages = block_table.shape
    _check("paged_attn_decode_append", lib().paged_attn_decode_append(
        pool.handle, layer, n_req, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(block_table),
        _ptr(tags), max_pages, _ptr(seq_lens_before), _ptr(out), _ptr(lse), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def paged_attn_chunk(pool: Pool, layer, q, cu_q, block_table, tags, seq_lens, out, ws,
                     stream=None):
    n_req, max_pages = block_table.shape
    _check("paged_attn_chunk", lib().paged_attn_chunk(
        pool.handle, layer, n_req, _ptr(q), _ptr(cu_q), int(q.shape[0]), _ptr(block_table),
        _ptr(tags), max_pages, _ptr(seq_lens), _ptr(out), _ptr(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def kv_partition_pages(block_table, tags, seq_lens, list8, list3, counts, stream=None):
    n_req, max_pages = block_table.shape
    _check("kv_partition_pages", lib().kv_partition_pages(
        n_req, _ptr(block_table), _ptr(tags), max_pages, _ptr(seq_lens), _ptr(list8), _ptr(list3),
        _ptr(counts), _stream(stream)))


def kv_pool_free_counts(pool: Pool):
    a, b = ctypes.c_int32(), ctypes.c_int32()
    _check("kv_pool_free_counts", lib().kv_pool_free_counts(pool.handle, ctypes.byref(a),
                                                             ctypes.byref(b)))
    return a.value, b.value


def kv_pool_read_free_lists(pool: Pool):
    f8 = np.zeros(pool.n_fp8, np.int32)
    f3 = np.zeros(max(pool.n_tq3, 1), np.int32)
    n8, n3 = ctypes.c_int32(), ctypes.c_int32()
    _check("kv_pool_read_free_lists", lib().kv_pool_read_free_lists(
        pool.handle, f8.ctypes.data, ctypes.byref(n8), f3.ctypes.data, ctypes.byref(n3)))
    return f8[: n8.value].copy(), f3[: n3.value].copy()


def kv_pool_counters(pool: Pool) -> dict:
    c = Counters()
    _check("kv_pool_counters", lib().kv_pool_counters(pool.handle, ctypes.byref(c)))
    return {n: getattr(c, n) for n, _ in Counters._fields_}


def paged_attn_set_deterministic(pool: Pool, enable: bool) -> None:
    _check("paged_attn_set_deterministic",
           lib().paged_attn_set_deterministic(pool.handle, int(bool(enable))))


def paged_attn_set_timing(pool: Pool, enable: bool) -> None:
    _check("paged_attn_set_timing", lib().paged_attn_set_timing(pool.handle, int(bool(enable))))


def paged_attn_last_times(pool: Pool) -> tuple:
    """(scan_us, merge_us) of the last timed paged_attn_decode call (waits for it)."""
    a, b = ctypes.c_float(), ctypes.c_float()
    _check("paged_attn_last_times", lib().paged_attn_last_times(pool.handle, ctypes.byref(a),
                                                                ctypes.byref(b)))
    return a.value, b.value


STREAM_PROBE_WORKGROUPS = 2048


def mkv_stream_read(buf, sink, stream=None):
    """Streaming-read probe (measurement only): reads the device tensor `buf`
    once; `sink` is a device int32 tensor of STREAM_PROBE_WORKGROUPS words."""
    assert sink.numel() >= STREAM_PROBE_WORKGROUPS
    _check("mkv_stream_read", lib().mkv_stream_read(
        _ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), _stream(stream)))


def mkv_fp64_probe(a, b, quot, root, half, stream=None):
    """Conformance probe (tests only): quot = a / b, root = sqrt(a), half =
    binary16(a), by the library's own compiled fp64 code (device tensors)."""
    n = a.numel()
    assert b.numel() == n and quot.numel() == n and root.numel() == n and half.numel() == n
    _check("mkv_fp64_probe", lib().mkv_fp64_probe(_ptr(a), _ptr(b), n, _ptr(quot), _ptr(root),
                                                  _ptr(half), _stream(stream)))


def paged_attn_decode_cohort_key(pool: Pool, n_req, max_pages, fused_append=True, scoring=False):
    key = ctypes.c_uint64()
    _check("paged_attn_decode_cohort_key", lib().paged_attn_decode_cohort_key(
        pool.handle, n_req, max_pages, int(bool(fused_append)), int(bool(scoring)),
        ctypes.byref(key)))
    return key.value


class DecodeStepGraph:
    """A decode step (per layer paged_attn_decode_append, then
    kv_migrate_to_tq3) captured once into a HIP graph and replayed for later
    steps of the same cohort (Sec. 4.1 graph path gated on a homogeneous
    cohort).  The step reads its inputs from fixed device buffers -- q
    [n_layers][n_req][Hq][d], k_new / v_new [n_layers][n_req][Hkv][d],
    seq_lens_before [n_req], seq_lens_after [n_req], anchor mask -- which the
    caller refills before each run.  run(key) replays only when `key` (the
    cohort key of the step about to run) equals the key captured; otherwise it
    fails closed to launching the same calls directly.  Host orchestration
    only: the work is the library's kernels either way."""

    def __init__(self, pool: Pool, block_table, tags, bufs: dict, out, lse, ws):
        self.pool, self.bt, self.tags, self.b, self.out, self.lse, self.ws = (
            pool, block_table, tags, bufs, out, lse, ws)
        n_req, max_pages = block_table.shape
        self.key = paged_attn_decode_cohort_key(pool, n_req, max_pages, True, False)
        self.graph = None
        self.replays = 0
        self.direct = 0

    def _step(self):
        b = self.b
        for layer in range(self.pool.n_layers):
            paged_attn_decode_append(self.pool, layer, b["q"][layer], b["k_new"][layer],
                                     b["v_new"][layer], self.bt, self.tags, b["seq_before"],
                                     self.out[layer], self.lse[layer], self.ws)
        kv_migrate_to_tq3(self.pool, self.bt, self.tags, b["anchor"], b["seq_after"])

    def capture(self):
        """Capture one step (every kernel instance it uses must have run once
        on this device before, so that no launch attribute is set inside)."""
        import torch
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.graph(g, stream=s):
            self._step()
        torch.cuda.current_stream().wait_stream(s)
        self.graph = g

    def run(self, key):
        if self.graph is not None and key == self.key:
            self.graph.replay()
            self.replays += 1
        else:
            self._step()
            self.direct += 1


class ControlBf16:
    """Dense bf16 control pages (measurement only): the same KV as the mixed
    pool held as bf16, for timing the mixed path against an uncompressed
    cache.  Page ids come from the caller's block table."""

    def __init__(self, n_layers, n_q_heads, n_kv_heads, head_dim, n_pages, device="cuda"):
        import torch
        self.n_layers, self.n_q_heads, self.n_kv_heads, self.d = n_layers, n_q_heads, n_kv_heads, head_dim
        self.n_pages = n_pages
        self.pages = torch.zeros((n_layers, n_pages, n_kv_heads, 2 * PAGE * head_dim),
                                 dtype=torch.int16, device=device)

    def write(self, layer, block_table, seq_lens_before, cu_new_tokens, k, v, stream=None):
        n_req, max_pages = block_table.shape
        _check("mkv_control_bf16_write", lib().mkv_control_bf16_write(
            _ptr(self.pages), self.n_pages, self.n_layers, self.n_kv_heads, self.d, layer, n_req,
            _ptr(block_table), max_pages, _ptr(seq_lens_before), _ptr(cu_new_tokens),
            int(k.shape[0]), _ptr(k), _ptr(v), _stream(stream)))

    def workspace(self, n_req, max_pages, device="cuda"):
        import torch
        b = ctypes.c_size_t()
        _check("mkv_control_bf16_workspace_bytes", lib().mkv_control_bf16_workspace_bytes(
            n_req, max_pages, self.n_kv_heads, self.n_q_heads, self.d, ctypes.byref(b)))
        return torch.empty(b.value, dtype=torch.uint8, device=device)

    def decode(self, layer, q, block_table, seq_lens, out, lse, ws, stream=None):
        n_req, max_pages = block_table.shape
        _check("mkv_control_bf16_decode", lib().mkv_control_bf16_decode(
            _ptr(self.pages), self.n_pages, self.n_layers, self.n_kv_heads, self.n_q_heads, self.d,
            layer, n_req, _ptr(q), _ptr(block_table), max_pages, _ptr(seq_lens), _ptr(out),
            _ptr(lse), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def kv_pool_check_errors(pool: Pool, clear=False) -> int:
    e = ctypes.c_uint32()
    _check("kv_pool_check_errors", lib().kv_pool_check_errors(pool.handle, ctypes.byref(e),
                                                               int(bool(clear))))
    return e.value
