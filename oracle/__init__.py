"""Minima-KV CPU oracle (test infrastructure only).

Plain, slow CPU implementation of what the MI355X hot path computes, written
from the paper (arXiv 2608.23834) — the C core lives in ``mkv_oracle.c`` and
this module marshals numpy arrays into it.  Only the tests, the smoke check and
the benchmark's CPU-baseline leg may import it; the product package never does
and shares no code with it.

Paper passages followed (by section / equation / algorithm):
  * Sec. 2.1, Eq. (kv-per-token): bytes per live token (``kv_bytes_per_token``)
  * Sec. 3.1: tiers R/A/S, FP8 Recent/Anchor, 3-bit rotated Stale codec
  * Alg. 1: Append, Retier, Promote, SealPrefix and Finish transitions
    (``Pool.append``, ``Pool.migrate``, ``Pool.promote``, ``Pool.acquire`` /
    ``Pool.release``, ``Pool.finish``); Sec. 4.4 reference counts
  * Sec. 3.2, Eq. (effective-bits): effective rate (``effective_bits``)
  * Sec. 3.3, Eq. (softmax-merge): partials and merge (``merge``)
  * Sec. 4.1: compact per-format lists, TQ3 page contents, the canary's
    active-cache byte counter (``canary_bytes``)
  * Sec. 4.3: FP8 -> TQ3 normalize-rotate-pack (``tq3_encode``)
  * Sec. 3.1, Eqs. (score-partial), (score-global-weight), (attention-score):
    page attention mass and its EWMA (``Pool.page_scores``)

Every function is pinned by CPU tests against closed forms, library routines
or brute force; none is "parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mkv_oracle.c")
_LIB_PATH = os.path.join(_HERE, "_build", "liborc.so")
_lib = None

PAGE = 16
TAG_R, TAG_A, TAG_S, TAG_NONE = 0, 1, 2, 0xFF
CODEBOOK = np.array([-2.25, -1.375, -0.75, -0.25, 0.25, 0.75, 1.375, 2.25])


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, no FMA contraction)."""
    os.makedirs(os.path.dirname(_LIB_PATH), exist_ok=True)
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call([
            "gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
            "-shared", "-std=c11", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        _lib = ctypes.CDLL(_LIB_PATH)
        _declare(_lib)
    return _lib


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return lib().orc_num_threads()


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _declare(L):
    vp, i32, i64, f32, f64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_double
    L.orc_e4m3_to_f64.restype = f64
    L.orc_e4m3_to_f64.argtypes = [ctypes.c_uint8]
    L.orc_e4m3_from_f32.restype = ctypes.c_uint8
    L.orc_e4m3_from_f32.argtypes = [f32]
    L.orc_e4m3_from_f32_array.argtypes = [vp, vp, i64]
    L.orc_f16_from_f64.restype = ctypes.c_uint16
    L.orc_f16_from_f64.argtypes = [f64]
    L.orc_f16_to_f64.restype = f64
    L.orc_f16_to_f64.argtypes = [ctypes.c_uint16]
    L.orc_f16_from_f64_array.argtypes = [vp, vp, i64]
    L.orc_hadamard_i64.argtypes = [vp, vp, i32]
    L.orc_tq3_decide.restype = i32
    L.orc_tq3_decide.argtypes = [i64, i64]
    L.orc_tq3_encode.argtypes = [i32, vp, f32, vp, f32, vp, vp, vp, vp, vp, vp]
    L.orc_tq3_dequant.argtypes = [i32, vp, vp, vp, vp, vp, vp, vp, vp]
    L.orc_tq3_pack.argtypes = [i32, vp, vp, vp, vp, vp, vp]
    L.orc_tq3_unpack.argtypes = [i32, vp, vp, vp, vp, vp, vp]
    L.orc_tq3_bit_pos.argtypes = [i32, i32, i32, i32, vp, vp]
    L.orc_fp8_k_off.restype = i64
    L.orc_fp8_k_off.argtypes = [i32, i32, i32]
    L.orc_fp8_v_off.restype = i64
    L.orc_fp8_v_off.argtypes = [i32, i32, i32]
    L.orc_tq3_region_bytes.restype = i64
    L.orc_tq3_region_bytes.argtypes = [i32]
    L.orc_tier.restype = i32
    L.orc_tier.argtypes = [i32, i32, i32, i32]
    L.orc_append.restype = i32
    L.orc_append.argtypes = [vp, i32, i32, vp, vp, i32, vp, vp, vp, vp]
    L.orc_migrate.restype = i32
    L.orc_migrate.argtypes = [vp, i32, vp, vp, i32, vp, vp]
    L.orc_pages_acquire.restype = i32
    L.orc_pages_acquire.argtypes = [vp, i32, vp, vp]
    L.orc_pages_release.restype = i32
    L.orc_pages_release.argtypes = [vp, i32, vp, vp]
    L.orc_request_finish.restype = i32
    L.orc_request_finish.argtypes = [vp, i32, vp, vp, vp, i32]
    L.orc_promote.restype = i32
    L.orc_promote.argtypes = [vp, i32, vp, vp, i32, vp, vp]
    L.orc_tq3_reconstruct_f32.argtypes = [i32, vp, vp, vp, vp, vp, vp, vp, vp]
    L.orc_partition.argtypes = [i32, vp, vp, i32, vp, vp, vp, vp]
    L.orc_reconstruct.argtypes = [vp, i32, i32, i32, vp, vp, i32, i32, vp, vp]
    L.orc_decode.argtypes = [vp, i32, i32, i32, vp, vp, vp, i32, vp, vp, vp]
    L.orc_chunk.argtypes = [vp, i32, i32, i32, vp, vp, vp, vp, i32, vp, vp, vp]
    L.orc_merge.argtypes = [i32, i32, vp, vp, vp, vp, vp]
    L.orc_page_scores.argtypes = [vp, i32, i32, i32, vp, vp, vp, i32, vp, vp, f64, vp, vp, vp]
    L.orc_num_threads.restype = i32
    L.orc_num_threads.argtypes = []


# --------------------------------------------------------------------------
# Scalar formats
# --------------------------------------------------------------------------
_E4M3_TABLE = None


def e4m3_to_f64(codes: np.ndarray) -> np.ndarray:
    """Value of OCP E4M3FN codes (NaN for 0x7F/0xFF)."""
    global _E4M3_TABLE
    if _E4M3_TABLE is None:
        L = lib()
        _E4M3_TABLE = np.array([L.orc_e4m3_to_f64(i) for i in range(256)])
    return _E4M3_TABLE[np.asarray(codes, dtype=np.uint8)]


def e4m3_from_f32(x: np.ndarray) -> np.ndarray:
    """Round fp32 -> E4M3FN: nearest, ties to even, saturate to +-448."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint8)
    lib().orc_e4m3_from_f32_array(_p(x), _p(out), x.size)
    return out


def f16_from_f64(x: np.ndarray) -> np.ndarray:
    """One round-to-nearest-even fp64 -> binary16 (bits), saturating at 65504."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().orc_f16_from_f64_array(_p(x), _p(out), x.size)
    return out


def f16_to_f64(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# TQ3 codec (Sec. 3.1, Sec. 4.1, Sec. 4.3)
# --------------------------------------------------------------------------
def hadamard_i64(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.int64)
    y = np.empty_like(x)
    lib().orc_hadamard_i64(_p(x), _p(y), x.size)
    return y


def tq3_decide(y: int, n2: int) -> int:
    return lib().orc_tq3_decide(int(y), int(n2))


def tq3_encode(d, k8, sK, v8, sV, sigma):
    """Encode one FP8 page-head (16 tokens, logical [t][c] code order)."""
    k8 = np.ascontiguousarray(k8, dtype=np.uint8).reshape(PAGE, d)
    v8 = np.ascontiguousarray(v8, dtype=np.uint8).reshape(PAGE, d)
    sigma = np.ascontiguousarray(sigma, dtype=np.int8)
    kc = np.empty((PAGE, d), np.uint8)
    vc = np.empty((PAGE, d), np.uint8)
    g = np.empty(PAGE, np.uint16)
    vs = np.empty(d, np.uint16)
    vz = np.empty(d, np.uint16)
    lib().orc_tq3_encode(d, _p(k8), float(sK), _p(v8), float(sV), _p(sigma), _p(kc), _p(g),
                         _p(vc), _p(vs), _p(vz))
    return dict(kcode=kc, gamma=g, vcode=vc, vscale=vs, vzero=vz)


def tq3_dequant(d, enc, sigma):
    sigma = np.ascontiguousarray(sigma, dtype=np.int8)
    kh = np.empty((PAGE, d))
    vh = np.empty((PAGE, d))
    lib().orc_tq3_dequant(d, _p(enc["kcode"]), _p(enc["gamma"]), _p(enc["vcode"]),
                          _p(enc["vscale"]), _p(enc["vzero"]), _p(sigma), _p(kh), _p(vh))
    return kh, vh


def tq3_reconstruct_f32(d, enc, sigma):
    """Promote's fp32 reconstruction of one TQ3 page-head: (k32, v32) [16][d]."""
    sigma = np.ascontiguousarray(sigma, dtype=np.int8)
    k32 = np.empty((PAGE, d), np.float32)
    v32 = np.empty((PAGE, d), np.float32)
    lib().orc_tq3_reconstruct_f32(d, _p(enc["kcode"]), _p(enc["gamma"]), _p(enc["vcode"]),
                                  _p(enc["vscale"]), _p(enc["vzero"]), _p(sigma), _p(k32), _p(v32))
    return k32, v32


def tq3_pack(d, enc) -> np.ndarray:
    region = np.empty(tq3_region_bytes(d), np.uint8)
    lib().orc_tq3_pack(d, _p(enc["kcode"]), _p(enc["gamma"]), _p(enc["vcode"]),
                       _p(enc["vscale"]), _p(enc["vzero"]), _p(region))
    return region


def tq3_unpack(d, region) -> dict:
    region = np.ascontiguousarray(region, dtype=np.uint8)
    kc = np.empty((PAGE, d), np.uint8)
    vc = np.empty((PAGE, d), np.uint8)
    g = np.empty(PAGE, np.uint16)
    vs = np.empty(d, np.uint16)
    vz = np.empty(d, np.uint16)
    lib().orc_tq3_unpack(d, _p(region), _p(kc), _p(g), _p(vc), _p(vs), _p(vz))
    return dict(kcode=kc, gamma=g, vcode=vc, vscale=vs, vzero=vz)


def tq3_bit_pos(d, q, b, k):
    by = ctypes.c_int()
    bi = ctypes.c_int()
    lib().orc_tq3_bit_pos(d, q, b, k, ctypes.byref(by), ctypes.byref(bi))
    return by.value, bi.value


def tq3_region_bytes(d: int) -> int:
    return 16 * d + 32


def fp8_region_bytes(d: int) -> int:
    return 2 * PAGE * d


def fp8_k_off(d, t, c):
    return lib().orc_fp8_k_off(d, t, c)


def fp8_v_off(d, t, c):
    return lib().orc_fp8_v_off(d, t, c)


def tier(p, seq_len, W, is_anchor):
    return lib().orc_tier(p, seq_len, W, int(bool(is_anchor)))


# --------------------------------------------------------------------------
# Pool state machine (Alg. 1) and attention (Sec. 3.3)
# --------------------------------------------------------------------------
class _CPool(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int), ("n_kv_heads", ctypes.c_int), ("d", ctypes.c_int),
                ("n_fp8", ctypes.c_int), ("n_tq3", ctypes.c_int), ("recent", ctypes.c_int),
                ("sigma", ctypes.c_void_p), ("fp8", ctypes.c_void_p),
                ("fp8_scale", ctypes.c_void_p), ("tq3", ctypes.c_void_p),
                ("fp8_stack", ctypes.c_void_p), ("fp8_top", ctypes.c_void_p),
                ("tq3_stack", ctypes.c_void_p), ("tq3_top", ctypes.c_void_p),
                ("rc8", ctypes.c_void_p), ("rc3", ctypes.c_void_p)]


class Pool:
    """Host mirror of the device pools, in the same byte layout.

    Free stacks: ids are handed out in the order of ``fp8_order`` /
    ``tq3_order``; released ids are pushed and reused last-in first-out."""

    def __init__(self, n_layers, n_q_heads, n_kv_heads, d, n_fp8, n_tq3, recent, sigma,
                 fp8_order=None, tq3_order=None):
        self.n_layers, self.n_q_heads, self.n_kv_heads, self.d = n_layers, n_q_heads, n_kv_heads, d
        self.n_fp8, self.n_tq3, self.recent = n_fp8, n_tq3, recent
        self.sigma = np.ascontiguousarray(sigma, dtype=np.int8)
        self.fp8 = np.zeros((n_layers, n_fp8, n_kv_heads, fp8_region_bytes(d)), np.uint8)
        self.fp8_scale = np.zeros((n_layers, n_fp8, n_kv_heads, 2), np.float32)
        self.tq3 = np.zeros((n_layers, n_tq3, n_kv_heads, tq3_region_bytes(d)), np.uint8)
        o8 = np.arange(n_fp8) if fp8_order is None else np.asarray(fp8_order)
        o3 = np.arange(n_tq3) if tq3_order is None else np.asarray(tq3_order)
        self.fp8_stack = np.ascontiguousarray(o8[::-1], dtype=np.int32)
        self.tq3_stack = np.ascontiguousarray(o3[::-1], dtype=np.int32)
        self.fp8_top = np.array([n_fp8], np.int32)
        self.tq3_top = np.array([n_tq3], np.int32)
        self.rc8 = np.zeros(n_fp8, np.int32)  # references per page (0: free)
        self.rc3 = np.zeros(max(n_tq3, 1), np.int32)

    def _c(self):
        s = _CPool(self.n_layers, self.n_kv_heads, self.d, self.n_fp8, self.n_tq3, self.recent,
                   self.sigma.ctypes.data, self.fp8.ctypes.data, self.fp8_scale.ctypes.data,
                   self.tq3.ctypes.data, self.fp8_stack.ctypes.data, self.fp8_top.ctypes.data,
                   self.tq3_stack.ctypes.data, self.tq3_top.ctypes.data,
                   self.rc8.ctypes.data, self.rc3.ctypes.data)
        self._keep = s
        return ctypes.byref(s)

    def append(self, layer, block_table, tags, seq_before, cu_new, k_bf16, v_bf16) -> int:
        n_req, max_pages = block_table.shape
        k = np.ascontiguousarray(k_bf16, dtype=np.uint16)
        v = np.ascontiguousarray(v_bf16, dtype=np.uint16)
        sb = np.ascontiguousarray(seq_before, dtype=np.int32)
        cu = np.ascontiguousarray(cu_new, dtype=np.int32)
        return lib().orc_append(self._c(), layer, n_req, _p(block_table), _p(tags), max_pages,
                                _p(sb), _p(cu), _p(k), _p(v))

    def migrate(self, block_table, tags, anchor, seq_lens) -> int:
        n_req, max_pages = block_table.shape
        sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
        an = None if anchor is None else np.ascontiguousarray(anchor, dtype=np.uint8)
        return lib().orc_migrate(self._c(), n_req, _p(block_table), _p(tags), max_pages,
                                 None if an is None else _p(an), _p(sl))

    def promote(self, block_table, tags, promote_mask, seq_lens) -> int:
        """Alg. 1 Promote of every Stale page whose mask entry is set."""
        n_req, max_pages = block_table.shape
        sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
        pm = np.ascontiguousarray(promote_mask, dtype=np.uint8)
        return lib().orc_promote(self._c(), n_req, _p(block_table), _p(tags), max_pages, _p(pm),
                                 _p(sl))

    def acquire(self, ids, tags) -> int:
        """Alg. 1 SealPrefix / prefix attach: one more reference per listed page."""
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        tg = np.ascontiguousarray(tags, dtype=np.uint8)
        return lib().orc_pages_acquire(self._c(), len(ids), _p(ids), _p(tg))

    def release(self, ids, tags) -> int:
        """Prefix eviction: drop one reference per listed page (pages freed)."""
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        tg = np.ascontiguousarray(tags, dtype=np.uint8)
        return lib().orc_pages_release(self._c(), len(ids), _p(ids), _p(tg))

    def finish(self, reqs, block_table, tags) -> int:
        """Alg. 1 Finish of the listed requests (ascending): rows released, unmapped."""
        n_req, max_pages = block_table.shape
        rq = np.ascontiguousarray(reqs, dtype=np.int32)
        return lib().orc_request_finish(self._c(), len(rq), _p(rq), _p(block_table), _p(tags),
                                        max_pages)

    def reconstruct(self, layer, r, h, block_table, tags, n_tok):
        n_req, max_pages = block_table.shape
        kh = np.empty((max(n_tok, 1), self.d))
        vh = np.empty((max(n_tok, 1), self.d))
        lib().orc_reconstruct(self._c(), layer, r, h, _p(block_table), _p(tags), max_pages, n_tok,
                              _p(kh), _p(vh))
        return kh[:n_tok], vh[:n_tok]

    def decode(self, layer, q_bf16, block_table, tags, seq_lens):
        n_req, max_pages = block_table.shape
        q = np.ascontiguousarray(q_bf16, dtype=np.uint16)
        sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
        out = np.zeros((n_req, self.n_q_heads, self.d))
        lse = np.zeros((n_req, self.n_q_heads))
        lib().orc_decode(self._c(), layer, n_req, self.n_q_heads, _p(q), _p(block_table), _p(tags),
                         max_pages, _p(sl), _p(out), _p(lse))
        return out, lse

    def page_scores(self, layer, q_bf16, block_table, tags, seq_lens, head_mask, beta, a):
        """Attention-score collector (Sec. 3.1 Eqs. score-partial ..
        attention-score): updates `a` [n_req][max_pages] in place; returns
        (q~ [n_req][max_pages][Hq], r [n_req][max_pages])."""
        n_req, max_pages = block_table.shape
        q = np.ascontiguousarray(q_bf16, dtype=np.uint16)
        sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
        hm = np.ascontiguousarray(head_mask, dtype=np.uint8)
        assert a.dtype == np.float64 and a.flags.c_contiguous and a.shape == (n_req, max_pages)
        qn = np.full((n_req, max_pages, self.n_q_heads), np.nan)
        rr = np.full((n_req, max_pages), np.nan)
        lib().orc_page_scores(self._c(), layer, n_req, self.n_q_heads, _p(q), _p(block_table),
                              _p(tags), max_pages, _p(sl), _p(hm), float(beta), _p(a), _p(qn),
                              _p(rr))
        return qn, rr

    def chunk(self, layer, q_bf16, cu_q, block_table, tags, seq_lens, sample_stride=1):
        n_req, max_pages = block_table.shape
        q = np.ascontiguousarray(q_bf16, dtype=np.uint16)
        cu = np.ascontiguousarray(cu_q, dtype=np.int32)
        sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
        out = np.full((q.shape[0], self.n_q_heads, self.d), np.nan)
        st = np.ascontiguousarray(np.broadcast_to(np.asarray(sample_stride, np.int32), (n_req,)))
        lib().orc_chunk(self._c(), layer, n_req, self.n_q_heads, _p(q), _p(cu), _p(block_table),
                        _p(tags), max_pages, _p(sl), _p(out), _p(st))
        return out


def partition(block_table, tags, seq_lens):
    """Compact per-format lists (Sec. 4.1): (lists8, lists3, counts)."""
    n_req, max_pages = block_table.shape
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    tg = np.ascontiguousarray(tags, dtype=np.uint8)
    sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
    o8 = np.full((n_req, max_pages, 2), -1, np.int32)
    o3 = np.full((n_req, max_pages, 2), -1, np.int32)
    cnt = np.zeros((n_req, 2), np.int32)
    lib().orc_partition(n_req, _p(bt), _p(tg), max_pages, _p(sl), _p(o8), _p(o3), _p(cnt))
    return o8, o3, cnt


def merge(m, l, obar):
    """Eq. (softmax-merge): partials (m_j, l_j, Obar_j) -> (O, lse)."""
    m = np.ascontiguousarray(m, dtype=np.float64)
    l = np.ascontiguousarray(l, dtype=np.float64)
    obar = np.ascontiguousarray(obar, dtype=np.float64)
    d = obar.shape[-1]
    out = np.empty(d)
    lse = np.empty(1)
    lib().orc_merge(m.size, d, _p(m), _p(l), _p(obar), _p(out), _p(lse))
    return out, lse[0]


# --------------------------------------------------------------------------
# Byte accounting (Sec. 2.1, Sec. 3.2, Sec. 4.1 / 6.3)
# --------------------------------------------------------------------------
def kv_bytes_per_token(n_full_layers, n_kv_heads, head_dim, bytes_per_scalar):
    """Eq. (kv-per-token): m = 2 * L_f * H_kv * d_h * s."""
    return 2 * n_full_layers * n_kv_heads * head_dim * bytes_per_scalar


def fp8_page_head_bytes(d, page=PAGE, with_scales=True):
    return 2 * page * d + (8 if with_scales else 0)


def tq3_page_head_bytes(d, page=PAGE):
    """3-bit K and V codes, fp16 gamma per token, fp16 V scale and zero per channel."""
    return 2 * page * 3 * d // 8 + 2 * page + 4 * d


def effective_bits(p_R, p_A, p_S, b_S, b_meta=0.0):
    """Eq. (effective-bits): b_eff = 8(p_R + p_A) + b_S p_S + b_meta."""
    return 8.0 * (p_R + p_A) + b_S * p_S + b_meta


def canary_bytes(n_fp8_page_layers, n_tq3_page_layers, page=1792, n_kv_heads=4, d=256):
    """Active-cache byte counter of the direct canary (Sec. 6.3) under the
    per-channel V metadata reading: FP8 page-layers are priced by their codes,
    TQ3 page-layers by codes + fp16 gamma per token + fp16 V scale/zero per
    channel; the full cache is priced in BF16 over all page-layers."""
    fp8 = n_fp8_page_layers * n_kv_heads * 2 * page * d
    tq3 = n_tq3_page_layers * n_kv_heads * (2 * page * 3 * d // 8 + 2 * page + 4 * d)
    full = (n_fp8_page_layers + n_tq3_page_layers) * n_kv_heads * 2 * page * d * 2
    return fp8 + tq3, full
