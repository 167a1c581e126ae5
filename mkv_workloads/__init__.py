"""Seeded synthetic inputs for the five Minima-KV workloads.

This module only draws data: bf16 Q/K/V tensors, sequence lengths, anchor page
sets, free-list orders and the rotation sign vector.  It holds none of the
method's arithmetic (no quantisation, tiering, rotation or attention), so both
the CPU oracle's tests and the GPU path can consume the same arrays.

The shapes follow the paper's deployment (Sec. 4.1 / Sec. 5.4: 16 full-attention
layers, 24 query heads, 4 KV heads, head dim 256) and its long-context canary
(Sec. 6.3: two requests of 59,008 prompt tokens).  Real model KV is not
available, so values are N(0,1) draws with per-channel log-normal scales
(sigma = 0.5) per layer, head and channel, which imitate the heavy channels of
real keys; the tiny config instead scales 4 key channels by 8.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

PAGE = 16


@dataclasses.dataclass(frozen=True)
class Workload:
    cfg_id: int
    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    recent: int            # Recent window W in tokens
    first_anchor_pages: int
    anchor_frac: float     # fraction of the remaining old pages drawn as anchors
    n_req: int
    ctx: tuple             # per-request context length (decode: seq_len)
    chunk: int = 0         # chunked-prefill query tokens per request (config 5)
    outlier_k_channels: int = 0
    lognormal_sigma: float = 0.5

    @property
    def seed(self) -> int:
        return 20260000 + self.cfg_id

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


# purposes of the derived streams
_K_SIGMA, _K_ANCHOR, _K_ORDER8, _K_ORDER3, _K_LENS, _K_OUTLIER = 1, 2, 3, 4, 5, 6
_K_Q, _K_K, _K_V, _K_SQ, _K_SK, _K_SV, _K_QC = 10, 11, 12, 13, 14, 15, 16


def _cfg4_lens(n, seed):
    g = _rng(seed, _K_LENS)
    return tuple(int(x) for x in g.integers(4096, 65536 + 1, size=n))


def workload(cfg_id: int) -> Workload:
    """The five workloads (tiny, single 16K, long pair, batch 64, chunk+migrate)."""
    if cfg_id == 1:
        return Workload(1, "tiny-decode-d128-ctx2048", 1, 8, 1, 128, 256, 4, 0.0, 1, (2048,),
                        outlier_k_channels=4)
    if cfg_id == 2:
        return Workload(2, "single-decode-16k", 16, 24, 4, 256, 1024, 4, 0.02, 1, (16384,))
    if cfg_id == 3:
        return Workload(3, "long-pair-2x59008", 16, 24, 4, 256, 2048, 8, 0.01, 2, (59008, 59008))
    if cfg_id == 4:
        return Workload(4, "batch64-ctx4k-64k", 16, 24, 4, 256, 1024, 4, 0.02, 64,
                        _cfg4_lens(64, 20260004))
    if cfg_id == 5:
        return Workload(5, "chunk512-vs-65536-migrate", 1, 24, 4, 256, 1024, 4, 0.02, 8,
                        (65536 + 512,) * 8, chunk=512)
    raise ValueError(cfg_id)


def scaled(w: Workload, ctx: tuple, n_layers: int | None = None, name: str | None = None,
           chunk: int | None = None) -> Workload:
    """Same geometry and distributions at other lengths (small parity cases)."""
    return dataclasses.replace(w, ctx=tuple(ctx), n_req=len(ctx),
                               n_layers=w.n_layers if n_layers is None else n_layers,
                               name=name or (w.name + "-scaled"),
                               chunk=w.chunk if chunk is None else chunk)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest even (inputs are finite)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> 16) & np.uint32(1))
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def rot_signs(w: Workload) -> np.ndarray:
    """The random +-1 vector of the rotation, one per pool."""
    g = _rng(w.seed, _K_SIGMA)
    return np.where(g.integers(0, 2, size=w.head_dim) == 1, 1, -1).astype(np.int8)


def free_order(w: Workload, n_pages: int, fmt: str) -> np.ndarray:
    """Order in which the pool hands out physical ids: a shuffled permutation,
    so block tables are random permutations of physical pages."""
    g = _rng(w.seed, _K_ORDER8 if fmt == "fp8" else _K_ORDER3)
    return g.permutation(n_pages).astype(np.int32)


def n_pages_of(seq_len: int) -> int:
    return (seq_len + PAGE - 1) // PAGE


def anchor_mask(w: Workload, max_pages: int, seq_lens=None) -> np.ndarray:
    """Anchor set per request: the first pages plus a uniform random draw of
    ``anchor_frac`` of the remaining old pages (count rounded half to even);
    "remaining" excludes the first pages and the pages of the Recent window."""
    lens = w.ctx if seq_lens is None else seq_lens
    m = np.zeros((len(lens), max_pages), np.uint8)
    for r, L in enumerate(lens):
        npg = n_pages_of(L)
        first = min(w.first_anchor_pages, npg)
        m[r, :first] = 1
        lo, hi = first, max(first, npg - w.recent // PAGE)
        remaining = hi - lo
        k = int(round(w.anchor_frac * remaining))  # Python round: half to even
        if k > 0:
            g = _rng(w.seed, _K_ANCHOR, r)
            pick = g.choice(np.arange(lo, hi), size=k, replace=False)
            m[r, pick] = 1
    return m


def _channel_scales(w: Workload, key: int, layer: int, n_heads: int) -> np.ndarray:
    g = _rng(w.seed, key, layer)
    return np.exp(w.lognormal_sigma * g.standard_normal((n_heads, w.head_dim))).astype(np.float32)


def kv_layer(w: Workload, layer: int, n_tok: int, token_offset: int = 0):
    """bf16 K and V for ``n_tok`` consecutive tokens (rows ``token_offset`` ..)
    of one layer, shape [n_tok][Hkv][d] (uint16 bits).  Rows are drawn
    independently per row block so any slice is reproducible."""
    H, d = w.n_kv_heads, w.head_dim
    out = []
    for key, skey in ((_K_K, _K_SK), (_K_V, _K_SV)):
        x = _rows(w.seed, key, layer, token_offset, n_tok, H * d).reshape(n_tok, H, d)
        if w.outlier_k_channels and key == _K_K:
            ch = _rng(w.seed, _K_OUTLIER).choice(d, size=w.outlier_k_channels, replace=False)
            x[:, :, ch] *= 8.0
        elif not w.outlier_k_channels:
            x *= _channel_scales(w, skey, layer, H)[None]
        out.append(bf16_round(x))
    return out[0], out[1]


def outlier_channels(w: Workload) -> np.ndarray:
    if not w.outlier_k_channels:
        return np.zeros(0, np.int64)
    return np.sort(_rng(w.seed, _K_OUTLIER).choice(w.head_dim, size=w.outlier_k_channels,
                                                   replace=False))


_BLOCK = 4096


def _rows(seed, key, layer, start, n, width):
    """N(0,1) rows [start, start+n) of a (virtually infinite) row stream;
    each block of 4096 rows has its own generator (blocks drawn in parallel)."""
    res = np.empty((n, width), np.float32)
    if n <= 0:
        return res
    b0, b1 = start // _BLOCK, (start + n - 1) // _BLOCK

    def one(b):
        g = _rng(seed, key, layer, b)
        blk = g.standard_normal((_BLOCK, width), dtype=np.float32)
        lo = max(start, b * _BLOCK)
        hi = min(start + n, (b + 1) * _BLOCK)
        res[lo - start:hi - start] = blk[lo - b * _BLOCK:hi - b * _BLOCK]

    if b1 - b0 >= 2:
        import concurrent.futures as cf
        with cf.ThreadPoolExecutor(max_workers=min(8, b1 - b0 + 1)) as ex:
            list(ex.map(one, range(b0, b1 + 1)))
    else:
        for b in range(b0, b1 + 1):
            one(b)
    return res


def q_decode(w: Workload, layer: int, step: int = 0) -> np.ndarray:
    """bf16 decode queries [n_req][Hq][d]."""
    g = _rng(w.seed, _K_Q, layer, step)
    x = g.standard_normal((w.n_req, w.n_q_heads, w.head_dim), dtype=np.float32)
    if not w.outlier_k_channels:
        x *= _channel_scales(w, _K_SQ, layer, w.n_q_heads)[None]
    return bf16_round(x)


def q_chunk(w: Workload, layer: int, n_per_req: int, step: int = 0) -> np.ndarray:
    """bf16 chunk queries [n_req * n_per_req][Hq][d]."""
    g = _rng(w.seed, _K_QC, layer, step)
    x = g.standard_normal((w.n_req * n_per_req, w.n_q_heads, w.head_dim), dtype=np.float32)
    x *= _channel_scales(w, _K_SQ, layer, w.n_q_heads)[None]
    return bf16_round(x)


def max_pages_for(w: Workload, extra_tokens: int = 0) -> int:
    return n_pages_of(max(w.ctx) + extra_tokens)


def kv_layer_device(w: Workload, layer: int, n_tok: int, device="cuda"):
    """bf16 K and V for ``n_tok`` tokens of one layer drawn on the device
    (torch's counter-based generator, seeded from the workload), shape
    [n_tok][Hkv][d] int16 bits.  Same distribution as ``kv_layer`` (N(0,1)
    times the per-(layer, head, channel) log-normal scales); used where the
    host generator would be too slow (the 64-request batch holds 2.2 M
    tokens).  Callers that check against the oracle copy rows back to the
    host, so both sides read identical bytes."""
    import torch
    H, d = w.n_kv_heads, w.head_dim
    out = []
    for key, skey in ((_K_K, _K_SK), (_K_V, _K_SV)):
        g = torch.Generator(device=device)
        g.manual_seed(int(np.random.SeedSequence(w.seed, spawn_key=(key, layer)).generate_state(1)[0]))
        x = torch.randn((n_tok, H, d), generator=g, device=device, dtype=torch.float32)
        if not w.outlier_k_channels:
            x *= torch.from_numpy(_channel_scales(w, skey, layer, H)).to(device)[None]
        out.append(x.to(torch.bfloat16).view(torch.int16))
        del x
    return out[0], out[1]
