"""Pins for the oracle's byte accounting against numbers the paper prints
(tests/golden/paper_numbers.json: Sec. 2.1, Sec. 3.2, Sec. 4.1, Sec. 6.3)."""
import json
import os

import pytest

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))


def g(key):
    return GOLD[key]["value"]


def test_bytes_per_token(orc):
    assert orc.kv_bytes_per_token(16, 4, 256, 2) == g("qwen_bf16_bytes_per_token")
    assert orc.kv_bytes_per_token(16, 4, 256, 1) == g("qwen_fp8_bytes_per_token")
    per = orc.kv_bytes_per_token(16, 4, 256, 2)
    assert per * 32768 / 2 ** 30 == g("bf16_gib_per_32k")
    assert per * 131072 / 2 ** 30 == g("bf16_gib_per_128k")


def test_canary_counter_reconciles_with_per_channel_v_metadata(orc):
    """The canary's active-cache counter is reproduced exactly by 18 FP8 and 47
    TQ3 page-layers of 1,792 tokens (9+24 and 9+23 blocks), with the TQ3 page
    priced as 3-bit K and V codes + fp16 gamma per token + fp16 V scale/zero
    per channel, and the full cache priced in BF16."""
    comp, full = orc.canary_bytes(18, 47)
    assert comp == g("canary_active_bytes_compressed")
    assert full == g("canary_active_bytes_full")
    assert round(full / comp, 4) == g("canary_compression")
    blocks = -(-g("canary_prompt_tokens") // g("canary_page_tokens"))
    assert blocks == g("canary_blocks_per_request")
    # the split is unique among small integer page counts
    sols = [(a, b) for a in range(0, 66) for b in range(0, 66)
            if orc.canary_bytes(a, b)[0] == g("canary_active_bytes_compressed")]
    assert sols == [(18, 47)]


def test_effective_rate(orc):
    kib = g("deploy_kib_per_token")
    bits = kib * 1024 * 8 / (2 * 16 * 4 * 256)
    assert round(bits, 2) == g("deploy_bits_per_scalar")
    assert round(16 / bits, 3) == g("deploy_vs_bf16")
    assert round(8 / bits, 3) == g("deploy_vs_fp8")
    # Eq. (effective-bits) with no metadata: all-FP8 is 8 bits, all-Stale b_S
    assert orc.effective_bits(1, 0, 0, 3.0) == 8.0
    assert orc.effective_bits(0, 0, 1, 3.0) == 3.0


def test_build_page_sizes(orc):
    # per token-head at 16-token pages, d = 256: FP8 512.5 B, TQ3 258 B, BF16 1024 B
    assert orc.fp8_page_head_bytes(256) / 16 == 512.5
    assert orc.tq3_page_head_bytes(256) / 16 == 258.0
