"""Conformance of the GPU's fp64 arithmetic that the bit-exact TQ3 metadata
rests on (Sec. 4.1: FP16 key-norm correction gamma and FP16 V scale/zero are
computed in fp64 and rounded once to binary16).  The library's own compiled
division, square root and binary16 rounding (mkv_fp64_probe) are compared bit
for bit with numpy's IEEE-754 float64 division and square root and numpy's
float64 -> float16 conversion (nearest-even; saturated here at 65504 as the
library defines it) on 10^8 random inputs per operation."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

N_BATCH, BATCH = 10, 10_000_000


def _doubles(torch, n, e_lo, e_hi, signed, gen):
    """Random finite doubles: uniform 52-bit significands, biased exponents
    uniform in [e_lo, e_hi] (e_lo = 0 gives subnormals), random sign."""
    mant = torch.randint(0, 1 << 52, (n,), dtype=torch.int64, device="cuda", generator=gen)
    ex = torch.randint(e_lo, e_hi + 1, (n,), dtype=torch.int64, device="cuda", generator=gen)
    bits = (ex << 52) | mant
    if signed:
        sg = torch.randint(0, 2, (n,), dtype=torch.int64, device="cuda", generator=gen)
        bits = bits | (sg << 63)
    return bits.view(torch.float64)


def test_fp64_div_sqrt_and_binary16_rounding_match_ieee():
    import torch
    import paper_2608_23834_amd as mk
    assert torch.cuda.is_available()
    gen = torch.Generator(device="cuda")
    gen.manual_seed(20261010)
    quot = torch.empty(BATCH, dtype=torch.float64, device="cuda")
    root = torch.empty_like(quot)
    half = torch.empty(BATCH, dtype=torch.int16, device="cuda")
    bad = {"div": 0, "sqrt": 0, "f16": 0}
    for k in range(N_BATCH):
        # even batches: the whole normal range (and subnormal operands); odd
        # batches: the ranges the encoders meet (ratios of integers near 1,
        # values around the binary16 range, including its subnormals and
        # saturation)
        if k % 2 == 0:
            a = _doubles(torch, BATCH, 0, 2046, False, gen)
            b = _doubles(torch, BATCH, 0, 2046, True, gen)
        else:  # every other odd batch with negative operands too (sqrt checked on a >= 0)
            a = _doubles(torch, BATCH, 1023 - 30, 1023 + 20, k % 4 == 3, gen)
            b = _doubles(torch, BATCH, 1023 - 8, 1023 + 8, True, gen)
        mk.mkv_fp64_probe(a, b, quot, root, half)
        torch.cuda.synchronize()
        an, bn = a.cpu().numpy(), b.cpu().numpy()
        with np.errstate(over="ignore", under="ignore"):
            q_ref = an / bn
            h_ref = an.astype(np.float16)
        pos = an >= 0
        r_ref = np.sqrt(np.where(pos, an, 0.0))
        h_ref = np.where(np.isinf(h_ref), np.copysign(np.float16(65504.0), h_ref), h_ref).astype(np.float16)
        bad["div"] += int(np.count_nonzero(quot.cpu().numpy().view(np.int64) != q_ref.view(np.int64)))
        r_gpu = root.cpu().numpy()
        bad["sqrt"] += int(np.count_nonzero((r_gpu.view(np.int64) != r_ref.view(np.int64)) & pos))
        bad["sqrt"] += int(np.count_nonzero(~np.isnan(r_gpu[~pos])))
        bad["f16"] += int(np.count_nonzero(half.cpu().numpy().view(np.uint16) != h_ref.view(np.uint16)))
        print(f"  batch {k}: mismatches so far {bad}", flush=True)
    assert bad == {"div": 0, "sqrt": 0, "f16": 0}, bad
