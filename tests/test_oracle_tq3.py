"""Pins for the oracle's TQ3 codec (Sec. 3.1 Stale tier, Sec. 4.1 page contents,
Sec. 4.3 normalize-rotate-pack).

Pinned by: scipy's Hadamard matrix, closed-form basis-vector round trips,
sign symmetry and scale invariance of the decisions, the quantizer's expected
distortion under N(0,1) by numerical integration, the kernel's algebraic
identity q.k_hat = gamma (Rq).mu_c / 1, exact cases of the V quantizer, and a
bijection check of the packed bit layout.
"""
import numpy as np
import pytest
import scipy.linalg
from scipy.integrate import quad
from scipy.stats import norm

D = (128, 256)


def e4m3_codes_for(orc, x):
    return orc.e4m3_from_f32(np.asarray(x, np.float32))


@pytest.mark.parametrize("d", D)
def test_hadamard_matches_scipy(orc, d):
    rng = np.random.default_rng(d)
    x = rng.integers(-229376, 229377, size=d).astype(np.int64)
    H = scipy.linalg.hadamard(d).astype(np.int64)
    assert np.array_equal(orc.hadamard_i64(x), H @ x)


def test_decide_matches_float_away_from_ties(orc):
    rng = np.random.default_rng(3)
    T = (orc.CODEBOOK[1:] + orc.CODEBOOK[:-1]) / 2
    for _ in range(20000):
        n2 = int(rng.integers(1, 2 ** 43))
        y = int(rng.normal() * np.sqrt(n2) * rng.choice([0.3, 1, 2.5]))
        z = y / np.sqrt(n2)
        if np.min(np.abs(z - T)) < 1e-9:
            continue
        assert orc.tq3_decide(y, n2) == int(np.sum(z > T))


def test_decide_exact_ties_go_low(orc):
    # z exactly on a threshold: y = T * sqrt(n2) with n2 a perfect square
    for tau16 in (-29, -17, -8, 0, 8, 17, 29):
        for s in (16, 160, 4096):
            n2 = s * s
            y = tau16 * s // 16
            if y * 16 != tau16 * s:
                continue
            T = tau16 / 16
            want = int(np.sum((orc.CODEBOOK[1:] + orc.CODEBOOK[:-1]) / 2 < T))
            assert orc.tq3_decide(y, n2) == want
    assert orc.tq3_decide(0, 12345) == 3


@pytest.mark.parametrize("d", D)
def test_basis_vector_round_trip(orc, d):
    """k = sK * e_j: every rotated coordinate is +-1, codes are 5 (mu = 0.75)
    for +1 and 2 (mu = -0.75) for -1, gamma = sK / (0.75 sqrt(d)), and the
    reconstruction is sK * e_j up to gamma's fp16 rounding."""
    rng = np.random.default_rng(d)
    sigma = np.where(rng.integers(0, 2, d) == 1, 1, -1).astype(np.int8)
    sK = np.float32(0.0123)
    for j in (0, 1, d // 3, d - 1):
        k8 = np.zeros((16, d), np.uint8)
        k8[:, j] = 0x38  # 1.0
        v8 = np.zeros((16, d), np.uint8)
        enc = orc.tq3_encode(d, k8, sK, v8, np.float32(1.0), sigma)
        H = scipy.linalg.hadamard(d)
        y = H[:, j] * sigma[j]
        want_codes = np.where(y > 0, 5, 2)
        assert np.array_equal(enc["kcode"], np.broadcast_to(want_codes, (16, d)))
        g = float(sK) / (0.75 * np.sqrt(d))
        assert np.all(enc["gamma"] == orc.f16_from_f64(np.array([g]))[0])
        kh, _ = orc.tq3_dequant(d, enc, sigma)
        e = np.zeros(d)
        e[j] = float(sK)
        g16 = orc.f16_to_f64(enc["gamma"][:1])[0]
        assert np.allclose(kh, e * g16 / g, atol=1e-15)


def _random_k8(orc, rng, d, n=16):
    x = rng.standard_normal((n, d)).astype(np.float32) * 40
    return e4m3_codes_for(orc, x)


@pytest.mark.parametrize("d", D)
def test_sign_symmetry_and_scale_invariance(orc, d):
    rng = np.random.default_rng(11)
    sigma = np.where(rng.integers(0, 2, d) == 1, 1, -1).astype(np.int8)
    v8 = np.zeros((16, d), np.uint8)
    T = (orc.CODEBOOK[1:] + orc.CODEBOOK[:-1]) / 2
    for _ in range(10):
        k8 = _random_k8(orc, rng, d)
        enc = orc.tq3_encode(d, k8, 1.0, v8, 1.0, sigma)
        neg = orc.tq3_encode(d, k8 ^ 0x80, 1.0, v8, 1.0, sigma)
        # rows where no rotated coordinate is a tie (incl. 0) obey c(-X) = 7 - c(X)
        X = orc.e4m3_to_f64(k8) * sigma[None, :]
        z = (X @ scipy.linalg.hadamard(d).T) / np.linalg.norm(X, axis=1, keepdims=True)
        clean = np.all(np.min(np.abs(z[..., None] - T), axis=-1) > 1e-12, axis=1)
        assert clean.any()
        assert np.array_equal(neg["kcode"][clean], 7 - enc["kcode"][clean])
        assert np.array_equal(neg["gamma"], enc["gamma"])
        # doubling every key value (exponent + 1) leaves the codes unchanged
        small = (k8 & 0x78) < 0x70  # stays finite after +1 exponent, and normal
        rows = np.all(small & ((k8 & 0x78) != 0) | ((k8 & 0x7F) == 0), axis=1)
        k8d = np.where((k8 & 0x7F) == 0, k8, k8 + 0x08).astype(np.uint8)
        dbl = orc.tq3_encode(d, k8d, 1.0, v8, 1.0, sigma)
        assert np.array_equal(dbl["kcode"][rows], enc["kcode"][rows])


def _codebook_mse():
    c = np.array([-2.25, -1.375, -0.75, -0.25, 0.25, 0.75, 1.375, 2.25])
    t = np.r_[-np.inf, (c[1:] + c[:-1]) / 2, np.inf]
    return sum(quad(lambda x, k=k: (x - c[k]) ** 2 * norm.pdf(x), t[k], t[k + 1])[0]
               for k in range(8))


def test_distortion_matches_quantizer_theory(orc):
    """Rotated, normalised coordinates are ~N(0,1); their quantisation error
    must match the codebook's expected distortion under N(0,1) (0.03489)."""
    d = 256
    rng = np.random.default_rng(5)
    sigma = np.where(rng.integers(0, 2, d) == 1, 1, -1).astype(np.int8)
    H = scipy.linalg.hadamard(d)
    errs = []
    for _ in range(40):
        k8 = _random_k8(orc, rng, d)
        enc = orc.tq3_encode(d, k8, 1.0, np.zeros((16, d), np.uint8), 1.0, sigma)
        X = orc.e4m3_to_f64(k8)
        z = ((X * sigma) @ H.T) / np.linalg.norm(X, axis=1, keepdims=True)
        errs.append((z - orc.CODEBOOK[enc["kcode"]]) ** 2)
    mse = np.mean(errs)
    want = _codebook_mse()
    assert abs(want - 0.03489) < 1e-4
    assert abs(mse - want) < 0.002, (mse, want)


@pytest.mark.parametrize("d", D)
def test_norm_preserved_and_reconstruction_error(orc, d):
    rng = np.random.default_rng(6)
    sigma = np.where(rng.integers(0, 2, d) == 1, 1, -1).astype(np.int8)
    sK = np.float32(0.05)
    k8 = _random_k8(orc, rng, d)
    enc = orc.tq3_encode(d, k8, sK, np.zeros((16, d), np.uint8), 1.0, sigma)
    kh, _ = orc.tq3_dequant(d, enc, sigma)
    k = orc.e4m3_to_f64(k8) * float(sK)
    nk, nh = np.linalg.norm(k, axis=1), np.linalg.norm(kh, axis=1)
    assert np.allclose(nh, nk, rtol=2.0 ** -10)  # gamma is fp16
    rel = np.sum((kh - k) ** 2, axis=1) / nk ** 2
    assert 0.02 < rel.mean() < 0.05  # ~ the 3-bit distortion, not a sign/transposition bug


@pytest.mark.parametrize("d", D)
def test_score_identity_for_rotated_query(orc, d):
    """q . k_hat = gamma * (R q) . mu_c with R = d^-1/2 H diag(sigma): the
    decode kernels rotate the query once instead of every key."""
    rng = np.random.default_rng(8)
    sigma = np.where(rng.integers(0, 2, d) == 1, 1, -1).astype(np.int8)
    k8 = _random_k8(orc, rng, d)
    enc = orc.tq3_encode(d, k8, 0.07, np.zeros((16, d), np.uint8), 1.0, sigma)
    kh, _ = orc.tq3_dequant(d, enc, sigma)
    q = rng.standard_normal(d)
    R = scipy.linalg.hadamard(d) * sigma[None, :] / np.sqrt(d)
    g = orc.f16_to_f64(enc["gamma"])
    lhs = kh @ q
    rhs = g * (orc.CODEBOOK[enc["kcode"]] @ (R @ q))
    assert np.allclose(lhs, rhs, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("d", D)
def test_value_quantizer_exact_cases(orc, d):
    sigma = np.ones(d, np.int8)
    k8 = np.zeros((16, d), np.uint8)
    # channel 0 constant; channel 1 an exact ramp 0..7 (x 0.5); others random
    rng = np.random.default_rng(9)
    v = rng.standard_normal((16, d)).astype(np.float32)
    v[:, 0] = 1.5
    v[:, 1] = 0.5 * np.array([0, 1, 2, 3, 4, 5, 6, 7, 7, 6, 5, 4, 3, 2, 1, 0])
    v8 = e4m3_codes_for(orc, v)
    sV = np.float32(0.25)
    enc = orc.tq3_encode(d, k8, 1.0, v8, sV, sigma)
    _, vh = orc.tq3_dequant(d, enc, sigma)
    vt = orc.e4m3_to_f64(v8) * float(sV)
    assert np.all(vh[:, 0] == vt[:, 0])
    assert np.array_equal(enc["vcode"][:, 1], [0, 1, 2, 3, 4, 5, 6, 7, 7, 6, 5, 4, 3, 2, 1, 0])
    assert np.all(vh[:, 1] == vt[:, 1])
    scale = orc.f16_to_f64(enc["vscale"])
    zero = orc.f16_to_f64(enc["vzero"])
    # error bound: half a step plus the fp16 rounding of the zero point
    bound = scale / 2 + np.abs(zero) * 2.0 ** -11 + np.abs(vt.max(0) - vt.min(0)) * 2.0 ** -11
    assert np.all(np.abs(vh - vt) <= bound[None, :] + 1e-12)


@pytest.mark.parametrize("d", D)
def test_pack_layout_is_a_bijection(orc, d):
    seen = set()
    nbytes = 3 * d // 32
    for q in range(d // 16):
        for b in range(4):
            for k in range(3):
                pos = orc.tq3_bit_pos(d, q, b, k)
                assert 0 <= pos[0] < nbytes and 0 <= pos[1] < 8
                seen.add(pos)
    assert len(seen) == nbytes * 8  # every bit of the chunk used exactly once


@pytest.mark.parametrize("d", D)
def test_pack_unpack_round_trip(orc, d):
    rng = np.random.default_rng(10)
    enc = dict(kcode=rng.integers(0, 8, (16, d)).astype(np.uint8),
               gamma=rng.integers(0, 0x7C00, 16).astype(np.uint16),
               vcode=rng.integers(0, 8, (16, d)).astype(np.uint8),
               vscale=rng.integers(0, 0x7C00, d).astype(np.uint16),
               vzero=rng.integers(0, 0xFC00, d).astype(np.uint16))
    region = orc.tq3_pack(d, enc)
    assert region.size == orc.tq3_region_bytes(d) == 16 * d + 32
    back = orc.tq3_unpack(d, region)
    for key in enc:
        assert np.array_equal(back[key], enc[key]), key


def test_region_sizes(orc):
    assert orc.tq3_region_bytes(256) == 4128 and orc.tq3_region_bytes(128) == 2080
    assert orc.tq3_page_head_bytes(256) == 4128 and orc.fp8_page_head_bytes(256) == 8200
