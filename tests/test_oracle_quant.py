"""Pins of the oracle's INT4 group quantizer (oracle/quant.py) against exact
rational arithmetic: the scale as bf16(float32(a / 7)) rounded exactly, each
code as the nearest grid point (ties to even), the extreme element at +-7,
the all-zero group, and exact dequantization."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import quant
from paper_2608_10362_amd import synth


def _round_to_bits(r: Fraction, mant_bits: int) -> Fraction:
    """Exact round-to-nearest-even of a positive rational to `mant_bits` significant bits."""
    if r == 0:
        return Fraction(0)
    e = 0
    while r >= 2:
        r /= 2
        e += 1
    while r < 1:
        r *= 2
        e -= 1
    scaled = r * (1 << (mant_bits - 1))
    fl = scaled.numerator // scaled.denominator
    rem = scaled - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return Fraction(fl, 1 << (mant_bits - 1)) * (Fraction(2) ** e)


def _bits_to_frac(b) -> Fraction:
    return Fraction(float(np.array([int(b) << 16], np.uint32).view(np.float32)[0]))


def _weights(N, K, seed):
    rng = np.random.default_rng(seed)
    w = rng.standard_normal((N, K)).astype(np.float32) * np.float32(0.02)
    w[0, :7] = np.float32(0.0)  # some exact zeros
    return synth.f32_to_bf16_bits(w)


@pytest.mark.parametrize("N,K", [(3, 256), (2, 136)])
def test_scales_are_the_exactly_rounded_max_over_seven(N, K):
    w = _weights(N, K, 1)
    q, s = quant.quantize_int4(w)
    assert s.shape == (N, (K + 127) // 128)
    for n in range(N):
        for g in range(s.shape[1]):
            a = max(abs(_bits_to_frac(b)) for b in w[n, g * 128:(g + 1) * 128])
            want = _round_to_bits(_round_to_bits(a / 7, 24), 8)  # float32 division, then bf16
            assert _bits_to_frac(s[n, g]) == want


@pytest.mark.parametrize("N,K", [(3, 256), (2, 136)])
def test_codes_are_the_nearest_grid_points_ties_to_even(N, K):
    w = _weights(N, K, 2)
    q, s = quant.quantize_int4(w)
    assert q.min() >= -8 and q.max() <= 7
    for n in range(N):
        for k in range(K):
            sf = _bits_to_frac(s[n, k // 128])
            wf = _bits_to_frac(w[n, k])
            if sf == 0:
                assert q[n, k] == 0
                continue
            # the code's distance is the smallest over the 16 codes; of two equally
            # close codes, the even one (round half to even of w / s)
            d = [abs(wf - c * sf) for c in range(-8, 8)]
            best = min(d)
            cands = [c for c in range(-8, 8) if d[c + 8] == best]
            want = cands[0] if len(cands) == 1 else [c for c in cands if c % 2 == 0][0]
            assert q[n, k] == want, (n, k)


def test_group_extreme_maps_to_seven_and_zero_groups_stay_zero():
    w = np.zeros((2, 256), np.float32)
    w[0, 5] = -0.05
    w[0, 9] = 0.01
    w[0, 130] = 0.03
    bits = synth.f32_to_bf16_bits(w)
    q, s = quant.quantize_int4(bits)
    assert q[0, 5] == -7 and q[0, 130] == 7
    assert (q[1] == 0).all() and (s[1] == 0).all()
    # one non-zero value alone in its group: its code is +-7, every other code 0
    assert np.count_nonzero(q[0, 128:]) == 1


def test_dequantized_weights_are_exact_and_within_half_a_step():
    w = _weights(4, 384, 3)
    q, s = quant.quantize_int4(w)
    deq = quant.dequantize_int4(q, s)
    wf = synth.bf16_bits_to_f32(w).astype(np.float64)
    sf = np.repeat(synth.bf16_bits_to_f32(s).astype(np.float64), 128, axis=1)
    assert np.all(np.abs(deq - wf) <= sf / 2 * (1 + 2 ** -7))
    # q * s is exact in float64 (4-bit integer times an 8-bit significand)
    for n in range(2):
        for k in range(0, 384, 37):
            assert Fraction(float(deq[n, k])) == int(q[n, k]) * _bits_to_frac(s[n, k // 128])


def test_int4_model_weights_replace_only_the_linear_layers():
    W = synth.make_weights(synth.LLAMA_1B, n_layers=1)
    Q = quant.int4_model_weights(W, n_layers=1)
    assert Q["lm_head"] is W["lm_head"] and Q["embed"] is W["embed"]
    for name in quant.LINEAR:
        assert Q["layers"][0][name].dtype == np.float64
        assert Q["layers"][0][name].shape == W["layers"][0][name].shape
    assert Q["layers"][0]["attn_norm"] is W["layers"][0]["attn_norm"]
