"""Pins of the fp8 (E4M3FN) KV oracle (CPU).

* encoding equals torch's float8_e4m3fn cast (round to nearest, ties to even)
  on float32 values inside the finite range, subnormals and ties included;
* closed forms: saturation at +-448, the smallest subnormal, ties at
  subnormal and normal spacing, exact values; decoding equals torch's for all
  254 finite codes;
* the fp8-KV decoder: cached steps equal recomputation, and its logits differ
  from the bf16-exact decoder by about the e4m3 rounding, not more;
* planted mistakes (truncation instead of rounding, no saturation) break a pin.
"""

import numpy as np
import pytest
import torch

from oracle import decoder as od
from oracle import fp8
from workload import SMALL_BF16, make_weights, random_tokens


def _torch_codes(x32):
    return torch.from_numpy(x32).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def _random_in_range(n, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(n) * np.exp(rng.uniform(-14, 6.5, n))
    x = x.astype(np.float32)
    return x[np.abs(x) < 448]


def encode_matches_torch(encode):
    x = _random_in_range(200000, 0)
    # exact ties: midpoints between neighbouring codes, both signs
    vals = fp8.e4m3_values()[:0x7F]
    mids = ((vals[:-1] + vals[1:]) / 2).astype(np.float32)
    x = np.concatenate([x, mids, -mids, vals.astype(np.float32)])
    return bool(np.array_equal(encode(x), _torch_codes(x)))


def closed_forms_hold(encode):
    cases = {448.0: 0x7E, 500.0: 0x7E, 1e30: 0x7E, -1000.0: 0xFE, 2.0 ** -9: 0x01,
             2.0 ** -10: 0x00, 3 * 2.0 ** -10: 0x02, 1.0: 0x38, 1.0625: 0x38,  # tie -> even
             1.1875: 0x3A, -2.0 ** -11: 0x80, 240.0: 0x77}
    got = encode(np.array(list(cases), dtype=np.float64))
    return bool(np.array_equal(got, np.array(list(cases.values()), dtype=np.uint8)))


def test_encode_matches_torch():
    assert encode_matches_torch(fp8.e4m3_encode)


def test_closed_forms_and_decode_table():
    assert closed_forms_hold(fp8.e4m3_encode)
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).double().numpy()
    np.testing.assert_array_equal(fp8.e4m3_decode(codes), ref)
    assert np.isnan(fp8.e4m3_decode([0x7F, 0xFF])).all()


def test_fp8_decoder_cached_equals_recompute_and_stays_close():
    shape = SMALL_BF16
    arrays = make_weights(shape, seed=3, bf16=True, std=0.05)
    w = od.ModelWeights.from_arrays(shape, arrays)
    tokens = random_tokens(24, shape.vocab, seed=4)
    scales = (0.5, 0.25)
    dec = od.Decoder(w, kv_fp8=scales)
    st = dec.new_state()
    inc = np.stack([dec.step(st, t) for t in tokens])
    full = od.recompute_logits(w, tokens, kv_fp8=scales)
    np.testing.assert_allclose(inc, full, rtol=0, atol=1e-10 * np.max(np.abs(full)))
    exact = od.recompute_logits(w, tokens)
    rel = np.max(np.abs(full - exact)) / np.max(np.abs(exact))
    assert 1e-5 < rel < 0.1, rel  # fp8 rounding is visible but modest


def _mut_truncate(x):
    a = np.asarray(x, dtype=np.float64)
    vals = fp8.e4m3_values()[:0x7F]
    mag = np.minimum(np.abs(a), 448.0)
    code = np.clip(np.searchsorted(vals, mag, side="right") - 1, 0, 0x7E).astype(np.uint8)
    return (code | (np.signbit(a).astype(np.uint8) << 7)).astype(np.uint8)


def _mut_no_saturation(x):
    a = np.asarray(x, dtype=np.float64)
    out = fp8.e4m3_encode(a)
    out[np.abs(a) > 464] |= 0x7F  # overflow to NaN
    return out


@pytest.mark.parametrize("mutant", [_mut_truncate, _mut_no_saturation])
def test_planted_mistakes_break_a_pin(mutant):
    assert not (encode_matches_torch(mutant) and closed_forms_hold(mutant))
