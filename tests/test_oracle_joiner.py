"""Pins for the oracle's decoder + joiner + log-softmax (Algorithm 1, decoder and joiner)."""
import numpy as np
import pytest
import scipy.special

import oracle
from paper_2211_00484_amd import synth
from ref_search import LayerJoiner


def _rand_case(seed, V=12, C=24, sigma=0.3, R=9):
    rng = np.random.default_rng(seed)
    model = synth.make_model(rng, V, C, sigma)
    enc = rng.standard_normal((R, C), dtype=np.float32)
    a = rng.integers(0, V, R).astype(np.int32)
    b = rng.integers(0, V, R).astype(np.int32)
    return model, enc, a, b


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("bf16", [False, True])
def test_matches_library_layers(seed, bf16):
    model, enc, a, b = _rand_case(seed)
    got = oracle.logp(model, enc, a, b, bf16=bf16)
    ref = LayerJoiner(model, bf16=bf16)
    for r in range(enc.shape[0]):
        np.testing.assert_allclose(got[r], ref(enc[r], int(a[r]), int(b[r])), rtol=0, atol=1e-12)


def test_zero_weight_gives_log_softmax_of_bias():
    model, enc, a, b = _rand_case(7)
    model.w_out[:] = 0.0
    got = oracle.logp(model, enc, a, b)
    want = scipy.special.log_softmax(model.b_out.astype(np.float64))
    for r in range(enc.shape[0]):
        np.testing.assert_allclose(got[r], want, atol=1e-13)


def test_normalised_over_full_vocab_including_blank():
    model, enc, a, b = _rand_case(3, V=40)
    got = oracle.logp(model, enc, a, b)
    np.testing.assert_allclose(np.exp(got).sum(axis=1), 1.0, atol=1e-12)


def test_tap0_weights_the_older_label():
    model, enc, a, b = _rand_case(11)
    model.conv[:, 0] = 0.0                      # older label can no longer matter
    base = oracle.logp(model, enc, a, b)
    other = oracle.logp(model, enc, (a + 1) % model.vocab_size, b)
    np.testing.assert_array_equal(base, other)
    changed = oracle.logp(model, enc, a, (b + 1) % model.vocab_size)
    assert np.abs(changed - base).max() > 1e-6


def test_tap1_weights_the_newer_label():
    model, enc, a, b = _rand_case(12)
    model.conv[:, 1] = 0.0
    base = oracle.logp(model, enc, a, b)
    np.testing.assert_array_equal(base, oracle.logp(model, enc, a, (b + 3) % model.vocab_size))
    assert np.abs(oracle.logp(model, enc, (a + 3) % model.vocab_size, b) - base).max() > 1e-6


def test_decoder_relu_and_tanh_closed_form():
    # Negative embedding with positive taps -> decoder output clamped to 0, so the
    # joiner sees tanh(enc).  With C = 1 and W[v] = v, z_v = v * tanh(e) + bias_v.
    V, C = 5, 1
    model = synth.Model(V, C, embed=-np.ones((V, C), np.float32),
                        conv=np.ones((C, 2), np.float32),
                        w_out=np.arange(V, dtype=np.float32).reshape(V, 1),
                        b_out=np.linspace(-0.5, 0.5, V).astype(np.float32))
    e = np.float32(0.75)
    got = oracle.logp(model, np.array([[e]], np.float32), np.array([2]), np.array([3]))[0]
    z = np.arange(V) * np.tanh(np.float64(e)) + model.b_out.astype(np.float64)
    np.testing.assert_allclose(got, z - scipy.special.logsumexp(z), atol=1e-14)


def test_bf16_rounding_is_round_to_nearest_even():
    # W values exactly between two bfloat16 neighbours must round to the even one.
    V, C = 3, 1
    one_plus_half_ulp = np.float32(1.0 + 2.0 ** -8)          # tie between 1 and 1 + 2^-7
    three_half_ulps = np.float32(1.0 + 3 * 2.0 ** -8)        # tie between 1+2^-7 and 1+2^-6
    w = np.array([[one_plus_half_ulp], [three_half_ulps], [0.0]], np.float32)
    model = synth.Model(V, C, embed=np.zeros((V, C), np.float32), conv=np.zeros((C, 2), np.float32),
                        w_out=w, b_out=np.zeros(V, np.float32))
    enc = np.array([[np.arctanh(0.5)]], np.float32)          # h = 0.5, exact in bf16 after rounding
    got = oracle.logp(model, enc, np.array([0]), np.array([0]), bf16=True)[0]
    assert abs(np.tanh(np.float64(enc[0, 0])) - 0.5) < 1e-7
    hb = 0.5                                                 # nearest bfloat16 of h
    z = np.array([1.0 * hb, (1.0 + 2.0 ** -6) * hb, 0.0])
    np.testing.assert_allclose(got, z - scipy.special.logsumexp(z), atol=1e-14)
