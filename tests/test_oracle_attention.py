"""Pins of the decode-attention oracle (oracle.attention).

  * a single cached position: the output is that position's value row;
  * identical keys: uniform weights, the output is the mean of the values;
  * one key far ahead of the others: the output is its value row;
  * window semantics: a window covering the whole history equals full
    attention, a window of 1 returns the current value row, and a window of
    Lw equals full attention over the last Lw positions only;
  * GQA: two heads of one group with the same query give the same output, and
    heads read their own group's cache;
  * FlowKV's chunk recurrence (Eq. 6-12, left to right) reproduces the plain
    softmax for several chunk sizes, including chunks that do not divide the
    range.
"""
import numpy as np
import pytest

import oracle
from oracle.attention import attended_range, decode_attention, decode_attention_chunked


def bf16(a):
    return oracle.f32_to_bf16(np.asarray(a, dtype=np.float32))


def rand_case(H, G, d, L, seed):
    rng = np.random.default_rng(seed)
    q = bf16(rng.standard_normal((H, d)))
    K = bf16(rng.standard_normal((G, L, d)))
    V = bf16(rng.standard_normal((G, L, d)))
    return q, K, V


def test_single_position_returns_its_value():
    q, K, V = rand_case(4, 2, 64, 8, 0)
    o, _ = decode_attention(q, K, V, t=0, window=0, scale=0.125)
    vals = oracle.bf16_to_f32(V).astype(np.float64)
    assert np.array_equal(o[:2], np.broadcast_to(vals[0, 0], (2, 64)))
    assert np.array_equal(o[2:], np.broadcast_to(vals[1, 0], (2, 64)))


def test_identical_keys_average_the_values():
    q, K, V = rand_case(2, 1, 32, 10, 1)
    K[:] = K[0, 0]
    o, _ = decode_attention(q, K, V, t=9, window=0, scale=0.5)
    mean = oracle.bf16_to_f32(V).astype(np.float64)[0].mean(axis=0)
    assert np.allclose(o, mean, rtol=0, atol=1e-14)


def test_dominant_key_selects_its_value():
    q, K, V = rand_case(1, 1, 16, 12, 2)
    q[:] = bf16(np.ones((1, 16)))
    K[:] = bf16(np.zeros((1, 12, 16)))
    K[0, 5] = bf16(np.full(16, 8.0))          # score 128 vs 0 for the rest
    o, _ = decode_attention(q, K, V, t=11, window=0, scale=1.0)
    assert np.allclose(o[0], oracle.bf16_to_f32(V)[0, 5], rtol=0, atol=1e-50)


def test_window_semantics():
    q, K, V = rand_case(2, 1, 32, 40, 3)
    full, _ = decode_attention(q, K, V, t=29, window=0, scale=0.2)
    wide, _ = decode_attention(q, K, V, t=29, window=64, scale=0.2)
    assert np.array_equal(full, wide)
    one, _ = decode_attention(q, K, V, t=29, window=1, scale=0.2)
    assert np.array_equal(one, np.broadcast_to(oracle.bf16_to_f32(V).astype(np.float64)[0, 29], (2, 32)))
    w8, _ = decode_attention(q, K, V, t=29, window=8, scale=0.2)
    tail, _ = decode_attention(q, K[:, 22:30], V[:, 22:30], t=7, window=0, scale=0.2)
    assert np.allclose(w8, tail, rtol=0, atol=1e-15)
    assert attended_range(29, 8) == (22, 30) and attended_range(5, 8) == (0, 6) and attended_range(5, 0) == (0, 6)


def test_gqa_mapping():
    q, K, V = rand_case(8, 4, 32, 16, 4)
    q[1] = q[0]
    o, _ = decode_attention(q, K, V, t=15, window=0, scale=0.25)
    assert np.array_equal(o[0], o[1])
    # head 2 reads group 1: replacing group 0's cache does not change it
    K2, V2 = K.copy(), V.copy()
    K2[0], V2[0] = K[2], V[2]
    o2, _ = decode_attention(q, K2, V2, t=15, window=0, scale=0.25)
    assert np.array_equal(o[2:], o2[2:])


@pytest.mark.parametrize("chunk", [1, 7, 64, 256, 1000])
@pytest.mark.parametrize("window", [0, 100])
def test_chunk_recurrence_reproduces_softmax(chunk, window):
    q, K, V = rand_case(4, 2, 64, 300, 5)
    o, _ = decode_attention(q, K, V, t=270, window=window, scale=0.125)
    oc = decode_attention_chunked(q, K, V, t=270, window=window, scale=0.125, chunk=chunk)
    assert np.allclose(oc, o, rtol=1e-12, atol=1e-13)
