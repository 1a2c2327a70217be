"""Pins of the oracle's causal attention (the last-layer prefill attention
whose QK^T tiles QER reads, Sec. 3.3): closed forms and invariants that a
dropped term, a wrong sign, a wrong key/value head or a missing causal mask
would break."""
import numpy as np
import pytest

import oracle


def rand(shape, seed, scale=1.0):
    return (np.random.default_rng([2609, 3675, 95, seed]).standard_normal(shape) * scale).astype(np.float32)


def to_bf16(x):
    return (np.ascontiguousarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def test_first_row_is_its_own_value():
    Q, K, V = rand((5, 3, 16), 1), rand((5, 3, 16), 2), rand((5, 3, 16), 3)
    O = oracle.attention(Q, K, V)
    assert np.array_equal(O[0], V[0].astype(np.float64))


@pytest.mark.parametrize("H_q,H_kv", [(2, 2), (4, 2), (3, 1)])
def test_uniform_logits_give_prefix_means(H_q, H_kv):
    L, d = 37, 32
    Q = np.zeros((L, H_q, d), np.float32)
    K, V = rand((L, H_kv, d), 4), rand((L, H_kv, d), 5)
    O = oracle.attention(Q, K, V)
    pref = np.cumsum(V.astype(np.float64), axis=0) / np.arange(1, L + 1)[:, None, None]
    g = np.arange(H_q) * H_kv // H_q
    assert np.allclose(O, pref[:, g], rtol=1e-12, atol=1e-12)


def test_two_keys_closed_form():
    # q1 = (a, 0, ...), k0 = (1, 0, ...), k1 = (0, 1, ...): s_10 = a*scale, s_11 = 0
    d, a, scale = 16, 3.0, 0.5
    Q = np.zeros((2, 1, d), np.float32)
    K = np.zeros((2, 1, d), np.float32)
    Q[1, 0, 0] = a
    K[0, 0, 0] = 1
    K[1, 0, 1] = 1
    V = rand((2, 1, d), 6)
    O = oracle.attention(Q, K, V, scale=scale)
    w0 = 1.0 / (1.0 + np.exp(-a * scale))          # sigmoid(s_10 - s_11)
    expect = w0 * V[0, 0].astype(np.float64) + (1 - w0) * V[1, 0].astype(np.float64)
    assert np.allclose(O[1, 0], expect, rtol=1e-14, atol=1e-14)


def test_hard_attention_limit():
    L, d = 12, 16
    Q, K, V = rand((L, 2, d), 7), rand((L, 2, d), 8), rand((L, 2, d), 9)
    O = oracle.attention(Q, K, V, scale=1e4)
    for i in range(L):
        for h in range(2):
            s = K[:i + 1, h].astype(np.float64) @ Q[i, h].astype(np.float64)
            assert np.allclose(O[i, h], V[np.argmax(s), h], atol=1e-6)


def test_causal():
    L, d = 20, 16
    Q, K, V = rand((L, 2, d), 10), rand((L, 2, d), 11), rand((L, 2, d), 12)
    O = oracle.attention(Q, K, V)
    K2, V2 = K.copy(), V.copy()
    K2[13:] = rand((L - 13, 2, d), 13)
    V2[13:] = rand((L - 13, 2, d), 14)
    O2 = oracle.attention(Q, K2, V2)
    assert np.array_equal(O[:13], O2[:13])
    assert not np.allclose(O[13:], O2[13:])


def test_key_shift_invariance():
    # adding c to every key shifts row i's logits by the constant <q_i, c>
    L, d = 25, 32
    q8 = lambda x: (np.round(x * 8) / 8).astype(np.float32)   # K + c stays exact in fp32
    Q, K, V = rand((L, 2, d), 15), q8(rand((L, 2, d), 16)), rand((L, 2, d), 17)
    c = q8(rand((1, 2, d), 18))
    O = oracle.attention(Q, K, V)
    O2 = oracle.attention(Q, (K + c).astype(np.float32), V)
    assert np.allclose(O, O2, rtol=1e-9, atol=1e-9)


def test_grouped_heads_equal_repeated_heads():
    L, d, H_q, H_kv = 19, 16, 6, 2
    Q, K, V = rand((L, H_q, d), 19), rand((L, H_kv, d), 20), rand((L, H_kv, d), 21)
    rep = H_q // H_kv
    O = oracle.attention(Q, K, V)
    O2 = oracle.attention(Q, np.repeat(K, rep, axis=1), np.repeat(V, rep, axis=1))
    assert np.array_equal(O, O2)


def test_one_hot_values_give_causal_weights():
    # V = identity rows: o_i is the weight vector, non-negative, summing to 1, zero past i
    L, d = 16, 16
    Q, K = rand((L, 1, d), 22, 2.0), rand((L, 1, d), 23)
    V = np.eye(L, d, dtype=np.float32)[:, None, :]
    O = oracle.attention(Q, K, V)[:, 0]
    assert np.all(O >= 0)
    assert np.allclose(O.sum(axis=1), 1.0, atol=1e-12)
    assert np.all(np.triu(O, 1) == 0)
    # and the weights order as the logits do
    for i in range(1, L):
        s = K[:i + 1, 0].astype(np.float64) @ Q[i, 0].astype(np.float64)
        assert np.array_equal(np.argsort(O[i, :i + 1], kind="stable"), np.argsort(s, kind="stable"))


def test_rows_subset_and_bf16_inputs():
    L, d = 30, 32
    Q, K, V = rand((L, 4, d), 24), rand((L, 2, d), 25), rand((L, 2, d), 26)
    Qb, Kb, Vb = to_bf16(Q), to_bf16(K), to_bf16(V)
    full = oracle.attention(Qb, Kb, Vb)
    rows = np.array([29, 0, 7, 7], np.int32)
    assert np.array_equal(oracle.attention(Qb, Kb, Vb, rows=rows), full[rows])
    # bf16 bits read as the fp32 values they denote
    dec = lambda x: (x.astype(np.uint32) << 16).view(np.float32)
    assert np.array_equal(full, oracle.attention(dec(Qb), dec(Kb), dec(Vb)))
    with pytest.raises(ValueError):
        oracle.attention(Q, K, V, rows=np.array([L], np.int32))
