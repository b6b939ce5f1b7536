"""Pins of the oracle's QKV generation (Eq. 1) from outside the oracle: closed forms
for one-hot embeddings and one-hot weights (which also fix the head order), brute
force with exactly rounded sums on tiny shapes, exact power-of-two scaling, and a
planted transposition."""
import math

import numpy as np
import pytest

from oracle import hack_oracle as O


def _f16(seed, shape, scale=1.0):
    g = np.random.default_rng(seed)
    return (g.standard_normal(shape, dtype=np.float32) * np.float32(scale)).astype(np.float16)


def test_one_hot_embeddings_return_weight_columns():
    """E = [I 0]: token t's Q/K/V channels are column t of W (exactly; no rounding)."""
    Hq, Hkv, d, hidden, L = 4, 2, 8, 16, 10
    W = _f16(1, ((Hq + 2 * Hkv) * d, hidden))
    E = np.zeros((L, hidden), np.float16)
    E[np.arange(L), np.arange(L)] = 1.0
    Q, K, V = O.project_qkv(E, W, Hq, Hkv, d)
    for t in range(L):
        col = W[:, t]
        assert np.array_equal(Q[:, t, :].reshape(-1), col[:Hq * d])
        assert np.array_equal(K[:, t, :].reshape(-1), col[Hq * d:(Hq + Hkv) * d])
        assert np.array_equal(V[:, t, :].reshape(-1), col[(Hq + Hkv) * d:])


def test_one_hot_weight_lands_on_its_head_channel_and_token():
    """A single non-zero weight at (output channel n, input i) gives exactly one
    non-zero output, E[t, i] * w, at Q/K/V head n // d, channel n % d, for every t."""
    Hq, Hkv, d, hidden, L = 4, 2, 8, 16, 5
    E = _f16(2, (L, hidden))
    for n, kind in ((3, "q"), (Hq * d + 9, "k"), ((Hq + Hkv) * d + 15, "v")):
        W = np.zeros(((Hq + 2 * Hkv) * d, hidden), np.float16)
        W[n, 7] = 0.5
        Q, K, V = O.project_qkv(E, W, Hq, Hkv, d)
        arr = {"q": Q, "k": K, "v": V}[kind]
        base = {"q": 0, "k": Hq * d, "v": (Hq + Hkv) * d}[kind]
        h, c = divmod(n - base, d)
        want = (E[:, 7].astype(np.float64) * 0.5).astype(np.float16)
        assert np.array_equal(arr[h, :, c], want)
        assert np.count_nonzero(Q) + np.count_nonzero(K) + np.count_nonzero(V) == np.count_nonzero(want)


def test_brute_force_exactly_rounded_sums():
    """Tiny shapes: each output is the exactly rounded sum (math.fsum of the exact
    fp16 x fp16 products) rounded once to fp16."""
    Hq, Hkv, d, hidden, L = 2, 1, 4, 24, 3
    E, W = _f16(3, (L, hidden)), _f16(4, ((Hq + 2 * Hkv) * d, hidden), 0.2)
    Q, K, V = O.project_qkv(E, W, Hq, Hkv, d)
    got = np.concatenate([Q.transpose(1, 0, 2).reshape(L, -1), K.transpose(1, 0, 2).reshape(L, -1),
                          V.transpose(1, 0, 2).reshape(L, -1)], axis=1)
    for t in range(L):
        for n in range(W.shape[0]):
            exact = math.fsum(float(E[t, i]) * float(W[n, i]) for i in range(hidden))
            assert got[t, n] == np.float16(exact), (t, n)


def test_power_of_two_scaling_is_exact():
    Hq, Hkv, d, hidden, L = 2, 1, 8, 32, 6
    E, W = _f16(5, (L, hidden)), _f16(6, ((Hq + 2 * Hkv) * d, hidden), 0.1)
    a = O.project_qkv(E, W, Hq, Hkv, d)
    b = O.project_qkv((E.astype(np.float32) * 4).astype(np.float16), W, Hq, Hkv, d)
    for x, y in zip(a, b):
        assert np.array_equal((x.astype(np.float32) * 4).astype(np.float16), y)


def test_token_subset_matches_full_projection():
    Hq, Hkv, d, hidden, L = 2, 1, 8, 32, 9
    E, W = _f16(7, (L, hidden)), _f16(8, ((Hq + 2 * Hkv) * d, hidden), 0.1)
    full = O.project_qkv(E, W, Hq, Hkv, d)
    part = O.project_qkv(E, W, Hq, Hkv, d, tokens=[0, 4, 8])
    for x, y in zip(full, part):
        assert np.array_equal(x[:, [0, 4, 8]], y)


def test_planted_transposed_weights_are_caught(monkeypatch):
    """A projection that reads W's rows as input channels (E W instead of E W^T) fails
    the one-hot-weight pin."""
    real = O.project_qkv

    def wrong(E, W, q_heads, kv_heads, head_dim, tokens=None):
        Wt = np.asarray(W, np.float16)
        sq = np.zeros((Wt.shape[0], Wt.shape[0]), np.float16)
        k = min(Wt.shape)
        sq[:, :k] = Wt[:, :k]
        return real(E[:, :sq.shape[1]] if E.shape[1] >= sq.shape[1] else
                    np.pad(E, ((0, 0), (0, sq.shape[1] - E.shape[1]))), sq.T, q_heads, kv_heads, head_dim, tokens)

    monkeypatch.setattr(O, "project_qkv", wrong)
    with pytest.raises(AssertionError):
        test_one_hot_weight_lands_on_its_head_channel_and_token()


def test_prefill_from_embeddings_equals_projection_then_attention():
    """With one-hot embeddings and weights whose columns hold given Q/K/V values, the
    prefill from embeddings equals quantize-then-attend of those values (the
    projection is exact there), for a causal 40-token prompt with GQA."""
    Hq, Hkv, d, pi, bits, L = 4, 2, 128, 32, 2, 40
    hidden = L
    Qv, Kv, Vv = _f16(9, (Hq, L, d)), _f16(10, (Hkv, L, d)), _f16(11, (Hkv, L, d))
    # W column t = token t's [Q heads | K heads | V heads] channels
    W = np.concatenate([Qv.transpose(0, 2, 1).reshape(Hq * d, L), Kv.transpose(0, 2, 1).reshape(Hkv * d, L),
                        Vv.transpose(0, 2, 1).reshape(Hkv * d, L)])
    E = np.eye(L, hidden, dtype=np.float16)[None]
    out, Q, seqs = O.prefill_from_embeddings(E, W, Hq, Hkv, d, bits, pi)
    assert np.array_equal(Q[0], Qv)
    ref_seqs = [[O.quantize_sequence(Kv[h], Vv[h], bits, pi, seq=0, head=h, kv_heads=Hkv) for h in range(Hkv)]]
    ref = O.attend_prefill(Qv[None], ref_seqs, Hkv, True)
    assert np.array_equal(out, ref)
    for h in range(Hkv):
        assert np.array_equal(seqs[0][h].k_codes, ref_seqs[0][h].k_codes)
        assert np.array_equal(seqs[0][h].v_codes, ref_seqs[0][h].v_codes)
