"""Pins of the oracle's homomorphic products (Eq. 4) and quantized attention
(Sec. 5.3, Eq. 2-3) against exact identities, brute force on tiny inputs and
closed-form special cases.  Planted mistakes at the end show each pin bites."""
import math

import numpy as np
import pytest

from oracle import hack_oracle as O


def _f16(seed, shape, scale=1.0):
    g = np.random.default_rng(seed)
    return (g.standard_normal(shape, dtype=np.float32) * np.float32(scale)).astype(np.float16)


def _random_quantized(seed, n, bits):
    g = np.random.default_rng(seed)
    codes = g.integers(0, 1 << bits, size=n)
    return codes, float(g.normal()), float(abs(g.normal()) + 0.01)


# ---------------------------------------------------------------- Eq. 4 -------------
def _eq4_identity_error(hq):
    """max relative gap between Eq. 4 and the dequantize-then-multiply product."""
    worst = 0.0
    for seed in range(50):
        for n in (16, 32, 64):
            a, ma, sa = _random_quantized(seed, n, 8)
            b, mb, sb = _random_quantized(seed + 1000, n, 2)
            _, est = hq(a, ma, sa, b, mb, sb)
            exact = float(np.dot(sa * a + ma, sb * b + mb))
            worst = max(worst, abs(est - exact) / max(1.0, abs(exact)))
    return worst


def test_eq4_is_exact_identity():
    assert _eq4_identity_error(O.hq_partition) < 1e-12


def test_eq4_brute_force_tiny():
    """Pure-Python loops over dequantized elements on a 3x4 @ 4x2 case."""
    g = np.random.default_rng(11)
    A = g.integers(0, 256, size=(3, 4)); B = g.integers(0, 4, size=(4, 2))
    ma = g.normal(size=(3, 1)); sa = np.abs(g.normal(size=(3, 1))) + .1
    mb = g.normal(size=(1, 2)); sb = np.abs(g.normal(size=(1, 2))) + .1
    prods, C = O.hq_matmul(A, ma, sa, B, mb, sb, 4)
    for i in range(3):
        for j in range(2):
            acc = 0.0
            ip = 0
            for z in range(4):
                acc += (sa[i, 0] * A[i, z] + ma[i, 0]) * (sb[0, j] * B[z, j] + mb[0, j])
                ip += int(A[i, z]) * int(B[z, j])
            assert abs(C[i, j] - acc) < 1e-12 * max(1, abs(acc))
            assert prods[i, j, 0] == ip


def test_eq4_symmetric_special_case():
    """With both minima 0 only the scaled integer product remains (symmetric quantization)."""
    a, _, sa = _random_quantized(3, 32, 8)
    b, _, sb = _random_quantized(4, 32, 4)
    prod, est = O.hq_partition(a, 0.0, sa, b, 0.0, sb)
    assert est == sa * sb * prod


def test_multi_partition_sum_equals_dequantized_matmul():
    """Sec. 5.2: with several partitions along Z, AB = A1B1 + A2B2 + ... each by Eq. 4."""
    g = np.random.default_rng(5)
    M, Z, N, pi = 5, 128, 7, 32
    A = g.integers(0, 256, size=(M, Z)); B = g.integers(0, 4, size=(Z, N))
    ma = g.normal(size=(M, Z // pi)); sa = np.abs(g.normal(size=(M, Z // pi))) + .1
    mb = g.normal(size=(Z // pi, N)); sb = np.abs(g.normal(size=(Z // pi, N))) + .1
    _, C = O.hq_matmul(A, ma, sa, B, mb, sb, pi)
    Ad = np.repeat(sa, pi, axis=1) * A + np.repeat(ma, pi, axis=1)
    Bd = np.repeat(sb, pi, axis=0) * B + np.repeat(mb, pi, axis=0)
    assert np.allclose(C, Ad @ Bd, rtol=1e-12, atol=1e-9)


# --------------------------------------------------- attention pins ------------------
def _seq(seed, L, bits=2, pi=32, d=128):
    k = _f16(seed, (L, d)); v = _f16(seed + 1, (L, d))
    return k, v, O.quantize_sequence(k, v, bits, pi)


def _dequant_scores(q, sq):
    """q_hat . k_hat / sqrt(d) in float64 from independently dequantized operands."""
    qc, qm, qs, _ = O.quantize_query(q, sq.partition)
    qhat = np.repeat(qs, sq.partition) * qc + np.repeat(qm, sq.partition)
    return O.dequantize_k(sq) @ qhat / math.sqrt(q.shape[0])


@pytest.mark.parametrize("L,pi,bits", [(1, 32, 2), (33, 32, 2), (100, 64, 4), (256, 32, 2)])
def test_scores_equal_dequantized_product(L, pi, bits):
    q = _f16(9, (128,))
    _, _, sq = _seq(L, L, bits, pi)
    S, prods, qc, _, _ = O.scores(q, sq)
    ref = _dequant_scores(q, sq)
    assert np.allclose(S, ref, rtol=1e-12, atol=1e-10)
    for p in range(128 // pi):   # integer partition products against a direct sum
        sl = slice(p * pi, (p + 1) * pi)
        assert np.array_equal(prods[:, p], (sq.k_codes[:, sl] * qc[sl]).sum(1))


def _pv_pin_gap(pv_fn, L, tail_mode):
    """max |pv_fn - (dequantized P blocks) @ (dequantized V blocks) - open-block term|."""
    _, v, sq = _seq(21, L)
    g = np.random.default_rng(3)
    prob = g.random(L); prob /= prob.sum()
    O_ = pv_fn(prob, sq, 8, tail_mode)
    Pi, F, T = sq.partition, sq.full_blocks, sq.tail_tokens
    ref = np.zeros(128)
    for blk in range(F):
        pc, pm, ps, _ = O.quantize_partition(prob[blk * Pi:(blk + 1) * Pi], 8, "f64")
        vhat = sq.v_scale[blk] * sq.v_codes[blk] + sq.v_min[blk]
        ref += (ps * pc + pm) @ vhat
    if T:
        pt = prob[F * Pi:]
        if tail_mode == O.TAIL_FP16:
            ref += pt @ v[F * Pi:].astype(np.float64)
        else:
            pc, pm, ps, _ = O.quantize_partition(pt, 8, "f64")
            vhat = sq.v_scale[F] * sq.v_codes[F, :T] + sq.v_min[F]
            ref += (ps * pc + pm) @ vhat
    return np.abs(O_ - ref).max() / max(1e-300, np.abs(ref).max())


@pytest.mark.parametrize("L,tail_mode", [(64, 0), (77, 0), (77, 1), (5, 1)])
def test_pv_equals_dequantized_product(L, tail_mode):
    assert _pv_pin_gap(O.pv_blocks, L, tail_mode) < 1e-12


@pytest.mark.parametrize("L", [64, 80, 20])
def test_zero_query_gives_mean_of_values(L):
    """q = 0: S = 0, P uniform 1/L, every P block constant (codes 0, min 1/L), so O is the
    mean of the dequantized full blocks plus (1/L) times the fp16 open block."""
    _, v, sq = _seq(31, L)
    O_ = O.decode_row(np.zeros(128, np.float16), sq)
    F, T, Pi = sq.full_blocks, sq.tail_tokens, sq.partition
    total = O.dequantize_v_blocks(sq).sum(0) if F else np.zeros(128)
    total = total + v[F * Pi:].astype(np.float64).sum(0)
    assert np.allclose(O_, total / L, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("L", [64, 20])
def test_causal_first_row_is_first_value(L):
    """Row 0 of causal prefill has P = [1, 0, ...]: the first block quantizes to codes
    [255, 0, ...] with min 0 and scale 1/255, so O_0 = v_hat_0 (or the fp16 v_0 when
    token 0 is in the open block)."""
    k, v, sq = _seq(41, L)
    Q = _f16(42, (1, 1, L, 128))
    O_ = O.attend_prefill(Q, [[sq]], 1, causal=True, rows=[(0, 0, 0)])[0, 0, 0]
    if L >= sq.partition:
        ref = sq.v_scale[0] * sq.v_codes[0, 0] + sq.v_min[0]
    else:
        ref = v[0].astype(np.float64)
    assert np.allclose(O_, ref, rtol=1e-6, atol=1e-6)


def test_prefill_last_row_equals_decode():
    L = 96
    k, v, sq = _seq(51, L)
    Q = _f16(52, (1, 2, L, 128))
    last = O.attend_prefill(Q, [[sq]], 1, causal=True, rows=[(0, 1, L - 1)])[0, 1, L - 1]
    dec = O.decode_row(Q[0, 1, L - 1], sq)
    assert np.array_equal(last, dec.astype(np.float32))


def test_noncausal_prefill_rows_equal_decode():
    L = 40
    k, v, sq = _seq(55, L)
    Q = _f16(56, (1, 1, L, 128))
    out = O.attend_prefill(Q, [[sq]], 1, causal=False, rows=[(0, 0, i) for i in (0, 17, 39)])
    for i in (0, 17, 39):
        assert np.array_equal(out[0, 0, i], O.decode_row(Q[0, 0, i], sq).astype(np.float32))


def test_gqa_heads_with_same_query_match():
    L = 70
    _, _, sq0 = _seq(61, L)
    _, _, sq1 = _seq(62, L)
    q = np.repeat(_f16(63, (1, 1, 128)), 8, axis=1)          # 8 q heads, 2 kv heads
    out = O.attend_decode(q, [[sq0, sq1]], 2)
    for h in range(1, 4):
        assert np.array_equal(out[0, h], out[0, 0])
        assert np.array_equal(out[0, 4 + h], out[0, 4])
    assert not np.array_equal(out[0, 0], out[0, 4])


def test_more_bits_approach_unquantized_attention():
    L = 200
    k = _f16(71, (L, 128)); v = _f16(72, (L, 128)); q = _f16(73, (128,))
    ref = O.attention_unquantized(q, k, v)
    errs = []
    for bits in (2, 4, 8):
        sq = O.quantize_sequence(k, v, bits, 32)
        errs.append(np.abs(O.decode_row(q, sq) - ref).max())
    assert errs[0] > errs[1] > errs[2]
    assert errs[2] < 0.02 * np.abs(ref).max()


def test_softmax_rows_sum_to_one():
    S = np.random.default_rng(1).normal(size=(10, 300)) * 20
    for row in S:
        assert abs(O.softmax(row).sum() - 1) < 1e-12


def test_stochastic_sequence_is_deterministic_and_seeded():
    k = _f16(81, (40, 128)); v = _f16(82, (40, 128))
    a = O.quantize_sequence(k, v, 2, 32, O.STOCHASTIC, seed=5, seq=1, head=2, kv_heads=4)
    b = O.quantize_sequence(k, v, 2, 32, O.STOCHASTIC, seed=5, seq=1, head=2, kv_heads=4)
    c = O.quantize_sequence(k, v, 2, 32, O.STOCHASTIC, seed=6, seq=1, head=2, kv_heads=4)
    assert np.array_equal(a.k_codes, b.k_codes) and np.array_equal(a.v_codes, b.v_codes)
    assert not np.array_equal(a.k_codes, c.k_codes)


def test_append_equivalence_of_prefix_quantization():
    """K partitions of earlier tokens never change when tokens are appended (Sec. 5.3);
    full V blocks never change either; only the open block does."""
    k = _f16(91, (70, 128)); v = _f16(92, (70, 128))
    a = O.quantize_sequence(k[:40], v[:40], 2, 32)
    b = O.quantize_sequence(k, v, 2, 32)
    assert np.array_equal(a.k_codes, b.k_codes[:40])
    assert np.array_equal(a.v_codes[0], b.v_codes[0])
    assert not np.array_equal(a.v_codes[1, :8], b.v_codes[1, :8]) or a.v_min[1].tolist() != b.v_min[1].tolist()


def test_pack_cache_layout_roundtrip():
    """The byte format decodes back to the oracle's codes and metadata (contiguous and paged)."""
    L, H, pi, bits = 77, 2, 32, 2
    seqs = [[O.quantize_sequence(_f16(100 + h, (L, 128)), _f16(200 + h, (L, 128)), bits, pi)
             for h in range(H)]]
    for page_tokens, table, pages in ((128, None, 1), (64, np.array([[3, 1]]), 4)):
        out = O.pack_cache(seqs, H, 128, bits, pi, page_tokens, pages, table)
        for h in range(H):
            sq = seqs[0][h]
            for t in (0, 33, 76):
                pg = t // page_tokens if table is None else table[0][t // page_tokens]
                pg = 0 if table is None else pg
                row = out["k_codes"][pg, h, t % page_tokens]
                assert np.array_equal(O.unpack_codes(row, bits), sq.k_codes[t])
                assert np.array_equal(out["k_meta"][pg, h, t % page_tokens, :, 0].astype(np.float64), sq.k_min[t])
            blk = 1
            pg = 0 if table is None else table[0][blk * pi // page_tokens]
            bi = (blk * pi % page_tokens) // pi
            assert np.array_equal(O.unpack_codes(out["v_codes"][pg, h, bi], bits), sq.v_codes[blk].T)
            assert np.array_equal(out["v_tail"][0, h, :sq.tail_tokens], sq.v_tail)


# ------------------------------------------------------- planted mistakes -------------
def _eq4_dropped_term(a, ma, sa, b, mb, sb):
    prod, _ = O.hq_partition(a, ma, sa, b, mb, sb)
    a = np.asarray(a); b = np.asarray(b)
    return prod, sa * sb * prod + sa * mb * a.sum() + len(a) * ma * mb


def _eq4_swapped_sums(a, ma, sa, b, mb, sb):
    prod, _ = O.hq_partition(a, ma, sa, b, mb, sb)
    a = np.asarray(a); b = np.asarray(b)
    return prod, sa * sb * prod + sa * mb * b.sum() + ma * sb * a.sum() + len(a) * ma * mb


def test_planted_eq4_mistakes_are_caught():
    assert _eq4_identity_error(_eq4_dropped_term) > 1e-3
    assert _eq4_identity_error(_eq4_swapped_sums) > 1e-3


def test_planted_score_mistakes_are_caught(monkeypatch):
    q = _f16(9, (128,))
    _, _, sq = _seq(33, 33, 2, 32)
    ref = _dequant_scores(q, sq)
    real = O.quantize_query

    def wrong_sum(qrow, pi, bits=8, sr=None):
        c, m, s, tot = real(qrow, pi, bits, sr)
        return c, m, s, tot[::-1].copy()           # sums of the wrong partitions
    monkeypatch.setattr(O, "quantize_query", wrong_sum)
    S, _, _, _, _ = O.scores(q, sq)
    assert not np.allclose(S, ref, rtol=1e-6)
    monkeypatch.setattr(O, "quantize_query", real)
    sq.k_min = -sq.k_min                            # a sign slip in the K minima
    S, _, _, _, _ = O.scores(q, sq)
    sq.k_min = -sq.k_min
    assert not np.allclose(S, _dequant_scores(q, sq), rtol=1e-6)


def test_planted_pv_mistake_is_caught():
    """Using n = Pi instead of n = T for the re-quantized open block, or dropping the
    cached-sum term, breaks the PV pin."""
    def wrong_count(prob, sq, bits, mode):
        F, T, Pi = sq.full_blocks, sq.tail_tokens, sq.partition
        pc, pm, ps, _ = O.quantize_partition(prob[F * Pi:], bits, "f64")
        return O.pv_blocks(prob, sq, bits, mode) + (Pi - T) * pm * sq.v_min[F]

    def dropped_sum_term(prob, sq, bits, mode):
        out = O.pv_blocks(prob, sq, bits, mode)
        Pi = sq.partition
        for blk in range(sq.full_blocks):
            pc, pm, ps, _ = O.quantize_partition(prob[blk * Pi:(blk + 1) * Pi], bits, "f64")
            out = out - pm * sq.v_scale[blk] * sq.v_sum[blk]
        return out
    assert _pv_pin_gap(wrong_count, 77, O.TAIL_REQUANT) > 1e-6
    assert _pv_pin_gap(dropped_sum_term, 77, O.TAIL_FP16) > 1e-6


def test_empty_sequence_packs_and_attends():
    sq = O.quantize_sequence(_f16(1, (0, 128)), _f16(2, (0, 128)), 2, 32)
    out = O.pack_cache([[sq]], 1, 128, 2, 32, 64, 1)
    assert not out["k_codes"].any() and not out["v_tail"].any()
    assert np.all(O.decode_row(_f16(3, (128,)), sq) == 0)


# ---- stochastic rounding of the transient Q and P codes (reading R4) ----------------
def test_qp_index_layout_and_distinctness():
    """((seq*H_q + head) * 2^20 + row) * 2^24 + col: the closed form, and distinct values
    over a small grid of (seq, head, row, col) by brute force."""
    assert int(O.qp_index(1, 4, 2, 3, 5)) == ((1 * 4 + 2) * 2 ** 20 + 3) * 2 ** 24 + 5
    seen = set()
    for b in range(3):
        for h in range(4):
            for i in range(3):
                cols = O.qp_index(b, 4, h, i, np.arange(300))
                seen.update(int(x) for x in cols)
    assert len(seen) == 3 * 4 * 3 * 300


def test_element_index_layout_and_distinctness():
    """Stored K/V elements (reading R4): ((seq*H_kv + head) * 2^32 + token) * d + channel.
    The closed form, and distinct values over a small grid of (seq, head, token,
    channel) by brute force, so no two stored elements share a threshold."""
    assert int(O.element_index(1, 4, 2, 3, 5, 128)) == ((1 * 4 + 2) * 2 ** 32 + 3) * 128 + 5
    seen = set()
    for b in range(3):
        for h in range(4):
            idx = O.element_index(b, 4, h, np.arange(50)[:, None], np.arange(128)[None, :], 128)
            seen.update(int(x) for x in idx.ravel())
    assert len(seen) == 3 * 4 * 50 * 128


def test_stochastic_sequence_draws_each_elements_own_threshold():
    """quantize_sequence under stochastic rounding gives K partition (t, p) and V block
    (blk, channel c) the thresholds of their own elements: the codes equal a direct
    quantize_partition call with u taken at those elements' indices (a swapped token and
    channel, or the wrong stream, changes them)."""
    L, d, pi, bits, seed, seq, head, H = 70, 128, 32, 2, 9, 2, 1, 3
    k, v = _f16(31, (L, d)), _f16(32, (L, d))
    sq = O.quantize_sequence(k, v, bits, pi, O.STOCHASTIC, seed, seq, head, H)
    near = O.quantize_sequence(k, v, bits, pi)
    assert not np.array_equal(sq.k_codes, near.k_codes)
    for t, p in ((0, 0), (5, 3), (69, 2)):
        ch = np.arange(p * pi, (p + 1) * pi)
        u = O.stochastic_threshold(seed, O.STREAM_K, O.element_index(seq, H, head, t, ch, d))
        c, m, s, tot = O.quantize_partition(k[t, ch][None, :], bits, "f16", O.STOCHASTIC, u[None, :])
        assert np.array_equal(sq.k_codes[t, ch], c[0]) and sq.k_sum[t, p] == tot[0]
    for blk, c_ in ((0, 0), (1, 77), (1, 127)):
        toks = np.arange(blk * pi, (blk + 1) * pi)
        u = O.stochastic_threshold(seed, O.STREAM_V, O.element_index(seq, H, head, toks, c_, d))
        c, m, s, tot = O.quantize_partition(v[toks, c_][None, :], bits, "f16", O.STOCHASTIC, u[None, :])
        assert np.array_equal(sq.v_codes[blk, :, c_], c[0]) and sq.v_sum[blk, c_] == tot[0]


def test_stochastic_query_codes_are_floor_or_ceil_and_unbiased():
    """Over 4000 seeds each Q code is floor(t) or floor(t)+1 with t = (x-m)*fl(1/s) in
    float32 (R3), and the mean dequantized value s*c + m approaches x (E[c] = t)."""
    q = _f16(21, (128,))
    n = 4000
    acc = np.zeros(128)
    c0, m0, s0, _ = O.quantize_query(q, 32)              # nearest: same m, s
    x = q.astype(np.float32).reshape(4, 32)
    t = (x - m0[:, None].astype(np.float32)) * (np.float32(1) / s0[:, None].astype(np.float32))
    fl = np.floor(t).reshape(128)
    for seed in range(n):
        c, m, s, _ = O.quantize_query(q, 32, 8, O.QPStochastic(seed, 0, 1, 0, 0))
        assert np.array_equal(m, m0) and np.array_equal(s, s0)
        assert np.all((c == fl) | (c == fl + 1))
        acc += np.repeat(s, 32) * c + np.repeat(m, 32)
    mean = acc / n
    sigma = np.repeat(s0, 32) / 2 / math.sqrt(n)          # |c - t| < 1, so sd(s c) <= s/2
    assert np.all(np.abs(mean - q.astype(np.float64)) <= 5 * sigma + 1e-12)


def test_stochastic_p_blocks_are_unbiased():
    """For a fixed probability row, the mean over seeds of the Eq. 4 output of the
    stochastically quantized P blocks approaches p . V_hat (the dequantized V blocks) plus
    the fp16 open block: the closed form of unbiased rounding."""
    _, _, sq = _seq(41, 3 * 32 + 9, 2, 32)
    g = np.random.default_rng(5)
    prob = g.random(sq.length)
    prob /= prob.sum()
    vhat = np.concatenate([sq.v_codes[k] * sq.v_scale[k][None, :] + sq.v_min[k][None, :]
                           for k in range(sq.full_blocks)])
    exact = prob[:vhat.shape[0]] @ vhat + prob[vhat.shape[0]:] @ sq.v_tail.astype(np.float64)
    n = 1500
    outs = np.stack([O.pv_blocks(prob, sq, 8, O.TAIL_FP16, O.QPStochastic(seed, 0, 1, 0, 0)) for seed in range(n)])
    near = O.pv_blocks(prob, sq, 8, O.TAIL_FP16)
    # spread of one call around the exact value: at most one code step s_p per element
    bound = 5 * outs.std(axis=0) / math.sqrt(n) + 1e-12
    assert np.all(np.abs(outs.mean(axis=0) - exact) <= bound)
    assert not np.allclose(outs[0], outs[1])             # different seeds, different codes
    assert np.abs(near - exact).max() > 0                # nearest rounding is not the closed form


# ---- operation counts of Sec. 5.2 / 5.3 ------------------------------------------
def test_eq4_operation_count_matches_the_paper():
    """Evaluating Eq. 4 element by element with an operation counter gives 2MZN integer
    operations and 9MN + MZ + NZ correction operations (plus the M + N products of the
    per-row and per-column factors, a lower-order term), and the same C as the
    vectorised Eq. 4."""
    g = np.random.default_rng(17)
    for M, Z, N in ((1, 8, 5), (3, 16, 2), (4, 7, 6)):
        A = g.integers(0, 4, size=(M, Z)); B = g.integers(0, 4, size=(Z, N))
        ma, sa = g.normal(size=M), np.abs(g.normal(size=M)); mb, sb = g.normal(size=N), np.abs(g.normal(size=N))
        C, iops, fops = O.count_eq4_ops(A, ma, sa, B, mb, sb)
        int_cost, corr_cost = O.hq_matmul_cost(M, Z, N)
        assert iops == int_cost == 2 * M * Z * N
        assert fops == corr_cost + M + N
        _, ref = O.hq_matmul(A, ma[:, None], sa[:, None], B, mb[None, :], sb[None, :], Z)
        assert np.allclose(C, ref, rtol=1e-12, atol=1e-12)


def test_decode_cost_model_break_even_points():
    """Sec. 5.3: per decode step the correction costs 10(d + L) + 2dL, and 10(d + L) once
    the code sums are cached; dequantizing K and V costs 4dL.  With d = 128 the
    dequantization exceeds the correction for L > 2.5 and exceeds it tenfold for L > 30
    (exactly 31.07: the paper's 30 is approximate)."""
    d = 128
    assert O.decode_approximation_cost(d, 100, sums_cached=False) == 10 * (d + 100) + 2 * d * 100
    assert O.decode_approximation_cost(d, 100) == 10 * (d + 100)
    assert O.dequantization_cost(d, 2) < O.decode_approximation_cost(d, 2)
    assert O.dequantization_cost(d, 3) > O.decode_approximation_cost(d, 3)
    exact = 10 * d / (4 * d - 10)
    assert 2.5 < exact < 2.6
    ten = 100 * d / (4 * d - 100)
    assert 31 < ten < 31.1
    assert O.dequantization_cost(d, 31) < 10 * O.decode_approximation_cost(d, 31)
    assert O.dequantization_cost(d, 32) > 10 * O.decode_approximation_cost(d, 32)
