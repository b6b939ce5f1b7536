"""GPU parity of prefill attention (hack_attend_prefill) against the oracle: the
output within max|d| <= 2e-3 * max|O| over the call (P codes come from the GPU's
own exp, so a code may flip at a rounding boundary)."""
import numpy as np
import pytest
import torch

from oracle import hack_oracle as O

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    return gpu_util


def _run_prefill(gu, case, causal):
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth
    L = case.max_len
    Q = synth.normal_f16(case.seed, "q", (case.batch, case.Hq, L, case.d), sub=7)
    out = hk.hack_attend_prefill(case.layout, case.cache, torch.from_numpy(Q).to(gu.DEV), causal)
    torch.cuda.synchronize()
    return Q, out.cpu().numpy()


CASES = [
    # bits, pi, group, kv_heads, L, causal, paged page, Q/P bits
    (4, 64, 4, 2, 200, True, 0, 8),
    (4, 64, 4, 2, 200, False, 0, 8),
    (2, 32, 4, 2, 131, True, 0, 8),
    (2, 64, 8, 1, 96, True, 0, 8),
    (4, 32, 1, 2, 33, True, 0, 8),
    (2, 32, 2, 1, 1, True, 0, 8),
    (4, 64, 4, 1, 64, True, 128, 8),
    (2, 32, 4, 1, 300, False, 64, 8),
    (4, 64, 4, 2, 200, True, 0, 4),
    (2, 32, 8, 1, 131, False, 0, 4),
    # partition 128: one K partition per token, 128-token V blocks, u16 code sums
    (2, 128, 4, 2, 300, True, 0, 8),
    (4, 128, 4, 1, 129, False, 0, 8),
    (4, 128, 8, 1, 200, True, 256, 8),
    (2, 128, 2, 2, 127, True, 0, 4),
]


@pytest.mark.parametrize("bits,pi,group,H,L,causal,paged,qp", CASES)
def test_attend_prefill_matches_oracle(bits, pi, group, H, L, causal, paged, qp):
    gu = _gpu()
    gu.announce(f"prefill bits={bits} pi={pi} G={group} H={H} L={L} causal={causal} paged={paged} qp={qp}")
    case = gu.Case(300 + bits + pi + L, 1 if L > 150 else 2, H, [L] * (1 if L > 150 else 2), bits, pi,
                   group=group, paged_page=paged, qp_bits=qp).quantize()
    Q, got = _run_prefill(gu, case, causal)
    ref = O.attend_prefill(Q, case.oracle_seqs(), H, causal=causal, qp_bits=qp)
    err = gu.rel_err(got, ref)
    print(f"max|d|/|O|inf = {err:.3e}")
    assert err <= TOL


def test_prefill_full_size_sampled_rows():
    """Batch 1, 32/8 heads, 8192 tokens, 4-bit K/V, partition 64, causal: sampled rows."""
    gu = _gpu()
    gu.announce("full-size prefill_l8192 (sampled rows)")
    L = 8192
    case = gu.Case(1003, 1, 8, [L], 4, 64, group=4).quantize()
    Q, got = _run_prefill(gu, case, True)
    rows = [(0, 0, 0), (0, 1, 63), (0, 2, 64), (0, 5, 1000), (0, 9, 4095), (0, 17, 4096),
            (0, 26, 7000), (0, 31, L - 1), (0, 12, L - 64), (0, 3, 2047)]
    pairs = {(b, h // 4) for b, h, _ in rows}
    seqs = case.oracle_seqs(pairs)
    ref = O.attend_prefill(Q, seqs, 8, causal=True, rows=rows)
    g = np.stack([got[b, h, i] for b, h, i in rows])
    r = np.stack([ref[b, h, i] for b, h, i in rows])
    err = float(np.abs(g - r).max() / np.abs(r).max())
    # context only (not a gate): the same rows against unquantized float64 attention
    exact = np.stack([O.attention_unquantized(Q[b, h, i], case.k[b, h // 4], case.v[b, h // 4], causal_row=i)
                      for b, h, i in rows])
    ctx = float(np.abs(g - exact).max() / np.abs(exact).max())
    print(f"sampled rows max|d|/|O|inf = {err:.3e} vs the oracle; {ctx:.3e} vs unquantized attention")
    assert err <= TOL


def test_prefill_last_row_matches_decode():
    """The last causal prefill row and a decode step with the same query agree."""
    gu = _gpu()
    from paper_2502_03589_amd import hack as hk
    gu.announce("prefill last row vs decode")
    L = 160
    case = gu.Case(77, 1, 2, [L], 2, 32, group=4).quantize()
    Q, got = _run_prefill(gu, case, True)
    q_last = np.ascontiguousarray(Q[:, :, L - 1, :])
    dec = hk.hack_attend_decode(case.layout, case.cache, torch.from_numpy(q_last).to(gu.DEV), case.lens_dev, L)
    torch.cuda.synchronize()
    d = dec.cpu().numpy()
    assert np.abs(d - got[:, :, L - 1, :]).max() <= TOL * np.abs(d).max()


@pytest.mark.parametrize("bits,pi,group,H,L,causal,qp", [(4, 64, 4, 2, 200, True, 8), (2, 32, 8, 1, 131, False, 4)])
def test_stochastic_prefill_matches_oracle(bits, pi, group, H, L, causal, qp):
    """Stochastic rounding of K/V, Q and P in prefill against the oracle drawing the same
    SplitMix64 thresholds."""
    gu = _gpu()
    gu.announce(f"stochastic prefill bits={bits} pi={pi} G={group} H={H} L={L} causal={causal} qp={qp}")
    case = gu.Case(500 + bits + pi + L, 1, H, [L], bits, pi, group=group, rounding=O.STOCHASTIC,
                   qp_bits=qp).quantize()
    Q, got = _run_prefill(gu, case, causal)
    ref = O.attend_prefill(Q, case.oracle_seqs(), H, causal=causal, qp_bits=qp, stochastic_seed=case.seed)
    err = gu.rel_err(got, ref)
    print(f"max|d|/|O|inf = {err:.3e}")
    assert err <= TOL
