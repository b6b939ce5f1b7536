"""GPU parity of decode attention with a partition of 128 (Sec. 5.2, 5.3, Eq. 4):
one K partition per token row, V blocks of 128 tokens, on the int8-dot kernel.
Compared with the oracle within 2e-3 max|O| (the same bar as partitions 32 and
64), over ragged lengths that leave open blocks of every kind, several chunks per
sequence, kv groups of 1-8 heads, paged caches, 4-bit Q/P, the three open-block
modes, cached sums on and off (bit-identical outputs) and stochastic Q/P."""
import numpy as np
import pytest
import torch

from oracle import hack_oracle as O

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _env():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2502_03589_amd import hack as hk
    from tests import gpu_util as gu
    return hk, gu


CASES = [
    # bits, group, kv_heads, lens, tail_mode, paged page, Q/P bits
    (2, 4, 2, [256, 1, 127, 129, 600], 0, 0, 8),
    (2, 4, 2, [256, 1, 127, 129, 600], 1, 0, 8),
    (4, 8, 2, [77, 129, 1000], 0, 0, 8),
    (4, 2, 2, [63, 700, 1], 1, 0, 8),
    (2, 1, 3, [128, 383, 2500], 0, 0, 8),
    (2, 4, 2, [0, 50, 5000], 0, 512, 8),
    (4, 6, 1, [2048 + 17, 400], 1, 1024, 8),
    (2, 4, 2, [256, 1, 127, 129, 600], 0, 0, 4),
    (4, 8, 2, [77, 129, 1000], 1, 0, 4),
    (2, 3, 1, [1, 2, 3], 0, 0, 8),
    (4, 5, 1, [128 * 7, 1], 1, 0, 8),
    (2, 7, 2, [512, 513, 1023], 2, 1024, 8),
]


@pytest.mark.parametrize("bits,group,H,lens,tail,paged,qp", CASES)
def test_attend_decode_p128_matches_oracle(bits, group, H, lens, tail, paged, qp):
    hk, gu = _env()
    gu.announce(f"decode p128 bits={bits} G={group} H={H} lens={lens} tail={tail} paged={paged} qp={qp}")
    case = gu.Case(131 + bits + group, len(lens), H, lens, bits, 128, group=group, paged_page=paged,
                   qp_bits=qp).quantize()
    out = hk.hack_attend_decode(case.layout, case.cache, torch.from_numpy(case.q).to(gu.DEV), case.lens_dev,
                                case.max_len, tail)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = O.attend_decode(case.q, case.oracle_seqs(), H, qp, tail)
    err = gu.rel_err(got, ref)
    print(f"max|d|/|O|inf = {err:.3e}")
    assert err <= TOL
    for b, L in enumerate(lens):
        if L == 0:
            assert np.all(got[b] == 0)


@pytest.mark.parametrize("bits,tail", [(2, 0), (4, 1)])
def test_p128_without_cached_sums_is_bit_identical(bits, tail):
    hk, gu = _env()
    lens = [256, 1, 127, 129, 1600]
    gu.announce(f"decode p128 no sums bits={bits} tail={tail}")
    case = gu.Case(141 + bits, len(lens), 2, lens, bits, 128, group=4).quantize()
    lay0 = hk.hack_kv_layout_make(case.d, case.H, bits, 128, case.page_tokens, 8, O.NEAREST_EVEN, case.seed,
                                  sums_cached=False)
    cache0 = hk.KVCache(lay0, case.num_pages, case.batch, None, gu.DEV)
    lens0 = torch.from_numpy(case.lens.copy()).to(gu.DEV)
    k = torch.from_numpy(np.ascontiguousarray(case.k[:, :, :case.max_len])).to(gu.DEV)
    v = torch.from_numpy(np.ascontiguousarray(case.v[:, :, :case.max_len])).to(gu.DEV)
    hk.hack_quantize(lay0, cache0, k, v, lens0, case.max_len)
    q = torch.from_numpy(case.q).to(gu.DEV)
    ref = hk.hack_attend_decode(case.layout, case.cache, q, case.lens_dev, case.max_len, tail)
    got = hk.hack_attend_decode(lay0, cache0, q, lens0, case.max_len, tail)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
    err = gu.rel_err(got.cpu().numpy(), O.attend_decode(case.q, case.oracle_seqs(), 2, 8, tail))
    print(f"max|d|/|O|inf = {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("bits,group,H,lens,tail,qp", [
    (2, 4, 2, [256, 1, 127, 300], 0, 8),
    (4, 8, 1, [77, 1000], 1, 8),
    (2, 4, 1, [500, 129], 0, 4),
])
def test_stochastic_p128_matches_oracle(bits, group, H, lens, tail, qp):
    hk, gu = _env()
    gu.announce(f"stochastic decode p128 bits={bits} G={group} H={H} lens={lens} tail={tail} qp={qp}")
    case = gu.Case(151 + bits, len(lens), H, lens, bits, 128, group=group, rounding=O.STOCHASTIC,
                   qp_bits=qp).quantize()
    out = hk.hack_attend_decode(case.layout, case.cache, torch.from_numpy(case.q).to(gu.DEV), case.lens_dev,
                                case.max_len, tail)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = O.attend_decode(case.q, case.oracle_seqs(), H, qp, tail, stochastic_seed=case.seed)
    err = gu.rel_err(got, ref)
    print(f"max|d|/|O|inf = {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("bits,group,H,lens,tail", [
    (2, 4, 2, [125, 127, 128, 300, 0], 0),
    (2, 4, 2, [125, 127, 128, 300, 0], 1),
    (4, 8, 1, [126, 127, 511], 2),
])
def test_p128_decode_step_equals_append_then_decode(bits, group, H, lens, tail):
    """hack_decode_step at partition 128 writes the same cache bytes and lengths as
    hack_append and returns what hack_attend_decode returns after it, over steps that
    close a block; the end state matches the oracle."""
    hk, gu = _env()
    gu.announce(f"decode step p128 bits={bits} G={group} H={H} lens={lens} tail={tail}")
    steps = 4
    a = gu.Case(161 + bits, len(lens), H, lens, bits, 128, group=group, spare_tokens=steps).quantize()
    b = gu.Case(161 + bits, len(lens), H, lens, bits, 128, group=group, spare_tokens=steps).quantize()
    lens_in = b.lens_dev.clone()
    lens_out = torch.zeros_like(lens_in)
    for step in range(steps):
        cur = a.lens_dev.cpu().numpy()
        kn = torch.from_numpy(np.stack([a.k[s, :, cur[s]] for s in range(a.batch)])).to(gu.DEV)
        vn = torch.from_numpy(np.stack([a.v[s, :, cur[s]] for s in range(a.batch)])).to(gu.DEV)
        q = torch.from_numpy(gu.synth.normal_f16(a.seed + 1000 + step, "q", (a.batch, a.Hq, a.d))).to(gu.DEV)
        ml = int(cur.max())
        hk.hack_append(a.layout, a.cache, kn, vn, a.lens_dev, ml, tail)
        ref_out = hk.hack_attend_decode(a.layout, a.cache, q, a.lens_dev, ml + 1, tail)
        got = hk.hack_decode_step(b.layout, b.cache, kn, vn, q, lens_in, lens_out, ml, tail)
        torch.cuda.synchronize()
        assert torch.equal(lens_out, a.lens_dev)
        assert torch.equal(got, ref_out)
        lens_in, lens_out = lens_out, lens_in
    ra, rb = a.sections(), b.sections()
    for name in ra:
        assert np.array_equal(ra[name], rb[name]), name
    a.lens = a.lens_dev.cpu().numpy()
    if tail == O.TAIL_DEQUANT:  # the open block is the result of requantizing appends
        seqs = [[None] * H for _ in lens]
        for s_, L0 in enumerate(lens):
            for h in range(H):
                sq = O.quantize_sequence(a.k[s_, h, :L0], a.v[s_, h, :L0], bits, 128)
                for t in range(L0, L0 + steps):
                    sq = O.append_requantizing(sq, a.k[s_, h, t], a.v[s_, h, t], bits)
                seqs[s_][h] = sq
    else:
        seqs = a.oracle_seqs()
    qlast = gu.synth.normal_f16(a.seed + 1000 + steps - 1, "q", (a.batch, a.Hq, a.d))
    err = gu.rel_err(got.cpu().numpy(), O.attend_decode(qlast, seqs, H, 8, tail))
    print(f"max|d|/|O|inf vs oracle after {steps} steps = {err:.3e}")
    assert err <= TOL


def test_p128_qk_export_reports_unsupported():
    hk, gu = _env()
    gu.announce("p128 unsupported entry points")
    case = gu.Case(171, 2, 2, [300, 129], 2, 128, group=4).quantize()
    with pytest.raises(hk.HackError) as e:
        hk.hack_debug_qk_products(case.layout, case.cache, torch.from_numpy(case.q).to(gu.DEV), case.lens_dev,
                                  case.max_len)
    assert e.value.status == 2


@pytest.mark.parametrize("bits", [2, 4])
def test_full_size_p128_decode_sampled(bits):
    """decode_llama8b_l4096's shapes at partition 128 (batch 16, 32/8 heads, 4096
    tokens, x10 outliers on 4 K channels), in the launch configuration the partition
    sweep times: outputs of sampled rows against the oracle, and the split-K merge
    over the full chunk count."""
    hk, gu = _env()
    gu.announce(f"full-size p128 decode bits={bits} (sampled)")
    case = gu.Case(1128 + bits, 16, 8, [4096] * 16, bits, 128, group=4, outliers=4).quantize()
    out = hk.hack_attend_decode(case.layout, case.cache, torch.from_numpy(case.q).to(gu.DEV), case.lens_dev, 4096)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    pairs = {(0, 0), (7, 4), (15, 7)}
    seqs = case.oracle_seqs(pairs)
    rows = [(b, h * 4 + g) for (b, h) in pairs for g in range(4)]
    ref = O.attend_decode(case.q, seqs, 8, rows=rows)
    got_rows = np.stack([got[b, h] for b, h in rows])
    ref_rows = np.stack([ref[b, h] for b, h in rows])
    err = float(np.abs(got_rows - ref_rows).max() / np.abs(ref_rows).max())
    print(f"sampled rows max|d|/|O|inf = {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("bits,tail", [(2, 0), (4, 1)])
def test_p128_long_context_sampled(bits, tail):
    """Partition 128 at the long-context size: batch 2, 8/2 heads, 131072 + 77 tokens
    (chunks of 64 spans, an open block of 77 tokens), one sampled pair per sequence."""
    hk, gu = _env()
    L = 131072 + 77
    gu.announce(f"long-context p128 bits={bits} tail={tail} L={L}")
    case = gu.Case(1300 + bits, 2, 2, [L, L - 200], bits, 128, group=4).quantize()
    out = hk.hack_attend_decode(case.layout, case.cache, torch.from_numpy(case.q).to(gu.DEV), case.lens_dev,
                                case.max_len, tail)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    pairs = {(0, 1), (1, 0)}
    seqs = case.oracle_seqs(pairs)
    rows = [(b, h * 4 + g) for (b, h) in pairs for g in range(4)]
    ref = O.attend_decode(case.q, seqs, 2, 8, tail, rows=rows)
    got_rows = np.stack([got[b, h] for b, h in rows])
    ref_rows = np.stack([ref[b, h] for b, h in rows])
    err = float(np.abs(got_rows - ref_rows).max() / np.abs(ref_rows).max())
    print(f"sampled rows max|d|/|O|inf = {err:.3e}")
    assert err <= TOL


def test_p128_split_merge_sees_each_calls_records():
    """Back-to-back partition-128 decode calls on one workspace with alternating
    queries and several chunks per sequence: the merging workgroup must read the
    current call's records, and every call leaves the counters at zero."""
    hk, gu = _env()
    gu.announce("p128 split-K merge over repeated calls")
    case = gu.Case(1808, 4, 2, [2000, 1999, 1500, 2048], 2, 128, group=4).quantize()
    qa = case.q
    qb = gu.synth.normal_f16(1809, "q", qa.shape)
    seqs = case.oracle_seqs()
    refs = [O.attend_decode(q, seqs, case.H, 8, 0) for q in (qa, qb)]
    qd = [torch.from_numpy(q).to(gu.DEV) for q in (qa, qb)]
    ws = hk.decode_workspace(case.layout, case.batch, case.Hq, case.max_len)
    outs = [torch.empty((case.batch, case.Hq, case.d), dtype=torch.float32, device=gu.DEV) for _ in range(40)]
    for it, out in enumerate(outs):  # queued back to back, no host synchronization in between
        hk.hack_attend_decode(case.layout, case.cache, qd[it % 2], case.lens_dev, case.max_len, out=out, workspace=ws)
    torch.cuda.synchronize()
    for it, out in enumerate(outs):
        err = gu.rel_err(out.cpu().numpy(), refs[it % 2])
        assert err <= TOL, f"call {it}: {err:.3e}"
    nbytes = hk.hack_decode_workspace_bytes(case.layout, case.batch, case.Hq, case.max_len)
    raw = ws.view(torch.uint8)[:nbytes].cpu().numpy()
    # the counters come first (one int32 per (sequence, kv head, four-head group)); all are back at zero
    B, H, G = case.batch, case.H, case.G
    assert not np.any(raw[:B * H * ((G + 3) // 4) * 4])


def test_p128_decode_step_paged():
    """hack_decode_step at partition 128 on a paged cache (512-token pages): same bytes
    and outputs as append then decode."""
    hk, gu = _env()
    lens = [510, 511, 1023, 40]
    gu.announce(f"decode step p128 paged lens={lens}")
    a = gu.Case(1811, len(lens), 2, lens, 2, 128, group=4, paged_page=512, spare_tokens=3).quantize()
    b = gu.Case(1811, len(lens), 2, lens, 2, 128, group=4, paged_page=512, spare_tokens=3).quantize()
    lens_in, lens_out = b.lens_dev.clone(), torch.zeros_like(b.lens_dev)
    for step in range(3):
        cur = a.lens_dev.cpu().numpy()
        kn = torch.from_numpy(np.stack([a.k[s, :, cur[s]] for s in range(a.batch)])).to(gu.DEV)
        vn = torch.from_numpy(np.stack([a.v[s, :, cur[s]] for s in range(a.batch)])).to(gu.DEV)
        q = torch.from_numpy(gu.synth.normal_f16(1900 + step, "q", (a.batch, a.Hq, a.d))).to(gu.DEV)
        ml = int(cur.max())
        hk.hack_append(a.layout, a.cache, kn, vn, a.lens_dev, ml, 1)
        ref_out = hk.hack_attend_decode(a.layout, a.cache, q, a.lens_dev, ml + 1, 1)
        got = hk.hack_decode_step(b.layout, b.cache, kn, vn, q, lens_in, lens_out, ml, 1)
        torch.cuda.synchronize()
        assert torch.equal(lens_out, a.lens_dev)
        assert torch.equal(got, ref_out)
        lens_in, lens_out = lens_out, lens_in
    ra, rb = a.sections(), b.sections()
    for name in ra:
        assert np.array_equal(ra[name], rb[name]), name
