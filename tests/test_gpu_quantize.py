"""GPU parity of quantize-on-write (hack_quantize, hack_append) against the oracle:
every stored byte (codes, fp16 min/scale, sums, fp16 open block) must match."""
import numpy as np
import pytest
import torch

from oracle import hack_oracle as O

pytestmark = pytest.mark.gpu


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    return gpu_util


@pytest.mark.parametrize("bits,pi,paged,rounding", [
    (2, 32, 0, 0), (4, 32, 0, 0), (2, 64, 0, 0), (4, 64, 0, 0), (2, 128, 0, 0), (4, 16, 0, 0),
    (2, 32, 64, 0), (4, 64, 128, 0), (2, 32, 0, 1), (4, 64, 64, 1),
])
def test_quantize_bytes_bit_exact(bits, pi, paged, rounding):
    gu = _gpu()
    lens = [1, pi - 1, pi, pi + 1, 3 * pi + 7, 0]
    gu.announce(f"quantize bits={bits} pi={pi} paged={paged} rounding={rounding} lens={lens}")
    case = gu.Case(11 + bits + pi, len(lens), 2, lens, bits, pi, paged_page=paged, rounding=rounding).quantize()
    got = gu.as_sections(case.sections(), case)
    ref = case.oracle_bytes(case.oracle_seqs())
    for name in ref:
        assert np.array_equal(got[name], ref[name]), name


def test_quantize_outlier_channels_bit_exact():
    gu = _gpu()
    gu.announce("quantize with x10 outlier K channels")
    case = gu.Case(1002, 2, 2, [300, 129], 2, 32, outliers=4).quantize()
    got = gu.as_sections(case.sections(), case)
    ref = case.oracle_bytes(case.oracle_seqs())
    for name in ref:
        assert np.array_equal(got[name], ref[name]), name


@pytest.mark.parametrize("tail_mode,bits,pi,paged", [(0, 2, 32, 0), (1, 2, 32, 0), (0, 4, 64, 128), (1, 4, 32, 64)])
def test_append_equals_quantize_of_longer_prefix(tail_mode, bits, pi, paged):
    """Appending tokens one at a time produces the bytes a fresh quantize of the longer
    sequence produces (K rows, full V blocks, fp16 open block; the open block's codes
    too in REQUANT mode)."""
    gu = _gpu()
    lens = [pi - 3, 2 * pi - 1, 5, 3 * pi]
    steps = pi + 4
    gu.announce(f"append tail_mode={tail_mode} bits={bits} pi={pi} paged={paged} steps={steps}")
    case = gu.Case(77 + tail_mode, len(lens), 2, lens, bits, pi, paged_page=paged, spare_tokens=steps).quantize()
    for step in range(steps):
        case.append(step, tail_mode)
    assert np.array_equal(case.lens_dev.cpu().numpy(), np.asarray(lens) + steps)
    got = gu.as_sections(case.sections(), case)
    ref = case.oracle_bytes(case.oracle_seqs())
    km, vm, tm = gu.valid_masks(case, include_open_block=(tail_mode == O.TAIL_REQUANT))
    for name in ("k_codes", "k_meta", "k_sums"):
        assert np.array_equal(got[name][km], ref[name][km]), name
    for name in ("v_codes", "v_meta", "v_sums"):
        assert np.array_equal(got[name][vm], ref[name][vm]), name
    assert np.array_equal(got["v_tail"][tm], ref["v_tail"][tm])


@pytest.mark.parametrize("bits,pi,paged", [(2, 32, 0), (4, 64, 128), (2, 16, 64), (4, 32, 128)])
def test_append_requantizing_open_block_bit_exact(bits, pi, paged):
    """TAIL_DEQUANT: every append dequantizes the open V block's codes to fp16, adds the
    new value and quantizes the block again; the cache after a run of appends (closing
    a block on the way) equals the oracle's chain of requantizing appends byte for
    byte, and decode attention over it matches the oracle."""
    gu = _gpu()
    from paper_2502_03589_amd import hack as hk
    lens = [pi - 3, 2 * pi - 1, 5, 3 * pi]
    steps = pi + 4
    H = 2
    gu.announce(f"requantizing append bits={bits} pi={pi} paged={paged} steps={steps}")
    case = gu.Case(88 + bits, len(lens), H, lens, bits, pi, paged_page=paged, spare_tokens=steps).quantize()
    for step in range(steps):
        case.append(step, O.TAIL_DEQUANT)
    got = gu.as_sections(case.sections(), case)
    seqs = []
    for b, L0 in enumerate(lens):
        row = []
        for h in range(H):
            sq = O.quantize_sequence(case.k[b, h, :L0], case.v[b, h, :L0], bits, pi)
            for t in range(L0, L0 + steps):
                sq = O.append_requantizing(sq, case.k[b, h, t], case.v[b, h, t], bits)
            row.append(sq)
        seqs.append(row)
    ref = case.oracle_bytes(seqs)
    km, vm, _ = gu.valid_masks(case, include_open_block=True)
    for name in ("k_codes", "k_meta", "k_sums"):
        assert np.array_equal(got[name][km], ref[name][km]), name
    for name in ("v_codes", "v_meta", "v_sums"):
        assert np.array_equal(got[name][vm], ref[name][vm]), name
    # the attention kernels take partitions of 32 and 64 and pages that hold whole spans
    if pi % 32 == 0 and (paged == 0 or paged % (4 * pi) == 0):
        out = hk.hack_attend_decode(case.layout, case.cache, torch.from_numpy(case.q).to(gu.DEV), case.lens_dev,
                                    case.max_len, O.TAIL_DEQUANT)
        refo = O.attend_decode(case.q, seqs, H, 8, O.TAIL_DEQUANT)
        err = gu.rel_err(out.cpu().numpy(), refo)
        print(f"max|d|/|O|inf = {err:.3e}")
        assert err <= 2e-3
