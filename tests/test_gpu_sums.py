"""GPU parity of summation elimination switched off (Sec. 5.3): a cache without code
sums gives the same codes, (min, scale) and open block, and decode attention that
rebuilds each partition sum from the packed codes gives bit-identical outputs to the
one that reads the cached sums (and so matches the oracle within 2e-3 max|O|)."""
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


def _twin(hk, gu, case):
    """The same inputs quantized into a cache of the same format without sums."""
    lay = hk.hack_kv_layout_make(case.d, case.H, case.bits, case.pi, case.page_tokens, case.qp_bits,
                                 case.rounding, case.seed, sums_cached=False)
    cache = hk.KVCache(lay, case.num_pages, case.batch, case.table, gu.DEV)
    lens = torch.from_numpy(case.lens.copy()).to(gu.DEV)
    k = torch.from_numpy(np.ascontiguousarray(case.k[:, :, :case.max_len])).to(gu.DEV)
    v = torch.from_numpy(np.ascontiguousarray(case.v[:, :, :case.max_len])).to(gu.DEV)
    hk.hack_quantize(lay, cache, k, v, lens, case.max_len)
    return lay, cache, lens


@pytest.mark.parametrize("bits,pi,group,H,lens,tail,paged,qp", [
    (2, 32, 4, 2, [256, 1, 31, 33, 300], 0, 0, 8),
    (2, 32, 8, 2, [77, 129, 1000], 1, 0, 8),
    (4, 32, 4, 2, [500, 63], 0, 0, 8),
    (2, 64, 2, 2, [64, 65, 700], 0, 256, 8),
    (4, 64, 8, 1, [2048 + 17, 400], 1, 256, 4),
])
def test_decode_without_cached_sums_is_bit_identical(bits, pi, group, H, lens, tail, paged, qp):
    hk, gu = _env()
    gu.announce(f"no sums: bits={bits} pi={pi} G={group} H={H} lens={lens} tail={tail} paged={paged} qp={qp}")
    case = gu.Case(61 + bits + pi + group, len(lens), H, lens, bits, pi, group=group, paged_page=paged,
                   qp_bits=qp).quantize()
    lay0, cache0, lens0 = _twin(hk, gu, case)
    for name in ("k_codes", "k_meta", "v_codes", "v_meta", "v_tail"):
        assert torch.equal(cache0.buffers[name], case.cache.buffers[name]), name
    q = torch.from_numpy(case.q).to(gu.DEV)
    ref = hk.hack_attend_decode(case.layout, case.cache, q, case.lens_dev, case.max_len, tail)
    got = hk.hack_attend_decode(lay0, cache0, q, lens0, case.max_len, tail)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
    oracle = O.attend_decode(case.q, case.oracle_seqs(), H, qp, tail)
    err = gu.rel_err(got.cpu().numpy(), oracle)
    print(f"max|d|/|O|inf = {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("tail", [0, 1])
def test_decode_step_without_cached_sums(tail):
    """Appending tokens (and closing V blocks) into a cache without sums, then attending,
    matches the same steps on a cache with sums, output for output."""
    hk, gu = _env()
    bits, pi, group, H = 2, 32, 4, 2
    lens = [pi - 2, 3 * pi - 1, 5]
    steps = 6
    gu.announce(f"no sums decode_step tail={tail}")
    case = gu.Case(91 + tail, len(lens), H, lens, bits, pi, group=group, spare_tokens=steps).quantize()
    lay0, cache0, lens0 = _twin(hk, gu, case)
    kd = torch.from_numpy(case.k).to(gu.DEV)
    vd = torch.from_numpy(case.v).to(gu.DEV)
    q = torch.from_numpy(case.q).to(gu.DEV)
    cap = case.page_tokens
    ws1 = hk.decode_workspace(case.layout, case.batch, case.Hq, cap)
    ws0 = hk.decode_workspace(lay0, case.batch, case.Hq, cap)
    out1 = torch.empty((case.batch, case.Hq, case.d), dtype=torch.float32, device=gu.DEV)
    out0 = torch.empty_like(out1)
    l1a, l1b = case.lens_dev, torch.zeros_like(case.lens_dev)
    l0a, l0b = lens0, torch.zeros_like(lens0)
    for step in range(steps):
        idx = torch.from_numpy(case.lens + step).long().to(gu.DEV)
        kn = kd[torch.arange(case.batch, device=gu.DEV), :, idx].contiguous()
        vn = vd[torch.arange(case.batch, device=gu.DEV), :, idx].contiguous()
        hk.bind_decode_step(case.layout, case.cache, kn, vn, q, l1a, l1b, cap - 1, tail, out1, ws1)(
            torch.cuda.current_stream())
        hk.bind_decode_step(lay0, cache0, kn, vn, q, l0a, l0b, cap - 1, tail, out0, ws0)(
            torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert torch.equal(out0, out1), step
        l1a, l1b = l1b, l1a
        l0a, l0b = l0b, l0a
