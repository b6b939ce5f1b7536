"""GPU parity of the fused QKV generation (hack_project_qkv, Eq. 1 fused with the
quantize-on-write of Sec. 5.2-5.3) and of the prefill from embeddings against the
oracle.

Where the projection is exact in fp32 and in float64 alike (embeddings and weights
of few significant bits, so every partial sum is representable), both sides round the
same number to fp16: the query heads and every cache byte must be bit-exact.  With
N(0,1)-like values the GPU sums in fp32 and the oracle in float64, so an fp16 result
can differ by one unit in the last place; those cases are bounded instead, and the
prefill output is gated at 2e-3 * max|O| as everywhere else."""
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


def exact_inputs(seed, B, L, hidden, N):
    """Embeddings k/4 and weights j/64 with |k|, |j| <= 8: each product is a multiple of
    2^-8 of magnitude <= 1/4, so any sum over 4096 terms needs at most 19 bits."""
    g = np.random.default_rng(seed)
    E = (g.integers(-8, 9, size=(B, L, hidden)) / 4.0).astype(np.float16)
    W = (g.integers(-8, 9, size=(N, hidden)) / 64.0).astype(np.float16)
    return E, W


def realistic_inputs(seed, B, L, hidden, N):
    from paper_2502_03589_amd import synth
    E = synth.normal_f16(seed, "misc", (B, L, hidden), sub=1)
    W = (synth.normal_f16(seed, "misc", (N, hidden), sub=2).astype(np.float32) / np.sqrt(hidden)).astype(np.float16)
    return E, W


class ProjCase:
    def __init__(self, gu, seed, B, Hkv, G, L, hidden, bits, pi, paged=0, rounding=O.NEAREST_EVEN, exact=True):
        from paper_2502_03589_amd import hack as hk
        from paper_2502_03589_amd import synth
        self.B, self.H, self.G, self.Hq, self.L, self.hidden = B, Hkv, G, Hkv * G, L, hidden
        self.bits, self.pi, self.seed, self.rounding = bits, pi, seed, rounding
        N = (self.Hq + 2 * Hkv) * 128
        self.E, self.W = (exact_inputs if exact else realistic_inputs)(seed, B, L, hidden, N)
        if paged:
            self.page_tokens = paged
            table, pages = synth.page_table(seed, np.full(B, L), paged)
            self.table_np, self.num_pages = table, pages
            self.table = torch.from_numpy(table).to(gu.DEV)
        else:
            self.page_tokens = max(pi, -(-L // pi) * pi)
            self.table_np, self.table, self.num_pages = None, None, B
        self.layout = hk.hack_kv_layout_make(128, Hkv, bits, pi, self.page_tokens, 8, rounding, seed)
        self.cache = hk.KVCache(self.layout, self.num_pages, B, self.table, gu.DEV)
        self.e_dev = torch.from_numpy(self.E).to(gu.DEV)
        self.w_dev = torch.from_numpy(self.W).to(gu.DEV)

    def oracle(self):
        qs, seqs = [], []
        for b in range(self.B):
            Q, K, V = O.project_qkv(self.E[b], self.W, self.Hq, self.H, 128)
            qs.append(Q)
            seqs.append([O.quantize_sequence(K[h], V[h], self.bits, self.pi, self.rounding, self.seed, b, h, self.H)
                         for h in range(self.H)])
        return np.stack(qs), seqs


def _cache_view(gu, pc):
    """The device cache as the oracle's section arrays (gpu_util's reshaping)."""
    class _C:
        pass
    c = _C()
    c.d, c.pi, c.bits, c.H, c.batch = 128, pc.pi, pc.bits, pc.H, pc.B
    c.page_tokens, c.num_pages, c.layout, c.table_np = pc.page_tokens, pc.num_pages, pc.layout, pc.table_np
    c.lens = np.full(pc.B, pc.L)
    torch.cuda.synchronize()
    raw = {n: b.cpu().numpy() for n, b in pc.cache.buffers.items()}
    return c, gu.as_sections(raw, c)


@pytest.mark.parametrize("bits,pi,paged,rounding,L", [
    (2, 32, 0, 0, 300), (4, 64, 0, 0, 300), (2, 16, 256, 0, 300), (4, 128, 0, 0, 129),
    (2, 64, 256, 1, 300), (4, 32, 0, 1, 1),
])
def test_project_bit_exact_where_the_projection_is_exact(bits, pi, paged, rounding, L):
    gu = _gpu()
    from paper_2502_03589_amd import hack as hk
    gu.announce(f"project exact bits={bits} pi={pi} paged={paged} rounding={rounding} L={L}")
    pc = ProjCase(gu, 61 + bits + pi, 2, 2, 4, L, 256, bits, pi, paged, rounding, exact=True)
    q = hk.hack_project_qkv(pc.layout, pc.cache, pc.e_dev, pc.w_dev, pc.Hq)
    Qref, seqs = pc.oracle()
    case, raw = _cache_view(gu, pc)
    assert np.array_equal(q.cpu().numpy().view(np.uint16), Qref.view(np.uint16))
    ref = O.pack_cache(seqs, pc.H, 128, bits, pi, pc.page_tokens, pc.num_pages, pc.table_np, pc.B)
    km, vm, tm = gu.valid_masks(case, include_open_block=True)
    for name, mask in (("k_codes", km), ("k_meta", km), ("k_sums", km), ("v_codes", vm), ("v_meta", vm),
                       ("v_sums", vm), ("v_tail", tm)):
        assert np.array_equal(raw[name][mask], ref[name][mask]), name


@pytest.mark.parametrize("B,Hkv,G,bits,pi,L", [(1, 1, 3, 2, 32, 300), (2, 3, 1, 4, 64, 520)])
def test_project_odd_head_counts_bit_exact(B, Hkv, G, bits, pi, L):
    """Output heads are computed two to a tile: 5 and 9 heads give tiles that mix a query
    and a key head, and a last tile with a single value head (its second half reads
    clamped weight rows and is never stored)."""
    gu = _gpu()
    from paper_2502_03589_amd import hack as hk
    gu.announce(f"project odd heads B={B} Hkv={Hkv} G={G} bits={bits} pi={pi} L={L}")
    pc = ProjCase(gu, 90 + Hkv + G, B, Hkv, G, L, 192, bits, pi, exact=True)
    q = hk.hack_project_qkv(pc.layout, pc.cache, pc.e_dev, pc.w_dev, pc.Hq)
    Qref, seqs = pc.oracle()
    case, raw = _cache_view(gu, pc)
    assert np.array_equal(q.cpu().numpy().view(np.uint16), Qref.view(np.uint16))
    ref = O.pack_cache(seqs, pc.H, 128, bits, pi, pc.page_tokens, pc.num_pages, pc.table_np, pc.B)
    km, vm, tm = gu.valid_masks(case, include_open_block=True)
    for name, mask in (("k_codes", km), ("k_meta", km), ("k_sums", km), ("v_codes", vm), ("v_meta", vm),
                       ("v_sums", vm), ("v_tail", tm)):
        assert np.array_equal(raw[name][mask], ref[name][mask]), name


def _ulps(a, b):
    """|a - b| in fp16 units in the last place (both finite, compared as ordered ints)."""
    ia = a.view(np.int16).astype(np.int32)
    ib = b.view(np.int16).astype(np.int32)
    ia = np.where(ia < 0, -32768 - ia, ia)
    ib = np.where(ib < 0, -32768 - ib, ib)
    return np.abs(ia - ib)


def _within_fp32_sum_bound(got16, E, W, q_heads, kv_heads, tokens=None):
    """Each fp16 query value is the fp32 sum of its `hidden` exact products rounded to
    fp16: |got - exact| <= half an fp16 ulp of the larger of the two + hidden * 2^-24 *
    sum_i |E_i W_i| (the error bound of a recursive fp32 sum; any order is covered).
    Returns the largest ratio of the error to that bound."""
    Ef = np.asarray(E, np.float64)
    if tokens is not None:
        Ef = Ef[np.asarray(tokens)]
    Wf = np.asarray(W, np.float64)[:q_heads * 128]
    exact = Ef @ Wf.T                                         # [n][Hq*128]
    absdot = np.abs(Ef) @ np.abs(Wf).T
    g = got16.astype(np.float64).transpose(1, 0, 2).reshape(exact.shape)
    mag = np.maximum(np.abs(exact), np.abs(g))
    ulp = np.where(mag < 2.0 ** -14, 2.0 ** -24, 2.0 ** (np.floor(np.log2(np.maximum(mag, 2.0 ** -14))) - 10))
    bound = 0.5 * ulp + Ef.shape[1] * 2.0 ** -24 * absdot
    return float(np.max(np.abs(g - exact) / bound))


def test_prefill_from_embeddings_matches_oracle():
    """N(0,1) embeddings, weights of variance 1/hidden: query heads within one fp16 ulp
    of the oracle's (nearly all equal), cache codes equal except where an fp16 K/V value
    fell on the other side of a rounding boundary, and the prefill output of the whole
    path (projection, quantization, attention) within the gate."""
    gu = _gpu()
    from paper_2502_03589_amd import hack as hk
    gu.announce("prefill from embeddings B=1 H=2 G=4 L=700 hidden=1024")
    pc = ProjCase(gu, 77, 1, 2, 4, 700, 1024, 4, 64, exact=False)
    out, q = hk.hack_prefill_from_embeddings(pc.layout, pc.cache, pc.e_dev, pc.w_dev, pc.Hq, True)
    torch.cuda.synchronize()
    Qref, seqs = pc.oracle()
    qn = q.cpu().numpy()
    ul = _ulps(qn, Qref)
    ratio = _within_fp32_sum_bound(qn[0], pc.E[0], pc.W, pc.Hq, pc.H)
    print(f"Q: max {ul.max()} ulp, {np.mean(ul == 0):.4f} equal to the oracle; error / fp32-sum bound <= {ratio:.3f}")
    assert ratio <= 1.0 and np.mean(ul == 0) >= 0.99
    case, raw = _cache_view(gu, pc)
    ref = O.pack_cache(seqs, pc.H, 128, pc.bits, pc.pi, pc.page_tokens, pc.num_pages, None, pc.B)
    km, _, _ = gu.valid_masks(case, include_open_block=True)
    kc_diff = np.mean(raw["k_codes"][km] != ref["k_codes"][km])
    print(f"K code bytes differing: {kc_diff:.4%}")
    assert kc_diff < 0.02
    rows = [(0, h, i) for h in range(pc.Hq) for i in range(0, 700, 7)]
    want = O.attend_prefill(Qref, seqs, pc.H, True, rows=rows)
    got = out.cpu().numpy()
    g = np.stack([got[b, h, i] for b, h, i in rows])
    w = np.stack([want[b, h, i] for b, h, i in rows])
    err = float(np.abs(g - w).max() / np.abs(w).max())
    print(f"sampled rows max|d|/|O|inf = {err:.3e}")
    assert err <= TOL


def test_full_size_projection_sampled():
    """The prefill workload's shapes with a Llama-3-8B-sized hidden dimension (8192
    tokens, 32/8 heads, hidden 4096, 4-bit K/V, partition 64): sampled tokens' query
    heads within one ulp, and their K partitions' codes against the oracle's."""
    gu = _gpu()
    from paper_2502_03589_amd import hack as hk
    gu.announce("full-size projection 8192 x 4096 -> 48 heads (sampled)")
    pc = ProjCase(gu, 1003, 1, 8, 4, 8192, 4096, 4, 64, exact=False)
    q = hk.hack_project_qkv(pc.layout, pc.cache, pc.e_dev, pc.w_dev, pc.Hq)
    torch.cuda.synchronize()
    toks = [0, 1, 127, 128, 4095, 5000, 8190, 8191]
    Q, K, V = O.project_qkv(pc.E[0], pc.W, pc.Hq, pc.H, 128, tokens=toks)
    qg = q.cpu().numpy()[0][:, toks]
    ul = _ulps(qg, Q)
    ratio = _within_fp32_sum_bound(qg, pc.E[0], pc.W, pc.Hq, pc.H, tokens=toks)
    print(f"Q: max {ul.max()} ulp, {np.mean(ul == 0):.4f} equal to the oracle; error / fp32-sum bound <= {ratio:.3f}")
    assert ratio <= 1.0 and np.mean(ul == 0) >= 0.99
    case, raw = _cache_view(gu, pc)
    diff = 0
    for j, t in enumerate(toks):
        for h in range(pc.H):
            sq = O.quantize_sequence(K[h, j:j + 1], V[h, j:j + 1], 4, 64)
            packed = O.pack_codes(sq.k_codes.reshape(1, 2, 64), 4).reshape(-1)
            diff += int(np.sum(raw["k_codes"][0, h, t] != packed))
    print(f"sampled K code bytes differing: {diff} of {len(toks) * pc.H * 64}")
    assert diff <= 0.02 * len(toks) * pc.H * 64
