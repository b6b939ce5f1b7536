"""Plain CPU oracle for HACK's quantized attention (arXiv 2502.03589).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import or call this module; the product path
(the HIP library and its Python binding) never does.  It shares no code with
the HIP path: the only thing both sides consume is the seeded input arrays.

What it computes (citations are to the paper):
  * asymmetric per-partition b-bit quantization: min, scale = (max-min)/(2^b-1),
    code = round((x-min)/scale)                          (Sec. 5.2, quantizer definition)
  * the homomorphic product of two quantized partitions (Eq. 4) and its sum
    over several partitions along the inner dimension     (Sec. 5.2, Eq. 4 and the block sum after it)
  * attention O = softmax(Q K^T / sqrt(d_h)) V           (Sec. 4, Eq. 2 and Eq. 3)
    with Q quantized to 8 bits, K/V to b bits along the contraction
    dimension, P quantized to 8 bits per V block, and both products done by
    Eq. 4 using the cached code sums                       (Sec. 5.3, summation elimination)
  * QKV generation Q = E W_Q, K = E W_K, V = E W_V from the prompt's embeddings
    (Sec. 4, Eq. 1), in float64 rounded to fp16, in front of the quantizer
  * the open (last, partial) block of V kept in fp16 and multiplied
    unquantized (requantization elimination, Sec. 5.3), or re-quantized from its
    fp16 originals with n = T elements (the re-quantizing alternative).

Precision: the quantizer of stored K/V and of Q uses float32 operations in a
fixed order (so the codes are single-valued); every product and correction is
int64 / float64.  P is quantized in float64.

Readings where the paper is silent or garbled:
  R1  bits b general: scale = (max-min)/(2^b-1) (the text writes 2^2-1).
  R2  stored scale is the float32 scale rounded *up* to fp16 so that
      (max-min)/s <= 2^b-1; min is stored exactly (it is an input value).
  R3  arithmetic order: s32 = fl(fl(max-min)/Q); r = fl(1/s); t = fl(fl(x-min)*r).
  R4  rounding: nearest-even by default; stochastic rounding rounds up with
      probability frac(t), with thresholds from SplitMix64 (Steele, Lea and
      Flood, 2014) so both sides draw identical numbers.
  R5  a constant partition (s == 0) has all codes 0.
  R6  packing: b-bit codes LSB-first in order of the partition's elements.
  R7  P is the normalized softmax row, quantized per V block of the row; in
      causal attention the masked zeros inside a block are quantized like any
      other element.
  R8  grouped-query attention: q head h uses kv head h // (H_q / H_kv).
  R9  output is float32.
  R15 the requantizing alternative to requantization elimination (Sec. 5.3): the
      open V block keeps only codes; an append dequantizes them to fp16,
      x_hat = fp16(fl(fl(s*c) + m)), adds the new value and quantizes the block again
      with n = T + 1 (so the error of every earlier requantization is kept).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

NEAREST_EVEN = 0
STOCHASTIC = 1
TAIL_FP16 = 0
TAIL_REQUANT = 1
TAIL_DEQUANT = 2
STREAM_K = 1
STREAM_V = 2
STREAM_Q = 3
STREAM_P = 4

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_MIX1 = np.uint64(0xBF58476D1CE4E5B9)
_MIX2 = np.uint64(0x94D049BB133111EB)


# ----------------------------------------------------------------------------
# Random thresholds for stochastic rounding (reading R4)
# ----------------------------------------------------------------------------
def splitmix64(x) -> np.ndarray:
    """SplitMix64 output for state x (Steele, Lea and Flood, OOPSLA 2014):
    z = x + golden; z = (z ^ z>>30) * C1; z = (z ^ z>>27) * C2; return z ^ z>>31."""
    z = np.asarray(x, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = z + _GOLDEN
        z = (z ^ (z >> np.uint64(30))) * _MIX1
        z = (z ^ (z >> np.uint64(27))) * _MIX2
    return z ^ (z >> np.uint64(31))


def element_index(seq: int, kv_heads: int, head: int, token, channel, head_dim: int):
    """Canonical index of a stored K/V element: ((seq*H_kv + head) * 2^32 + token) * d + channel."""
    base = np.uint64((seq * kv_heads + head)) << np.uint64(32)
    with np.errstate(over="ignore"):
        return (base + np.asarray(token, dtype=np.uint64)) * np.uint64(head_dim) + np.asarray(channel, dtype=np.uint64)


def stochastic_threshold(seed: int, stream: int, idx) -> np.ndarray:
    """u = (SplitMix64(seed ^ (stream << 56) ^ idx) >> 40) * 2^-24, a float32 in [0, 1)."""
    key = np.uint64(seed) ^ (np.uint64(stream) << np.uint64(56))
    h = splitmix64(np.asarray(idx, dtype=np.uint64) ^ key)
    return (h >> np.uint64(40)).astype(np.float32) * np.float32(2.0 ** -24)


def qp_index(seq: int, q_heads: int, head: int, row, col):
    """Canonical index of a transient Q or P element (reading R4): query head `head` of
    sequence `seq`, query row `row` (0 in decode), column `col` (channel of Q, key token
    of P): ((seq*H_q + head) * 2^20 + row) * 2^24 + col."""
    with np.errstate(over="ignore"):
        base = (np.uint64(seq * q_heads + head) << np.uint64(20)) + np.asarray(row, dtype=np.uint64)
        return (base << np.uint64(24)) + np.asarray(col, dtype=np.uint64)


@dataclasses.dataclass
class QPStochastic:
    """Stochastic rounding of the Q and P codes of one query row (reading R4): the
    thresholds of stream STREAM_Q (Q channels) and STREAM_P (P key tokens)."""
    seed: int
    seq: int
    q_heads: int
    head: int
    row: int = 0

    def u(self, stream: int, cols) -> np.ndarray:
        return stochastic_threshold(self.seed, stream, qp_index(self.seq, self.q_heads, self.head, self.row, cols))


# ----------------------------------------------------------------------------
# Quantizer of one partition (Sec. 5.2; readings R1-R5)
# ----------------------------------------------------------------------------
def round_up_to_f16(s32):
    """Smallest fp16 value >= s32 (s32 >= 0), returned as float32 (reading R2)."""
    s32 = np.asarray(s32, np.float32)
    h = s32.astype(np.float16)
    bump = h.astype(np.float32) < s32
    h = np.where(bump, np.nextafter(h, np.float16(np.inf)), h)
    return h.astype(np.float32)


def quantize_partition(x, bits: int, meta: str = "f16", rounding: int = NEAREST_EVEN, u=None):
    """Quantize partitions (Sec. 5.2): each row along the last axis of x is one partition.

    meta='f16' : stored K/V (float32 arithmetic, scale rounded up to fp16)
    meta='f32' : transient Q (float32 arithmetic, float32 scale)
    meta='f64' : transient P (float64 arithmetic)
    Per partition: m = min, s = (max - m) / (2^b - 1), r = 1/s, t = (x - m) r,
    code = min(2^b - 1, round(t)); a partition with s == 0 has all codes 0.
    Returns (codes int64 [..., n], minimum [...], scale [...], sum of codes int64 [...])."""
    qmax = (1 << bits) - 1
    ft = np.float64 if meta == "f64" else np.float32
    xf = np.asarray(x).astype(ft)
    lo = xf.min(axis=-1, keepdims=True)
    hi = xf.max(axis=-1, keepdims=True)
    s = ((hi - lo).astype(ft) / ft(qmax)).astype(ft)
    if meta == "f16":
        s = round_up_to_f16(s)
    zero = s == 0
    r = (ft(1.0) / np.where(zero, ft(1.0), s)).astype(ft)
    t = ((xf - lo).astype(ft) * r).astype(ft)
    if rounding == NEAREST_EVEN:
        c = np.rint(t)
    else:
        fl = np.floor(t)
        c = fl + (np.asarray(u) < (t - fl))
    c = np.minimum(c, qmax).astype(np.int64)
    c = np.where(zero, 0, c)
    return c, lo[..., 0], s[..., 0], c.sum(axis=-1)


def sum_bytes(bits: int, partition: int) -> int:
    """Storage of a cached code sum: b + ceil(log2 Pi) bits, rounded to 1 or 2 bytes (Sec. 5.3, Sec. 6)."""
    need = bits + math.ceil(math.log2(partition))
    return 1 if need <= 8 else 2


def pack_codes(codes, bits: int) -> np.ndarray:
    """Pack b-bit codes LSB-first in element order along the last axis (reading R6):
    element e goes to bits [(e*b) mod 8, ...) of byte floor(e*b/8)."""
    codes = np.asarray(codes, dtype=np.int64)
    per = 8 // bits
    n = codes.shape[-1]
    shifted = codes << ((np.arange(n) % per) * bits)
    grouped = shifted.reshape(codes.shape[:-1] + (n // per, per))
    return grouped.sum(axis=-1).astype(np.uint8)   # fields are disjoint, so sum == bitwise or


def unpack_codes(data, bits: int) -> np.ndarray:
    """Inverse of pack_codes along the last axis."""
    data = np.asarray(data, dtype=np.int64)
    per = 8 // bits
    fields = (data[..., None] >> (np.arange(per) * bits)) & ((1 << bits) - 1)
    return fields.reshape(data.shape[:-1] + (data.shape[-1] * per,))


# ----------------------------------------------------------------------------
# Homomorphic product (Eq. 4) and multi-partition sum
# ----------------------------------------------------------------------------
def hq_partition(a_codes, m_a, s_a, b_codes, m_b, s_b):
    """One partition of n aligned elements (Eq. 4):
    sum_z a_z b_z ~= s_a s_b sum a'b' + s_a m_b sum a' + m_a s_b sum b' + n m_a m_b.
    Returns (integer product sum a'b', float64 estimate)."""
    a = np.asarray(a_codes, dtype=np.int64)
    b = np.asarray(b_codes, dtype=np.int64)
    n = a.shape[0]
    prod = int(np.dot(a, b))
    sa = int(a.sum())
    sb = int(b.sum())
    m_a = float(m_a); s_a = float(s_a); m_b = float(m_b); s_b = float(s_b)
    est = s_a * s_b * prod + s_a * m_b * sa + m_a * s_b * sb + n * m_a * m_b
    return prod, est


def hq_matmul(a_codes, m_a, s_a, b_codes, m_b, s_b, partition: int):
    """C = A B with A (M x Z) partitioned along rows' Z and B (Z x N) along columns' Z
    into partitions of `partition` elements; each block by Eq. 4, then summed (Sec. 5.2).
    m_a, s_a: [M][Z/partition]; m_b, s_b: [Z/partition][N].  Returns (C' int64 [M][N][parts], C fp64)."""
    A = np.asarray(a_codes, dtype=np.int64)
    B = np.asarray(b_codes, dtype=np.int64)
    M, Z = A.shape
    N = B.shape[1]
    parts = Z // partition
    prods = np.zeros((M, N, parts), np.int64)
    C = np.zeros((M, N), np.float64)
    for p in range(parts):
        sl = slice(p * partition, (p + 1) * partition)
        Ap, Bp = A[:, sl], B[sl, :]
        prod = Ap @ Bp
        sa = Ap.sum(axis=1)[:, None]
        sb = Bp.sum(axis=0)[None, :]
        ma = np.asarray(m_a, np.float64)[:, p][:, None]
        sa_ = np.asarray(s_a, np.float64)[:, p][:, None]
        mb = np.asarray(m_b, np.float64)[p, :][None, :]
        sb_ = np.asarray(s_b, np.float64)[p, :][None, :]
        prods[:, :, p] = prod
        C += sa_ * sb_ * prod + sa_ * mb * sa + ma * sb_ * sb + partition * ma * mb
    return prods, C


# ----------------------------------------------------------------------------
# Quantized KV of one (sequence, kv head)
# ----------------------------------------------------------------------------
@dataclasses.dataclass
class SeqKV:
    """Quantized K/V of one sequence and one kv head.

    K: each token's d values in d/Pi partitions along the head dimension.
    V: each channel's values in Pi-token blocks along the sequence; the open
       block (T = L mod Pi tokens) is kept in fp16 and also re-quantized with n=T."""
    length: int
    partition: int
    k_codes: np.ndarray   # int64 [L][d]
    k_min: np.ndarray     # float64 (fp16 values) [L][P]
    k_scale: np.ndarray   # [L][P]
    k_sum: np.ndarray     # int64 [L][P]
    v_codes: np.ndarray   # int64 [NB][Pi][d]   (NB = F + (T > 0))
    v_min: np.ndarray     # [NB][d]
    v_scale: np.ndarray   # [NB][d]
    v_sum: np.ndarray     # int64 [NB][d]
    v_count: np.ndarray   # int64 [NB]  valid tokens per block (Pi, or T for the open block)
    v_tail: np.ndarray    # float16 [T][d]

    @property
    def full_blocks(self) -> int:
        return self.length // self.partition

    @property
    def tail_tokens(self) -> int:
        return self.length - self.full_blocks * self.partition


def quantize_sequence(k, v, bits: int, partition: int, rounding: int = NEAREST_EVEN,
                      seed: int = 0, seq: int = 0, head: int = 0, kv_heads: int = 1) -> SeqKV:
    """Quantize one sequence's K [L][d] and V [L][d] (fp16) as the paper lays them out:
    K partitions along d (Sec. 5.3, QK^T partitioning), V blocks of Pi tokens along
    the sequence per channel (Sec. 5.3, PV partitioning); the open V block stays fp16
    (requantization elimination, Sec. 5.3) and is also quantized with n = T."""
    k = np.asarray(k, np.float16)
    v = np.asarray(v, np.float16)
    L, d = k.shape
    Pi = partition
    P = d // Pi
    # K: partition p of token t holds channels [p*Pi, (p+1)*Pi)
    uk = None
    if rounding == STOCHASTIC:
        tok = np.arange(L)[:, None, None]
        ch = np.arange(d).reshape(1, P, Pi)
        uk = stochastic_threshold(seed, STREAM_K, element_index(seq, kv_heads, head, tok, ch, d))
    kc, km, ks, ksum = quantize_partition(k.reshape(L, P, Pi), bits, "f16", rounding, uk)
    F = L // Pi
    T = L - F * Pi
    NB = F + (1 if T > 0 else 0)
    vc = np.zeros((NB, Pi, d), np.int64)
    vm = np.zeros((NB, d)); vs = np.zeros((NB, d)); vsum = np.zeros((NB, d), np.int64)
    vcount = np.zeros(NB, np.int64)
    # V: block blk, channel c holds tokens [blk*Pi, blk*Pi + n) of channel c
    for blk in range(NB):
        n = Pi if blk < F else T
        toks = np.arange(blk * Pi, blk * Pi + n)
        uv = None
        if rounding == STOCHASTIC:
            uv = stochastic_threshold(seed, STREAM_V,
                                      element_index(seq, kv_heads, head, toks[None, :], np.arange(d)[:, None], d))
        c, m, s_, tot = quantize_partition(v[toks, :].T, bits, "f16", rounding, uv)   # [d][n]
        vc[blk, :n, :] = c.T
        vm[blk] = m; vs[blk] = s_; vsum[blk] = tot
        vcount[blk] = n
    return SeqKV(L, Pi, kc.reshape(L, d), km.astype(np.float64), ks.astype(np.float64), ksum,
                 vc, vm, vs, vsum, vcount, v[F * Pi:L].copy())


def dequantize_to_f16(codes, m, s) -> np.ndarray:
    """x_hat = fp16(fl32(fl32(s * c) + m)) (reading R15): float32 product, then sum,
    then rounding to fp16 (the quantizer's inputs are fp16 values)."""
    c = np.asarray(codes).astype(np.float32)
    prod = (np.asarray(s, np.float32) * c).astype(np.float32)
    return (prod + np.asarray(m, np.float32)).astype(np.float32).astype(np.float16)


def append_requantizing(sq: SeqKV, k_row, v_row, bits: int, rounding: int = NEAREST_EVEN, seed: int = 0,
                        seq: int = 0, head: int = 0, kv_heads: int = 1) -> SeqKV:
    """Append token L = sq.length with the requantizing open block (reading R15): the
    token's K partitions are quantized as usual; the open V block's codes are
    dequantized to fp16, the new value is added and the block is quantized again with
    n = T + 1 (a block that reaches Pi tokens is closed with those codes)."""
    k_row = np.asarray(k_row, np.float16)
    v_row = np.asarray(v_row, np.float16)
    L, Pi = sq.length, sq.partition
    d = k_row.shape[0]
    P = d // Pi
    uk = None
    if rounding == STOCHASTIC:
        uk = stochastic_threshold(seed, STREAM_K, element_index(seq, kv_heads, head, L, np.arange(d).reshape(P, Pi), d))
    kc, km, ks, ksum = quantize_partition(k_row.reshape(P, Pi), bits, "f16", rounding, uk)
    F, T = sq.full_blocks, sq.tail_tokens
    vc, vm, vs, vsum, vcount = sq.v_codes, sq.v_min, sq.v_scale, sq.v_sum, sq.v_count
    if T == 0:                                   # the token opens a new block
        vc = np.concatenate([vc, np.zeros((1, Pi, d), np.int64)])
        vm = np.concatenate([vm, np.zeros((1, d))]); vs = np.concatenate([vs, np.zeros((1, d))])
        vsum = np.concatenate([vsum, np.zeros((1, d), np.int64)]); vcount = np.concatenate([vcount, [0]])
        vals = v_row[None, :]
    else:
        old = dequantize_to_f16(vc[F, :T, :], vm[F][None, :], vs[F][None, :])   # [T][d]
        vals = np.concatenate([old, v_row[None, :]])
    uv = None
    if rounding == STOCHASTIC:
        toks = F * Pi + np.arange(T + 1)
        uv = stochastic_threshold(seed, STREAM_V, element_index(seq, kv_heads, head, toks[None, :], np.arange(d)[:, None], d))
    c, m, s_, tot = quantize_partition(vals.T, bits, "f16", rounding, uv)          # [d][T+1]
    vc = vc.copy(); vm = vm.copy(); vs = vs.copy(); vsum = vsum.copy(); vcount = vcount.copy()
    vc[F, :, :] = 0
    vc[F, :T + 1, :] = c.T
    vm[F] = m; vs[F] = s_; vsum[F] = tot; vcount[F] = T + 1
    tail = np.concatenate([sq.v_tail, v_row[None, :]]) if T + 1 < Pi else np.zeros((0, d), np.float16)
    return SeqKV(L + 1, Pi, np.concatenate([sq.k_codes, kc.reshape(1, d)]),
                 np.concatenate([sq.k_min, km.astype(np.float64)[None, :]]),
                 np.concatenate([sq.k_scale, ks.astype(np.float64)[None, :]]),
                 np.concatenate([sq.k_sum, ksum[None, :]]), vc, vm, vs, vsum, vcount, tail)


def dequantize_k(sq: SeqKV) -> np.ndarray:
    """x_hat = s * code + min per K partition, float64 [L][d]."""
    P = sq.k_min.shape[1]
    Pi = sq.partition
    out = np.zeros(sq.k_codes.shape)
    for p in range(P):
        sl = slice(p * Pi, (p + 1) * Pi)
        out[:, sl] = sq.k_scale[:, p:p + 1] * sq.k_codes[:, sl] + sq.k_min[:, p:p + 1]
    return out


def dequantize_v_blocks(sq: SeqKV) -> np.ndarray:
    """x_hat per full V block, float64 [F*Pi][d]."""
    F = sq.full_blocks
    rows = []
    for blk in range(F):
        rows.append(sq.v_scale[blk][None, :] * sq.v_codes[blk] + sq.v_min[blk][None, :])
    return np.concatenate(rows, 0) if rows else np.zeros((0, sq.k_codes.shape[1]))


# ----------------------------------------------------------------------------
# Operation counts of Sec. 5.2 / 5.3 (one partition spanning the inner dimension)
# ----------------------------------------------------------------------------
def hq_matmul_cost(M: int, Z: int, N: int) -> tuple:
    """(integer products, correction) of C = A B by Eq. 4 for A (M x Z), B (Z x N) as
    one partition: 2MZN for sum a'b'; 2MN (s_a s_b times it), MN + MZ (m_b s_a sum a'),
    MN + NZ (m_a s_b sum b'), 2MN (Z m_a m_b) and 3MN (adding the terms): 9MN + MZ + NZ."""
    return 2 * M * Z * N, 9 * M * N + M * Z + N * Z


def decode_approximation_cost(d: int, L: int, sums_cached: bool = True) -> int:
    """Correction cost of one decode step (q K^T with M=1, Z=d, N=L; P V with M=1,
    Z=L, N=d): 10(d + L) + 2dL; caching the K and V code sums (summation
    elimination) removes the 2dL of their per-step recomputation."""
    qk = hq_matmul_cost(1, d, L)[1]
    pv = hq_matmul_cost(1, L, d)[1]
    return qk + pv - (2 * d * L if sums_cached else 0)


def dequantization_cost(d: int, L: int) -> int:
    """Dequantizing K and V of one step, x = s c + m per element: 4dL."""
    return 4 * d * L


def count_eq4_ops(a_codes, m_a, s_a, b_codes, m_b, s_b) -> tuple:
    """Eq. 4 for A (M x Z) and B (Z x N) as one partition, evaluated element by element
    while counting every arithmetic operation.  Returns (C, integer ops, correction ops):
    per row of A its code sum (Z additions) and s_a * sum a' (1 multiplication), per
    column of B likewise, then per output element s_a s_b (A'B') (2), m_b (s_a sum a')
    (1), m_a (s_b sum b') (1), Z m_a m_b (2) and three additions."""
    A = np.asarray(a_codes, np.int64)
    B = np.asarray(b_codes, np.int64)
    M, Z = A.shape
    N = B.shape[1]
    iops = 0
    fops = 0
    u = []
    for i in range(M):                      # s_a[i] * sum_z a'[i][z]
        t = 0
        for z in range(Z):
            t += int(A[i, z]); fops += 1
        u.append(float(s_a[i]) * t); fops += 1
    v = []
    for j in range(N):                      # s_b[j] * sum_z b'[z][j]
        t = 0
        for z in range(Z):
            t += int(B[z, j]); fops += 1
        v.append(float(s_b[j]) * t); fops += 1
    C = np.zeros((M, N))
    for i in range(M):
        for j in range(N):
            p = 0
            for z in range(Z):
                p += int(A[i, z]) * int(B[z, j]); iops += 2
            t1 = float(s_a[i]) * float(s_b[j]) * p; fops += 2
            t2 = float(m_b[j]) * u[i]; fops += 1
            t3 = float(m_a[i]) * v[j]; fops += 1
            t4 = Z * float(m_a[i]) * float(m_b[j]); fops += 2
            C[i, j] = t1 + t2 + t3 + t4; fops += 3
    return C, iops, fops


# ----------------------------------------------------------------------------
# Attention on quantized operands (Sec. 5.3 with Eq. 2-4)
# ----------------------------------------------------------------------------
def quantize_query(q, partition: int, bits: int = 8, sr: Optional[QPStochastic] = None):
    """Q row quantized per partition along d with float32 metadata (Sec. 5.1: Q uses 8 bits);
    rounded to nearest, or stochastically with the thresholds of `sr`."""
    q = np.asarray(q, np.float16)
    d = q.shape[0]
    P = d // partition
    if sr is None:
        c, m, s, tot = quantize_partition(q.reshape(P, partition), bits, "f32")
    else:
        u = sr.u(STREAM_Q, np.arange(d)).reshape(P, partition)
        c, m, s, tot = quantize_partition(q.reshape(P, partition), bits, "f32", STOCHASTIC, u)
    return c.reshape(d), m.astype(np.float64), s.astype(np.float64), tot


def scores(q, sq: SeqKV, qp_bits: int = 8, upto: Optional[int] = None, sr: Optional[QPStochastic] = None):
    """S_j = (1/sqrt(d)) sum_p Eq4(q'_p, k'_{j,p}) for j < upto, using the cached K sums.
    Returns (S float64 [upto], integer products int64 [upto][P], q codes, q min, q scale)."""
    d = sq.k_codes.shape[1]
    Pi = sq.partition
    P = d // Pi
    L = sq.length if upto is None else upto
    qc, qm, qs, qsum = quantize_query(q, Pi, qp_bits, sr)
    S = np.zeros(L)
    prods = np.zeros((L, P), np.int64)
    for p in range(P):
        sl = slice(p * Pi, (p + 1) * Pi)
        C = sq.k_codes[:L, sl] @ qc[sl]
        prods[:, p] = C
        sk = sq.k_scale[:L, p]
        mk = sq.k_min[:L, p]
        S += qs[p] * sk * C + qs[p] * mk * qsum[p] + qm[p] * sk * sq.k_sum[:L, p] + Pi * qm[p] * mk
    S = S / math.sqrt(d)
    return S, prods, qc, qm, qs


def _quantize_p(p, qp_bits: int, sr: Optional[QPStochastic], first: int):
    """One V block's probabilities (key tokens first, first+1, ...) quantized in float64."""
    if sr is None:
        return quantize_partition(p, qp_bits, "f64")
    return quantize_partition(p, qp_bits, "f64", STOCHASTIC, sr.u(STREAM_P, first + np.arange(len(p))))


def pv_blocks(prob, sq: SeqKV, qp_bits: int, tail_mode: int, sr: Optional[QPStochastic] = None):
    """O_c = sum over V blocks of Eq4(P'_block, V'_block,c) plus the open block
    (fp16 and unquantized P in TAIL_FP16 mode; re-quantized with n=T in TAIL_REQUANT mode)."""
    d = sq.k_codes.shape[1]
    Pi = sq.partition
    F, T = sq.full_blocks, sq.tail_tokens
    O = np.zeros(d)
    for blk in range(F):
        pc, pm, ps, psum = _quantize_p(prob[blk * Pi:(blk + 1) * Pi], qp_bits, sr, blk * Pi)
        D = pc @ sq.v_codes[blk]                      # int64 [d]
        O += ps * sq.v_scale[blk] * D + ps * sq.v_min[blk] * psum \
            + pm * sq.v_scale[blk] * sq.v_sum[blk] + Pi * pm * sq.v_min[blk]
    if T > 0:
        pt = prob[F * Pi:F * Pi + T]
        if tail_mode == TAIL_FP16:
            O += pt @ sq.v_tail.astype(np.float64)
        else:
            pc, pm, ps, psum = _quantize_p(pt, qp_bits, sr, F * Pi)
            D = pc @ sq.v_codes[F, :T]
            O += ps * sq.v_scale[F] * D + ps * sq.v_min[F] * psum \
                + pm * sq.v_scale[F] * sq.v_sum[F] + T * pm * sq.v_min[F]
    return O


def softmax(S):
    """Row softmax (Eq. 3), max-subtracted, float64."""
    e = np.exp(S - S.max())
    return e / e.sum()


def decode_row(q, sq: SeqKV, qp_bits: int = 8, tail_mode: int = TAIL_FP16, sr: Optional[QPStochastic] = None):
    """One decode query row over the whole cached sequence (Sec. 5.3, L_Q = 1)."""
    if sq.length == 0:
        return np.zeros(sq.k_codes.shape[1])
    S, _, _, _, _ = scores(q, sq, qp_bits, sr=sr)
    return pv_blocks(softmax(S), sq, qp_bits, tail_mode, sr)


def prefill_row(q, sq: SeqKV, i: int, causal: bool, qp_bits: int = 8, sr: Optional[QPStochastic] = None):
    """Prefill row i (L_Q = L_KV, Sec. 5.3): causal rows see tokens j <= i; P is zero
    past i and its blocks are quantized over all Pi entries (reading R7)."""
    L = sq.length
    upto = i + 1 if causal else L
    S, _, _, _, _ = scores(q, sq, qp_bits, upto, sr)
    prob = np.zeros(L)
    prob[:upto] = softmax(S)
    return pv_blocks(prob, sq, qp_bits, TAIL_FP16, sr)


# ----------------------------------------------------------------------------
# QKV generation in front of prefill attention (Sec. 4, Eq. 1; fused with
# quantization and attention in the paper's prefill kernel, Sec. 6)
# ----------------------------------------------------------------------------
def project_qkv(E, W, q_heads: int, kv_heads: int, head_dim: int, tokens=None):
    """Eq. 1: Q^h = E W_Q^h, K^h = E W_K^h, V^h = E W_V^h for one sequence.

    E: fp16 [L][hidden], the prompt's embeddings.  W: fp16 [(H_q + 2 H_kv) * d][hidden],
    one row per output channel: the H_q query heads' d channels, then the H_kv key
    heads', then the H_kv value heads' (the transposes of W_Q, W_K, W_V side by side).
    The products are summed in float64 and rounded once to fp16, the precision of the
    K/V values the quantizer takes (and of the Q the attention takes).  `tokens`
    optionally restricts the rows (a list of token indices).
    Returns fp16 Q [H_q][n][d], K [H_kv][n][d], V [H_kv][n][d]."""
    E = np.asarray(E, np.float16)
    W = np.asarray(W, np.float16)
    if tokens is not None:
        E = E[np.asarray(tokens)]
    n = E.shape[0]
    d = head_dim
    out = (E.astype(np.float64) @ W.astype(np.float64).T).astype(np.float16)   # [n][N]
    heads = out.reshape(n, q_heads + 2 * kv_heads, d).transpose(1, 0, 2)
    return (np.ascontiguousarray(heads[:q_heads]), np.ascontiguousarray(heads[q_heads:q_heads + kv_heads]),
            np.ascontiguousarray(heads[q_heads + kv_heads:]))


def prefill_from_embeddings(E, W, q_heads: int, kv_heads: int, head_dim: int, bits: int, partition: int,
                            causal: bool = True, qp_bits: int = 8, rows=None, rounding: int = NEAREST_EVEN,
                            seed: int = 0):
    """The paper's prefill (Sec. 6): QKV generation (Eq. 1), quantization of K and V
    (Sec. 5.2-5.3) and attention with homomorphic quantization, for a batch.
    E: fp16 [B][L][hidden].  Returns (O float32 [B][H_q][L][d], Q fp16 [B][H_q][L][d],
    seqs[b][h] SeqKV).  `rows` restricts the attention to (b, h_q, i) triples."""
    E = np.asarray(E, np.float16)
    B = E.shape[0]
    Qs, seqs = [], []
    for b in range(B):
        Q, K, V = project_qkv(E[b], W, q_heads, kv_heads, head_dim)
        Qs.append(Q)
        seqs.append([quantize_sequence(K[h], V[h], bits, partition, rounding, seed, b, h, kv_heads)
                     for h in range(kv_heads)])
    Q = np.stack(Qs)
    return attend_prefill(Q, seqs, kv_heads, causal, qp_bits, rows), Q, seqs


def attend_decode(q, seqs, kv_heads: int, qp_bits: int = 8, tail_mode: int = TAIL_FP16, rows=None,
                  stochastic_seed: Optional[int] = None):
    """q [B][H_q][d] fp16; seqs[b][h_kv] SeqKV.  Returns O float32 [B][H_q][d].
    `rows` optionally restricts the work to a list of (b, h_q) pairs (others stay 0).
    With `stochastic_seed`, Q and P codes are rounded stochastically (reading R4)."""
    B, Hq, d = q.shape
    G = Hq // kv_heads
    O = np.zeros((B, Hq, d), np.float64)
    todo = rows if rows is not None else [(b, h) for b in range(B) for h in range(Hq)]
    for b, h in todo:
        sr = None if stochastic_seed is None else QPStochastic(stochastic_seed, b, Hq, h, 0)
        O[b, h] = decode_row(q[b, h], seqs[b][h // G], qp_bits, tail_mode, sr)
    return O.astype(np.float32)


def attend_prefill(Q, seqs, kv_heads: int, causal: bool = True, qp_bits: int = 8, rows=None,
                   stochastic_seed: Optional[int] = None):
    """Q [B][H_q][L][d] fp16.  Returns O float32 [B][H_q][L][d].
    `rows` optionally restricts the work to a list of (b, h_q, i) triples.
    With `stochastic_seed`, Q and P codes are rounded stochastically (reading R4)."""
    B, Hq, L, d = Q.shape
    G = Hq // kv_heads
    O = np.zeros((B, Hq, L, d), np.float64)
    todo = rows if rows is not None else [(b, h, i) for b in range(B) for h in range(Hq) for i in range(L)]
    for b, h, i in todo:
        sr = None if stochastic_seed is None else QPStochastic(stochastic_seed, b, Hq, h, i)
        O[b, h, i] = prefill_row(Q[b, h, i], seqs[b][h // G], i, causal, qp_bits, sr)
    return O.astype(np.float32)


def attention_unquantized(q, k, v, causal_row: Optional[int] = None):
    """Plain softmax(q k^T / sqrt(d)) v in float64 for one row (context only, not a gate)."""
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    q = np.asarray(q, np.float64)
    L = k.shape[0] if causal_row is None else causal_row + 1
    S = k[:L] @ q / math.sqrt(q.shape[0])
    return softmax(S) @ v[:L]


# ----------------------------------------------------------------------------
# The compressed byte format (the bytes a prefill instance would send, Sec. 5.1)
# ----------------------------------------------------------------------------
def pack_cache(seqs, kv_heads: int, head_dim: int, bits: int, partition: int,
               page_tokens: int, num_pages: int, block_table=None, batch: Optional[int] = None):
    """Lay the quantized sequences out in the library's byte format.

    Sections (all little-endian):
      k_codes [pages][H][page_tokens][d*b/8]        codes of each token, partitions in order
      k_meta  [pages][H][page_tokens][d/Pi][2] f16  (min, scale)
      k_sums  [pages][H][page_tokens][d/Pi]         u8 or u16
      v_codes [pages][H][page_tokens/Pi][d][Pi*b/8] codes of each channel over a block
      v_meta  [pages][H][page_tokens/Pi][d][2] f16
      v_sums  [pages][H][page_tokens/Pi][d]
      v_tail  [B][H][Pi][d] f16                     open block, fp16
    Token t of sequence s lives on page table[s][t // page_tokens] at slot t % page_tokens;
    without a table, sequence s uses page s.  The open block's re-quantized codes
    (n = T) are stored at its block slot with zero codes past T."""
    B = len(seqs) if batch is None else batch
    d, Pi = head_dim, partition
    P = d // Pi
    sdt = np.uint8 if sum_bytes(bits, Pi) == 1 else np.uint16
    bpp = page_tokens // Pi
    out = {
        "k_codes": np.zeros((num_pages, kv_heads, page_tokens, d * bits // 8), np.uint8),
        "k_meta": np.zeros((num_pages, kv_heads, page_tokens, P, 2), np.float16),
        "k_sums": np.zeros((num_pages, kv_heads, page_tokens, P), sdt),
        "v_codes": np.zeros((num_pages, kv_heads, bpp, d, Pi * bits // 8), np.uint8),
        "v_meta": np.zeros((num_pages, kv_heads, bpp, d, 2), np.float16),
        "v_sums": np.zeros((num_pages, kv_heads, bpp, d), sdt),
        "v_tail": np.zeros((B, kv_heads, Pi, d), np.float16),
    }

    def page_of(s, t):
        return int(block_table[s][t // page_tokens]) if block_table is not None else s

    for s in range(B):
        for h in range(kv_heads):
            sq = seqs[s][h]
            L = sq.length
            kbytes = pack_codes(sq.k_codes.reshape(L, P, Pi), bits).reshape(L, d * bits // 8)
            vbytes = pack_codes(np.transpose(sq.v_codes, (0, 2, 1)), bits)   # [NB][d][Pi*b/8]
            for t0 in range(0, L, page_tokens):
                t1 = min(L, t0 + page_tokens)
                pg = page_of(s, t0)
                out["k_codes"][pg, h, :t1 - t0] = kbytes[t0:t1]
                out["k_meta"][pg, h, :t1 - t0, :, 0] = sq.k_min[t0:t1]
                out["k_meta"][pg, h, :t1 - t0, :, 1] = sq.k_scale[t0:t1]
                out["k_sums"][pg, h, :t1 - t0] = sq.k_sum[t0:t1]
            for blk in range(sq.v_codes.shape[0]):
                pg = page_of(s, blk * Pi)
                bi = (blk * Pi % page_tokens) // Pi
                out["v_codes"][pg, h, bi] = vbytes[blk]
                out["v_meta"][pg, h, bi, :, 0] = sq.v_min[blk]
                out["v_meta"][pg, h, bi, :, 1] = sq.v_scale[blk]
                out["v_sums"][pg, h, bi] = sq.v_sum[blk]
            out["v_tail"][s, h, :sq.tail_tokens] = sq.v_tail
    return out
