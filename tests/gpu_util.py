"""Helpers shared by the GPU parity tests: seeded inputs, caches on the device,
and the oracle's view of the same data.  Imported by tests only."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import hack_oracle as O
from paper_2502_03589_amd import hack as hk
from paper_2502_03589_amd import synth

DEV = torch.device("cuda:0")


def announce(msg: str):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


class Case:
    """K/V/q inputs, a device cache written by hack_quantize, and the oracle's sequences."""

    def __init__(self, seed, batch, kv_heads, lens, bits, pi, group=4, d=128, paged_page=0,
                 rounding=O.NEAREST_EVEN, spare_tokens=0, outliers=0, qp_bits=8):
        self.seed, self.batch, self.H, self.d = seed, batch, kv_heads, d
        self.bits, self.pi, self.G, self.Hq = bits, pi, group, group * kv_heads
        self.lens = np.asarray(lens, np.int32)
        self.max_len = int(self.lens.max()) if len(self.lens) else 0
        total = self.max_len + spare_tokens
        self.k = synth.normal_f16(seed, "k", (batch, kv_heads, max(total, 1), d))
        if outliers:
            ch = synth.outlier_channels(seed, d, outliers)
            self.k = synth.scale_channels_f16(self.k, ch, 10.0)
        self.v = synth.normal_f16(seed, "v", (batch, kv_heads, max(total, 1), d))
        self.q = synth.normal_f16(seed, "q", (batch, self.Hq, d))
        self.rounding = rounding
        self.qp_bits = qp_bits
        if paged_page:
            self.page_tokens = paged_page
            lens_cap = np.maximum(self.lens + spare_tokens, 1)
            table, pages = synth.page_table(seed, lens_cap, paged_page)
            self.table_np, self.num_pages = table, pages
            self.table = torch.from_numpy(table).to(DEV)
        else:
            cap = max(pi, ((total + pi - 1) // pi) * pi)
            self.page_tokens = cap
            self.table_np, self.table, self.num_pages = None, None, batch
        self.layout = hk.hack_kv_layout_make(d, kv_heads, bits, pi, self.page_tokens, qp_bits, rounding, seed)
        self.cache = hk.KVCache(self.layout, self.num_pages, batch, self.table, DEV)
        self.lens_dev = torch.from_numpy(self.lens.copy()).to(DEV)

    # ---- device side -------------------------------------------------------------
    def quantize(self):
        k = torch.from_numpy(np.ascontiguousarray(self.k[:, :, :self.max_len])).to(DEV)
        v = torch.from_numpy(np.ascontiguousarray(self.v[:, :, :self.max_len])).to(DEV)
        hk.hack_quantize(self.layout, self.cache, k, v, self.lens_dev, self.max_len)
        return self

    def append(self, step, tail_mode):
        """Append the token at position lens (per sequence) from the stored inputs."""
        cur = self.lens_dev.cpu().numpy()
        kn = np.stack([self.k[b, :, cur[b]] for b in range(self.batch)])
        vn = np.stack([self.v[b, :, cur[b]] for b in range(self.batch)])
        hk.hack_append(self.layout, self.cache, torch.from_numpy(kn).to(DEV), torch.from_numpy(vn).to(DEV),
                       self.lens_dev, int(cur.max()), tail_mode)
        self.lens = cur + 1
        self.max_len = int(self.lens.max())

    def sections(self):
        torch.cuda.synchronize()
        return {n: b.cpu().numpy() for n, b in self.cache.buffers.items()}

    # ---- oracle side -------------------------------------------------------------
    def oracle_seqs(self, pairs=None):
        out = [[None] * self.H for _ in range(self.batch)]
        for b in range(self.batch):
            for h in range(self.H):
                if pairs is not None and (b, h) not in pairs:
                    continue
                L = int(self.lens[b])
                out[b][h] = O.quantize_sequence(self.k[b, h, :L], self.v[b, h, :L], self.bits, self.pi,
                                                self.rounding, self.seed, b, h, self.H)
        return out

    def oracle_bytes(self, seqs):
        return O.pack_cache(seqs, self.H, self.d, self.bits, self.pi, self.page_tokens, self.num_pages,
                            self.table_np, self.batch)


def as_sections(raw: dict, case: Case) -> dict:
    """Reshape the raw device byte buffers into the oracle's section arrays."""
    P = case.d // case.pi
    pt, pages, H, d, pi, bits = case.page_tokens, case.num_pages, case.H, case.d, case.pi, case.bits
    sdt = np.uint8 if case.layout.sum_bytes == 1 else np.uint16
    n = lambda a, cnt: a[:cnt]
    return {
        "k_codes": n(raw["k_codes"], pages * H * pt * d * bits // 8).reshape(pages, H, pt, d * bits // 8),
        "k_meta": n(raw["k_meta"], pages * H * pt * P * 4).view(np.float16).reshape(pages, H, pt, P, 2),
        "k_sums": n(raw["k_sums"], pages * H * pt * P * case.layout.sum_bytes).view(sdt).reshape(pages, H, pt, P),
        "v_codes": n(raw["v_codes"], pages * H * pt * d * bits // 8).reshape(pages, H, pt // pi, d, pi * bits // 8),
        "v_meta": n(raw["v_meta"], pages * H * (pt // pi) * d * 4).view(np.float16).reshape(pages, H, pt // pi, d, 2),
        "v_sums": n(raw["v_sums"], pages * H * (pt // pi) * d * case.layout.sum_bytes).view(sdt).reshape(pages, H, pt // pi, d),
        "v_tail": n(raw["v_tail"], case.batch * H * pi * d * 2).view(np.float16).reshape(case.batch, H, pi, d),
    }


def valid_masks(case: Case, include_open_block: bool):
    """Boolean masks of the slots a sequence of the current lengths owns."""
    pt, pi, H = case.page_tokens, case.pi, case.H
    km = np.zeros((case.num_pages, H, pt), bool)
    vm = np.zeros((case.num_pages, H, pt // pi), bool)
    tm = np.zeros((case.batch, H, pi), bool)
    for b in range(case.batch):
        L = int(case.lens[b])
        F, T = L // pi, L % pi
        for t in range(L):
            pg = b if case.table_np is None else case.table_np[b][t // pt]
            km[pg, :, t % pt] = True
        nb = F + (1 if (T and include_open_block) else 0)
        for blk in range(nb):
            pg = b if case.table_np is None else case.table_np[b][blk * pi // pt]
            vm[pg, :, (blk * pi % pt) // pi] = True
        tm[b, :, :T] = True
    return km, vm, tm


def rel_err(got, ref):
    return float(np.abs(np.asarray(got, np.float64) - ref).max() / max(np.abs(ref).max(), 1e-30))
