"""Helpers of the GPU parity tests: move seeded inputs to the device and read
the library's cache buffers back according to the documented layout (the
offsets are recomputed here from the layout formula, not asked of the
library)."""
import numpy as np

import workloads
from oracle import cache as ocache

KIVI, QUAROT, TURBO, RTN, KIVI_RTN = 0, 1, 2, 3, 4


def dev(bits16, dtype, device="cuda"):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits16).view(np.int16))
    t = t.view(torch.float16 if dtype == workloads.F16 else torch.bfloat16)
    return t.to(device)


def host_bits(t):
    """uint16 bit patterns of a 16-bit torch tensor."""
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


class Layout:
    """Byte layout of a cache (mirrors the description in include/rq.h)."""

    def __init__(self, family, n_layers, batch, H, cap, R, bits):
        self.family, self.L, self.B, self.H = family, n_layers, batch, H
        self.cap, self.R = cap, R
        self.bits = np.asarray(bits).reshape(n_layers, H, 2)
        # metadata bytes per block of each kind (KIVI-style 512, per-token 64)
        self.mb = (512 if family in (KIVI, KIVI_RTN) else 64,
                   512 if family == KIVI else 64)

    def region_off(self, l, h, kind):
        flat = self.bits.reshape(-1)
        i = (l * self.H + h) * 2 + kind
        return int(sum(self.B * self.cap * 16 * int(b) for b in flat[:i]))

    def k_words(self, codes_u8, l, b, h, n_tok):
        bk = int(self.bits[l, h, 0])
        base = self.region_off(l, h, 0) + b * self.cap * 16 * bk
        raw = codes_u8[base: base + n_tok * 16 * bk]
        return raw.view(np.uint32).reshape(n_tok, 4, bk)

    def v_words(self, codes_u8, l, b, h, n_blk):
        bv = int(self.bits[l, h, 1])
        base = self.region_off(l, h, 1) + b * self.cap * 16 * bv
        raw = codes_u8[base: base + n_blk * 128 * 4 * bv]
        return raw.view(np.uint32).reshape(n_blk, 128, bv)

    def meta(self, meta_u8, l, b, h, kind, n_blk):
        nblk_cap = self.cap // 32
        mk, mv = self.mb
        layer = self.H * self.B * nblk_cap * (mk + mv)
        base = (l * layer + h * self.B * nblk_cap * (mk + mv) + kind * self.B * nblk_cap * mk
                + b * nblk_cap * self.mb[kind])
        raw = meta_u8[base: base + n_blk * self.mb[kind]].view(np.float16)
        if self.mb[kind] == 512:
            return raw.reshape(n_blk, 4, 2, 32)
        return raw.reshape(n_blk, 32)

    def ring(self, resid_u16, l, b, h, kind):
        slots = self.R + 32
        layer = self.B * self.H * 2 * slots * 128
        base = l * layer + (((b * self.H + h) * 2 + kind) * slots) * 128
        return resid_u16[base: base + slots * 128].reshape(slots, 128)


def compare_unit(lay, bufs, l, b, h, unit, k16, v16):
    """Assert the device cache of unit (l, b, h) equals the oracle unit
    bit for bit (codes, metadata, residual window).  k16/v16: uint16 input
    bits [T][128] of this unit."""
    codes_u8, meta_u8, resid_u16 = bufs
    nq, T = unit.nq, unit.T
    np.testing.assert_array_equal(lay.k_words(codes_u8, l, b, h, nq),
                                  unit.k_words)
    np.testing.assert_array_equal(lay.v_words(codes_u8, l, b, h, nq // 32),
                                  unit.v_words)
    for kind, want in ((0, unit.k_meta), (1, unit.v_meta)):
        got = lay.meta(meta_u8, l, b, h, kind, nq // 32)
        np.testing.assert_array_equal(got.view(np.uint16),
                                      np.asarray(want).view(np.uint16))
    for kind, src in ((0, k16), (1, v16)):
        ring = lay.ring(resid_u16, l, b, h, kind)
        for t in range(nq, T):
            np.testing.assert_array_equal(ring[ocache.ring_slot(t, lay.R)],
                                          src[t])


def read_buffers(kvc):
    return (kvc.codes.cpu().numpy(), kvc.meta.cpu().numpy(),
            kvc.resid.cpu().numpy().view(np.uint16))
