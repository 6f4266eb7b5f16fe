"""Quantized KV cache of one (layer, batch entry, kv-head) unit (oracle).

Residual window (a reading: the paper does not describe one; the workload
definitions ask for a 16-bit window of the most recent tokens): tokens are
quantized in blocks of 32 once they are older than the window, so with T
cached tokens and window R the quantized prefix is
    nq = max(0, floor((T - R) / 32) * 32)
and tokens nq .. T-1 stay exact in the 16-bit input type, in a ring of
R + 32 slots (token t in slot t mod (R + 32)).  The same rule serves every
quantizer family.

Layout of one unit, all little-endian (the byte layout is this library's;
see ``fmt`` for chunks and pair order):

  K codes  [token][chunk q = 0..3][b_K words]      chunk q = channels 32q..32q+31
  V codes  [block][channel 0..127][b_V words]      a chunk = the 32 tokens of a block
  KIVI meta, per block, K then V:
           K: [chunk q][s(32, pair order), z(32, pair order)]  fp16
           V: [channel group cg][s(32 tokens, pair order), z(...)]  fp16
  QuaRot meta, per block: [32 tokens, pair order] fp16 scale
  TurboQuant meta, per block: [32 tokens, pair order] fp16 norm
  KIVI_RTN (the "mixed" family: KIVI's per-channel asymmetric keys with
  RTN's per-token symmetric values, each side its own quantizer as the
  paper's K/V separation allows, Sec. 3.4): K meta as KIVI, V meta as RTN
"""
import numpy as np

from . import fmt, quant

KIVI, QUAROT, TURBO, RTN, KIVI_RTN = 0, 1, 2, 3, 4


def n_quantized(T, R):
    return max(0, ((T - R) // 32) * 32)


def ring_slot(t, R):
    return t % (R + 32)


def pack_keys(codes, b):
    """codes[T][128] -> words[T][4][b]."""
    T = codes.shape[0]
    return fmt.pack_chunks(codes.reshape(T, 4, 32), b)


def pack_values(codes, b):
    """codes[T][128] (T % 32 == 0) -> words[T/32][128][b]."""
    T = codes.shape[0]
    blk = codes.reshape(T // 32, 32, 128).transpose(0, 2, 1)
    return fmt.pack_chunks(blk, b)


def unpack_keys(words, b):
    T = words.shape[0]
    return fmt.unpack_chunks(words, b).reshape(T, 128)


def unpack_values(words, b):
    nb = words.shape[0]
    return fmt.unpack_chunks(words, b).transpose(0, 2, 1).reshape(nb * 32, 128)


def kivi_meta_keys(s, z):
    """s, z fp16[nblk][128] -> fp16[nblk][4][2][32] (pair order)."""
    nb = s.shape[0]
    s4 = fmt.to_pair_order(s.reshape(nb, 4, 32))
    z4 = fmt.to_pair_order(z.reshape(nb, 4, 32))
    return np.stack([s4, z4], axis=2)


def kivi_meta_values(s, z):
    """s, z fp16[T][4] -> fp16[T/32][4][2][32] (tokens in pair order)."""
    T = s.shape[0]
    s4 = fmt.to_pair_order(s.reshape(T // 32, 32, 4).transpose(0, 2, 1))
    z4 = fmt.to_pair_order(z.reshape(T // 32, 32, 4).transpose(0, 2, 1))
    return np.stack([s4, z4], axis=2)


def token_meta(s):
    """Per-token fp16 values [T] -> [T/32][32] pair order."""
    T = s.shape[0]
    return fmt.to_pair_order(s.reshape(T // 32, 32))


class Unit:
    """Oracle cache of one unit, built from the first T tokens of k, v
    (float32 [T][128], exact values of the 16-bit inputs)."""

    def __init__(self, family, k, v, bk, bv, R, rotation=None):
        """rotation: the (layer, kv-head) rotation for TurboQuant (float64
        [128][128], the exact bf16 values), else None."""
        self.family, self.bk, self.bv, self.R = family, bk, bv, R
        T = k.shape[0]
        self.T = T
        self.nq = nq = n_quantized(T, R)
        kq, vq = k[:nq], v[:nq]
        if family == KIVI:
            uk, sk, zk = quant.kivi_quant_keys(kq, bk)
            uv, sv, zv = quant.kivi_quant_values(vq, bv)
            self.k_hat = quant.kivi_dequant_keys(uk, sk, zk)
            self.v_hat = quant.kivi_dequant_values(uv, sv, zv)
            self.k_meta = kivi_meta_keys(sk, zk)
            self.v_meta = kivi_meta_values(sv, zv)
        elif family == QUAROT:
            uk, sk = quant.quarot_quant(kq, bk)
            uv, sv = quant.quarot_quant(vq, bv)
            self.k_hat = quant.quarot_dequant(uk, sk, bk)
            self.v_hat = quant.quarot_dequant(uv, sv, bv)
            self.k_meta = token_meta(sk)
            self.v_meta = token_meta(sv)
        elif family == RTN:
            uk, sk = quant.rtn_quant(kq, bk)
            uv, sv = quant.rtn_quant(vq, bv)
            self.k_hat = quant.rtn_dequant(uk, sk, bk)
            self.v_hat = quant.rtn_dequant(uv, sv, bv)
            self.k_meta = token_meta(sk)
            self.v_meta = token_meta(sv)
        elif family == KIVI_RTN:
            uk, sk, zk = quant.kivi_quant_keys(kq, bk)
            uv, sv = quant.rtn_quant(vq, bv)
            self.k_hat = quant.kivi_dequant_keys(uk, sk, zk)
            self.v_hat = quant.rtn_dequant(uv, sv, bv)
            self.k_meta = kivi_meta_keys(sk, zk)
            self.v_meta = token_meta(sv)
        elif family == TURBO:
            uk, nk, self.k_t = quant.turbo_quant(kq, rotation, bk)
            uv, nv, self.v_t = quant.turbo_quant(vq, rotation, bv)
            self.k_hat = quant.turbo_dequant(uk, nk, rotation, bk)
            self.v_hat = quant.turbo_dequant(uv, nv, rotation, bv)
            self.k_meta = token_meta(nk)
            self.v_meta = token_meta(nv)
        else:
            raise NotImplementedError(family)
        self.k_codes, self.v_codes = uk, uv
        self.k_words = pack_keys(uk, bk)
        self.v_words = pack_values(uv, bv)
        # residual ring
        cap = R + 32
        self.ring_k = np.zeros((cap, 128), dtype=np.float32)
        self.ring_v = np.zeros((cap, 128), dtype=np.float32)
        for t in range(nq, T):
            self.ring_k[ring_slot(t, R)] = k[t]
            self.ring_v[ring_slot(t, R)] = v[t]
        self.k_res = np.asarray(k[nq:T], dtype=np.float64)
        self.v_res = np.asarray(v[nq:T], dtype=np.float64)

    def keys(self):
        """Effective keys seen by attention: dequantized prefix + residual."""
        return np.concatenate([self.k_hat, self.k_res], axis=0)

    def values(self):
        return np.concatenate([self.v_hat, self.v_res], axis=0)
