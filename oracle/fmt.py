"""Number formats and the packed-code format (oracle).

The paper stores per-head bit-widths in a small static table that the
quantizer indexes in O(1) (Sec. 3.4 "Pipeline summary"; Appendix "Runtime
Analysis"), and counts the cache as b bits per element (Appendix "Memory
Footprint").  It does not fix a byte layout; the one below is this
library's, and packed codes are compared bit for bit against it.

Chunk: 32 codes of one b-bit stream (b = 1..8) occupy exactly b 32-bit
words.  Words are little-endian uint32.

b = 3: every code is one 3-bit field.  The three words form one 96-bit
stream (stream bit 32k + j is bit j of word k), cut into four quarters of
24 bits; quarter q (0..3) holds, for i = 0..3,
    code  4q + i       at stream bit  24q + 3i,
    code  16 + 4q + i  at stream bit  24q + 12 + 3i,
so that moving the upper 12 bits of a quarter up by 4 puts codes
(4q + i, 16 + 4q + i) at bits (3i, 16 + 3i) of one word.  Two fields cross
a word boundary (codes 6 and 25).

Other widths: the code bits are split into planes whose widths are the
binary digits of b, widest first (b=5 -> 4,1; b=6 -> 4,2; b=7 -> 4,2,1;
b=1,2,4,8 -> one plane); plane p holds code bits [o_p, o_p + w_p).  A plane
of width w is w words; word d of it holds, for k = 0 .. 16/w - 1,
    the field of code  d*16/w + k       at bit  k*w,
    the field of code  16 + d*16/w + k  at bit  16 + k*w,
so that every 16-bit half-word pair (bit k*w, bit 16 + k*w) carries codes
(i, i + 16).

Pair order of a 32-entry sequence s[0..31]: s[0], s[16], s[1], s[17], ...,
s[15], s[31].  Per-group metadata is stored in pair order.
"""
import numpy as np

CHUNK = 32
F16_MAX = 65504.0


def planes(b):
    """Plane widths of a b-bit code, widest first (b = 3: one field)."""
    if not 1 <= b <= 8:
        raise ValueError("bits must be in 1..8")
    if b == 3:
        return [3]
    return [w for w in (8, 4, 2, 1) if b & w]


def stream3_bit(i):
    """Stream bit of code i (0..31) of a three-bit chunk."""
    j = i % 16
    return 24 * (j // 4) + 3 * (j % 4) + (12 if i >= 16 else 0)


def _pack3(codes, out):
    for i in range(CHUNK):
        pos = stream3_bit(i)
        word, bit = divmod(pos, 32)
        c = codes[..., i]
        out[..., word] |= (c << np.uint32(bit)) & np.uint32(0xFFFFFFFF)
        if bit + 3 > 32:
            out[..., word + 1] |= c >> np.uint32(32 - bit)
    return out


def _unpack3(words, codes):
    x = [words[..., k].astype(np.int64) for k in range(3)]
    for i in range(CHUNK):
        pos = stream3_bit(i)
        word, bit = divmod(pos, 32)
        v = x[word] >> bit
        if bit + 3 > 32:
            v = v | (x[word + 1] << (32 - bit))
        codes[..., i] = v & 7
    return codes


def pack_chunks(codes, b):
    """codes[..., 32] (integers < 2^b) -> words[..., b] uint32."""
    codes = np.asarray(codes, dtype=np.uint32)
    assert codes.shape[-1] == CHUNK
    if np.any(codes >> b):
        raise ValueError("code out of range")
    out = np.zeros(codes.shape[:-1] + (b,), dtype=np.uint32)
    if b == 3:
        return _pack3(codes, out)
    word = 0
    shift = 0
    for w in planes(b):
        per = 16 // w
        mask = np.uint32((1 << w) - 1)
        for d in range(w):
            acc = np.zeros(codes.shape[:-1], dtype=np.uint32)
            for k in range(per):
                lo = (codes[..., d * per + k] >> shift) & mask
                hi = (codes[..., 16 + d * per + k] >> shift) & mask
                acc |= lo << np.uint32(k * w)
                acc |= hi << np.uint32(16 + k * w)
            out[..., word] = acc
            word += 1
        shift += w
    return out


def unpack_chunks(words, b):
    """Inverse of pack_chunks: words[..., b] -> codes[..., 32] (int64)."""
    words = np.asarray(words, dtype=np.uint32)
    assert words.shape[-1] == b
    codes = np.zeros(words.shape[:-1] + (CHUNK,), dtype=np.int64)
    if b == 3:
        return _unpack3(words, codes)
    word = 0
    shift = 0
    for w in planes(b):
        per = 16 // w
        mask = (1 << w) - 1
        for d in range(w):
            x = words[..., word].astype(np.int64)
            for k in range(per):
                codes[..., d * per + k] |= ((x >> (k * w)) & mask) << shift
                codes[..., 16 + d * per + k] |= (
                    (x >> (16 + k * w)) & mask) << shift
            word += 1
        shift += w
    return codes


PAIR_ORDER = np.array([i // 2 + 16 * (i % 2) for i in range(CHUNK)])


def to_pair_order(x):
    """x[..., 32] -> x[..., PAIR_ORDER]."""
    return np.asarray(x)[..., PAIR_ORDER]


def from_pair_order(x):
    inv = np.argsort(PAIR_ORDER)
    return np.asarray(x)[..., inv]


# ------------------------------------------------------------ 16-bit floats
def f16_sat(x):
    """Round float32 to fp16 (nearest-even), saturating at +-65504."""
    x = np.clip(np.asarray(x, dtype=np.float32), -F16_MAX, F16_MAX)
    return x.astype(np.float16)


def widen16(bits, is_bf16):
    """Exact float32 value of fp16 / bf16 bit patterns."""
    bits = np.asarray(bits, dtype=np.uint16)
    if is_bf16:
        return (bits.astype(np.uint32) << 16).view(np.float32)
    return bits.view(np.float16).astype(np.float32)
