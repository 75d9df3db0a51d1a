"""Sampling walk oracle: the round at temperature T > 0.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What the method computes: under sampling the walk draws a token from the
verified row of its current node and descends while the draw is a child in
the tree; the last draw becomes the next root.  Every committed token is then
a draw from the target's own distribution, so the output distribution is that
of sampling the target token by token (the paper's limitations section and
its temperature-1 results in App. C).

Readings (also listed in the design notes):

* A draw from softmax(z / T) is taken by the Gumbel-max rule: the token of
  largest z_w / T + g_w, with g_w = -ln(-ln u_w) and u_w uniform on (0, 1),
  lowest index on ties.  Every row gets its own draw; rows the walk does not
  visit are never read, so drawing all rows up front changes nothing.
* The uniforms come from the counter-based generator Philox4x32-10 (Salmon,
  Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11),
  written here from its definition: key (seed_lo, seed_hi), counter
  (w // 4, node, sequence, round), word w % 4 of the output;
  u = ((x >> 9) + 0.5) * 2^-23: 23 bits, so that k + 0.5 still fits fp32's
  24-bit significand; u is then exact and lies in [2^-24, 1 - 2^-24].
* The logarithms are computed by one fixed fp32 recipe that the GPU repeats
  operation for operation (IEEE-rounded +, -, *, /, no fused multiply-add):
  ln t = e ln 2 + 2 atanh(s), t = m 2^e with m in [sqrt(1/2), sqrt(2)),
  s = (m - 1) / (m + 1), atanh(s) = s (1 + s^2/3 + s^4/5 + s^6/7 + s^8/9).
  With that range m - 1 is exact and t near 1 keeps e = 0, so the relative
  error stays a few ulp even as t -> 1; the Gumbel transform needs exactly
  that, since -ln u -> 0 as u -> 1.  Both sides then draw the same tokens bit
  for bit.  The recipe's error against ln is below 3e-7 relative and the
  Gumbel noise is within 2e-6 of -ln(-ln u) for every one of the 2^23
  uniforms (both pinned in the tests), far inside what a sampler can show.
* z / T is one IEEE fp32 division (bf16 logits are widened exactly first).
"""

import numpy as np

from . import accept as _acc

_M0, _M1 = np.uint64(0xD2511F53), np.uint64(0xCD9E8D57)
_W0, _W1 = np.uint32(0x9E3779B9), np.uint32(0xBB67AE85)
_MASK = np.uint64(0xFFFFFFFF)


def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds.  ctr: uint32 array [..., 4]; key: uint32 [..., 2]."""
    c = [np.asarray(ctr[..., i], dtype=np.uint32) for i in range(4)]
    k0 = np.asarray(key[..., 0], dtype=np.uint32)
    k1 = np.asarray(key[..., 1], dtype=np.uint32)
    for r in range(10):
        if r > 0:
            k0 = (k0 + _W0).astype(np.uint32)
            k1 = (k1 + _W1).astype(np.uint32)
        p0 = c[0].astype(np.uint64) * _M0
        p1 = c[2].astype(np.uint64) * _M1
        hi0, lo0 = (p0 >> np.uint64(32)).astype(np.uint32), (p0 & _MASK).astype(np.uint32)
        hi1, lo1 = (p1 >> np.uint64(32)).astype(np.uint32), (p1 & _MASK).astype(np.uint32)
        c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
    return np.stack(c, axis=-1)


def uniforms(seed, round_, seq, node, vocab):
    """u_w for w < vocab of row (seq, node) in round ``round_``: float32 in (0, 1)."""
    w = np.arange(vocab, dtype=np.uint64)
    ctr = np.zeros((vocab, 4), dtype=np.uint32)
    ctr[:, 0] = (w >> np.uint64(2)).astype(np.uint32)
    ctr[:, 1] = node
    ctr[:, 2] = seq
    ctr[:, 3] = round_
    key = np.zeros((vocab, 2), dtype=np.uint32)
    key[:, 0] = np.uint32(seed & 0xFFFFFFFF)
    key[:, 1] = np.uint32((seed >> 32) & 0xFFFFFFFF)
    x = philox4x32_10(ctr, key)[np.arange(vocab), (w & np.uint64(3)).astype(np.int64)]
    return ((x >> np.uint32(9)).astype(np.float32) + np.float32(0.5)) * np.float32(2.0 ** -23)


_LN2 = np.float32(0.6931471805599453)
_ODD = [np.float32(1.0 / k) for k in (9, 7, 5, 3)]
_SQRT2_MANT = np.uint32(0x3504F3)   # mantissa field of sqrt(2) rounded down


def ln_f32(t):
    """ln t for positive normal float32 t, by the fixed recipe of the module header."""
    t = np.asarray(t, dtype=np.float32)
    bits = t.view(np.uint32)
    e = ((bits >> np.uint32(23)) & np.uint32(0xFF)).astype(np.int32) - 127
    mant = bits & np.uint32(0x007FFFFF)
    high = mant > _SQRT2_MANT           # m >= sqrt(2): halve m, so m in [sqrt(1/2), sqrt(2))
    e = e + high.astype(np.int32)
    m = (mant | np.where(high, np.uint32(0x3F000000), np.uint32(0x3F800000))).view(np.float32)
    s = (m - np.float32(1.0)) / (m + np.float32(1.0))
    s2 = s * s
    acc = _ODD[0]
    for c in _ODD[1:]:
        acc = acc * s2 + c
    acc = acc * s2 + np.float32(1.0)
    atanh2 = np.float32(2.0) * (s * acc)
    return e.astype(np.float32) * _LN2 + atanh2


def gumbel(u):
    """g = -ln(-ln u) in float32 by the fixed recipe."""
    return -ln_f32(-ln_f32(u))


def _as_f32(z):
    if hasattr(z, "detach"):
        t = z.detach().to("cpu")
        if str(t.dtype) in ("torch.bfloat16", "torch.float16"):
            t = t.float()
        z = t.numpy()
    return np.asarray(z, dtype=np.float32)


def sample_row(z, temperature, seed, round_, seq, node):
    """The draw from softmax(z / T) of one row: argmax of z / T + g, lowest index on ties."""
    z = _as_f32(z)
    y = z / np.float32(temperature) + gumbel(uniforms(seed, round_, seq, node, z.shape[0]))
    return int(np.argmax(y))


def sampling_walk(logits, parents, tokens, temperature, seed, round_, seq):
    """One sequence's sampling walk.  Returns (draws of every row, a, path, next_root)."""
    n = len(parents)
    draws = [sample_row(logits[v], temperature, seed, round_, seq, v) for v in range(n)]
    a, path, nr = _acc.greedy_walk(draws, parents, tokens)
    return draws, a, path, nr
