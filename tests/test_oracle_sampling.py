"""Pins for the sampling-walk oracle (CPU only): Philox4x32-10 against its
published known-answer vectors, the fixed fp32 logarithm against ln, the
Gumbel noise's moments, the Gumbel-max draw against softmax by a chi-square
test, and the whole sampling walk on the tiny decoder: the committed tokens'
joint distribution equals that of sampling the target token by token."""

import math

import numpy as np
import pytest
from scipy import stats

from oracle import accept as OA
from oracle import sampling as S
from oracle import tiny_model as T


def _kat(ctr, key):
    return [int(v) for v in S.philox4x32_10(np.array([ctr], np.uint32), np.array([key], np.uint32))[0]]


def test_philox_known_answers():
    # Random123's known-answer vectors for Philox4x32-10
    assert _kat([0, 0, 0, 0], [0, 0]) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert _kat([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2) == [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]
    assert _kat([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0]) == \
        [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]


def test_uniforms_are_open_interval_and_uniform():
    u = S.uniforms(seed=12345, round_=3, seq=1, node=2, vocab=200000)
    assert u.dtype == np.float32 and u.min() > 0 and u.max() < 1
    # every value the mapping can take is exact, inside (0, 1) and distinct
    k = np.arange(2 ** 23, dtype=np.uint32)
    uk = (k.astype(np.float32) + np.float32(0.5)) * np.float32(2.0 ** -23)
    assert np.array_equal(uk.astype(np.float64), (k.astype(np.float64) + 0.5) / 2.0 ** 23)
    assert uk[0] == 2.0 ** -24 and uk[-1] == 1 - 2.0 ** -24
    assert stats.kstest(u.astype(np.float64), "uniform").pvalue > 1e-3
    assert not np.array_equal(u, S.uniforms(seed=12345, round_=4, seq=1, node=2, vocab=200000))


def test_fixed_logarithm_matches_ln():
    one = np.float32(1.0)
    near_one = np.concatenate([one - np.arange(1, 5000, dtype=np.float32) * np.float32(2.0 ** -24),
                               one + np.arange(1, 5000, dtype=np.float32) * np.float32(2.0 ** -23)])
    sqrt2 = np.float32(np.sqrt(2.0))
    around_sqrt2 = np.nextafter(sqrt2, np.float32(np.inf)) * np.float32(2.0) ** np.arange(-3, 3, dtype=np.float32)
    t = np.concatenate([np.float32(2.0) ** np.arange(-126, 127, dtype=np.float32),
                        np.random.default_rng(0).uniform(1e-8, 30.0, 100000).astype(np.float32),
                        near_one, around_sqrt2, sqrt2 * np.float32(2.0) ** np.arange(-3, 3, dtype=np.float32),
                        np.array([np.finfo(np.float32).tiny, np.finfo(np.float32).max], np.float32)])
    ref = np.log(t.astype(np.float64))
    got = S.ln_f32(t).astype(np.float64)
    err = np.abs(got - ref) / np.where(ref == 0, 1.0, np.abs(ref))   # relative, also as t -> 1
    assert err.max() < 3e-7
    assert S.ln_f32(np.float32(1.0)) == 0.0


def test_gumbel_noise_is_accurate_for_every_uniform():
    """All 2^23 uniforms the generator can produce: the fixed-recipe Gumbel
    value is within 2e-6 of -ln(-ln u) (the largest u = 1 - 2^-24 gives
    ln 2^24 - ..., about 16.64; the smallest u = 2^-24 about -2.81)."""
    k = np.arange(2 ** 23, dtype=np.uint32)
    u = (k.astype(np.float32) + np.float32(0.5)) * np.float32(2.0 ** -23)
    g = S.gumbel(u).astype(np.float64)
    ref = -np.log(-np.log(u.astype(np.float64)))
    assert np.abs(g - ref).max() < 2e-6
    assert abs(g[-1] - (-np.log(-np.log1p(-2.0 ** -24)))) < 1e-5 and abs(g[0] + np.log(24 * np.log(2))) < 1e-5


def test_gumbel_moments():
    g = S.gumbel(S.uniforms(seed=7, round_=0, seq=0, node=0, vocab=400000)).astype(np.float64)
    assert abs(g.mean() - 0.5772156649) < 0.01            # Euler-Mascheroni
    assert abs(g.var() - math.pi ** 2 / 6) < 0.03


def test_gumbel_max_draws_follow_softmax():
    z = np.array([0.3, -1.0, 2.0, 0.0, 1.2, -0.5], dtype=np.float32)
    for temperature in (1.0, 0.5):
        zz = z.astype(np.float64) / temperature
        p = np.exp(zz - zz.max())
        p /= p.sum()
        counts = np.zeros(len(z))
        for r in range(6000):
            counts[S.sample_row(z, temperature, seed=99, round_=r, seq=0, node=0)] += 1
        assert stats.chisquare(counts, p * counts.sum()).pvalue > 1e-3


def test_ties_and_masked_tokens():
    z = np.array([-np.inf, 5.0, -np.inf], dtype=np.float32)
    assert all(S.sample_row(z, 1.0, seed=1, round_=r, seq=0, node=0) == 1 for r in range(50))


def _joint_exact(m, prompt, k):
    """p(t1..tk | prompt) of sampling the target token by token, as a dict."""
    out = {(): 1.0}
    for _ in range(k):
        nxt = {}
        for seq, pr in out.items():
            lg, _ = m.forward_causal(list(prompt) + list(seq))
            p = np.exp(lg[-1] - lg[-1].max())
            p /= p.sum()
            for t in range(m.vocab):
                nxt[seq + (t,)] = pr * p[t]
        out = nxt
    return out


def test_sampling_walk_preserves_the_target_distribution():
    """Two tokens after the prompt, GLANCE rounds with the sampling walk against
    token-by-token sampling of a 12-token tiny decoder (chi-square)."""
    m = T.TinyDecoder(3, vocab=12, d_model=16, n_layers=1, n_q_heads=2, n_kv_heads=1, head_dim=8, d_ff=32)
    prompt = [1, 5, 7]
    exact = _joint_exact(m, prompt, 3)   # root t1, then t2, t3
    lg0, _ = m.forward_causal(prompt)
    counts = {}
    n_runs = 3000
    rng = np.random.default_rng(0)
    for run in range(n_runs):
        seed = 1000 + run
        out = []
        # the root: a draw from the prompt's last row (node 0 of a one-node tree)
        root = S.sample_row(lg0[-1].astype(np.float32), 1.0, seed, 0, 0, 0)
        out.append(root)
        rnd = 1
        while len(out) < 3:
            ctx = list(prompt) + out[:-1]
            # a small tree: two children of the root, one grandchild under the first
            kids = rng.choice(m.vocab, size=2, replace=False)
            parents, tokens = [-1, 0, 0, 1], [out[-1], int(kids[0]), int(kids[1]), int(rng.integers(m.vocab))]
            rows = m.verify_tree(ctx, parents, tokens)
            _, a, path, nr = S.sampling_walk(rows.astype(np.float32), parents, tokens, 1.0, seed, rnd, 0)
            out.extend(int(tokens[c]) for c in path[1:])
            out.append(int(nr))
            rnd += 1
        key = tuple(out[:3])
        counts[key] = counts.get(key, 0) + 1
    # bin outcomes with a small expected count together
    keys = sorted(exact, key=lambda k: -exact[k])
    obs, exp, rest_o, rest_e = [], [], 0, 0.0
    for k in keys:
        e = exact[k] * n_runs
        if e >= 8:
            obs.append(counts.get(k, 0))
            exp.append(e)
        else:
            rest_o += counts.get(k, 0)
            rest_e += e
    obs.append(rest_o)
    exp.append(rest_e)
    assert len(obs) >= 8
    assert stats.chisquare(obs, np.array(exp) * sum(obs) / sum(exp)).pvalue > 1e-3


def test_gumbel_bound_by_leading_zeros():
    """g(u) <= -ln(1 - u) <= (clz(r) - 8) ln 2 with r = 2^23 - 1 - k for the
    uniform u = (k + 0.5) 2^-23 (since -ln u >= 1 - u and 1 - u >= r 2^-23).
    For u >= 1/2, clz(r) - 8 = min(L, 23) + 1 with L the leading one bits of
    k; for u < 1/2 the same expression with L the leading zero bits is >= ln 2,
    above g(1/2) = -ln ln 2.  So (min(L, 23) + 1) ln 2, L the leading bits
    equal to the top bit, bounds the noise from the integer alone, which lets
    a sampler skip the logarithms of tokens that cannot win; (min(L, 23) - 1)
    ln 2 (u >= 1/2) and -2.82 (u < 1/2) bound it from below, which gives a
    sampler a running best before any logarithm.  Checked for every k on the
    fixed recipe's values, with 2^-16 to spare for its rounding."""
    k = np.arange(2 ** 23, dtype=np.uint32)
    u = (k.astype(np.float32) + np.float32(0.5)) * np.float32(2.0 ** -23)
    g = S.gumbel(u).astype(np.float64)
    top = (k >> np.uint32(22)) & np.uint32(1)
    flipped = np.where(top == 1, np.uint32(0x7FFFFF) - k, k).astype(np.int64)   # leading equal bits -> zeros
    lead = np.full(k.shape, 23, dtype=np.int64)
    nz = flipped > 0
    lead[nz] = 22 - np.floor(np.log2(flipped[nz].astype(np.float64))).astype(np.int64)
    bound = (np.minimum(lead, 23) + 1) * np.log(2.0)
    assert np.all(g <= bound + 2.0 ** -16)
    # and from below: for u >= 1/2, -ln u <= (1 - u) / u <= 2 (1 - u), so
    # g >= -ln 2 - ln(1 - u) >= (min(L, 23) - 1) ln 2; for u < 1/2, g >= g(2^-24) > -2.82
    top1 = top == 1
    lower = np.where(top1, (np.minimum(lead, 23) - 1) * np.log(2.0), -2.82)
    assert np.all(g >= lower)
    # a tighter integer-only form: with r = 2^23 - 1 - k and F the fp32 bits of
    # float(r), F 2^-23 - 127 <= log2 r (exponent plus mantissa fraction, since
    # log2(1 + f) >= f on [0, 1]), so g <= -ln(1 - u) <= (23 - (F 2^-23 - 127)) ln 2;
    # r = 0 gives 150 ln 2, far above the largest noise.  Computed in fp32 as a
    # sampler would (the scaling by 2^-23 is exact).
    r32 = (np.uint32(0x7FFFFF) - k).astype(np.uint32)
    lg = r32.astype(np.float32).view(np.uint32).astype(np.float32) * np.float32(2.0 ** -23) - np.float32(127.0)
    tight = (np.float32(23.0) - lg).astype(np.float64) * np.log(2.0)
    assert np.all(g <= tight + 2.0 ** -16)
    assert np.mean(tight - g) < 0.5 < np.mean(bound - g)   # tighter on average than the leading-bit form
    # a tighter lower bound for u >= 1/2: -ln u <= (1 - u) / u gives
    # g >= -ln(1 - u) - 2 (1 - u), and with F the fp32 bits of float(r + 1),
    # log2(r + 1) <= F 2^-23 - 127 + 0.0861 (the largest gap between
    # log2(1 + f) and f), so g >= (23 - 0.0862 - (F 2^-23 - 127)) ln 2 - 2 (r + 1) 2^-23
    r1 = (np.uint32(0x800000) - k).astype(np.uint32)
    lg1 = r1.astype(np.float32).view(np.uint32).astype(np.float32) * np.float32(2.0 ** -23) - np.float32(127.0)
    lo_tight = (np.float32(22.9138) - lg1) * np.float32(0.6931472) - \
        np.float32(2.0) * (r1.astype(np.float32) * np.float32(2.0 ** -23))
    assert np.all(g[top1] >= lo_tight[top1].astype(np.float64) + 2.0 ** -16)
    # the same bound read as clz(r) - 8 for u >= 1/2
    r = (np.uint32(0x7FFFFF) - k).astype(np.int64)
    hi = top == 1
    clz = np.where(r > 0, 31 - np.floor(np.log2(np.maximum(r, 1).astype(np.float64))).astype(np.int64), 32)
    assert np.array_equal((clz - 8)[hi], (np.minimum(lead, 23) + 1)[hi])
