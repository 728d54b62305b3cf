"""Pins of the oracle's rANS coder (the entropy coder the paper pairs with the
wavefront decode, Sec. III-C; symbols under the mean-scale Gaussian of
Sec. II-A).  Each check ties it to something outside it:

* tables: every level sums to 2^16 with every frequency >= 1, is symmetric,
  has the support ceil(6 T_l), and each frequency is 1 + floor(p (2^16 - K))
  for the Gaussian mass p evaluated independently with scipy (s = 0 also takes
  what the rounding left over); the code-length
  loss against the exact distribution is below 0.05 bits a symbol;
* three single-symbol streams worked by hand (tests/golden);
* round trip of random symbols at random levels, with escapes of one, two and
  three chunks and the int32 extremes;
* code length: every stream's size is its information content plus 32..64
  bits (the final state's excess over the initial one), to 1 bit (a coder
  using other probabilities than its tables, or tables other than the
  Gaussian, fails this);
* the model decode that reads its symbols from the streams equals the decode
  from the symbols themselves.
"""
import os

import numpy as np
import pytest
from scipy.stats import norm

import oracle
from paper_2607_19082_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def level_freqs(n, base, cum, l):
    c = cum[base[l]:base[l + 1]].astype(np.int64)
    return c, np.diff(c)


def gauss_mass(n, sigma):
    s = np.arange(-n, n + 1)
    p = norm.cdf((s + 0.5) / sigma) - norm.cdf((s - 0.5) / sigma)
    return np.append(p, 2 * norm.sf((n + 0.5) / sigma))


def test_tables_against_the_gaussian():
    t = inputs.scale_table()
    n, base, cum = oracle.rans_tables(t)
    for l, sigma in enumerate(t.astype(np.float64)):
        assert n[l] == max(1, int(np.ceil(6 * sigma)))
        c, f = level_freqs(n, base, cum, l)
        K = 2 * n[l] + 2
        assert len(f) == K and c[0] == 0 and c[-1] == 1 << 16
        assert f.min() >= 1
        assert np.array_equal(f[:2 * n[l] + 1], f[:2 * n[l] + 1][::-1])
        p = gauss_mass(n[l], sigma)
        R = (1 << 16) - K
        d = p * R - (f - 1)
        assert d[n[l]] <= 1e-6                 # the mode takes what rounding left over
        d[n[l]] = 0.5
        assert np.all(d > -1e-6) and np.all(d < 1 + 1e-6), l
        q = f / 65536.0
        kl = np.sum(p[p > 0] * np.log2(p[p > 0] / q[p > 0]))
        assert kl < (1e-3 if sigma < 10 else 0.05), (l, kl)


def test_hand_worked_streams():
    table = inputs.scale_table()
    with open(os.path.join(GOLDEN, "rans_level0_examples.txt")) as f:
        rows = [list(map(int, line.split())) for line in f if line.strip() and not line.startswith("#")]
    assert len(rows) == 3
    for s, *words in rows:
        assert all(0 <= v < 2 ** 32 for v in words)
        sym = np.array(s, np.int32).reshape(1, 1, 1, 1)
        bits, off = oracle.rans_encode(sym, np.zeros_like(sym), table)
        assert list(bits) == words and list(off) == [0, len(words)]
        assert oracle.rans_decode(bits, off, np.zeros_like(sym), table)[0, 0, 0, 0] == s


def random_case(seed, B=2, H=3, W=17, M=5):
    rng = np.random.default_rng(seed)
    t = inputs.scale_table()
    idx = rng.integers(0, len(t), size=(B, H, W, M)).astype(np.int32)
    sigma = t[idx].astype(np.float64)
    sym = np.rint(rng.normal(size=idx.shape) * sigma).astype(np.int64)
    # escapes: one, two and three chunks, and the int32 extremes
    ext = [2 ** 31 - 1, -2 ** 31, 40000, -40000, 2 ** 20 + 5, -(2 ** 29), 5000, -1600]
    flat = sym.reshape(-1)
    pos = rng.choice(flat.size, size=len(ext), replace=False)
    flat[pos] = ext
    return t, np.clip(sym, -2 ** 31, 2 ** 31 - 1).astype(np.int32), idx


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_round_trip(seed):
    t, sym, idx = random_case(seed)
    bits, off = oracle.rans_encode(sym, idx, t)
    assert off[-1] == len(bits)
    assert np.array_equal(oracle.rans_decode(bits, off, idx, t), sym)


def test_code_length_matches_information_content():
    t, sym, idx = random_case(3, B=1, H=4, W=400, M=3)
    sym = np.clip(sym, -6 * t.max(), 6 * t.max()).astype(np.int32)   # escapes of one chunk at most
    n, base, cum = oracle.rans_tables(t)
    bits, off = oracle.rans_encode(sym, idx, t)
    B, H, W, M = sym.shape
    for i in range(H):
        for c in range(M):
            info = 0.0
            for j in range(W):
                l, s = idx[0, i, j, c], sym[0, i, j, c]
                cl, f = level_freqs(n, base, cum, l)
                u = s + n[l] if abs(s) <= n[l] else 2 * n[l] + 1
                info += 16 - np.log2(f[u])
                if u == 2 * n[l] + 1:                # plus 16 bits per 15-bit chunk of the escape value
                    e = 2 * (abs(int(s)) - n[l] - 1) + (s < 0)
                    info += 16 * max(1, -(-int(e).bit_length() // 15))
            k = i * M + c
            size = 32.0 * (int(off[k + 1]) - int(off[k]))
            assert info + 32 - 1 <= size <= info + 64 + 1, (i, c, size, info)


@pytest.mark.parametrize("B,H,W", [(1, 5, 7), (2, 4, 6)])
def test_model_decode_from_streams(B, H, W):
    M = 16
    w = inputs.make_weights(M, 1)
    table = inputs.scale_table()
    psi = inputs.make_psi(B, H, W, M)
    sym = inputs.make_symbols(B, H, W, M, 2.0, 32)
    m = oracle.Model(w, table, H, W, B)
    ref = m.decode(psi, sym)
    bits, off = oracle.rans_encode(sym, ref["idx"][..., 0, :], table)
    got, s = m.decode_bits(psi, bits, off)
    assert np.array_equal(s, sym)
    assert all(np.array_equal(got[k], ref[k]) for k in ref)
    # streams coded at other scale indices do not give the symbols back
    other, off2 = oracle.rans_encode(sym, (ref["idx"][..., 0, :] + 9) % len(table), table)
    try:
        _, s2 = m.decode_bits(psi, other, off2)
        assert not np.array_equal(s2, sym)
    except RuntimeError:
        pass
