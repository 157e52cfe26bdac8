"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle through a route that does not retype its own
formula: the paper's unsigned-code mask applied bit by bit (brute.py), a
bitwise mask, hand-worked values, numpy's int64 matmul, an im2col
convolution, the bit-plane identity, exact rational dequantisation, and
properties any correct mask must have.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import brute
from conftest import read_golden

from paper_2608_03057_amd import inputs

RNG = np.random.default_rng(12345)
ALL_W = np.arange(-128, 128, dtype=np.int64)


def rand_i8(shape, rng=RNG):
    return rng.integers(-128, 128, size=shape, dtype=np.int64).astype(np.int8)


# ------------------------------------------------------------------ the mask

@pytest.mark.parametrize("b", range(1, 9))
def test_mask_exhaustive_vs_unsigned_codes(b):
    """Sec. 3.1 Eq. truncquant + Sec. 3.2.1 Eqs. lsb_extraction/lsb_masking
    on the unsigned code Q = w + 128, one bit at a time, for every w."""
    got = oracle.mask(ALL_W.astype(np.int8), b).astype(np.int64)
    want = np.array([brute.masked_weight(int(w), b) for w in ALL_W])
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("b", range(1, 9))
def test_mask_exhaustive_vs_bitwise_and(b):
    """Dropping the k low two's-complement bits is an AND with ~(2^k - 1)."""
    k = 8 - b
    got = oracle.mask(ALL_W.astype(np.int8), b)
    want = (ALL_W & ~((1 << k) - 1)).astype(np.int8)
    np.testing.assert_array_equal(got, want)


def test_mask_worked_values():
    rows = read_golden("mask_worked_values.txt")
    assert len(rows) >= 10
    for w, b, wb in rows:
        assert int(oracle.mask(np.array([w], np.int8), b)[0]) == wb, (w, b)
        assert brute.masked_weight(w, b) == wb, (w, b)


def test_mask_properties():
    W = ALL_W.astype(np.int8)
    for b in range(1, 9):
        k = 8 - b
        Wb = oracle.mask(W, b).astype(np.int64)
        # idempotent
        np.testing.assert_array_equal(oracle.mask(Wb.astype(np.int8), b), Wb)
        # bounded: 0 <= W - W_b <= 2^k - 1
        d = ALL_W - Wb
        assert d.min() >= 0 and d.max() <= (1 << k) - 1
        # App. G.2 Eq. hw_multi_lsb: the dropped block is sum_{p<k} 2^p bit_p(W)
        u = ALL_W & 0xFF
        lsb = sum(((u >> p) & 1) << p for p in range(k)) if k else 0
        np.testing.assert_array_equal(d, lsb)
        # the result has no bit set below position k
        assert np.all((Wb & ((1 << k) - 1)) == 0)
        # nested / monotone in b
        for b2 in range(1, b + 1):
            Wb2 = oracle.mask(W, b2).astype(np.int64)
            np.testing.assert_array_equal(oracle.mask(Wb.astype(np.int8), b2), Wb2)
            assert np.all(Wb2 <= Wb) and np.all(Wb <= ALL_W)
    # b = 8 is the identity; b = 1 keeps only the sign plane
    np.testing.assert_array_equal(oracle.mask(W, 8), W)
    assert set(oracle.mask(W, 1).tolist()) == {-128, 0}


@pytest.mark.parametrize("b", [0, 9, -1, 100])
def test_mask_rejects_bits_outside_1_8(b):
    with pytest.raises(ValueError):
        oracle.mask(np.zeros(4, np.int8), b)


# --------------------------------------------------------------- the product

@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (3, 5, 7), (17, 33, 64), (40, 24, 1153)])
def test_b8_equals_numpy_int64_matmul(M, N, K):
    X, W = rand_i8((M, K)), rand_i8((N, K))
    acc, _ = oracle.masked_linear(X, W, 1.0, np.ones(N, np.float32), 8)
    np.testing.assert_array_equal(acc, X.astype(np.int64) @ W.astype(np.int64).T)


@pytest.mark.parametrize("b", range(1, 9))
def test_masked_product_linearity(b):
    """acc(X, W_b) = X W^T - X (W - W_b)^T, with W_b from a bitwise mask."""
    M, N, K = 9, 13, 301
    X, W = rand_i8((M, K)), rand_i8((N, K))
    k = 8 - b
    dropped = W.astype(np.int64) & ((1 << k) - 1)
    want = X.astype(np.int64) @ W.astype(np.int64).T - X.astype(np.int64) @ dropped.T
    acc, _ = oracle.masked_linear(X, W, 1.0, np.ones(N, np.float32), b)
    np.testing.assert_array_equal(acc, want)


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_agreement(seed):
    rng = np.random.default_rng(seed)
    M, N, K = (int(v) for v in rng.integers(1, 17, size=3))
    X, W = rand_i8((M, K), rng), rand_i8((N, K), rng)
    X[0, 0] = -128
    W[0, 0] = -128
    sw = rng.uniform(1e-3, 1e-2, size=N).astype(np.float32)
    bias = rng.uniform(-1, 1, size=N).astype(np.float32)
    for b in range(1, 9):
        acc, y = oracle.masked_linear(X, W, 0.02, sw, b, bias)
        bacc, by = brute.masked_linear(X.tolist(), W.tolist(), 0.02, sw.tolist(), b,
                                       bias.tolist())
        np.testing.assert_array_equal(acc, np.array(bacc))
        np.testing.assert_allclose(y, np.array(by), rtol=1e-14, atol=1e-14)


def test_special_cases():
    N, K = 7, 40
    W = rand_i8((N, K))
    sw = np.ones(N, np.float32)
    for b in range(1, 9):
        acc, _ = oracle.masked_linear(np.zeros((3, K), np.int8), W, 1.0, sw, b)
        assert not acc.any()
        # a one-hot activation row returns the masked weight column
        for j in (0, 17, K - 1):
            x = np.zeros((1, K), np.int8)
            x[0, j] = 1
            acc, _ = oracle.masked_linear(x, W, 1.0, sw, b)
            want = np.array([brute.masked_weight(int(W[n, j]), b) for n in range(N)])
            np.testing.assert_array_equal(acc[0], want)


def test_empty_shapes():
    acc, y = oracle.masked_linear(np.zeros((0, 5), np.int8), np.zeros((3, 5), np.int8),
                                  1.0, np.ones(3, np.float32), 4)
    assert acc.shape == (0, 3)
    acc, y = oracle.masked_linear(np.zeros((2, 0), np.int8), np.zeros((3, 0), np.int8),
                                  1.0, np.ones(3, np.float32), 4)
    assert not acc.any() and not y.any()


def test_overflow_bound():
    """|acc| <= 128 * 128 * K: K = 131071 fits int32, K = 131072 does not."""
    for K, ok in ((131071, True), (131072, False)):
        X = np.full((1, K), -128, np.int8)
        W = np.full((1, K), -128, np.int8)
        if ok:
            acc, _ = oracle.masked_linear(X, W, 1.0, np.ones(1, np.float32), 8)
            assert int(acc[0, 0]) == 16384 * K
        else:
            with pytest.raises(OverflowError):
                oracle.masked_linear(X, W, 1.0, np.ones(1, np.float32), 8)


def test_entries_match_full():
    M, N, K = 20, 30, 77
    X, W = rand_i8((M, K)), rand_i8((N, K))
    sw = RNG.uniform(1e-3, 1e-2, size=N).astype(np.float32)
    bias = RNG.uniform(-1, 1, size=N).astype(np.float32)
    rows = RNG.integers(0, M, 50)
    cols = RNG.integers(0, N, 50)
    for b in (8, 5, 1):
        acc, y = oracle.masked_linear(X, W, 0.02, sw, b, bias)
        ea, ey = oracle.masked_linear_entries(X, W, 0.02, sw, b, rows, cols, bias)
        np.testing.assert_array_equal(ea, acc[rows, cols])
        np.testing.assert_array_equal(ey, y[rows, cols])


# ------------------------------------------------------------ dequantisation

def test_dequant_exact_rational():
    """y = acc * sx * sw[n] (+ bias): fp64 within 2 roundings of the exact
    rational value (App. A.1 dequantisation, zero points zero)."""
    M, N, K = 6, 11, 50
    X, W = rand_i8((M, K)), rand_i8((N, K))
    sw = RNG.uniform(1e-3, 1e-2, size=N).astype(np.float32)
    bias = RNG.uniform(-1, 1, size=N).astype(np.float32)
    sx = np.float32(0.02)
    for b in (8, 3):
        acc, y = oracle.masked_linear(X, W, float(sx), sw, b, bias)
        for m in range(M):
            for n in range(N):
                exact = Fraction(int(acc[m, n])) * Fraction(float(sx)) * Fraction(float(sw[n])) \
                    + Fraction(float(bias[n]))
                mag = abs(Fraction(int(acc[m, n])) * Fraction(float(sx)) * Fraction(float(sw[n]))) \
                    + abs(Fraction(float(bias[n])))
                assert abs(Fraction(y[m, n]) - exact) <= mag * Fraction(3, 2 ** 53)


def test_dequant_power_of_two_scales_exact():
    M, N, K = 4, 5, 33
    X, W = rand_i8((M, K)), rand_i8((N, K))
    sw = np.array([2.0 ** -e for e in range(7, 7 + N)], np.float32)
    acc, y = oracle.masked_linear(X, W, 0.25, sw, 6)
    np.testing.assert_array_equal(y, acc.astype(np.float64) * 0.25 * sw.astype(np.float64))


# --------------------------------------------------------------- convolution

def im2col_conv(X, Wt, b):
    """3x3/pad 1 conv as an explicit patch matrix times the masked weight."""
    H, Wd, Ci = X.shape
    Co = Wt.shape[0]
    Xp = np.zeros((H + 2, Wd + 2, Ci), np.int64)
    Xp[1:-1, 1:-1] = X
    cols = np.zeros((H * Wd, 9 * Ci), np.int64)
    for h in range(H):
        for w in range(Wd):
            cols[h * Wd + w] = Xp[h:h + 3, w:w + 3, :].reshape(-1)
    k = 8 - b
    Wm = Wt.astype(np.int64) & ~((1 << k) - 1)
    return (cols @ Wm.reshape(Co, -1).T).reshape(H, Wd, Co)


@pytest.mark.parametrize("H,Wd,Ci,Co", [(1, 1, 1, 1), (4, 5, 3, 6), (7, 3, 16, 9)])
def test_conv_direct_vs_im2col(H, Wd, Ci, Co):
    X = rand_i8((H, Wd, Ci))
    Wt = rand_i8((Co, 3, 3, Ci))
    sw = np.ones(Co, np.float32)
    for b in (8, 6, 2):
        acc, _ = oracle.conv3x3(X, Wt, 1.0, sw, b)
        np.testing.assert_array_equal(acc, im2col_conv(X, Wt, b))


def test_conv_single_tap():
    """A centre-only kernel reduces the conv to a per-pixel linear layer."""
    H, Wd, Ci, Co = 5, 6, 8, 4
    X = rand_i8((H, Wd, Ci))
    Wt = np.zeros((Co, 3, 3, Ci), np.int8)
    Wt[:, 1, 1, :] = rand_i8((Co, Ci))
    acc, _ = oracle.conv3x3(X, Wt, 1.0, np.ones(Co, np.float32), 5)
    lin, _ = oracle.masked_linear(X.reshape(-1, Ci), Wt[:, 1, 1, :], 1.0,
                                  np.ones(Co, np.float32), 5)
    np.testing.assert_array_equal(acc.reshape(-1, Co), lin)


def test_conv_entries_match_full():
    H, Wd, Ci, Co = 5, 6, 7, 9
    X = rand_i8((H, Wd, Ci))
    Wt = rand_i8((Co, 3, 3, Ci))
    sw = RNG.uniform(1e-3, 1e-2, Co).astype(np.float32)
    bias = RNG.uniform(-1, 1, Co).astype(np.float32)
    pix = RNG.integers(0, H * Wd, 60)
    cols = RNG.integers(0, Co, 60)
    for b in (8, 4):
        acc, y = oracle.conv3x3(X, Wt, 0.02, sw, b, bias)
        ea, ey = oracle.conv3x3_entries(X, Wt, 0.02, sw, b, pix, cols, bias)
        np.testing.assert_array_equal(ea, acc.reshape(-1, Co)[pix, cols])
        np.testing.assert_array_equal(ey, y.reshape(-1, Co)[pix, cols])


# ---------------------------------------------------------------- bit planes

def words_by_channel(planes, N):
    """[nb, q, kb, r, w, f] plane words as [q, kb, n, w], n = 32*nb + 16*f + r."""
    NB, Q, KB, R, Wn, F = planes.shape
    assert (R, Wn, F) == (16, 4, 2)
    return planes.transpose(1, 2, 0, 5, 3, 4).reshape(Q, KB, NB * 32, 4)[:, :, :N, :]


def unpack(planes, N, K):
    """Bit plane q (q = 7 - p) back to a {0,1} int64 array [8 x N x K].
    Element j: e = j % 128 is sub-step e // 32, half (e % 32) // 16, group
    (e % 16) // 4, byte e % 4; word 2*half + sub-step // 2, and plane p's bit
    at (8*byte + 4*(sub-step % 2) + group + p) mod 32."""
    planes = words_by_channel(planes, N)
    Q, KB, N, _ = planes.shape
    j = np.arange(K)
    r = j % 128
    s, h, i, c = r // 32, (r % 32) // 16, (r % 16) // 4, r % 4
    w = 2 * h + s // 2
    g = 4 * (s % 2) + i
    words = planes[:, j // 128, :, :]                        # [8, K, N, 4]
    words = np.take_along_axis(words, np.broadcast_to(w[None, :, None, None],
                                                      words.shape[:3] + (1,)), 3)[..., 0]
    p = (7 - np.arange(Q))[:, None]                          # [8, 1]
    pos = (8 * c[None, :] + g[None, :] + p) % 32             # [8, K]
    bits = (words.astype(np.int64) >> pos[:, :, None]) & 1
    return bits.transpose(0, 2, 1)


def test_planes_bit_position_worked_example():
    """Positions worked out by hand from the layout definition, as
    (nb, q, kb, r, w, f) and as the flat word index
    (((nb*8 + q)*KB + kb)*16 + r)*8 + 2*w + f, here KB = 1:
    element (0, 0) = 1 (sub-step 0, half 0, group 0, byte 0) sets bit
    (0 + 0 + p=0) = 0 of word (0, 7, 0, 0, 0, 0), flat 7*128 = 896;
    element (0, 5) = -128 (group 1, byte 1) sets bit (8 + 1 + 7) = 16 of
    word (0, 0, 0, 0, 0, 0) of the sign plane, flat 0;
    element (0, 63) = -128 (sub-step 1, half 1, group 3, byte 3: word
    2*1 + 0 = 2) sets bit (24 + 4 + 3 + 7) mod 32 = 6 of word (0, 0, 0, 0, 2, 0),
    flat 4;
    element (0, 100) = 2 (sub-step 3, half 0, group 1, byte 0: word 1) sets
    bit (0 + 4 + 1 + 1) = 6 of word (0, 6, 0, 0, 1, 0) of plane p = 1, flat
    6*128 + 2 = 770;
    element (17, 0) = -128 (channel 17: nb 0, f 1, r 1) sets bit 7 of word
    (0, 0, 0, 1, 0, 1), flat 8 + 1 = 9;
    element (33, 127) = 1 (channel 33: nb 1, f 0, r 1; sub-step 3, half 1,
    group 3, byte 3: word 3) sets bit (24 + 4 + 3 + 0) = 31 of word
    (1, 7, 0, 1, 3, 0), flat (15*16 + 1)*8 + 6 = 1934."""
    W = np.zeros((40, 128), np.int8)
    W[0, 0] = 1
    W[0, 5] = -128
    W[0, 63] = -128
    W[0, 100] = 2
    W[17, 0] = -128
    W[33, 127] = 1
    planes = oracle.pack_planes(W)
    assert planes.shape == (2, 8, 1, 16, 4, 2)
    expect = {896: 1 << 0, 0: 1 << 16, 4: 1 << 6, 770: 1 << 6, 9: 1 << 7, 1934: 1 << 31}
    flat = planes.reshape(-1)
    for idx, v in expect.items():
        assert int(flat[idx]) == v, idx
    assert np.count_nonzero(flat) == len(expect)
    assert planes[0, 7, 0, 0, 0, 0] == 1 and planes[1, 7, 0, 1, 3, 0] == 1 << 31
    assert planes[0, 0, 0, 1, 0, 1] == 1 << 7 and planes[0, 6, 0, 0, 1, 0] == 1 << 6


@pytest.mark.parametrize("N,K", [(1, 1), (5, 31), (7, 32), (3, 100), (4, 300), (40, 200)])
def test_planes_round_trip(N, K):
    W = rand_i8((N, K))
    W[0, 0] = -128
    planes = oracle.pack_planes(W)
    assert planes.shape == ((N + 31) // 32, 8, (K + 127) // 128, 16, 4, 2)
    bits = unpack(planes, N, K)
    coef = np.array([-128] + [1 << p for p in range(6, -1, -1)])   # q = 0 is the sign plane
    np.testing.assert_array_equal(np.tensordot(coef, bits, 1), W.astype(np.int64))
    # every bit past K and past N is zero: the total popcount equals that of
    # the N x K elements
    total = sum(bin(int(v)).count("1") for v in planes.reshape(-1))
    assert total == int(bits.sum())


def unpack_weights(P, N, K):
    """Inverse of the packed layout by reshaping: [NB][KS][half][row][16]."""
    NB, KS = (N + 31) // 32, 4 * ((K + 127) // 128)
    full = np.asarray(P).reshape(NB, KS, 2, 32, 16).transpose(0, 3, 1, 2, 4)
    return full.reshape(NB * 32, KS * 32)


def test_packed_weights_worked_positions():
    """Byte positions derived by hand from the layout definition (unit
    (n//32, k//32) of 1 KB, lane n%32 + 32*((k%32)//16), byte k%16)."""
    N, K = 40, 200                       # KS = 8
    W = np.zeros((N, K), np.int8)
    cases = {(0, 0): 0, (31, 15): 31 * 16 + 15, (0, 16): 32 * 16, (0, 32): 1024,
             (33, 50): ((1 * 8 + 1) * 64 + 33) * 16 + 2, (39, 199): ((8 + 6) * 64 + 7) * 16 + 7}
    for i, (nk, pos) in enumerate(cases.items()):
        W[nk] = i + 1
    P = oracle.pack_weights(W)
    assert P.size == 64 * 256
    for i, (nk, pos) in enumerate(cases.items()):
        assert P[pos] == i + 1, (nk, pos)
    assert np.count_nonzero(P) == len(cases)


@pytest.mark.parametrize("N,K", [(1, 1), (5, 31), (32, 128), (33, 129), (70, 300)])
def test_packed_weights_round_trip(N, K):
    rng = np.random.default_rng(N * 1000 + K)
    W = rng.integers(-128, 128, (N, K), dtype=np.int64).astype(np.int8)
    P = oracle.pack_weights(W)
    assert P.size == 32 * ((N + 31) // 32) * 128 * ((K + 127) // 128)
    full = unpack_weights(P, N, K)
    assert np.array_equal(full[:N, :K], W)
    assert not full[N:].any() and not full[:, K:].any()


@pytest.mark.parametrize("b", range(1, 9))
def test_bit_plane_identity(b):
    """X W_b^T = sum_{p >= 8-b} c_p 2^p X P_p^T, c_7 = -1 (App. G.2: read
    only the top b planes)."""
    M, N, K = 6, 9, 70
    X, W = rand_i8((M, K)), rand_i8((N, K))
    bits = unpack(oracle.pack_planes(W), N, K)
    total = np.zeros((M, N), np.int64)
    for q in range(b):
        p = 7 - q
        c = -1 if p == 7 else 1
        total += c * (1 << p) * (X.astype(np.int64) @ bits[q].T)
    acc, _ = oracle.masked_linear(X, W, 1.0, np.ones(N, np.float32), b)
    np.testing.assert_array_equal(acc, total)


# ------------------------------------------------------------------ schedule

def test_stage_map_golden():
    for row in read_golden("stage_map.txt"):
        T, S, stages = row[0], row[1], row[2:]
        assert len(stages) == T
        assert [oracle.stage_of_step(t, S, T) for t in range(T)] == stages


@pytest.mark.parametrize("t,S,T", [(-1, 4, 20), (20, 4, 20), (0, 0, 20), (0, 5, 4), (0, 1, 0)])
def test_stage_map_rejects(t, S, T):
    with pytest.raises(ValueError):
        oracle.stage_of_step(t, S, T)


def _small_layers(rng):
    layers = []
    for (M, K, N) in ((5, 40, 7), (3, 33, 4)):
        layers.append(dict(X=rand_i8((M, K), rng), W=rand_i8((N, K), rng),
                           sw=rng.uniform(1e-3, 1e-2, N).astype(np.float32)))
    layers.append(dict(kind="conv3x3", X=rand_i8((3, 4, 5), rng), W=rand_i8((6, 3, 3, 5), rng),
                       sw=rng.uniform(1e-3, 1e-2, 6).astype(np.float32)))
    return layers


def test_schedule_properties():
    rng = np.random.default_rng(7)
    layers = _small_layers(rng)
    S, T = 4, 20
    table = rng.integers(2, 9, size=(len(layers), S))
    # a constant-8 table equals the static 8-bit layer
    res = oracle.run_schedule(layers, np.full((len(layers), S), 8), S, T, 0, T, 0.02)
    for layer, (acc, y, b) in zip(layers, res):
        if layer.get("kind") == "conv3x3":
            want = oracle.conv3x3(layer["X"], layer["W"], 0.02, layer["sw"], 8)
        else:
            want = oracle.masked_linear(layer["X"], layer["W"], 0.02, layer["sw"], 8)
        assert b == 8
        np.testing.assert_array_equal(acc, want[0])
    # one step per stage leaves that stage's single-layer result
    for s in range(S):
        t = s * (T // S) + 2
        res = oracle.run_schedule(layers, table, S, T, t, t + 1, 0.02)
        for l, (layer, (acc, y, b)) in enumerate(zip(layers, res)):
            assert b == table[l][s]
            if layer.get("kind") == "conv3x3":
                want = oracle.conv3x3(layer["X"], layer["W"], 0.02, layer["sw"], b)
            else:
                want = oracle.masked_linear(layer["X"], layer["W"], 0.02, layer["sw"], b)
            np.testing.assert_array_equal(acc, want[0])
            np.testing.assert_array_equal(y, want[1])
    # an empty range writes nothing
    assert oracle.run_schedule(layers, table, S, T, 7, 7, 0.02) == [None] * len(layers)
    with pytest.raises(ValueError):
        oracle.run_schedule(layers, table, S, T, 5, 21, 0.02)


# ----------------------------------------------------------------- generator

def test_generator_published_value_and_ranges():
    import torch
    # SplitMix64 from state 0: first output 0xE220A8397B1DCDAF (published)
    v = int(inputs.splitmix64(torch.tensor([0], dtype=torch.int64))) & (2 ** 64 - 1)
    assert v == 0xE220A8397B1DCDAF
    wl = inputs.workload(0)
    X = inputs.x_full(wl, 0)
    assert X.shape == (256, 1152) and int(X.min()) >= -127 and int(X.max()) <= 127
    W = inputs.w_full(wl, 0)
    assert W.shape == (1152, 1152) and abs(float(W.float().std()) - 32) < 1
    sw = inputs.sw_full(wl, 0)
    assert float(sw.min()) >= 1e-3 and float(sw.max()) < 1e-2
    t = inputs.b_table(inputs.workload(4))
    assert t.shape == (112, 4) and int(t.min()) == 2 and int(t.max()) == 8
    assert abs(float(t.float().mean()) - 5) < 0.3
    # counter-based: sampled rows equal the same rows of the full tensor
    rows = [0, 17, 255]
    np.testing.assert_array_equal(inputs.x_rows(wl, 0, rows).numpy(), X[rows].numpy())


# ------------------------------------------- activation quantizer (App. A.1.2)

def test_act_quant_exact_grid_and_ties():
    """Ranges whose scale is exactly 1 or 2: codes are x - min (scaled), and
    halves round to even (round to nearest, ties to even)."""
    a, z, q = oracle.act_quant(np.array([0.0, 2.5, 3.5, 100.0, 255.0], np.float32))
    assert (a, z) == (1.0, 0.0)
    assert q.tolist() == [0, 2, 4, 100, 255]
    a, z, q = oracle.act_quant(np.array([-128.0, -0.5, 0.5, 1.5, 127.0], np.float32))
    assert (a, z) == (1.0, 128.0)
    assert q.tolist() == [0, 128, 128, 130, 255]
    a, z, q = oracle.act_quant(np.array([0.0, 1.0, 3.0, 5.0, 510.0], np.float32))
    assert (a, z) == (2.0, 0.0)
    assert q.tolist() == [0, 0, 2, 2, 255]


def test_act_quant_constant_tensor():
    a, z, q = oracle.act_quant(np.full(7, -3.25, np.float32))
    assert a == 1.0 and z == 3.25 and not q.any()
    assert a * (0 - z) == -3.25          # dequantises to the constant exactly


@pytest.mark.parametrize("seed", range(4))
def test_act_quant_properties(seed):
    """min -> 0, max -> 255, codes monotone in x, and the dequantised value
    alpha (Q - z) within alpha/2 of x (plus single-precision slack, which
    matters when the range is narrow against its offset and z is large)."""
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(5000) * (10.0 ** rng.uniform(-3, 3)) + rng.uniform(-5, 5))
    x = x.astype(np.float32)
    a, z, q = oracle.act_quant(x)
    assert q[np.argmin(x)] == 0 and q[np.argmax(x)] == 255
    order = np.argsort(x, kind="stable")
    assert np.all(np.diff(q[order].astype(np.int64)) >= 0)
    span = float(x.max()) - float(x.min())
    assert abs(a - span / 255) <= 1e-6 * span / 255
    xhat = a * (q.astype(np.float64) - z)
    # single-precision slack of x/alpha + z (and of alpha, z themselves), in
    # units of alpha: a few ulps of the largest magnitude involved
    slack = 8 * 2.0 ** -24 * (np.abs(x.astype(np.float64)) / a + abs(z) + 255)
    assert np.all(np.abs(xhat - x.astype(np.float64)) <= a * (0.5 + slack))


def test_weight_colsums():
    """b = 8 equals the plain row sum; lower b equals the row sum of the
    two's-complement AND mask (a different route from the oracle's floor);
    and the dropped-bit identity colsum_8 - colsum_b = sum of the low bits."""
    rng = np.random.default_rng(3)
    W = rng.integers(-128, 128, (37, 300)).astype(np.int8)
    cs = oracle.weight_colsums(W)
    w64 = W.astype(np.int64)
    assert np.array_equal(cs[7], w64.sum(axis=1))
    for b in range(1, 9):
        k = 8 - b
        anded = w64 & ~((1 << k) - 1)
        assert np.array_equal(cs[b - 1], anded.sum(axis=1)), b
        low = (W.view(np.uint8).astype(np.int64) & ((1 << k) - 1)).sum(axis=1)
        assert np.array_equal(cs[7] - cs[b - 1], low), b


@pytest.mark.parametrize("b", [8, 5, 2])
def test_asym_linear_factored_form_and_signed_codes(b):
    """sum_k alpha (Q - z) sw W_b (the oracle's definition) equals the
    factored zero-point form alpha sw (Q W_b^T - z colsum_b) computed with
    numpy int64 matmul, and acc is the int64 product of the signed codes."""
    rng = np.random.default_rng(b)
    Q = rng.integers(0, 256, (9, 200)).astype(np.uint8)
    W = rng.integers(-128, 128, (11, 200)).astype(np.int8)
    sw = rng.uniform(1e-3, 1e-2, 11).astype(np.float32)
    bias = rng.uniform(-1, 1, 11).astype(np.float32)
    alpha, z = 0.0173, 121.37
    acc, y = oracle.masked_linear_asym(Q, W, alpha, z, sw, b, bias)
    k = 8 - b
    Wb = W.astype(np.int64) & ~((1 << k) - 1)
    colsum = Wb.sum(axis=1)
    accQ = Q.astype(np.int64) @ Wb.T
    assert np.array_equal(acc, (Q.astype(np.int64) - 128) @ Wb.T)
    assert np.array_equal(accQ, acc + 128 * colsum)
    ref = alpha * sw.astype(np.float64) * (accQ - z * colsum) + bias
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_asym_linear_reduces_to_symmetric():
    """With z = 128 and alpha = sx the asymmetric layer is the symmetric one
    on the codes Q - 128."""
    rng = np.random.default_rng(11)
    Q = rng.integers(0, 256, (6, 96)).astype(np.uint8)
    W = rng.integers(-128, 128, (5, 96)).astype(np.int8)
    sw = rng.uniform(1e-3, 1e-2, 5).astype(np.float32)
    for b in (8, 3):
        acc_a, y_a = oracle.masked_linear_asym(Q, W, 0.02, 128.0, sw, b)
        acc_s, y_s = oracle.masked_linear((Q.astype(np.int16) - 128).astype(np.int8), W, 0.02,
                                          sw, b)
        assert np.array_equal(acc_a, acc_s)
        assert np.allclose(y_a, y_s, rtol=1e-12, atol=1e-15)


def test_asym_entries_match_full():
    rng = np.random.default_rng(12)
    Q = rng.integers(0, 256, (13, 150)).astype(np.uint8)
    W = rng.integers(-128, 128, (17, 150)).astype(np.int8)
    sw = rng.uniform(1e-3, 1e-2, 17).astype(np.float32)
    acc, y = oracle.masked_linear_asym(Q, W, 0.05, 100.25, sw, 4)
    rows = rng.integers(0, 13, 40)
    cols = rng.integers(0, 17, 40)
    ae, ye = oracle.masked_linear_asym_entries(Q, W, 0.05, 100.25, sw, 4, rows, cols)
    assert np.array_equal(ae, acc[rows, cols])
    assert np.allclose(ye, y[rows, cols], rtol=1e-13, atol=0)


# ---------------------------------------------------- 16-bit low-rank branch

BF16_WORKED = [
    (1.0, 0x3F80),                      # exact
    (1 + 2 ** -8, 0x3F80),              # halfway between 1 and 1 + 2^-7: even mantissa
    (1 + 3 * 2 ** -8, 0x3F82),          # halfway between 1 + 2^-7 and 1 + 2^-6: even
    (1 + 2 ** -8 + 2 ** -20, 0x3F81),   # just above halfway
    (-2.5, 0xC020),
    (0.0, 0x0000),
    (-0.0, 0x8000),
    (3.140625, 0x4049),                 # 1.5703125 * 2, mantissa 73/128
    (65504.0, 0x4780),                  # largest fp16 value rounds up to 2^16
    (2.0 ** -133, 0x0001),              # smallest bfloat16 subnormal
    (1.5 * 2.0 ** -133, 0x0002),        # subnormal tie: even
]


@pytest.mark.parametrize("x,bits", BF16_WORKED)
def test_bf16_round_worked_values(x, bits):
    assert int(oracle.bf16_round(np.array([x], np.float32))[0]) == bits


def test_bf16_value_decodes():
    got = oracle.bf16_value([0x3F80, 0xC020, 0x0001, 0x4049, 0x3F82, 0x8000])
    assert got.tolist() == [1.0, -2.5, 2.0 ** -133, 3.140625, 1 + 2 ** -6, 0.0]


def test_bf16_round_matches_torch_rne():
    """The frexp/rint route against torch's float32 -> bfloat16 conversion
    (round to nearest even), on random values, exact ties and subnormals."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    base = rng.standard_normal(4000).astype(np.float32) * np.float32(37.0)
    finite = rng.integers(0, 0x7F00, 2000) | (rng.integers(0, 2, 2000) << 15)
    ties = (oracle.bf16_value(finite).astype(np.float32).view(np.uint32)
            | np.uint32(0x8000)).view(np.float32)
    tiny = (rng.integers(1, 1 << 23, 500).astype(np.uint32)).view(np.float32)
    x = np.concatenate([base, ties, tiny, -tiny])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    assert np.array_equal(oracle.bf16_round(x), ref)


def _lowrank_case(seed, M, K, r, N):
    x = inputs.activations_f32(seed, np.arange(M), K, "outlier").numpy()
    D = inputs.bf16_bits(seed, 1, (r, K)).numpy()
    U = inputs.bf16_bits(seed, 2, (N, r)).numpy()
    return x, D, U


def test_lowrank_exact_rational_tiny():
    """T and lr against exact rational arithmetic on the bfloat16 values."""
    x, D, U = _lowrank_case(31, 3, 7, 2, 4)
    T, lr = oracle.lowrank(x, D, U)
    xt = [[Fraction(float(v)) for v in row] for row in oracle.bf16_value(oracle.bf16_round(x))]
    Df = [[Fraction(float(v)) for v in row] for row in oracle.bf16_value(D)]
    Uf = [[Fraction(float(v)) for v in row] for row in oracle.bf16_value(U)]
    for m in range(3):
        Tm = [sum(xt[m][k] * Df[j][k] for k in range(7)) for j in range(2)]
        for j in range(2):
            assert abs(Fraction(T[m, j]) - Tm[j]) <= abs(Tm[j]) * Fraction(1, 2 ** 50)
        for n in range(4):
            e = sum(Tm[j] * Uf[n][j] for j in range(2))
            mag = sum(abs(Tm[j] * Uf[n][j]) for j in range(2))
            assert abs(Fraction(lr[m, n]) - e) <= mag * Fraction(1, 2 ** 48)


def test_lowrank_merged_weight():
    """(x~ D^T) U^T equals x~ (U D)^T: the branch is one rank-r linear map."""
    x, D, U = _lowrank_case(32, 9, 300, 16, 40)
    _, lr = oracle.lowrank(x, D, U)
    xt = oracle.bf16_value(oracle.bf16_round(x))
    merged = xt @ (oracle.bf16_value(U) @ oracle.bf16_value(D)).T
    mag = np.abs(xt) @ (np.abs(oracle.bf16_value(U)) @ np.abs(oracle.bf16_value(D))).T
    assert np.all(np.abs(lr - merged) <= 1e-13 * mag)


def test_lowrank_one_hot():
    """D = e_j e_k^T, U = 2 e_n e_j^T: the branch copies 2 * bf16(x[:, k]) to
    column n and zero elsewhere."""
    x, _, _ = _lowrank_case(33, 5, 12, 4, 6)
    D = np.zeros((4, 12), np.uint16)
    U = np.zeros((6, 4), np.uint16)
    D[2, 7] = 0x3F80                     # 1.0
    U[3, 2] = 0x4000                     # 2.0
    T, lr = oracle.lowrank(x, D, U)
    xt = oracle.bf16_value(oracle.bf16_round(x))
    expect = np.zeros((5, 6))
    expect[:, 3] = 2.0 * xt[:, 7]
    assert np.array_equal(lr, expect)
    assert np.array_equal(T[:, 2], xt[:, 7]) and not T[:, [0, 1, 3]].any()


def test_lowrank_entries_match_full():
    x, D, U = _lowrank_case(34, 11, 130, 32, 21)
    _, lr = oracle.lowrank(x, D, U)
    rng = np.random.default_rng(3)
    rows, cols = rng.integers(0, 11, 50), rng.integers(0, 21, 50)
    e = oracle.lowrank_entries(x, D, U, rows, cols)
    assert np.allclose(e, lr[rows, cols], rtol=1e-13, atol=0)


# ------------------------------------------------------ weight quantizer

def test_weight_quant_exact_grid_and_clamp():
    """A row on the grid min + j alpha (alpha = 2/256 exactly): code j, the
    midpoints floor to j, and max (j = 256) clamps to 255."""
    j = np.arange(257)
    on = np.concatenate([-1.0 + j / 128.0, [0.0]]).astype(np.float32)
    mid = np.concatenate([[-1.0], -1.0 + (np.arange(256) + 0.5) / 128.0, [1.0]])
    W = np.stack([on, mid.astype(np.float32)])
    Q, alpha, z, sw = oracle.weight_quant(W)
    assert alpha.tolist() == [2.0 ** -7] * 2 and z.tolist() == [128.0] * 2
    assert Q[0].tolist() == np.minimum(j, 255).tolist() + [128]
    assert Q[1, 1:257].tolist() == list(range(256)) and Q[1, 0] == 0 and Q[1, 257] == 255
    assert sw[0] == np.float32(np.float32(2.0 ** -7 * 256) / np.float32(255.0))


def test_weight_quant_truncquant_prefix():
    """Eq. truncquant: the (n-1)-bit code is the n-bit code without its LSB,
    for every n, so masking the stored 8-bit code reproduces the coarser
    quantizers; for weights normalised to [0, 1] the 8-bit code is
    floor(256 w) (the printed Q_n = floor(W 2^n), clamped at w = 1)."""
    rng = np.random.default_rng(21)
    W = rng.standard_normal((6, 500)).astype(np.float32)
    Q8 = oracle.weight_quant(W, 8)[0].astype(np.int64)
    for n in range(1, 8):
        Qn = oracle.weight_quant(W, n)[0].astype(np.int64)
        assert np.array_equal(Qn, Q8 >> (8 - n)), n
    u = (rng.integers(0, 4097, (3, 300)) / 4096.0).astype(np.float32)
    u[:, 0], u[:, 1] = 0.0, 1.0
    Qu = oracle.weight_quant(u, 8)[0].astype(np.int64)
    assert np.array_equal(Qu, np.minimum(np.floor(u.astype(np.float64) * 256), 255))


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_weight_quant_properties(seed):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((9, 777)) * rng.uniform(0.01, 3.0, (9, 1))
         + rng.uniform(-2, 2, (9, 1))).astype(np.float32)
    Q, alpha, z, sw = oracle.weight_quant(W)
    for n in range(9):
        assert Q[n, W[n].argmin()] == 0 and Q[n, W[n].argmax()] == 255
        order = np.argsort(W[n], kind="stable")
        assert np.all(np.diff(Q[n, order].astype(int)) >= 0)
        # floor: alpha (Q - z) <= w < alpha (Q + 1 - z), up to fp32 slack
        a, zz = float(alpha[n]), float(z[n])
        w = W[n].astype(np.float64)
        lo = a * (Q[n] - zz)
        slack = 8 * 2.0 ** -24 * (np.abs(w) + a * (abs(zz) + 256))
        assert np.all(lo <= w + slack) and np.all(w < lo + a + slack)
        assert abs(float(sw[n]) - a * 256 / 255) <= 2.0 ** -23 * a


def test_weight_quant_constant_row():
    Q, alpha, z, sw = oracle.weight_quant(np.full((2, 5), -0.5, np.float32))
    assert not Q.any() and alpha.tolist() == [1.0, 1.0] and z.tolist() == [0.5, 0.5]


def test_row_sums():
    X = rand_i8((5, 37))
    assert oracle.row_sums(X).tolist() == [sum(int(v) for v in row) for row in X]


@pytest.mark.parametrize("b", [8, 5, 1])
def test_layer_dequant_reduces_to_masked_linear(b):
    X, W = rand_i8((11, 90)), rand_i8((13, 90))
    sw = RNG.uniform(1e-3, 1e-2, 13).astype(np.float32)
    acc, y = oracle.layer_dequant(X, W, sw, b, sx=0.02)
    ra, ry = oracle.masked_linear(X, W, 0.02, sw, b)
    assert np.array_equal(acc, ra)
    mag = 0.02 * (np.abs(X.astype(np.float64)) @ np.abs(oracle.mask(W, b).astype(np.float64)).T
                  ) * sw.astype(np.float64)
    assert np.all(np.abs(y - ry) <= 1e-13 * mag)


@pytest.mark.parametrize("b", [8, 6, 3])
def test_layer_dequant_factored_zero_points(b):
    """sum_k x_hat w_hat_b against the expanded form through numpy's int64
    matmul: symmetric activations give sx sw (acc + (128 - zw) rowsum(X));
    asymmetric ones add (128 - zx) colsum_b and K (128 - zx)(128 - zw)."""
    X, W = rand_i8((7, 150)), rand_i8((9, 150))
    sw = RNG.uniform(1e-3, 1e-2, 9).astype(np.float32)
    zw = RNG.uniform(60, 190, 9).astype(np.float32)
    Wb = oracle.mask(W, b).astype(np.int64)
    acc = X.astype(np.int64) @ Wb.T
    rs = X.astype(np.int64).sum(1)[:, None]
    cs = Wb.sum(1)[None, :]
    swd, zwd = sw.astype(np.float64), zw.astype(np.float64)
    a1, y1 = oracle.layer_dequant(X, W, sw, b, sx=0.02, zw=zw)
    e1 = 0.02 * swd * (acc + (128.0 - zwd) * rs)
    assert np.array_equal(a1, acc)
    assert np.all(np.abs(y1 - e1) <= 1e-12 * (np.abs(0.02 * swd) * (np.abs(acc) + np.abs(
        (128 - zwd) * rs))))
    ax, zx = 0.031, 97.25
    a2, y2 = oracle.layer_dequant(X, W, sw, b, act=(ax, zx), zw=zw)
    e2 = ax * swd * (acc + (128 - zx) * cs + (128.0 - zwd) * (rs + 150 * (128 - zx)))
    mag = ax * swd * (np.abs(acc) + np.abs((128 - zx) * cs) + np.abs((128 - zwd) * rs)
                      + 150 * np.abs((128 - zx) * (128 - zwd)))
    assert np.all(np.abs(y2 - e2) <= 1e-12 * mag)


def test_layer_dequant_exact_rational_tiny():
    X, W = rand_i8((2, 5)), rand_i8((3, 5))
    sw = np.array([0.25, 0.5, 0.125], np.float32)
    zw = np.array([100.5, 130.0, 77.25], np.float32)
    acc, y = oracle.layer_dequant(X, W, sw, 4, act=(0.5, 3.75), zw=zw)
    Wb = oracle.mask(W, 4)
    for m in range(2):
        for n in range(3):
            e = sum((Fraction(1, 2) * (int(X[m, k]) + 128 - Fraction(15, 4)))
                    * (Fraction(float(sw[n])) * (int(Wb[n, k]) + 128 - Fraction(float(zw[n]))))
                    for k in range(5))
            assert Fraction(y[m, n]) == e


def test_layer_dequant_entries_match_full():
    X, W = rand_i8((9, 64)), rand_i8((10, 64))
    sw = RNG.uniform(1e-3, 1e-2, 10).astype(np.float32)
    zw = RNG.uniform(0, 255, 10).astype(np.float32)
    bias = RNG.uniform(-1, 1, 10).astype(np.float32)
    acc, y = oracle.layer_dequant(X, W, sw, 6, act=(0.02, 130.5), zw=zw, bias=bias)
    rows, cols = RNG.integers(0, 9, 30), RNG.integers(0, 10, 30)
    ae, ye = oracle.layer_dequant_entries(X, W, sw, 6, rows, cols, act=(0.02, 130.5), zw=zw,
                                          bias=bias)
    assert np.array_equal(ae, acc[rows, cols])
    assert np.allclose(ye, y[rows, cols], rtol=1e-13, atol=0)


# ------------------------------------------------ BitOPs and cycle accounting

def _golden_rows(name):
    from conftest import golden_path
    rows = []
    for line in open(golden_path(name)):
        line = line.strip()
        if line and not line.startswith("#"):
            rows.append(line.split())
    return rows


def test_rel_bitops_matches_printed_table():
    """Every (A-bit, Eff. W-bit, Rel. BitOPs) triple the quality table prints
    satisfies Rel = W A / 64 to its two printed decimals, and the schedule
    accounting of a one-layer schedule at that constant precision gives it."""
    for a, w100, rel100 in (map(int, r) for r in _golden_rows("bitops_quality.txt")):
        assert round(w100 / 100 * a / 64, 2) == rel100 / 100
    for a, b in ((8, 8), (8, 4), (4, 4), (16, 8)):
        c = oracle.schedule_cost([100], [[b]], 1, 1, 0, 1, a)
        assert c["rel_bitops"] == b * a / 64 and c["b_eff"] == b


def test_tpe_cycle_laws_match_printed_tables():
    rows = _golden_rows("tpe_cycles.txt")
    for r in rows:
        if r[0] == "measured":
            assert oracle.tpe_cycles_measured([int(v) for v in r[1:5]]) == int(r[5])
        elif r[0] == "fetch":
            assert oracle.fetch_planes(r[1], 8, 4) == int(r[2])
        else:
            assert oracle.tpe_tile_cycles(r[0], int(r[1])) == int(r[2])


def test_schedule_cost_hand_worked():
    """Two layers (100 and 300 MACs), S = 2 stages over T = 4 steps, table
    [[8, 4], [2, 6]]: steps 0, 1 at (8, 2), steps 2, 3 at (4, 6)."""
    c = oracle.schedule_cost([100, 300], [[8, 4], [2, 6]], 2, 4, 0, 4, 8)
    macs = 4 * 400
    bw = 2 * (100 * 8 + 300 * 2) + 2 * (100 * 4 + 300 * 6)
    assert c["macs"] == macs and c["b_eff"] == bw / macs
    assert c["b_mean"] == (8 + 2 + 8 + 2 + 4 + 6 + 4 + 6) / 8
    assert c["rel_bitops"] == bw * 8 / (64 * macs)
    assert c["rel_cycles_measured"] == bw / (8 * macs)
    num = 2 * (100 * (570 * 8 + 2603) + 300 * (570 * 2 + 2603)) + \
        2 * (100 * (570 * 4 + 2603) + 300 * (570 * 6 + 2603))
    assert c["rel_cycles_as_a4"] == num / (macs * (570 * 8 + 2603))
    # a sub-range of steps counts only those steps
    c2 = oracle.schedule_cost([100, 300], [[8, 4], [2, 6]], 2, 4, 3, 4, 8)
    assert c2["macs"] == 400 and c2["b_eff"] == (100 * 4 + 300 * 6) / 400
