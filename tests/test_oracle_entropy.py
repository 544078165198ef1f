"""Pins of the entropy-coding oracle (oracle/entropy.py) against things other
than itself: the Gaussian from scipy.stats, brute-force index search, a worked
example done by hand from the rANS definition, lossless round trips, and the
length bounds of rANS (Duda 2013): the output of a stream lies between the
ideal code length plus 16 bits and plus 32 bits per lane state."""
import numpy as np
import pytest
from scipy.stats import norm

from oracle import entropy as E


def test_scale_table_is_geometric_and_monotone():
    s = E.scale_table().astype(np.float64)
    assert s.dtype == np.float64 and len(s) == E.NS
    assert abs(s[0] - 0.11) < 1e-7 and abs(s[-1] - 256.0) < 1e-4
    r = s[1:] / s[:-1]
    assert np.all(r > 1.0) and np.allclose(r, (256.0 / 0.11) ** (1 / 63), rtol=1e-6)


def test_scale_index_is_the_smallest_covering_scale():
    tab = E.scale_table().astype(np.float64)
    rng = np.random.default_rng(3)
    sig = np.concatenate([np.exp(rng.uniform(np.log(0.01), np.log(1000.0), 2000)), tab,
                          np.nextafter(tab, np.inf), np.nextafter(tab, -np.inf), [0.0, 1e9]])
    k = E.scale_index(sig)
    for s, kk in zip(sig, k):
        cover = [j for j in range(E.NS) if tab[j] >= s]
        assert kk == (cover[0] if cover else E.NS - 1)


@pytest.mark.parametrize("j", [0, 1, 7, 20, 31, 45, 63])
def test_tables_are_valid_quantised_gaussians(j):
    R, f, c = E.table(j)
    sigma = float(E.scale_table()[j])
    assert R == max(int(np.ceil(8.0 * sigma)), 32)
    n = 2 * R + 2
    assert len(f) == n and np.all(f >= 1) and int(f.sum()) == E.M
    assert np.array_equal(c, np.concatenate([[0], np.cumsum(f)[:-1]]))
    q = np.arange(-R, R + 1)
    p = norm.cdf((q + 0.5) / sigma) - norm.cdf((q - 0.5) / sigma)
    p_esc = 2.0 * norm.sf((R + 0.5) / sigma)
    err = np.abs(f[:-1] / E.M - p)
    # floor(p (M - n)) + 1 is within n p / M + 1 / M of p M; the mode also takes the remainder (< n)
    bound = (n * p + 1.0) / E.M + 1e-12
    bound[R] += n / E.M
    assert np.all(err <= bound)
    assert abs(f[-1] / E.M - p_esc) <= (n * p_esc + 1.0) / E.M + 1e-12
    assert np.all(np.diff(f[: R + 1]) >= 0) and np.all(np.diff(f[R:-1]) <= 0)  # unimodal, peak at q = 0


def test_worked_example_one_symbol():
    # Scale 0 (sigma 0.11) has R = 32: every symbol but q = 0 has probability
    # below 2^-17, so f = 1 for q = -32 .. -1, 1 .. 32 and ESC, and
    # f(0) = 65536 - 65 = 65471 with start 32.
    R, f, c = E.table(0)
    assert R == 32 and f[R] == 65471 and c[R] == 32 and np.all(np.delete(f, R) == 1)
    # Encoding q = 0 from x = 65536: no renormalisation (65536 < 65471 * 65536);
    # x = (65536 div 65471) * 65536 + (65536 mod 65471) + 32 = 65536 + 65 + 32 = 65633.
    # Lane 0 ends at 65633 -> words (1, 97); the other 63 lanes stay at 65536 -> (1, 0).
    words = E.encode_stream(np.array([0]), np.array([0]))
    assert words == [1, 97] + [1, 0] * 63
    q, ok = E.decode_stream(words, np.array([0]))
    assert ok and list(q) == [0]


def test_worked_example_escape():
    # q = -40 at scale 0 escapes (|q| > R = 32): ESC (start 65535, f 1), then the
    # field 32768 + (40 - 33) = 32775 with f = 1.  From x = 65536: the field
    # needs renormalisation (65536 >= 1 * 65536): word 0, x = 1, then
    # x = 1 * 65536 + 0 + 32775 = 98311; ESC: again 98311 >= 65536: word
    # 98311 mod 65536 = 32775, x = 1, then x = 65536 + 65535 = 131071.
    # Decoding order: states (131071 -> 1, 65535), then the words of ESC's
    # renormalisation (32775), then the field's (0).
    words = E.encode_stream(np.array([-40]), np.array([0]))
    assert words == [1, 65535] + [1, 0] * 63 + [32775, 0]
    q, ok = E.decode_stream(words, np.array([0]))
    assert ok and list(q) == [-40]


def test_all_escape_stream_meets_the_two_word_bound():
    # Every symbol escapes at the smallest scale: each sub-symbol moves at most
    # one word, so a full stream holds at most 128 + 2 * 8192 words; with
    # frequency 1 the field always moves one, so the bound is nearly reached.
    rng = np.random.default_rng(9)
    q = rng.integers(33, 32768, E.STREAM) * rng.choice([-1, 1], E.STREAM)
    k = np.zeros(E.STREAM, dtype=np.int64)
    words = E.encode_stream(q, k)
    assert 128 + 2 * E.STREAM - 64 <= len(words) <= 128 + 2 * E.STREAM
    out, ok = E.decode_stream(words, k)
    assert ok and np.array_equal(out, q)


def _symbols(n, seed, esc_every=0):
    rng = np.random.default_rng(seed)
    sig = np.exp(rng.uniform(np.log(0.05), np.log(400.0), n))
    k = E.scale_index(sig)
    q = np.rint(rng.standard_normal(n) * sig).astype(np.int64)
    if esc_every:
        q[::esc_every] = rng.integers(-32768, 32768, len(q[::esc_every]))
        q[: min(n, 2)] = [-32768, 32767][: min(n, 2)]
    return np.clip(q, -32768, 32767), k


@pytest.mark.parametrize("n,esc", [(1, 0), (63, 5), (64, 0), (65, 3), (E.STREAM - 1, 41),
                                   (E.STREAM, 0), (E.STREAM + 1, 17), (20000, 97)])
def test_round_trip_and_length_bounds(n, esc):
    q, k = _symbols(n, seed=n, esc_every=esc)
    data = E.encode(q, k)
    out, ok = E.decode(data, k)
    assert ok and np.array_equal(out, q)
    ns = (n + E.STREAM - 1) // E.STREAM
    header = 20 + 2 * ns + ((-2 * ns) % 4)
    payload_bits = 8 * (len(data) - header)
    ideal = E.ideal_bits(q, k)
    assert ideal + 16 * E.LANES * ns - 1e-6 * n <= payload_bits <= ideal + 32 * E.LANES * ns + 1e-3 * n + 64


def test_corrupted_containers_are_rejected():
    q, k = _symbols(3000, seed=5, esc_every=50)
    data = E.encode(q, k)
    bad_magic = b"X" + data[1:]
    assert not E.decode(bad_magic, k)[1]
    assert not E.decode(data[: len(data) // 2], k)[1]
    assert not E.decode(data, k[:-1])[1]  # symbol count does not match the header
    flipped = bytearray(data)
    flipped[-3] ^= 0x5A
    out, ok = E.decode(bytes(flipped), k)
    assert not ok or not np.array_equal(out, q)
