"""The seeded input generator: known answers, row addressability, moments.  CPU only."""
import math

import numpy as np

import synth as S
from synth import configs as CF


def test_splitmix64_published_vector():
    # SplitMix64 (Vigna) with state 1234567: the first five outputs of its published test vector.
    want = [6457827717110365317, 3203168211198807973, 9817491932198370423,
            4593380528125082431, 16408922859458223821]
    assert [int(x) for x in S.raw64(1234567, np.arange(5))] == want


def test_bf16_round_nearest_even():
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -2.5, 1 + 2 ** -8 + 2 ** -20], dtype=np.float32)
    assert list(S.f32_to_bf16_bits(x)) == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x3F81]
    assert np.array_equal(S.bf16_bits_to_f32(np.array([0x3F80, 0xC020], np.uint16)), [1.0, -2.5])


def test_rows_are_addressable():
    full = S.tensor_f32(7, S.TID_VALUES, (50, 12), 0.3)
    rows = np.array([49, 0, 17, 17])
    assert np.array_equal(S.rows_f32(7, S.TID_VALUES, rows, 12, 0.3), full[rows])


def test_moments_and_bounds():
    x = S.normal_f32(S.stream_key(1, 2), np.arange(1 << 20), 0.25).astype(np.float64)
    assert abs(x.mean()) < 3 * 0.25 / math.sqrt(len(x)) * 2
    assert abs(x.std() - 0.25) < 0.002
    assert np.abs(x).max() <= 0.25 * math.sqrt(3) * 2 * 1.0001
    # distinct tensors and seeds give distinct streams
    assert S.stream_key(1, 2) != S.stream_key(2, 1) != S.stream_key(1, 3)


def test_permutation_and_clusters():
    p = S.permutation(3, S.TID_PERM, 1000)
    assert np.array_equal(np.sort(p), np.arange(1000))
    assert not np.array_equal(p, np.arange(1000))
    cfg = CF.C5.with_tokens(64)
    qr, qc = CF.queries(cfg)
    assert qr.shape == (64, 4, 128) and qr.dtype == np.float32
    part, _ = CF.queries(cfg, tokens=np.array([5, 9]))
    assert np.array_equal(part, qr[[5, 9]])


def test_config_shapes():
    assert CF.C3.n_slots == 20_070_400 and CF.C3.bag == 64
    assert CF.C5.n_values == 1_048_576 and CF.C5.n_slots == 4_194_304
    assert CF.C2.n_values == 1 << 20
