"""The seeded input generator: Philox4x32-10 known answers, slice regeneration, distributions."""
import numpy as np

import synth
from synth.workloads import WORKLOADS


def test_philox_known_answer_vectors():
    # Known-answer vectors published with the Random123 library (Salmon et al., SC'11) for Philox4x32-10.
    assert synth.philox((0, 0, 0, 0), (0, 0)) == (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)
    assert synth.philox((0xFFFFFFFF,) * 4, (0xFFFFFFFF, 0xFFFFFFFF)) == (0x408F276D, 0x41C83B0E, 0xA20BC7C6,
                                                                        0x6D5451FD)
    assert synth.philox((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0)) == (
        0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)


def test_slices_regenerate_exactly():
    full = synth.normal_f32(10_001, stream=7, std=0.02)
    part = synth.normal_f32(333, stream=7, std=0.02, start=4_567)
    assert (full[4_567:4_900] == part).all()
    lab = synth.labels_zipf(5000, 32000)
    assert (synth.labels_zipf(100, 32000, start=1234) == lab[1234:1334]).all()


def test_bf16_is_round_to_nearest_even_of_fp32():
    f = synth.normal_f32(100_000, stream=9, std=3.0)
    b = synth.bf16_to_f32(synth.normal_bf16(100_000, stream=9, std=3.0))
    # RNE to 8 significant bits (7 stored): relative error at most 2^-8
    assert (np.abs(b - f) <= np.abs(f) * 2.0 ** -8 + 1e-30).all()
    bits = b.view(np.uint32)
    assert (bits & 0xFFFF == 0).all()


def test_distributions():
    x = synth.normal_f32(2_000_000, stream=1, std=2.0).astype(np.float64)
    assert abs(x.mean()) < 0.01 and abs(x.std() - 2.0) < 0.01
    y = synth.labels_uniform(200_000, 10)
    cnt = np.bincount(y, minlength=10)
    assert y.min() == 0 and y.max() == 9 and np.abs(cnt / 2e4 - 1).max() < 0.05
    V = 1000
    z = synth.labels_zipf(400_000, V, a=1.1)
    pmf = np.arange(1, V + 1, dtype=np.float64) ** -1.1
    pmf /= pmf.sum()
    emp = np.bincount(z, minlength=V) / z.size
    assert np.abs(emp[:10] - pmf[:10]).max() < 3e-3


def test_ignored_fraction():
    y = synth.labels_uniform(100_000, 50)
    yi = synth.with_ignored(y, 0.05)
    frac = (yi == -100).mean()
    assert 0.045 < frac < 0.055 and ((yi == y) | (yi == -100)).all()


def test_workload_table_sizes():
    w = {x.name: x for x in WORKLOADS}
    assert w["tiny_linear_c10"].P == w["tiny_linear_c10"].head_params == 1290
    assert w["lm_8b_v128256"].P == 476 * 4096 * 4096 + 3429 * 4096
    for x in WORKLOADS:
        assert x.head_params <= x.P
        segs = x.segments()
        assert sum(s[1] for s in segs) == x.P
