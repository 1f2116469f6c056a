"""Input generator: determinism, shapes, storage-precision rounding."""
import numpy as np

from paper_2608_02123_amd.synth import CONFIGS, Workload, bf16_bits, make_inputs, round_to_bf16


def _rne_bf16_by_frexp(x):
    """Same rounding written as scaling of the significand (ties to even by np.rint)."""
    m, e = np.frexp(np.asarray(x, np.float64))
    return np.ldexp(np.rint(m * 256.0) / 256.0, e).astype(np.float32)


def test_bf16_rounding_matches_significand_rounding():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(200000) * s for s in (1e-3, 0.02, 1.0, 3.0, 1e4)])
    # exact ties: values halfway between two bf16 neighbours
    base = round_to_bf16(rng.standard_normal(1000)).astype(np.float64)
    ulp = np.abs(base) * 2.0 ** -8
    x = np.concatenate([x, base + ulp / 2, base - ulp / 2, [0.0, -0.0, 1.0, -2.5]])
    assert np.array_equal(round_to_bf16(x), _rne_bf16_by_frexp(x))
    bf16_bits(round_to_bf16(x))  # representable


def test_deterministic_and_shaped():
    w = Workload("t", V=3000, B=3, N=8, k=4, r=64, R=2, dtype="bf16", peak="decay")
    a, b = make_inputs(w), make_inputs(w)
    for key in ("L", "E", "W", "h", "root", "prefix_len"):
        assert np.array_equal(a[key], b[key])
    assert a["L"].shape == (2, 3, 3000) and a["E"].shape == (3000, 64)
    assert a["W"].shape == (64, 3000) and a["h"].shape == (2, 3, 64)
    bf16_bits(a["L"]), bf16_bits(a["E"]), bf16_bits(a["W"])
    assert ((0 <= a["root"]) & (a["root"] < 3000)).all()
    # requests draw independent logits and roots; the head is shared
    assert not np.array_equal(a["L"][0], a["L"][1])


def test_peaks_present():
    w = CONFIGS["tiny"]
    inp = make_inputs(w)
    # +8 on three tokens per depth on top of N(0, 9): the max is far out in the tail
    assert (inp["L"][0].max(axis=1) > 8.0).all()
