"""The seeded input generator: bf16 rounding, determinism, sampled rows."""
import numpy as np
import pytest

import workloads


def test_bf16_rounding_matches_torch_round_to_nearest_even():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * 10,
        np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -1.0 - 2.0 ** -8, 0.0, -0.0, 65504.0, 1e-40],
                 dtype=np.float32),
    ])
    ours = workloads.float32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    # ties go to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7
    assert ours[-7] == 0x3F80 and ours[-6] == 0x3F82


def test_bf16_widening_roundtrip():
    bits = np.arange(0, 0x7F80, 7, dtype=np.uint16)
    np.testing.assert_array_equal(workloads.float32_to_bf16_bits(workloads.bf16_bits_to_float32(bits)), bits)


def test_workloads_match_the_paper_token_counts():
    c = workloads.WORKLOADS
    assert c[4].N == 92 * 2048 == 368 * 512
    assert c[5].N == 1024 * 1024
    assert [c[i].d for i in range(1, 6)] == [64, 64, 128, 128, 64]
    assert abs(c[4].counted_flops()["total"] / 1e12 - 127.234) < 1e-3
    assert c[4].scale == np.float32(1 / np.sqrt(128))


def test_inputs_are_deterministic_and_stress_head_is_scaled():
    w = workloads.Workload(99, "tiny", 2, 3, 40, 8, True, 1.0, 7, 8.0, "full", (5, 8))
    a = workloads.make_inputs(w)
    b = workloads.make_inputs(w)
    for n in ("q", "k", "v", "dout"):
        np.testing.assert_array_equal(a[n], b[n])
        assert a[n].shape == (2, 3, 40, 8) and a[n].dtype == np.uint16
    f = {n: workloads.bf16_bits_to_float32(a[n]) for n in a}
    assert np.std(f["q"][:, 0]) > 5 * np.std(f["q"][:, 1:])
    assert np.std(f["v"][:, 0]) < 2 * np.std(f["v"][:, 1:])


def test_sampled_rows_distinct_and_in_range():
    for cid in (3, 4, 5):
        w = workloads.WORKLOADS[cid]
        r = workloads.sampled_query_rows(w)
        assert r.shape == (256, 3)
        assert len({tuple(x) for x in r}) == 256
        assert (r[:, 0] < w.B).all() and (r[:, 1] < w.H).all() and (r[:, 2] < w.N).all()
        kr = workloads.sampled_key_rows(w)
        assert not np.array_equal(r, kr)
