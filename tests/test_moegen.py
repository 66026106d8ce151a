"""The seeded input generator: reproducibility, exact expert loads, bf16 rounding."""
import numpy as np
import pytest
import torch

import moegen
import oracle


def test_round_bf16_matches_torch_rne():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38, -3.0e38, 1e-40],
                                 dtype=np.float32)]).astype(np.float32)
    want = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(moegen.round_bf16(a), want)


def test_seeded_and_reproducible():
    a = moegen.make_inputs("tiny")
    b = moegen.make_inputs("tiny")
    c = moegen.make_inputs("tiny", seed=5)
    for name in ("x", "logits", "w_gate", "w_up", "w_down"):
        assert np.array_equal(getattr(a, name), getattr(b, name))
        assert not np.array_equal(getattr(a, name), getattr(c, name))


def test_distributions():
    cfg = moegen.CONFIGS["tiny"].scaled(T=2048)
    I = moegen.make_inputs(cfg)
    assert abs(I.x.std() - 1.0) < 0.01
    assert abs(I.w_gate.std() - 1 / np.sqrt(cfg.H)) < 0.002
    assert abs(I.w_down.std() - 1 / np.sqrt(cfg.F)) < 0.002
    # router logits of std 0.02 * sqrt(H)
    assert abs(I.logits.std() - 0.02 * np.sqrt(cfg.H)) < 0.02
    bf = moegen.make_inputs(moegen.CONFIGS["mixtral4k"].scaled(T=64, H=256, F=512))
    assert bf.x.dtype == np.uint16 and bf.w_gate.shape == (8, 512, 256) and bf.w_down.shape == (8, 256, 512)
    assert abs(moegen.as_f64(bf.x).std() - 1.0) < 0.02


def test_zipf_counts():
    # c_r proportional to r^-1.2 over 8 experts, R = 65536, by largest remainder
    c = moegen.zipf_counts(8, 65536, 1.2)
    q = np.arange(1, 9) ** -1.2
    q = q / q.sum() * 65536
    assert c.sum() == 65536 and (np.abs(c - q) < 1).all()
    assert c.tolist() == [28091, 12227, 7516, 5322, 4072, 3272, 2719, 2317]
    assert 0.42 < c[0] / 65536 < 0.44


@pytest.mark.parametrize("T,E,k", [(64, 8, 2), (100, 7, 3), (50, 5, 5), (33, 64, 1)])
def test_exact_count_assignment(T, E, k):
    rng = np.random.default_rng(T * E + k)
    counts = moegen.largest_remainder(rng.random(E) + 0.01, T * k)
    counts = np.minimum(counts, T)
    # restore the total if the cap at T removed rows
    short = T * k - counts.sum()
    for e in np.argsort(counts):
        add = min(short, T - counts[e])
        counts[e] += add
        short -= add
    chosen, relabel = moegen.exact_count_assignment(counts, T, k, rng)
    assert all(len(set(r)) == k for r in chosen.tolist())
    assert np.array_equal(np.bincount(chosen.ravel(), minlength=E), counts[np.argsort(relabel)])


def test_constructed_logits_route_to_chosen_sets():
    cfg = moegen.MoEConfig("zipf-small", T=512, H=128, E=8, k=2, F=128, seed=7, routing="zipf")
    I = moegen.make_inputs(cfg)
    ids, _ = oracle.route(I.logits, cfg.k, 1)
    assert np.array_equal(np.sort(ids, 1), np.sort(I.chosen, 1))
    assert np.array_equal(np.bincount(ids.ravel(), minlength=8), I.target_counts)
    assert sorted(I.target_counts.tolist(), reverse=True) == moegen.zipf_counts(8, 1024, 1.2).tolist()


def test_lognormal_counts_pinned_small():
    rng = np.random.default_rng(4)
    c = moegen.lognormal_counts(rng, 64, 131072 * 4, 1.0, (1, 17, 31))
    assert c.sum() == 131072 * 4
    assert sorted(c)[:3] == [1, 17, 31]
    assert c.max() > 20000 and c.max() <= 131072


def test_uniform_routing():
    cfg = moegen.MoEConfig("u", T=16, H=64, E=8, k=3, F=64, routing="uniform")
    I = moegen.make_inputs(cfg)
    assert (I.logits == 0).all()


def test_cap_counts_keeps_the_sum_and_the_cap():
    c = moegen.cap_counts(np.array([335, 300, 100, 10, 1, 278]), 256)
    assert c.sum() == 1024 and c.max() <= 256
    assert list(c) == [256, 256, 245, 10, 1, 256]          # excess to the largest with room
    same = np.array([5, 4, 3])
    assert np.array_equal(moegen.cap_counts(same, 5), same)
