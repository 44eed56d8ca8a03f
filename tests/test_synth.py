"""The seeded input generator: reproducible, row-addressable, shaped like the workloads."""
import numpy as np

import synth


def test_rows_and_groups_are_independently_addressable():
    w = synth.variant(synth.workloads()["qwen3_8b_single"], V=3000, K=3)
    full = synth.generate(w)
    part = synth.generate(w, rows=[0, 5], bk=[(0, 2), (0, 1)])
    assert np.array_equal(part[0, 0], full[0, 0, 2])
    assert np.array_equal(part[1, 1], full[5, 0, 1])
    again = synth.generate(w)
    assert np.array_equal(full, again)
    other_round = synth.generate(w, round=1)
    assert not np.array_equal(full, other_round)


def test_value_distribution_and_boosts():
    w = synth.variant(synth.workloads()["qwen3_8b_single"], K=2)
    x = synth.decode(w, synth.generate(w))
    t = x[0, 0, 0]
    assert abs(t.mean()) < 0.05 and abs(t.std() - 3.0) < 0.05
    # 20 boosted tokens per row sit about 8 above their draw
    assert (t > 3 * 4.9).sum() == 0 or (t > 3 * 4.9).sum() <= 20
    for i, s in enumerate(w.scales):
        d = x[1 + i, 0, 0] - t
        assert abs(d.std() - s) < 0.03 * s + 0.01


def test_permutation_puts_smallest_scale_on_b_mod_n():
    w = synth.workloads()["batched_serving"]
    ranks = w.scale_ranks(0)
    for b in range(w.B):
        assert ranks[b, b % w.N] == 0
        assert sorted(ranks[b]) == list(range(w.N))
    w5 = synth.workloads()["large_pool_stream"]
    assert np.array_equal(w5.scale_ranks(500), (w5.N - 1) - w5.scale_ranks(0))
    assert np.array_equal(w5.scale_ranks(499), w5.scale_ranks(0))


def test_tree_shape_and_seeded_path_ends():
    w = synth.workloads()["draft_tree"]
    par = w.parent()
    assert len(par) == 64 and par[0] == -1 and np.all(par[1:] < np.arange(1, 64))
    depth = np.zeros(64, dtype=int)
    for n in range(1, 64):
        depth[n] = depth[par[n]] + 1
    assert list(np.bincount(depth)) == [1, 3, 6, 12, 24, 18]
    ends = w.path_end()
    has_child = np.zeros(64, bool)
    has_child[par[1:]] = True
    assert np.all(~has_child[ends])
    assert np.array_equal(ends, w.path_end())


def test_bf16_rounding_is_nearest_even():
    w = synth.variant(synth.workloads()["tiny_chain"], V=1000)
    wb = synth.variant(w, dtype=synth.BF16)
    f = synth.generate(w)
    b = synth.generate(wb)
    # target rows: bf16 must be the RNE rounding of the fp32 value
    u = f[0].view(np.uint32).astype(np.uint64)
    rne = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    assert np.array_equal(rne, b[0])
