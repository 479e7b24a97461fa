"""The seeded input generator: published SplitMix64 outputs, rounding,
determinism, page-table validity and the shape of the length distributions."""
import numpy as np

from paper_2608_22788_amd import synth


def test_splitmix64_published_vectors():
    # SplitMix64 started from state 0: outputs 1..3 (Vigna's reference code)
    z = synth._mix64(np.array([(k * synth.GAMMA) & synth.MASK64 for k in (1, 2, 3)], dtype=np.uint64))
    assert [int(x) for x in z] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_draws_are_counter_based():
    a = synth.draws(5, synth.S_K, np.arange(100))
    b = synth.draws(5, synth.S_K, np.arange(40, 60))
    assert np.array_equal(a[40:60], b)
    assert not np.array_equal(a, synth.draws(6, synth.S_K, np.arange(100)))
    assert not np.array_equal(a, synth.draws(5, synth.S_V, np.arange(100)))


def test_bf16_rounding_nearest_even():
    f = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20, -2.5, 3.0e38, np.inf, np.nan],
                 dtype=np.float32)
    got = synth.f32_to_bf16_bits(f)
    assert list(got) == [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC020, 0x7F62, 0x7F80, 0x7FC0]
    back = synth.bf16_bits_to_f32(got[:5])
    assert np.array_equal(back, np.array([1.0, 1.0, 1 + 2 ** -6, 1 + 2 ** -7, -2.5], np.float32))


def test_normals_moments():
    x = synth.bf16_bits_to_f32(synth.normal_bf16_range(0, synth.S_K, 0, 1 << 20)).astype(np.float64)
    assert abs(x.mean()) < 0.005 and abs(x.std() - 1.0) < 0.005
    assert np.abs(x).max() < 6.7


def test_uniform_int_inclusive():
    v = synth.uniform_int(synth.draws(1, synth.S_LEN_A, np.arange(200000)), 16, 256)
    assert v.min() == 16 and v.max() == 256


def test_length_distributions():
    bulk = np.concatenate([synth.lengths_bulk(s, 256) for s in range(40)])
    resp_med = np.median(bulk) - 640
    assert 1800 < resp_med < 2300
    assert bulk.max() <= 1024 + 16384 and bulk.min() >= 256 + 1
    sw = np.concatenate([synth.lengths_sweep(s, 512) for s in range(20)])
    assert sw.min() >= 512 + 1024 and sw.max() <= 512 + 65536
    # Pareto(1024, 1.5): P(X > 4096) = 4^-1.5 = 1/8
    assert abs((sw - 512 > 4096).mean() - 0.125) < 0.01
    mtp = synth.draw_lengths(synth.CONFIGS["mtp"], 0)
    assert ((mtp >= 16384) & (mtp <= 65536)).all()


def test_page_table_is_a_permutation():
    wl = synth.make_workload("bulk", seed=0)
    npg = (wl.ctx_lens.astype(np.int64) + 15) // 16
    used = np.concatenate([wl.page_table[b, :npg[b]] for b in range(wl.B)])
    assert np.array_equal(np.sort(used), np.arange(wl.num_pages))
    assert wl.num_pages == npg.sum()
    wl2 = synth.make_workload("bulk", seed=0)
    assert np.array_equal(wl.page_table, wl2.page_table)


def test_subset_keeps_values():
    wl = synth.make_workload("tiny", seed=0)
    sub = wl.subset([2, 0])
    kp, skp = wl.k_pages(), sub.k_pages()
    q, sq = wl.q_values(), sub.q_values()
    for i, b in enumerate([2, 0]):
        n = (int(wl.ctx_lens[b]) + 15) // 16
        for j in range(n):
            assert np.array_equal(kp[wl.page_table[b, j]], skp[sub.page_table[i, j]])
        assert np.array_equal(q[b], sq[i])


def test_poison_marks_only_unused_slots():
    wl = synth.make_workload("tiny", seed=3, poison=True, spare_pages=2)
    kp = wl.k_pages()
    used = wl.used_slots()
    nan = kp == synth.BF16_NAN
    assert nan[~used[:, None, :, None].repeat(wl.Hkv, 1).repeat(wl.D, 3)].all()
    assert not nan[used[:, None, :, None].repeat(wl.Hkv, 1).repeat(wl.D, 3)].any()
    assert (wl.page_table[:, -1] >= 0).all()
