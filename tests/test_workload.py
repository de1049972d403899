"""The seeded input generator (CPU): known answers, host library vs restatement,
distribution, and the validity of every workload schedule."""
import numpy as np
import pytest

from workload import configs, gen


def test_splitmix64_known_answer():
    # First output of SplitMix64 started from state 0 (the published generator).
    assert gen.mix64(0 + gen.GAMMA) == 0xE220A8397B1DCDAF
    assert gen.draw(0, 0) == 0xE220A8397B1DCDAF


def test_host_library_matches_restatement():
    lib = gen.host_lib()
    for seed, stream in ((1, 3), (1003, 5), (2**40 + 7, 6)):
        key = gen.stream_key(seed, stream)
        assert lib.wl_host_stream_key(seed, stream) == key
        for j in (0, 1, 2, 12345, 2**40):
            assert lib.wl_host_draw(key, j) == gen.draw(key, j)
    key = gen.stream_key(5, 3)
    a = gen.fill_host(5, 3, "f32", (2, 3, 4, 5), 17, (100, 30, 5, 1))
    ref = np.array([gen.normal_ref(key, 17 + i0 * 100 + i1 * 30 + i2 * 5 + i3)
                    for i0 in range(2) for i1 in range(3) for i2 in range(4) for i3 in range(5)],
                   np.float32)
    assert np.array_equal(a.view(np.float32).ravel(), ref)
    b = gen.fill_host(5, 3, "bf16", (2, 3, 4, 5), 17, (100, 30, 5, 1))
    assert np.array_equal(b.ravel(), np.array([gen.bf16_rne_ref(x) for x in ref], np.uint16))


def test_bf16_round_to_nearest_even():
    # halfway cases round to the even neighbour; others to the nearest
    cases = {0x3F808000: 0x3F80, 0x3F818000: 0x3F82, 0x3F808001: 0x3F81, 0x3F807FFF: 0x3F80,
             0xBF80C000: 0xBF81}
    lib = gen.host_lib()
    for u, want in cases.items():
        f = float(np.array(u, np.uint32).view(np.float32))
        assert gen.bf16_rne_ref(f) == want
        assert lib.wl_host_bf16_rne(f) == want


def test_values_are_standardised():
    x = gen.fill_host(3, gen.S_PREFILL_K, "f32", (1, 1, 1, 400_000), 0, (0, 0, 0, 1))
    f = x.view(np.float32).astype(np.float64)
    assert abs(f.mean()) < 0.01 and abs(f.std() - 1.0) < 0.01 and np.abs(f).max() < 6.0
    # exact multiples of 2^-17
    assert np.all(f * 131072.0 == np.round(f * 131072.0))


def test_counters_are_shape_independent():
    """A prefilled token's value depends on (query, layer, head, t, d), not on the length."""
    a = gen.prefill_host(9, "k", qid=4, n_layers=2, n_kv_heads=3, length=10, head_dim=8, dtype="bf16")
    b = gen.prefill_host(9, "k", qid=4, n_layers=2, n_kv_heads=3, length=25, head_dim=8, dtype="bf16")
    assert np.array_equal(a, b[:, :, :10])
    c = gen.prefill_host(9, "v", qid=4, n_layers=2, n_kv_heads=3, length=10, head_dim=8, dtype="bf16")
    assert not np.array_equal(a, c)


@pytest.mark.parametrize("name", sorted(configs.CONFIGS))
def test_schedule_is_valid(name):
    w = configs.CONFIGS[name]()
    assert len(w.init_lens) == w.batch and max(w.init_lens) == w.L0
    assert min(w.init_lens) >= 1
    live = set(range(w.batch))
    qids = set(range(w.batch))
    assert len(w.steps) == w.n_steps
    for e in w.steps:
        assert set(e.evict) <= live and e.evict == sorted(set(e.evict))
        live -= set(e.evict)
        assert not set(e.insert) & live
        live |= set(e.insert)
        assert len(e.insert) == len(e.insert_lens) == len(e.insert_qids)
        assert all(1 <= n < gen.TMAX for n in e.insert_lens)
        assert not set(e.insert_qids) & qids
        qids |= set(e.insert_qids)
    assert w.capacity() >= w.L0 + w.n_steps + 1


def test_config_laws():
    w = configs.skew_b256_l32768()
    longs = [n for n in w.init_lens if n > 1024]
    assert len(longs) == round(0.1 * w.batch)
    assert all(16384 <= n <= 32768 for n in longs)
    w3 = configs.llama7b_b64_l4096()
    assert all(32 <= n <= 4096 for n in w3.init_lens)
    ins = [n for e in w3.steps for n in e.insert_lens]
    assert 2.0 < len(ins) / w3.n_steps < 6.5          # Poisson(4) arrivals
