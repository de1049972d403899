"""HIP path vs the oracle on whole schedules (GPU): K/V ring and mask bit-exact
after every operation, attention within tolerance after every layer."""
import pytest

from tests import parity
from workload import configs

pytestmark = pytest.mark.gpu

SMALL = {
    # fp32, the tiny configuration: 4 slots, 4 heads, D=64, L=128, one insert into slot 2
    "tiny-f32": (configs.tiny_f32(), {}),
    # MHA bf16 D=128, rows spanning three 256-token splits, ragged tails
    "mha-bf16-d128": (configs.small("bf16", 2, 6, 8, 8, 128, L0=600, n_steps=4, n_evict=2, seed=31), {}),
    # GQA 4:1, bf16 D=128
    "gqa4-bf16-d128": (configs.small("bf16", 2, 5, 8, 2, 128, L0=300, n_steps=4, n_evict=2, seed=32), {}),
    # GQA 8:1, 64-token splits: many items per row and the combine kernel
    "gqa8-bf16-d128-split64": (configs.small("bf16", 1, 4, 16, 2, 128, L0=200, n_steps=3, n_evict=1, seed=33),
                               {"split": 64}),
    # fp32 D=128 (a token row spans 32 lanes), GQA 2:1
    "gqa2-f32-d128-split64": (configs.small("f32", 2, 4, 4, 2, 128, L0=150, n_steps=3, n_evict=2, seed=34),
                              {"split": 64}),
    # bf16 D=64 (8 lanes per row, 8 rows per instruction)
    "gqa2-bf16-d64-split64": (configs.small("bf16", 1, 7, 4, 2, 64, L0=500, n_steps=4, n_evict=3, seed=35),
                              {"split": 64}),
    # fp32 D=64 GQA 8:1
    "gqa8-f32-d64": (configs.small("f32", 1, 3, 8, 1, 64, L0=90, n_steps=3, n_evict=1, seed=36), {}),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_schedule_parity(name):
    w, kw = SMALL[name]
    print(f"[parity] {name}: {w.name}", flush=True)
    err = parity.run(w, **kw)
    print(f"[parity] {name}: max abs error {err:.3g}", flush=True)


@pytest.mark.parametrize("name", ["tiny-f32", "mha-bf16-d128", "gqa8-bf16-d128-split64", "gqa2-f32-d128-split64"])
def test_schedule_parity_separate_buffers(name):
    """The same schedules with K and V in two allocations of their own (packed
    layers) instead of one allocation interleaved by layer."""
    w, kw = SMALL[name]
    print(f"[parity] {name} separate buffers: {w.name}", flush=True)
    err = parity.run(w, layout="separate", **kw)
    print(f"[parity] {name} separate buffers: max abs error {err:.3g}", flush=True)


@pytest.mark.parametrize("name", ["mha-bf16-d128", "gqa2-f32-d128-split64"])
def test_schedule_parity_padded_layer_stride(name):
    """K and V with a layer stride beyond their rows (padding between layers):
    results as above, and the padding is never written."""
    w, kw = SMALL[name]
    print(f"[parity] {name} padded layer stride: {w.name}", flush=True)
    err = parity.run(w, layout="padded", **kw)
    print(f"[parity] {name} padded layer stride: max abs error {err:.3g}", flush=True)


def test_ring_wraparound_tight_capacity():
    """Capacity = the most the run can need: releases and growths move the window
    base across the end of the ring again and again."""
    w = configs.small("bf16", 1, 6, 4, 4, 64, L0=160, n_steps=10, n_evict=3, seed=41)
    cap = w.L0 + w.n_steps + 1
    print(f"[parity] wraparound cap={cap}", flush=True)
    parity.run(w, capacity=cap, split=64)


def test_explicit_scale():
    w = configs.small("f32", 1, 3, 2, 2, 64, L0=70, n_steps=2, n_evict=1, seed=42)
    parity.run(w, scale=0.3)


@pytest.mark.parametrize("name,release_every,scrub", [
    ("mha-bf16-d128", 3, True),                # release only every third step, then a closing release
    ("gqa8-bf16-d128-split64", 2, False),      # no placeholder bytes written at all
    ("tiny-f32", 1, False),
    ("gqa2-f32-d128-split64", 100, True),      # no release until the closing one
    ("gqa2-bf16-d64-split64", 100, False),
])
def test_schedule_parity_release_and_scrub(name, release_every, scrub):
    """Evictions without BATON_RELEASE (L keeps its leading placeholder columns
    until a later release, sec. 4.1 "Resources releasing") and without
    BATON_SCRUB (the finished queries' tokens stay as stale bytes that the mask
    alone excludes, sec. 4.1 KV_Cache paragraph): the live tokens, the mask and
    every output as the oracle says."""
    w, kw = SMALL[name]
    print(f"[parity] {name} release every {release_every}, scrub {scrub}", flush=True)
    err = parity.run(w, release_every=release_every, scrub=scrub, **kw)
    print(f"[parity] {name} release every {release_every}, scrub {scrub}: max abs error {err:.3g}", flush=True)


@pytest.mark.parametrize("scrub", [True, False])
def test_ring_wraparound_rare_release(scrub):
    """A tight ring with release every fourth step only: L grows past its
    leading placeholders, growth on insertion follows each release, and the
    window wraps around the end of the ring."""
    w = configs.small("bf16", 1, 6, 4, 4, 64, L0=160, n_steps=12, n_evict=3, seed=43)
    cap = w.L0 + w.n_steps + 1
    print(f"[parity] wraparound, release every 4, scrub {scrub}, cap={cap}", flush=True)
    parity.run(w, capacity=cap, split=64, release_every=4, scrub=scrub)


@pytest.mark.parametrize("name,scale", [
    ("mha-bf16-d128", 1.0),                    # the VALU kernel, bf16 (scores of spread ~11)
    ("gqa8-bf16-d128-split64", 1.0),           # the matrix-core kernel, 8 q-heads per kv-head
    ("gqa4-bf16-d128", 1.5),
    ("gqa2-f32-d128-split64", 1.0),            # the VALU kernel, fp32
    ("mha-bf16-d128", -1.0),                   # a negative scale
    ("gqa8-bf16-d128-split64", -0.7),
])
def test_peaked_softmax(name, scale):
    """A scale of 1 at head_dim 128 (about 11 times 1/sqrt(128)) makes each
    softmax nearly one-hot: the largest weights dwarf the rest, many fall below
    fp32's normal range and the bf16-rounded weights of the matrix-core kernel
    matter most."""
    w, kw = SMALL[name]
    print(f"[parity] {name} scale {scale}", flush=True)
    err = parity.run(w, scale=scale, **kw)
    print(f"[parity] {name} scale {scale}: max abs error {err:.3g}", flush=True)
