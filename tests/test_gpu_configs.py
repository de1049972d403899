"""The HIP path at the benchmark workloads' full sizes (GPU), in the launch
configuration bench.py times.  b32-L2048 is compared whole against the
materialized oracle; larger ones at sampled (step, layer, slot) points (whole
K/V rows bit-exact, every q-head's output within tolerance), with metadata at
every step and, at the end, the placeholder invariant over the whole ring."""
import pytest

from tests import parity
from workload import configs

pytestmark = pytest.mark.gpu


def test_b32_l2048_whole():
    w = configs.b32_l2048()
    print(f"[configs] b32-L2048 whole: B={w.batch} L0={w.L0} steps={w.n_steps}", flush=True)
    err = parity.run(w, check_every_op=False)
    print(f"[configs] b32-L2048 max abs error {err:.3g}", flush=True)


@pytest.mark.parametrize("name,steps,layers,kw", [
    ("7b-b64-L4096", {0, 31, 63}, {0, 17, 31}, {}),
    ("skew-b256-L32768", {0, 7, 15}, {0}, {}),
    ("skew-growth-b256-L32768", {0, 1, 8, 16}, {0}, {}),
])
def test_sampled(name, steps, layers, kw):
    w = configs.CONFIGS[name]()
    print(f"[configs] {name} sampled: B={w.batch} L0={w.L0} layers={w.n_layers} steps={w.n_steps}",
          flush=True)
    err, n = parity.run_sampled(w, steps, layers, **kw)
    print(f"[configs] {name}: {n} outputs checked, max abs error {err:.3g}", flush=True)
    assert n > 0


def test_70b_gqa_resident_layers():
    """70b-gqa-b128-L8192's per-layer shape (GQA 64/8, B=128, L=8192) with 24 of its 80
    layers resident -- the dense padded 80-layer cache (343.6 GB) exceeds HBM."""
    w = configs.gqa70b_b128_l8192(n_steps=6, n_layers=24)
    print(f"[configs] 70b-gqa-b128-L8192 24 layers sampled", flush=True)
    err, n = parity.run_sampled(w, {0, 5}, {0, 23}, n_slots=3)
    print(f"[configs] 70b-gqa-b128-L8192: {n} outputs checked, max abs error {err:.3g}", flush=True)


def test_b32_l2048_no_pd_sampled():
    """b32-L2048's schedule without prefill/decode separation, as bench.py --no-pd
    runs it (2 + 16 steps, every step prefilling two queries inside the batch)."""
    w = configs.b32_l2048(18)
    print(f"[configs] b32-L2048 no-P&D sampled: capacity {w.capacity_no_pd()}", flush=True)
    err, n = parity.run_sampled_no_pd(w, {0, 1, 9, 17}, heads=(0, 31))
    print(f"[configs] b32-L2048 no-P&D: {n} outputs checked, max abs error {err:.3g}", flush=True)
    assert n > 0
