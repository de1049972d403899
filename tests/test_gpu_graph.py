"""A decode step captured in a HIP graph (GPU): the mask and every layer's
attention, enqueued through torch's capture stream, then replayed.  The
library's kernels carry the step's state (L, base, the work list) by value and
record no memset, so each replay redoes the same step: the outputs equal those
of the step run eagerly on a twin cache, bit for bit, replay after replay with
other work in between, and so does the cache (the replayed append writes the
same column with the same values)."""
import numpy as np
import pytest
import torch

from tests import parity
from workload import configs, driver

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [("bf16", 2, 6, 8, 8, 128), ("bf16", 2, 5, 16, 2, 128)],
                         ids=["mha-bf16", "gqa8-bf16"])
def test_decode_step_in_a_hip_graph(shape):
    dtype, NL, B, Hq, Hkv, D = shape
    w = configs.small(dtype, NL, B, Hq, Hkv, D, L0=700, n_steps=2, n_evict=1, seed=51)
    eager, _ = driver.open_cache(w, split=256)
    graphed, inputs = driver.open_cache(w, split=256)
    dec = [inputs.decode(0, layer) for layer in range(NL)]
    torch.cuda.synchronize()

    mask_e = eager.build_mask()
    want = [eager.decode_attn(layer, *dec[layer]) for layer in range(NL)]
    torch.cuda.synchronize()

    # everything the captured calls touch exists before the capture
    mask_g = torch.empty_like(mask_e)
    outs = [torch.empty_like(x) for x in want]
    graphed.workspace()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed.build_mask(out=mask_g)
        for layer in range(NL):
            graphed.decode_attn(layer, *dec[layer], out=outs[layer])
    torch.cuda.synchronize()
    print(f"[graph] {shape}: captured {NL} layers", flush=True)
    for rep in range(3):
        for o in outs:
            o.fill_(float("nan"))            # eager work between the replays
        _ = torch.randn(1 << 16, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(mask_g, mask_e), f"replay {rep}: mask"
        for layer in range(NL):
            assert np.array_equal(parity.host_bits(outs[layer]), parity.host_bits(want[layer])), \
                f"replay {rep} layer {layer}: outputs differ from the eager step"
    eager.advance()
    graphed.advance()
    torch.cuda.synchronize()
    assert eager.query() == graphed.query()
    assert np.array_equal(parity.host_bits(eager.k), parity.host_bits(graphed.k))
    assert np.array_equal(parity.host_bits(eager.v), parity.host_bits(graphed.v))
    del g
    eager.close()
    graphed.close()


@pytest.mark.parametrize("shape", [("bf16", 1, 6, 8, 8, 128), ("bf16", 1, 5, 16, 2, 128)],
                         ids=["mha-bf16", "gqa8-bf16"])
def test_decode_step_over_holey_rows_in_a_hip_graph(shape):
    """After in-batch prefill steps the rows keep one-token runs behind their
    holes, which the attention reads as gathered items (token lists in the
    workspace, written by the captured work-list launch): a decode step over
    such rows replays bit for bit like the eager one."""
    dtype, NL, B, Hq, Hkv, D = shape
    w = configs.small(dtype, NL, B, Hq, Hkv, D, L0=200, n_steps=6, n_evict=1, new_hi=60, seed=52)
    eager, inputs = driver.open_cache(w, no_pd=True)
    graphed, _ = driver.open_cache(w, no_pd=True)
    for s, ev in enumerate(w.steps):
        for c in (eager, graphed):
            driver.run_step_no_pd(c, inputs, s, ev, mask=False)
    s = len(w.steps)
    dec = [inputs.decode(s, layer) for layer in range(NL)]
    torch.cuda.synchronize()

    mask_e = eager.build_mask()
    want = [eager.decode_attn(layer, *dec[layer]) for layer in range(NL)]
    torch.cuda.synchronize()

    mask_g = torch.empty_like(mask_e)
    outs = [torch.empty_like(x) for x in want]
    graphed.workspace()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed.build_mask(out=mask_g)
        for layer in range(NL):
            graphed.decode_attn(layer, *dec[layer], out=outs[layer])
    torch.cuda.synchronize()
    print(f"[graph holey] {shape}: captured {NL} layers after {s} prefill steps", flush=True)
    for rep in range(3):
        for o in outs:
            o.fill_(float("nan"))
        _ = torch.randn(1 << 16, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(mask_g, mask_e), f"replay {rep}: mask"
        for layer in range(NL):
            assert np.array_equal(parity.host_bits(outs[layer]), parity.host_bits(want[layer])), \
                f"replay {rep} layer {layer}: outputs differ from the eager step"
    eager.advance()
    graphed.advance()
    torch.cuda.synchronize()
    assert eager.query() == graphed.query()
    assert np.array_equal(parity.host_bits(eager.k), parity.host_bits(graphed.k))
    assert np.array_equal(parity.host_bits(eager.v), parity.host_bits(graphed.v))
    del g
    eager.close()
    graphed.close()
