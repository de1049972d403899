"""Baton without prefill/decode separation on the GPU (sec. 4.1): new queries
prefilled inside the batch (baton_shape_insert), holes left in the other rows,
the holey mask, causal prefill attention and later decode steps over holey
rows -- in lockstep with the materialized oracle: ring bit for bit, mask bit
for bit, token counts, every output within tolerance, and positions that hold
no token left untouched."""
import json
import os

import numpy as np
import pytest

from tests import oracle_pins, parity

pytestmark = pytest.mark.gpu

SHAPES = [("f32", 1, 4, 4, 4, 64), ("f32", 2, 5, 8, 2, 128), ("bf16", 2, 6, 8, 8, 128),
          ("bf16", 1, 5, 16, 2, 128), ("bf16", 1, 4, 4, 2, 64)]


def _sid(s):
    return f"{s[0]}-{s[1]}x{s[2]}-{s[3]}/{s[4]}x{s[5]}"


def _golden_ops():
    """The hand-derived replay's operations (tests/golden/inbatch_prefill_replay.json)."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "inbatch_prefill_replay.json")
    ops, s = [], 0
    for op in json.load(open(path))["ops"]:
        if op["op"] in ("embed", "shape"):
            ops.append((op["op"], op["slots"], op["lens"], op["qids"]))
        elif op["op"] == "evict":
            ops.append(("evict", op["slots"]))
        else:
            ops.append(("step", s))
            s += 1
    return ops


def _random_ops(seed, B, steps, max_len):
    rng = np.random.default_rng(seed)
    ops, qid, s = [], 0, 0
    for op in oracle_pins._random_ops_shaped(rng, B, steps, max_len):
        if op[0] in ("embed", "shape"):
            qids = list(range(qid, qid + len(op[1])))
            qid += len(op[1])
            ops.append((op[0], op[1], op[2], qids))
            if op[0] == "shape":
                ops.append(("step", s))
                s += 1
        elif op[0] == "evict":
            ops.append(op)
        else:
            ops.append(("step", s))
            s += 1
    return ops


@pytest.mark.parametrize("shape", SHAPES, ids=_sid)
def test_golden_story(shape):
    dtype, NL, _, Hq, Hkv, D = shape
    err = parity.run_script((dtype, NL, 3, Hq, Hkv, D), _golden_ops(), capacity=64)
    print(f"[inbatch golden] {shape}: max abs error {err:.3g}", flush=True)


@pytest.mark.parametrize("shape", [s for s in SHAPES if s[1] > 1], ids=_sid)
def test_random_sequences_separate_buffers(shape):
    """Prefill steps with K and V in two allocations of their own (packed layers)."""
    dtype, NL, B, Hq, Hkv, D = shape
    ops = _random_ops(7, B, steps=10, max_len=70)
    err = parity.run_script(shape, ops, capacity=2048, split=64, layout="separate")
    print(f"[inbatch random] {shape} separate buffers: {len(ops)} ops, max abs error {err:.3g}", flush=True)


@pytest.mark.parametrize("shape", SHAPES, ids=_sid)
@pytest.mark.parametrize("seed", [0, 1])
def test_random_sequences(shape, seed):
    dtype, NL, B, Hq, Hkv, D = shape
    ops = _random_ops(seed * 10 + len(shape[0]), B, steps=14, max_len=70)
    err = parity.run_script(shape, ops, capacity=2048, split=64)
    print(f"[inbatch random] {shape} seed {seed}: {len(ops)} ops, max abs error {err:.3g}", flush=True)


def test_long_prompts_and_wrap():
    """Prompts spanning many tiles and key blocks (up to 300 tokens), several
    prefills in one step with different lengths, a ring that wraps."""
    ops = [("embed", [0, 1, 2], [100, 40, 7], [0, 1, 2]), ("step", 0),
           ("evict", [1]), ("shape", [1], [300], [3]), ("step", 1), ("step", 2),
           ("evict", [0, 2]), ("shape", [2, 0], [129, 33], [4, 5]), ("step", 3),
           ("evict", [1]), ("embed", [1], [60], [6]), ("step", 4),
           ("evict", [2]), ("shape", [2], [250], [7]), ("step", 5), ("step", 6)]
    for shape in (("bf16", 1, 3, 8, 8, 128), ("bf16", 1, 3, 16, 2, 64), ("f32", 1, 3, 4, 2, 128)):
        err = parity.run_script(shape, ops, capacity=800, split=64)
        print(f"[inbatch long] {shape}: max abs error {err:.3g}", flush=True)


def test_extract_with_holes():
    """A query with holes stored aside and re-inserted: its tokens come back in
    order without the holes, and it decodes on as the oracle says."""
    ops = [("embed", [0, 1], [20, 9], [0, 1]), ("step", 0),
           ("shape", [2], [12], [2]), ("step", 1), ("step", 2),
           ("evict", [1]), ("shape", [1], [5], [3]), ("step", 3),
           ("extract", [0, 2], "holey"), ("evict", [0, 2]), ("step", 4),
           ("embed_saved", [3, 0], "holey"), ("step", 5), ("step", 6)]
    for shape in (("bf16", 2, 4, 8, 2, 128), ("f32", 1, 4, 4, 4, 64)):
        err = parity.run_script(shape, ops, capacity=256, split=64)
        print(f"[inbatch extract] {shape}: max abs error {err:.3g}", flush=True)


@pytest.mark.parametrize("scale", [1.0, -0.5])
def test_peaked_and_negative_scale(scale):
    """Prompts and decode rows with a peaked softmax (scale 1 at head_dim 128)
    and with a negative scale, whose sign the prefill kernel folds into q."""
    ops = [("embed", [0, 1, 2], [100, 40, 7], [0, 1, 2]), ("step", 0),
           ("evict", [1]), ("shape", [1], [200], [3]), ("step", 1), ("step", 2),
           ("evict", [0, 2]), ("shape", [2, 0], [129, 33], [4, 5]), ("step", 3), ("step", 4)]
    for shape in (("bf16", 1, 3, 8, 8, 128), ("bf16", 1, 3, 16, 2, 64), ("f32", 1, 3, 4, 2, 128)):
        err = parity.run_script(shape, ops, capacity=600, split=64, scale=scale)
        print(f"[inbatch scale {scale}] {shape}: max abs error {err:.3g}", flush=True)


def test_holes_with_unscrubbed_evictions():
    """In-batch prefill and holes after evictions that leave stale tokens
    (no BATON_SCRUB) and do not release: live tokens, mask and outputs as the
    oracle says."""
    ops = [("embed", [0, 1, 2], [30, 12, 50], [0, 1, 2]), ("step", 0),
           ("evict", [1], False, False), ("shape", [1], [20], [3]), ("step", 1),
           ("evict", [2], False, False), ("embed", [2], [9], [4]), ("step", 2),
           ("evict", [0], True, False), ("shape", [0], [6], [5]), ("step", 3), ("step", 4),
           ("evict", [], True, False), ("step", 5)]
    for shape in (("bf16", 2, 3, 8, 2, 128), ("f32", 1, 3, 4, 4, 64)):
        err = parity.run_script(shape, ops, capacity=256, split=64)
        print(f"[inbatch stale] {shape}: max abs error {err:.3g}", flush=True)


@pytest.mark.parametrize("shape", [("f32", 1, 3, 4, 4, 128), ("bf16", 1, 3, 8, 8, 128), ("bf16", 1, 3, 4, 4, 64),
                                   ("bf16", 1, 3, 16, 2, 128), ("bf16", 1, 3, 8, 4, 64)], ids=_sid)
def test_gathered_items(shape):
    """A row that lives through many prefill steps keeps a short run (the
    tokens it decoded since the last one) behind each hole; the attention
    kernels read such runs as gathered items of at most one pass of a
    workgroup (VALU: 32, 64 and 128 tokens for the first three shapes, more
    than the split at head_dim 64; matrix cores, grouped heads: 64):
    slot 0 ends with some 70 tokens in short runs behind 19 holes (several
    gathered items, the last with the current token), slot 1 (a 10-token
    prompt) is short runs only, slot 2 is prefilled again and again with
    prompts of 3-40 tokens."""
    prompts = [5, 23, 40, 7, 31, 12, 3, 37]
    ops = [("embed", [0], [100], [0]), ("shape", [1], [10], [1]), ("step", 0)]
    s, qid = 1, 2
    for c in range(18):
        if c:
            ops.append(("evict", [2]))
        ops += [("shape", [2], [prompts[c % len(prompts)]], [qid]), ("step", s)]
        qid, s = qid + 1, s + 1
        for _ in range(c % 5 + 1):
            ops.append(("step", s))
            s += 1
    err = parity.run_script(shape, ops, capacity=1024, split=64)
    print(f"[inbatch gathered] {shape}: {s} steps, max abs error {err:.3g}", flush=True)


@pytest.mark.parametrize("shape", [("bf16", 1, 4, 8, 2, 128), ("bf16", 1, 4, 4, 4, 64), ("f32", 1, 4, 4, 4, 128)],
                         ids=_sid)
def test_many_holes_rows_of_different_ages(shape):
    """Sixty holes held by rows of different ages: slot 0 lives through every
    prefill step, slot 1 is prefilled again and again, slot 2 is embedded
    (prefilled elsewhere) after 20 of them and slot 3 prefilled in the batch
    after 40, so each row holds its own suffix of the hole list.  The run
    behind a hole is the prefill step's one token and up to two decode steps,
    or (twice) 66 decode steps: listed runs, runs cut into a piece of the
    split (64) and a remainder, and back-to-back short runs in one work list
    (66 tokens are listed at head_dim 64, whose gathered items hold 128)."""
    prompts = [5, 23, 40, 7, 31, 12, 3, 37, 2, 18]
    ops = [("embed", [0], [150], [0]), ("step", 0)]
    s, qid = 1, 1
    for c in range(60):
        if c:
            ops.append(("evict", [1]))
        if c == 20:
            ops.append(("embed", [2], [90], [qid]))
            qid += 1
        slots, lens = [1], [prompts[c % len(prompts)]]
        if c == 40:
            slots, lens = [1, 3], [lens[0], 25]
        ops += [("shape", slots, lens, list(range(qid, qid + len(slots)))), ("step", s)]
        qid, s = qid + len(slots), s + 1
        for _ in range(66 if c in (10, 35) else c % 3):
            ops.append(("step", s))
            s += 1
    err = parity.run_script(shape, ops, capacity=2048, split=64)
    print(f"[inbatch many holes] {shape}: {s} steps, max abs error {err:.3g}", flush=True)
