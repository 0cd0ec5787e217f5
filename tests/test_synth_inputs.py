"""Properties of the seeded synthetic inputs that the parity tests rely on (CPU only).

The large workloads cut every weight tensor from one periodic stream of draws.
A kernel or residency bug that confuses expert e with expert e' can only be
seen if the two experts' bytes differ, so every expert blob of the
benchmark workloads (every layer, the shared experts included) must be
distinct -- and distinct part by part, since the gate/up and the down
matrices are read by different kernels.
"""
import hashlib

import numpy as np
import pytest

import synth


def _keys(wl):
    for l in range(wl.L):
        for e in range(wl.E):
            yield l, e
        if wl.shared:
            yield l, None


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_every_expert_blob_part_is_distinct(cfg):
    """Hash the first 16 Ki elements of each matrix of every blob (packed nibbles and scales separately for
    int4): all distinct per part, so no two blobs share a gate/up or a down matrix (distinct prefixes imply
    distinct contents)."""
    wl = synth.workload(cfg)
    seen = {}
    n = 0
    for l, e in _keys(wl):
        for name, part in synth.expert_blob_prefixes(wl, l, e, n=16384).items():
            h = hashlib.blake2b(part.tobytes(), digest_size=16).digest()
            other = seen.setdefault((name, h), (l, e))
            assert other == (l, e), f"cfg{cfg}: part {name} of {(l, e)} equals that of {other}"
        n += 1
    assert n == wl.L * (wl.E + (1 if wl.shared else 0))


@pytest.mark.parametrize("cfg", [3, 4, 5])
def test_window_starts_are_distinct_and_group_aligned(cfg):
    """Every tensor of a repeating stream starts at its own group-aligned element."""
    wl = synth.workload(cfg)
    P = synth._pool_size(wl)
    starts = [synth._tensor_offset(wl, l, "router") for l in range(wl.L)]
    starts += [synth._tensor_offset(wl, l, "expert" if e is not None else "shared", e or 0) for l, e in _keys(wl)]
    assert all(s % synth.GROUP == 0 and 0 <= s < P for s in starts)
    assert len(set(starts)) == len(starts)


@pytest.mark.parametrize("cfg", [3, 5])
def test_prefixes_are_the_blobs_own_bytes(cfg):
    """The prefix helper reads the same windows as expert_blob (checked on a few keys, shared included)."""
    wl = synth.workload(cfg, L=2)
    lay = synth.blob_layout(wl.H, wl.I, wl.dtype)
    for l, e in [(0, 0), (0, 64), (1, 255), (1, None)]:
        blob = synth.expert_blob(wl, l, e)
        for name, part in synth.expert_blob_prefixes(wl, l, e, n=4096).items():
            off = lay[name][0]
            assert np.array_equal(blob[off:off + part.size], part), (l, e, name)


def test_experts_sixty_four_apart_differ_at_the_largest_expert_count():
    """The case a 2^26-element period used to alias: experts e and e + 64 of a 256-expert int4 layer."""
    wl = synth.workload(5, L=1)
    assert not np.array_equal(synth.expert_blob(wl, 0, 0), synth.expert_blob(wl, 0, 64))
    wl3 = synth.workload(3)
    assert not np.array_equal(synth.expert_blob(wl3, 0, 3), synth.expert_blob(wl3, 0, 67))


def test_layer_experts_matches_expert_blob_on_a_repeating_stream():
    wl = synth.workload(2)
    lay = synth.layer_experts(wl, 0)
    for e in (0, 1, 77, 127):
        assert np.array_equal(lay[e], synth.expert_blob(wl, 0, e))


def test_small_workloads_keep_independent_consecutive_windows():
    """Workloads that fit one period draw every weight independently (consecutive windows, no repeats)."""
    wl = synth.workload(1)
    assert not synth._stream_repeats(wl)
    assert synth._tensor_offset(wl, 0, "expert", 1) - synth._tensor_offset(wl, 0, "expert", 0) == 3 * wl.I * wl.H
