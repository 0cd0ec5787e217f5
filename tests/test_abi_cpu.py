"""CPU checks of the C-ABI library: it loads, exports every declared entry point,
and its residency runtime (host-simulation mode, no HIP calls) makes the same
decisions as the oracle's LRU."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
import paper_2605_29135_amd as moe
from paper_2605_29135_amd import binding

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_library_exports_exactly_the_header_entry_points():
    names = moe.header_symbols()
    assert "moe_route_topk" in names and "expert_cache_lookup" in names
    lib = moe.lib()
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if re.search(r" T ", ln)}
    assert exported == set(names)


def test_workspace_bytes_covers_activations_and_group_table():
    for T, k, I in [(1, 8, 768), (4, 8, 512), (16, 8, 512), (16, 16, 128)]:
        n = moe.moe_ffn_workspace_bytes(T, k, I)
        assert n >= 4 * (T * k + T) * I + 4 * (4 + 3 * (T * k + 1) + T * k + T)
        assert n % 256 == 0


class SimStore:
    """Host store whose expert (l, e) blob is filled with a tag of its key."""

    def __init__(self, L, E, eb=256, layer_stride=None):
        self.L, self.E, self.eb = L, E, eb
        self.buf = np.zeros(L * E * eb, np.uint8)
        for l in range(L):
            for e in range(E):
                self.buf[(l * E + e) * eb:(l * E + e + 1) * eb] = np.frombuffer(
                    np.full(eb // 4, l * E + e, np.int32).tobytes(), np.uint8)
        self.layer_stride = E * eb if layer_stride is None else layer_stride

    def cache(self, C_slots, preload=False, policy=moe.MOE_POLICY_LRU, charge_max=0):
        return moe.ExpertCache(self.L, self.E, self.eb, C_slots * self.eb, self.buf.ctypes.data,
                               self.layer_stride, self.eb, preload=preload, host_sim=True, policy=policy,
                               charge_max=charge_max)


def _pool_key(cache, slot, eb):
    _, pool = cache.slot_table()
    return np.frombuffer(C.string_at(pool + int(slot) * eb, eb), np.int32)


def _table(cache, L, E):
    t, _ = cache.slot_table()
    return np.frombuffer(C.string_at(t, 4 * L * E), np.int32)


def _as_tuples(ev):
    return [tuple(int(v) for v in e) for e in ev]


def _random_trace(rng, steps, L, E, n):
    return [(int(rng.integers(0, L)), rng.integers(0, E, size=n)) for _ in range(steps)]


@pytest.mark.parametrize("seed,L,E,n,C_slots", [(0, 2, 12, 3, 5), (1, 3, 16, 8, 8), (2, 1, 40, 8, 20),
                                                 (3, 4, 128, 8, 60)])
def test_sim_cache_matches_oracle_lru(seed, L, E, n, C_slots):
    rng = np.random.default_rng(seed)
    st = SimStore(L, E)
    c = st.cache(C_slots)
    o = oracle.LRU(C_slots, L, E)
    for t, (l, ids) in enumerate(_random_trace(rng, 300, L, E, n)):
        slots, hit = c.lookup(t, l, ids)
        assert o.lookup(t, l, ids) == oracle.OK
        for i, e in enumerate(ids):
            assert slots[i] == o.slot_of(l, int(e))
            # the filled slot holds that expert's blob
            assert (_pool_key(c, slots[i], st.eb) == l * E + e).all()
        c.release()
    assert _as_tuples(c.trace()) == _as_tuples(o.events())
    s, so = c.stats(), o.stats()
    assert (s["hits"], s["misses"], s["evictions"]) == (so["hits"], so["misses"], so["evictions"])
    assert s["occupancy"] == o.occupancy() <= C_slots
    assert s["h2d_bytes"] == s["misses"] * st.eb
    table = _table(c, L, E)
    for l in range(L):
        for e in range(E):
            assert table[l * E + e] == o.slot_of(l, e)


def test_sim_cache_prefetch_matches_oracle():
    rng = np.random.default_rng(7)
    L, E, C_slots = 2, 20, 9
    st = SimStore(L, E)
    c = st.cache(C_slots)
    o = oracle.LRU(C_slots, L, E)
    for t in range(400):
        l = int(rng.integers(0, L))
        ids = rng.integers(0, E, size=int(rng.integers(1, 5)))
        pre = bool(rng.random() < 0.3)
        if pre:
            c.prefetch(t, l, ids)
        else:
            c.lookup(t, l, ids)
        assert o.lookup(t, l, ids, prefetch=pre) == oracle.OK
    assert _as_tuples(c.trace()) == _as_tuples(o.events())
    assert c.stats()["prefetches"] == o.stats()["prefetches"] > 0


@pytest.mark.parametrize("seed,L,E,n,C_slots,Q", [(0, 2, 12, 3, 5, 0), (1, 3, 16, 8, 8, 1), (2, 1, 40, 8, 20, 3),
                                                   (3, 4, 128, 8, 60, 32), (4, 2, 20, 4, 9, 2)])
def test_sim_cache_rotary_matches_oracle(seed, L, E, n, C_slots, Q):
    """The rotary slot group against the oracle's: demand lookups and prefetches, event for event."""
    rng = np.random.default_rng(50 + seed)
    st = SimStore(L, E)
    c = st.cache(C_slots, policy=moe.MOE_POLICY_ROTARY, charge_max=Q)
    o = oracle.Rotary(C_slots, L, E, charge_max=Q)
    for t in range(400):
        l = int(rng.integers(0, L))
        ids = rng.integers(0, E, size=int(rng.integers(1, n + 1)))
        pre = bool(rng.random() < 0.2)
        if pre:
            c.prefetch(t, l, ids)
        else:
            slots, _ = c.lookup(t, l, ids)
            for i, e in enumerate(ids):
                assert (_pool_key(c, slots[i], st.eb) == l * E + e).all()
            c.release()
        assert o.lookup(t, l, ids, prefetch=pre) == oracle.OK
    assert _as_tuples(c.trace()) == _as_tuples(o.events())
    s, so = c.stats(), o.stats()
    assert (s["hits"], s["misses"], s["prefetches"], s["evictions"]) == \
        (so["hits"], so["misses"], so["prefetches"], so["evictions"])
    assert s["occupancy"] == o.occupancy() <= C_slots
    table = _table(c, L, E)
    assert all(table[l * E + e] == o.slot_of(l, e) for l in range(L) for e in range(E))


def test_sim_cache_rotary_rejects_bad_charge():
    st = SimStore(1, 4)
    for q in (-1, 65536):
        with pytest.raises(moe.MoeError):
            st.cache(2, policy=moe.MOE_POLICY_ROTARY, charge_max=q)
    with pytest.raises(moe.MoeError):
        st.cache(2, policy=7)


def test_sim_cache_golden_step_sets():
    lines = [ln.split() for ln in open(os.path.join(GOLDEN, "lru_step_sets.txt"))
             if ln.strip() and not ln.startswith("#")]
    st = SimStore(1, 8)
    c = st.cache(3)
    for l in lines:
        if l[0] != "op":
            continue
        arrow = l.index("->")
        t, layer, ids, want = int(l[2]), int(l[3]), [int(v) for v in l[4:arrow]], int(l[arrow + 1])
        try:
            (c.prefetch if l[1] == "prefetch" else c.lookup)(t, layer, ids)
            got = 0
        except moe.MoeError as e:
            got = e.code
        assert got == want
    expect = [tuple(int(v) for v in l[1:]) for l in lines if l[0] == "ev"]
    assert _as_tuples(c.trace()) == expect


def test_sim_cache_layer_aliasing_keeps_keys_distinct():
    L, E = 3, 6
    st = SimStore(L, E, layer_stride=0)  # every layer reads layer 0's blobs
    c = st.cache(4)
    c.lookup(0, 0, [1])
    c.lookup(1, 2, [1])
    ev = c.trace()
    assert [int(e["kind"]) for e in ev] == [moe.EVENT_MISS, moe.EVENT_MISS]
    assert (_pool_key(c, int(ev[1]["slot"]), st.eb) == 1).all()


def test_sim_cache_preload_and_errors():
    L, E = 2, 5
    st = SimStore(L, E)
    c = st.cache(L * E, preload=True)
    assert list(_table(c, L, E)) == list(range(L * E))
    c.lookup(0, 1, [4, 0])
    assert c.stats()["misses"] == 0 and c.stats()["hits"] == 2
    small = st.cache(2)
    with pytest.raises(moe.MoeError) as ei:
        small.lookup(0, 0, [0, 1, 2])
    assert ei.value.code == -4  # budget
    with pytest.raises(moe.MoeError) as ei:
        small.lookup(0, 0, [5])
    assert ei.value.code == -2  # range
    with pytest.raises(moe.MoeError) as ei:
        small.lookup(0, 2, [0])
    assert ei.value.code == -1  # layer
    assert small.stats()["occupancy"] == 0 and len(small.trace()) == 0
    with pytest.raises(moe.MoeError) as ei:
        st.cache(0)
    assert ei.value.code == -4
    with pytest.raises(moe.MoeError) as ei:
        st.cache(L * E - 1, preload=True)
    assert ei.value.code == -4


def _zipf_steps(rng, L, E, k, steps, s=1.1):
    p = 1.0 / np.arange(1, E + 1) ** s
    p /= p.sum()
    perms = [rng.permutation(E) for _ in range(L)]
    out = []
    for t in range(steps):
        for layer in range(L):
            ids = np.sort(perms[layer][rng.choice(E, k, replace=False, p=p)]).astype(np.int32)
            out.append(layer * E + ids)
    return out


@pytest.mark.parametrize("seed,L,E,k,steps,C", [(0, 2, 16, 2, 60, 5), (1, 4, 32, 4, 200, 24),
                                                 (2, 40, 128, 8, 64, 682), (3, 3, 8, 8, 30, 8)])
def test_opt_fills_matches_oracle(seed, L, E, k, steps, C):
    """The library's offline bound (host code) equals the oracle's on Zipf traces, up to config 4's shape."""
    trace = _zipf_steps(np.random.default_rng(seed), L, E, k, steps)
    got = moe.moe_opt_fills(trace, L * E, C)
    assert got == oracle.opt_misses(trace, L * E, C)
    o = oracle.LRU(C, L, E)
    for i, keys in enumerate(trace):
        assert o.lookup(i, int(keys[0]) // E, keys % E) == oracle.OK
    assert got <= o.stats()["misses"]


def test_opt_fills_rejects_bad_traces():
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_opt_fills([[0, 1, 2]], 3, 2)
    assert ei.value.code == -4
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_opt_fills([[0, 5]], 3, 2)
    assert ei.value.code == -2
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_opt_fills([[1, 1]], 3, 2)
    assert ei.value.code == -1
    assert moe.moe_opt_fills([], 3, 2) == 0
