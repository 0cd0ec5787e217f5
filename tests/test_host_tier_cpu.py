"""The host tier on the CPU: the oracle's model of its residency rule against a hand-derived trace and its
invariants, the library's rule (host-simulated cache, through the C ABI) against that model event for event,
and the library's host GEMV tier (moe_host_expert_ffn) against the oracle's expert FFN.

The paper's run recipe keeps some layers' experts in host memory and computes them on host cores (sec. 6,
Fig. 3); which experts the host serves is the library's rule (moe_cache_desc.host_layers / host_quota)."""
import ctypes as C
import os

import numpy as np
import pytest

import oracle
import paper_2605_29135_amd as moe
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def _tuples(ev):
    return [tuple(int(v) for v in e) for e in ev]


def _apply(model, lines):
    for ln in lines:
        if ln[0] == "op":
            arrow = ln.index("->")
            st = model.lookup(int(ln[2]), int(ln[3]), [int(v) for v in ln[4:arrow]], prefetch=ln[1] == "prefetch")
            assert st == int(ln[arrow + 1]), ln


# ------------------------------------------------------------ oracle pins ---
def test_golden_host_tier_trace():
    lines = _golden("host_tier.txt")
    kv = {ln[0]: ln[1:] for ln in lines}
    h = oracle.HostTier(oracle.LRU(int(kv["capacity"][0]), int(kv["layers"][0]), int(kv["experts"][0])),
                        int(kv["host_layers"][0]), int(kv["host_quota"][0]))
    _apply(h, lines)
    assert _tuples(h.events()) == [tuple(int(v) for v in ln[1:]) for ln in lines if ln[0] == "ev"]
    st = dict(zip(kv["stats"][0::2], (int(v) for v in kv["stats"][1::2])))
    assert h.stats() == st


def _trace(rng, steps, L, E, n, pf_every=0):
    out = []
    for t in range(steps):
        out.append((t, int(rng.integers(0, L)), rng.integers(0, E, size=n), False))
        if pf_every and t % pf_every == pf_every - 1:
            out.append((t, int(rng.integers(0, L)), rng.integers(0, E, size=2), True))
    return out


@pytest.mark.parametrize("seed", range(4))
def test_host_tier_without_host_share_is_plain_lru(seed):
    rng = np.random.default_rng(seed)
    L, E, C_ = 3, 16, 7
    h, o = oracle.HostTier(oracle.LRU(C_, L, E), 0, 0), oracle.LRU(C_, L, E)
    for t, l, ids, pf in _trace(rng, 200, L, E, 4, pf_every=7):
        assert h.lookup(t, l, ids, prefetch=pf) == o.lookup(t, l, ids, prefetch=pf)
    assert _tuples(h.events()) == _tuples(o.events())
    assert h.stats()["host"] == 0


@pytest.mark.parametrize("seed,N,Q", [(0, 0, 1), (1, 1, 2), (2, 0, 3), (3, 2, 1)])
def test_host_tier_invariants(seed, N, Q):
    """Host layers never touch a slot; elsewhere a lookup's host share is at most Q experts, none of them
    resident, and it keeps (within Q) every non-resident expert the layer's previous share held; the slot
    table sees exactly the rest; counts add up."""
    rng = np.random.default_rng(seed)
    L, E, C_ = 3, 12, 6
    h = oracle.HostTier(oracle.LRU(C_, L, E), N, Q)
    prev = [set() for _ in range(L)]
    n_ev = 0
    n_demand = 0
    for t, l, ids, pf in _trace(rng, 300, L, E, 3, pf_every=5):
        resident = {e for e in range(E) if h.slot_of(l, e) >= 0}
        assert h.lookup(t, l, ids, prefetch=pf) == oracle.OK
        ev = h.events(n_ev)
        n_ev += ev.size
        R = sorted({int(i) for i in ids})
        if pf:  # a prefetch logs its non-resident ids only, never a host event
            assert [int(e) for e in ev["expert"]] == sorted(set(R) - resident)
            assert not (ev["kind"] == oracle.HOST).any()
            continue
        assert [int(e) for e in ev["expert"]] == R
        n_demand += len(R)
        host = {int(e) for e in ev["expert"][ev["kind"] == oracle.HOST]}
        assert (ev["slot"][ev["kind"] == oracle.HOST] == -1).all()
        if l < N:
            assert host == set(R)
        else:
            assert len(host) <= Q and not (host & resident)
            sticky = {e for e in R if e in prev[l] and e not in resident}
            assert sticky <= host
            fresh = sorted(set(R) - resident - sticky)
            assert host - sticky == set(fresh[:max(0, Q - len(sticky))])
        prev[l] = host
    s = h.stats()
    assert s["hits"] + s["misses"] + s["host"] == n_demand


def test_host_tier_errors_change_nothing():
    h = oracle.HostTier(oracle.LRU(2, 1, 8), 0, 1)
    assert h.lookup(0, 0, [1, 2]) == oracle.OK
    before = _tuples(h.events())
    assert h.lookup(1, 0, [3, 4, 5]) == oracle.ERR_BUDGET
    assert h.lookup(1, 0, [9]) == oracle.ERR_RANGE
    assert _tuples(h.events()) == before and h.prev[0] == {1}


# ------------------------------------------- library rule (host simulation) ---
class _Store:
    def __init__(self, L, E, eb=256):
        self.L, self.E, self.eb = L, E, eb
        self.buf = np.zeros(L * E * eb, np.uint8)

    def cache(self, C_slots, host_layers, host_quota):
        return moe.ExpertCache(self.L, self.E, self.eb, C_slots * self.eb, self.buf.ctypes.data, self.E * self.eb,
                               self.eb, host_sim=True, host_layers=host_layers, host_quota=host_quota)


def test_library_host_tier_golden_trace():
    lines = _golden("host_tier.txt")
    kv = {ln[0]: ln[1:] for ln in lines}
    st = _Store(int(kv["layers"][0]), int(kv["experts"][0]))
    c = st.cache(int(kv["capacity"][0]), int(kv["host_layers"][0]), int(kv["host_quota"][0]))
    for ln in lines:
        if ln[0] != "op":
            continue
        arrow = ln.index("->")
        t, l, ids = int(ln[2]), int(ln[3]), [int(v) for v in ln[4:arrow]]
        want = int(ln[arrow + 1])
        if want == oracle.OK:
            if ln[1] == "prefetch":
                c.prefetch(t, l, ids)
            else:
                c.lookup(t, l, ids)
                c.release()
        else:
            with pytest.raises(moe.MoeError) as ei:
                c.lookup(t, l, ids)
            assert ei.value.code == want
    assert _tuples(c.trace()) == [tuple(int(v) for v in ln[1:]) for ln in lines if ln[0] == "ev"]
    s = c.stats()
    assert (s["hits"], s["misses"], s["prefetches"], s["evictions"], s["host_computed"]) == (4, 5, 1, 3, 9)
    assert s["lookups"] == 4 + 5 + 9


@pytest.mark.parametrize("seed,L,E,n,C_slots,N,Q", [(0, 3, 16, 4, 7, 1, 1), (1, 4, 32, 8, 20, 0, 3),
                                                    (2, 2, 64, 8, 12, 0, 2), (3, 5, 24, 6, 10, 2, 4)])
def test_library_host_tier_matches_oracle(seed, L, E, n, C_slots, N, Q):
    """Random lookups and prefetches: decisions event for event, the slots returned (MOE_SLOT_HOST for the
    host's share), the device slot table and the counters."""
    rng = np.random.default_rng(seed)
    st = _Store(L, E)
    c = st.cache(C_slots, N, Q)
    o = oracle.HostTier(oracle.LRU(C_slots, L, E), N, Q)
    n_ev = 0
    for t, l, ids, pf in _trace(rng, 400, L, E, n, pf_every=6):
        assert o.lookup(t, l, ids, prefetch=pf) == oracle.OK
        ev = o.events(n_ev)
        n_ev += ev.size
        if pf:
            c.prefetch(t, l, ids)
            continue
        slots, hit = c.lookup(t, l, ids)
        c.release()
        kind = {int(e): int(k) for e, k in zip(ev["expert"], ev["kind"])}
        for i, e in enumerate(ids):
            if kind[int(e)] == oracle.HOST:
                assert slots[i] == moe.MOE_SLOT_HOST and hit[i] == 0
            else:
                assert slots[i] == o.slot_of(l, int(e)) >= 0
                assert hit[i] == (kind[int(e)] == oracle.HIT)
    assert _tuples(c.trace()) == _tuples(o.events())
    s, so = c.stats(), o.stats()
    assert (s["hits"], s["misses"], s["prefetches"], s["evictions"], s["host_computed"]) == \
        (so["hits"], so["misses"], so["prefetches"], so["evictions"], so["host"])
    t_ptr, _ = c.slot_table()
    table = np.frombuffer(C.string_at(t_ptr, 4 * L * E), np.int32)
    for l in range(L):
        for e in range(E):
            assert table[l * E + e] == o.slot_of(l, e)


def test_fill_clock_needs_device_residency():
    st = _Store(2, 8)
    with pytest.raises(moe.MoeError):
        moe.ExpertCache(2, 8, 256, 4 * 256, st.buf.ctypes.data, 8 * 256, 256, host_sim=True, fill_clock=True)


def test_library_host_tier_rejects_bad_settings():
    st = _Store(2, 8)
    for N, Q in [(-1, 0), (3, 0), (0, -1), (0, 9)]:
        with pytest.raises(moe.MoeError):
            st.cache(4, N, Q)
    with pytest.raises(moe.MoeError):  # not with preload
        moe.ExpertCache(2, 8, 256, 16 * 256, st.buf.ctypes.data, 8 * 256, 256, host_sim=True, preload=True,
                        host_quota=1)


# ------------------------------------------------------- host GEMV tier ---
def _blobs(wl, seed):
    rng = np.random.default_rng(seed)
    gu = rng.normal(0, 0.02, (wl.E, 2 * wl.I, wl.H)).astype(np.float32)
    d = rng.normal(0, 0.02, (wl.E, wl.H, wl.I)).astype(np.float32)
    from blobs import make_blob
    return np.stack([make_blob(gu[e], d[e], wl.dtype) for e in range(wl.E)])


@pytest.mark.parametrize("dtype,H,I", [(synth.F32, 256, 128), (synth.BF16, 512, 384), (synth.BF16, 2048, 768),
                                       (synth.INT4G128, 512, 256), (synth.INT4G128, 2048, 512)])
def test_host_expert_ffn_matches_oracle(dtype, H, I):
    """y = sum_j w_j FFN_j(x) in fp32 on host cores against the fp64 oracle on the same stored weights, for
    0..k experts (weights in rank order), on 1, 3 and 8 threads: results equal bit for bit across thread
    counts (each output row is summed by one thread in rank order) and within 1e-5 normwise of the oracle."""
    wl = synth.Workload("host tier", H=H, E=6, k=4, I=I, dtype=dtype, cfg_id=150 + dtype)
    ex = _blobs(wl, dtype)
    rng = np.random.default_rng(3)
    x = rng.standard_normal(H).astype(np.float32)
    tiers = [moe.HostTier(n) for n in (1, 3, 8)]
    for n in range(0, wl.k + 1):
        ids = rng.choice(wl.E, n, replace=False).astype(np.int32)
        w = rng.random(n).astype(np.float32)
        ys = [t.expert_ffn(x, [ex[e] for e in ids], w, H, I, dtype) for t in tiers]
        for y in ys[1:]:
            assert np.array_equal(y, ys[0])
        if n == 0:
            assert not ys[0].any()
            continue
        ref = oracle.moe_ffn(x[None], ids[None], w[None].astype(np.float64), ex, H, I, dtype)[0]
        err = np.abs(ys[0] - ref).max() / np.abs(ref).max()
        assert err <= 1e-5, (n, err)
    for t in tiers:
        t.close()


def test_host_expert_ffn_rejects_bad_arguments():
    t = moe.HostTier(2)
    x = np.zeros(256, np.float32)
    blob = np.zeros(synth.expert_bytes(256, 128, synth.BF16), np.uint8)
    for H, I, dtype, n in [(200, 128, synth.BF16, 1), (256, 100, synth.BF16, 1), (256, 128, 7, 1),
                           (256, 128, synth.BF16, 17)]:
        with pytest.raises(moe.MoeError):
            t.expert_ffn(x, [blob] * n, np.ones(n, np.float32), H, I, dtype)
    t.close()
    with pytest.raises(moe.MoeError):
        moe.HostTier(-1)
