"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Hand-derived golden cases (tests/golden/), brute force on small inputs,
textbook special cases and invariants.  CPU only.
"""
import itertools
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle
import synth
from blobs import decode_blob, make_blob, swiglu_dense

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def _kv(lines):
    return {ln[0]: ln[1:] for ln in lines}


# ------------------------------------------------------------- routing ---
def test_golden_topk_softmax():
    g = _kv(_golden_lines("topk_softmax.txt"))
    z = np.array([float(v) for v in g["logits"]], np.float32)[None]
    ids, w, st = oracle.topk_softmax(z, int(g["k"][0]))
    assert st == oracle.OK
    assert ids[0].tolist() == [int(v) for v in g["ids"]]
    np.testing.assert_allclose(w[0], [float(v) for v in g["weights"]], rtol=1e-15, atol=0)


def _sorted_topk(z, k):
    return sorted(range(z.size), key=lambda e: (-float(z[e]), e))[:k]


@pytest.mark.parametrize("E,k", [(4, 1), (4, 2), (16, 2), (16, 16), (128, 8), (256, 8)])
def test_topk_matches_full_sort_with_ties(E, k):
    rng = np.random.default_rng(E * 100 + k)
    # few distinct values -> many ties; include both signed zeros
    vals = np.array([-2.0, -0.0, 0.0, 0.5, 1.0, 3.0], np.float32)
    z = vals[rng.integers(0, vals.size, size=(40, E))]
    ids, w, st = oracle.topk_softmax(z, k)
    assert st == oracle.OK
    for t in range(z.shape[0]):
        assert ids[t].tolist() == _sorted_topk(z[t], k)


def test_topk_k1_is_argmax_weight_one():
    z = np.random.default_rng(1).standard_normal((64, 32)).astype(np.float32)
    z[3, [4, 9]] = 10.0  # tie: np.argmax keeps the first
    ids, w, _ = oracle.topk_softmax(z, 1)
    assert ids[:, 0].tolist() == np.argmax(z, axis=1).tolist()
    assert (w == 1.0).all()


def test_topk_kE_is_plain_softmax():
    z = np.random.default_rng(2).standard_normal((16, 12)).astype(np.float32) * 3
    ids, w, _ = oracle.topk_softmax(z, 12)
    for t in range(16):
        ref = scipy.special.softmax(z[t].astype(np.float64))
        np.testing.assert_allclose(w[t], ref[ids[t]], rtol=1e-13)


def test_topk_invariants():
    z = np.random.default_rng(3).standard_normal((200, 128)).astype(np.float32)
    k = 8
    ids, w, _ = oracle.topk_softmax(z, k)
    assert ((ids >= 0) & (ids < 128)).all()
    assert all(len(set(r)) == k for r in ids.tolist())
    assert (np.diff(w, axis=1) <= 0).all()
    assert np.abs(w.sum(axis=1) - 1.0).max() <= k * 2.0 ** -52
    # the selected logits dominate the rest
    for t in range(200):
        rest = np.delete(z[t], ids[t])
        assert z[t, ids[t]].min() >= rest.max()


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf])
def test_topk_nonfinite_is_error(bad):
    z = np.zeros((3, 8), np.float32)
    z[1, 5] = bad
    ids, w, st = oracle.topk_softmax(z, 2)
    assert st == oracle.ERR_NONFINITE
    assert ids[1].tolist() == [-1, -1]
    assert ids[0].tolist() == [0, 1] and ids[2].tolist() == [0, 1]


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_router_logits_exact_on_integers(dtype):
    rng = np.random.default_rng(4)
    E, H, T = 16, 256, 5
    wi = rng.integers(-8, 9, size=(E, H))
    xi = rng.integers(-8, 9, size=(T, H))
    w = wi.astype(np.float32) if dtype == synth.F32 else synth.bf16_bits(wi.astype(np.float32))
    z = oracle.router_logits(xi.astype(np.float32), w, dtype)
    assert (z == (xi @ wi.T).astype(np.float64)).all()


def test_rmsnorm_closed_forms():
    H = 128
    x = np.zeros((3, H), np.float32)
    x[0, :2] = [3.0, 4.0]          # mean square 25/128
    x[1, :] = -2.5                 # constant row
    x[2, 5] = 1e-3                 # tiny row: eps dominates
    h = oracle.rmsnorm(x, eps=1e-6)
    np.testing.assert_allclose(h[0, :2], np.array([3.0, 4.0]) / math.sqrt(25 / 128 + 1e-6), rtol=1e-15)
    assert (h[0, 2:] == 0).all()
    np.testing.assert_allclose(h[1], -2.5 / math.sqrt(6.25 + 1e-6), rtol=1e-15)
    v = float(np.float32(1e-3))
    np.testing.assert_allclose(h[2, 5], v / math.sqrt(v * v / 128 + 1e-6), rtol=1e-15)


def test_rmsnorm_invariants():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((6, 2048)).astype(np.float32) * 3
    h = oracle.rmsnorm(x)
    np.testing.assert_allclose((h ** 2).mean(axis=1), 1.0, rtol=1e-6)   # unit RMS (eps is tiny)
    np.testing.assert_allclose(oracle.rmsnorm(x * np.float32(4.0)), h, rtol=1e-6)  # positive scale drops out
    np.testing.assert_allclose(oracle.rmsnorm(-x), -h, rtol=1e-15)


# ---------------------------------------------------------- expert FFN ---
def test_golden_swiglu_expert():
    lines = _golden_lines("swiglu_expert.txt")
    H = int(next(l for l in lines if l[0] == "H")[1])
    I = int(next(l for l in lines if l[0] == "I")[1])
    gu = np.zeros((2 * I, H), np.float32)
    d = np.zeros((H, I), np.float32)
    x = np.zeros(H, np.float32)
    y_ref = np.zeros(H)
    for l in lines:
        if l[0] == "weights":
            (gu if l[1] == "gu" else d)[int(l[2]), int(l[3])] = float(l[4])
        elif l[0] == "x":
            x[int(l[1])] = float(l[2])
        elif l[0] == "y":
            y_ref[int(l[1])] = float(l[2])
    for dtype in (synth.F32, synth.BF16):
        y = oracle.expert_forward(x, make_blob(gu, d, dtype), H, I, dtype)
        np.testing.assert_allclose(y, y_ref, rtol=1e-15, atol=0)


def _random_experts(rng, E, H, I, dtype, scale=0.05):
    blobs = [make_blob(rng.standard_normal((2 * I, H)) * scale, rng.standard_normal((H, I)) * scale, dtype)
             for _ in range(E)]
    return np.stack(blobs)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16, synth.INT4G128])
@pytest.mark.parametrize("shared", [False, True])
def test_ffn_matches_dense_all_experts_masked(dtype, shared):
    """Dense evaluation of every expert, weights masked to the top-k."""
    rng = np.random.default_rng(10 + dtype)
    E, H, I, T, k = 6, 128, 256, 3, 2
    ex = _random_experts(rng, E, H, I, dtype)
    sh = _random_experts(rng, 1, H, I, dtype)[0] if shared else None
    x = rng.standard_normal((T, H)).astype(np.float32)
    z = rng.standard_normal((T, E)).astype(np.float32)
    ids, w, _ = oracle.topk_softmax(z, k)
    y = oracle.moe_ffn(x, ids, w, ex, H, I, dtype, sh)
    dense = np.stack([swiglu_dense(x, *decode_blob(ex[e], H, I, dtype)) for e in range(E)], axis=1)
    mask = np.zeros((T, E))
    mask[np.arange(T)[:, None], ids] = w
    ref = np.einsum("te,teh->th", mask, dense)
    if shared:
        ref += swiglu_dense(x, *decode_blob(sh, H, I, dtype))
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-14)


def test_ffn_single_expert_is_plain_swiglu():
    rng = np.random.default_rng(11)
    H, I = 256, 128
    gu = rng.standard_normal((2 * I, H)).astype(np.float32) * 0.05
    d = rng.standard_normal((H, I)).astype(np.float32) * 0.05
    x = rng.standard_normal((1, H)).astype(np.float32)
    y = oracle.moe_ffn(x, np.array([[0]]), np.array([[1.0]]), make_blob(gu, d, synth.F32)[None], H, I, synth.F32)
    g = x.astype(np.float64) @ gu[0::2].T.astype(np.float64)
    u = x.astype(np.float64) @ gu[1::2].T.astype(np.float64)
    ref = (g * scipy.special.expit(g) * u) @ d.T.astype(np.float64)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-15)


def test_ffn_zero_up_rows_give_zero():
    rng = np.random.default_rng(12)
    H, I = 128, 128
    gu = rng.standard_normal((2 * I, H)).astype(np.float32)
    gu[1::2] = 0.0
    d = rng.standard_normal((H, I)).astype(np.float32)
    y = oracle.expert_forward(rng.standard_normal(H).astype(np.float32), make_blob(gu, d, synth.BF16), H, I,
                              synth.BF16)
    assert (y == 0.0).all()


def test_ffn_identical_experts_independent_of_routing():
    rng = np.random.default_rng(13)
    E, H, I, T, k = 8, 128, 128, 4, 3
    one = _random_experts(rng, 1, H, I, synth.BF16)[0]
    ex = np.stack([one] * E)
    x = rng.standard_normal((T, H)).astype(np.float32)
    ys = []
    for s in range(3):
        z = np.random.default_rng(100 + s).standard_normal((T, E)).astype(np.float32)
        ids, w, _ = oracle.topk_softmax(z, k)
        ys.append(oracle.moe_ffn(x, ids, w, ex, H, I, synth.BF16))
    single = np.stack([oracle.expert_forward(x[t], one, H, I, synth.BF16) for t in range(T)])
    for y in ys:
        np.testing.assert_allclose(y, single, rtol=1e-12, atol=1e-15)


def test_layer_permutation_equivariance():
    """Relabelling experts (router rows and blobs together) leaves the layer output unchanged."""
    rng = np.random.default_rng(14)
    E, H, I, T, k = 8, 128, 128, 5, 3
    ex = _random_experts(rng, E, H, I, synth.BF16)
    wr = synth.bf16_bits(rng.standard_normal((E, H)).astype(np.float32) * 0.1)
    x = rng.standard_normal((T, H)).astype(np.float32)
    perm = rng.permutation(E)

    def layer(wr_, ex_):
        z = oracle.router_logits(x, wr_, synth.BF16).astype(np.float32)
        ids, w, _ = oracle.topk_softmax(z, k)
        return oracle.moe_ffn(x, ids, w, ex_, H, I, synth.BF16)

    np.testing.assert_allclose(layer(wr, ex), layer(wr[perm], ex[perm]), rtol=1e-12, atol=1e-15)


def test_ffn_rejects_out_of_range_ids():
    ex = np.zeros((2, synth.expert_bytes(128, 128, synth.BF16)), np.uint8)
    with pytest.raises(ValueError):
        oracle.moe_ffn(np.zeros((1, 128), np.float32), np.array([[2]]), np.array([[1.0]]), ex, 128, 128, synth.BF16)


# ---------------------------------------------------------------- int4 ---
def test_int4_nibble_table_and_scales():
    table = {int(a): int(b) for a, b in _golden_lines("int4_nibbles.txt")}
    H = I = 128
    blob = np.zeros(synth.expert_bytes(H, I, synth.INT4G128), np.uint8)
    lay = synth.blob_layout(H, I, synth.INT4G128)
    oq, _, _ = lay["gu_q"]
    os_, _, _ = lay["gu_s"]
    # row 3 of W_gu: element c holds nibble c % 16; group 0 scale 0.5, group 0 of row 4 scale -3
    for c in range(H):
        nib = c % 16
        byte = oq + 3 * (H // 2) + c // 2
        blob[byte] |= nib if c % 2 == 0 else nib << 4
    blob[os_ + 2 * 3:os_ + 2 * 4] = synth.bf16_bits(np.array([0.5], np.float32)).view(np.uint8)
    for c in range(H):
        assert oracle.expert_weight(blob, H, I, synth.INT4G128, "gu", 3, c) == 0.5 * table[c % 16]
    blob[oq + 4 * (H // 2)] = 0x9F  # low nibble 15 -> -1, high nibble 9 -> -7
    blob[os_ + 2 * 4:os_ + 2 * 5] = synth.bf16_bits(np.array([-3.0], np.float32)).view(np.uint8)
    assert oracle.expert_weight(blob, H, I, synth.INT4G128, "gu", 4, 0) == 3.0
    assert oracle.expert_weight(blob, H, I, synth.INT4G128, "gu", 4, 1) == 21.0


def test_int4_roundtrip_and_quantizer_bound():
    rng = np.random.default_rng(15)
    H, I = 256, 128
    gu = rng.standard_normal((2 * I, H)).astype(np.float32) * 0.02
    d = rng.standard_normal((H, I)).astype(np.float32) * 0.02
    blob = make_blob(gu, d, synth.INT4G128)
    dgu, dd = decode_blob(blob, H, I, synth.INT4G128)
    for which, m, dm in (("gu", gu, dgu), ("d", d, dd)):
        rows, cols = m.shape
        for r, c in zip(rng.integers(0, rows, 200), rng.integers(0, cols, 200)):
            assert oracle.expert_weight(blob, H, I, synth.INT4G128, which, int(r), int(c)) == dm[r, c]
        # quantizer: every group's error is at most half a step (plus the bf16 scale rounding)
        s = np.abs(m).reshape(rows, cols // 128, 128).max(axis=2) / 7.0
        err = np.abs(m - dm).reshape(rows, cols // 128, 128).max(axis=2)
        assert (err <= 0.5 * s * (1 + 2.0 ** -7) + 1e-3 * s).all()


# ----------------------------------------------------------------- LRU ---
def _events_tuples(ev):
    return [tuple(int(v) for v in e) for e in ev]


def test_golden_lru_textbook():
    lines = _golden_lines("lru_textbook.txt")
    kv = {l[0]: l[1:] for l in lines if not l[0].lstrip("-").isdigit()}
    C, E = int(kv["capacity"][0]), int(kv["experts"][0])
    ref = [int(v) for v in kv["reference"]]
    c = oracle.LRU(C, 1, E)
    for t, e in enumerate(ref):
        assert c.lookup(t, 0, [e]) == oracle.OK
    assert c.stats()["misses"] == int(kv["faults"][0])
    expect = [tuple(int(v) for v in l) for l in lines if l[0].lstrip("-").isdigit()]
    assert _events_tuples(c.events()) == expect


def test_golden_lru_step_sets():
    lines = _golden_lines("lru_step_sets.txt")
    kv = {l[0]: l[1:] for l in lines if l[0] in ("capacity", "experts")}
    c = oracle.LRU(int(kv["capacity"][0]), 1, int(kv["experts"][0]))
    for l in lines:
        if l[0] == "op":
            arrow = l.index("->")
            t, layer, ids = int(l[2]), int(l[3]), [int(v) for v in l[4:arrow]]
            assert c.lookup(t, layer, ids, prefetch=(l[1] == "prefetch")) == int(l[arrow + 1])
    expect = [tuple(int(v) for v in l[1:]) for l in lines if l[0] == "ev"]
    assert _events_tuples(c.events()) == expect


def _random_trace(rng, steps, L, E, n):
    return [(int(rng.integers(0, L)), rng.integers(0, E, size=n)) for _ in range(steps)]


def _step_stack_hits(trace, C):
    """Brute force: hit iff (distinct keys used in later steps) + (keys of its
    last step with a larger id) < C."""
    hits = []
    last_step = {}
    step_sets = []
    for s, (layer, ids) in enumerate(trace):
        R = sorted(set(int(i) for i in ids))
        out = []
        for e in R:
            key = (layer, e)
            if key not in last_step:
                out.append(False)
                continue
            s0 = last_step[key]
            newer = set()
            for s1 in range(s0 + 1, s):
                newer |= step_sets[s1]
            # keys of step s0 stamped after `key`: the same layer, a larger id
            newer |= {kk for kk in step_sets[s0] if kk[1] > e}
            out.append(len(newer) < C)
        for e in R:
            last_step[(layer, e)] = s
        step_sets.append({(layer, e) for e in R})
        hits.append(out)
    return hits


@pytest.mark.parametrize("seed", range(6))
def test_lru_hits_match_step_stack_distance(seed):
    rng = np.random.default_rng(200 + seed)
    L, E, n = 2, 12, int(rng.integers(1, 5))
    trace = _random_trace(rng, 120, L, E, n)
    for C in range(n, 3 * E):
        c = oracle.LRU(C, L, E)
        got = []
        for t, (layer, ids) in enumerate(trace):
            first = len(c.events())
            assert c.lookup(t, layer, ids) == oracle.OK
            got.append([int(ev["kind"]) == oracle.HIT for ev in c.events(first)])
        assert got == _step_stack_hits(trace, C), f"C={C}"


def _recency_list_model(trace, C):
    """Brute force with an explicit recency list (most recent last) and a slot array."""
    recency, slots, events = [], [None] * C, []
    for t, (layer, ids) in enumerate(trace):
        R = sorted(set(int(i) for i in ids))
        step_keys = {(layer, e) for e in R}
        for e in R:
            key = (layer, e)
            if key in recency:
                recency.remove(key)
                recency.append(key)
                events.append((t, layer, e, 0, slots.index(key), -1))
                continue
            if None in slots:
                s, victim = slots.index(None), -1
            else:
                vk = next(kk for kk in recency if kk not in step_keys)
                s, victim = slots.index(vk), vk[0] * 1000 + vk[1]
                recency.remove(vk)
            slots[s] = key
            recency.append(key)
            events.append((t, layer, e, 1, s, victim))
    return events


@pytest.mark.parametrize("seed", range(4))
def test_lru_slots_and_victims_match_recency_list(seed):
    rng = np.random.default_rng(300 + seed)
    L, E = 3, 1000
    trace = [(int(rng.integers(0, L)), rng.integers(0, 10, size=int(rng.integers(1, 4)))) for _ in range(300)]
    for C in (3, 4, 7, 12):
        c = oracle.LRU(C, L, E)
        for t, (layer, ids) in enumerate(trace):
            c.lookup(t, layer, ids)
        assert _events_tuples(c.events()) == _recency_list_model(trace, C)


def test_lru_cyclic_trace_misses_every_time():
    C = 5
    c = oracle.LRU(C, 1, C + 1)
    for t in range(10 * (C + 1)):
        c.lookup(t, 0, [t % (C + 1)])
    assert c.stats() == dict(hits=0, misses=10 * (C + 1), prefetches=0, evictions=10 * (C + 1) - C)


def test_lru_compulsory_misses_only_when_everything_fits():
    rng = np.random.default_rng(16)
    trace = _random_trace(rng, 500, 4, 16, 8)
    distinct = {(l, int(e)) for l, ids in trace for e in ids}
    c = oracle.LRU(len(distinct), 4, 16)
    for t, (l, ids) in enumerate(trace):
        c.lookup(t, l, ids)
    st = c.stats()
    assert st["misses"] == len(distinct) and st["evictions"] == 0


def test_lru_inclusion_and_counts():
    rng = np.random.default_rng(17)
    L, E, n = 3, 32, 8
    trace = _random_trace(rng, 400, L, E, n)
    lookups = sum(len(set(ids.tolist())) for _, ids in trace)
    prev_hits = None
    prev_miss = None
    for C in range(n, L * E + 1, 5):
        c = oracle.LRU(C, L, E)
        occ = []
        for t, (l, ids) in enumerate(trace):
            c.lookup(t, l, ids)
            occ.append(c.occupancy())
        st = c.stats()
        assert st["hits"] + st["misses"] == lookups
        assert max(occ) <= C
        hits = {(int(e["t"]), int(e["expert"])) for e in c.events() if e["kind"] == oracle.HIT}
        if prev_hits is not None:
            assert prev_hits <= hits and st["misses"] <= prev_miss
        prev_hits, prev_miss = hits, st["misses"]


def test_lru_preload_all_resident():
    L, E = 2, 5
    c = oracle.LRU(L * E, L, E, preload=True)
    assert [c.slot_of(l, e) for l in range(L) for e in range(E)] == list(range(L * E))
    for t in range(20):
        c.lookup(t, t % L, [(t * 3) % E, (t * 7 + 1) % E])
    assert c.stats()["misses"] == 0


def test_lru_errors():
    c = oracle.LRU(2, 2, 4)
    assert c.lookup(0, 0, [4]) == oracle.ERR_RANGE
    assert c.lookup(0, 0, [-1]) == oracle.ERR_RANGE
    assert c.lookup(0, 2, [0]) == oracle.ERR_ARG
    assert c.lookup(0, 0, [0, 1, 2]) == oracle.ERR_BUDGET
    assert c.lookup(0, 0, [1, 1, 0, 1]) == oracle.OK  # duplicates count once
    assert c.occupancy() == 2 and len(c.events()) == 2
    with pytest.raises(ValueError):
        oracle.LRU(0, 1, 1)


# ------------------------------------------------------- rotary slot group ---
def test_golden_rotary_fifo_belady_anomaly():
    g = {}
    for line in _golden_lines("rotary_fifo_belady.txt"):
        g[line[0]] = [int(v) for v in line[1:]]
    ref = g["reference"]
    for C in (3, 4):
        c = oracle.Rotary(C, 1, 8, charge_max=0)
        lru = oracle.LRU(C, 1, 8)
        for t, e in enumerate(ref):
            assert c.lookup(t, 0, [e]) == oracle.OK
            lru.lookup(t, 0, [e])
        ev = c.events()
        miss = ev[ev["kind"] == oracle.MISS]
        assert c.stats()["misses"] == g[f"fifo{C}_faults"][0]
        assert miss["t"].tolist() == g[f"fifo{C}_fault_steps"]
        assert [v for v in miss["victim_key"].tolist() if v >= 0] == g[f"fifo{C}_victims"]
        if C == 3:
            assert miss["slot"].tolist() == g["fifo3_slots"]
        assert lru.stats()["misses"] == g[f"lru{C}_faults"][0]


def _second_chance_queue_model(trace, C, Q):
    """Generalised second chance written as a queue: entries wait in a queue in the order the hand meets
    them; the front entry goes to the back if the step needs it, or if it still holds a charge (spending
    one); otherwise it leaves and the newcomer joins at the back.  Hits add a charge up to Q.  trace items:
    (layer, ids, prefetch).  Returns (t, layer, expert, kind, slot, victim_key) tuples, victim keys as
    layer * 1000 + expert."""
    from collections import deque
    q = deque()                 # [key, slot] in hand order
    charge, slot_of, free = {}, {}, list(range(C))
    events = []
    for t, (layer, ids, pf) in enumerate(trace):
        R = sorted(set(int(e) for e in ids))
        need = {(layer, e) for e in R}
        for e in R:
            key = (layer, e)
            if key in slot_of:
                if not pf:
                    charge[key] = min(charge[key] + 1, Q)
                    events.append((t, layer, e, 0, slot_of[key], -1))
                continue
            if free:
                s, victim = free.pop(0), -1
                q.append([key, s])
            else:
                while True:
                    k0, s0 = q[0]
                    q.rotate(-1)
                    if k0 in need:
                        continue
                    if charge[k0] > 0:
                        charge[k0] -= 1
                        continue
                    break
                # the victim is now at the back: it becomes the newcomer's entry
                q[-1] = [key, s0]
                s, victim = s0, k0[0] * 1000 + k0[1]
                del slot_of[k0], charge[k0]
            slot_of[key], charge[key] = s, 0
            events.append((t, layer, e, 2 if pf else 1, s, victim))
    return events


@pytest.mark.parametrize("seed", range(4))
def test_rotary_matches_second_chance_queue(seed):
    rng = np.random.default_rng(700 + seed)
    L, E = 3, 1000
    trace = [(int(rng.integers(0, L)), rng.integers(0, 12, size=int(rng.integers(1, 4))), bool(rng.random() < 0.15))
             for _ in range(400)]
    for C in (3, 4, 7, 12):
        for Q in (0, 1, 2, 5):
            c = oracle.Rotary(C, L, E, charge_max=Q)
            for t, (layer, ids, pf) in enumerate(trace):
                assert c.lookup(t, layer, ids, prefetch=pf) == oracle.OK
            assert _events_tuples(c.events()) == _second_chance_queue_model(trace, C, Q)


def test_rotary_without_charge_evicts_in_entry_order():
    rng = np.random.default_rng(41)
    C = 6
    c = oracle.Rotary(C, 1, 40, charge_max=0)
    order = []
    for t in range(300):
        e = int(rng.integers(0, 40))
        c.lookup(t, 0, [e])
        ev = c.events()[-1]
        if ev["kind"] == oracle.MISS:
            if ev["victim_key"] >= 0:
                assert ev["victim_key"] == order.pop(0)   # the oldest entry leaves, hits notwithstanding
            order.append(e)
    assert len(order) == C


def test_rotary_charge_keeps_a_hot_expert():
    # expert 0 is used every step beside a cyclic sweep over C others: cyclic replacement evicts it once per
    # turn of the hand, a charged ring never does (each pass spends one charge, each step restores one)
    C = 5
    for Q, evicted in ((0, True), (1, False), (3, False)):
        c = oracle.Rotary(C, 1, 40, charge_max=Q)
        for t in range(200):
            c.lookup(2 * t, 0, [0])
            c.lookup(2 * t + 1, 0, [1 + t % C])
        ev = c.events()
        assert bool((ev["victim_key"] == 0).any()) == evicted


def test_rotary_counts_occupancy_and_compulsory_misses():
    rng = np.random.default_rng(43)
    L, E, n = 3, 32, 8
    trace = _random_trace(rng, 400, L, E, n)
    lookups = sum(len(set(ids.tolist())) for _, ids in trace)
    for C in (n, 13, 40):
        c = oracle.Rotary(C, L, E, charge_max=3)
        for t, (l, ids) in enumerate(trace):
            c.lookup(t, l, ids)
            assert c.occupancy() <= C
            assert all(c.slot_of(l, int(e)) >= 0 for e in ids)  # the step's experts are resident together
        st = c.stats()
        assert st["hits"] + st["misses"] == lookups
    distinct = {(l, int(e)) for l, ids in trace for e in ids}
    c = oracle.Rotary(len(distinct), L, E, charge_max=3)
    for t, (l, ids) in enumerate(trace):
        c.lookup(t, l, ids)
    assert c.stats()["misses"] == len(distinct) and c.stats()["evictions"] == 0


def test_rotary_errors_and_preload():
    c = oracle.Rotary(2, 2, 4, charge_max=1)
    assert c.lookup(0, 0, [4]) == oracle.ERR_RANGE
    assert c.lookup(0, 2, [0]) == oracle.ERR_ARG
    assert c.lookup(0, 0, [0, 1, 2]) == oracle.ERR_BUDGET
    with pytest.raises(ValueError):
        oracle.Rotary(2, 1, 4, charge_max=-1)
    p = oracle.Rotary(6, 2, 3, charge_max=2, preload=True)
    assert [p.slot_of(l, e) for l in range(2) for e in range(3)] == list(range(6))


def test_golden_recall_contexts():
    lines = _golden_lines("recall_contexts.txt")
    tokens = [[[int(v) for v in ln[2 + 2 * l:4 + 2 * l]] for l in range(3)] for ln in lines if ln[0] == "token"]
    for ln in (ln for ln in lines if ln[0] == "recalled"):
        M, ov, want = int(ln[1]), int(ln[2]), [int(v) for v in ln[3:]]
        rec = oracle.Recall(M, 2, ov)
        got = []
        for t, sets in enumerate(tokens):
            who, calls = rec.step(t, sets)
            got.append(who)
            assert [l for l, _ in calls] == ([1, 2] if who >= 0 else [])
            if who >= 0:
                assert [c[1] for c in calls] == tokens[who][1:]
            if (M, ov, t) == (1, 1, 4):
                v = next(ln2 for ln2 in lines if ln2[0] == "calls_t4_1_1")[1:]
                assert calls == [(int(v[0]), [int(v[1]), int(v[2])]), (int(v[3]), [int(v[4]), int(v[5])])]
        assert got == want, (M, ov, got)


def test_recall_prefetch_of_a_recurring_context_turns_misses_into_prefetch_hits():
    # two alternating contexts that do not fit together: without recall every layer's set misses on each
    # return; with recall (exact signatures) each later layer's set is prefetched and found resident
    L, k, C = 4, 2, 8   # one context needs L * k = 8 slots
    A = [[10 * l + 1, 10 * l + 2] for l in range(L)]
    B = [[10 * l + 5, 10 * l + 6] for l in range(L)]
    seq = [A, B] * 6
    plain = oracle.replay_decode(oracle.LRU(C, L, 64), seq)
    rec = oracle.replay_decode(oracle.LRU(C, L, 64), seq, oracle.Recall(4, k))
    sp, sr = plain.stats(), rec.stats()
    assert sp["misses"] == len(seq) * L * k                      # every lookup misses
    assert sr["misses"] == 2 * L * k + (len(seq) - 2) * k         # only layer 0 misses once both are remembered
    assert sr["prefetches"] == (len(seq) - 2) * (L - 1) * k
    for cache in (oracle.Rotary(C, L, 64, 3), oracle.LRU(C, L, 64)):
        oracle.replay_decode(cache, seq, oracle.Recall(4, k))
        assert cache.occupancy() <= C


# ------------------------------------------------------ decoder attention ---
def _bf16(a):
    return synth.bf16_bits(np.asarray(a, np.float32))


def _f(bits):
    return synth.bf16_to_f32(np.asarray(bits, np.uint16)).astype(np.float64)


def test_golden_rope_4d_and_properties():
    g = {ln[0]: [float(v) for v in ln[1:]] for ln in _golden_lines("rope_4d.txt")}
    out = oracle.rope(np.array(g["v"]), int(g["p"][0]), g["theta"][0])
    assert np.allclose(out, g["rotated"], rtol=0, atol=1e-12)
    rng = np.random.default_rng(3)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    assert np.array_equal(oracle.rope(q, 0), q)                                        # position 0: identity
    assert abs(np.linalg.norm(oracle.rope(q, 777)) - np.linalg.norm(q)) < 1e-9        # a rotation
    a = oracle.rope(q, 40) @ oracle.rope(k, 13)
    b = oracle.rope(q, 1040) @ oracle.rope(k, 1013)                                   # only m - n matters
    assert abs(a - b) < 1e-8


def _attn_weights(H, n_heads, n_kv, d, wq=None, wk=None, wv=None, wo=None, seed=0):
    rng = np.random.default_rng(seed)
    rnd = lambda r, c: rng.standard_normal((r, c)) * 0.05
    wq = rnd(n_heads * d, H) if wq is None else wq
    wk = rnd(n_kv * d, H) if wk is None else wk
    wv = rnd(n_kv * d, H) if wv is None else wv
    wo = rnd(H, n_heads * d) if wo is None else wo
    return _bf16(np.vstack([wq, wk, wv])), _bf16(wo)


def test_attention_single_position_returns_the_value_heads():
    H, n_heads, n_kv, d = 64, 4, 2, 16
    wqkv, wo = _attn_weights(H, n_heads, n_kv, d)
    x = np.random.default_rng(1).standard_normal(H).astype(np.float32)
    kc = np.zeros((n_kv, 8, d), np.uint16)
    vc = np.zeros_like(kc)
    y = oracle.attention_decode(x, wqkv, wo, kc, vc, 0, n_heads, n_kv)
    h = oracle.rmsnorm(x)[0]
    v = _f(_bf16(_f(wqkv[(n_heads + n_kv) * d:]) @ h)).reshape(n_kv, d)   # bf16 as the cache holds it
    att = np.concatenate([v[j // (n_heads // n_kv)] for j in range(n_heads)])
    assert np.allclose(y, x + _f(wo) @ att, rtol=0, atol=1e-9)
    assert np.array_equal(vc[:, 0], _bf16(v.astype(np.float32)))


def test_attention_zero_query_attends_uniformly():
    H, n_heads, n_kv, d, p = 32, 2, 1, 16, 5
    wqkv, wo = _attn_weights(H, n_heads, n_kv, d, wq=np.zeros((n_heads * d, H)))
    rng = np.random.default_rng(2)
    kc = _bf16(rng.standard_normal((n_kv, 8, d)))
    vc = _bf16(rng.standard_normal((n_kv, 8, d)))
    x = rng.standard_normal(H).astype(np.float32)
    y = oracle.attention_decode(x, wqkv, wo, kc, vc, p, n_heads, n_kv)
    mean_v = _f(vc[0, :p + 1]).mean(axis=0)     # positions 0..p, the new value included
    assert np.allclose(y, x + _f(wo) @ np.concatenate([mean_v, mean_v]), rtol=0, atol=1e-9)


def test_attention_two_positions_closed_form():
    """One head, d = 8, position 1: q = rope(rmsnorm(e0-ish)) makes the score of cached key alpha e0 equal to
    alpha cos(1) (up to the norms' eps), the new key and value are zero: y = x + beta sigma(score) 1.  Fixes the
    1/sqrt(d) scale, the rotation angle and pairing, the query norm, the softmax over both positions, W_o and
    the residual."""
    d = H = 8
    alpha, beta, eps = 2.0, 0.5, 1e-6
    wqkv, wo = _attn_weights(H, 1, 1, d, wq=np.eye(d), wk=np.zeros((d, H)), wv=np.zeros((d, H)), wo=np.eye(H))
    kc = np.zeros((1, 4, d), np.uint16)
    vc = np.zeros_like(kc)
    kc[0, 0] = _bf16(alpha * np.eye(d)[0])
    vc[0, 0] = _bf16(np.full(d, beta))
    x = (3.0 * np.eye(d)[0]).astype(np.float32)
    y = oracle.attention_decode(x, wqkv, wo, kc, vc, 1, 1, 1, theta=500.0, eps=eps)
    h0 = 3.0 / np.sqrt(9.0 / d + eps)                 # rmsnorm(x)[0]
    q0 = h0 / np.sqrt(h0 * h0 / d + eps)              # the query head's own norm
    score = q0 * np.cos(1.0) * alpha / np.sqrt(d)     # dims (0, 4) turned by 1 rad at position 1
    w0 = 1.0 / (1.0 + np.exp(-score))                 # softmax over (score, 0)
    assert np.allclose(y, x + beta * w0 * np.ones(d), rtol=0, atol=1e-7)


def test_attention_query_groups_share_their_key_value_head():
    n_heads, n_kv, d, p = 4, 2, 4, 3
    H = n_heads * d
    z = np.zeros((n_heads * d, H))
    wqkv, wo = _attn_weights(H, n_heads, n_kv, d, wq=z, wk=np.zeros((n_kv * d, H)), wv=np.zeros((n_kv * d, H)),
                             wo=np.eye(H))
    kc = np.zeros((n_kv, 4, d), np.uint16)
    vc = np.zeros_like(kc)
    vc[0, :p] = _bf16(np.ones(d))
    vc[1, :p] = _bf16(np.full(d, 2.0))
    x = np.random.default_rng(4).standard_normal(H).astype(np.float32)
    y = oracle.attention_decode(x, wqkv, wo, kc, vc, p, n_heads, n_kv)
    # uniform over 4 positions, the new value zero: heads 0, 1 read kv head 0, heads 2, 3 kv head 1
    assert np.allclose(y - x, np.r_[np.full(2 * d, 0.75), np.full(2 * d, 1.5)], rtol=0, atol=1e-12)


# ------------------------------------------------------------ OPT bound ---
def _golden_kv(name):
    kv = {}
    for line in open(os.path.join(GOLDEN, name)):
        if line.strip() and not line.startswith("#"):
            key, *vals = line.split()
            kv[key] = [int(v) for v in vals]
    return kv


def _brute_min_fills(steps, C):
    """Exhaustive search over every eviction choice: the fewest fills that keep each step's keys resident
    together with C slots (no prefetching: keys enter only when a step needs them)."""
    from functools import lru_cache

    @lru_cache(maxsize=None)
    def go(i, pos, resident):
        if i == len(steps):
            return 0
        st = steps[i]
        if pos == len(st):
            return go(i + 1, 0, resident)
        k = st[pos]
        if k in resident:
            return go(i, pos + 1, resident)
        if len(resident) < C:
            return 1 + go(i, pos + 1, resident | {k})
        best = None
        for v in resident:
            if v in st:  # the step's own keys stay resident
                continue
            r = 1 + go(i, pos + 1, (resident - {v}) | {k})
            best = r if best is None else min(best, r)
        return best if best is not None else 10 ** 9

    return go(0, 0, frozenset())


def test_opt_textbook_example():
    g = _golden_kv("opt_textbook.txt")
    steps = [[k] for k in g["reference"]]
    assert oracle.opt_misses(steps, g["experts"][0], g["capacity"][0]) == g["faults"][0] == len(g["fault_steps"])


@pytest.mark.parametrize("seed", range(150))
def test_opt_equals_exhaustive_search(seed):
    rng = np.random.default_rng(seed)
    n_keys = int(rng.integers(3, 8))
    C = int(rng.integers(1, 5))
    steps = []
    for _ in range(int(rng.integers(1, 13))):
        m = int(rng.integers(1, min(C, n_keys) + 1))
        steps.append(sorted(rng.choice(n_keys, m, replace=False).tolist()))
    assert oracle.opt_misses(steps, n_keys, C) == _brute_min_fills(tuple(tuple(s) for s in steps), C)


def test_opt_bounds_lru_and_simple_cases():
    rng = np.random.default_rng(11)
    E, L, k = 32, 2, 4
    p = 1.0 / np.arange(1, E + 1) ** 1.1
    p /= p.sum()
    steps, keys = [], []
    for t in range(300):
        layer = t % L
        ids = np.sort(rng.choice(E, k, replace=False, p=p)).astype(np.int32)
        steps.append((layer, ids))
        keys.append(layer * E + ids)
    distinct = len(np.unique(np.concatenate(keys)))
    prev = None
    for C in (k, 6, 10, 16, 24, distinct):
        o = oracle.LRU(C, L, E)
        for t, (layer, ids) in enumerate(steps):
            assert o.lookup(t, layer, ids) == oracle.OK
        lru = o.stats()["misses"]
        opt = oracle.opt_misses(keys, L * E, C)
        assert distinct <= opt <= lru
        if prev is not None:
            assert opt <= prev  # more slots never need more fills
        prev = opt
    assert oracle.opt_misses(keys, L * E, distinct) == distinct  # everything fits: compulsory fills only
    assert oracle.opt_misses([[0, 1, 2]], 3, 2) == -1  # a step larger than the cache
