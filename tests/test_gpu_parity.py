"""Parity of the HIP path (through the C ABI) with the CPU oracle, on MI355X.

Tolerances: router logits normwise 1e-5 per token; top-k ids bit-exact given
the GPU's own fp32 logits; weights |w - w_ref| <= 1e-5 * max(1, |w_ref|);
expert FFN output normwise max|y - y_ref| / max|y_ref| per token <= 1e-5 (fp32
weights), 1e-2 (bf16), 3e-2 (int4) against the fp64 oracle on the same stored
weights; residency event logs byte-equal to the oracle replaying the same calls.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2605_29135_amd as moe
import synth

pytestmark = pytest.mark.gpu

TOL = {synth.F32: 1e-5, synth.BF16: 1e-2, synth.INT4G128: 3e-2}
DEV = torch.device("cuda:0")


@pytest.fixture(scope="module", autouse=True)
def _init():
    moe.moe_init(0)
    yield
    torch.cuda.synchronize()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def normwise(y, ref):
    y = np.atleast_2d(y).astype(np.float64)
    ref = np.atleast_2d(ref)
    return float(np.max(np.abs(y - ref).max(axis=1) / np.maximum(np.abs(ref).max(axis=1), 1e-30)))


def check_route(x, wr, rdtype, k, bias=None, norm=False):
    """Run moe_route_topk and check it against the oracle; returns (ids, weights) on the host."""
    h = torch.empty(x.shape, dtype=torch.float32, device=DEV) if (norm and x is not None) else None
    logits, ids, w = moe.moe_route_topk(None if x is None else dev(x), None if wr is None else dev(wr), rdtype, k,
                                        E=(wr.shape[0] if wr is not None else bias.shape[1]),
                                        logit_bias=None if bias is None else dev(bias), rmsnorm=norm, x_norm=h)
    moe.moe_sync_check()
    z = logits.cpu().numpy()
    if x is not None:
        xin = x
        if norm:
            href = oracle.rmsnorm(x)
            assert normwise(h.cpu().numpy(), href) <= 1e-6
            xin = href.astype(np.float32)
        zref = oracle.router_logits(xin, wr, rdtype) + (0 if bias is None else bias)
        assert normwise(z, zref) <= 1e-5
    o_ids, o_w, st = oracle.topk_softmax(z, k)
    assert st == oracle.OK
    g_ids, g_w = ids.cpu().numpy(), w.cpu().numpy()
    assert (g_ids == o_ids).all()
    assert (np.abs(g_w - o_w) <= 1e-5 * np.maximum(1.0, np.abs(o_w))).all()
    return g_ids, g_w


# ----------------------------------------------------------------- route ---
@pytest.mark.parametrize("cfg,T", [(1, 1), (2, 1), (3, 1), (3, 4), (3, 16), (2, 37)])
@pytest.mark.parametrize("norm", [False, True])
def test_route_parity_configs(cfg, T, norm):
    wl = synth.workload(cfg)
    wr = synth.router_weights(wl, 0)
    for step in range(3):
        x = synth.hidden_states(wl, step, T=T) * np.float32(1.0 + step)
        check_route(x, wr, wl.router_dtype, wl.k, norm=norm)


@pytest.mark.parametrize("norm", [False, True])
def test_route_prefill_chunk_and_ragged_tiles(norm):
    """Many-token routing (the matrix-core router): config 5's 2048-token chunk over 256 experts, a ragged
    70 x 130 case whose last token and expert tiles are partial, and hidden sizes that give a block's waves
    several rounds of loads or nothing to do."""
    wl = synth.workload(5, L=1)
    check_route(synth.prefill_states(wl), synth.router_weights(wl, 0), wl.router_dtype, wl.k, norm=norm)
    rng = np.random.default_rng(130)
    x = (rng.standard_normal((70, 384)) * 3.0).astype(np.float32)
    wr = synth.bf16_bits(rng.standard_normal((130, 384)).astype(np.float32) * 0.05)
    bias = rng.standard_normal((70, 130)).astype(np.float32)
    check_route(x, wr, synth.BF16, 5, bias, norm=norm)
    # the H range split over a block's waves: two rounds of loads per wave (H 4096), and fewer k steps than
    # waves (H 128: half the waves add nothing)
    for T_, H_, E_ in ((20, 4096, 48), (17, 128, 40)):
        x = (rng.standard_normal((T_, H_)) * 2.0).astype(np.float32)
        wr = synth.bf16_bits(rng.standard_normal((E_, H_)).astype(np.float32) * 0.05)
        check_route(x, wr, synth.BF16, 4, norm=norm)


def test_route_with_mask_bias_selects_the_drawn_sets():
    wl = synth.workload(3, T=16)
    wr = synth.router_weights(wl, 0)
    sets = synth.routing_sets(wl, steps=4, T=16)
    for t in range(4):
        bias = synth.mask_logits(wl, sets[t, 0])
        ids, _ = check_route(synth.hidden_states(wl, t, T=16), wr, wl.router_dtype, wl.k, bias)
        assert (np.sort(ids, axis=1) == sets[t, 0]).all()


@pytest.mark.parametrize("E,k", [(16, 16), (256, 1), (256, 16), (64, 3), (130, 5)])
def test_route_ties_and_edge_k(E, k):
    rng = np.random.default_rng(E + k)
    vals = np.array([-1.0, -0.0, 0.0, 0.25, 2.0], np.float32)
    bias = vals[rng.integers(0, vals.size, size=(9, E))]
    check_route(None, None, synth.F32, k, bias)
    H = 256
    x = rng.standard_normal((9, H)).astype(np.float32)
    wr = synth.bf16_bits(rng.standard_normal((E, H)).astype(np.float32) * 0.05)
    check_route(x, wr, synth.BF16, k, bias)


def test_route_nonfinite_raises_and_marks_token():
    bias = np.zeros((3, 32), np.float32)
    bias[1, 7] = np.nan
    _, ids, w = moe.moe_route_topk(None, None, synth.F32, 4, E=32, logit_bias=dev(bias))
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_sync_check()
    assert ei.value.code == -3
    assert (ids.cpu().numpy()[1] == -1).all() and (w.cpu().numpy()[1] == 0).all()
    assert (ids.cpu().numpy()[0] == [0, 1, 2, 3]).all()
    moe.moe_sync_check()  # flags were cleared


def test_route_rejects_bad_arguments():
    x = torch.zeros((1, 256), device=DEV)
    w = torch.zeros((300, 256), device=DEV)
    with pytest.raises(moe.MoeError):
        moe.moe_route_topk(x, w, synth.F32, 8)  # E > 256
    with pytest.raises(moe.MoeError):
        moe.moe_route_topk(x, w[:16], synth.F32, 17)  # k > E
    moe.moe_route_topk(x[:0], w[:16], synth.F32, 2)  # T = 0 is a no-op


# ------------------------------------------------------------------- FFN ---
_EXPERTS = {}


def _experts(wl):
    """Layer 0's routed experts [E x expert_bytes] and shared blob (cached per workload shape)."""
    key = (wl.cfg_id, wl.H, wl.E, wl.I, wl.L, wl.dtype, wl.shared)
    if key not in _EXPERTS:
        _EXPERTS.clear()
        ex = synth.layer_experts(wl, 0)
        sh = synth.expert_blob(wl, 0, None) if wl.shared else None
        _EXPERTS[key] = (ex, sh)
    return _EXPERTS[key]


def check_ffn(wl, x, ids, w, ex, sh, slot_perm=None, accumulate=False):
    E, eb = ex.shape
    if slot_perm is not None:  # expert e lives in slot slot_perm[e]
        pool_np = np.empty_like(ex)
        pool_np[slot_perm] = ex
        slot_of = dev(slot_perm.astype(np.int32))
    else:
        pool_np, slot_of = ex, None
    pool = dev(pool_np.reshape(-1))
    xd = dev(x)
    base = np.random.default_rng(0).standard_normal(x.shape).astype(np.float32)
    y = dev(base) if accumulate else None
    y = moe.moe_expert_ffn_grouped(xd, dev(ids), dev(w), pool, eb, wl.dtype, wl.I, wl.E, slot_of=slot_of,
                                   shared_w=None if sh is None else dev(sh), y_out=y, accumulate=accumulate)
    moe.moe_sync_check()
    ref = oracle.moe_ffn(x, ids, w.astype(np.float64), ex, wl.H, wl.I, wl.dtype, sh)
    got = y.cpu().numpy() - (base if accumulate else 0)
    err = normwise(got, ref)
    assert err <= TOL[wl.dtype], err
    return err


@pytest.mark.parametrize("cfg,T", [(1, 1), (2, 1), (3, 1), (3, 4), (3, 16), (5, 1), (5, 4)])
def test_ffn_parity_configs(cfg, T):
    wl = synth.workload(cfg, T=T, L=1)
    ex, sh = _experts(wl)
    wr = synth.router_weights(wl, 0)
    for step in range(2):
        x = synth.hidden_states(wl, step, T=T)
        ids, w = check_route(x, wr, wl.router_dtype, wl.k)
        check_ffn(wl, x, ids, w, ex, sh)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16, synth.INT4G128])
def test_ffn_grouping_duplicates_slots_and_accumulate(dtype):
    """Tokens sharing experts, a permuted slot table, ragged shapes and the fused residual."""
    H = 2048 if dtype == synth.INT4G128 else 384
    wl = synth.Workload("ragged", H=H, E=24, k=6, I=384, dtype=dtype, router_dtype=synth.F32, shared=True,
                        cfg_id=90 + dtype)
    ex, sh = _experts(wl)
    rng = np.random.default_rng(dtype)
    for T in (2, 7, 16):
        x = rng.standard_normal((T, wl.H)).astype(np.float32)
        ids = np.stack([rng.choice(6, size=6, replace=False) for _ in range(T)]).astype(np.int32)  # heavy overlap
        w = rng.random((T, 6)).astype(np.float32)
        check_ffn(wl, x, ids, w, ex, sh, slot_perm=rng.permutation(wl.E))
        check_ffn(wl, x, ids, w, ex, None, accumulate=True)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16, synth.INT4G128])
def test_ffn_groups_of_many_tokens(dtype):
    """Groups holding more tokens than one LDS chunk of token rows (8 rows at H 2048): full and ragged last
    chunks, and a shared expert that every token uses."""
    wl = synth.Workload("many tokens", H=2048, E=12, k=4, I=256, dtype=dtype, router_dtype=synth.F32, shared=True,
                        cfg_id=120 + dtype)
    ex, sh = _experts(wl)
    rng = np.random.default_rng(120 + dtype)
    for T in (9, 13, 16):  # (at most 16 tokens per call)
        x = rng.standard_normal((T, wl.H)).astype(np.float32)
        ids = np.stack([rng.choice(5, size=4, replace=False) for _ in range(T)]).astype(np.int32)
        w = rng.random((T, 4)).astype(np.float32)
        check_ffn(wl, x, ids, w, ex, sh, slot_perm=rng.permutation(wl.E))


@pytest.mark.parametrize("dtype,H", [(synth.F32, 384), (synth.BF16, 256), (synth.BF16, 640), (synth.BF16, 3968),
                                     (synth.BF16, 4096), (synth.INT4G128, 256), (synth.INT4G128, 2176),
                                     (synth.INT4G128, 4224)])
def test_ffn_one_token_partial_chunks(dtype, H):
    """One-token decode at widths where the last 64-lane chunk of a row is only partly filled."""
    wl = synth.Workload("one-token widths", H=H, E=12, k=3, I=256, dtype=dtype, router_dtype=synth.F32, shared=True,
                        cfg_id=200 + H + dtype)
    ex, sh = _experts(wl)
    rng = np.random.default_rng(H + dtype)
    for _ in range(2):
        x = rng.standard_normal((1, wl.H)).astype(np.float32)
        ids = rng.choice(wl.E, size=(1, wl.k), replace=False).astype(np.int32)
        w = rng.random((1, wl.k)).astype(np.float32)
        check_ffn(wl, x, ids, w, ex, sh, slot_perm=rng.permutation(wl.E))
        check_ffn(wl, x, ids, w, ex, None, accumulate=True)


@pytest.mark.parametrize("scale", [2.0 ** -40, 1.0, 2.0 ** 40])
def test_ffn_int4_one_token_activation_range(scale):
    """The one-token int4 kernels hold x and the SwiGLU activations as fp16 scaled by a power of two per 32-element
    chunk: tiny and huge rows, and a row whose chunks span 2^-30 .. 2^30, keep fp16's relative precision
    (normwise error ~1e-4 against the fp64 oracle; bound 1e-3, well inside the int4 tolerance)."""
    wl = synth.Workload("int4 range", H=2048, E=16, k=4, I=512, dtype=synth.INT4G128, router_dtype=synth.F32,
                        shared=True, cfg_id=261)
    ex, sh = _experts(wl)
    rng = np.random.default_rng(261)
    ids = rng.choice(wl.E, size=(1, wl.k), replace=False).astype(np.int32)
    w = rng.random((1, wl.k)).astype(np.float32)
    x = rng.standard_normal((1, wl.H)) * scale
    rows = [x]
    if scale == 1.0:
        rows.append(x * 2.0 ** rng.integers(-30, 31, size=wl.H // 32).repeat(32))
    for xx in rows:
        assert check_ffn(wl, xx.astype(np.float32), ids, w, ex, sh) <= 1e-3


def test_ffn_invalid_ids_raise_and_contribute_nothing():
    wl = synth.Workload("bad-ids", H=256, E=8, k=2, I=128, dtype=synth.BF16, cfg_id=95)
    ex, _ = _experts(wl)
    x = np.random.default_rng(1).standard_normal((2, 256)).astype(np.float32)
    w = np.array([[0.6, 0.4], [0.5, 0.5]], np.float32)
    for T1 in (1, 2):
        ids = np.array([[3, 9], [1, 2]], np.int32)[:T1]
        y = moe.moe_expert_ffn_grouped(dev(x[:T1]), dev(ids), dev(w[:T1]), dev(ex.reshape(-1)), wl.expert_bytes,
                                       wl.dtype, wl.I, wl.E)
        with pytest.raises(moe.MoeError) as ei:
            moe.moe_sync_check()
        assert ei.value.code == -2
        ref = oracle.moe_ffn(x[:1], np.array([[3]]), np.array([[0.6]]), ex, wl.H, wl.I, wl.dtype)
        assert normwise(y.cpu().numpy()[:1], ref) <= 1e-2
    slot_of = dev(np.array([0, 1, 2, -1, 4, 5, 6, 7], np.int32))
    moe.moe_expert_ffn_grouped(dev(x[:1]), dev(np.array([[3, 1]], np.int32)), dev(w[:1]), dev(ex.reshape(-1)),
                               wl.expert_bytes, wl.dtype, wl.I, wl.E, slot_of=slot_of)
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_sync_check()
    assert ei.value.code == -8


def test_combine_parity():
    rng = np.random.default_rng(3)
    T, k, H = 5, 8, 2048
    yp = rng.standard_normal((T, k, H)).astype(np.float32)
    w = rng.random((T, k)).astype(np.float32)
    ys = rng.standard_normal((T, H)).astype(np.float32)
    y = moe.moe_combine(dev(yp), dev(w), dev(ys))
    ref = np.einsum("tk,tkh->th", w.astype(np.float64), yp.astype(np.float64)) + ys
    assert normwise(y.cpu().numpy(), ref) <= 1e-6
    base = dev(ys)
    moe.moe_combine(dev(yp), dev(w), None, y_out=base, accumulate=True)
    assert normwise(base.cpu().numpy(), ref) <= 1e-6


# ------------------------------------------------------- budgeted stack ---
def _pinned_store(wl, layers_alias=False):
    L_store = 1 if layers_alias else wl.L
    buf = moe.PinnedBuffer(L_store * wl.E * wl.expert_bytes)
    st = buf.array.reshape(L_store, wl.E * wl.expert_bytes)
    for l in range(L_store):
        synth.layer_experts(wl, l, st[l])
    return buf


class _Layers:
    """Host copies of a workload's per-layer weights for the oracle chains (built on first use)."""

    def __init__(self, wl, layers_alias=False):
        self.wl, self.alias, self._ex, self._sh, self._rt = wl, layers_alias, {}, {}, {}

    def experts(self, l):
        src = 0 if self.alias else l
        if src not in self._ex:
            self._ex[src] = synth.layer_experts(self.wl, src)
        return self._ex[src]

    def shared(self, l):
        if not self.wl.shared:
            return None
        if l not in self._sh:
            self._sh[l] = synth.expert_blob(self.wl, l, None)
        return self._sh[l]

    def router(self, l):
        if l not in self._rt:
            self._rt[l] = synth.router_weights(self.wl, l)
        return self._rt[l]


# The one-token int4 FFN takes its activations in fp16 (each rounded by at most 2^-11 relative, a normwise
# error of about 1e-4 in each layer's increment), so after layer 0 the oracle's chain state and the GPU's drift
# apart by that much and later layers' logits are compared within 1e-3; the other decode paths keep fp32
# activations (1e-5).  A layer routed with another layer's router is off by O(1).
DECODE_LOGIT_TOL = {synth.F32: 1e-5, synth.BF16: 1e-5, synth.INT4G128: 1e-3}


def oracle_routed_chain(wl, x0, g_logits, g_ids, g_w, layers, bias=None, logit_tol=None, attention=None,
                        logit_tol0=1e-5):
    """The fp64 oracle chain x <- x + MoE_l(rmsnorm(x)), l = 0..L-1, routed by the oracle itself.

    At each layer the oracle recomputes the router logits from its own chain state; the GPU's logits (bias
    taken off) must match them normwise per token (`logit_tol0` at layer 0, `logit_tol` later, where the chain
    states may have drifted apart by the kernels' own rounding).  The oracle's top-k of the GPU's fp32 logits must
    give the GPU's ids bit for bit and its weights within 1e-5 (the decision is taken on the same fp32 values),
    and the chain continues with the oracle's ids and weights.  A stack that routed a layer with the wrong
    router, an input that was not normalised, or the wrong experts fails here.  attention(l, x) -> x, when
    given, is each layer's attention block before its MoE block."""
    if logit_tol is None:
        logit_tol = DECODE_LOGIT_TOL[wl.dtype]
    xr = np.atleast_2d(x0).astype(np.float64)
    for l in range(wl.L):
        if attention is not None:
            xr = np.atleast_2d(attention(l, xr))
        hr = oracle.rmsnorm(xr.astype(np.float32)).astype(np.float32)
        zr = oracle.router_logits(hr, layers.router(l), wl.router_dtype)
        gz = np.atleast_2d(g_logits[l]).astype(np.float64) - (0.0 if bias is None else np.atleast_2d(bias[l]))
        err = normwise(gz, zr)
        assert err <= (logit_tol0 if l == 0 else logit_tol), f"layer {l}: router logits off by {err:.2e}"
        o_ids, o_w, st = oracle.topk_softmax(np.atleast_2d(g_logits[l]).astype(np.float32), wl.k)
        assert st == oracle.OK
        assert (o_ids == np.atleast_2d(g_ids[l])).all(), f"layer {l}: top-k ids differ from the oracle's"
        gw = np.atleast_2d(g_w[l])
        assert (np.abs(gw - o_w) <= 1e-5 * np.maximum(1.0, np.abs(o_w))).all(), f"layer {l}: top-k weights"
        xr = xr + oracle.moe_ffn(hr, o_ids, o_w, layers.experts(l), wl.H, wl.I, wl.dtype, layers.shared(l))
    return xr


def run_stack_and_check(wl, steps, capacity, layers_alias=False, check_steps=None, T=1, charge_max=None,
                        recall=0, recall_overlap=0, device=False, graph=False, host_layers=0, host_quota=0,
                        host_threads=0, fill_clock=False):
    """Decode `steps` steps through the stack; check events exactly and outputs within tolerance.  With
    charge_max the slots use the rotary policy (else LRU); with recall the stack recalls prior slot sets; with
    host_layers / host_quota a host tier computes its share of the experts on host cores."""
    buf = _pinned_store(wl, layers_alias)
    eb = wl.expert_bytes
    policy = moe.MOE_POLICY_LRU if charge_max is None else moe.MOE_POLICY_ROTARY
    cache = moe.ExpertCache(wl.L, wl.E, eb, capacity * eb + (wl.L * eb if wl.shared else 0), buf.ptr,
                            0 if layers_alias else wl.E * eb, eb, reserved_bytes=wl.L * eb if wl.shared else 0,
                            policy=policy, charge_max=charge_max or 0, device=device, host_layers=host_layers,
                            host_quota=host_quota, fill_clock=fill_clock)
    routers = [dev(synth.router_weights(wl, l)) for l in range(wl.L)]
    shared = [dev(synth.expert_blob(wl, l, None)) for l in range(wl.L)] if wl.shared else None
    stack = moe.MoeStack(cache, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, shared, max_tokens=T,
                         recall=recall, recall_overlap=recall_overlap, host_threads=host_threads)
    rec = oracle.Recall(recall, wl.k, recall_overlap) if recall else None
    sets = synth.routing_sets(wl, steps=steps, T=T)
    o = oracle.LRU(capacity, wl.L, wl.E) if charge_max is None else oracle.Rotary(capacity, wl.L, wl.E, charge_max)
    if host_layers or host_quota:
        o = oracle.HostTier(o, host_layers, host_quota)
    check_steps = set(range(steps) if check_steps is None else check_steps)
    layers = _Layers(wl, layers_alias)
    if graph:  # a replayed graph reads and writes the same buffers every step
        x_buf = torch.empty((T, wl.H), dtype=torch.float32, device=DEV)
        b_buf = torch.empty((wl.L, T, wl.E), dtype=torch.float32, device=DEV)
        ids_buf = torch.empty((wl.L, T, wl.k), dtype=torch.int32, device=DEV)
        w_buf = torch.empty((wl.L, T, wl.k), dtype=torch.float32, device=DEV)
        z_buf = torch.empty((wl.L, T, wl.E), dtype=torch.float32, device=DEV)
    for t in range(steps):
        x0 = synth.hidden_states(wl, t, T=T)
        bias = np.stack([synth.mask_logits(wl, sets[t, l]) for l in range(wl.L)])
        if graph:
            x, ids, w, z = x_buf, ids_buf, w_buf, z_buf
            x.copy_(dev(x0))
            b_buf.copy_(dev(bias))
            stack.decode_graph(t, x, b_buf, ids, w, z)
        else:
            x = dev(x0)
            ids = torch.empty((wl.L, T, wl.k), dtype=torch.int32, device=DEV)
            w = torch.empty((wl.L, T, wl.k), dtype=torch.float32, device=DEV)
            z = torch.empty((wl.L, T, wl.E), dtype=torch.float32, device=DEV)
            stack.decode_step(t, x, dev(bias), ids, w, z)
        moe.moe_sync_check()
        g_ids, g_w, g_z = ids.cpu().numpy(), w.cpu().numpy(), z.cpu().numpy()
        calls = dict(rec.step(t, [g_ids[l].reshape(-1) for l in range(wl.L)])[1]) if rec else {}
        for l in range(wl.L):
            assert (np.sort(g_ids[l], axis=1) == sets[t, l]).all()
            assert o.lookup(t, l, g_ids[l].reshape(-1)) == oracle.OK
            if l + 1 in calls:
                assert o.lookup(t, l + 1, calls[l + 1], prefetch=True) == oracle.OK
        if t in check_steps:
            # the fp64 oracle chain from the same input, routed by the oracle itself
            xr = oracle_routed_chain(wl, x0, g_z, g_ids, g_w, layers, bias=bias)
            assert normwise(x.cpu().numpy() - x0, xr - x0) <= TOL[wl.dtype]
    n_ev = len(cache.trace())
    for which in range(4):  # re-launch timing leaves the residency state alone
        assert stack.kernel_time(which, 5) > 0
    moe.moe_sync_check()
    assert len(cache.trace()) == n_ev
    ev = cache.trace()
    oev = o.events()
    assert len(ev) == len(oev)
    assert (ev.view(np.int32).reshape(-1, 6) == oev.view(np.int32).reshape(-1, 6)).all()
    s = cache.stats()
    assert s["occupancy"] <= capacity and s["misses"] == o.stats()["misses"]
    if capacity * eb <= 64 << 20:  # every resident expert's slot holds its whole blob, byte for byte
        torch.cuda.synchronize()  # (the cache's copy stream too: prefetches fill there)
        table_p, pool_p = cache.slot_table()
        table = _d2h(table_p, 4 * wl.L * wl.E).view(np.int32)
        pool = _d2h(pool_p, capacity * eb).reshape(capacity, eb)
        store = buf.array.reshape(-1, eb)
        for l in range(wl.L):
            for e in range(wl.E):
                sl = o.slot_of(l, e)
                assert table[l * wl.E + e] == sl
                if sl >= 0:
                    assert np.array_equal(pool[sl], store[e if layers_alias else l * wl.E + e]), (l, e)
    stack.close()
    cache.close()
    buf.close()
    return s


@pytest.mark.parametrize("device,charge_max,graph", [(False, None, False), (True, None, False), (True, 3, False),
                                                    (True, None, True), (True, 2, True)])
def test_budgeted_stack_small_evicting(device, charge_max, graph):
    """With device=True every lookup is a kernel (no host round trip); with graph=True each step is a replay
    of one captured graph.  The decisions are the same, and every replay is checked."""
    wl = synth.Workload("small stack", H=512, E=32, k=4, I=256, L=4, dtype=synth.BF16, routing="zipf_overlap",
                        cfg_id=97)
    s = run_stack_and_check(wl, steps=40, capacity=24, device=device, charge_max=charge_max, graph=graph)
    assert s["evictions"] > 0


def test_decode_graph_replays_equal_eager_steps():
    """Twin stacks on twin device caches: graph replays against eager steps, bit for bit, with eager work and
    synchronisations between the replays."""
    wl = synth.Workload("graph stack", H=2048, E=64, k=8, I=256, L=3, dtype=synth.INT4G128, shared=True,
                        routing="zipf_overlap", cfg_id=95)
    eb, cap = wl.expert_bytes, 30
    buf = _pinned_store(wl)
    routers = [dev(synth.router_weights(wl, l)) for l in range(wl.L)]
    shared = [dev(synth.expert_blob(wl, l, None)) for l in range(wl.L)]
    caches = [moe.ExpertCache(wl.L, wl.E, eb, (cap + wl.L) * eb, buf.ptr, wl.E * eb, eb, reserved_bytes=wl.L * eb,
                              device=True) for _ in range(2)]
    stacks = [moe.MoeStack(c, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, shared) for c in caches]
    sets = synth.routing_sets(wl, steps=12)
    x_buf = torch.empty((1, wl.H), dtype=torch.float32, device=DEV)
    b_buf = torch.empty((wl.L, 1, wl.E), dtype=torch.float32, device=DEV)
    ids_buf = torch.empty((wl.L, 1, wl.k), dtype=torch.int32, device=DEV)
    w_buf = torch.empty((wl.L, 1, wl.k), dtype=torch.float32, device=DEV)
    for t in range(12):
        x0 = dev(synth.hidden_states(wl, t))
        bias = dev(np.stack([synth.mask_logits(wl, sets[t, l]) for l in range(wl.L)]))
        xe = x0.clone()
        ids_e = torch.empty_like(ids_buf)
        w_e = torch.empty_like(w_buf)
        stacks[0].decode_step(t, xe, bias, ids_e, w_e)
        torch.cuda.synchronize()
        x_buf.copy_(x0)
        b_buf.copy_(bias)
        stacks[1].decode_graph(t, x_buf, b_buf, ids_buf, w_buf)
        moe.moe_sync_check()
        assert torch.equal(x_buf, xe) and torch.equal(ids_buf, ids_e) and torch.equal(w_buf, w_e), t
    ev0, ev1 = caches[0].trace(), caches[1].trace()
    assert len(ev0) == len(ev1) > 0 and (ev0.view(np.int32) == ev1.view(np.int32)).all()
    for which in range(4):
        assert stacks[1].kernel_time(which, 3) > 0
    moe.moe_sync_check()
    for s_, c in zip(stacks, caches):
        s_.close()
        c.close()
    buf.close()


@pytest.mark.parametrize("charge_max", [0, 3])
def test_budgeted_stack_rotary_slots(charge_max):
    """The stack over a rotary slot group: residency decisions event for event against the oracle's ring."""
    wl = synth.Workload("small stack", H=512, E=32, k=4, I=256, L=4, dtype=synth.BF16, routing="zipf_overlap",
                        cfg_id=97)
    s = run_stack_and_check(wl, steps=40, capacity=24, charge_max=charge_max)
    assert s["evictions"] > 0


@pytest.mark.parametrize("charge_max,overlap", [(None, 3), (2, 0)])
def test_budgeted_stack_recall_on_recurring_contexts(charge_max, overlap):
    """Reverse rotation: a token whose layer-0 set matches a remembered token's prefetches that token's
    later-layer sets; the log (lookups and prefetches) event for event against the oracle's replay."""
    wl = synth.Workload("topic stack", H=512, E=32, k=4, I=256, L=4, dtype=synth.BF16, routing="topics", topics=3,
                        cfg_id=96)
    s = run_stack_and_check(wl, steps=40, capacity=20, charge_max=charge_max, recall=4, recall_overlap=overlap)
    assert s["prefetches"] > 0 and s["evictions"] > 0


def test_budgeted_stack_tokens_and_shared_int4():
    wl = synth.Workload("int4 stack", H=2048, E=64, k=8, I=256, L=3, dtype=synth.INT4G128, shared=True,
                        routing="zipf_overlap", cfg_id=98)
    s = run_stack_and_check(wl, steps=12, capacity=40, T=4, check_steps=[0, 5, 11])
    assert s["evictions"] > 0


@pytest.mark.parametrize("graph", [False, True])
def test_budgeted_stack_int4_shared_device_one_token(graph):
    """One-token int4 steps with a shared expert under device residency: the gate/up launch streams each
    step's missing experts itself (rows, group scales and the down parts); outputs, decisions and every
    resident slot's bytes against the oracle and the host store."""
    wl = synth.Workload("int4 stack", H=2048, E=64, k=8, I=256, L=3, dtype=synth.INT4G128, shared=True,
                        routing="zipf_overlap", cfg_id=92)
    s = run_stack_and_check(wl, steps=16, capacity=30, device=True, graph=graph)
    assert s["evictions"] > 0


@pytest.mark.parametrize("graph", [False, True])
def test_fill_clock_times_the_fills_and_changes_nothing(graph):
    """MOE_CACHE_FILL_CLOCK: the demand fills of one-token device steps are timed (fill_ns > 0, stall_ns within
    it); decisions and outputs still match the oracle; without the flag both stay 0."""
    wl = synth.Workload("clock stack", H=512, E=32, k=4, I=256, L=4, dtype=synth.BF16, routing="zipf_overlap",
                        cfg_id=97)
    s = run_stack_and_check(wl, steps=16, capacity=24, device=True, graph=graph, fill_clock=True)
    assert s["misses"] > 0 and s["fill_ns"] > 0 and 0 <= s["stall_ns"] <= s["fill_ns"]
    s0 = run_stack_and_check(wl, steps=4, capacity=24, device=True)
    assert s0["fill_ns"] == 0 and s0["stall_ns"] == 0


@pytest.mark.parametrize("dtype,shared,N,Q,threads", [(synth.BF16, False, 1, 1, 0), (synth.BF16, False, 0, 2, 3),
                                                      (synth.INT4G128, True, 1, 2, 0)])
def test_budgeted_stack_host_tier(dtype, shared, N, Q, threads):
    """A host tier beside the slot table: layers below N, and up to Q non-resident experts per lookup elsewhere,
    are computed on host cores from the pinned store while the GPU runs the fills and the resident experts.
    Decisions event for event against the oracle's model of the rule, outputs against the oracle chain (routed
    by the oracle), and every resident slot byte for byte against the store."""
    H = 2048 if dtype == synth.INT4G128 else 512
    wl = synth.Workload("host tier stack", H=H, E=32, k=4, I=256, L=4, dtype=dtype, shared=shared,
                        routing="zipf_overlap", cfg_id=160 + dtype)
    s = run_stack_and_check(wl, steps=24, capacity=16, host_layers=N, host_quota=Q, host_threads=threads)
    assert s["host_computed"] > 0 and s["misses"] > 0 and s["evictions"] > 0


def test_host_tier_stack_rejects_what_it_cannot_run():
    wl = synth.Workload("host tier stack", H=512, E=16, k=2, I=128, L=2, dtype=synth.BF16, cfg_id=170)
    buf = _pinned_store(wl)
    eb = wl.expert_bytes
    routers = [dev(synth.router_weights(wl, l)) for l in range(wl.L)]
    cache = moe.ExpertCache(wl.L, wl.E, eb, 8 * eb, buf.ptr, wl.E * eb, eb, host_quota=1)
    for kw in (dict(max_tokens=2), dict(max_prefill_tokens=16), dict(prefetch=1)):
        with pytest.raises(moe.MoeError):
            moe.MoeStack(cache, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, None, **kw)
    cache.close()
    with pytest.raises(moe.MoeError):  # a host tier decides on the host
        moe.ExpertCache(wl.L, wl.E, eb, 8 * eb, buf.ptr, wl.E * eb, eb, host_quota=1, device=True)
    buf.close()


def test_preloaded_stack_kernel_time_repeats():
    """Timing re-launches on a preloaded stack (every expert resident): a two-layer graph repeats its launches,
    the repeats read rotated expert sets (or, with the flag, the step's own), and the stack's state is left alone,
    so the next step equals a twin stack's bit for bit.  Timing a route launch with the flag is rejected."""
    wl = synth.Workload("preloaded timing", H=512, E=16, k=2, I=128, L=2, dtype=synth.BF16, shared=True,
                        routing="zipf_overlap", cfg_id=171)
    eb = wl.expert_bytes
    buf = _pinned_store(wl)
    routers = [dev(synth.router_weights(wl, l)) for l in range(wl.L)]
    shared = [dev(synth.expert_blob(wl, l, None)) for l in range(wl.L)]
    caches = [moe.ExpertCache(wl.L, wl.E, eb, (wl.L * wl.E + wl.L) * eb, buf.ptr, wl.E * eb, eb,
                              reserved_bytes=wl.L * eb, preload=True) for _ in range(2)]
    stacks = [moe.MoeStack(c, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, shared) for c in caches]
    sets = synth.routing_sets(wl, steps=2)
    for t in range(2):
        x0 = dev(synth.hidden_states(wl, t))
        bias = dev(np.stack([synth.mask_logits(wl, sets[t, l]) for l in range(wl.L)]))
        outs = []
        for st in stacks:
            x = x0.clone()
            ids = torch.empty((wl.L, 1, wl.k), dtype=torch.int32, device=DEV)
            st.decode_step(t, x, bias, ids)
            outs.append((x, ids))
        moe.moe_sync_check()
        assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1]), t
        if t == 0:
            for which in (0, 1, 2, 3, 9, 10, 11):
                assert stacks[1].kernel_time(which, 2) > 0, which
            with pytest.raises(moe.MoeError):
                stacks[1].kernel_time(8, 1)
            moe.moe_sync_check()
    assert caches[1].stats()["misses"] == caches[0].stats()["misses"] == 0
    for s_, c in zip(stacks, caches):
        s_.close()
        c.close()
    buf.close()


@pytest.mark.parametrize("device", [False, True])
def test_budgeted_stack_full_size_config4_sampled(device):
    """The benchmark's configuration (40 layers, 6 GiB budget -> 682 slots), layers aliasing one host copy."""
    wl = synth.workload(4)
    s = run_stack_and_check(wl, steps=6, capacity=wl.capacity(), layers_alias=True, check_steps=[0, 5], device=device)
    assert s["capacity"] == 682 and s["misses"] > 0


def _d2h(ptr, nbytes):
    """Copy device memory the library owns (a raw pointer) to the host."""
    import ctypes as C
    hip = C.CDLL("libamdhip64.so")
    hip.hipMemcpy.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int]
    hip.hipMemcpy.restype = C.c_int
    out = np.empty(nbytes, np.uint8)
    assert hip.hipMemcpy(out.ctypes.data, ptr, nbytes, 2) == 0  # device to host
    return out


@pytest.mark.parametrize("rotary,Q,C,L,E,nmax,steps", [(False, 0, 24, 3, 32, 8, 300), (True, 3, 24, 3, 32, 8, 300),
                                                       (False, 0, 700, 40, 128, 40, 400),
                                                       (True, 32, 700, 40, 128, 40, 400),
                                                       (False, 0, 4096, 48, 256, 600, 120),
                                                       (True, 0, 4096, 48, 256, 600, 120)])
def test_device_lookups_match_oracle(rotary, Q, C, L, E, nmax, steps):
    """Lookups made by the device kernel: decisions, counters, slot table and slot contents against the
    oracle, for steps of up to nmax ids with repeats (prefill-sized at the largest capacity)."""
    eb = 256
    buf = moe.PinnedBuffer(L * E * eb)
    buf.array.view(np.int32).reshape(L * E, eb // 4)[:] = np.arange(L * E, dtype=np.int32)[:, None]
    cache = moe.ExpertCache(L, E, eb, C * eb, buf.ptr, E * eb, eb, device=True,
                            policy=moe.MOE_POLICY_ROTARY if rotary else moe.MOE_POLICY_LRU, charge_max=Q)
    o = oracle.Rotary(C, L, E, Q) if rotary else oracle.LRU(C, L, E)
    rng = np.random.default_rng(C + 7 * Q + int(rotary))
    ids = [rng.integers(0, E, size=int(rng.integers(1, nmax + 1))).astype(np.int32) for _ in range(steps)]
    layers = rng.integers(0, L, size=steps)
    ids_d = [dev(a) for a in ids]
    slots_d = [torch.empty(a.size, dtype=torch.int32, device=DEV) for a in ids]
    want_slots = []
    torch.cuda.synchronize()
    for t in range(steps):
        cache.lookup_device(t, int(layers[t]), ids_d[t], slots_d[t])
        assert o.lookup(t, int(layers[t]), ids[t]) == oracle.OK
        want_slots.append([o.slot_of(int(layers[t]), int(e)) for e in ids[t]])
    moe.moe_sync_check()
    assert all(slots_d[t].cpu().tolist() == want_slots[t] for t in range(steps))
    ev, oev = cache.trace(), o.events()
    assert len(ev) == len(oev)
    assert (ev.view(np.int32).reshape(-1, 6) == oev.view(np.int32).reshape(-1, 6)).all()
    st, so = cache.stats(), o.stats()
    assert (st["hits"], st["misses"], st["evictions"]) == (so["hits"], so["misses"], so["evictions"])
    assert st["occupancy"] == o.occupancy() and st["h2d_bytes"] == st["misses"] * eb
    table_p, pool_p = cache.slot_table()
    table = _d2h(table_p, 4 * L * E).view(np.int32)
    pool = _d2h(pool_p, C * eb).view(np.int32).reshape(C, eb // 4)
    for l in range(L):
        for e in range(E):
            s = o.slot_of(l, e)
            assert table[l * E + e] == s
            if s >= 0:
                assert (pool[s] == l * E + e).all()
    cache.close()
    buf.close()


@pytest.mark.parametrize("rotary,Q,C,L,E,nmax,steps", [(False, 0, 24, 3, 32, 8, 300), (True, 3, 24, 3, 32, 8, 300),
                                                       (False, 0, 700, 40, 128, 40, 300),
                                                       (True, 32, 700, 40, 128, 40, 300),
                                                       (False, 0, 4096, 48, 256, 600, 80)])
def test_device_prefetches_and_lookups_match_oracle(rotary, Q, C, L, E, nmax, steps):
    """Device prefetches (decisions on the stream, fills on the copy stream) interleaved with device lookups:
    every decision, the counters, the slot table and every slot's contents against the oracle replaying the
    same calls, prefetches included."""
    eb = 256
    buf = moe.PinnedBuffer(L * E * eb)
    buf.array.view(np.int32).reshape(L * E, eb // 4)[:] = np.arange(L * E, dtype=np.int32)[:, None]
    cache = moe.ExpertCache(L, E, eb, C * eb, buf.ptr, E * eb, eb, device=True,
                            policy=moe.MOE_POLICY_ROTARY if rotary else moe.MOE_POLICY_LRU, charge_max=Q)
    o = oracle.Rotary(C, L, E, Q) if rotary else oracle.LRU(C, L, E)
    rng = np.random.default_rng(11 * C + Q + int(rotary))
    ids = [rng.integers(0, E, size=int(rng.integers(1, nmax + 1))).astype(np.int32) for _ in range(steps)]
    layers = rng.integers(0, L, size=steps)
    pf = rng.random(steps) < 0.4
    ids_d = [dev(a) for a in ids]
    slots_d = [torch.empty(a.size, dtype=torch.int32, device=DEV) for a in ids]
    want_slots = {}
    torch.cuda.synchronize()
    for t in range(steps):
        if pf[t]:
            cache.prefetch_device(t, int(layers[t]), ids_d[t])
        else:
            cache.lookup_device(t, int(layers[t]), ids_d[t], slots_d[t])
        assert o.lookup(t, int(layers[t]), ids[t], prefetch=bool(pf[t])) == oracle.OK
        if not pf[t]:
            want_slots[t] = [o.slot_of(int(layers[t]), int(e)) for e in ids[t]]
    torch.cuda.synchronize()
    moe.moe_sync_check()
    assert all(slots_d[t].cpu().tolist() == w for t, w in want_slots.items())
    ev, oev = cache.trace(), o.events()
    assert len(ev) == len(oev)
    assert (ev.view(np.int32).reshape(-1, 6) == oev.view(np.int32).reshape(-1, 6)).all()
    st, so = cache.stats(), o.stats()
    assert st["prefetches"] > 0
    assert ((st["hits"], st["misses"], st["prefetches"], st["evictions"])
            == (so["hits"], so["misses"], so["prefetches"], so["evictions"]))
    assert st["occupancy"] == o.occupancy() and st["h2d_bytes"] == (st["misses"] + st["prefetches"]) * eb
    table_p, pool_p = cache.slot_table()
    table = _d2h(table_p, 4 * L * E).view(np.int32)
    pool = _d2h(pool_p, C * eb).view(np.int32).reshape(C, eb // 4)
    for l in range(L):
        for e in range(E):
            s = o.slot_of(l, e)
            assert table[l * E + e] == s
            if s >= 0:
                assert (pool[s] == l * E + e).all()
    cache.close()
    buf.close()


@pytest.mark.parametrize("case", ["all_free", "free_then_victims", "eight_victims", "nine_victims", "m64", "m65"])
def test_device_lookup_one_pass_boundaries(case):
    """The device LRU's one-pass placement (at most 64 experts and 8 victims in a step) and the lane walk beyond
    it, at their boundaries, against the oracle event for event: misses into free slots only; free slots then
    victims in one step; exactly 8 and 9 victims; 64 and 65 experts in one step."""
    L, E, eb = 2, 160, 256
    C = {"all_free": 40, "free_then_victims": 10, "eight_victims": 16, "nine_victims": 16, "m64": 100,
         "m65": 100}[case]
    steps = {"all_free": [list(range(8)), list(range(8, 20))],
             "free_then_victims": [list(range(8)), list(range(20, 26))],        # 2 free + 4 victims
             "eight_victims": [list(range(16)), list(range(30, 38))],           # 8 victims
             "nine_victims": [list(range(16)), list(range(30, 39))],            # 9 victims: the lane walk
             "m64": [list(range(64)), list(range(30, 94)), list(range(100, 110))],
             "m65": [list(range(65)), list(range(30, 95)), list(range(100, 110))]}[case]
    buf = moe.PinnedBuffer(L * E * eb)
    buf.array.view(np.int32).reshape(L * E, eb // 4)[:] = np.arange(L * E, dtype=np.int32)[:, None]
    cache = moe.ExpertCache(L, E, eb, C * eb, buf.ptr, E * eb, eb, device=True)
    o = oracle.LRU(C, L, E)
    rng = np.random.default_rng(len(case))
    for t, ids in enumerate(steps):
        ids = np.array(rng.permutation(ids), np.int32)  # any order: decisions follow ascending ids
        slots = torch.empty(ids.size, dtype=torch.int32, device=DEV)
        cache.lookup_device(t, 1, dev(ids), slots)
        assert o.lookup(t, 1, ids) == oracle.OK
        moe.moe_sync_check()
        assert slots.cpu().tolist() == [o.slot_of(1, int(e)) for e in ids]
    ev, oev = cache.trace(), o.events()
    assert len(ev) == len(oev) and (ev.view(np.int32).reshape(-1, 6) == oev.view(np.int32).reshape(-1, 6)).all()
    st, so = cache.stats(), o.stats()
    assert (st["hits"], st["misses"], st["evictions"]) == (so["hits"], so["misses"], so["evictions"])
    pool = _d2h(cache.slot_table()[1], C * eb).view(np.int32).reshape(C, eb // 4)
    for e in range(E):
        s_ = o.slot_of(1, e)
        if s_ >= 0:
            assert (pool[s_] == E + e).all()
    cache.close()
    buf.close()


def test_device_lookup_errors_change_nothing():
    L, E, C, eb = 2, 16, 4, 256
    buf = moe.PinnedBuffer(L * E * eb)
    cache = moe.ExpertCache(L, E, eb, C * eb, buf.ptr, E * eb, eb, device=True)
    cache.lookup_device(0, 0, dev(np.array([1, 2, 2], np.int32)))
    moe.moe_sync_check()
    slots = dev(np.full(5, 7, np.int32))
    cache.lookup_device(1, 1, dev(np.array([3, 16], np.int32)), slots_out=slots[:2])
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_sync_check()
    assert ei.value.code == -2
    assert (slots.cpu().numpy()[:2] == -1).all() and slots.cpu().numpy()[2] == 7  # no rank placed
    cache.lookup_device(2, 1, dev(np.arange(5, dtype=np.int32)), slots_out=slots)
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_sync_check()
    assert ei.value.code == -4
    assert (slots.cpu().numpy() == -1).all()
    ev = cache.trace()
    assert len(ev) == 2 and cache.stats()["misses"] == 2
    with pytest.raises(moe.MoeError):
        cache.lookup(3, 0, np.array([1], np.int32))
    with pytest.raises(moe.MoeError):
        cache.prefetch(3, 0, np.array([1], np.int32))
    with pytest.raises(moe.MoeError):
        cache.lookup_device(3, 2, dev(np.array([1], np.int32)))
    with pytest.raises(moe.MoeError):
        cache.prefetch_device(3, 2, dev(np.array([1], np.int32)))
    cache.prefetch_device(3, 0, dev(np.array([-1], np.int32)))
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_sync_check()
    assert ei.value.code == -2
    cache.prefetch_device(4, 0, dev(np.arange(5, dtype=np.int32)))
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_sync_check()
    assert ei.value.code == -4
    st = cache.stats()
    assert len(cache.trace()) == 2 and st["misses"] == 2 and st["prefetches"] == 0
    cache.close()
    with pytest.raises(moe.MoeError):
        moe.ExpertCache(L, E, eb, 5000 * eb, buf.ptr, E * eb, eb, device=True)
    buf.close()


def test_full_size_config2_every_output():
    wl = synth.workload(2)
    ex, _ = _experts(wl)
    wr = synth.router_weights(wl, 0)
    pool = dev(ex.reshape(-1))
    for step in range(4):
        x = synth.hidden_states(wl, step)
        ids, w = check_route(x, wr, wl.router_dtype, wl.k)
        y = moe.moe_expert_ffn_grouped(dev(x), dev(ids), dev(w), pool, wl.expert_bytes, wl.dtype, wl.I, wl.E)
        moe.moe_sync_check()
        ref = oracle.moe_ffn(x, ids, w.astype(np.float64), ex, wl.H, wl.I, wl.dtype)
        assert normwise(y.cpu().numpy(), ref) <= TOL[wl.dtype]


def test_cache_rejects_pageable_host_memory():
    host = np.zeros(4 * 256, np.uint8)
    with pytest.raises(moe.MoeError) as ei:
        moe.ExpertCache(1, 4, 256, 2 * 256, host.ctypes.data, 0, 256)
    assert ei.value.code == -5


# --------------------------------------------------------------- prefill ---
# The grouped MFMA path rounds the token rows and the SwiGLU activations to bf16
# for the matrix cores (int4 weights are dequantised to bf16): per product the
# relative rounding is <= 2**-8, which over H ~ 2e3 random-sign terms stays far
# inside the bf16 / int4 tolerances below.
PREFILL_TOL = {synth.BF16: 1e-2, synth.INT4G128: 3e-2}


def run_prefill(wl, x, ids, w, ex, sh, slot_perm=None):
    E, eb = ex.shape
    if slot_perm is not None:
        pool_np = np.empty_like(ex)
        pool_np[slot_perm] = ex
        slot_of = dev(slot_perm.astype(np.int32))
    else:
        pool_np, slot_of = ex, None
    y = moe.moe_prefill_grouped(dev(x), dev(ids), dev(w), dev(pool_np.reshape(-1)), eb, wl.dtype, wl.I, wl.E,
                                slot_of=slot_of, shared_w=None if sh is None else dev(sh))
    moe.moe_sync_check()
    return y.cpu().numpy()


@pytest.mark.parametrize("dtype", [synth.BF16, synth.INT4G128])
@pytest.mark.parametrize("shared", [False, True])
def test_prefill_parity_small_ragged(dtype, shared):
    H = 2048 if dtype == synth.INT4G128 else 256
    wl = synth.Workload("prefill-small", H=H, E=16, k=4, I=256, dtype=dtype, router_dtype=synth.F32, shared=shared,
                        cfg_id=80 + dtype)
    ex, sh = _experts(wl)
    rng = np.random.default_rng(7 + dtype)
    for T in (1, 37, 130):
        x = rng.standard_normal((T, wl.H)).astype(np.float32)
        z = rng.standard_normal((T, wl.E)).astype(np.float32)
        z[:, 3] += 2.0  # one popular expert: its group spans several 64-row tiles
        ids, w, _ = oracle.topk_softmax(z, wl.k)
        w = w.astype(np.float32)
        y = run_prefill(wl, x, ids, w, ex, sh, slot_perm=rng.permutation(wl.E))
        ref = oracle.moe_ffn(x, ids, w.astype(np.float64), ex, wl.H, wl.I, wl.dtype, sh)
        assert normwise(y, ref) <= PREFILL_TOL[dtype]


def test_prefill_config5_chunk():
    """Config 5's 2048-token chunk (E 256, top-8, int4-g128, shared expert) routed by its router."""
    wl = synth.workload(5, L=1)
    ex, sh = _experts(wl)
    wr = synth.router_weights(wl, 0)
    x = synth.prefill_states(wl)
    _, ids_d, w_d = moe.moe_route_topk(dev(x), dev(wr), wl.router_dtype, wl.k, rmsnorm=False)
    ids, w = ids_d.cpu().numpy(), w_d.cpu().numpy()
    counts = np.bincount(ids.reshape(-1), minlength=wl.E)
    assert counts.max() > 64  # some groups span more than one tile
    y = run_prefill(wl, x, ids, w, ex, sh)
    # every token against the decode kernel (fp32 activations), 16 tokens per call
    pool = dev(ex.reshape(-1))
    ws = torch.empty(moe.moe_ffn_workspace_bytes(16, wl.k, wl.I), dtype=torch.uint8, device=DEV)
    y_dec = np.empty_like(y)
    shd = dev(sh)
    for t0 in range(0, wl.prefill, 16):
        yd = moe.moe_expert_ffn_grouped(dev(x[t0:t0 + 16]), ids_d[t0:t0 + 16].contiguous(),
                                        w_d[t0:t0 + 16].contiguous(), pool, wl.expert_bytes, wl.dtype, wl.I, wl.E,
                                        shared_w=shd, workspace=ws)
        y_dec[t0:t0 + 16] = yd.cpu().numpy()
    moe.moe_sync_check()
    assert normwise(y, y_dec) <= PREFILL_TOL[wl.dtype]
    # sampled tokens against the oracle
    sample = np.random.default_rng(0).choice(wl.prefill, 12, replace=False)
    ref = oracle.moe_ffn(x[sample], ids[sample], w[sample].astype(np.float64), ex, wl.H, wl.I, wl.dtype, sh)
    assert normwise(y[sample], ref) <= PREFILL_TOL[wl.dtype]


def test_prefill_invalid_ids_contribute_nothing():
    wl = synth.Workload("prefill-bad", H=256, E=8, k=2, I=128, dtype=synth.BF16, cfg_id=96)
    ex, _ = _experts(wl)
    x = np.random.default_rng(2).standard_normal((3, 256)).astype(np.float32)
    ids = np.array([[3, 9], [1, 2], [5, -1]], np.int32)
    w = np.full((3, 2), 0.5, np.float32)
    y = moe.moe_prefill_grouped(dev(x), dev(ids), dev(w), dev(ex.reshape(-1)), wl.expert_bytes, wl.dtype, wl.I, wl.E)
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_sync_check()
    assert ei.value.code == -2
    ok_ids = np.array([[3], [1], [5]], np.int32)
    ref = oracle.moe_ffn(x, ok_ids, np.full((3, 1), 0.5), ex, wl.H, wl.I, wl.dtype)
    ref[1] += 0.5 * oracle.expert_forward(x[1], ex[2], wl.H, wl.I, wl.dtype)
    assert normwise(y.cpu().numpy(), ref) <= PREFILL_TOL[wl.dtype]


def test_prefill_rejects_fp32_weights():
    wl = synth.Workload("prefill-f32", H=256, E=4, k=2, I=128, dtype=synth.F32, cfg_id=97)
    ex, _ = _experts(wl)
    x = np.zeros((2, 256), np.float32)
    ids = np.array([[0, 1], [2, 3]], np.int32)
    w = np.full((2, 2), 0.5, np.float32)
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_prefill_grouped(dev(x), dev(ids), dev(w), dev(ex.reshape(-1)), wl.expert_bytes, wl.dtype, wl.I, wl.E)
    assert ei.value.code == -1


# ---------------------------------------------------------- stack prefill ---
# A prompt chunk's expert FFN rounds x and the activations to bf16 for the matrix cores (a normwise error of
# up to PREFILL_TOL in each layer's increment), so after layer 0 the oracle's chain state and the GPU's have
# drifted apart by up to that much of each increment so far, and the logits with them: later layers' logits
# are compared within half that tolerance (layer 0 within 1e-5).  A layer routed with another layer's router
# is off by O(1).
PREFILL_LOGIT_TOL = {synth.BF16: 5e-3, synth.INT4G128: 1.5e-2}


@pytest.mark.parametrize("dtype,shared", [(synth.BF16, False), (synth.INT4G128, True)])
def test_stack_prefill_then_decode_budgeted(dtype, shared):
    """A prompt chunk through a budgeted stack whose layers evict each other (one layer's experts fit, three
    do not), then decode steps on the same cache: the residency log equals the oracle LRU's, and outputs match
    the oracle chain routed by the GPU's ids."""
    H = 2048 if dtype == synth.INT4G128 else 512
    wl = synth.Workload("prefill stack", H=H, E=32, k=4, I=256, L=3, dtype=dtype, shared=shared,
                        routing="zipf_overlap", cfg_id=110 + dtype)
    capacity, T, steps = 40, 96, 3
    buf = _pinned_store(wl)
    eb = wl.expert_bytes
    reserved = wl.L * eb if shared else 0
    cache = moe.ExpertCache(wl.L, wl.E, eb, capacity * eb + reserved, buf.ptr, wl.E * eb, eb, reserved_bytes=reserved)
    routers = [dev(synth.router_weights(wl, l)) for l in range(wl.L)]
    shw = [dev(synth.expert_blob(wl, l, None)) for l in range(wl.L)] if shared else None
    stack = moe.MoeStack(cache, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, shw, max_tokens=1,
                         max_prefill_tokens=T)
    o = oracle.LRU(capacity, wl.L, wl.E)
    layers = _Layers(wl)
    x0 = np.random.default_rng(dtype).standard_normal((T, wl.H)).astype(np.float32)
    x = dev(x0)
    ids = torch.empty((wl.L, T, wl.k), dtype=torch.int32, device=DEV)
    w = torch.empty((wl.L, T, wl.k), dtype=torch.float32, device=DEV)
    z = torch.empty((wl.L, T, wl.E), dtype=torch.float32, device=DEV)
    stack.prefill(0, x, ids, w, z)
    moe.moe_sync_check()
    g_ids, g_w = ids.cpu().numpy(), w.cpu().numpy()
    for l in range(wl.L):
        assert o.lookup(0, l, g_ids[l].reshape(-1)) == oracle.OK
    xr = oracle_routed_chain(wl, x0, z.cpu().numpy(), g_ids, g_w, layers, logit_tol=PREFILL_LOGIT_TOL[wl.dtype])
    assert normwise(x.cpu().numpy() - x0, xr - x0) <= PREFILL_TOL[dtype]
    sets = synth.routing_sets(wl, steps=steps)
    for t in range(steps):
        xd0 = synth.hidden_states(wl, t)
        bias = np.stack([synth.mask_logits(wl, sets[t, l]) for l in range(wl.L)])
        xd = dev(xd0)
        di = torch.empty((wl.L, 1, wl.k), dtype=torch.int32, device=DEV)
        dw = torch.empty((wl.L, 1, wl.k), dtype=torch.float32, device=DEV)
        dz = torch.empty((wl.L, 1, wl.E), dtype=torch.float32, device=DEV)
        stack.decode_step(1 + t, xd, dev(bias), di, dw, dz)
        moe.moe_sync_check()
        for l in range(wl.L):
            assert o.lookup(1 + t, l, di.cpu().numpy()[l].reshape(-1)) == oracle.OK
        xr = oracle_routed_chain(wl, xd0, dz.cpu().numpy(), di.cpu().numpy(), dw.cpu().numpy(), layers, bias=bias)
        assert normwise(xd.cpu().numpy() - xd0, xr - xd0) <= TOL[dtype]
    ev, oev = cache.trace(), o.events()
    assert len(ev) == len(oev)
    assert (ev.view(np.int32).reshape(-1, 6) == oev.view(np.int32).reshape(-1, 6)).all()
    s = cache.stats()
    assert s["evictions"] > 0 and s["occupancy"] <= capacity
    stack.close()
    cache.close()
    buf.close()


@pytest.mark.parametrize("dtype", [synth.BF16, synth.INT4G128])
def test_stack_prefill_pipelined_device_prefetch(dtype):
    """Device LRU residency with room for two layers and a chunk that uses nearly every expert: the stack
    prefetches each layer's experts (fills on the copy stream) while the previous layer's FFN runs.  The
    decision log equals the oracle LRU's for the same sequence (prefetch layer 0; per layer: demand lookup,
    then prefetch of the next layer), outputs match the oracle chain, and decode steps continue on the cache."""
    H = 2048 if dtype == synth.INT4G128 else 512
    wl = synth.Workload("prefill pipe", H=H, E=16, k=4, I=256, L=4, dtype=dtype, shared=True,
                        routing="zipf_overlap", cfg_id=130 + dtype)
    capacity, T = 40, 64  # 2E <= 40 < L E: layers evict each other; T k = 256 >= 8 E
    buf = _pinned_store(wl)
    eb = wl.expert_bytes
    reserved = wl.L * eb
    cache = moe.ExpertCache(wl.L, wl.E, eb, capacity * eb + reserved, buf.ptr, wl.E * eb, eb,
                            reserved_bytes=reserved, device=True)
    routers = [dev(synth.router_weights(wl, l)) for l in range(wl.L)]
    shw = [dev(synth.expert_blob(wl, l, None)) for l in range(wl.L)]
    stack = moe.MoeStack(cache, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, shw, max_tokens=1,
                         max_prefill_tokens=T)
    x0 = np.random.default_rng(dtype + 3).standard_normal((T, wl.H)).astype(np.float32)
    x = dev(x0)
    ids = torch.empty((wl.L, T, wl.k), dtype=torch.int32, device=DEV)
    w = torch.empty((wl.L, T, wl.k), dtype=torch.float32, device=DEV)
    z = torch.empty((wl.L, T, wl.E), dtype=torch.float32, device=DEV)
    stack.prefill(0, x, ids, w, z)
    moe.moe_sync_check()
    g_ids, g_w = ids.cpu().numpy(), w.cpu().numpy()
    o = oracle.LRU(capacity, wl.L, wl.E)
    every = np.arange(wl.E, dtype=np.int32)
    assert o.lookup(0, 0, every, prefetch=True) == oracle.OK
    for l in range(wl.L):
        assert o.lookup(0, l, g_ids[l].reshape(-1)) == oracle.OK
        if l + 1 < wl.L:
            assert o.lookup(0, l + 1, every, prefetch=True) == oracle.OK
    layers = _Layers(wl)
    xr = oracle_routed_chain(wl, x0, z.cpu().numpy(), g_ids, g_w, layers, logit_tol=PREFILL_LOGIT_TOL[wl.dtype])
    assert normwise(x.cpu().numpy() - x0, xr - x0) <= PREFILL_TOL[dtype]
    sets = synth.routing_sets(wl, steps=3)
    for t in range(3):
        xd0 = synth.hidden_states(wl, t)
        bias = np.stack([synth.mask_logits(wl, sets[t, l]) for l in range(wl.L)])
        xd = dev(xd0)
        di = torch.empty((wl.L, 1, wl.k), dtype=torch.int32, device=DEV)
        dw = torch.empty((wl.L, 1, wl.k), dtype=torch.float32, device=DEV)
        dz = torch.empty((wl.L, 1, wl.E), dtype=torch.float32, device=DEV)
        stack.decode_step(1 + t, xd, dev(bias), di, dw, dz)
        moe.moe_sync_check()
        for l in range(wl.L):
            assert o.lookup(1 + t, l, di.cpu().numpy()[l].reshape(-1)) == oracle.OK
        xr = oracle_routed_chain(wl, xd0, dz.cpu().numpy(), di.cpu().numpy(), dw.cpu().numpy(), layers, bias=bias)
        assert normwise(xd.cpu().numpy() - xd0, xr - xd0) <= TOL[dtype]
    ev, oev = cache.trace(), o.events()
    assert len(ev) == len(oev)
    assert (ev.view(np.int32).reshape(-1, 6) == oev.view(np.int32).reshape(-1, 6)).all()
    s, so = cache.stats(), o.stats()
    assert (s["hits"], s["misses"], s["prefetches"], s["evictions"]) == \
        (so["hits"], so["misses"], so["prefetches"], so["evictions"])
    assert so["prefetches"] > 0 and so["evictions"] > 0
    stack.close()
    cache.close()
    buf.close()


def test_stack_prefill_config5_two_layers_sampled():
    """Config 5's full 2048-token chunk through two of its layers (6 GiB budget: 3923 slots), checked on
    sampled tokens against the oracle chain."""
    wl = synth.workload(5, L=2)
    buf = _pinned_store(wl)
    eb = wl.expert_bytes
    reserved = wl.L * eb
    cache = moe.ExpertCache(wl.L, wl.E, eb, wl.budget_bytes, buf.ptr, wl.E * eb, eb, reserved_bytes=reserved)
    routers = [dev(synth.router_weights(wl, l)) for l in range(wl.L)]
    shw = [dev(synth.expert_blob(wl, l, None)) for l in range(wl.L)]
    stack = moe.MoeStack(cache, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, shw, max_tokens=1,
                         max_prefill_tokens=wl.prefill)
    x0 = synth.prefill_states(wl)
    x = dev(x0)
    ids = torch.empty((wl.L, wl.prefill, wl.k), dtype=torch.int32, device=DEV)
    w = torch.empty((wl.L, wl.prefill, wl.k), dtype=torch.float32, device=DEV)
    z = torch.empty((wl.L, wl.prefill, wl.E), dtype=torch.float32, device=DEV)
    stack.prefill(0, x, ids, w, z)
    moe.moe_sync_check()
    sample = np.random.default_rng(5).choice(wl.prefill, 12, replace=False)
    g_ids, g_w, g_z = ids.cpu().numpy()[:, sample], w.cpu().numpy()[:, sample], z.cpu().numpy()[:, sample]
    xr = oracle_routed_chain(wl, x0[sample], g_z, g_ids, g_w, _Layers(wl), logit_tol=PREFILL_LOGIT_TOL[wl.dtype])
    assert normwise(x.cpu().numpy()[sample] - x0[sample], xr - x0[sample]) <= PREFILL_TOL[wl.dtype]
    s = cache.stats()
    assert s["misses"] == len(np.unique(ids.cpu().numpy()[0])) + len(np.unique(ids.cpu().numpy()[1]))
    stack.close()
    cache.close()
    buf.close()


def test_cache_prefetch_and_demand_fills_on_device():
    """Device residency ordering, with no host synchronisation between steps: prefetches fill on the copy
    stream, demand lookups fill on the compute stream, each FFN reads the pool through the device slot table.
    With 6 slots, demand lookups evict prefetched slots (possibly still filling) and hit prefetched experts.
    Every FFN output matches the oracle on the experts it asked for; the residency log matches the oracle's."""
    wl = synth.Workload("cache order", H=256, E=16, k=4, I=128, L=2, dtype=synth.BF16, cfg_id=120)
    C, steps = 6, 40
    buf = _pinned_store(wl)
    eb = wl.expert_bytes
    cache = moe.ExpertCache(wl.L, wl.E, eb, C * eb, buf.ptr, wl.E * eb, eb)
    table, pool = cache.slot_table()
    o = oracle.LRU(C, wl.L, wl.E)
    rng = np.random.default_rng(0)
    host = {l: synth.layer_experts(wl, l) for l in range(wl.L)}
    ids_np = np.stack([rng.choice(wl.E, wl.k, replace=False) for _ in range(steps)]).astype(np.int32)[:, None, :]
    w_np = rng.random((steps, 1, wl.k)).astype(np.float32)
    w_np /= w_np.sum(axis=2, keepdims=True)
    x_np = rng.standard_normal((steps, 1, wl.H)).astype(np.float32)
    ids_d, w_d, x_d = dev(ids_np), dev(w_np), dev(x_np)
    y_d = torch.zeros((steps, 1, wl.H), dtype=torch.float32, device=DEV)
    ws = torch.empty(moe.moe_ffn_workspace_bytes(1, wl.k, wl.I), dtype=torch.uint8, device=DEV)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    for t in range(steps):
        l = t % 2
        if t % 3 == 0:
            pf = rng.choice(wl.E, 3, replace=False).astype(np.int32)
            cache.prefetch(t, 1 - l, pf)
            assert o.lookup(t, 1 - l, pf, prefetch=True) == oracle.OK
        cache.lookup(t, l, ids_np[t].reshape(-1), stream)
        assert o.lookup(t, l, ids_np[t].reshape(-1)) == oracle.OK
        rc = moe.lib().moe_expert_ffn_grouped(
            x_d[t].data_ptr(), 1, wl.H, wl.I, wl.E, wl.k, ids_d[t].data_ptr(), w_d[t].data_ptr(),
            table + 4 * l * wl.E, pool, eb, wl.dtype, None, y_d[t].data_ptr(), ws.data_ptr(),
            ws.numel(), 0, stream.cuda_stream)
        assert rc == 0, moe.lib().moe_last_error()
        cache.release(stream)
    moe.moe_sync_check()
    y = y_d.cpu().numpy()
    for t in range(steps):
        ref = oracle.moe_ffn(x_np[t], ids_np[t], w_np[t].astype(np.float64), host[t % 2], wl.H, wl.I, wl.dtype)
        assert normwise(y[t], ref) <= TOL[wl.dtype], t
    ev, oev = cache.trace(), o.events()
    assert len(ev) == len(oev)
    assert (ev.view(np.int32).reshape(-1, 6) == oev.view(np.int32).reshape(-1, 6)).all()
    s = cache.stats()
    assert s["prefetches"] > 0 and s["evictions"] > 0
    cache.close()
    buf.close()


def test_cache_device_prefetch_and_demand_fills():
    """Device residency with device prefetches, no host synchronisation between steps: each step prefetches
    three experts of the other layer (fills on the copy stream, overlapping the FFN queued next), then looks up
    its own experts on the device (waiting for those fills) and runs the FFN through the device slot table.
    With 6 slots, prefetches evict slots earlier FFNs read and lookups evict prefetched slots. Every FFN
    output matches the oracle on the experts it asked for; the residency log matches the oracle's."""
    wl = synth.Workload("cache order", H=256, E=16, k=4, I=128, L=2, dtype=synth.BF16, cfg_id=121)
    C, steps = 6, 40
    buf = _pinned_store(wl)
    eb = wl.expert_bytes
    cache = moe.ExpertCache(wl.L, wl.E, eb, C * eb, buf.ptr, wl.E * eb, eb, device=True)
    table, pool = cache.slot_table()
    o = oracle.LRU(C, wl.L, wl.E)
    rng = np.random.default_rng(1)
    host = {l: synth.layer_experts(wl, l) for l in range(wl.L)}
    ids_np = np.stack([rng.choice(wl.E, wl.k, replace=False) for _ in range(steps)]).astype(np.int32)[:, None, :]
    pf_np = np.stack([rng.choice(wl.E, 3, replace=False) for _ in range(steps)]).astype(np.int32)
    w_np = rng.random((steps, 1, wl.k)).astype(np.float32)
    w_np /= w_np.sum(axis=2, keepdims=True)
    x_np = rng.standard_normal((steps, 1, wl.H)).astype(np.float32)
    ids_d, pf_d, w_d, x_d = dev(ids_np), dev(pf_np), dev(w_np), dev(x_np)
    y_d = torch.zeros((steps, 1, wl.H), dtype=torch.float32, device=DEV)
    ws = torch.empty(moe.moe_ffn_workspace_bytes(1, wl.k, wl.I), dtype=torch.uint8, device=DEV)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    for t in range(steps):
        l = t % 2
        if t % 3 != 2:
            cache.prefetch_device(t, 1 - l, pf_d[t], stream)
            assert o.lookup(t, 1 - l, pf_np[t], prefetch=True) == oracle.OK
        cache.lookup_device(t, l, ids_d[t].reshape(-1), None, stream)
        assert o.lookup(t, l, ids_np[t].reshape(-1)) == oracle.OK
        rc = moe.lib().moe_expert_ffn_grouped(
            x_d[t].data_ptr(), 1, wl.H, wl.I, wl.E, wl.k, ids_d[t].data_ptr(), w_d[t].data_ptr(),
            table + 4 * l * wl.E, pool, eb, wl.dtype, None, y_d[t].data_ptr(), ws.data_ptr(),
            ws.numel(), 0, stream.cuda_stream)
        assert rc == 0, moe.lib().moe_last_error()
    torch.cuda.synchronize()
    moe.moe_sync_check()
    y = y_d.cpu().numpy()
    for t in range(steps):
        ref = oracle.moe_ffn(x_np[t], ids_np[t], w_np[t].astype(np.float64), host[t % 2], wl.H, wl.I, wl.dtype)
        assert normwise(y[t], ref) <= TOL[wl.dtype], t
    ev, oev = cache.trace(), o.events()
    assert len(ev) == len(oev)
    assert (ev.view(np.int32).reshape(-1, 6) == oev.view(np.int32).reshape(-1, 6)).all()
    s = cache.stats()
    assert s["prefetches"] > 0 and s["evictions"] > 0
    cache.close()
    buf.close()


def test_stack_decode_with_prefetch():
    """One-token decode with speculative prefetch (2 experts per layer): the residency log equals the oracle
    LRU replaying the same demand lookups and prefetches, every prefetch picked the next layer's most often
    demanded non-resident experts (ties: lower id), and outputs match the oracle chain."""
    wl = synth.Workload("prefetch stack", H=512, E=32, k=4, I=256, L=3, dtype=synth.BF16, routing="zipf_overlap",
                        cfg_id=130)
    capacity, steps, P = 20, 30, 2
    buf = _pinned_store(wl)
    eb = wl.expert_bytes
    cache = moe.ExpertCache(wl.L, wl.E, eb, capacity * eb, buf.ptr, wl.E * eb, eb)
    routers = [dev(synth.router_weights(wl, l)) for l in range(wl.L)]
    stack = moe.MoeStack(cache, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, None, prefetch=P)
    sets = synth.routing_sets(wl, steps=steps)
    layers = _Layers(wl)
    for t in range(steps):
        x0 = synth.hidden_states(wl, t)
        bias = np.stack([synth.mask_logits(wl, sets[t, l]) for l in range(wl.L)])
        x = dev(x0)
        ids = torch.empty((wl.L, 1, wl.k), dtype=torch.int32, device=DEV)
        w = torch.empty((wl.L, 1, wl.k), dtype=torch.float32, device=DEV)
        z = torch.empty((wl.L, 1, wl.E), dtype=torch.float32, device=DEV)
        stack.decode_step(t, x, dev(bias), ids, w, z)
        moe.moe_sync_check()
        if t % 7 == 0:
            xr = oracle_routed_chain(wl, x0, z.cpu().numpy(), ids.cpu().numpy(), w.cpu().numpy(), layers, bias=bias)
            assert normwise(x.cpu().numpy() - x0, xr - x0) <= TOL[wl.dtype]
    ev = cache.trace()
    # replay: consecutive events of one call share (t, layer) and demand-or-prefetch kind
    kind_pf = ev["kind"] == moe.EVENT_PREFETCH
    key = ev["t"].astype(np.int64) * 4096 + ev["layer"] * 2 + kind_pf
    starts = np.flatnonzero(np.r_[True, key[1:] != key[:-1]])
    ends = np.r_[starts[1:], ev.size]
    o = oracle.LRU(capacity, wl.L, wl.E)
    counts = np.zeros((wl.L, wl.E), np.int64)
    n_pf = 0
    for a, b in zip(starts, ends):
        t, layer, ex = int(ev["t"][a]), int(ev["layer"][a]), ev["expert"][a:b]
        if kind_pf[a]:
            resident = np.array([o.slot_of(layer, e) >= 0 for e in range(wl.E)])
            cand = [e for e in range(wl.E) if not resident[e]]
            cand.sort(key=lambda e: (-counts[layer, e], e))
            assert sorted(ex.tolist()) == sorted(cand[:P])
            assert o.lookup(t, layer, ex, prefetch=True) == oracle.OK
            n_pf += b - a
        else:
            assert o.lookup(t, layer, ex) == oracle.OK
            counts[layer, ex] += 1
    oev = o.events()
    assert len(ev) == len(oev)
    assert (ev.view(np.int32).reshape(-1, 6) == oev.view(np.int32).reshape(-1, 6)).all()
    assert n_pf > 0 and cache.stats()["prefetches"] == n_pf
    stack.close()
    cache.close()
    buf.close()


# ------------------------------------------------------------- decoder attention ---
# bf16 weights and caches, fp32 arithmetic: the attention block's output (x + W_o Attn) is compared as its
# increment over x, normwise against the fp64 oracle.
ATTN_LOGIT_TOL = 2e-3  # logits after attention blocks whose new key or value may round to another bf16 value
ATTN_TOL = 1e-2


def _attn_case(H, n_heads, n_kv, d, max_pos, seed):
    rng = np.random.default_rng(seed)
    bf = lambda a: synth.bf16_bits(np.asarray(a, np.float32))
    wqkv = bf(rng.standard_normal(((n_heads + 2 * n_kv) * d, H)) * 0.02)
    wo = bf(rng.standard_normal((H, n_heads * d)) * 0.02)
    kc = bf(rng.standard_normal((n_kv, max_pos, d)))    # unit-RMS keys, as normalised heads are
    vc = bf(rng.standard_normal((n_kv, max_pos, d)))
    x = rng.standard_normal(H).astype(np.float32)
    return wqkv, wo, kc, vc, x


def _i16(a):  # bf16 bits as a torch-friendly int16 device tensor
    return dev(np.ascontiguousarray(a).view(np.int16))


@pytest.mark.parametrize("H,nh,nkv,d,max_pos,p", [(256, 4, 2, 64, 300, 0), (256, 4, 2, 64, 300, 1),
                                                  (256, 4, 2, 64, 300, 63), (256, 4, 2, 64, 300, 64),
                                                  (256, 4, 2, 64, 300, 65), (256, 8, 1, 32, 300, 299),
                                                  (512, 8, 2, 128, 256, 200), (2048, 32, 4, 128, 4096, 4095),
                                                  (256, 16, 1, 128, 200, 130), (256, 2, 2, 128, 200, 7),
                                                  (256, 4, 4, 32, 100, 99)])
def test_attention_decode_parity(H, nh, nkv, d, max_pos, p):
    wqkv, wo, kc, vc, x = _attn_case(H, nh, nkv, d, max_pos, seed=H + p)
    kc_o, vc_o = kc.copy(), vc.copy()
    y_ref = oracle.attention_decode(x, wqkv, wo, kc_o, vc_o, p, nh, nkv)
    xd, kd, vd = dev(x), _i16(moe.key_cache_layout(kc)), _i16(vc)
    moe.moe_attention_decode(xd, _i16(wqkv), _i16(wo), kd, vd, p, nh, nkv)
    moe.moe_sync_check()
    got = xd.cpu().numpy().astype(np.float64)
    assert normwise(got - x, y_ref - x) <= ATTN_TOL
    k_gpu = moe.key_cache_plain(kd.cpu().numpy().view(np.uint16))
    v_gpu = vd.cpu().numpy().view(np.uint16)
    others = np.arange(max_pos) != p
    assert np.array_equal(k_gpu[:, others], kc[:, others]) and np.array_equal(v_gpu[:, others], vc[:, others])
    f = lambda b: synth.bf16_to_f32(b).astype(np.float64)
    assert np.abs(f(k_gpu[:, p]) - f(kc_o[:, p])).max() <= 1e-2 * max(1.0, np.abs(f(kc_o[:, p])).max())
    assert np.abs(f(v_gpu[:, p]) - f(vc_o[:, p])).max() <= 1e-2 * max(1.0, np.abs(f(vc_o[:, p])).max())


@pytest.mark.parametrize("p", [0, 64, 70, 127])
def test_attention_decode_ignores_cache_content_past_p(p):
    """NaN keys and values at positions p and above (position p is written before it is read; the partial
    kernel's loads past the last position are clamped to p, with weight 0): output equals the oracle's."""
    H, nh, nkv, d, max_pos = 256, 8, 2, 128, 160
    wqkv, wo, kc, vc, x = _attn_case(H, nh, nkv, d, max_pos, seed=31 + p)
    kc[:, p:], vc[:, p:] = 0x7FC0, 0x7FC0  # bf16 quiet NaN
    kc_o, vc_o = kc.copy(), vc.copy()
    y_ref = oracle.attention_decode(x, wqkv, wo, kc_o, vc_o, p, nh, nkv)
    assert np.isfinite(y_ref).all()
    xd = dev(x)
    moe.moe_attention_decode(xd, _i16(wqkv), _i16(wo), _i16(moe.key_cache_layout(kc)), _i16(vc), p, nh, nkv)
    moe.moe_sync_check()
    got = xd.cpu().numpy().astype(np.float64)
    assert np.isfinite(got).all() and normwise(got - x, y_ref - x) <= ATTN_TOL


def test_attention_decode_sequence_appends_across_chunks():
    """70 tokens from an empty cache (the 64-position chunk boundary crossed), GPU and oracle each keeping
    their own caches; every step's output compared."""
    H, nh, nkv, d, max_pos = 256, 4, 1, 64, 96
    wqkv, wo, _, _, _ = _attn_case(H, nh, nkv, d, max_pos, seed=11)
    kc_o = np.zeros((nkv, max_pos, d), np.uint16)
    vc_o = np.zeros_like(kc_o)
    kd, vd = _i16(moe.key_cache_layout(kc_o)), _i16(vc_o)
    wq_d, wo_d = _i16(wqkv), _i16(wo)
    rng = np.random.default_rng(12)
    for p in range(70):
        x = rng.standard_normal(H).astype(np.float32)
        y_ref = oracle.attention_decode(x, wqkv, wo, kc_o, vc_o, p, nh, nkv)
        xd = dev(x)
        moe.moe_attention_decode(xd, wq_d, wo_d, kd, vd, p, nh, nkv)
        moe.moe_sync_check()
        assert normwise(xd.cpu().numpy().astype(np.float64) - x, y_ref - x) <= ATTN_TOL, p


def test_attention_decode_rejects_bad_arguments():
    H, nh, nkv, d, max_pos = 256, 4, 2, 64, 32
    wqkv, wo, kc, vc, x = _attn_case(H, nh, nkv, d, max_pos, seed=5)
    args = (_i16(wqkv), _i16(wo), _i16(moe.key_cache_layout(kc)), _i16(vc))
    for p, nh_, nkv_ in ((max_pos, nh, nkv), (-1, nh, nkv), (0, 4, 3), (0, 40, 2), (0, 6, 2)):
        with pytest.raises(moe.MoeError) as ei:
            moe.moe_attention_decode(dev(x), *args, p, nh_, nkv_)
        assert ei.value.code == -1


def test_stack_with_attention_blocks_matches_oracle_chain():
    """Each layer x <- x + Attn(rmsnorm(x)), then the MoE block, over a budgeted device cache; the oracle
    chain (its own caches, routed by the oracle) token by token.  A new key or value may round to a
    neighbouring bf16 value on one side only, so the chain states (and the logits) may differ by that much of
    an attention increment."""
    wl = synth.Workload("attn stack", H=256, E=16, k=2, I=128, L=3, dtype=synth.BF16, routing="zipf_overlap",
                        cfg_id=94)
    nh, nkv, d, max_pos, start = 4, 2, 64, 40, 20
    eb, cap = wl.expert_bytes, 10
    buf = _pinned_store(wl)
    cache = moe.ExpertCache(wl.L, wl.E, eb, cap * eb, buf.ptr, wl.E * eb, eb, device=True)
    routers = [dev(synth.router_weights(wl, l)) for l in range(wl.L)]
    blocks = [_attn_case(wl.H, nh, nkv, d, max_pos, seed=300 + l) for l in range(wl.L)]
    kc_o = [b[2].copy() for b in blocks]
    vc_o = [b[3].copy() for b in blocks]
    att = dict(n_heads=nh, n_kv=nkv, head_dim=d, max_pos=max_pos, theta=1.0e6, start_pos=start,
               w_qkv=[_i16(b[0]) for b in blocks], w_o=[_i16(b[1]) for b in blocks],
               k_cache=[_i16(moe.key_cache_layout(b[2])) for b in blocks], v_cache=[_i16(b[3]) for b in blocks])
    stack = moe.MoeStack(cache, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, None, attention=att)
    sets = synth.routing_sets(wl, steps=6)
    layers = _Layers(wl)
    for t in range(6):
        x0 = synth.hidden_states(wl, t)
        bias = np.stack([synth.mask_logits(wl, sets[t, l]) for l in range(wl.L)])
        x = dev(x0)
        ids = torch.empty((wl.L, 1, wl.k), dtype=torch.int32, device=DEV)
        w = torch.empty((wl.L, 1, wl.k), dtype=torch.float32, device=DEV)
        z = torch.empty((wl.L, 1, wl.E), dtype=torch.float32, device=DEV)
        stack.decode_step(t, x, dev(bias), ids, w, z)
        moe.moe_sync_check()
        g_ids, g_w = ids.cpu().numpy(), w.cpu().numpy()
        for l in range(wl.L):
            assert (np.sort(g_ids[l], axis=1) == sets[t, l]).all()
        attn = lambda l, xr: oracle.attention_decode(xr.reshape(-1).astype(np.float32), blocks[l][0], blocks[l][1],
                                                     kc_o[l], vc_o[l], start + t, nh, nkv)
        xr = oracle_routed_chain(wl, x0, z.cpu().numpy(), g_ids, g_w, layers, bias=bias, attention=attn,
                                 logit_tol0=ATTN_LOGIT_TOL, logit_tol=ATTN_LOGIT_TOL).reshape(-1)
        assert normwise(x.cpu().numpy().reshape(-1) - x0.reshape(-1), xr - x0.reshape(-1)) <= ATTN_TOL, t
    assert stack.kernel_time(4, 2) > 0
    moe.moe_sync_check()
    with pytest.raises(moe.MoeError):  # two tokens in one step
        stack.decode_step(6, dev(np.zeros((2, wl.H), np.float32)))
    stack.close()
    with pytest.raises(moe.MoeError):  # prefill with an attention block
        moe.MoeStack(cache, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, None, attention=att,
                     max_prefill_tokens=16)
    full = dict(att, start_pos=max_pos - 1)
    stack = moe.MoeStack(cache, wl.H, wl.I, wl.E, wl.k, wl.dtype, wl.router_dtype, routers, None, attention=full)
    stack.decode_step(100, dev(synth.hidden_states(wl, 7)))
    moe.moe_sync_check()
    with pytest.raises(moe.MoeError):  # the caches are full
        stack.decode_step(101, dev(synth.hidden_states(wl, 8)))
    stack.close()
    cache.close()
    buf.close()
