"""The expert FFN entry point that allocates nothing (moe_expert_ffn_grouped_noalloc), through the C ABI.

Its kernels are those of moe_expert_ffn_grouped, on the library's fixed per-device scratch instead of a
caller workspace, so its output must equal that entry point's bit for bit on the same inputs.  Two calls in a
row, the second with a smaller input, check that the shared array's leftovers from the first call do not
leak into the second.  Both are also checked against the oracle at the benchmark spec's tolerance.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2605_29135_amd as moe
import synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
TOL = {synth.F32: 1e-5, synth.BF16: 1e-2, synth.INT4G128: 3e-2}


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _normwise(y, ref):
    y, ref = np.atleast_2d(y).astype(np.float64), np.atleast_2d(ref)
    return float(np.max(np.abs(y - ref).max(axis=1) / np.maximum(np.abs(ref).max(axis=1), 1e-30)))


def _case(wl, T, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, wl.H)).astype(np.float32)
    ids = np.stack([rng.choice(wl.E, wl.k, replace=False) for _ in range(T)]).astype(np.int32)
    w = rng.random((T, wl.k)).astype(np.float32)
    w /= w.sum(axis=1, keepdims=True)
    return x, ids, w


@pytest.mark.parametrize("dtype", [synth.BF16, synth.INT4G128])
def test_noalloc_ffn_equals_workspace_ffn_on_two_calls(dtype):
    moe.moe_init(0)
    wl = synth.Workload("noalloc", H=2048, E=32, k=8, I=512, dtype=dtype, shared=True, cfg_id=77 + dtype)
    experts = synth.layer_experts(wl, 0)
    shared = synth.expert_blob(wl, 0, None)
    pool, sh = _dev(experts.reshape(-1)), _dev(shared)
    for T, seed in ((16, 1), (3, 2)):  # the second call is smaller than the first
        x, ids, w = _case(wl, T, seed)
        xd, idd, wd = _dev(x), _dev(ids), _dev(w)
        y_ws = moe.moe_expert_ffn_grouped(xd, idd, wd, pool, wl.expert_bytes, dtype, wl.I, wl.E, shared_w=sh)
        y_na = torch.full_like(y_ws, float("nan"))
        moe.moe_expert_ffn_grouped_noalloc(xd, idd, wd, pool, wl.expert_bytes, dtype, wl.I, wl.E, shared_w=sh,
                                           y_out=y_na)
        moe.moe_sync_check()
        assert torch.equal(y_na, y_ws), T
        ref = oracle.moe_ffn(x, ids, w, experts, wl.H, wl.I, dtype, shared)
        assert _normwise(y_na.cpu().numpy(), ref) <= TOL[dtype], T


def test_noalloc_ffn_rejects_inputs_beyond_the_fixed_scratch():
    moe.moe_init(0)
    H, I, E, k, T = 2048, 4096, 16, 16, 16  # (T*k + T) * I * 4 bytes = 4.25 MiB > 4 MiB
    assert moe.moe_ffn_workspace_bytes(T, k, I) > 4 << 20
    x = torch.zeros((T, H), dtype=torch.float32, device=DEV)
    ids = torch.zeros((T, k), dtype=torch.int32, device=DEV)
    w = torch.zeros((T, k), dtype=torch.float32, device=DEV)
    pool = torch.zeros(256, dtype=torch.uint8, device=DEV)
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_expert_ffn_grouped_noalloc(x, ids, w, pool, synth.expert_bytes(H, I, synth.BF16), synth.BF16, I, E)
    assert ei.value.code == -1 and "scratch" in str(ei.value)
    moe.moe_sync_check()
