"""ctypes binding of libmoe_budget.so: argument marshalling only.

Every step of the path runs in the library's HIP kernels; this module turns
torch tensors into device pointers and raises :class:`MoeError` on a non-zero
status.  There is no fallback: if the library is not built, loading fails.
"""
from __future__ import annotations

import ctypes as C
import os
import re

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmoe_budget.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "moe_budget.h")

MOE_OK = 0
ERR_NAMES = {-1: "INVALID_ARG", -2: "RANGE", -3: "NONFINITE", -4: "BUDGET", -5: "NOT_PINNED",
             -6: "HIP", -7: "COPY", -8: "NOT_RESIDENT"}
MOE_F32, MOE_BF16, MOE_INT4G128 = 0, 1, 2
MOE_ACCUMULATE = 1
MOE_ROUTE_RMSNORM = 1
MOE_POLICY_LRU = 0
MOE_POLICY_ROTARY = 1
MOE_CACHE_PRELOAD, MOE_CACHE_HOST_SIM, MOE_CACHE_DEVICE, MOE_CACHE_FILL_CLOCK = 1, 2, 4, 8
EVENT_HIT, EVENT_MISS, EVENT_PREFETCH, EVENT_HOST = 0, 1, 2, 3
MOE_SLOT_HOST = -2
MAX_DECODE_TOKENS = 16


class MoeError(RuntimeError):
    def __init__(self, code: int, where: str, msg: str):
        super().__init__(f"{where}: MOE_ERR_{ERR_NAMES.get(code, code)} ({code}): {msg}")
        self.code = code


class CacheDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("n_experts", C.c_int), ("expert_bytes", C.c_size_t),
                ("budget_bytes", C.c_size_t), ("reserved_bytes", C.c_size_t), ("host_base", C.c_void_p),
                ("host_layer_stride", C.c_size_t), ("host_expert_stride", C.c_size_t),
                ("policy", C.c_int), ("flags", C.c_int), ("charge_max", C.c_int), ("host_layers", C.c_int),
                ("host_quota", C.c_int)]


class CacheStats(C.Structure):
    _fields_ = [("lookups", C.c_uint64), ("hits", C.c_uint64), ("misses", C.c_uint64),
                ("prefetches", C.c_uint64), ("evictions", C.c_uint64), ("h2d_bytes", C.c_uint64),
                ("capacity", C.c_int32), ("occupancy", C.c_int32), ("stall_ns", C.c_uint64),
                ("fill_ns", C.c_uint64), ("host_computed", C.c_uint64)]


EVENT_DTYPE = np.dtype([("t", "<i4"), ("layer", "<i4"), ("expert", "<i4"),
                        ("kind", "<i4"), ("slot", "<i4"), ("victim_key", "<i4")])


class AttentionDesc(C.Structure):
    _fields_ = [("n_heads", C.c_int), ("n_kv", C.c_int), ("head_dim", C.c_int), ("max_pos", C.c_int),
                ("theta", C.c_float), ("start_pos", C.c_int), ("w_qkv", C.POINTER(C.c_void_p)),
                ("w_o", C.POINTER(C.c_void_p)), ("k_cache", C.POINTER(C.c_void_p)), ("v_cache", C.POINTER(C.c_void_p))]


class StackDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("H", C.c_int), ("I", C.c_int), ("E", C.c_int), ("k", C.c_int),
                ("w_dtype", C.c_int), ("router_dtype", C.c_int), ("router_w", C.POINTER(C.c_void_p)),
                ("shared_w", C.POINTER(C.c_void_p)), ("cache", C.c_void_p), ("max_tokens", C.c_int),
                ("max_prefill_tokens", C.c_int), ("prefetch", C.c_int), ("recall", C.c_int),
                ("recall_overlap", C.c_int), ("attention", C.POINTER(AttentionDesc)), ("host_threads", C.c_int)]


_lib = None


def lib() -> C.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built: run __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        P, I, SZ, U64P = C.c_void_p, C.c_int, C.c_size_t, C.POINTER(C.c_uint64)
        sig = {
            "moe_init": [I], "moe_last_error": [], "moe_sync_check": [P],
            "moe_route_topk": [P, P, I, I, I, I, I, P, P, P, P, I, P, P],
            "moe_ffn_workspace_bytes": [I, I, I],
            "moe_expert_ffn_grouped": [P, I, I, I, I, I, P, P, P, P, SZ, I, P, P, P, SZ, I, P],
            "moe_expert_ffn_grouped_noalloc": [P, I, I, I, I, I, P, P, P, P, SZ, I, P, P, I, P],
            "moe_combine": [P, P, P, I, I, I, P, I, P],
            "moe_attention_decode": [P, I, I, I, I, P, P, P, P, I, I, C.c_float, P, SZ, P],
            "moe_prefill_workspace_bytes": [I, I, I, I, I],
            "moe_prefill_grouped": [P, I, I, I, I, I, P, P, P, P, SZ, I, P, P, P, SZ, I, P],
            "expert_cache_create": [C.POINTER(CacheDesc), C.POINTER(P)],
            "expert_cache_destroy": [P],
            "expert_cache_lookup": [P, I, I, P, I, P, P, P],
            "expert_cache_lookup_device": [P, I, I, P, I, P, P],
            "expert_cache_prefetch_device": [P, I, I, P, I, P],
            "expert_cache_prefetch": [P, I, I, P, I],
            "expert_cache_release": [P, P],
            "expert_cache_slot_table": [P, C.POINTER(P), C.POINTER(P)],
            "expert_cache_stats": [P, C.POINTER(CacheStats)],
            "expert_cache_trace": [P, SZ, P, SZ, C.POINTER(SZ)],
            "moe_stack_create": [C.POINTER(StackDesc), C.POINTER(P)],
            "moe_host_tier_create": [I, C.POINTER(P)],
            "moe_host_tier_destroy": [P],
            "moe_host_expert_ffn": [P, P, I, I, I, I, P, P, P],
            "moe_stack_destroy": [P],
            "moe_stack_decode_step": [P, I, P, I, P, P, P, P, P],
            "moe_stack_decode_graph": [P, I, P, P, P, P, P, P],
            "moe_stack_kernel_time": [P, I, I, P, C.POINTER(C.c_double)],
            "moe_stack_prefill": [P, I, P, I, P, P, P, P],
            "moe_hbm_read_probe": [P, SZ, P, P],
            "moe_opt_fills": [P, P, I, I, I, U64P],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = I
        L.moe_last_error.restype = C.c_char_p
        L.moe_ffn_workspace_bytes.restype = SZ
        L.moe_prefill_workspace_bytes.restype = SZ
        _lib = L
    return _lib


def header_symbols() -> list[str]:
    """Entry points declared in include/moe_budget.h."""
    with open(HEADER) as f:
        return re.findall(r"^MOE_API\s+[\w\s\*]*?\b(\w+)\s*\(", f.read(), flags=re.M)


def _check(code: int, where: str) -> None:
    if code != MOE_OK:
        raise MoeError(code, where, lib().moe_last_error().decode(errors="replace"))


# ------------------------------------------------------------ marshalling ---
def _dev(t, name: str, dtype=None):
    """Device pointer of a contiguous CUDA tensor (or 0 for None)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    return t.data_ptr()


def _stream(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


# ------------------------------------------------------------ entry points ---
def moe_init(device: int = 0) -> None:
    _check(lib().moe_init(device), "moe_init")


def moe_sync_check(stream=None) -> None:
    _check(lib().moe_sync_check(_stream(stream)), "moe_sync_check")


def moe_route_topk(x, w_router, w_dtype: int, k: int, *, E: int | None = None, logit_bias=None,
                   logits=None, ids=None, weights=None, rmsnorm: bool = False, x_norm=None, stream=None):
    """Router logits and top-k; returns (logits [T x E], ids [T x k], weights [T x k]).

    With ``rmsnorm`` the router reads x / rms(x) and, if ``x_norm`` is given,
    stores that normalised input there."""
    import torch
    src = x if x is not None else logit_bias
    T = src.shape[0]
    H = x.shape[1] if x is not None else 0
    E = E if E is not None else (w_router.shape[0] if w_router is not None else logit_bias.shape[1])
    dev = src.device
    logits = torch.empty((T, E), dtype=torch.float32, device=dev) if logits is None else logits
    ids = torch.empty((T, k), dtype=torch.int32, device=dev) if ids is None else ids
    weights = torch.empty((T, k), dtype=torch.float32, device=dev) if weights is None else weights
    _check(lib().moe_route_topk(_dev(x, "x", torch.float32), _dev(w_router, "w_router"), w_dtype, T, H, E, k,
                                _dev(logit_bias, "logit_bias", torch.float32),
                                _dev(logits, "logits", torch.float32), _dev(ids, "ids", torch.int32),
                                _dev(weights, "weights", torch.float32), MOE_ROUTE_RMSNORM if rmsnorm else 0,
                                _dev(x_norm, "x_norm", torch.float32), _stream(stream)), "moe_route_topk")
    return logits, ids, weights


def moe_ffn_workspace_bytes(T: int, k: int, I: int) -> int:
    return int(lib().moe_ffn_workspace_bytes(T, k, I))


def moe_expert_ffn_grouped(x, ids, weights, pool, expert_bytes: int, w_dtype: int, I: int, E: int, *,
                           slot_of=None, shared_w=None, y_out=None, workspace=None, accumulate: bool = False,
                           stream=None):
    """y = sum_j w_j FFN_{ids_j}(x) (+ shared); returns y_out [T x H]."""
    import torch
    T, H = x.shape
    k = ids.shape[1]
    y_out = torch.empty((T, H), dtype=torch.float32, device=x.device) if y_out is None else y_out
    nws = moe_ffn_workspace_bytes(T, k, I)
    if workspace is None:
        workspace = torch.empty(max(nws, 256), dtype=torch.uint8, device=x.device)
    _check(lib().moe_expert_ffn_grouped(
        _dev(x, "x", torch.float32), T, H, I, E, k, _dev(ids, "ids", torch.int32),
        _dev(weights, "weights", torch.float32), _dev(slot_of, "slot_of", torch.int32), _dev(pool, "pool"),
        expert_bytes, w_dtype, _dev(shared_w, "shared_w"), _dev(y_out, "y_out", torch.float32),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        MOE_ACCUMULATE if accumulate else 0, _stream(stream)), "moe_expert_ffn_grouped")
    return y_out


def moe_expert_ffn_grouped_noalloc(x, ids, weights, pool, expert_bytes: int, w_dtype: int, I: int, E: int, *,
                                   slot_of=None, shared_w=None, y_out=None, accumulate: bool = False, stream=None):
    """moe_expert_ffn_grouped on the library's fixed per-device scratch (the call allocates nothing; pass
    y_out to keep this wrapper from allocating it); returns y_out [T x H]."""
    import torch
    T, H = x.shape
    k = ids.shape[1]
    y_out = torch.empty((T, H), dtype=torch.float32, device=x.device) if y_out is None else y_out
    _check(lib().moe_expert_ffn_grouped_noalloc(
        _dev(x, "x", torch.float32), T, H, I, E, k, _dev(ids, "ids", torch.int32),
        _dev(weights, "weights", torch.float32), _dev(slot_of, "slot_of", torch.int32), _dev(pool, "pool"),
        expert_bytes, w_dtype, _dev(shared_w, "shared_w"), _dev(y_out, "y_out", torch.float32),
        MOE_ACCUMULATE if accumulate else 0, _stream(stream)), "moe_expert_ffn_grouped_noalloc")
    return y_out


def moe_prefill_workspace_bytes(T: int, k: int, E: int, H: int, I: int) -> int:
    return int(lib().moe_prefill_workspace_bytes(T, k, E, H, I))


def moe_prefill_grouped(x, ids, weights, pool, expert_bytes: int, w_dtype: int, I: int, E: int, *,
                        slot_of=None, shared_w=None, y_out=None, workspace=None, accumulate: bool = False,
                        stream=None):
    """Prefill-chunk expert FFN (grouped bf16 MFMA GEMMs); returns y_out [T x H]."""
    import torch
    T, H = x.shape
    k = ids.shape[1]
    y_out = torch.empty((T, H), dtype=torch.float32, device=x.device) if y_out is None else y_out
    nws = moe_prefill_workspace_bytes(T, k, E, H, I)
    if workspace is None:
        workspace = torch.empty(max(nws, 256), dtype=torch.uint8, device=x.device)
    _check(lib().moe_prefill_grouped(
        _dev(x, "x", torch.float32), T, H, I, E, k, _dev(ids, "ids", torch.int32),
        _dev(weights, "weights", torch.float32), _dev(slot_of, "slot_of", torch.int32), _dev(pool, "pool"),
        expert_bytes, w_dtype, _dev(shared_w, "shared_w"), _dev(y_out, "y_out", torch.float32),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        MOE_ACCUMULATE if accumulate else 0, _stream(stream)), "moe_prefill_grouped")
    return y_out


def moe_opt_fills(steps, n_keys: int, capacity: int) -> int:
    """Fewest fills any replacement policy needs for `steps` (arrays of distinct keys, each step's keys
    resident together) with `capacity` slots (host-side analysis in the library)."""
    arrs = [np.ascontiguousarray(np.asarray(s_, np.int32).reshape(-1)) for s_ in steps]
    keys = np.ascontiguousarray(np.concatenate(arrs) if arrs else np.zeros(0, np.int32), dtype=np.int32)
    offsets = np.zeros(len(arrs) + 1, np.int32)
    offsets[1:] = np.cumsum([a.size for a in arrs])
    out = C.c_uint64()
    _check(lib().moe_opt_fills(keys.ctypes.data, offsets.ctypes.data, len(arrs), n_keys, capacity, C.byref(out)),
           "moe_opt_fills")
    return out.value


def moe_opt_fills_flat(keys, offsets, n_keys: int, capacity: int) -> int:
    """moe_opt_fills on a flat trace: keys int32 [n], offsets int32 [steps + 1]."""
    keys = np.ascontiguousarray(keys, dtype=np.int32)
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    out = C.c_uint64()
    _check(lib().moe_opt_fills(keys.ctypes.data, offsets.ctypes.data, offsets.size - 1, n_keys, capacity,
                               C.byref(out)), "moe_opt_fills")
    return out.value


def moe_hbm_read_probe(buf, sink, stream=None):
    """Stream the device tensor `buf` once with the expert kernels' 16-byte loads (measurement aid)."""
    import torch
    nbytes = buf.numel() * buf.element_size()
    _check(lib().moe_hbm_read_probe(_dev(buf, "buf"), nbytes, _dev(sink, "sink", torch.float32), _stream(stream)),
           "moe_hbm_read_probe")


def moe_attention_workspace_bytes(n_heads: int, n_kv: int, head_dim: int, max_pos: int) -> int:
    return int(lib().moe_attention_workspace_bytes(n_heads, n_kv, head_dim, max_pos))


def key_cache_layout(k_plain: np.ndarray) -> np.ndarray:
    """[n_kv, max_pos, d] keys -> the library's key-cache layout [n_kv, d/8, max_pos, 8]."""
    n_kv, max_pos, d = k_plain.shape
    return np.ascontiguousarray(k_plain.reshape(n_kv, max_pos, d // 8, 8).transpose(0, 2, 1, 3))


def key_cache_plain(k_lib: np.ndarray) -> np.ndarray:
    """Inverse of key_cache_layout: [n_kv, d/8, max_pos, 8] -> [n_kv, max_pos, d]."""
    n_kv, dc, max_pos, _ = k_lib.shape
    return np.ascontiguousarray(k_lib.transpose(0, 2, 1, 3)).reshape(n_kv, max_pos, dc * 8)


def moe_attention_decode(x, w_qkv, w_o, k_cache, v_cache, p: int, n_heads: int, n_kv: int, theta: float = 1.0e6,
                         workspace=None, stream=None):
    """x <- x + W_o Attn(rmsnorm(x)) at position p, in place on the device fp32 tensor x [H].  k_cache
    (bf16/int16 [n_kv, d/8, max_pos, 8]) and v_cache ([n_kv, max_pos, d]) receive position p."""
    import torch
    H = x.numel()
    n_kv_, max_pos, d = v_cache.shape
    nws = moe_attention_workspace_bytes(n_heads, n_kv, d, max_pos)
    if workspace is None:
        workspace = torch.empty(max(nws, 256), dtype=torch.uint8, device=x.device)
    _check(lib().moe_attention_decode(_dev(x, "x", torch.float32), H, n_heads, n_kv, d, _dev(w_qkv, "w_qkv"),
                                      _dev(w_o, "w_o"), _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"), max_pos,
                                      p, theta, _dev(workspace, "workspace"),
                                      workspace.numel() * workspace.element_size(), _stream(stream)),
           "moe_attention_decode")
    return x


def moe_combine(y_partial, weights, y_shared=None, y_out=None, accumulate: bool = False, stream=None):
    """y[t] = sum_j weights[t,j] * y_partial[t,j] (+ y_shared[t])."""
    import torch
    T, k, H = y_partial.shape
    y_out = torch.empty((T, H), dtype=torch.float32, device=y_partial.device) if y_out is None else y_out
    _check(lib().moe_combine(_dev(y_partial, "y_partial", torch.float32), _dev(weights, "weights", torch.float32),
                             _dev(y_shared, "y_shared", torch.float32), T, k, H,
                             _dev(y_out, "y_out", torch.float32), MOE_ACCUMULATE if accumulate else 0,
                             _stream(stream)), "moe_combine")
    return y_out


class HostTier:
    """Owner of one moe_host_tier (a pool of host threads computing experts from host memory)."""

    def __init__(self, threads: int = 0):
        h = C.c_void_p()
        _check(lib().moe_host_tier_create(threads, C.byref(h)), "moe_host_tier_create")
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            lib().moe_host_tier_destroy(self._h)
            self._h = None

    __del__ = close

    def expert_ffn(self, x, blobs, weights, H: int, I: int, w_dtype: int):
        """y = sum_j weights[j] FFN_j(x) over host blobs (numpy uint8 arrays or addresses); numpy in and out."""
        xa = np.ascontiguousarray(x, dtype=np.float32).reshape(-1)
        keep = [b if isinstance(b, int) else np.ascontiguousarray(b) for b in blobs]
        ptrs = (C.c_void_p * max(1, len(keep)))(*[b if isinstance(b, int) else b.ctypes.data for b in keep])
        wa = np.ascontiguousarray(weights, dtype=np.float32).reshape(-1)
        y = np.empty(H, np.float32)
        _check(lib().moe_host_expert_ffn(self._h, xa.ctypes.data, H, I, w_dtype, len(keep), ptrs, wa.ctypes.data,
                                         y.ctypes.data), "moe_host_expert_ffn")
        return y


class ExpertCache:
    """Owner of one expert_cache (slot table in HBM over a pinned host store; LRU or rotary replacement)."""

    def __init__(self, n_layers: int, n_experts: int, expert_bytes: int, budget_bytes: int, host_base: int,
                 host_layer_stride: int, host_expert_stride: int, reserved_bytes: int = 0,
                 preload: bool = False, host_sim: bool = False, policy: int = MOE_POLICY_LRU,
                 charge_max: int = 0, device: bool = False, host_layers: int = 0, host_quota: int = 0,
                 fill_clock: bool = False):
        d = CacheDesc(n_layers, n_experts, expert_bytes, budget_bytes, reserved_bytes, host_base,
                      host_layer_stride, host_expert_stride, policy,
                      (MOE_CACHE_PRELOAD if preload else 0) | (MOE_CACHE_HOST_SIM if host_sim else 0) |
                      (MOE_CACHE_DEVICE if device else 0) | (MOE_CACHE_FILL_CLOCK if fill_clock else 0),
                      charge_max, host_layers, host_quota)
        h = C.c_void_p()
        _check(lib().expert_cache_create(C.byref(d), C.byref(h)), "expert_cache_create")
        self._h = h
        self.L, self.E, self.host_sim = n_layers, n_experts, host_sim

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None):
            lib().expert_cache_destroy(self._h)
            self._h = None

    __del__ = close

    def lookup(self, step: int, layer: int, ids, stream=None):
        """Host-side lookup; returns (slots int32 [n], hit uint8 [n])."""
        a = np.ascontiguousarray(np.asarray(ids).reshape(-1), dtype=np.int32)
        slots = np.empty(a.size, np.int32)
        hit = np.empty(a.size, np.uint8)
        s = None if self.host_sim else _stream(stream)
        _check(lib().expert_cache_lookup(self._h, step, layer, a.ctypes.data, a.size, slots.ctypes.data,
                                         hit.ctypes.data, s), "expert_cache_lookup")
        return slots, hit

    def lookup_device(self, step: int, layer: int, ids, slots_out=None, stream=None):
        """Device lookup (MOE_CACHE_DEVICE): enqueues the lookup of device int32 ids and its fills; slots_out
        (device int32, optional) receives each id's slot."""
        import torch
        _check(lib().expert_cache_lookup_device(self._h, step, layer, _dev(ids, "ids", torch.int32), ids.numel(),
                                                _dev(slots_out, "slots_out", torch.int32), _stream(stream)),
               "expert_cache_lookup_device")

    def prefetch_device(self, step: int, layer: int, ids, stream=None):
        """Device prefetch (MOE_CACHE_DEVICE): decisions on `stream`, fills on the cache's copy stream."""
        import torch
        _check(lib().expert_cache_prefetch_device(self._h, step, layer, _dev(ids, "ids", torch.int32), ids.numel(),
                                                  _stream(stream)), "expert_cache_prefetch_device")

    def prefetch(self, step: int, layer: int, ids):
        a = np.ascontiguousarray(np.asarray(ids).reshape(-1), dtype=np.int32)
        _check(lib().expert_cache_prefetch(self._h, step, layer, a.ctypes.data, a.size), "expert_cache_prefetch")

    def release(self, stream=None):
        _check(lib().expert_cache_release(self._h, None if self.host_sim else _stream(stream)),
               "expert_cache_release")

    def slot_table(self):
        """(slot table address, pool address) as integers."""
        t, p = C.c_void_p(), C.c_void_p()
        _check(lib().expert_cache_slot_table(self._h, C.byref(t), C.byref(p)), "expert_cache_slot_table")
        return t.value, p.value

    def stats(self) -> dict:
        st = CacheStats()
        _check(lib().expert_cache_stats(self._h, C.byref(st)), "expert_cache_stats")
        return {f: getattr(st, f) for f, _ in CacheStats._fields_}

    def trace(self, first: int = 0, cap: int | None = None) -> np.ndarray:
        out = []
        while True:
            n_want = 1 << 16 if cap is None else cap - sum(len(o) for o in out)
            if n_want <= 0:
                break
            buf = np.empty(n_want, EVENT_DTYPE)
            n = C.c_size_t()
            _check(lib().expert_cache_trace(self._h, first, buf.ctypes.data, n_want, C.byref(n)),
                   "expert_cache_trace")
            out.append(buf[:n.value])
            first += n.value
            if n.value < n_want:
                break
        return np.concatenate(out) if out else np.empty(0, EVENT_DTYPE)


class MoeStack:
    """Owner of one moe_stack (decode steps and prefill chunks over L MoE layers on a cache)."""

    def __init__(self, cache: ExpertCache, H: int, I: int, E: int, k: int, w_dtype: int, router_dtype: int,
                 router_w: list, shared_w: list | None = None, max_tokens: int = 1, max_prefill_tokens: int = 0,
                 prefetch: int = 0, recall: int = 0, recall_overlap: int = 0, attention: dict | None = None,
                 host_threads: int = 0):
        self._router = (C.c_void_p * len(router_w))(*[_dev(w, "router_w") for w in router_w])
        self._shared = None
        if shared_w is not None:
            self._shared = (C.c_void_p * len(shared_w))(*[_dev(w, "shared_w") for w in shared_w])
        self._keep = (router_w, shared_w, cache)
        att = None
        if attention is not None:  # dict: n_heads, n_kv, head_dim, max_pos, theta, start_pos, w_qkv, w_o, k_cache, v_cache
            arr = lambda ts, nm: (C.c_void_p * len(ts))(*[_dev(t, nm) for t in ts])
            self._att_arrays = [arr(attention[nm], nm) for nm in ("w_qkv", "w_o", "k_cache", "v_cache")]
            att = AttentionDesc(attention["n_heads"], attention["n_kv"], attention["head_dim"], attention["max_pos"],
                                attention.get("theta", 1.0e6), attention.get("start_pos", 0),
                                *[C.cast(a, C.POINTER(C.c_void_p)) for a in self._att_arrays])
            self._att = att
            self._keep = self._keep + (attention,)
        d = StackDesc(len(router_w), H, I, E, k, w_dtype, router_dtype,
                      C.cast(self._router, C.POINTER(C.c_void_p)),
                      C.cast(self._shared, C.POINTER(C.c_void_p)) if self._shared is not None else None,
                      cache.handle, max_tokens, max_prefill_tokens, prefetch, recall, recall_overlap,
                      C.pointer(att) if att is not None else None, host_threads)
        h = C.c_void_p()
        _check(lib().moe_stack_create(C.byref(d), C.byref(h)), "moe_stack_create")
        self._h = h
        self.L, self.E, self.k = len(router_w), E, k

    def close(self):
        if getattr(self, "_h", None):
            lib().moe_stack_destroy(self._h)
            self._h = None

    __del__ = close

    def decode_step(self, step: int, x, logit_bias=None, ids_out=None, weights_out=None, logits_out=None,
                    stream=None):
        """x <- x + MoE_l(x) over every layer, in place on the device tensor x [T x H]."""
        import torch
        T = x.shape[0]
        _check(lib().moe_stack_decode_step(self._h, step, _dev(x, "x", torch.float32), T,
                                           _dev(logit_bias, "logit_bias", torch.float32),
                                           _dev(ids_out, "ids_out", torch.int32),
                                           _dev(weights_out, "weights_out", torch.float32),
                                           _dev(logits_out, "logits_out", torch.float32), _stream(stream)),
               "moe_stack_decode_step")

    def decode_graph(self, step: int, x, logit_bias=None, ids_out=None, weights_out=None, logits_out=None,
                     stream=None):
        """One-token decode step as a replayed HIP graph (device residency); keep the tensors fixed."""
        import torch
        if x.shape[0] != 1:
            raise ValueError("decode_graph takes one token")
        _check(lib().moe_stack_decode_graph(self._h, step, _dev(x, "x", torch.float32),
                                            _dev(logit_bias, "logit_bias", torch.float32),
                                            _dev(ids_out, "ids_out", torch.int32),
                                            _dev(weights_out, "weights_out", torch.float32),
                                            _dev(logits_out, "logits_out", torch.float32), _stream(stream)),
               "moe_stack_decode_graph")
        return x

    def prefill(self, step: int, x, ids_out=None, weights_out=None, logits_out=None, stream=None):
        """Prompt chunk: x <- x + MoE_l(rmsnorm(x)) over every layer, in place on the device tensor x [T x H]."""
        import torch
        T = x.shape[0]
        _check(lib().moe_stack_prefill(self._h, step, _dev(x, "x", torch.float32), T,
                                       _dev(ids_out, "ids_out", torch.int32),
                                       _dev(weights_out, "weights_out", torch.float32),
                                       _dev(logits_out, "logits_out", torch.float32), _stream(stream)),
               "moe_stack_prefill")
        return x

    def kernel_time(self, which: int, n: int = 200, stream=None) -> float:
        """Mean ms of one launch of kernel `which` (0 route, 1 gate/up, 2 down, 3 the whole expert FFN as
        the decode step issues it, 4 attention), each layer's launch of the last step replayed n times from a
        graph (repeated to at least 32 launches; a stack without a budget rotates the repeats' experts unless
        8 is added to `which`)."""
        ms = C.c_double()
        _check(lib().moe_stack_kernel_time(self._h, which, n, _stream(stream), C.byref(ms)), "moe_stack_kernel_time")
        return ms.value


class PinnedBuffer:
    """Page-locked host memory from hipHostMalloc, viewed as a numpy uint8 array.

    The expert store must be pinned for asynchronous host-to-device fills.  (A
    torch pinned tensor would round a 48 GB request up to a power of two.)"""

    def __init__(self, nbytes: int):
        hip = C.CDLL("libamdhip64.so")
        hip.hipHostMalloc.argtypes = [C.POINTER(C.c_void_p), C.c_size_t, C.c_uint]
        hip.hipHostMalloc.restype = C.c_int
        hip.hipHostFree.argtypes = [C.c_void_p]
        hip.hipHostFree.restype = C.c_int
        self._hip = hip
        p = C.c_void_p()
        rc = hip.hipHostMalloc(C.byref(p), max(1, nbytes), 0)
        if rc != 0 or not p.value:
            raise MemoryError(f"hipHostMalloc({nbytes}) failed with {rc}")
        self.ptr = p.value
        self.nbytes = nbytes
        self.array = np.ctypeslib.as_array((C.c_uint8 * max(1, nbytes)).from_address(self.ptr))[:nbytes]

    def close(self):
        if getattr(self, "ptr", None):
            self.array = None
            self._hip.hipHostFree(self.ptr)
            self.ptr = None

    __del__ = close
