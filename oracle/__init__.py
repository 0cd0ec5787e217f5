"""CPU oracle for the MoE decode step under an expert budget -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  The arithmetic lives in ``moe_oracle.c`` and
``attention_oracle.c`` (plain C, fp64); this module builds them with gcc and
marshals numpy arrays into them.
It shares no code with the HIP library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
_SRCS = [_SRC, os.path.join(_HERE, "attention_oracle.c")]
_LIB = os.path.join(_HERE, "libmoe_oracle.so")

F32, BF16, INT4G128 = 0, 1, 2
OK, ERR_ARG, ERR_RANGE, ERR_NONFINITE, ERR_BUDGET = 0, -1, -2, -3, -4
HIT, MISS, PREFETCH, HOST = 0, 1, 2, 3

EVENT_DTYPE = np.dtype([("t", "<i4"), ("layer", "<i4"), ("expert", "<i4"),
                        ("kind", "<i4"), ("slot", "<i4"), ("victim_key", "<i4")])


def build() -> str:
    """Compile ``libmoe_oracle.so`` (gcc -O2, OpenMP over output rows)."""
    tmp = _LIB + ".tmp"
    subprocess.run(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
                    "-o", tmp, *_SRCS, "-lm"], check=True)
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < max(os.path.getmtime(f) for f in _SRCS):
            build()
        _lib = C.CDLL(_LIB)
        P, I32, SZ, D = C.c_void_p, C.c_int, C.c_size_t, C.POINTER(C.c_double)
        _lib.oracle_rmsnorm.argtypes = [P, I32, I32, C.c_double, P]
        _lib.oracle_router_logits.argtypes = [P, P, I32, I32, I32, I32, P]
        _lib.oracle_topk_softmax.argtypes = [P, I32, I32, I32, P, P]
        _lib.oracle_expert_forward.argtypes = [P, I32, I32, P, I32, P]
        _lib.oracle_moe_ffn.argtypes = [P, I32, I32, I32, I32, I32, P, P, P, SZ, I32, P, P]
        _lib.oracle_expert_bytes.argtypes = [I32, I32, I32]
        _lib.oracle_expert_bytes.restype = SZ
        _lib.oracle_expert_weight.argtypes = [P, I32, I32, I32, I32, I32, I32]
        _lib.oracle_expert_weight.restype = C.c_double
        _lib.oracle_lru_new.argtypes = [I32, I32, I32, I32]
        _lib.oracle_lru_new.restype = P
        _lib.oracle_rotary_new.argtypes = [I32, I32, I32, I32, I32]
        _lib.oracle_rope.argtypes = [P, I32, I32, C.c_double]
        _lib.oracle_rope.restype = None
        _lib.oracle_attention_decode.argtypes = [P, I32, I32, I32, I32, P, P, P, P, I32, I32, C.c_double,
                                                 C.c_double, P]
        _lib.oracle_rotary_new.restype = P
        _lib.oracle_lru_free.argtypes = [P]
        _lib.oracle_lru_lookup.argtypes = [P, I32, I32, P, I32, I32]
        _lib.oracle_lru_n_events.argtypes = [P]
        _lib.oracle_lru_n_events.restype = SZ
        _lib.oracle_lru_events.argtypes = [P, SZ, P, SZ]
        _lib.oracle_lru_events.restype = SZ
        _lib.oracle_lru_stats.argtypes = [P, P]
        _lib.oracle_lru_slot_of.argtypes = [P, I32, I32]
        _lib.oracle_lru_occupancy.argtypes = [P]
        _lib.oracle_opt_misses.argtypes = [P, P, I32, I32, I32]
        _lib.oracle_opt_misses.restype = C.c_longlong
        del D
    return _lib


def _p(a: np.ndarray) -> int:
    return a.ctypes.data


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def threads_used() -> int:
    """OpenMP threads the oracle's parallel loops run on (OpenMP's own count, as set or defaulted)."""
    return int(lib().omp_get_max_threads())


def set_threads(n: int) -> None:
    """Run the oracle's parallel loops on n threads from now on (OpenMP's omp_set_num_threads); the results
    do not depend on it, since every output row is summed by one thread in a fixed order."""
    lib().omp_set_num_threads(C.c_int(int(n)))


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), for reporting the oracle's timings."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def expert_bytes(H: int, I: int, dtype: int) -> int:
    return int(lib().oracle_expert_bytes(H, I, dtype))


def expert_weight(blob: np.ndarray, H: int, I: int, dtype: int, which: str, r: int, c: int) -> float:
    """Dequantised weight (r, c) of matrix ``which`` ('gu' or 'd') of an expert blob."""
    b = _c(blob, np.uint8)
    return float(lib().oracle_expert_weight(_p(b), dtype, H, I, 0 if which == "gu" else 1, r, c))


RMS_EPS = 1e-6


def rmsnorm(x: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    """fp64 ``x / sqrt(mean(x^2) + eps)`` per row of fp32 ``x [T x H]``."""
    x = _c(np.atleast_2d(x), np.float32)
    T, H = x.shape
    h = np.empty((T, H), dtype=np.float64)
    st = lib().oracle_rmsnorm(_p(x), T, H, eps, _p(h))
    if st != OK:
        raise ValueError(f"oracle_rmsnorm status {st}")
    return h


def router_logits(x: np.ndarray, w_router: np.ndarray, w_dtype: int) -> np.ndarray:
    """fp64 logits ``[T x E]`` of fp32 ``x [T x H]`` against ``w_router [E x H]`` (f32 or bf16 bits)."""
    x = _c(x, np.float32)
    w = _c(w_router, np.float32 if w_dtype == F32 else np.uint16)
    T, H = x.shape
    E = w.shape[0]
    z = np.empty((T, E), dtype=np.float64)
    st = lib().oracle_router_logits(_p(x), _p(w), w_dtype, T, H, E, _p(z))
    if st != OK:
        raise ValueError(f"oracle_router_logits status {st}")
    return z


def topk_softmax(z: np.ndarray, k: int):
    """Top-k ids (rank order) and fp64 softmax weights of fp32 logits ``z [T x E]``.

    Returns (ids int32 [T x k], weights float64 [T x k], status)."""
    z = _c(z, np.float32)
    T, E = z.shape
    ids = np.empty((T, k), dtype=np.int32)
    w = np.empty((T, k), dtype=np.float64)
    st = lib().oracle_topk_softmax(_p(z), T, E, k, _p(ids), _p(w))
    return ids, w, st


def expert_forward(x: np.ndarray, blob: np.ndarray, H: int, I: int, dtype: int) -> np.ndarray:
    x = _c(x, np.float32).reshape(H)
    b = _c(blob, np.uint8)
    y = np.empty(H, dtype=np.float64)
    st = lib().oracle_expert_forward(_p(x), H, I, _p(b), dtype, _p(y))
    if st != OK:
        raise ValueError(f"oracle_expert_forward status {st}")
    return y


def moe_ffn(x: np.ndarray, ids: np.ndarray, w: np.ndarray, experts: np.ndarray, H: int, I: int,
            dtype: int, shared: np.ndarray | None = None) -> np.ndarray:
    """fp64 ``y [T x H]`` = weighted sum of the selected experts (+ shared expert).

    ``experts`` is ``[E x expert_bytes]`` uint8 (one blob per routed expert)."""
    x = _c(x, np.float32)
    T = x.shape[0]
    ids = _c(ids, np.int32).reshape(T, -1)
    k = ids.shape[1]
    w = _c(w, np.float64).reshape(T, k)
    ex = np.ascontiguousarray(experts, dtype=np.uint8)
    E, stride = ex.shape
    sh = None if shared is None else _c(shared, np.uint8)
    y = np.empty((T, H), dtype=np.float64)
    st = lib().oracle_moe_ffn(_p(x), T, H, I, E, k, _p(ids), _p(w), _p(ex), stride, dtype,
                              None if sh is None else _p(sh), _p(y))
    if st != OK:
        raise ValueError(f"oracle_moe_ffn status {st}")
    return y


class LRU:
    """LRU expert-slot table (the oracle's residency state machine)."""

    def __init__(self, capacity: int, L: int, E: int, preload: bool = False):
        self._h = lib().oracle_lru_new(capacity, L, E, int(preload))
        if not self._h:
            raise ValueError("oracle_lru_new: invalid arguments")
        self.C, self.L, self.E = capacity, L, E


    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h:
            lib().oracle_lru_free(h)

    def lookup(self, t: int, layer: int, ids, prefetch: bool = False) -> int:
        a = _c(np.atleast_1d(ids), np.int32)
        return lib().oracle_lru_lookup(self._h, t, layer, _p(a), a.size, int(prefetch))

    def events(self, first: int = 0) -> np.ndarray:
        n = int(lib().oracle_lru_n_events(self._h))
        out = np.empty(max(0, n - first), dtype=EVENT_DTYPE)
        if out.size:
            lib().oracle_lru_events(self._h, first, _p(out), out.size)
        return out

    def stats(self) -> dict:
        s = np.zeros(4, dtype=np.uint64)
        lib().oracle_lru_stats(self._h, _p(s))
        return dict(hits=int(s[0]), misses=int(s[1]), prefetches=int(s[2]), evictions=int(s[3]))

    def slot_of(self, layer: int, expert: int) -> int:
        return int(lib().oracle_lru_slot_of(self._h, layer, expert))

    def occupancy(self) -> int:
        return int(lib().oracle_lru_occupancy(self._h))


class Rotary(LRU):
    """Rotary slot group (paper sec. 4, Figs. 1-2): slots on a ring swept by a hand; hits charge their slot
    (up to charge_max), a miss rotates the hand forward past the step's own slots and charged slots (each
    giving up one charge) to the first uncharged slot.  charge_max = 0 is cyclic (FIFO) replacement."""

    def __init__(self, capacity: int, L: int, E: int, charge_max: int, preload: bool = False):
        self._h = lib().oracle_rotary_new(capacity, L, E, charge_max, int(preload))
        if not self._h:
            raise ValueError("oracle_rotary_new: invalid arguments")
        self.C, self.L, self.E = capacity, L, E

class HostTier:
    """A slot table with a host tier (the paper's run recipe keeps the experts of some layers in host memory
    and computes them on host cores, sec. 6 and Fig. 3; this is the rule the library's cache applies, which
    the paper leaves open).  Each demand lookup of a step's experts R (ascending, distinct) at layer l:

    1. an id outside [0, E) is a range error, a step needing more experts than there are slots a budget
       error; either changes nothing;
    2. the host's share: all of R when l < host_layers; otherwise, of the experts of R that hold no slot,
       first those the host served at layer l's previous demand lookup, then the others in ascending order
       while the share is smaller than host_quota;
    3. the rest of R goes through the slot table's own policy (the LRU or rotary object `table`), exactly as
       a lookup of that subset; the host's share takes no slot and no recency stamp;
    4. layer l remembers its share for its next demand lookup.

    Prefetches pass straight to the table.  The decision log is the table's events with one event
    (t, l, e, HOST, -1, -1) per host-served expert, merged in ascending expert order within each lookup."""

    def __init__(self, table: LRU, host_layers: int, host_quota: int):
        self.table, self.N, self.Q = table, int(host_layers), int(host_quota)
        self.prev = [set() for _ in range(table.L)]
        self._log = []
        self._seen = 0  # table events already merged into the log
        self.host = 0

    def _take_table_events(self):
        ev = self.table.events(self._seen)
        self._seen += ev.size
        return ev

    def lookup(self, t: int, layer: int, ids, prefetch: bool = False) -> int:
        R = sorted({int(i) for i in np.atleast_1d(ids)})
        if prefetch:
            st = self.table.lookup(t, layer, np.array(R, np.int32), prefetch=True)
            self._log.extend(self._take_table_events().tolist())
            return st
        if any(e < 0 or e >= self.table.E for e in R):
            return ERR_RANGE
        if len(R) > self.table.C:
            return ERR_BUDGET
        if layer < self.N:
            host = set(R)
        else:
            absent = [e for e in R if self.table.slot_of(layer, e) < 0]
            host = {e for e in absent if e in self.prev[layer]}
            for e in absent:
                if len(host) >= self.Q:
                    break
                host.add(e)
        self.prev[layer] = host
        rest = [e for e in R if e not in host]
        st = self.table.lookup(t, layer, np.array(rest, np.int32)) if rest else OK
        if st != OK:
            return st
        table_ev = {int(ev[2]): tuple(ev) for ev in self._take_table_events().tolist()}
        for e in R:
            self._log.append((t, layer, e, HOST, -1, -1) if e in host else table_ev[e])
        self.host += len(host)
        return OK

    def events(self, first: int = 0) -> np.ndarray:
        return np.array(self._log[first:], dtype=EVENT_DTYPE)

    def stats(self) -> dict:
        return dict(self.table.stats(), host=self.host)

    def slot_of(self, layer: int, expert: int) -> int:
        return self.table.slot_of(layer, expert)


class Recall:
    """Reverse rotation of the slot group (paper sec. 4, Fig. 2: when an earlier context recurs the
    residency returns to the slot set it had).  Our reading: a token's context signature is its layer-0
    expert set (the routing result of its hidden state, Fig. 1); up to `capacity` past tokens are remembered
    with their expert set at every layer.  A token whose signature shares at least `overlap` experts (0 means
    all k) with a remembered one recalls the one sharing the most (ties: the most recently stored), and the
    slot group is asked to bring back that token's set of each later layer.  After the token, it is
    remembered in place of a remembered token with the same signature, else of the oldest."""

    def __init__(self, capacity: int, k: int, overlap: int = 0):
        self.capacity, self.k = capacity, k
        self.need = overlap if overlap else k
        self.snaps = []   # [signature (frozenset), per-layer sets, order stored, token]
        self.n = 0

    def step(self, t: int, sets):
        """Token t's expert sets per layer (lists of k ids).  Returns (recalled token or -1, [(layer, ids)]
        for layers 1..L-1), then remembers token t."""
        s0 = frozenset(int(e) for e in sets[0])
        best, best_n = None, -1
        for snap in self.snaps:
            n = len(s0 & snap[0])
            if n >= self.need and (n > best_n or (n == best_n and snap[2] > best[2])):
                best, best_n = snap, n
        calls = [] if best is None else [(l, list(best[1][l])) for l in range(1, len(sets))]
        self.n += 1
        new = [s0, [[int(e) for e in st] for st in sets], self.n, t]
        for i, snap in enumerate(self.snaps):
            if snap[0] == s0:
                self.snaps[i] = new
                break
        else:
            if len(self.snaps) < self.capacity:
                self.snaps.append(new)
            else:
                i = min(range(len(self.snaps)), key=lambda j: self.snaps[j][2])
                self.snaps[i] = new
        return (-1 if best is None else best[3]), calls


def replay_decode(cache, token_sets, recall: Recall | None = None):
    """Drive an oracle slot table (LRU or Rotary) the way one-token decode does: per token, per layer, the
    demand lookup of that layer's set, then (with recall) the prefetch of the recalled next-layer set."""
    for t, sets in enumerate(token_sets):
        calls = dict(recall.step(t, sets)[1]) if recall is not None else {}
        for l, ids in enumerate(sets):
            cache.lookup(t, l, ids)
            if l + 1 in calls:
                cache.lookup(t, l + 1, calls[l + 1], prefetch=True)
    return cache


ROPE_THETA = 1.0e6


def rope(v: np.ndarray, p: int, theta: float = ROPE_THETA) -> np.ndarray:
    """Rotary position embedding (rotate-half form) of fp64 head vector(s) ``v [..., d]`` at position p."""
    out = np.array(v, dtype=np.float64, copy=True)
    flat = out.reshape(-1, out.shape[-1])
    for row in flat:
        lib().oracle_rope(_p(row), row.size, p, theta)
    return flat.reshape(out.shape)


def attention_decode(x, w_qkv, w_o, k_cache, v_cache, p: int, n_heads: int, n_kv: int,
                     theta: float = ROPE_THETA, eps: float = RMS_EPS) -> np.ndarray:
    """x + Attn(rmsnorm(x)) for one token at position p; k_cache / v_cache (bf16 bits, uint16
    [n_kv x max_pos x head_dim]) hold positions < p and receive position p in place.  Returns fp64 [H]."""
    x = _c(np.asarray(x).reshape(-1), np.float32)
    H = x.size
    n_kv_, max_pos, d = k_cache.shape
    assert n_kv_ == n_kv and v_cache.shape == k_cache.shape
    assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous and k_cache.dtype == np.uint16
    wq = _c(w_qkv, np.uint16)
    wo = _c(w_o, np.uint16)
    y = np.empty(H, np.float64)
    st = lib().oracle_attention_decode(_p(x), H, n_heads, n_kv, d, _p(wq), _p(wo), _p(k_cache), _p(v_cache),
                                       max_pos, p, theta, eps, _p(y))
    if st != OK:
        raise ValueError(f"oracle_attention_decode status {st}")
    return y

def opt_misses(steps, n_keys: int, capacity: int) -> int:
    """Fewest fills any replacement policy needs for `steps` (a list of arrays of distinct keys, each step's
    keys resident together) with `capacity` slots: Belady's farthest-next-use rule at step granularity.
    Returns -1 if a step needs more than `capacity` keys."""
    keys = np.concatenate([np.asarray(st, np.int32).reshape(-1) for st in steps]) if steps else np.zeros(0, np.int32)
    offsets = np.zeros(len(steps) + 1, np.int32)
    offsets[1:] = np.cumsum([len(np.asarray(st).reshape(-1)) for st in steps])
    keys = np.ascontiguousarray(keys, np.int32)
    return int(lib().oracle_opt_misses(keys.ctypes.data, offsets.ctypes.data, len(steps), n_keys, capacity))
