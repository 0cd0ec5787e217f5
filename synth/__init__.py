"""Seeded synthetic inputs for the MoE decode path (weights, hidden states, routing).

This module is shared by the CPU oracle's tests, the HIP path's tests and the
benchmark.  It holds *input generation only*: random draws, the bf16/int4
storage encodings of the generated weights, and the byte layout of an expert
blob.  None of the method's arithmetic (routing, softmax, SwiGLU, combine,
residency) lives here.

Recipe (every draw comes from NumPy PCG64 keyed by ``SeedSequence(seed,
spawn_key=...)`` so any tensor can be rebuilt on its own):

* Weights.  Every weight tensor of a workload is a window of one stream of
  N(0, sigma_w) draws that repeats with period ``P`` elements
  (``P = min(2**26, total elements rounded up to 128)``).  The tensors are
  enumerated per layer: the router ``[E x H]``, then routed experts 0..E-1
  (each ``W_gu`` then ``W_d``), then the shared expert if the workload has
  one.  When the whole workload fits in one period (small workloads) the
  windows are consecutive, so every draw is independent.  The large stacks
  re-use the stream, which keeps generation of 48 GB host stores to memcpy
  speed; there tensor number q of the enumeration starts at element
  ``128 * ((q * 0x9E3779B1) mod P/128)`` of the stream.  The multiplier is
  odd, so q -> start is a bijection on the P/128 group-aligned starts: no two
  tensors (up to P/128 = 524 288 of them) start at the same place, and no two
  expert blobs are byte-identical.  fp32 draws are stored as fp32, bf16 by
  round-to-nearest-even, int4 by the group-128 symmetric quantizer below.
* Hidden states: fresh N(0, 1) fp32 per decode step (and per token).
* Routing for the Zipf workloads: per layer a seeded permutation maps Zipf
  ranks r = 1..E (p_r proportional to r**-s) to experts; a token's expert set
  is a Plackett-Luce draw without replacement (Gumbel top-k on log p).  With
  overlap q, each expert of the previous step's set at the same layer is kept
  with probability q and the rest is refilled from experts outside that set.
  The set reaches the router as an additive logit mask of +64 on its members.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from functools import lru_cache

import numpy as np

# ---------------------------------------------------------------- dtypes ---
F32, BF16, INT4G128 = 0, 1, 2
DTYPE_NAMES = {F32: "f32", BF16: "bf16", INT4G128: "int4g128"}
GROUP = 128          # int4 quantisation group along the reduction dimension
MASK_LOGIT = 64.0    # additive router mask that realises a drawn expert set
_POOL_MAX = 1 << 26

_KEY_WEIGHTS, _KEY_X, _KEY_ROUTE, _KEY_PREFILL_X = 0, 1, 2, 3


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and recipe of one synthetic MoE workload."""
    name: str
    H: int                 # hidden size
    E: int                 # routed experts per layer
    k: int                 # experts selected per token
    I: int                 # expert intermediate size
    L: int = 1             # layers
    dtype: int = BF16      # expert weight storage type
    router_dtype: int = BF16
    shared: bool = False   # one always-active shared expert per layer (intermediate I)
    T: int = 1             # tokens per decode step
    steps: int = 1
    budget_bytes: int | None = None   # expert-slot HBM budget; None = all resident
    routing: str = "router"           # "router" | "zipf" | "zipf_overlap" | "topics"
    zipf_s: float = 1.1
    overlap: float = 0.7
    topics: int = 4                   # "topics": latent contexts the tokens move between
    topic_stay: float = 0.9           # "topics": chance a token keeps the previous token's context
    topic_keep: float = 0.85          # "topics": chance each expert of the context's profile set is drawn
    prefill: int = 0       # prefill chunk length (tokens); 0 = none
    sigma_w: float = 0.02
    seed: int = 0
    cfg_id: int = 0

    @property
    def expert_bytes(self) -> int:
        return expert_bytes(self.H, self.I, self.dtype)

    @property
    def router_bytes(self) -> int:
        return self.E * self.H * (4 if self.router_dtype == F32 else 2)

    def capacity(self) -> int:
        """Routed-expert slots that fit the budget (shared experts are charged first)."""
        if self.budget_bytes is None:
            return self.L * self.E
        reserved = self.L * self.expert_bytes if self.shared else 0
        return max(0, (self.budget_bytes - reserved) // self.expert_bytes)


GiB = 1 << 30

# The five workloads the method is measured on (shapes of a Qwen-class MoE).
CONFIGS = {
    1: Workload("cfg1: 1 layer fp32 H256 E16 k2 I128, T=1 x 64 steps, all resident",
                H=256, E=16, k=2, I=128, dtype=F32, router_dtype=F32, steps=64, cfg_id=1),
    2: Workload("cfg2: 1 layer bf16 H2048 E128 k8 I768, T=1 x 1000 steps, all resident",
                H=2048, E=128, k=8, I=768, steps=1000, cfg_id=2),
    3: Workload("cfg3: 1 layer bf16 H2048 E256 k8 I512 + shared, Zipf(1.1), T in {1,4,16}",
                H=2048, E=256, k=8, I=512, shared=True, steps=1000, routing="zipf", cfg_id=3),
    4: Workload("cfg4: 40-layer bf16 H2048 E128 k8 I768 decode, 6 GiB LRU budget, Zipf(1.1) 70% overlap",
                H=2048, E=128, k=8, I=768, L=40, steps=2048, budget_bytes=6 * GiB,
                routing="zipf_overlap", cfg_id=4),
    5: Workload("cfg5: 48-layer int4-g128 H2048 E256 k8 I512 + shared, prefill 2048 + 512 decode, 6 GiB",
                H=2048, E=256, k=8, I=512, L=48, dtype=INT4G128, shared=True, steps=512,
                budget_bytes=6 * GiB, routing="zipf_overlap", prefill=2048, cfg_id=5),
}


def workload(cfg: int, **overrides) -> Workload:
    return dataclasses.replace(CONFIGS[cfg], **overrides)


# ---------------------------------------------------------- expert blob ---
def expert_bytes(H: int, I: int, dtype: int) -> int:
    """Bytes of one expert blob ``[W_gu ; W_d]`` (layout in :func:`blob_layout`)."""
    return sum(n for _, _, n in blob_layout(H, I, dtype).values())


def blob_layout(H: int, I: int, dtype: int) -> dict:
    """Byte layout of one expert blob: name -> (offset, row-shape, nbytes).

    * ``gu``: gate/up rows ``[2I x H]`` interleaved (row 2i = gate i, row
      2i+1 = up i), row-major.
    * ``d``: down rows ``[H x I]``, row-major.
    * int4-g128: each matrix is stored as packed nibbles ``[rows x K/2]`` (low
      nibble = even element, two's complement in [-8, 7]) followed by its bf16
      scales ``[rows x K/128]``.
    """
    if H % GROUP or I % GROUP:
        raise ValueError("H and I must be multiples of 128")
    out, off = {}, 0
    if dtype in (F32, BF16):
        es = 4 if dtype == F32 else 2
        for name, rows, cols in (("gu", 2 * I, H), ("d", H, I)):
            n = rows * cols * es
            out[name] = (off, (rows, cols), n)
            off += n
    elif dtype == INT4G128:
        for name, rows, cols in (("gu", 2 * I, H), ("d", H, I)):
            nq = rows * cols // 2
            out[name + "_q"] = (off, (rows, cols // 2), nq)
            off += nq
            ns = rows * (cols // GROUP) * 2
            out[name + "_s"] = (off, (rows, cols // GROUP), ns)
            off += ns
    else:
        raise ValueError(f"unknown dtype {dtype}")
    return out


# ------------------------------------------------------ storage encodings ---
def bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16) by round-to-nearest-even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def quantize_int4g128(w: np.ndarray):
    """Fixture quantizer: symmetric int4 per group of 128 consecutive elements.

    s = bf16_rne(max|w_g| / 7);  q = clamp(rne(w / s), -8, 7);  q = 0 where s = 0.
    Returns (packed uint8 [n/2], scale bits uint16 [n/128]) for a flat fp32 array.
    """
    w = np.ascontiguousarray(w, dtype=np.float32).reshape(-1, GROUP)
    amax = np.abs(w).max(axis=1)
    s_bits = bf16_bits(amax / np.float32(7.0))
    s = bf16_to_f32(s_bits)
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.where(s[:, None] > 0, np.rint(w / s[:, None]), 0.0)
    q = np.clip(q, -8, 7).astype(np.int8).reshape(-1)
    nib = (q.astype(np.uint8) & np.uint8(0xF))
    packed = (nib[0::2] | (nib[1::2] << np.uint8(4))).astype(np.uint8)
    return packed, s_bits


def unpack_int4(packed: np.ndarray) -> np.ndarray:
    """Packed bytes -> int8 values in [-8, 7] (low nibble first)."""
    p = np.asarray(packed, dtype=np.uint8)
    lo = (p & 0xF).astype(np.int8)
    hi = (p >> 4).astype(np.int8)
    lo = np.where(lo > 7, lo - 16, lo).astype(np.int8)
    hi = np.where(hi > 7, hi - 16, hi).astype(np.int8)
    out = np.empty(p.size * 2, dtype=np.int8)
    out[0::2] = lo.reshape(-1)
    out[1::2] = hi.reshape(-1)
    return out


# ------------------------------------------------------------ the stream ---
def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=tuple(key))))


def _elements_per_layer(wl: Workload) -> int:
    n_exp = 3 * wl.I * wl.H
    return wl.E * wl.H + wl.E * n_exp + (n_exp if wl.shared else 0)


def _pool_size(wl: Workload) -> int:
    total = wl.L * _elements_per_layer(wl)
    return min(_POOL_MAX, -(-total // GROUP) * GROUP)


_POOL_CHUNK = 1 << 22


@lru_cache(maxsize=4)
def _pool_f32(seed: int, cfg_id: int, P: int, sigma: float) -> np.ndarray:
    """The periodic N(0, sigma) stream's first period, in chunks of 2**22 drawn in parallel."""
    out = np.empty(P, dtype=np.float32)
    starts = list(range(0, P, _POOL_CHUNK))

    def fill(i_s):
        i, s = i_s
        n = min(_POOL_CHUNK, P - s)
        _rng(seed, cfg_id, _KEY_WEIGHTS, i).standard_normal(n, dtype=np.float32, out=out[s:s + n])

    with ThreadPoolExecutor(8) as ex:
        list(ex.map(fill, enumerate(starts)))
    out *= np.float32(sigma)
    return out


@lru_cache(maxsize=4)
def _pool_enc(seed: int, cfg_id: int, P: int, sigma: float, dtype: int):
    f = _pool_f32(seed, cfg_id, P, sigma)
    if dtype == F32:
        return f
    # encode in chunks of 2**22 elements (whole int4 groups) on a thread pool
    starts = list(range(0, P, _POOL_CHUNK))
    if dtype == BF16:
        out = np.empty(P, dtype=np.uint16)

        def enc(s):
            out[s:s + _POOL_CHUNK] = bf16_bits(f[s:s + _POOL_CHUNK])
    elif dtype == INT4G128:
        out = (np.empty(P // 2, dtype=np.uint8), np.empty(P // GROUP, dtype=np.uint16))

        def enc(s):
            q, sc = quantize_int4g128(f[s:s + _POOL_CHUNK])
            out[0][s // 2:s // 2 + q.size] = q
            out[1][s // GROUP:s // GROUP + sc.size] = sc
    else:
        raise ValueError(dtype)
    with ThreadPoolExecutor(8) as ex:
        list(ex.map(enc, starts))
    return out


def _window(pool: np.ndarray, off: int, n: int, unit: int = 1) -> np.ndarray:
    """Elements [off, off+n) of the periodic extension of ``pool`` (indices in ``unit`` steps)."""
    P = pool.size
    off, n = off // unit, n // unit
    off %= P
    if off + n <= P:
        return pool[off:off + n]
    out = np.empty(n, dtype=pool.dtype)
    i = 0
    while i < n:
        take = min(n - i, P - off)
        out[i:i + take] = pool[off:off + take]
        i += take
        off = 0
    return out


_START_MULT = 0x9E3779B1  # odd: tensor number -> window start is a bijection modulo P/128


def _stream_repeats(wl: Workload) -> bool:
    return wl.L * _elements_per_layer(wl) > _pool_size(wl)


def _tensor_number(wl: Workload, layer: int, which: str, expert: int = 0) -> int:
    """Position of a weight tensor in the enumeration (router, experts 0..E-1, shared) per layer."""
    base = layer * (wl.E + 2)
    if which == "router":
        return base
    if which == "expert":
        if not 0 <= expert < wl.E:
            raise ValueError(f"expert {expert} outside [0, {wl.E})")
        return base + 1 + expert
    if which == "shared":
        return base + 1 + wl.E
    raise ValueError(which)


def _tensor_offset(wl: Workload, layer: int, which: str, expert: int = 0) -> int:
    """Element offset of a weight tensor in the (periodic) stream."""
    if _stream_repeats(wl):
        groups = _pool_size(wl) // GROUP
        q = _tensor_number(wl, layer, which, expert)
        if q >= groups:
            raise ValueError("more tensors than distinct window starts")
        return GROUP * ((q * _START_MULT) % groups)
    base = layer * _elements_per_layer(wl)
    if which == "router":
        return base
    n_exp = 3 * wl.I * wl.H
    base += wl.E * wl.H
    if which == "expert":
        return base + expert * n_exp
    if which == "shared":
        return base + wl.E * n_exp
    raise ValueError(which)


def _encode_window(wl: Workload, dtype: int, off: int, n: int) -> bytes | np.ndarray:
    P = _pool_size(wl)
    pool = _pool_enc(wl.seed, wl.cfg_id, P, wl.sigma_w, dtype)
    if dtype == F32:
        return _window(pool, off, n)
    if dtype == BF16:
        return _window(pool, off, n)
    packed, scales = pool
    return _window(packed, off, n, 2), _window(scales, off, n, GROUP)


def router_weights(wl: Workload, layer: int = 0) -> np.ndarray:
    """Router weights ``[E x H]``: fp32 array, or bf16 bits as uint16."""
    w = _encode_window(wl, wl.router_dtype, _tensor_offset(wl, layer, "router"), wl.E * wl.H)
    return np.array(w).reshape(wl.E, wl.H)


def _blob_parts(wl: Workload, layer: int, expert: int | None, prefix: int | None = None) -> dict:
    """The encoded parts of one expert blob (name in :func:`blob_layout` -> uint8 bytes), or with
    ``prefix`` only the encoding of each matrix's first ``prefix`` elements (a multiple of 128)."""
    off = _tensor_offset(wl, layer, "shared" if expert is None else "expert", expert or 0)
    H, I = wl.H, wl.I
    n_gu = 2 * I * H
    parts = {}
    for name, o, n in (("gu", off, n_gu), ("d", off + n_gu, H * I)):
        if prefix is not None:
            n = min(n, prefix)
        if wl.dtype in (F32, BF16):
            parts[name] = np.asarray(_encode_window(wl, wl.dtype, o, n)).view(np.uint8)
        else:
            q, s = _encode_window(wl, wl.dtype, o, n)
            parts[name + "_q"] = np.asarray(q)
            parts[name + "_s"] = np.asarray(s).view(np.uint8)
    return parts


def expert_blob(wl: Workload, layer: int, expert: int | None) -> np.ndarray:
    """One expert's blob as uint8 bytes.  ``expert=None`` = the layer's shared expert."""
    out = np.empty(wl.expert_bytes, dtype=np.uint8)
    lay = blob_layout(wl.H, wl.I, wl.dtype)
    for name, part in _blob_parts(wl, layer, expert).items():
        b, _, nb = lay[name]
        out[b:b + nb] = part
    return out


def expert_blob_prefixes(wl: Workload, layer: int, expert: int | None, n: int = 4096) -> dict:
    """The first bytes of each part of an expert blob: the encoding of each matrix's first ``n`` elements
    (packed nibbles and scales separately for int4).  Distinct prefixes prove distinct blobs."""
    if n % GROUP:
        raise ValueError("prefix must be a multiple of 128 elements")
    return _blob_parts(wl, layer, expert, prefix=n)


def layer_experts(wl: Workload, layer: int, out: np.ndarray | None = None) -> np.ndarray:
    """All routed experts of a layer as ``[E x expert_bytes]`` uint8 (written into ``out`` if given)."""
    eb = wl.expert_bytes
    if out is None:
        out = np.empty((wl.E, eb), dtype=np.uint8)
    out = out.reshape(wl.E, eb)
    if wl.dtype in (F32, BF16) and not _stream_repeats(wl):
        # consecutive experts are consecutive windows, so the layout of
        # [E x (gu | d)] is one contiguous window of the encoded stream
        off = _tensor_offset(wl, layer, "expert", 0)
        flat = np.asarray(_encode_window(wl, wl.dtype, off, wl.E * 3 * wl.I * wl.H))
        out.reshape(-1)[:] = flat.view(np.uint8)
    else:
        for e in range(wl.E):
            out[e] = expert_blob(wl, layer, e)
    return out


def fill_host_store(wl: Workload, store: np.ndarray, threads: int = 8) -> None:
    """Write every layer's routed experts into ``store`` viewed as ``[L x E x expert_bytes]``."""
    st = store.reshape(wl.L, wl.E * wl.expert_bytes)
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(lambda l: layer_experts(wl, l, st[l]), range(wl.L)))


# ------------------------------------------------------- hidden states ---
def hidden_states(wl: Workload, step: int, T: int | None = None) -> np.ndarray:
    """Decode-step input ``[T x H]`` fp32, N(0, 1), fresh per step."""
    T = wl.T if T is None else T
    return _rng(wl.seed, wl.cfg_id, _KEY_X, T, step).standard_normal((T, wl.H), dtype=np.float32)


def prefill_states(wl: Workload, T: int | None = None) -> np.ndarray:
    T = wl.prefill if T is None else T
    return _rng(wl.seed, wl.cfg_id, _KEY_PREFILL_X, T).standard_normal((T, wl.H), dtype=np.float32)


# ------------------------------------------------------------- routing ---
def zipf_log_probs(wl: Workload, layer: int, rng: np.random.Generator) -> np.ndarray:
    perm = rng.permutation(wl.E)
    ranks = np.empty(wl.E, dtype=np.int64)
    ranks[perm] = np.arange(1, wl.E + 1)
    logp = -wl.zipf_s * np.log(ranks.astype(np.float64))
    return logp - np.log(np.exp(logp).sum())


def _gumbel_topk(scores: np.ndarray, m: int) -> np.ndarray:
    idx = np.argpartition(-scores, m - 1)[:m] if m < scores.size else np.arange(scores.size)
    return np.sort(idx)


def topic_sequence(wl: Workload, steps: int, T: int) -> np.ndarray:
    """Context of each (step, token) for "topics" routing ``[steps x T]``: a Markov chain that keeps the
    previous token's context with probability topic_stay, else moves to one of the others uniformly."""
    rng = _rng(wl.seed, wl.cfg_id, _KEY_ROUTE, 1 << 20)
    z = np.zeros((steps, T), dtype=np.int64)
    for tok in range(T):
        for t in range(1, steps):
            z[t, tok] = z[t - 1, tok]
            if rng.random() >= wl.topic_stay:
                z[t, tok] = (z[t - 1, tok] + 1 + rng.integers(0, wl.topics - 1)) % wl.topics
    return z


def routing_sets(wl: Workload, steps: int | None = None, T: int | None = None) -> np.ndarray:
    """Drawn expert sets ``[steps x L x T x k]`` int32 (ascending ids per set)."""
    steps = wl.steps if steps is None else steps
    T = wl.T if T is None else T
    E, k = wl.E, wl.k
    out = np.empty((steps, wl.L, T, k), dtype=np.int32)
    z = topic_sequence(wl, steps, T) if wl.routing == "topics" else None
    for l in range(wl.L):
        rng = _rng(wl.seed, wl.cfg_id, _KEY_ROUTE, l)
        logp = zipf_log_probs(wl, l, rng)
        if wl.routing == "zipf":
            g = rng.gumbel(size=(steps, T, E))
            sc = logp[None, None, :] + g
            top = np.argpartition(-sc, k - 1, axis=-1)[..., :k]
            out[:, l] = np.sort(top, axis=-1)
        elif wl.routing == "zipf_overlap":
            for tok in range(T):
                prev = None
                for t in range(steps):
                    if prev is None:
                        s = _gumbel_topk(logp + rng.gumbel(size=E), k)
                    else:
                        keep = prev[rng.random(k) < wl.overlap]
                        g = logp + rng.gumbel(size=E)
                        g[prev] = -np.inf
                        s = np.sort(np.concatenate([keep, _gumbel_topk(g, k - keep.size)])) \
                            if keep.size < k else keep
                    out[t, l, tok] = s
                    prev = s
        elif wl.routing == "topics":
            # each context has its own Zipf ranking of the layer's experts and a profile set drawn from it;
            # a token keeps each profile expert with probability topic_keep and refills from its context
            logps = [zipf_log_probs(wl, l, _rng(wl.seed, wl.cfg_id, _KEY_ROUTE, l, c + 1)) for c in range(wl.topics)]
            profile = [_gumbel_topk(lp + rng.gumbel(size=E), k) for lp in logps]
            for tok in range(T):
                for t in range(steps):
                    c = int(z[t, tok])
                    keep = profile[c][rng.random(k) < wl.topic_keep]
                    g = logps[c] + rng.gumbel(size=E)
                    g[profile[c]] = -np.inf
                    out[t, l, tok] = np.sort(np.concatenate([keep, _gumbel_topk(g, k - keep.size)])) \
                        if keep.size < k else keep
        else:
            raise ValueError(f"workload routing {wl.routing!r} draws no sets")
    return out


def mask_logits(wl: Workload, sets: np.ndarray) -> np.ndarray:
    """Additive router mask ``[T x E]`` fp32 for one (step, layer): +64 on each drawn expert."""
    T = sets.shape[0]
    m = np.zeros((T, wl.E), dtype=np.float32)
    m[np.arange(T)[:, None], sets] = MASK_LOGIT
    return m
