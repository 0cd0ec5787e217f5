"""Test-side helpers: build and decode expert blobs with plain numpy.

Independent of both the oracle's C and the HIP library: the tests use these
to construct hand-made weights and to evaluate experts densely.
"""
import numpy as np

import synth


def make_blob(gu: np.ndarray, d: np.ndarray, dtype: int) -> np.ndarray:
    """Blob from dense fp32 matrices W_gu [2I x H] (interleaved rows) and W_d [H x I].

    bf16 stores the RNE-rounded values; int4 uses the fixture quantizer."""
    gu = np.ascontiguousarray(gu, np.float32)
    d = np.ascontiguousarray(d, np.float32)
    if dtype == synth.F32:
        return np.concatenate([gu.view(np.uint8).ravel(), d.view(np.uint8).ravel()])
    if dtype == synth.BF16:
        return np.concatenate([synth.bf16_bits(gu).view(np.uint8).ravel(),
                               synth.bf16_bits(d).view(np.uint8).ravel()])
    parts = []
    for m in (gu, d):
        q, s = synth.quantize_int4g128(m.ravel())
        parts += [q, s.view(np.uint8)]
    return np.concatenate(parts)


def decode_blob(blob: np.ndarray, H: int, I: int, dtype: int):
    """Dense float64 (W_gu [2I x H], W_d [H x I]) of a blob."""
    lay = synth.blob_layout(H, I, dtype)
    b = np.ascontiguousarray(blob, np.uint8)
    out = []
    for name, (rows, cols) in (("gu", (2 * I, H)), ("d", (H, I))):
        if dtype in (synth.F32, synth.BF16):
            o, _, n = lay[name]
            raw = b[o:o + n]
            m = raw.view(np.float32) if dtype == synth.F32 else synth.bf16_to_f32(raw.view(np.uint16))
            out.append(m.astype(np.float64).reshape(rows, cols))
        else:
            oq, _, nq = lay[name + "_q"]
            os_, _, ns = lay[name + "_s"]
            q = synth.unpack_int4(b[oq:oq + nq]).astype(np.float64).reshape(rows, cols)
            s = synth.bf16_to_f32(b[os_:os_ + ns].view(np.uint16)).astype(np.float64).reshape(rows, cols // 128)
            out.append(q * np.repeat(s, 128, axis=1))
    return out[0], out[1]


def swiglu_dense(x: np.ndarray, gu: np.ndarray, d: np.ndarray) -> np.ndarray:
    """SwiGLU expert on rows of x (float64): W_d (silu(W_g x) * W_u x)."""
    x = np.asarray(x, np.float64)
    g = x @ gu[0::2].T
    u = x @ gu[1::2].T
    a = g / (1.0 + np.exp(-g)) * u
    return a @ d.T
