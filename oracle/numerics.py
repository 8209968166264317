"""Elementary operations of the oracle, in fp64.

Readings (the paper fixes none of these; the synthetic decoders follow the
common dense-decoder design whose costs Appendix C counts):
  * RMSNorm: y = x / sqrt(mean(x^2) + eps) * g, eps = 1e-6.
  * RoPE: rotate-half pairing (i, i + D/2), angle pos * base^(-2i/D), base 1e4.
  * Storage rounding: cache entries are stored in the weight storage type; bf16
    is round-to-nearest-even to 8 significant bits, applied to the exact value.
"""
import numpy as np


def round_to_storage(x: np.ndarray, wdtype: str) -> np.ndarray:
    """Round fp64 values to the cache storage type and return them as fp64."""
    x = np.asarray(x, dtype=np.float64)
    if wdtype == "f32":
        return x.astype(np.float32).astype(np.float64)
    if wdtype != "bf16":
        raise ValueError(wdtype)
    # x = m * 2**e with 0.5 <= |m| < 1; bf16 keeps 8 significant bits, and its
    # smallest step (subnormal range) is 2**-133. Scaling by a power of two is exact.
    _, e = np.frexp(x)
    q = np.ldexp(1.0, np.maximum(e - 8, -133))
    return np.rint(x / q) * q


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns (uint16)."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x: np.ndarray, pos, base: float) -> np.ndarray:
    """Rotate-half rotary embedding of x[..., heads, D] at integer position(s) pos.

    pos is a scalar or an array broadcastable to x.shape[:-2]."""
    D = x.shape[-1]
    half = D // 2
    inv = base ** (-(2.0 * np.arange(half, dtype=np.float64)) / D)
    ang = np.asarray(pos, dtype=np.float64)[..., None, None] * inv
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def head_stats(logits: np.ndarray):
    """(argmax with lowest index on ties, max softmax probability, top-1 minus top-2 gap).

    The confidence is the softmax probability of the best token at temperature
    one (Section 2 "Confidence gate"; Section 10 names it the probability of
    the best token)."""
    j = int(np.argmax(logits))            # numpy returns the first maximum
    m = logits[j]
    conf = 1.0 / float(np.sum(np.exp(logits - m)))
    gap = float(m - np.partition(logits, -2)[-2]) if logits.size > 1 else np.inf
    return j, conf, gap


MEASURES = ("maxprob", "margin", "negentropy")


def confidence_measures(logits: np.ndarray) -> dict:
    """The three softmax confidence measures the paper compares (Section 10:
    probability of the best token, margin between the best and second-best
    probabilities, negative entropy of the distribution), at temperature one,
    in fp64:
      maxprob    = p_(1)
      margin     = p_(1) - p_(2)            (0 when the two best tie)
      negentropy = sum_i p_i log p_i        (<= 0; 0 log 0 = 0)
    """
    x = np.asarray(logits, dtype=np.float64)
    p = np.exp(x - x.max())
    p /= p.sum()
    top = np.sort(p)[::-1]
    nz = p[p > 0]
    return {"maxprob": float(top[0]),
            "margin": float(top[0] - top[1]) if p.size > 1 else float(top[0]),
            "negentropy": float(np.sum(nz * np.log(nz)))}

