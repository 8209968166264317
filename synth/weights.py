"""Seeded weight and prompt generation.

Recipe (fixed, documented, reproducible for any thread count):
  * Tensors are produced in the order given by ``tensor_names``.
  * A matrix with n elements is drawn in chunks of CHUNK elements; chunk c of
    tensor i uses ``numpy.random.default_rng([seed, i, c])`` and
    ``standard_normal(dtype=float32)``, scaled by init_std (0.02) in fp32.
  * Readout matrices are the identity plus that noise (the fitting procedure's
    starting point, identity and zero offset, plus a perturbation).
  * bf16 storage keeps the top 16 bits of the fp32 value after
    round-to-nearest-even; arrays of dtype uint16 carry those bit patterns.
  * RMSNorm gains are one, the final norm gain is ``final_norm_gain``; readout
    offsets are zero. Gains and offsets are always fp32.
Matrices are canonical [out, in] row-major.
"""
from concurrent.futures import ThreadPoolExecutor
import os

import numpy as np

from .configs import ModelConfig

CHUNK = 1 << 22


def tensor_names(cfg: ModelConfig):
    names = ["embed"]
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        names += [p + "attn_norm", p + "wq", p + "wk", p + "wv", p + "wo",
                  p + "mlp_norm", p + "w_gate", p + "w_up", p + "w_down"]
    names.append("final_norm")
    for L in cfg.readout_layers:
        names += [f"readout.{L}.w", f"readout.{L}.b"]
    return names


def tensor_shape(cfg: ModelConfig, name: str):
    H, A, K, D, F, V = (cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                        cfg.ffn, cfg.vocab)
    leaf = name.split(".")[-1]
    if name == "embed":
        return (V, H)
    if leaf in ("attn_norm", "mlp_norm") or name == "final_norm" or leaf == "b":
        return (H,)
    return {"wq": (A * D, H), "wk": (K * D, H), "wv": (K * D, H), "wo": (H, A * D),
            "w_gate": (F, H), "w_up": (F, H), "w_down": (H, F), "w": (H, H)}[leaf]


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """fp32 array -> uint16 bf16 bit patterns, round to nearest, ties to even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def _fill_chunk(out, flat_out_is_bf16, seed, idx, c, n, std, add_identity_cols):
    lo = c * CHUNK
    hi = min(n, lo + CHUNK)
    rng = np.random.default_rng([seed, idx, c])
    v = rng.standard_normal(hi - lo, dtype=np.float32)
    v *= np.float32(std)
    if add_identity_cols:
        # identity entries of an [H, H] matrix sit at flat positions k*(H+1)
        H = add_identity_cols
        first = (lo + H) // (H + 1) * (H + 1)
        pos = np.arange(first, hi, H + 1, dtype=np.int64)
        v[pos - lo] += np.float32(1.0)
    if flat_out_is_bf16:
        out[lo:hi] = bf16_bits_from_f32(v)
    else:
        out[lo:hi] = v


def generate_weights(cfg: ModelConfig, seed: int | None = None, threads: int | None = None):
    """Return {name: ndarray}. Matrices are uint16 (bf16 bits) or float32; gains fp32."""
    seed = cfg.seed if seed is None else seed
    threads = threads or min(16, len(os.sched_getaffinity(0)))
    out = {}
    jobs = []
    for idx, name in enumerate(tensor_names(cfg)):
        shape = tensor_shape(cfg, name)
        leaf = name.split(".")[-1]
        if len(shape) == 1:
            if name == "final_norm":
                out[name] = np.full(shape, cfg.final_norm_gain, dtype=np.float32)
            elif leaf == "b":
                out[name] = np.zeros(shape, dtype=np.float32)
            else:
                out[name] = np.ones(shape, dtype=np.float32)
            continue
        is_bf16 = cfg.wdtype == "bf16"
        arr = np.empty(shape, dtype=np.uint16 if is_bf16 else np.float32)
        flat = arr.reshape(-1)
        n = flat.size
        ident = cfg.hidden if leaf == "w" else 0
        for c in range((n + CHUNK - 1) // CHUNK):
            jobs.append((flat, is_bf16, seed, idx, c, n, cfg.init_std, ident))
        out[name] = arr
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(lambda j: _fill_chunk(*j), jobs))
    return out


def prompts(cfg: ModelConfig, seed: int, length: int) -> np.ndarray:
    """Uniform-random token ids in [0, V)."""
    return np.random.default_rng(seed).integers(0, cfg.vocab, length, dtype=np.int64).astype(np.int32)
