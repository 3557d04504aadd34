"""Seeded synthetic inputs shared by the CPU oracle, the tests and the benchmark.

This module produces *inputs only*: random bits, uniforms, normals and integer
labels, keyed by (seed, virtual worker, minibatch, tensor id).  It contains no
part of the training method's arithmetic.  Both sides of every parity test
consume the arrays it returns, so they see identical bits.

Generator (counter based, every element computed independently):
  * SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
    generators", OOPSLA 2014): z = x + 0x9E3779B97F4A7C15;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9; z = (z ^ (z >> 27)) * 0x94D049BB133111EB;
    return z ^ (z >> 31).
  * A stream key is SplitMix64 chained over (seed, vw, minibatch, tensor_id).
  * Element i of a stream is SplitMix64(key + i * 0x9E3779B97F4A7C15).
  * Uniform in (0, 1): ((bits >> 11) + 0.5) * 2**-53.
  * Normal: Box-Muller on uniforms (2i, 2i+1): sqrt(-2 ln u1) * cos(2 pi u2) and
    the matching sin term for odd outputs.
  * Labels: floor(u * classes).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "stream_key", "bits", "uniform", "normal", "labels",
    "T_X", "T_Y", "T_DY", "T_LABELS", "T_W0", "T_PROBE",
]

# tensor ids used throughout the repository
T_X = 1        # stage input activations / images
T_DY = 2       # upstream gradient at the stage output
T_LABELS = 3   # class labels for a loss head
T_W0 = 4       # initial weights (layer index is folded in by the caller)
T_Y = 5        # auxiliary per-test tensors
T_PROBE = 6    # probes for identities (adjoint tests and the like)

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_MASK = (1 << 64) - 1


def _mix_scalar(x: int) -> int:
    z = (x + 0x9E3779B97F4A7C15) & _MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def stream_key(seed: int, vw: int, minibatch: int, tensor_id: int) -> int:
    """64-bit key of one stream: SplitMix64 chained over the four integers."""
    k = _mix_scalar(seed & _MASK)
    for v in (vw, minibatch, tensor_id):
        k = _mix_scalar((k ^ (v & _MASK)) & _MASK)
    return k


def bits(key: int, n: int, offset: int = 0) -> np.ndarray:
    """n raw 64-bit outputs (elements offset .. offset+n-1) of the stream `key`."""
    with np.errstate(over="ignore"):
        i = np.arange(offset, offset + n, dtype=np.uint64)
        x = np.uint64(key) + i * _GOLDEN
        z = x + _GOLDEN
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def uniform(key: int, n: int, offset: int = 0) -> np.ndarray:
    """n uniforms in the open interval (0, 1) as float64."""
    b = bits(key, n, offset)
    return ((b >> np.uint64(11)).astype(np.float64) + 0.5) * (2.0 ** -53)


def normal(key: int, n: int, std: float = 1.0, dtype=np.float32) -> np.ndarray:
    """n normals N(0, std^2), Box-Muller on consecutive uniform pairs."""
    m = (n + 1) // 2
    u = uniform(key, 2 * m)
    u1, u2 = u[0::2], u[1::2]
    r = np.sqrt(-2.0 * np.log(u1))
    out = np.empty(2 * m, dtype=np.float64)
    out[0::2] = r * np.cos(2.0 * np.pi * u2)
    out[1::2] = r * np.sin(2.0 * np.pi * u2)
    out = out[:n]
    if std != 1.0:
        out *= std
    return out.astype(dtype, copy=False)


def labels(key: int, n: int, classes: int) -> np.ndarray:
    """n integer labels, uniform over [0, classes), as int32."""
    u = uniform(key, n)
    lab = np.floor(u * classes).astype(np.int64)
    np.minimum(lab, classes - 1, out=lab)
    return lab.astype(np.int32)


def initial_weights(segments, seed: int) -> np.ndarray:
    """Initial flat weight vector from a list of parameter segments.

    ``segments`` lists (kind, count, fan_in) in flat-vector order, kind one of
    "w" (He-normal: N(0, 2/fan_in)), "b" / "beta" (zeros), "gamma" (ones).
    Segment i of kind "w" draws from stream (seed, 0, i, T_W0)."""
    parts = []
    for i, (kind, count, fan_in) in enumerate(segments):
        if kind == "w":
            std = float(np.sqrt(2.0 / fan_in))
            parts.append(normal(stream_key(seed, 0, i, T_W0), count, std))
        elif kind == "gamma":
            parts.append(np.ones(count, np.float32))
        else:
            parts.append(np.zeros(count, np.float32))
    return np.concatenate(parts) if parts else np.zeros(0, np.float32)
