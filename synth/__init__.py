"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module holds no arithmetic of the method itself: it only turns seeds into
numbers (weights, prompt ids, group-length schedules).  Both the CPU oracle and
the GPU path consume what it produces; the GPU library also re-implements the
weight generator on the device (``ham_init_weights``) from the same published
definitions, and the tests compare the two.

Definitions (all integer arithmetic is modulo 2**64):

* SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
  generators", OOPSLA 2014; reference C code by S. Vigna): the ``i``-th output
  (0-based) of the stream seeded with ``s`` is ``mix(s + (i + 1) * GAMMA)`` with
  ``GAMMA = 0x9E3779B97F4A7C15`` and the finaliser
  ``z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27; z *= 0x94D049BB133111EB;
  z ^= z >> 31``.  Counter-based by construction: ``sm(s, i)``.
* Tensor keys: ``key = sm(seed, tensor_id)``; element ``i`` of a tensor (row-major
  index in its logical shape) uses ``r1 = sm(key, 2 i)``, ``r2 = sm(key, 2 i + 1)``.
* Normal deviate: Box-Muller, cosine branch (Box and Muller 1958):
  ``u1 = ((r1 >> 11) + 1) * 2**-53`` in (0, 1], ``u2 = (r2 >> 11) * 2**-53`` in
  [0, 1), ``n = sqrt(-2 ln u1) * cos(2 pi u2)`` in float64.  The weight is
  ``fp32(n * 0.02)`` (round to nearest even), then bf16 by round to nearest even
  for bf16 models.  Norm gains are 1 and there are no biases.
* Prompt ids: ``key_b = sm(seed, b)``; ``id = ((sm(key_b, i) >> 32) * V) >> 32``.
* Group-length schedule (a geometric law with p = 1/2, capped at G):
  ``key_b = sm(seed, b)``; ``L(b, s) = min(G, 1 + ctz(sm(key_b, s)))`` with
  ``ctz(0) = 64``.  Step 0 is the group emitted by prefill, step s >= 1 the group
  emitted by the s-th macro-step.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
M1 = 0xBF58476D1CE4E5B9
M2 = 0x94D049BB133111EB
MASK = (1 << 64) - 1

# Tensor identifiers of the generated model (fixed; the device generator uses the
# same numbering).  Per-layer tensors: LAYER_BASE + LAYER_STRIDE * j + t, where
# j counts base layers first (0..L-1) and then micro-decoder layers (L..L+M-1).
T_EMBED, T_RELPOS, T_AQ, T_AK, T_AV, T_AO, T_ALIN, T_LMHEAD, T_STOP = range(9)
LAYER_BASE = 16
LAYER_STRIDE = 8
L_WQ, L_WK, L_WV, L_WO, L_WG, L_WU, L_WD = range(7)

_U64 = np.uint64


def _mix64(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> _U64(30))
    z = z * _U64(M1)
    z = z ^ (z >> _U64(27))
    z = z * _U64(M2)
    return z ^ (z >> _U64(31))


def sm_scalar(seed: int, i: int) -> int:
    """i-th output of the SplitMix64 stream seeded with ``seed`` (Python ints)."""
    z = (seed + (i + 1) * GAMMA) & MASK
    z ^= z >> 30
    z = (z * M1) & MASK
    z ^= z >> 27
    z = (z * M2) & MASK
    return z ^ (z >> 31)


def sm_array(seed: int, idx: np.ndarray) -> np.ndarray:
    """Vectorised ``sm(seed, idx)`` for a uint64 index array."""
    with np.errstate(over="ignore"):
        z = _U64(seed & MASK) + (idx.astype(np.uint64) + _U64(1)) * _U64(GAMMA)
        return _mix64(z)


def tensor_key(seed: int, tensor_id: int) -> int:
    return sm_scalar(seed, tensor_id)


def layer_tensor_id(j: int, t: int) -> int:
    return LAYER_BASE + LAYER_STRIDE * j + t


def _normal_chunk(key: int, i0: int, i1: int) -> np.ndarray:
    i = np.arange(i0, i1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        r1 = sm_array(key, i * _U64(2))
        r2 = sm_array(key, i * _U64(2) + _U64(1))
    u1 = ((r1 >> _U64(11)).astype(np.float64) + 1.0) * (2.0 ** -53)
    u2 = (r2 >> _U64(11)).astype(np.float64) * (2.0 ** -53)
    rad = np.sqrt(-2.0 * np.log(u1))
    ang = (2.0 * np.pi) * u2
    n = rad * np.cos(ang)
    return (n * 0.02).astype(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest even); returns the uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = (b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(u: np.ndarray) -> np.ndarray:
    return (u.astype(np.uint32) << np.uint32(16)).view(np.float32)


_CHUNK = 1 << 21


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def normal_tensor(seed: int, tensor_id: int, count: int, bf16: bool) -> np.ndarray:
    """All ``count`` elements of one generated tensor, in row-major order.

    Returns float32 values, or uint16 bf16 bit patterns when ``bf16`` is set.
    """
    key = tensor_key(seed, tensor_id)
    out = np.empty(count, dtype=np.uint16 if bf16 else np.float32)

    def job(i0: int) -> None:
        i1 = min(count, i0 + _CHUNK)
        v = _normal_chunk(key, i0, i1)
        out[i0:i1] = f32_to_bf16_bits(v) if bf16 else v

    starts = range(0, count, _CHUNK)
    if count > 2 * _CHUNK:
        with ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(job, starts))
    else:
        for s in starts:
            job(s)
    return out


def normal_elements(seed: int, tensor_id: int, idx: np.ndarray, bf16: bool) -> np.ndarray:
    """Selected elements (row-major indices) of one generated tensor."""
    key = tensor_key(seed, tensor_id)
    idx = np.asarray(idx, dtype=np.uint64)
    with np.errstate(over="ignore"):
        r1 = sm_array(key, idx * _U64(2))
        r2 = sm_array(key, idx * _U64(2) + _U64(1))
    u1 = ((r1 >> _U64(11)).astype(np.float64) + 1.0) * (2.0 ** -53)
    u2 = (r2 >> _U64(11)).astype(np.float64) * (2.0 ** -53)
    v = ((np.sqrt(-2.0 * np.log(u1)) * np.cos((2.0 * np.pi) * u2)) * 0.02).astype(np.float32)
    return f32_to_bf16_bits(v) if bf16 else v


def prompt_ids(seed: int, batch: int, length: int, vocab: int) -> np.ndarray:
    """Uniform-random prompt ids, int32 [batch][length]."""
    out = np.empty((batch, length), dtype=np.int32)
    i = np.arange(length, dtype=np.uint64)
    for b in range(batch):
        r = sm_array(sm_scalar(seed, b), i)
        with np.errstate(over="ignore"):
            out[b] = (((r >> _U64(32)) * _U64(vocab)) >> _U64(32)).astype(np.int32)
    return out


def _ctz64(r: np.ndarray) -> np.ndarray:
    r = r.astype(np.uint64)
    out = np.full(r.shape, 64, dtype=np.int64)
    nz = r != 0
    with np.errstate(over="ignore"):
        below = (r[nz] & (~r[nz] + _U64(1))) - _U64(1)  # ones below the lowest set bit
    out[nz] = np.bitwise_count(below).astype(np.int64)
    return out


def group_schedule(seed: int, batch: int, steps: int, max_group: int) -> np.ndarray:
    """Forced group lengths, int32 [batch][steps]; column 0 is the prefill group."""
    out = np.empty((batch, steps), dtype=np.int32)
    s = np.arange(steps, dtype=np.uint64)
    for b in range(batch):
        r = sm_array(sm_scalar(seed, b), s)
        out[b] = np.minimum(max_group, 1 + _ctz64(r)).astype(np.int32)
    return out
