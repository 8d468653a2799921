"""Seeded synthetic inputs shared by the CPU oracle and the HIP path.

This module only draws numbers and packs them into the storage formats the
two sides consume.  It holds none of the projection's arithmetic: no block
products, no supports, no activations.  Every tensor is drawn from
``numpy.random.default_rng([config_id, tensor_id])`` so that the oracle and
the GPU receive bit-identical inputs.

Storage formats
---------------
* ``"f32"``: IEEE binary32 values.
* ``"bf16"``: bfloat16, obtained from the binary32 draw by round-to-nearest-
  even on the upper 16 bits.  The generator returns both the raw ``uint16``
  bit patterns (what the GPU receives) and their exact float64 values (what
  the oracle receives).
"""

from __future__ import annotations

import dataclasses

import numpy as np

__all__ = [
    "Tensor",
    "gaussian",
    "f32_to_bf16_bits",
    "bf16_bits_to_f64",
    "cyclic_types",
    "sequence_types",
    "decode_positions",
    "equal_widths",
]


@dataclasses.dataclass
class Tensor:
    """A synthetic tensor in its storage format plus its exact float64 value."""

    raw: np.ndarray  # float32 array, or uint16 bf16 bit patterns
    exact: np.ndarray  # float64, exactly the stored values
    dtype: str  # "f32" or "bf16"


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round binary32 values to bfloat16 (nearest, ties to even); return bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = (u + 0x7FFF + lsb) >> 16
    nan = np.isnan(x)
    out = rounded.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    """Exact float64 values of bfloat16 bit patterns."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def gaussian(config_id: int, tensor_id: int, shape, std: float = 1.0,
             dtype: str = "bf16") -> Tensor:
    """i.i.d. N(0, std^2) draw, stored as ``dtype``."""
    rng = np.random.default_rng([int(config_id), int(tensor_id)])
    x = (rng.standard_normal(size=shape) * std).astype(np.float32)
    if dtype == "f32":
        return Tensor(raw=x, exact=x.astype(np.float64), dtype="f32")
    if dtype == "bf16":
        bits = f32_to_bf16_bits(x)
        return Tensor(raw=bits, exact=bf16_bits_to_f64(bits), dtype="bf16")
    raise ValueError(f"unknown dtype {dtype!r}")


def cyclic_types(M: int, q: int, seq_len: int | None = None,
                 offset: int = 0) -> np.ndarray:
    """Row types ``(position + offset) mod q``.

    ``seq_len`` makes the position restart at every sequence boundary, as
    for a batch of ``M // seq_len`` sequences laid out back to back.
    """
    b = np.arange(M, dtype=np.int64)
    pos = b % seq_len if seq_len else b
    return ((pos + offset) % q).astype(np.int32)


def sequence_types(M: int, q: int, seq_len: int) -> np.ndarray:
    """Position-in-sequence mod q for ``M`` rows of back-to-back sequences."""
    return cyclic_types(M, q, seq_len=seq_len)


def decode_positions(config_id: int, M: int, max_pos: int = 2048) -> np.ndarray:
    """Random decode positions in ``[0, max_pos)`` for ``M`` sequences."""
    rng = np.random.default_rng([int(config_id), 1000])
    return rng.integers(0, max_pos, size=M).astype(np.int64)


def equal_widths(total: int, q: int) -> list[int]:
    """``q`` equal group widths summing to ``total``."""
    if total % q:
        raise ValueError(f"{total} is not divisible by q={q}")
    return [total // q] * q
