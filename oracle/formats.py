"""Decoders for the storage formats the oracle reads (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` use this package; the product path never does.

* bf16: the upper 16 bits of an IEEE-754 binary32 value.
* OCP FP8 E4M3 ("e4m3fn"): 1 sign bit, 4 exponent bits (bias 7), 3 mantissa
  bits; exponent field 0 encodes subnormals m/8 * 2^-6; S.1111.111 is NaN;
  there is no infinity, so the largest finite magnitude is 1.75 * 2^8 = 448.
"""
import numpy as np


def decode_bf16(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64 values (exact)."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def decode_e4m3(codes) -> np.ndarray:
    """OCP E4M3 codes (uint8) -> float64 values (exact; NaN for S.1111.111)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    normal = np.ldexp(1.0 + m / 8.0, (e - 7).astype(np.int64))
    subnormal = np.ldexp(m / 8.0, -6)
    v = sign * np.where(e == 0, subnormal, normal)
    return np.where((e == 15) & ((c & 7) == 7), np.nan, v)


def decode_weight(entry, fmt: str) -> np.ndarray:
    """One stored weight tensor -> float64.

    ``fmt`` is ``"f32"`` (float32 array), ``"bf16"`` (uint16 bit patterns) or
    ``"e4m3"`` (a ``(codes [out, in], bf16 scale bits [out])`` pair whose
    value is ``decode(code) * scale[row]``)."""
    if fmt == "f32":
        return np.asarray(entry, dtype=np.float64)
    if fmt == "bf16":
        return decode_bf16(entry)
    if fmt == "e4m3":
        codes, scale_bits = entry
        return decode_e4m3(codes) * decode_bf16(scale_bits)[:, None]
    raise ValueError(f"unknown weight format {fmt!r}")


def decode_states(x, fmt: str) -> np.ndarray:
    """Stored activations (float32 or bf16 bits) -> float64."""
    return np.asarray(x, dtype=np.float64) if fmt == "f32" else decode_bf16(x)
