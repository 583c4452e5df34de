"""Seeded synthetic inputs for the colour-restricted tensor path.

This module only draws random inputs. It holds none of the method's
arithmetic: no colour hash, no page-table filter, no copy, no triad, no GEMV.
Both the CPU oracle's tests and the GPU path's tests and bench take their
inputs from here, so that the two sides see identical bytes.

Recipe (the paper's own workloads -- the Apollo trace and the eleven DNN
models of its evaluation -- are not available; these shapes stand in for its
memory-bound latency-sensitive layers and its memory-heavy best-effort
kernels, paper section 7.2 and section 9.1.1):

* page addresses: ``integers(0, 2**36) << 12`` (uniform 4 KiB-aligned
  48-bit addresses), ``default_rng(seed)``;
* XOR masks: each mask ``integers(0, 2**(41 - b)) << b`` with
  b = max(8, ``min_bit``) (every bit of b..40 set with probability 1/2),
  drawn from ``default_rng(mask_seed)``; ``min_bit`` is the largest page
  shift of the configuration, so that no mask bit falls inside a page and
  every page has one colour (the paper colours whole sectors); the whole set
  of K masks is redrawn from the same stream until the masks, and also the
  masks cut down to their K + 2 lowest bits b..b+K+1, are linearly
  independent over GF(2): then all 2**K colours exist and every aligned run
  of 2**(K+2) pages holds each colour equally often (consecutive pages
  interleave over the colours, as hardware channel hashes interleave
  consecutive blocks over channels), so small pools reach every colour;
* fp32 data: N(0,1), or U[-1,1) built as ``2*u - 1`` from numpy's 24-bit
  float32 uniforms (every value is a multiple of 2**-23);
* bf16 data: float32 N(0, sigma) rounded to nearest-even to bf16 bits;
* fp16 data: uniform random 16-bit patterns (NaN/Inf payloads included).
"""
from __future__ import annotations

import numpy as np

ADDR_BITS = 48
MASK_LO_BIT = 8
MASK_HI_BIT = 40


def gf2_rank(vectors) -> int:
    """Rank over GF(2) of a list of integers read as bit vectors."""
    basis = []  # kept reduced: each element has a distinct leading bit
    for v in vectors:
        v = int(v)
        for b in basis:
            v = min(v, v ^ b)
        if v:
            basis.append(v)
            basis.sort(reverse=True)
    return len(basis)


def xor_masks(n_masks: int, seed: int = 1, min_bit: int = 12,
              lo_bit: int = MASK_LO_BIT, hi_bit: int = MASK_HI_BIT):
    """K random masks on address bits max(lo_bit, min_bit)..hi_bit, full rank.

    Returns a list of python ints.  Bits below ``min_bit`` (the page shift)
    stay clear, so a page of 2**min_bit bytes hashes to one colour.  Redraws
    the whole set from one stream until the masks have GF(2) rank K, and so
    have the masks cut down to their K + 2 lowest bits (when the bit range
    holds that many).
    """
    if not 1 <= n_masks <= 8:
        raise ValueError("1 <= n_masks <= 8")
    lo = max(lo_bit, min_bit)
    if hi_bit - lo + 1 < n_masks:
        raise ValueError("not enough mask bits above min_bit for full rank")
    rng = np.random.default_rng(seed)
    width = hi_bit - lo + 1
    window = ((1 << min(n_masks + 2, width)) - 1) << lo
    while True:
        masks = [int(rng.integers(0, 2 ** width)) << lo for _ in range(n_masks)]
        if gf2_rank(masks) == n_masks and gf2_rank([m & window for m in masks]) == n_masks:
            return masks


def page_addresses(n: int, seed: int = 0, page_bits: int = 12,
                   addr_bits: int = ADDR_BITS) -> np.ndarray:
    """n uniform random page-aligned addresses below 2**addr_bits (uint64)."""
    rng = np.random.default_rng(seed)
    return (rng.integers(0, 2 ** (addr_bits - page_bits), size=n, dtype=np.uint64)
            << np.uint64(page_bits)).astype(np.uint64)


def colour_set_bits(colours) -> list:
    """A 256-bit colour set as four little-endian uint64 words."""
    words = [0, 0, 0, 0]
    for c in colours:
        c = int(c)
        if not 0 <= c < 256:
            raise ValueError("colour out of range")
        words[c >> 6] |= 1 << (c & 63)
    return words


def cu_mask_bits(cus) -> list:
    """A 256-bit compute-unit set as four little-endian uint64 words."""
    return colour_set_bits(cus)


def uniform_f32(n: int, seed: int = 0) -> np.ndarray:
    """U[-1,1) float32; every value is an exact multiple of 2**-23."""
    rng = np.random.default_rng(seed)
    u = rng.random(n, dtype=np.float32)
    return (u * np.float32(2.0) - np.float32(1.0)).astype(np.float32)


def normal_f32(n: int, seed: int = 0, sigma: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(n, dtype=np.float32) * np.float32(sigma)).astype(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bf16 bit patterns (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return rounded.astype(np.uint16)


def normal_bf16(n: int, seed: int = 0, sigma: float = 1.0) -> np.ndarray:
    """N(0, sigma) as bf16 bit patterns (uint16)."""
    return f32_to_bf16_bits(normal_f32(n, seed, sigma))


def random_u16(n: int, seed: int = 0) -> np.ndarray:
    """Uniform random 16-bit patterns (used as fp16 payloads)."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, 2 ** 16, size=n, dtype=np.uint16)


def random_bytes(n: int, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, 256, size=n, dtype=np.uint8)


def random_permutation(n: int, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.permutation(n).astype(np.uint32)


def random_cu_subset(num_cus: int, k: int, seed: int = 0) -> list:
    rng = np.random.default_rng(seed)
    return sorted(int(c) for c in rng.choice(num_cus, size=k, replace=False))
