"""CPU oracle for the colour-restricted tensor path -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It wraps ``oracle.c`` (plain C,
single-threaded, built with gcc) with numpy-array entry points.  Nothing in
the HIP library imports it, and it imports nothing from the HIP library.

Parity status: every function is pinned by ``tests/test_oracle_pins.py``
(invariants, closed forms, brute force, library routines); none is
"parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

F32, BF16, F16 = 0, 1, 2

_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with gcc (no contraction, no fast-math)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math",
                               "-shared", "-fPIC", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"])
        os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=False)
        L = ctypes.CDLL(LIB)
        u32, u64, i32, vp = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p
        L.oracle_colour.argtypes = [u64, vp, u32]
        L.oracle_colour.restype = u32
        L.oracle_colour_popcount.argtypes = [u64, vp, u32]
        L.oracle_colour_popcount.restype = u32
        L.oracle_classify.argtypes = [vp, u64, vp, u32, vp, vp]
        L.oracle_classify.restype = None
        L.oracle_pagetable.argtypes = [vp, u32, u64, u32, u64, vp, u64, vp]
        L.oracle_pagetable.restype = u64
        L.oracle_lut_colour.argtypes = [u64, vp, u64, u64, u32]
        L.oracle_lut_colour.restype = u32
        L.oracle_classify_lut.argtypes = [vp, u64, vp, u64, u64, u32, vp, vp]
        L.oracle_classify_lut.restype = None
        L.oracle_pagetable_lut.argtypes = [vp, u64, u64, u32, u64, u32, u64, vp, u64, vp]
        L.oracle_pagetable_lut.restype = u64
        L.oracle_relayout.argtypes = [vp, vp, vp, vp, u64, u32]
        L.oracle_relayout.restype = None
        L.oracle_triad.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.c_float, u64, u32]
        L.oracle_triad.restype = None
        L.oracle_decode.argtypes = [u32, i32]
        L.oracle_decode.restype = ctypes.c_double
        L.oracle_gemv.argtypes = [vp, vp, i32, u32, u32, vp, i32, u32, u32, vp, vp]
        L.oracle_gemv.restype = None
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return ctypes.c_void_p(a.ctypes.data)


def _masks(masks) -> np.ndarray:
    return np.ascontiguousarray(np.array([int(m) for m in masks], dtype=np.uint64))


def colour(addr: int, masks) -> int:
    m = _masks(masks)
    return int(lib().oracle_colour(int(addr), _ptr(m), len(m)))


def colour_popcount(addr: int, masks) -> int:
    m = _masks(masks)
    return int(lib().oracle_colour_popcount(int(addr), _ptr(m), len(m)))


def classify(addrs: np.ndarray, masks, with_hist: bool = True):
    """Returns (colours uint8[n], hist uint64[2^K] or None)."""
    a = np.ascontiguousarray(addrs, dtype=np.uint64)
    m = _masks(masks)
    colours = np.empty(a.size, dtype=np.uint8)
    hist = np.empty(1 << len(m), dtype=np.uint64) if with_hist else None
    lib().oracle_classify(_ptr(a), a.size, _ptr(m), len(m), _ptr(colours),
                          _ptr(hist) if hist is not None else None)
    return colours, hist


def pagetable(masks, origin: int, page_shift: int, pool_pages: int, colour_set_words,
              n_needed: int):
    """Returns (pt uint32[min(found, n_needed)], found)."""
    m = _masks(masks)
    s = np.ascontiguousarray(np.array([int(w) for w in colour_set_words], dtype=np.uint64))
    assert s.size == 4
    pt = np.zeros(max(n_needed, 1), dtype=np.uint32)
    found = int(lib().oracle_pagetable(_ptr(m), len(m), int(origin), int(page_shift),
                                       int(pool_pages), _ptr(s), int(n_needed), _ptr(pt)))
    return pt[:min(found, n_needed)].copy(), found


def relayout(dst_pool: np.ndarray, pt_dst: np.ndarray, src_pool: np.ndarray,
             pt_src: np.ndarray, n_bytes: int, page_shift: int) -> None:
    """In place on dst_pool (any dtype; addressed as bytes)."""
    pd = np.ascontiguousarray(pt_dst, dtype=np.uint32)
    ps = np.ascontiguousarray(pt_src, dtype=np.uint32)
    lib().oracle_relayout(_ptr(dst_pool), _ptr(pd), _ptr(src_pool), _ptr(ps),
                          int(n_bytes), int(page_shift))


def triad(a_pool, pt_a, b_pool, pt_b, c_pool, pt_c, s: float, n: int, page_shift: int) -> None:
    """In place on a_pool: a = fmaf(s, c, b) through the three page tables."""
    pa, pb, pc = (np.ascontiguousarray(p, dtype=np.uint32) for p in (pt_a, pt_b, pt_c))
    lib().oracle_triad(_ptr(a_pool), _ptr(pa), _ptr(b_pool), _ptr(pb), _ptr(c_pool), _ptr(pc),
                       float(s), int(n), int(page_shift))


def decode(bits: int, dtype: int) -> float:
    return float(lib().oracle_decode(int(bits), int(dtype)))


def gemv(w_pool, pt_w, w_dtype: int, M: int, K: int, x, x_dtype: int, B: int,
         page_shift: int, with_absdot: bool = True):
    """Returns (y float64[B, M], absdot float64[B, M] or None)."""
    pw = np.ascontiguousarray(pt_w, dtype=np.uint32)
    xx = np.ascontiguousarray(x)
    y = np.empty((B, M), dtype=np.float64)
    ad = np.empty((B, M), dtype=np.float64) if with_absdot else None
    lib().oracle_gemv(_ptr(w_pool), _ptr(pw), int(w_dtype), int(M), int(K), _ptr(xx),
                      int(x_dtype), int(B), int(page_shift), _ptr(y),
                      _ptr(ad) if ad is not None else None)
    return y, ad


def lut_colour(addr: int, lut: np.ndarray, origin: int, lut_shift: int) -> int:
    t = np.ascontiguousarray(lut, dtype=np.uint8)
    return int(lib().oracle_lut_colour(int(addr), _ptr(t), int(origin), t.size, int(lut_shift)))


def classify_lut(addrs: np.ndarray, lut: np.ndarray, origin: int, lut_shift: int,
                 with_hist: bool = True):
    """Returns (colours uint8[n], hist uint64[256] or None)."""
    a = np.ascontiguousarray(addrs, dtype=np.uint64)
    t = np.ascontiguousarray(lut, dtype=np.uint8)
    colours = np.empty(a.size, dtype=np.uint8)
    hist = np.empty(256, dtype=np.uint64) if with_hist else None
    lib().oracle_classify_lut(_ptr(a), a.size, _ptr(t), int(origin), t.size, int(lut_shift),
                              _ptr(colours), _ptr(hist) if hist is not None else None)
    return colours, hist


def pagetable_lut(lut: np.ndarray, origin: int, lut_shift: int, addr_origin: int,
                  page_shift: int, pool_pages: int, colour_set_words, n_needed: int):
    """Returns (pt uint32[min(found, n_needed)], found)."""
    t = np.ascontiguousarray(lut, dtype=np.uint8)
    s = np.ascontiguousarray(np.array([int(w) for w in colour_set_words], dtype=np.uint64))
    assert s.size == 4
    pt = np.zeros(max(n_needed, 1), dtype=np.uint32)
    found = int(lib().oracle_pagetable_lut(_ptr(t), int(origin), t.size, int(lut_shift),
                                           int(addr_origin), int(page_shift), int(pool_pages),
                                           _ptr(s), int(n_needed), _ptr(pt)))
    return pt[:min(found, n_needed)].copy(), found
