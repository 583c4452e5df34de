"""Python binding of libsgdrc, the MI355X colour-restricted tensor path.

Argument marshalling only: every operation runs in the HIP kernels of
``libsgdrc.so``; there is no fallback.  If the library has not been built
(``python -m paper_2407_13996_amd.build``) every entry point raises.

Device buffers are passed as torch tensors (or raw integer device
addresses); streams as ``torch.cuda.Stream`` objects, raw ``hipStream_t``
integers, or None for torch's current stream.  The function names match the
C ABI in ``include/sgdrc.h``.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libsgdrc.so")

OK, EINVAL, ENOMEM, ENODEV, EHIP = 0, -22, -12, -19, -5
F32, BF16, F16 = 0, 1, 2
DEVERR_PT_RANGE = 1
DEVFLAG_GATE_FALLBACK = 2
DEVERR_SUSPENDED_DROPPED = 4
DEVERR_HANDBACK = 8
MAX_MASKS = 8
BM_BE_WEIGHT, BM_LS_TENSOR, BM_ACTIVATION = 0, 1, 2
BM_MONOPOLY, BM_COLOCATED = 0, 1
BM_ALL, BM_PART = 0, 1


class SgdrcError(RuntimeError):
    def __init__(self, code: int, message: str, n_found: int | None = None):
        super().__init__(f"sgdrc error {code}: {message}")
        self.code = code
        self.n_found = n_found


class Hash(ctypes.Structure):
    _fields_ = [("n_masks", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("masks", ctypes.c_uint64 * MAX_MASKS)]


class ColourSet(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_uint64 * 4)]


class CuMask(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_uint64 * 4)]


class ColourTable(ctypes.Structure):
    _fields_ = [("lut", ctypes.c_void_p), ("origin", ctypes.c_uint64), ("entries", ctypes.c_uint64),
                ("shift", ctypes.c_uint32), ("reserved", ctypes.c_uint32)]


class Paged(ctypes.Structure):
    _fields_ = [("pool", ctypes.c_void_p), ("pt", ctypes.c_void_p),
                ("pool_pages", ctypes.c_uint64)]


class GemvPlan(ctypes.Structure):
    _fields_ = [("path", ctypes.c_uint32), ("rows", ctypes.c_uint32), ("loads", ctypes.c_uint32),
                ("batch_cols", ctypes.c_uint32), ("tiles", ctypes.c_uint64),
                ("sum_depth", ctypes.c_uint32), ("x_once", ctypes.c_uint32)]


GEMV_VALU, GEMV_MFMA = 0, 1


class RelayoutItem(ctypes.Structure):
    _fields_ = [("dst", Paged), ("src", Paged), ("n_bytes", ctypes.c_uint64),
                ("page_shift", ctypes.c_uint32), ("reserved", ctypes.c_uint32)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libsgdrc.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2407_13996_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, u32, u64, i32 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int
        P = ctypes.POINTER
        sigs = {
            "sgdrc_init": ([i32, P(vp)], i32),
            "sgdrc_destroy": ([vp], i32),
            "sgdrc_num_cus": ([vp], i32),
            "sgdrc_cu_key": ([vp, u32, P(u32)], i32),
            "sgdrc_last_error": ([], ctypes.c_char_p),
            "sgdrc_device_error": ([vp, P(u32)], i32),
            "sgdrc_set_worklog": ([vp, vp, vp, u64], i32),
            "sgdrc_last_tiles": ([vp, vp, P(u64)], i32),
            "sgdrc_last_schedule": ([vp, vp, P(u32)], i32),
            "sgdrc_set_timelog": ([vp, vp, vp, u32], i32),
            "sgdrc_wallclock_khz": ([vp, P(u32)], i32),
            "set_cu_mask": ([vp, vp, P(CuMask)], i32),
            "sgdrc_set_stream_occupancy": ([vp, vp, u32], i32),
            "sgdrc_set_eviction_flag": ([vp, vp, vp], i32),
            "sgdrc_resume": ([vp, vp], i32),
            "sgdrc_signal_flag": ([vp, vp, vp, u32, vp], i32),
            "sgdrc_suspended": ([vp, vp, P(u64)], i32),
            "sgdrc_set_eviction_hook": ([vp, vp, u32], i32),
            "sgdrc_stream_release": ([vp, vp], i32),
            "colour_alloc_pagetable_noalloc": ([vp, P(Hash), u64, u32, u64, P(ColourSet), u64, vp,
                                                vp, vp], i32),
            "sgdrc_tidal_masks": ([u32, P(u32), u32, u32, u32, P(CuMask), P(CuMask)], i32),
            "sgdrc_bm_create": ([vp, P(vp)], i32),
            "sgdrc_bm_destroy": ([vp], i32),
            "sgdrc_bm_register": ([vp, u32, P(Paged), P(Paged), u64, u32, vp, P(u32)], i32),
            "sgdrc_bm_set_state": ([vp, i32, vp], i32),
            "sgdrc_bm_state": ([vp, P(i32)], i32),
            "sgdrc_bm_input": ([vp, u32, P(Paged), P(i32)], i32),
            "sgdrc_bm_output": ([vp, u32, P(Paged), P(i32)], i32),
            "sgdrc_bm_acquire": ([vp, u64, P(u32)], i32),
            "sgdrc_bm_release": ([vp, u32], i32),
            "colour_classify": ([vp, P(Hash), vp, u64, vp, vp, vp], i32),
            "colour_alloc_pagetable": ([vp, P(Hash), u64, u32, u64, P(ColourSet), u64, vp,
                                        P(u64), vp], i32),
            "bimodal_relayout": ([vp, P(Paged), P(Paged), u64, u32, vp], i32),
            "bimodal_relayout_batch": ([vp, P(RelayoutItem), u32, vp], i32),
            "colored_stream": ([vp, P(Paged), P(Paged), P(Paged), ctypes.c_float, u64, u32, vp],
                               i32),
            "colored_gemv": ([vp, P(Paged), i32, u32, u32, vp, i32, u32, vp, u32, vp], i32),
            "colored_gemv_plan": ([u32, i32, u32, u32, i32, u32, P(GemvPlan)], i32),
            "colour_classify_table": ([vp, P(ColourTable), vp, u64, vp, vp, vp], i32),
            "colour_alloc_pagetable_table": ([vp, P(ColourTable), u64, u32, u64, P(ColourSet), u64,
                                              vp, P(u64), vp], i32),
        }
        for name, (args, res) in sigs.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def last_error() -> str:
    return lib().sgdrc_last_error().decode()


def _check(rc: int, n_found: int | None = None) -> None:
    if rc != OK:
        raise SgdrcError(rc, last_error(), n_found)


def _addr(x) -> int | None:
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    return int(x)


def _stream(s):
    if s is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if hasattr(s, "cuda_stream"):
        return ctypes.c_void_p(s.cuda_stream)
    return ctypes.c_void_p(int(s))


def make_hash(masks) -> Hash:
    masks = [int(m) for m in masks]
    h = Hash()
    h.n_masks = len(masks)
    h.reserved = 0
    for i, m in enumerate(masks[:MAX_MASKS]):
        h.masks[i] = m
    return h


def make_set(words, cls=ColourSet):
    s = cls()
    for i, w in enumerate(words):
        s.bits[i] = int(w)
    return s


def words_of(indices) -> list:
    words = [0, 0, 0, 0]
    for c in indices:
        words[int(c) >> 6] |= 1 << (int(c) & 63)
    return words


def paged(pool, pt, pool_pages: int) -> Paged:
    """A Paged descriptor; it keeps references to tensors passed for pool and
    pt so that their memory stays allocated while the descriptor lives."""
    p = Paged(_addr(pool), _addr(pt), int(pool_pages))
    p._keep = (pool, pt)
    return p


class Context:
    """One libsgdrc context on a HIP device."""

    def __init__(self, device: int = 0):
        h = ctypes.c_void_p()
        _check(lib().sgdrc_init(int(device), ctypes.byref(h)))
        self.handle = h
        self.device = device

    @property
    def num_cus(self) -> int:
        n = lib().sgdrc_num_cus(self.handle)
        if n < 0:
            _check(n)
        return n

    def cu_key(self, cu: int) -> int:
        k = ctypes.c_uint32()
        _check(lib().sgdrc_cu_key(self.handle, int(cu), ctypes.byref(k)))
        return k.value

    def device_error(self) -> int:
        f = ctypes.c_uint32()
        _check(lib().sgdrc_device_error(self.handle, ctypes.byref(f)))
        return f.value

    def set_worklog(self, cu_tiles=None, tile_visits=None) -> None:
        cap = 0 if tile_visits is None else int(tile_visits.numel())
        _check(lib().sgdrc_set_worklog(self.handle, _addr(cu_tiles), _addr(tile_visits), cap))

    def last_tiles(self, stream=None) -> int:
        t = ctypes.c_uint64()
        _check(lib().sgdrc_last_tiles(self.handle, _stream(stream), ctypes.byref(t)))
        return t.value

    def last_schedule(self, stream=None) -> str:
        """'static' or 'queue': how the last launch on ``stream`` took its tiles."""
        v = ctypes.c_uint32()
        _check(lib().sgdrc_last_schedule(self.handle, _stream(stream), ctypes.byref(v)))
        return "static" if v.value == 1 else "queue"

    def set_timelog(self, stream=None, slots=None) -> None:
        """Log {start, end} device-clock ticks of each later launch on
        ``stream`` into ``slots`` (int64 device tensor of 2 * n entries,
        used cyclically); None switches the log off."""
        n = 0 if slots is None else int(slots.numel()) // 2
        if slots is not None and n == 0:
            raise ValueError("slots must hold at least one {start, end} pair")
        _check(lib().sgdrc_set_timelog(self.handle, _stream(stream), _addr(slots), n))

    @property
    def wallclock_khz(self) -> int:
        k = ctypes.c_uint32()
        _check(lib().sgdrc_wallclock_khz(self.handle, ctypes.byref(k)))
        return k.value

    def close(self) -> None:
        if self.handle is not None and self.handle.value:
            _check(lib().sgdrc_destroy(self.handle))
        self.handle = None


def _h(ctx):
    return ctx.handle if isinstance(ctx, Context) else ctx


def set_cu_mask(ctx, stream, cus) -> None:
    """cus: iterable of logical CU indices, or None for all CUs."""
    m = None if cus is None else ctypes.byref(make_set(words_of(cus), CuMask))
    _check(lib().set_cu_mask(_h(ctx), _stream(stream), m))


def set_stream_occupancy(ctx, stream, max_wgs_per_cu: int) -> None:
    """Cap the workgroups per CU of later launches on ``stream`` (0 = no cap)."""
    _check(lib().sgdrc_set_stream_occupancy(_h(ctx), _stream(stream), int(max_wgs_per_cu)))


def set_eviction_flag(ctx, stream, flag) -> None:
    """Make later colored_stream / bimodal_relayout launches on ``stream``
    preemptible by the device word ``flag`` (an int32 CUDA tensor of at
    least one element, or a raw address); None switches it off."""
    _check(lib().sgdrc_set_eviction_flag(_h(ctx), _stream(stream), _addr(flag)))


def set_eviction_hook(ctx, stream, tile: int) -> None:
    """Testing aid: later preemptible launches on ``stream`` act as if the
    eviction flag rose at tile index ``tile`` (0 switches it off)."""
    _check(lib().sgdrc_set_eviction_hook(_h(ctx), _stream(stream), int(tile)))


def stream_release(ctx, stream) -> None:
    """Forget the context's state for ``stream`` (mask, cap, flags, queues)."""
    _check(lib().sgdrc_stream_release(_h(ctx), _stream(stream)))


def resume(ctx, stream=None) -> None:
    """Enqueue the continuation of the stream's last preemptible launch."""
    _check(lib().sgdrc_resume(_h(ctx), _stream(stream)))


def signal_flag(ctx, stream, flag, value: int, stamp=None) -> None:
    """Enqueue on ``stream`` a device store of ``value`` to ``flag`` (and of
    the device clock to ``stamp``, an int64 tensor element, if given)."""
    _check(lib().sgdrc_signal_flag(_h(ctx), _stream(stream), _addr(flag), int(value),
                                   _addr(stamp)))


def suspended(ctx, stream=None) -> int:
    """Wait for ``stream``; tiles its last preemptible launch has left (0 = done)."""
    t = ctypes.c_uint64()
    _check(lib().sgdrc_suspended(_h(ctx), _stream(stream), ctypes.byref(t)))
    return t.value


def _cus_of(m: CuMask, n: int) -> list:
    return [i for i in range(n) if (m.bits[i >> 6] >> (i & 63)) & 1]


def tidal_masks(num_cus: int, ls_cus, window: int, granule: int = 1):
    """Sliding-window CU reservation: (LS CUs, BE CUs) as lists of logical CUs
    for the queued latency-sensitive kernels' CU needs ``ls_cus``."""
    q = [int(x) for x in ls_cus]
    arr = (ctypes.c_uint32 * max(len(q), 1))(*q)
    ls, be = CuMask(), CuMask()
    _check(lib().sgdrc_tidal_masks(int(num_cus), arr, len(q), int(window), int(granule),
                                   ctypes.byref(ls), ctypes.byref(be)))
    return _cus_of(ls, num_cus), _cus_of(be, num_cus)


def colour_classify(ctx, masks, addrs, colours, hist=None, stream=None) -> None:
    _check(lib().colour_classify(_h(ctx), ctypes.byref(make_hash(masks)), _addr(addrs),
                                 int(addrs.numel()), _addr(colours), _addr(hist),
                                 _stream(stream)))


def colour_alloc_pagetable(ctx, masks, addr_origin: int, page_shift: int, pool_pages: int,
                           colours, n_needed: int, pt, stream=None) -> int:
    """Returns n_found; raises SgdrcError (code ENOMEM, .n_found) on shortfall."""
    found = ctypes.c_uint64()
    rc = lib().colour_alloc_pagetable(_h(ctx), ctypes.byref(make_hash(masks)), int(addr_origin),
                                      int(page_shift), int(pool_pages),
                                      ctypes.byref(make_set(words_of(colours))), int(n_needed),
                                      _addr(pt), ctypes.byref(found), _stream(stream))
    _check(rc, found.value)
    return found.value


def colour_alloc_pagetable_noalloc(ctx, masks, addr_origin: int, page_shift: int,
                                   pool_pages: int, colours, n_needed: int, pt, n_found,
                                   stream=None) -> None:
    """Asynchronous, allocation-free page-table build: the table goes to
    ``pt`` and the count of qualifying pages to ``n_found`` (a device int64
    tensor of one element); no shortfall error."""
    _check(lib().colour_alloc_pagetable_noalloc(_h(ctx), ctypes.byref(make_hash(masks)),
                                                int(addr_origin), int(page_shift),
                                                int(pool_pages),
                                                ctypes.byref(make_set(words_of(colours))),
                                                int(n_needed), _addr(pt), _addr(n_found),
                                                _stream(stream)))


def colour_table(lut, origin: int, shift: int) -> ColourTable:
    """Descriptor of a colour table (uint8 device tensor, one entry per
    2^shift-byte partition from ``origin``); keeps a reference to ``lut``."""
    t = ColourTable(_addr(lut), int(origin), int(lut.numel()), int(shift), 0)
    t._keep = lut
    return t


def colour_classify_table(ctx, table: ColourTable, addrs, colours, hist=None, stream=None) -> None:
    _check(lib().colour_classify_table(_h(ctx), ctypes.byref(table), _addr(addrs),
                                       int(addrs.numel()), _addr(colours), _addr(hist),
                                       _stream(stream)))


def colour_alloc_pagetable_table(ctx, table: ColourTable, addr_origin: int, page_shift: int,
                                 pool_pages: int, colours, n_needed: int, pt, stream=None) -> int:
    """Returns n_found; raises SgdrcError (code ENOMEM, .n_found) on shortfall."""
    found = ctypes.c_uint64()
    rc = lib().colour_alloc_pagetable_table(_h(ctx), ctypes.byref(table), int(addr_origin),
                                            int(page_shift), int(pool_pages),
                                            ctypes.byref(make_set(words_of(colours))),
                                            int(n_needed), _addr(pt), ctypes.byref(found),
                                            _stream(stream))
    _check(rc, found.value)
    return found.value


def bimodal_relayout(ctx, dst: Paged, src: Paged, n_bytes: int, page_shift: int,
                     stream=None) -> None:
    _check(lib().bimodal_relayout(_h(ctx), ctypes.byref(dst), ctypes.byref(src), int(n_bytes),
                                  int(page_shift), _stream(stream)))


def bimodal_relayout_batch(ctx, items, stream=None) -> None:
    """``items``: (dst Paged, src Paged, n_bytes, page_shift) tuples, copied
    as bimodal_relayout would, in one launch per 32 items."""
    arr = (RelayoutItem * max(len(items), 1))()
    for i, (dst, src, n_bytes, shift) in enumerate(items):
        arr[i] = RelayoutItem(dst, src, int(n_bytes), int(shift), 0)
    _check(lib().bimodal_relayout_batch(_h(ctx), arr, len(items), _stream(stream)))


def colored_stream(ctx, a: Paged, b: Paged, c: Paged, s: float, n_elems: int, page_shift: int,
                   stream=None) -> None:
    _check(lib().colored_stream(_h(ctx), ctypes.byref(a), ctypes.byref(b), ctypes.byref(c),
                                float(s), int(n_elems), int(page_shift), _stream(stream)))


def colored_gemv(ctx, w: Paged, w_dtype: int, M: int, K: int, x, x_dtype: int, batch: int, y,
                 page_shift: int, stream=None) -> None:
    _check(lib().colored_gemv(_h(ctx), ctypes.byref(w), int(w_dtype), int(M), int(K), _addr(x),
                              int(x_dtype), int(batch), _addr(y), int(page_shift),
                              _stream(stream)))


def gemv_plan(allowed_cus: int, w_dtype: int, M: int, K: int, x_dtype: int, batch: int) -> dict:
    """The launch plan colored_gemv takes for this shape on ``allowed_cus``
    CUs (host-only; no device needed)."""
    p = GemvPlan()
    _check(lib().colored_gemv_plan(int(allowed_cus), int(w_dtype), int(M), int(K), int(x_dtype),
                                 int(batch), ctypes.byref(p)))
    return {"path": "mfma" if p.path == GEMV_MFMA else "valu", "rows": p.rows, "loads": p.loads,
            "batch_cols": p.batch_cols, "tiles": p.tiles, "sum_depth": p.sum_depth,
            "x_once": bool(p.x_once)}


class Bimodal:
    """The bimodal tensor runtime: tensor forms by class and co-location
    state.  ``ctx`` may be None (activations only)."""

    def __init__(self, ctx=None):
        h = ctypes.c_void_p()
        _check(lib().sgdrc_bm_create(_h(ctx) if ctx is not None else None, ctypes.byref(h)))
        self.handle = h
        self.has_ctx = ctx is not None
        self._keep = []

    def _st(self, stream):
        # a runtime without context never moves data: no stream needed
        return _stream(stream) if (self.has_ctx or stream is not None) else None

    def register(self, cls: int, all_form: Paged, part_form: Paged, n_bytes: int,
                 page_shift: int, stream=None) -> int:
        i = ctypes.c_uint32()
        _check(lib().sgdrc_bm_register(self.handle, int(cls), ctypes.byref(all_form),
                                       ctypes.byref(part_form), int(n_bytes), int(page_shift),
                                       self._st(stream), ctypes.byref(i)))
        self._keep.append((all_form, part_form))
        return i.value

    def set_state(self, state: int, stream=None) -> None:
        _check(lib().sgdrc_bm_set_state(self.handle, int(state), self._st(stream)))

    @property
    def state(self) -> int:
        v = ctypes.c_int()
        _check(lib().sgdrc_bm_state(self.handle, ctypes.byref(v)))
        return v.value

    def input(self, tid: int):
        """(descriptor, form) a kernel reads tensor ``tid`` through."""
        p, w = Paged(), ctypes.c_int()
        _check(lib().sgdrc_bm_input(self.handle, int(tid), ctypes.byref(p), ctypes.byref(w)))
        return p, w.value

    def output(self, tid: int):
        """(descriptor, form) a kernel writes tensor ``tid`` through."""
        p, w = Paged(), ctypes.c_int()
        _check(lib().sgdrc_bm_output(self.handle, int(tid), ctypes.byref(p), ctypes.byref(w)))
        return p, w.value

    def acquire(self, n_bytes: int) -> int:
        i = ctypes.c_uint32()
        _check(lib().sgdrc_bm_acquire(self.handle, int(n_bytes), ctypes.byref(i)))
        return i.value

    def release(self, tid: int) -> None:
        _check(lib().sgdrc_bm_release(self.handle, int(tid)))

    def close(self) -> None:
        if self.handle is not None and self.handle.value:
            _check(lib().sgdrc_bm_destroy(self.handle))
        self.handle = None
