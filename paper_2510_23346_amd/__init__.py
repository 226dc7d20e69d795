"""MI355X (gfx950) block-diagonal LoRA shard library -- Python binding.

A thin ctypes layer over ``libbdlora.so`` (C ABI in ``include/bdlora.h``):
it checks and marshals arguments (tensor pointers, shapes, the current HIP
stream) and calls the library; every step of the computation runs in the
library's HIP kernels.  PyTorch is used only for device memory and streams.
The library must have been built (``python -m paper_2510_23346_amd.build``);
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "COLUMN", "ROW", "BDLoRAError", "lib", "lib_path", "Pool", "ProjDesc", "build_plan",
    "adapter_elems", "pool_size", "pack_weight", "HEADER_FUNCTIONS", "DECODE_MAX_T", "DECODE_PLAN_IN_MAIN_T",
    "DECODE_PLAN_IN_MAIN_BYTES", "decode_plans_in_main",
    "ACT_NONE", "ACT_SILU_MUL", "WEIGHT_BF16", "WEIGHT_INT4_G128", "pack_weight_int4",
    "packed_weight_bytes", "MAX_SEGMENTS", "Segments", "layout_slot_bytes", "pack_adapter_layout",
]

COLUMN, ROW = 0, 1
MAX_SLICES = 4
DECODE_MAX_T = 64       # BDLORA_DECODE_MAX_T: largest batch that takes the decode launches
DECODE_PLAN_IN_MAIN_T = 32            # BDLORA_DECODE_PLAN_IN_MAIN_T
DECODE_PLAN_IN_MAIN_BYTES = 1572864    # BDLORA_DECODE_PLAN_IN_MAIN_BYTES


def decode_plans_in_main(T, d_ins):
    """Whether a decode call of T tokens over projections with inputs
    ``d_ins`` skips the plan launch (the rule stated in bdlora.h)."""
    act = 2 * T * sum(int(k) for k in d_ins)
    return 1 <= T <= 16 or (T <= DECODE_PLAN_IN_MAIN_T and act <= DECODE_PLAN_IN_MAIN_BYTES)
MAX_SEGMENTS = 256      # BDLORA_MAX_SEGMENTS: most segments of a batch given as segments
STATIC_SCRATCH_BYTES = 32 << 20   # BDLORA_STATIC_SCRATCH_BYTES: static scratch of forward_layer_static
ACT_NONE, ACT_SILU_MUL = 0, 1   # BDLORA_ACT_*: activation between the MLP's projections
# BDLORA_PATH_*: launch sequence of a forward (0: none yet)
PATHS = {0: "", 1: "decode", 2: "tile64", 3: "medium", 4: "large"}
WEIGHT_BF16, WEIGHT_INT4_G128 = 0, 1   # BDLORA_WEIGHT_*: base weight formats
_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libbdlora.so")
_LIB = None

STATUS = {0: "OK", -1: "INVALID_ARG", -2: "OOM", -3: "BAD_ADAPTER", -4: "SHAPE", -5: "HIP",
          -6: "UNSUPPORTED"}

# functions the C header declares, with ctypes signatures
_c = ctypes
_P = _c.c_void_p
_I = _c.c_int32
_IP = _c.POINTER(_c.c_int32)
_LP = _c.POINTER(_c.c_int64)


class ProjDesc(ctypes.Structure):
    _fields_ = [("kind", _c.c_int32), ("d_in", _c.c_int32), ("n_slices", _c.c_int32),
                ("slice_out", _c.c_int32 * MAX_SLICES), ("weight_format", _c.c_int32)]


class _Segs(ctypes.Structure):
    _fields_ = [("n_seg", _c.c_int32), ("start", _IP), ("len", _IP), ("slot", _IP)]


_SP = _c.POINTER(_Segs)

_SIGS = {
    "bdlora_create_pool": (_I, [_c.POINTER(ProjDesc), _I, _I, _I, _I, _c.c_int64, _I, _c.POINTER(_P)]),
    "bdlora_pool_slots": (_I, [_P, _IP]),
    "bdlora_layout_slot_bytes": (_I, [_c.POINTER(ProjDesc), _I, _I, _LP]),
    "bdlora_pack_adapter_layout": (_I, [_c.POINTER(ProjDesc), _I, _I, _I, _c.POINTER(_P), _c.POINTER(_P), _P]),
    "bdlora_destroy_pool": (_I, [_P]),
    "bdlora_load_adapter": (_I, [_P, _I, _I, _c.c_float, _c.POINTER(_P), _c.POINTER(_P)]),
    "bdlora_unload_adapter": (_I, [_P, _I]),
    "bdlora_slot_bytes": (_c.c_int64, [_P]),
    "bdlora_pack_adapter_host": (_I, [_P, _I, _c.POINTER(_P), _c.POINTER(_P), _P]),
    "bdlora_load_adapter_packed": (_I, [_P, _I, _I, _c.c_float, _P, _P]),
    "bdlora_load_adapters_packed": (_I, [_P, _I, _I, _IP, _c.POINTER(_c.c_float), _P, _P]),
    "bdlora_forward_shard": (_I, [_P, _I, _P, _P, _P, _SP, _I, _P, _P]),
    "bdlora_forward_layer": (_I, [_P, _I, _IP, _c.POINTER(_P), _c.POINTER(_P), _c.POINTER(_P), _P, _SP, _I, _P]),
    "bdlora_forward_mlp": (_I, [_P, _I, _IP, _I, _P, _c.POINTER(_P), _P, _P, _P, _SP, _I, _P]),
    "bdlora_forward_layer_static": (_I, [_P, _I, _IP, _c.POINTER(_P), _c.POINTER(_P), _c.POINTER(_P), _P, _SP, _I,
                                         _P]),
    "bdlora_build_plan": (_I, [_IP, _I, _IP, _I, _IP, _IP, _IP, _IP, _IP, _IP]),
    "bdlora_plan_device": (_I, [_P, _P, _I, _P, _P, _P, _P, _P, _P, _P]),
    "bdlora_get_device_error": (_I, [_P, _P, _IP]),
    "bdlora_pack_weight": (_I, [_P, _P, _I, _I, _P]),
    "bdlora_packed_weight_bytes": (_c.c_size_t, [_I, _I, _I]),
    "bdlora_pack_weight_int4": (_I, [_P, _P, _P, _I, _I, _P]),
    "bdlora_adapter_elems": (_I, [_c.POINTER(ProjDesc), _I, _I, _LP]),
    "bdlora_pool_size": (_I, [_c.POINTER(ProjDesc), _I, _I, _I, _I, _LP, _LP]),
    "bdlora_pool_bytes": (_I, [_P, _LP]),
    "bdlora_profile_begin": (_I, [_P, _I]),
    "bdlora_profile_end": (_I, [_P, _c.POINTER(_c.c_float), _IP]),
    "bdlora_last_path": (_I, [_P, _IP]),
    "bdlora_last_error": (_c.c_char_p, []),
}
HEADER_FUNCTIONS = tuple(_SIGS)


class BDLoRAError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """Load ``libbdlora.so`` (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2510_23346_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _LIB = L
    return _LIB


def _check(rc: int):
    if rc != 0:
        raise BDLoRAError(rc, lib().bdlora_last_error().decode())


def _descs(projs, weight_formats=None) -> Tuple[ctypes.Array, List[Tuple[int, int, Tuple[int, ...]]]]:
    norm = []
    for p in projs:
        if hasattr(p, "d_in"):               # workloads.ProjSpec or similar
            kind = ROW if getattr(p, "kind", "column") in ("row", ROW) else COLUMN
            norm.append((kind, int(p.d_in), tuple(int(s) for s in p.slices)))
        else:
            kind, d_in, slices = p
            kind = ROW if kind in ("row", ROW) else COLUMN
            norm.append((kind, int(d_in), tuple(int(s) for s in slices)))
    arr = (ProjDesc * max(1, len(norm)))()
    if weight_formats is None:
        weight_formats = [WEIGHT_BF16] * len(norm)
    elif isinstance(weight_formats, int):
        weight_formats = [weight_formats] * len(norm)
    if len(weight_formats) != len(norm):
        raise ValueError("one weight format per projection")
    for i, (kind, d_in, slices) in enumerate(norm):
        arr[i].weight_format = int(weight_formats[i])
        if not 1 <= len(slices) <= MAX_SLICES:
            raise ValueError("a projection has 1..4 slices")
        arr[i].kind = kind
        arr[i].d_in = d_in
        arr[i].n_slices = len(slices)
        for j, s in enumerate(slices):
            arr[i].slice_out[j] = s
    return arr, norm


def adapter_elems(projs, rank: int) -> int:
    arr, norm = _descs(projs)
    out = _c.c_int64()
    _check(lib().bdlora_adapter_elems(arr, len(norm), int(rank), _c.byref(out)))
    return out.value


def pool_size(projs, max_slots: int, max_rank: int, max_tokens: int) -> Tuple[int, int]:
    arr, norm = _descs(projs)
    a, b = _c.c_int64(), _c.c_int64()
    _check(lib().bdlora_pool_size(arr, len(norm), int(max_slots), int(max_rank), int(max_tokens),
                                  _c.byref(a), _c.byref(b)))
    return a.value, b.value


def pack_weight(W, W_packed=None, stream=None):
    """Pack a base weight ``W [N, K]`` (nn.Linear layout, bf16 device tensor)
    into the fragment layout forward calls take; returns the packed tensor."""
    N, K = int(W.shape[0]), int(W.shape[1])
    if W_packed is None:
        W_packed = W.new_empty((N, K))
    if tuple(W_packed.shape) != (N, K) or not W.is_contiguous() or not W_packed.is_contiguous():
        raise ValueError("W and W_packed must be contiguous [N, K] tensors")
    _check(lib().bdlora_pack_weight(_ptr(W), _ptr(W_packed), N, K, _stream_handle(stream)))
    return W_packed


def packed_weight_bytes(weight_format: int, N: int, K: int) -> int:
    """Bytes of a packed base weight (0 if the format does not take the shape)."""
    return int(lib().bdlora_packed_weight_bytes(int(weight_format), int(N), int(K)))


def pack_weight_int4(q, scales, W_packed=None, stream=None):
    """Pack an INT4 base weight for forward calls: ``q`` uint8 device tensor
    ``[N, K/2]`` (nibbles q+8, low nibble = even input), ``scales`` bf16
    ``[N, K/128]``; returns the packed uint8 tensor."""
    N, K2 = int(q.shape[0]), int(q.shape[1])
    K = 2 * K2
    nbytes = packed_weight_bytes(WEIGHT_INT4_G128, N, K)
    if nbytes == 0:
        raise ValueError("an INT4 base weight needs N a multiple of 64 and K of 128")
    if tuple(scales.shape) != (N, K // 128) or scales.element_size() != 2:
        raise ValueError(f"scales must be a 2-byte [N, K/128] = [{N}, {K // 128}] tensor")
    if q.element_size() != 1 or not q.is_contiguous() or not scales.is_contiguous():
        raise ValueError("q must be a contiguous uint8 tensor, scales contiguous")
    if W_packed is None:
        import torch
        W_packed = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    if W_packed.numel() * W_packed.element_size() < nbytes:
        raise ValueError(f"W_packed must hold {nbytes} bytes")
    _check(lib().bdlora_pack_weight_int4(_ptr(q), _ptr(scales), _ptr(W_packed), N, K, _stream_handle(stream)))
    return W_packed


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(_IP)


class Segments:
    """A batch in run-length form (``bdlora_segments``): segment ``i``
    covers tokens ``start[i] .. start[i] + len[i] - 1`` and uses adapter
    ``slot[i]`` (-1: none).  ``Segments.from_ids(ids)`` makes the maximal
    runs of a per-token id vector."""

    def __init__(self, start, length, slot):
        self.start = np.ascontiguousarray(np.asarray(start, dtype=np.int32))
        self.len = np.ascontiguousarray(np.asarray(length, dtype=np.int32))
        self.slot = np.ascontiguousarray(np.asarray(slot, dtype=np.int32))
        if not (self.start.shape == self.len.shape == self.slot.shape) or self.start.ndim != 1:
            raise ValueError("start, len and slot must be 1-D arrays of one length")
        self._c = _Segs(int(self.start.size), _i32p(self.start), _i32p(self.len), _i32p(self.slot))

    @classmethod
    def from_ids(cls, ids) -> "Segments":
        ids = np.asarray(ids, dtype=np.int64).reshape(-1)
        if ids.size == 0:
            return cls([], [], [])
        cut = np.flatnonzero(np.diff(ids) != 0) + 1
        start = np.concatenate([[0], cut])
        length = np.diff(np.concatenate([start, [ids.size]]))
        return cls(start, length, ids[start])

    @property
    def n_seg(self) -> int:
        return int(self.start.size)

    @property
    def T(self) -> int:
        return int(self.len.sum())

    def ref(self):
        return _c.byref(self._c)


def _batch(ids, segs):
    """(ids pointer, segments pointer, T) for a forward call: exactly one of
    device ``ids`` and host ``segs``."""
    if (ids is None) == (segs is None):
        raise ValueError("give exactly one of ids and segs")
    if segs is not None:
        if not isinstance(segs, Segments):
            segs = Segments.from_ids(segs)
        return 0, segs.ref(), segs.T, segs
    return _ptr(ids), None, int(ids.shape[0]), None


def layout_slot_bytes(projs, max_rank: int) -> int:
    """Bytes of one adapter slot of any pool with these projections and
    max_rank (pure host)."""
    arr, norm = _descs(projs)
    out = _c.c_int64()
    _check(lib().bdlora_layout_slot_bytes(arr, len(norm), int(max_rank), _c.byref(out)))
    return out.value


def _flat_factors(projs, rank: int, A, B):
    flatA, flatB, keep = [], [], []
    for p, (_, d_in, slices) in enumerate(projs):
        for s, n in enumerate(slices):
            a = np.ascontiguousarray(np.asarray(A[p][s]).view(np.uint16) if rank else np.zeros((d_in, 0), np.uint16))
            b = np.ascontiguousarray(np.asarray(B[p][s]).view(np.uint16) if rank else np.zeros((0, n), np.uint16))
            if a.shape != (d_in, rank) or b.shape != (rank, n):
                raise ValueError(f"adapter factor shapes {a.shape}, {b.shape} do not match "
                                 f"({d_in}, {rank}), ({rank}, {n})")
            keep += [a, b]
            flatA.append(a.ctypes.data)
            flatB.append(b.ctypes.data)
    pa = (_c.c_void_p * max(1, len(flatA)))(*flatA)
    pb = (_c.c_void_p * max(1, len(flatB)))(*flatB)
    return pa, pb, keep


def pack_adapter_layout(projs, max_rank: int, rank: int, A, B, out=None):
    """Pack one adapter into the slot layout of pools with these projections
    and max_rank, on the host without a pool or GPU; returns the uint8
    slab (``out`` if given)."""
    arr, norm = _descs(projs)
    nbytes = layout_slot_bytes(projs, max_rank)
    if out is None:
        out = np.empty(nbytes, dtype=np.uint8)
    n = out.numel() * out.element_size() if hasattr(out, "numel") else out.nbytes
    if n < nbytes:
        raise ValueError(f"out must hold {nbytes} bytes")
    ptr = out.data_ptr() if hasattr(out, "data_ptr") else out.ctypes.data
    pa, pb, keep = _flat_factors(norm, int(rank), A, B)
    _check(lib().bdlora_pack_adapter_layout(arr, len(norm), int(max_rank), int(rank), pa, pb, ptr))
    del keep
    return out


def build_plan(loaded: Sequence[int], ids: Sequence[int]):
    """Host plan (see ``bdlora_build_plan``).  Returns ``(status, vid,
    groups, perm)`` with ``groups`` a list of ``(slot, start, count)``."""
    ld = np.ascontiguousarray(np.asarray(loaded, dtype=np.int32))
    ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32))
    T = int(ids.size)
    G = max(1, min(T, ld.size))
    vid = np.empty(max(T, 1), np.int32)
    perm = np.empty(max(T, 1), np.int32)
    gs, gst, gc = (np.empty(G, np.int32) for _ in range(3))
    ng = _c.c_int32(0)
    rc = lib().bdlora_build_plan(_i32p(ld), int(ld.size), _i32p(ids) if T else None, T, _i32p(vid),
                                 _i32p(gs), _i32p(gst), _i32p(gc), _i32p(perm), _c.byref(ng))
    if rc not in (0, -3):
        _check(rc)
    n = ng.value
    groups = [(int(gs[i]), int(gst[i]), int(gc[i])) for i in range(n)]
    nperm = sum(c for _, _, c in groups)
    return rc, vid[:T].copy(), groups, perm[:nperm].copy()


def _ptr(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    raise TypeError(f"expected a device tensor or an int pointer, got {type(x)}")


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


class Pool:
    """A GPU-resident adapter pool for a fixed list of shard projections.

    ``projs``: sequence of ``(kind, d_in, slices)`` (kind "column"/"row")
    or objects with ``kind``, ``d_in`` and ``slices`` attributes.
    """

    def __init__(self, projs, max_slots: int, max_rank: int, max_tokens: int, device: int = 0,
                 weight_formats=None, pool_bytes: int = 0):
        self._arr, self.projs = _descs(projs, weight_formats)
        self.weight_formats = [int(self._arr[i].weight_format) for i in range(len(self.projs))]
        self.max_rank, self.max_tokens = int(max_rank), int(max_tokens)
        self.device = int(device)
        h = _c.c_void_p()
        _check(lib().bdlora_create_pool(self._arr, len(self.projs), int(max_slots), self.max_rank,
                                        self.max_tokens, int(pool_bytes), self.device, _c.byref(h)))
        self._h = h
        n = _c.c_int32()
        _check(lib().bdlora_pool_slots(h, _c.byref(n)))
        self.max_slots = n.value
        self.loaded = np.zeros(self.max_slots, np.int32)

    # -- lifetime ---------------------------------------------------------
    def close(self):
        if getattr(self, "_h", None):
            _check(lib().bdlora_destroy_pool(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def handle(self):
        return self._h

    @property
    def bytes(self) -> int:
        out = _c.c_int64()
        _check(lib().bdlora_pool_bytes(self._h, _c.byref(out)))
        return out.value

    # -- adapters ---------------------------------------------------------
    @property
    def slot_bytes(self) -> int:
        return int(lib().bdlora_slot_bytes(self._h))

    def pack_adapter_host(self, rank: int, A, B, out=None):
        """Pack one adapter on the host into the pool's slot layout (for a
        host-side adapter cache).  ``out``: a CPU uint8 tensor or numpy array
        of ``slot_bytes`` bytes (pinned memory makes later loads
        asynchronous); returns it."""
        if out is None:
            out = np.empty(self.slot_bytes, dtype=np.uint8)
        n = out.numel() * out.element_size() if hasattr(out, "numel") else out.nbytes
        if n < self.slot_bytes:
            raise ValueError(f"out must hold {self.slot_bytes} bytes")
        ptr = out.data_ptr() if hasattr(out, "data_ptr") else out.ctypes.data
        pa, pb, keep = _flat_factors(self.projs, int(rank), A, B)
        _check(lib().bdlora_pack_adapter_host(self._h, int(rank), pa, pb, ptr))
        del keep
        return out

    def load_adapter_packed(self, slot: int, rank: int, scale: float, slab, stream=None):
        """Enqueue the copy of a host-packed slab into ``slot`` on ``stream``
        (asynchronous for pinned memory; keep ``slab`` alive until the stream
        has passed the copy)."""
        n = slab.numel() * slab.element_size() if hasattr(slab, "numel") else slab.nbytes
        if n < self.slot_bytes:
            raise ValueError(f"slab must hold {self.slot_bytes} bytes")
        ptr = slab.data_ptr() if hasattr(slab, "data_ptr") else slab.ctypes.data
        _check(lib().bdlora_load_adapter_packed(self._h, int(slot), int(rank), float(scale), ptr,
                                                _stream_handle(stream)))
        self.loaded[int(slot)] = 1

    def load_adapters_packed(self, first_slot: int, ranks, scales, slabs, stream=None):
        """Enqueue one copy of ``len(ranks)`` host-packed slabs (back to back
        in ``slabs``) into the consecutive slots from ``first_slot``."""
        n = len(ranks)
        nbytes = slabs.numel() * slabs.element_size() if hasattr(slabs, "numel") else slabs.nbytes
        if len(scales) != n or nbytes < n * self.slot_bytes:
            raise ValueError(f"slabs must hold {n} x {self.slot_bytes} bytes, one rank and scale each")
        ptr = slabs.data_ptr() if hasattr(slabs, "data_ptr") else slabs.ctypes.data
        r = (_c.c_int32 * max(1, n))(*[int(x) for x in ranks])
        sc = (_c.c_float * max(1, n))(*[float(x) for x in scales])
        _check(lib().bdlora_load_adapters_packed(self._h, int(first_slot), n, r, sc, ptr, _stream_handle(stream)))
        self.loaded[int(first_slot):int(first_slot) + n] = 1

    def load_adapter(self, slot: int, rank: int, scale: float, A, B):
        """``A[p][s]``: uint16 bf16 bits ``[d_in, rank]``; ``B[p][s]``:
        ``[rank, slice_out]`` (paper layout), for every projection p and
        slice s of the pool."""
        pa, pb, keep = _flat_factors(self.projs, int(rank), A, B)
        _check(lib().bdlora_load_adapter(self._h, int(slot), int(rank), float(scale), pa, pb))
        self.loaded[int(slot)] = 1
        del keep

    def unload_adapter(self, slot: int):
        _check(lib().bdlora_unload_adapter(self._h, int(slot)))
        self.loaded[int(slot)] = 0

    # -- forward ----------------------------------------------------------
    def _check_io(self, p, X, W, out, T):
        if not 0 <= int(p) < len(self.projs):
            return                               # the library reports the bad index
        kind, d_in, slices = self.projs[p]
        n = sum(slices)
        if self.weight_formats[p] != WEIGHT_BF16 and hasattr(W, "shape"):
            need = packed_weight_bytes(self.weight_formats[p], n, d_in)
            if W.numel() * W.element_size() < need or not W.is_contiguous():
                raise ValueError(f"packed INT4 W must be a contiguous buffer of {need} bytes")
            W = None
        for name, t, shape in (("X", X, (T, d_in)), ("W", W, (n, d_in)), ("out", out, (T, n))):
            if hasattr(t, "shape"):
                if tuple(t.shape) != shape:
                    raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {shape}")
                if t.element_size() != 2 or not t.is_contiguous():
                    raise ValueError(f"{name} must be a contiguous 2-byte (bf16) tensor")

    def forward_shard(self, proj: int, X, W, ids, out, T: Optional[int] = None, stream=None, segs=None):
        """One projection: ``out = X W^T + scale (X A) B`` per token.  The
        adapters come as device ``ids`` or as host ``segs`` (a
        :class:`Segments` or a per-token id sequence turned into runs); pass
        ``ids=None`` with ``segs``."""
        ip, sp, T0, keep = _batch(ids, segs)
        T = T0 if T is None else int(T)
        self._check_io(proj, X, W, out, T)
        _check(lib().bdlora_forward_shard(self._h, int(proj), _ptr(X), _ptr(W), ip or None, sp, T, _ptr(out),
                                          _stream_handle(stream)))
        del keep

    def forward_layer(self, projs: Sequence[int], Xs, Ws, outs, ids, T: Optional[int] = None, stream=None,
                      segs=None):
        """Several projections sharing the token batch, in one launch set."""
        ip, sp, T0, keep = _batch(ids, segs)
        T = T0 if T is None else int(T)
        n = len(projs)
        for i, p in enumerate(projs):
            self._check_io(p, Xs[i], Ws[i], outs[i], T)
        pr = (_c.c_int32 * n)(*[int(p) for p in projs])
        xs = (_c.c_void_p * n)(*[_ptr(x) for x in Xs])
        ws = (_c.c_void_p * n)(*[_ptr(w) for w in Ws])
        os_ = (_c.c_void_p * n)(*[_ptr(o) for o in outs])
        _check(lib().bdlora_forward_layer(self._h, n, pr, xs, ws, os_, ip or None, sp, T, _stream_handle(stream)))
        del keep

    def forward_layer_static(self, projs: Sequence[int], Xs, Ws, outs, ids, T: Optional[int] = None,
                             stream=None, segs=None):
        """``forward_layer`` for decode batches (T <= DECODE_MAX_T) with its
        per-batch scratch in the library's static device array: the call
        allocates nothing.  Calls on one GPU share that array (serialize
        them)."""
        ip, sp, T0, keep = _batch(ids, segs)
        T = T0 if T is None else int(T)
        n = len(projs)
        for i, p in enumerate(projs):
            self._check_io(p, Xs[i], Ws[i], outs[i], T)
        pr = (_c.c_int32 * n)(*[int(p) for p in projs])
        xs = (_c.c_void_p * n)(*[_ptr(x) for x in Xs])
        ws = (_c.c_void_p * n)(*[_ptr(w) for w in Ws])
        os_ = (_c.c_void_p * n)(*[_ptr(o) for o in outs])
        _check(lib().bdlora_forward_layer_static(self._h, n, pr, xs, ws, os_, ip or None, sp, T,
                                                 _stream_handle(stream)))
        del keep

    def forward_mlp(self, act: int, first: Sequence[int], down: int, X, W_first, W_down, out, ids,
                    T: Optional[int] = None, stream=None, segs=None):
        """One device's share of a BD-LoRA MLP (Alg. 1): ``first`` = [proj]
        (act ACT_NONE) or [gate, up] (ACT_SILU_MUL), then the row projection
        ``down``; ``out`` is down's partial output."""
        ip, sp, T0, keep = _batch(ids, segs)
        T = T0 if T is None else int(T)
        n = len(first)
        for i, p in enumerate(first):
            self._check_io(p, X, W_first[i], None, T)
        self._check_io(down, None, W_down, out, T)
        pr = (_c.c_int32 * max(n, 1))(*[int(p) for p in first])
        ws = (_c.c_void_p * max(n, 1))(*[_ptr(w) for w in W_first])
        _check(lib().bdlora_forward_mlp(self._h, int(act), pr, int(down), _ptr(X), ws, _ptr(W_down), _ptr(out),
                                        ip or None, sp, T, _stream_handle(stream)))
        del keep

    def plan_device(self, ids, vid, gslot, gstart, gcount, perm, n_groups, T: Optional[int] = None, stream=None):
        T = int(ids.shape[0]) if T is None else int(T)
        _check(lib().bdlora_plan_device(self._h, _ptr(ids), T, _ptr(vid), _ptr(gslot), _ptr(gstart),
                                        _ptr(gcount), _ptr(perm), _ptr(n_groups), _stream_handle(stream)))

    def device_error(self, stream=None) -> int:
        f = _c.c_int32(0)
        _check(lib().bdlora_get_device_error(self._h, _stream_handle(stream), _c.byref(f)))
        return f.value

    # -- timing hooks -----------------------------------------------------
    def profile_begin(self, n: int):
        _check(lib().bdlora_profile_begin(self._h, int(n)))

    def profile_end(self) -> Tuple[List[float], int]:
        """Mean milliseconds of the four timed intervals, and the calls recorded."""
        ms = (_c.c_float * 4)()
        n = _c.c_int32()
        _check(lib().bdlora_profile_end(self._h, ms, _c.byref(n)))
        return [ms[0], ms[1], ms[2], ms[3]], n.value

    def last_path(self) -> str:
        """Launch sequence of the last forward: 'decode', 'tile64', 'medium', 'large' ('' before any)."""
        v = _c.c_int32(0)
        _check(lib().bdlora_last_path(self._h, _c.byref(v)))
        return PATHS[v.value]
