"""ctypes binding of libarchead.so (argument marshalling only).

Every step of the forward runs in the library's HIP kernels; this module only
turns torch tensors into pointers, sizes and the caller's stream.  It fails
loudly when the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libarchead.so")
HOST_LIB_PATH = os.path.join(_PKG, "libarchead_host.so")

ABI_VERSION = 3
OK, E_INVALID_ARG, E_MISALIGNED, E_UNSUPPORTED, E_WORKSPACE, E_HIP = range(6)
F32, BF16, F16, I32, I64, I8, U8, I5 = range(8)
INT4_V1 = 1
OP_LOGITS, OP_LOGITS_CE, OP_ARGMAX, OP_TOPK, OP_FIDELITY = 0, 1, 2, 3, 4
TOPK_MAX = 64
(LAUNCH_GEMV_BLOCKS_PER_CU, LAUNCH_GEMV_GRID, LAUNCH_DEC_BLOCKS, LAUNCH_MID_BLOCKS,
 LAUNCH_TILE_WAVES, LAUNCH_TILE_ROWS, LAUNCH_T_SPIN_LIMIT) = range(7)
NOALLOC_SCRATCH_BYTES = 4 << 20   # ARCHEAD_NOALLOC_SCRATCH_BYTES of include/archead.h


class ArcheadError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"archead status {status}: {msg}")
        self.status = status


class Desc(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_uint32), ("V", ctypes.c_int64),
                ("d", ctypes.c_int64), ("g", ctypes.c_int64),
                ("r_c", ctypes.c_int64), ("r_r", ctypes.c_int64),
                ("g_v", ctypes.c_int64), ("g_b", ctypes.c_int64),
                ("int4_encoding", ctypes.c_int32), ("scale_dtype", ctypes.c_int32),
                ("factor_dtype", ctypes.c_int32), ("core_u_dtype", ctypes.c_int32)]

    @classmethod
    def make(cls, V, d, g, rc, rr, gV=None, gB=None, abi=ABI_VERSION,
             enc=INT4_V1, scale_dtype=F16, factor_dtype=I8, core_u_dtype=I8):
        return cls(abi, V, d, g, rc, rr, d if gV is None else gV,
                   d if gB is None else gB, enc, scale_dtype, factor_dtype, core_u_dtype)


class BuildDesc(ctypes.Structure):
    """archead_build_desc: shape and parameters of a head construction."""
    _fields_ = [("abi_version", ctypes.c_uint32), ("V", ctypes.c_int64), ("d", ctypes.c_int64),
                ("N", ctypes.c_int64), ("g", ctypes.c_int64), ("r_c", ctypes.c_int64),
                ("r_r", ctypes.c_int64), ("g_b", ctypes.c_int64), ("p", ctypes.c_double),
                ("lam", ctypes.c_double), ("oversample", ctypes.c_int64),
                ("power_iters", ctypes.c_int64)]


class Ptrs(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "res_codes", "res_scales", "core_u", "core_u_scale", "core_v",
        "core_v_scale", "corr_a", "corr_a_scale", "corr_b", "corr_b_scale",
        "res_row_scales")]


_SIGS = {
    "archead_validate_desc": (ctypes.c_int, [ctypes.POINTER(Desc)]),
    "archead_create": (ctypes.c_int, [ctypes.POINTER(Desc), ctypes.POINTER(Ptrs),
                                      ctypes.POINTER(ctypes.c_void_p)]),
    "archead_destroy": (None, [ctypes.c_void_p]),
    "archead_workspace_bytes": (ctypes.c_size_t, [ctypes.c_void_p, ctypes.c_int64,
                                                  ctypes.c_int]),
    "archead_logits": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_void_p, ctypes.c_int,
                                      ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t,
                                      ctypes.c_void_p]),
    "archead_logits_ce": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_int64, ctypes.c_void_p, ctypes.c_int,
                                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_size_t, ctypes.c_void_p]),
    "archead_logits_argmax": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                             ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "archead_logit_fidelity_head": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p,
                                                   ctypes.c_int64, ctypes.c_int64,
                                                   ctypes.c_void_p, ctypes.c_int64,
                                                   ctypes.c_void_p, ctypes.c_void_p,
                                                   ctypes.c_void_p, ctypes.c_void_p,
                                                   ctypes.c_void_p, ctypes.c_size_t,
                                                   ctypes.c_void_p]),
    "archead_logits_topk": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                           ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                           ctypes.c_size_t, ctypes.c_void_p]),
    "archead_logits_noalloc": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                              ctypes.c_int64, ctypes.c_void_p, ctypes.c_int,
                                              ctypes.c_int64, ctypes.c_void_p]),
    "archead_fidelity_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int64, ctypes.c_int64]),
    "archead_logit_fidelity": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                              ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                              ctypes.c_void_p]),
    "archead_build_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(BuildDesc)]),
    "archead_build_head": (ctypes.c_int, [ctypes.POINTER(BuildDesc), ctypes.c_void_p,
                                          ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                          ctypes.c_void_p, ctypes.POINTER(Ptrs), ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                          ctypes.c_void_p]),
    "archead_set_gemv_max_m": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64]),
    "archead_get_gemv_max_m": (ctypes.c_int64, [ctypes.c_void_p]),
    "archead_set_dec_range": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64]),
    "archead_get_dec_range": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64),
                                             ctypes.POINTER(ctypes.c_int64)]),
    "archead_set_mid_range": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64]),
    "archead_get_mid_range": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64),
                                             ctypes.POINTER(ctypes.c_int64)]),
    "archead_set_timing_events": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p,
                                                 ctypes.c_void_p]),
    "archead_set_launch": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64]),
    "archead_get_launch": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int,
                                          ctypes.POINTER(ctypes.c_int64)]),
    "archead_prepared_bytes": (ctypes.c_size_t, [ctypes.c_void_p]),
    "archead_prepare": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_void_p]),
    "archead_packed_bytes": (ctypes.c_uint64, [ctypes.POINTER(Desc)]),
    "archead_pack_int4": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_void_p]),
    "archead_pack_int5": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_void_p]),
    "archead_unpack_int5": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                           ctypes.c_void_p]),
    "archead_unpack_int4": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                           ctypes.c_void_p]),
    "archead_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "archead_last_error": (ctypes.c_char_p, []),
}

HOST_SYMBOLS = ("archead_validate_desc", "archead_set_gemv_max_m", "archead_set_timing_events",
                "archead_get_gemv_max_m", "archead_set_dec_range", "archead_get_dec_range",
                "archead_set_mid_range", "archead_get_mid_range",
                "archead_set_launch", "archead_get_launch",
                "archead_packed_bytes", "archead_pack_int4", "archead_pack_int5",
                "archead_unpack_int5",
                "archead_unpack_int4", "archead_status_str", "archead_last_error")

_libs = {}


def _load(path: str, names) -> ctypes.CDLL:
    if path in _libs:
        return _libs[path]
    if not os.path.exists(path):
        raise RuntimeError(
            f"{os.path.basename(path)} is not built; run "
            "`python -m paper_2608_02703_amd.build` (or __graft_entry__.build())")
    h = ctypes.CDLL(path)
    for n in names:
        res, args = _SIGS[n]
        f = getattr(h, n)
        f.restype = res
        f.argtypes = args
    _libs[path] = h
    return h


def lib() -> ctypes.CDLL:
    """The HIP library (all entry points).  ARCHEAD_LIB may name another
    build of it (tuning experiments)."""
    return _load(os.environ.get("ARCHEAD_LIB", LIB_PATH), list(_SIGS))


def host_lib(path: Optional[str] = None) -> ctypes.CDLL:
    """A host-only build of the argument checks and packers (g++)."""
    return _load(path or HOST_LIB_PATH, HOST_SYMBOLS)


def _check(st: int, L=None):
    if st != OK:
        L = L or lib()
        raise ArcheadError(st, L.archead_last_error().decode())


def validate_desc(desc: Desc, L=None) -> int:
    L = L or lib()
    return L.archead_validate_desc(ctypes.byref(desc))


def packed_bytes(desc: Desc, L=None) -> int:
    L = L or lib()
    return int(L.archead_packed_bytes(ctypes.byref(desc)))


def pack_int4(codes: np.ndarray, L=None) -> np.ndarray:
    L = L or lib()
    c = np.ascontiguousarray(codes, dtype=np.int8)
    rows, d = c.shape
    out = np.empty((rows, d // 2), dtype=np.uint8)
    _check(L.archead_pack_int4(c.ctypes.data, rows, d, out.ctypes.data), L)
    return out


def pack_int5(codes: np.ndarray, L=None) -> np.ndarray:
    """int codes [rows, r] in [-16, 15] -> ARCHEAD_I5 words uint32 [rows, ceil(r/6)]."""
    L = L or lib()
    c = np.ascontiguousarray(codes, dtype=np.int8)
    rows, r = c.shape
    out = np.empty((rows, (r + 5) // 6), dtype=np.uint32)
    _check(L.archead_pack_int5(c.ctypes.data, rows, r, out.ctypes.data), L)
    return out


def unpack_int5(words: np.ndarray, r: int, L=None) -> np.ndarray:
    L = L or lib()
    w = np.ascontiguousarray(words, dtype=np.uint32)
    if w.shape[1] != (r + 5) // 6:
        raise ValueError("ARCHEAD_I5 rows must hold ceil(r / 6) words")
    out = np.empty((w.shape[0], r), dtype=np.int8)
    _check(L.archead_unpack_int5(w.ctypes.data, w.shape[0], r, out.ctypes.data), L)
    return out


def unpack_int4(packed: np.ndarray, d: int, L=None) -> np.ndarray:
    L = L or lib()
    p = np.ascontiguousarray(packed, dtype=np.uint8)
    rows = p.shape[0]
    if p.shape[1] * 2 != d:
        raise ValueError("packed row length must be d/2")
    out = np.empty((rows, d), dtype=np.int8)
    _check(L.archead_unpack_int4(p.ctypes.data, rows, d, out.ctypes.data), L)
    return out


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def logit_fidelity(ref, test):
    """Per-position fidelity of `test` logits to reference logits `ref`, both
    fp32 [M, V] CUDA tensors with unit column stride (archead_logit_fidelity):
    returns (kl fp32 [M], sq fp32 [M], ref_idx int64 [M], rank int64 [M]) on
    the same device, computed on the current stream."""
    import torch
    if ref.dtype != torch.float32 or test.dtype != torch.float32:
        raise TypeError("logits must be float32")
    if ref.dim() != 2 or ref.shape != test.shape:
        raise ValueError("ref and test must both be [M, V]")
    if ref.stride(1) != 1 or test.stride(1) != 1:
        raise ValueError("logit rows must be contiguous")
    M, V = ref.shape
    dev = ref.device
    kl = torch.empty(M, dtype=torch.float32, device=dev)
    sq = torch.empty(M, dtype=torch.float32, device=dev)
    idx = torch.empty(M, dtype=torch.int64, device=dev)
    rank = torch.empty(M, dtype=torch.int64, device=dev)
    L = lib()
    if M == 0:
        return kl, sq, idx, rank
    ws = torch.empty(int(L.archead_fidelity_workspace_bytes(M, V)), dtype=torch.uint8, device=dev)
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    _check(L.archead_logit_fidelity(_ptr(ref), ref.stride(0), _ptr(test), test.stride(0), M, V,
                                    _ptr(kl), _ptr(sq), _ptr(idx), _ptr(rank), _ptr(ws),
                                    ws.numel(), stream), L)
    return kl, sq, idx, rank


def build_head(W, H, rc: int, rr: int, g: int, p: float = 0.75, lam: float = 1e-3, gB=None,
               oversample: int = 8, power_iters: int = 4, seed: int = 0,
               return_factors: bool = False):
    """archead_build_head: construct a packed head on the GPU from a dense
    head W (fp32 [V, d] CUDA tensor) and calibration hidden states H (fp32
    [N, d] CUDA tensor), with the randomized SVD's Gaussian sketch drawn here
    from a seeded torch generator.  Returns a PackedHead over the written
    buffers (and the unquantized A_w, B_w as fp64 tensors when
    return_factors)."""
    import torch
    if W.dtype != torch.float32 or H.dtype != torch.float32 or W.dim() != 2 or H.dim() != 2:
        raise TypeError("W and H must be 2-D float32 tensors")
    if W.stride(1) != 1 or H.stride(1) != 1 or W.shape[1] != H.shape[1]:
        raise ValueError("W and H need unit column stride and the same width d")
    V, d = W.shape
    N = H.shape[0]
    gB = d if gB is None else gB
    dev = W.device
    desc = BuildDesc(ABI_VERSION, V, d, N, g, rc, rr, gB, p, lam, oversample, power_iters)
    L = lib()
    need = int(L.archead_build_workspace_bytes(ctypes.byref(desc)))
    if need == 0:
        raise ArcheadError(E_INVALID_ARG, "invalid construction descriptor")

    def buf(shape, dtype):
        n = int(np.prod(shape))
        return torch.zeros(shape, dtype=dtype, device=dev) if n else None
    bufs = {"res_codes": buf((V, d // 2), torch.uint8), "res_scales": buf((V, d // g), torch.float16),
            "core_u": buf((V, rc), torch.int8), "core_u_scale": buf((V,), torch.float16) if rc else None,
            "core_v": buf((rc, d), torch.int8), "core_v_scale": buf((rc, 1), torch.float16) if rc else None,
            "corr_a": buf((V, rr), torch.int8), "corr_a_scale": buf((V,), torch.float16) if rr else None,
            "corr_b": buf((rr, d), torch.int8),
            "corr_b_scale": buf((rr, d // gB), torch.float16) if rr else None,
            "res_row_scales": None}
    k = rr + oversample if rr else 0
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    omega = torch.randn((max(k, 1), d), dtype=torch.float64, device=dev, generator=gen)
    a_w = torch.empty((V, rr), dtype=torch.float64, device=dev) if (return_factors and rr) else None
    b_w = torch.empty((rr, d), dtype=torch.float64, device=dev) if (return_factors and rr) else None
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    ptrs = Ptrs(*[_ptr(bufs.get(n)) for n in PackedHead.BUFFERS])
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    _check(L.archead_build_head(ctypes.byref(desc), _ptr(W), W.stride(0), _ptr(H), H.stride(0),
                                _ptr(omega), ctypes.byref(ptrs), _ptr(a_w), _ptr(b_w), _ptr(ws),
                                ws.numel(), stream), L)
    del ws
    ph = PackedHead(V, d, g, rc, rr, bufs, d, gB)
    return (ph, a_w, b_w) if return_factors else ph


class PackedHead:
    """A packed head resident on the current GPU plus its library handle.

    ``buffers`` maps the buffer names to torch tensors on the device (the
    caller keeps ownership; the handle only borrows them).  A uint8
    ``res_scales`` selects 8-bit group scale codes, with ``res_row_scales``
    (fp16 [V]) the per-row scale; an int32 ``core_u`` of ceil(rc/6) columns
    holds ARCHEAD_I5 words (5-bit codes)."""

    BUFFERS = ("res_codes", "res_scales", "core_u", "core_u_scale", "core_v",
               "core_v_scale", "corr_a", "corr_a_scale", "corr_b", "corr_b_scale",
               "res_row_scales")

    def __init__(self, V, d, g, rc, rr, buffers: dict, gV=None, gB=None):
        import torch  # noqa: F401  (device memory only)
        self.V, self.d, self.g, self.rc, self.rr = V, d, g, rc, rr
        self.gV = d if gV is None else gV
        self.gB = d if gB is None else gB
        self.buffers = buffers
        sc = buffers.get("res_scales")
        u8 = sc is not None and str(sc.dtype) == "torch.uint8"
        cu = buffers.get("core_u")
        i5 = cu is not None and str(cu.dtype) == "torch.int32"
        self.desc = Desc.make(V, d, g, rc, rr, self.gV, self.gB, scale_dtype=U8 if u8 else F16,
                              core_u_dtype=I5 if i5 else I8)
        self.ptrs = Ptrs(*[_ptr(buffers.get(n)) for n in self.BUFFERS])
        self._lib = lib()
        h = ctypes.c_void_p()
        _check(self._lib.archead_create(ctypes.byref(self.desc), ctypes.byref(self.ptrs),
                                        ctypes.byref(h)), self._lib)
        self.handle = h
        self._ws = {}
        self._prep = None

    @classmethod
    def from_arrays(cls, h, device="cuda"):
        """Upload a head given as numpy arrays (the attributes of
        synth.HeadArrays) to ``device``."""
        import torch
        bufs = {}
        for n in cls.BUFFERS:
            a = getattr(h, n, None)
            if a is None:
                bufs[n] = None
                continue
            a = np.ascontiguousarray(a)
            if a.size == 0:
                bufs[n] = None
                continue
            if a.dtype == np.float16:
                t = torch.from_numpy(a.view(np.int16)).view(torch.float16)
            elif a.dtype == np.uint32:               # ARCHEAD_I5 words
                t = torch.from_numpy(a.view(np.int32))
            elif a.dtype == np.uint8:
                t = torch.from_numpy(a)
            else:
                t = torch.from_numpy(a.astype(np.int8, copy=False))
            bufs[n] = t.to(device)
        return cls(h.V, h.d, h.g, h.rc, h.rr, bufs, getattr(h, "gV", None),
                   getattr(h, "gB", None))

    def close(self):
        if getattr(self, "handle", None):
            self._lib.archead_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ------------------------------------------------------------------
    def set_gemv_max_m(self, m: int):
        _check(self._lib.archead_set_gemv_max_m(self.handle, m), self._lib)

    def set_dec_range(self, min_m: int, max_m: int):
        _check(self._lib.archead_set_dec_range(self.handle, min_m, max_m), self._lib)

    def set_mid_range(self, min_m: int, max_m: int):
        _check(self._lib.archead_set_mid_range(self.handle, min_m, max_m), self._lib)

    def set_launch(self, knob: int, value: int):
        """archead_set_launch: one of the LAUNCH_* settings (0, or -1 for
        LAUNCH_T_SPIN_LIMIT, restores the built-in choice)."""
        _check(self._lib.archead_set_launch(self.handle, knob, value), self._lib)

    def get_launch(self, knob: int) -> int:
        v = ctypes.c_int64()
        _check(self._lib.archead_get_launch(self.handle, knob, ctypes.byref(v)), self._lib)
        return v.value

    def force_path(self, path: str):
        """Route every M to one kernel: "dec" (MFMA decode), "mid" (several
        tokens per pass over the head), "gemv" (decode GEMV), "tiled"
        (many-token MFMA) or "auto" (the built-in choice).  Shapes a kernel
        does not support still take another one."""
        off, every = (1, 0), (1, 10 ** 9)
        dec, mid, gemv = {"dec": (every, off, -1), "mid": (off, every, -1),
                          "gemv": (off, off, 10 ** 9), "tiled": (off, off, 0),
                          "auto": ((-1, -1), (-1, -1), -1)}[path]
        self.set_dec_range(*dec)
        self.set_mid_range(*mid)
        self.set_gemv_max_m(gemv)

    def set_timing_events(self, start, stop):
        """start / stop: torch.cuda.Event objects already recorded once (so
        their HIP events exist), or None to switch timing off."""
        p0 = ctypes.c_void_p(start.cuda_event) if start is not None else None
        p1 = ctypes.c_void_p(stop.cuda_event) if stop is not None else None
        _check(self._lib.archead_set_timing_events(self.handle, p0, p1), self._lib)

    def prepare(self, enable: bool = True):
        """Keep the many-token kernel's head-derived tables in a buffer owned
        by this object (built once, on the current stream), or drop it."""
        import torch
        if not enable:
            _check(self._lib.archead_prepare(self.handle, None, 0, None), self._lib)
            self._prep = None
            return
        n = int(self._lib.archead_prepared_bytes(self.handle))
        if n == 0:
            raise ValueError("this head shape has no many-token kernel")
        dev = torch.device("cuda", torch.cuda.current_device())
        buf = torch.empty(n, dtype=torch.uint8, device=dev)
        _check(self._lib.archead_prepare(self.handle, _ptr(buf), n, self._stream(dev)),
               self._lib)
        self._prep = buf

    def prepared_bytes(self) -> int:
        """archead_prepared_bytes: size of the many-token kernel's head-derived
        tables kept by prepare() (0 where the head has no such kernel)."""
        return int(self._lib.archead_prepared_bytes(self.handle))

    def workspace_bytes(self, M: int, op: int = OP_LOGITS) -> int:
        return int(self._lib.archead_workspace_bytes(self.handle, M, op))

    def workspace(self, M: int, op: int, device):
        import torch
        n = self.workspace_bytes(M, op)
        key = (str(device), n)
        ws = self._ws.get(key)
        if ws is None:
            ws = torch.empty(max(n, 256), dtype=torch.uint8, device=device)
            self._ws = {key: ws}
        return ws

    @staticmethod
    def _stream(device):
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)

    def logits(self, x, out=None, out_dtype=None, ws=None):
        """x: torch.bfloat16 [M, d] (row stride may exceed d) on the GPU."""
        import torch
        if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
            raise ValueError("x must be a 2-D bf16 tensor with unit column stride")
        M = x.shape[0]
        if out is None:
            out = torch.empty((M, self.V), dtype=out_dtype or torch.float32,
                              device=x.device)
        code = {torch.float32: F32, torch.bfloat16: BF16}[out.dtype]
        ws = self.workspace(M, OP_LOGITS, x.device) if ws is None else ws
        _check(self._lib.archead_logits(
            self.handle, _ptr(x), M, x.stride(0), _ptr(out), code, out.stride(0),
            _ptr(ws), ws.numel(), self._stream(x.device)), self._lib)
        return out

    def logits_noalloc(self, x, out=None, out_dtype=None):
        """archead_logits_noalloc: the logits with the library's static
        workspace (no workspace tensor).  x: torch.bfloat16 [M, d] on the GPU."""
        import torch
        if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
            raise ValueError("x must be a 2-D bf16 tensor with unit column stride")
        M = x.shape[0]
        if out is None:
            out = torch.empty((M, self.V), dtype=out_dtype or torch.float32,
                              device=x.device)
        code = {torch.float32: F32, torch.bfloat16: BF16}[out.dtype]
        _check(self._lib.archead_logits_noalloc(
            self.handle, _ptr(x), M, x.stride(0), _ptr(out), code, out.stride(0),
            self._stream(x.device)), self._lib)
        return out

    def logits_argmax(self, x, idx=None, max_logit=None, ws=None):
        """Greedy next token: returns (idx int64 [M], max_logit fp32 [M]), the
        smallest vocabulary index of each token's largest logit."""
        import torch
        if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
            raise ValueError("x must be a 2-D bf16 tensor with unit column stride")
        M = x.shape[0]
        idx = torch.empty(M, dtype=torch.int64, device=x.device) if idx is None else idx
        if max_logit is None:
            max_logit = torch.empty(M, dtype=torch.float32, device=x.device)
        ws = self.workspace(M, OP_ARGMAX, x.device) if ws is None else ws
        _check(self._lib.archead_logits_argmax(
            self.handle, _ptr(x), M, x.stride(0), _ptr(idx), _ptr(max_logit), _ptr(ws),
            ws.numel(), self._stream(x.device)), self._lib)
        return idx, max_logit

    def logits_topk(self, x, k, vals=None, idx=None, ws=None):
        """Top-k selection: returns (vals fp32 [M, k], idx int64 [M, k]), each
        token's k largest logits in decreasing order, equal logits by
        increasing index (archead_logits_topk)."""
        import torch
        if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
            raise ValueError("x must be a 2-D bf16 tensor with unit column stride")
        M = x.shape[0]
        if vals is None:
            vals = torch.empty((M, k), dtype=torch.float32, device=x.device)
        if idx is None:
            idx = torch.empty((M, k), dtype=torch.int64, device=x.device)
        if idx.dim() != 2 or idx.stride(1) != 1 or vals.dim() != 2 or vals.stride(1) != 1 or \
                vals.stride(0) != idx.stride(0):
            raise ValueError("vals and idx must be 2-D with unit column stride and one row stride")
        ws = self.workspace(M, OP_TOPK, x.device) if ws is None else ws
        _check(self._lib.archead_logits_topk(
            self.handle, _ptr(x), M, x.stride(0), int(k), _ptr(vals), _ptr(idx), idx.stride(0),
            _ptr(ws), ws.numel(), self._stream(x.device)), self._lib)
        return vals, idx

    def logit_fidelity_head(self, x, dense, ws=None):
        """Fidelity of this head to a dense bf16 head [V, d] on the tokens x,
        in the head's tile pass (archead_logit_fidelity_head): returns (kl
        fp32 [M], sq fp32 [M], ref_idx int64 [M], rank int64 [M])."""
        import torch
        if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
            raise ValueError("x must be a 2-D bf16 tensor with unit column stride")
        if dense.dtype != torch.bfloat16 or dense.dim() != 2 or dense.stride(1) != 1:
            raise ValueError("dense must be a 2-D bf16 tensor with unit column stride")
        M = x.shape[0]
        kl = torch.empty(M, dtype=torch.float32, device=x.device)
        sq = torch.empty(M, dtype=torch.float32, device=x.device)
        ref_idx = torch.empty(M, dtype=torch.int64, device=x.device)
        rank = torch.empty(M, dtype=torch.int64, device=x.device)
        ws = self.workspace(M, OP_FIDELITY, x.device) if ws is None else ws
        _check(self._lib.archead_logit_fidelity_head(
            self.handle, _ptr(x), M, x.stride(0), _ptr(dense), dense.stride(0), _ptr(kl),
            _ptr(sq), _ptr(ref_idx), _ptr(rank), _ptr(ws), ws.numel(), self._stream(x.device)),
            self._lib)
        return kl, sq, ref_idx, rank

    def logits_ce(self, x, targets, ce=None, mean=None, ws=None):
        """Fused log-softmax + cross-entropy; returns (ce [M], mean [1])."""
        import torch
        if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
            raise ValueError("x must be a 2-D bf16 tensor with unit column stride")
        M = x.shape[0]
        code = {torch.int32: I32, torch.int64: I64}[targets.dtype]
        ce = torch.empty(M, dtype=torch.float32, device=x.device) if ce is None else ce
        mean = torch.empty(1, dtype=torch.float32, device=x.device) if mean is None else mean
        ws = self.workspace(M, OP_LOGITS_CE, x.device) if ws is None else ws
        _check(self._lib.archead_logits_ce(
            self.handle, _ptr(x), M, x.stride(0), _ptr(targets), code, _ptr(ce),
            _ptr(mean), _ptr(ws), ws.numel(), self._stream(x.device)), self._lib)
        return ce, mean
