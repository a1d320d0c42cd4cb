"""ctypes binding of libdeepreduce.so (include/deepreduce.h).

Argument marshalling only: every function below passes torch device tensors'
pointers and the current HIP stream to the C ABI entry point of the same name
and raises ``DeepReduceError`` on a non-OK status.  No step of the codec runs
here.  The library must be built (``python -m paper_2102_03112_amd.build``);
``lib()`` raises if it is missing.
"""
from __future__ import annotations

import ctypes
import os
import struct
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdeepreduce.so")

DR_OK, DR_EINVAL, DR_ECAPACITY, DR_EDEVICE, DR_ENOTSUP = 0, -1, -2, -3, -4
R_NONZERO = (1 << 64) - 1
FLAG_NONFINITE, FLAG_DEC_MISMATCH, FLAG_COUNT, FLAG_CAPACITY, FLAG_STALLED = 1, 2, 4, 8, 16
VALUES_DENSE, VALUES_SPARSE = 0, 1
FILTER_STANDARD, FILTER_PARTITIONED = 0, 1
HEADER_BYTES = 64
HEADER_MAGIC = 0x31435244

EXPORTS = [
    "dr_bloom_params", "dr_sigma_bits", "dr_workspace_bytes", "dr_last_error", "dr_sparsify_topr",
    "dr_bloom_encode", "dr_bloom_decode", "dr_curvefit_encode", "dr_curvefit_decode", "dr_payload_layout",
    "dr_payload_encode", "dr_payload_decode", "dr_payload_decode_sum", "dr_roundtrip", "dr_trace_begin",
    "dr_trace_end", "dr_check_ranges", "dr_roundtrip_static",
]


class DeepReduceError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


class DrConfig(ctypes.Structure):
    _fields_ = [
        ("n_tensors", ctypes.c_uint64),
        ("offsets_h", ctypes.POINTER(ctypes.c_uint64)),
        ("ratio_num", ctypes.c_uint64),
        ("ratio_den", ctypes.c_uint64),
        ("fpr", ctypes.c_double),
        ("degree", ctypes.c_uint32),
        ("n_seg", ctypes.c_uint32),
        ("policy", ctypes.c_uint32),
        ("seed", ctypes.c_uint32),
        ("segmentation", ctypes.c_uint32),
        ("fit_model", ctypes.c_uint32),
        ("value_source", ctypes.c_uint32),
        ("filter_layout", ctypes.c_uint32),
    ]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2102_03112_amd.build`")
    # torch carries its own HIP runtime; loading it first makes the library
    # bind to that same runtime, so torch's device pointers and streams are
    # valid in the library's calls
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    vp, u32, u64, sz, st = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_size_t, ctypes.c_int
    cfgp = ctypes.POINTER(DrConfig)
    sig = {
        "dr_bloom_params": (st, [u64, ctypes.c_double, ctypes.POINTER(u64), ctypes.POINTER(u32)]),
        "dr_sigma_bits": (u32, [u64]),
        "dr_workspace_bytes": (sz, [u64, u64]),
        "dr_last_error": (ctypes.c_char_p, []),
        "dr_sparsify_topr": (st, [vp, u64, u64, vp, vp, vp, vp, sz, vp]),
        "dr_bloom_encode": (st, [vp, vp, u64, u64, u32, vp, vp, vp, sz, vp]),
        "dr_bloom_decode": (st, [vp, u64, u32, u64, vp, u64, vp, vp, sz, vp]),
        "dr_curvefit_encode": (st, [vp, vp, u64, u32, u32, vp, vp, vp, vp, sz, vp]),
        "dr_curvefit_decode": (st, [vp, vp, vp, u64, u32, u32, vp, vp, vp, sz, vp]),
        "dr_payload_layout": (sz, [cfgp, ctypes.POINTER(u64)]),
        "dr_payload_encode": (st, [vp, cfgp, vp, sz, vp, vp, sz, vp]),
        "dr_payload_decode": (st, [vp, cfgp, vp, vp, vp, vp, vp, sz, vp]),
        "dr_payload_decode_sum": (st, [ctypes.POINTER(vp), u32, cfgp, ctypes.c_float, vp, vp, vp, sz, vp]),
        "dr_roundtrip": (st, [vp, cfgp, vp, sz, vp, vp, vp, vp, vp, sz, vp]),
        "dr_trace_begin": (st, [vp]),
        "dr_trace_end": (st, [ctypes.c_char_p, sz]),
        "dr_check_ranges": (st, [cfgp, ctypes.POINTER(u64)]),
        "dr_roundtrip_static": (st, [vp, cfgp, vp, sz, vp, vp, vp, vp, vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def last_error() -> str:
    return lib().dr_last_error().decode()


def _check(fn: str, status: int):
    if status != DR_OK:
        raise DeepReduceError(fn, status, last_error())


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream=None):
    import torch

    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


# ---------------------------------------------------------------------------
# host-only helpers
# ---------------------------------------------------------------------------


def bloom_params(n_items: int, fpr: float) -> tuple[int, int]:
    m = ctypes.c_uint64()
    k = ctypes.c_uint32()
    _check("dr_bloom_params", lib().dr_bloom_params(n_items, fpr, ctypes.byref(m), ctypes.byref(k)))
    return int(m.value), int(k.value)


def sigma_bits(n: int) -> int:
    return int(lib().dr_sigma_bits(n))


def workspace_bytes(d: int, n_tensors: int = 1) -> int:
    return int(lib().dr_workspace_bytes(d, n_tensors))


def workspace(d: int, n_tensors: int = 1, device="cuda"):
    """A device scratch buffer of dr_workspace_bytes(d, n_tensors) bytes."""
    import torch

    ws = torch.empty(workspace_bytes(d, n_tensors) + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:]


# ---------------------------------------------------------------------------
# the codec's entry points
# ---------------------------------------------------------------------------


def sparsify_topr(g, r: int, idx_out, val_out, n_out, ws, stream=None):
    _check("dr_sparsify_topr", lib().dr_sparsify_topr(
        _ptr(g), g.numel(), r, _ptr(idx_out), _ptr(val_out), _ptr(n_out), _ptr(ws), ws.numel(), _stream(stream)))


def bloom_encode(idx, n_dev, n_cap: int, m_bits: int, k: int, bits_out, ws, stream=None, flags_out=None):
    _check("dr_bloom_encode", lib().dr_bloom_encode(
        _ptr(idx), _ptr(n_dev), n_cap, m_bits, k, _ptr(bits_out), _ptr(flags_out), _ptr(ws), ws.numel(),
        _stream(stream)))


def bloom_decode(bits, m_bits: int, k: int, d: int, idx_out, cap: int, n_out, ws, stream=None):
    _check("dr_bloom_decode", lib().dr_bloom_decode(
        _ptr(bits), m_bits, k, d, _ptr(idx_out), cap, _ptr(n_out), _ptr(ws), ws.numel(), _stream(stream)))


def curvefit_encode(vals, n_dev, n_cap: int, degree: int, n_seg: int, coef_out, sigma_out, ws, stream=None,
                    flags_out=None):
    _check("dr_curvefit_encode", lib().dr_curvefit_encode(
        _ptr(vals), _ptr(n_dev), n_cap, degree, n_seg, _ptr(coef_out), _ptr(sigma_out), _ptr(flags_out), _ptr(ws),
        ws.numel(), _stream(stream)))


def curvefit_decode(coef, sigma, n_dev, n_cap: int, degree: int, n_seg: int, vals_out, ws, stream=None,
                    flags_out=None):
    _check("dr_curvefit_decode", lib().dr_curvefit_decode(
        _ptr(coef), _ptr(sigma), _ptr(n_dev), n_cap, degree, n_seg, _ptr(vals_out), _ptr(flags_out), _ptr(ws),
        ws.numel(), _stream(stream)))


class Config:
    """A dr_config together with the host offsets array it points to."""

    def __init__(self, offsets, ratio, fpr: float, degree: int, n_seg: int, policy: int = 0, seed: int = 0,
                 segmentation: int = 0, fit_model: int = 0, value_source: int = VALUES_DENSE,
                 filter_layout: int = FILTER_STANDARD):
        self.offsets = np.ascontiguousarray(np.asarray(offsets, dtype=np.uint64))
        self._off_c = (ctypes.c_uint64 * self.offsets.size)(*[int(x) for x in self.offsets])
        num, den = (R_NONZERO, 1) if ratio is None else ratio
        self.c = DrConfig(self.offsets.size - 1, self._off_c, num, den, fpr, degree, n_seg, policy, seed,
                          segmentation, fit_model, value_source, filter_layout)
        self.ratio, self.fpr, self.degree, self.n_seg = ratio, fpr, degree, n_seg
        self.policy, self.seed, self.segmentation, self.fit_model = policy, seed, segmentation, fit_model
        self.value_source = value_source
        self.filter_layout = filter_layout

    @property
    def n_tensors(self) -> int:
        return self.offsets.size - 1

    @property
    def d(self) -> int:
        return int(self.offsets[-1])

    @classmethod
    def from_workload(cls, w, policy: int = 0, seed: int = 0, segmentation: int = 0, n_seg=None, fit_model: int = 0,
                      value_source: int = VALUES_DENSE, filter_layout: int = FILTER_STANDARD):
        return cls(w.offsets(), w.ratio, w.fpr, w.degree, w.n_seg if n_seg is None else n_seg, policy, seed,
                   segmentation, fit_model, value_source, filter_layout)


def check_ranges(cfg: Config) -> tuple[int, str]:
    """Host-only: the number of kernel index ranges of cfg's plan that would
    leave their buffers, and the first one's description."""
    v = ctypes.c_uint64()
    _check("dr_check_ranges", lib().dr_check_ranges(ctypes.byref(cfg.c), ctypes.byref(v)))
    return int(v.value), last_error()


def payload_layout(cfg: Config) -> tuple[int, list]:
    off = (ctypes.c_uint64 * (cfg.n_tensors + 1))()
    total = int(lib().dr_payload_layout(ctypes.byref(cfg.c), off))
    if total == 0:
        raise DeepReduceError("dr_payload_layout", DR_EINVAL, last_error())
    return total, [int(x) for x in off]


def payload_encode(g, cfg: Config, payload, counts_out, ws, stream=None):
    _check("dr_payload_encode", lib().dr_payload_encode(
        _ptr(g), ctypes.byref(cfg.c), _ptr(payload), payload.numel(), _ptr(counts_out), _ptr(ws), ws.numel(),
        _stream(stream)))


def payload_decode(payload, cfg: Config, dense_out, idx_out, val_out, counts_out, ws, stream=None):
    _check("dr_payload_decode", lib().dr_payload_decode(
        _ptr(payload), ctypes.byref(cfg.c), _ptr(dense_out), _ptr(idx_out), _ptr(val_out), _ptr(counts_out),
        _ptr(ws), ws.numel(), _stream(stream)))


def payload_decode_sum(payloads, cfg: Config, scale: float, dense_out, counts_out, ws, stream=None):
    """dense_out = scale * (sum of the dense gradients the payloads decode to)."""
    arr = (ctypes.c_void_p * max(1, len(payloads)))(*[_ptr(p) for p in payloads])
    _check("dr_payload_decode_sum", lib().dr_payload_decode_sum(
        arr, len(payloads), ctypes.byref(cfg.c), scale, _ptr(dense_out), _ptr(counts_out), _ptr(ws), ws.numel(),
        _stream(stream)))


def roundtrip(g, cfg: Config, payload, dense_out, idx_out, val_out, counts_out, ws, stream=None):
    _check("dr_roundtrip", lib().dr_roundtrip(
        _ptr(g), ctypes.byref(cfg.c), _ptr(payload), payload.numel(), _ptr(dense_out), _ptr(idx_out),
        _ptr(val_out), _ptr(counts_out), _ptr(ws), ws.numel(), _stream(stream)))


def roundtrip_static(g, cfg: Config, payload, dense_out, idx_out, val_out, counts_out, stream=None):
    """dr_roundtrip with the library's static scratch instead of a workspace."""
    _check("dr_roundtrip_static", lib().dr_roundtrip_static(
        _ptr(g), ctypes.byref(cfg.c), _ptr(payload), payload.numel(), _ptr(dense_out), _ptr(idx_out),
        _ptr(val_out), _ptr(counts_out), _stream(stream)))


def trace_begin(stream=None):
    _check("dr_trace_begin", lib().dr_trace_begin(_stream(stream)))


def trace_end() -> dict:
    """{kernel: (launches, total_ms)} for the kernels launched since trace_begin."""
    buf = ctypes.create_string_buffer(1 << 16)
    _check("dr_trace_end", lib().dr_trace_end(buf, len(buf)))
    out = {}
    for line in buf.value.decode().splitlines():
        name, cnt, ms = line.rsplit(" ", 2)
        out[name] = (int(cnt), float(ms))
    return out


# ---------------------------------------------------------------------------
# reading a payload container on the host
# ---------------------------------------------------------------------------


@dataclass
class Record:
    d: int
    n_selected: int
    n_positives: int
    n_values: int
    m_bits: int
    k: int
    hash_id: int
    policy: int
    seed: int
    deg_eff: int
    seg_eff: int
    sigma_b: int
    rec_bytes: int
    seg_mode: int
    model: int
    value_source: int
    bits: np.ndarray
    coef: np.ndarray
    knots: np.ndarray  # starts of runs 1 .. S_eff-1 (chord segmentation), else empty
    sigma: np.ndarray


def parse_record(buf: bytes | np.ndarray, start: int) -> Record:
    """Split one payload record (header layout in include/deepreduce.h)."""
    b = np.asarray(buf, dtype=np.uint8)
    hdr = bytes(b[start:start + HEADER_BYTES])
    (magic, hbytes, d, n_sel, n_pos, n_v, m_bits, k, hid, pol, seed, de, se, sb, rb,
     seg) = struct.unpack("<16I", hdr)
    if magic != HEADER_MAGIC or hbytes != HEADER_BYTES:
        raise ValueError(f"bad record header at {start}")
    at = start + HEADER_BYTES
    bits = b[at: at + m_bits // 8].view("<u4").copy()
    at += m_bits // 8
    ncoef = se * (de + 1)
    coef = b[at: at + 4 * ncoef].view("<f4").copy()
    at += 4 * ncoef
    seg, model, vsrc = seg & 0xFF, (seg >> 8) & 0xFF, seg >> 16
    nkn = se - 1 if seg == 1 and se > 1 else 0
    knots = b[at: at + 4 * nkn].view("<u4").copy()
    at += 4 * nkn
    nw = (n_v * sb + 31) // 32
    sigma = b[at: at + 4 * nw].view("<u4").copy()
    return Record(d, n_sel, n_pos, n_v, m_bits, k, hid, pol, seed, de, se, sb, rb, seg, model, vsrc, bits, coef,
                  knots, sigma)
