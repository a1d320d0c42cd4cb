"""CPU oracle for the DeepReduce sparse-tensor codec (arXiv 2102.03112).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only ``tests/``, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import this
package.  The heavy loops live in ``drref.c`` (plain C99, single-threaded);
this module marshals numpy arrays into it and strings the steps of one codec
round trip together in the paper's order.  It shares no code with the GPU
library and never imports it.

Parity status of each function is recorded in its docstring; every function
here is pinned by a test in ``tests/test_oracle_*.py`` against something other
than itself (a worked example from the paper, a closed form, published test
vectors, brute force, or an independent library routine).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libdrref.so")
_lib = None

OK, EINVAL, ECAPACITY = 0, -1, -2
R_NONZERO = (1 << 64) - 1  # "select every nonzero" instead of a top-r count
# index policies (Section 4; Sections 10.4, 10.5)
POLICY_P0, POLICY_RANDOM, POLICY_LEFTMOST, POLICY_MIDDLE, POLICY_RIGHTMOST = 0, 1, 2, 3, 4
NO_SLOT = 0xFFFFFFFF
# segmentation of the sorted values (Section 5)
SEG_EQUAL, SEG_CHORD = 0, 1
MAX_SEG = 4096
# value models (Section 5): polynomial, double exponential
FIT_POLY, FIT_DEXP = 0, 1
# filter layouts: every hash over the whole array, or hash j over part j of k
LAYOUT_STANDARD, LAYOUT_PARTITIONED = 0, 1
# the record header's hash id of each layout
HASH_ID = {LAYOUT_STANDARD: 1, LAYOUT_PARTITIONED: 2}
# where the sender takes the coded values (Section 4): the dense gradient g,
# or the sparsified gradient (g on the selection, 0 elsewhere)
VALUES_DENSE, VALUES_SPARSE = 0, 1


class OracleError(RuntimeError):
    pass


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build

        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    u8p = ctypes.POINTER(ctypes.c_uint8)
    u32p = ctypes.POINTER(ctypes.c_uint32)
    u64p = ctypes.POINTER(ctypes.c_uint64)
    f32p = ctypes.POINTER(ctypes.c_float)
    f64p = ctypes.POINTER(ctypes.c_double)
    u32, u64 = ctypes.c_uint32, ctypes.c_uint64
    sig = {
        "drref_murmur3_32": (u32, [u8p, u64, u32]),
        "drref_bloom_pos": (u64, [u32, u32, u64]),
        "drref_bloom_pos_many": (None, [u32p, u64, u32, u64, u64p]),
        "drref_bloom_params": (ctypes.c_int, [u64, ctypes.c_double, u64p, u32p]),
        "drref_topr": (ctypes.c_int, [f32p, u64, u64, u32p]),
        "drref_nonzero": (ctypes.c_int, [f32p, u64, u32p, u64, u64p]),
        "drref_bloom_encode": (ctypes.c_int, [u32p, u64, u64, u32, u32p]),
        "drref_bloom_query": (ctypes.c_int, [u32p, u64, u32, u64, u32p, u64, u64p]),
        "drref_part_start": (u64, [u32, u64, u32]),
        "drref_bloom_pos_layout_many": (None, [u32p, u64, u32, u64, u32, u32, u64p]),
        "drref_bloom_encode_layout": (ctypes.c_int, [u32p, u64, u64, u32, u32, u32p]),
        "drref_bloom_query_layout": (ctypes.c_int, [u32p, u64, u32, u32, u64, u32p, u64, u64p]),
        "drref_sort_desc": (ctypes.c_int, [f32p, u64, u32p]),
        "drref_lsq_fit": (ctypes.c_int, [f64p, f64p, u64, u32, f64p]),
        "drref_fit_shape": (None, [u64, u32, u32, u32p, u32p]),
        "drref_sigma_bits": (u32, [u64]),
        "drref_sigma_words": (u64, [u64]),
        "drref_curvefit_encode": (
            ctypes.c_int,
            [f32p, u64, u32, u32, f32p, f64p, u32p, u32p, u32p, u32p],
        ),
        "drref_curvefit_decode": (ctypes.c_int, [f32p, u32p, u64, u32, u32, f32p]),
        "drref_segment": (ctypes.c_int, [f32p, u64, u32, u32, u32, u64p, u32p]),
        "drref_seg_heuristic": (u32, [f32p, u64, u32]),
        "drref_curvefit_encode_seg": (
            ctypes.c_int,
            [f32p, u64, u32, u32, u32, f32p, f64p, u32p, u64p, u32p, u32p, u32p],
        ),
        "drref_curvefit_decode_seg": (ctypes.c_int, [f32p, u32p, u64, u32, u32, u64p, f32p]),
        "drref_curvefit_encode_ex": (
            ctypes.c_int,
            [f32p, u64, u32, u32, u32, u32, f32p, f64p, u32p, u64p, u32p, u32p, u32p, u32p],
        ),
        "drref_curvefit_decode_ex": (ctypes.c_int, [f32p, u32p, u64, u32, u32, u64p, u32, f32p]),
        "drref_dexp_fit": (ctypes.c_int, [f64p, f64p, u64, f64p, f64p]),
        "drref_perm": (u32, [u32, u64, u32]),
        "drref_policy_slots": (ctypes.c_int, [u64, u64, u32, u32, u32p, u64p]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _check(st: int, what: str):
    if st != OK:
        raise OracleError(f"{what}: status {st}")


# --------------------------------------------------------------------------
# hash family and Bloom parameters
# --------------------------------------------------------------------------


def murmur3_32(data: bytes, seed: int) -> int:
    """MurmurHash3_x86_32 of a byte string (Section 2 asks for k independent
    hash functions; this codec takes murmur3 with seeds 0..k-1)."""
    lib = _load()
    buf = (ctypes.c_uint8 * max(1, len(data))).from_buffer_copy(data or b"\0")
    return int(lib.drref_murmur3_32(buf, len(data), seed & 0xFFFFFFFF))


def bloom_pos(idx, j: int, m: int, k: int = 0, layout: int = LAYOUT_STANDARD) -> np.ndarray:
    """Bit positions of hash j for an array of indices: h_j(i) * m >> 32
    (standard layout), or floor(j m / k) + h_j(i) * q_j >> 32 within part j
    of size q_j (partitioned layout; needs k)."""
    lib = _load()
    idx = np.ascontiguousarray(idx, dtype=np.uint32)
    out = np.empty(idx.size, dtype=np.uint64)
    if layout == LAYOUT_STANDARD:
        lib.drref_bloom_pos_many(_ptr(idx, ctypes.c_uint32), idx.size, j, m, _ptr(out, ctypes.c_uint64))
    else:
        lib.drref_bloom_pos_layout_many(_ptr(idx, ctypes.c_uint32), idx.size, j, m, k, layout,
                                        _ptr(out, ctypes.c_uint64))
    return out


def part_start(j: int, m: int, k: int) -> int:
    """First bit of part j of a partitioned filter: floor(j m / k)."""
    return int(_load().drref_part_start(j, m, k))


def bloom_params(n: int, fpr: float) -> tuple[int, int]:
    """(m, k) from Remark 2 of Section 10.2, rounded as drref.c states."""
    lib = _load()
    m = ctypes.c_uint64()
    k = ctypes.c_uint32()
    _check(lib.drref_bloom_params(n, fpr, ctypes.byref(m), ctypes.byref(k)), "bloom_params")
    return int(m.value), int(k.value)


# --------------------------------------------------------------------------
# sparsification
# --------------------------------------------------------------------------


def ratio_count(d: int, num: int, den: int) -> int:
    """r = ceil(d * num / den) in integer arithmetic (the paper states r as a
    percentage of d, Section 6; rounding up is this codec's reading)."""
    return (d * num + den - 1) // den


def topr(g: np.ndarray, r: int) -> np.ndarray:
    """Indices of the r largest-magnitude entries, ascending (Section 10.2)."""
    lib = _load()
    g = np.ascontiguousarray(g, dtype=np.float32)
    S = np.empty(max(r, 1), dtype=np.uint32)
    _check(lib.drref_topr(_ptr(g, ctypes.c_float), g.size, r, _ptr(S, ctypes.c_uint32)), "topr")
    return S[:r]


def nonzero(g: np.ndarray) -> np.ndarray:
    """Support {i : g[i] != 0} of an inherently sparse gradient (Section 3)."""
    lib = _load()
    g = np.ascontiguousarray(g, dtype=np.float32)
    S = np.empty(max(g.size, 1), dtype=np.uint32)
    n = ctypes.c_uint64()
    _check(
        lib.drref_nonzero(_ptr(g, ctypes.c_float), g.size, _ptr(S, ctypes.c_uint32), g.size, ctypes.byref(n)),
        "nonzero",
    )
    return S[: n.value].copy()


# --------------------------------------------------------------------------
# Bloom filter
# --------------------------------------------------------------------------


def bloom_encode(S: np.ndarray, m: int, k: int, layout: int = LAYOUT_STANDARD) -> np.ndarray:
    """m-bit filter (m/32 LSB-first u32 words) holding every index of S."""
    lib = _load()
    S = np.ascontiguousarray(S, dtype=np.uint32)
    words = np.zeros(m // 32, dtype=np.uint32)
    if layout == LAYOUT_STANDARD:
        st = lib.drref_bloom_encode(_ptr(S, ctypes.c_uint32), S.size, m, k, _ptr(words, ctypes.c_uint32))
    else:
        st = lib.drref_bloom_encode_layout(_ptr(S, ctypes.c_uint32), S.size, m, k, layout,
                                           _ptr(words, ctypes.c_uint32))
    _check(st, "bloom_encode")
    return words


def bloom_query(words: np.ndarray, m: int, k: int, d: int, layout: int = LAYOUT_STANDARD) -> np.ndarray:
    """Policy P0's set P: every i in [0, d) the filter reports, ascending."""
    lib = _load()
    words = np.ascontiguousarray(words, dtype=np.uint32)
    cap = max(d, 1)
    P = np.empty(cap, dtype=np.uint32)
    n = ctypes.c_uint64()
    if layout == LAYOUT_STANDARD:
        st = lib.drref_bloom_query(_ptr(words, ctypes.c_uint32), m, k, d, _ptr(P, ctypes.c_uint32), cap,
                                   ctypes.byref(n))
    else:
        st = lib.drref_bloom_query_layout(_ptr(words, ctypes.c_uint32), m, k, layout, d, _ptr(P, ctypes.c_uint32),
                                          cap, ctypes.byref(n))
    _check(st, "bloom_query")
    return P[: n.value].copy()


# --------------------------------------------------------------------------
# curve fitting of the values
# --------------------------------------------------------------------------


def sort_desc(V: np.ndarray) -> np.ndarray:
    """perm[rank] = q: stable, signed descending order of V (Section 5)."""
    lib = _load()
    V = np.ascontiguousarray(V, dtype=np.float32)
    perm = np.empty(max(V.size, 1), dtype=np.uint32)
    _check(lib.drref_sort_desc(_ptr(V, ctypes.c_float), V.size, _ptr(perm, ctypes.c_uint32)), "sort_desc")
    return perm[: V.size]


def lsq_fit(x, y, D: int) -> np.ndarray:
    """Least-squares polynomial coefficients (increasing powers) of degree D
    through (x_j, y_j), normal equations in double (Section 5)."""
    lib = _load()
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.ascontiguousarray(y, dtype=np.float64)
    c = np.zeros(D + 1, dtype=np.float64)
    _check(lib.drref_lsq_fit(_ptr(x, ctypes.c_double), _ptr(y, ctypes.c_double), x.size, D, _ptr(c, ctypes.c_double)), "lsq_fit")
    return c


def fit_shape(n: int, D: int, S: int) -> tuple[int, int]:
    lib = _load()
    se = ctypes.c_uint32()
    de = ctypes.c_uint32()
    lib.drref_fit_shape(n, D, S, ctypes.byref(se), ctypes.byref(de))
    return int(se.value), int(de.value)


def sigma_bits(n: int) -> int:
    return int(_load().drref_sigma_bits(n))


def sigma_words(n: int) -> int:
    return int(_load().drref_sigma_words(n))


@dataclass
class FitPayload:
    coef: np.ndarray  # fp32, n_seg rows of degree+1
    coef64: np.ndarray  # the double-precision solution the fp32 rows round
    sigma: np.ndarray  # packed reorder map, u32 words
    n: int
    degree: int
    n_seg: int
    S_eff: int
    D_eff: int
    b: int
    seg_mode: int = SEG_EQUAL
    bounds: np.ndarray = None  # segment starts, S_eff + 1 entries (last = n)
    model: int = FIT_POLY  # the model used (a DEXP request on fewer than 4 values gives POLY)


def curvefit_encode(V: np.ndarray, degree: int, n_seg: int, seg_mode: int = SEG_EQUAL,
                    model: int = FIT_POLY) -> FitPayload:
    """Sort, segment, fit, and pack the reorder map (Sections 5 and 5.1).
    ``n_seg`` = 0 asks for the heuristic number of segments; ``seg_mode``
    chooses equal-count or chord segmentation (Section 5); ``model`` the
    polynomial or the double exponential (degree taken as 3: rows (a, b, c,
    d)).  The coefficient rows are n_seg (MAX_SEG for the heuristic) of
    degree+1."""
    lib = _load()
    V = np.ascontiguousarray(V, dtype=np.float32)
    n = V.size
    if model == FIT_DEXP:
        degree = 3
    cap = n_seg if n_seg else MAX_SEG
    coef = np.zeros(cap * (degree + 1), dtype=np.float32)
    coef64 = np.zeros(cap * (degree + 1), dtype=np.float64)
    sigma = np.zeros(max(sigma_words(n), 1), dtype=np.uint32)
    bounds = np.zeros(cap + 1, dtype=np.uint64)
    se, de, b, mo = ctypes.c_uint32(), ctypes.c_uint32(), ctypes.c_uint32(), ctypes.c_uint32()
    _check(
        lib.drref_curvefit_encode_ex(
            _ptr(V, ctypes.c_float), n, degree, n_seg, seg_mode, model, _ptr(coef, ctypes.c_float),
            _ptr(coef64, ctypes.c_double), _ptr(sigma, ctypes.c_uint32), _ptr(bounds, ctypes.c_uint64),
            ctypes.byref(se), ctypes.byref(de), ctypes.byref(b), ctypes.byref(mo),
        ),
        "curvefit_encode",
    )
    S_eff = int(se.value)
    return FitPayload(coef, coef64, sigma[: sigma_words(n)], n, degree, n_seg, S_eff, int(de.value), int(b.value),
                      seg_mode, bounds[: S_eff + 1].copy(), int(mo.value))


def dexp_fit(t: np.ndarray, y: np.ndarray) -> tuple[np.ndarray, float]:
    """(a, b, c, d) of the least-squares fit y ~ a e^(bt) + c e^(dt), and its
    residual sum of squares."""
    t = np.ascontiguousarray(t, dtype=np.float64)
    y = np.ascontiguousarray(y, dtype=np.float64)
    th = np.zeros(4)
    rss = ctypes.c_double()
    _check(_load().drref_dexp_fit(_ptr(t, ctypes.c_double), _ptr(y, ctypes.c_double), t.size,
                                  _ptr(th, ctypes.c_double), ctypes.byref(rss)), "dexp_fit")
    return th, float(rss.value)


def segment(C: np.ndarray, degree: int, n_seg: int, seg_mode: int) -> np.ndarray:
    """Segment starts (S_eff + 1 entries) of already sorted values C."""
    C = np.ascontiguousarray(C, dtype=np.float32)
    bounds = np.zeros(n_seg + 1, dtype=np.uint64)
    se = ctypes.c_uint32()
    _check(_load().drref_segment(_ptr(C, ctypes.c_float), C.size, degree, n_seg, seg_mode,
                                 _ptr(bounds, ctypes.c_uint64), ctypes.byref(se)), "segment")
    return bounds[: int(se.value) + 1].copy()


def seg_heuristic(C: np.ndarray, degree: int) -> int:
    """Heuristic number of segments for sorted values C (p + 1 pieces)."""
    C = np.ascontiguousarray(C, dtype=np.float32)
    return int(_load().drref_seg_heuristic(_ptr(C, ctypes.c_float), C.size, degree))


def curvefit_decode_seg(coef: np.ndarray, sigma: np.ndarray, n: int, degree: int, bounds: np.ndarray,
                        model: int = FIT_POLY) -> np.ndarray:
    """Reconstruct n values from coefficients, reorder map and segment starts."""
    lib = _load()
    coef = np.ascontiguousarray(coef, dtype=np.float32)
    sigma = np.ascontiguousarray(sigma, dtype=np.uint32)
    if sigma.size == 0:
        sigma = np.zeros(1, dtype=np.uint32)
    bounds = np.ascontiguousarray(bounds, dtype=np.uint64)
    out = np.empty(max(n, 1), dtype=np.float32)
    _check(lib.drref_curvefit_decode_ex(_ptr(coef, ctypes.c_float), _ptr(sigma, ctypes.c_uint32), n, degree,
                                        max(bounds.size - 1, 0), _ptr(bounds, ctypes.c_uint64), model,
                                        _ptr(out, ctypes.c_float)), "curvefit_decode_seg")
    return out[:n]


def curvefit_decode(coef: np.ndarray, sigma: np.ndarray, n: int, degree: int, n_seg: int) -> np.ndarray:
    """Reconstruct the n values from the coefficients and reorder map."""
    lib = _load()
    coef = np.ascontiguousarray(coef, dtype=np.float32)
    sigma = np.ascontiguousarray(sigma, dtype=np.uint32)
    if sigma.size == 0:
        sigma = np.zeros(1, dtype=np.uint32)
    out = np.empty(max(n, 1), dtype=np.float32)
    _check(
        lib.drref_curvefit_decode(_ptr(coef, ctypes.c_float), _ptr(sigma, ctypes.c_uint32), n, degree, n_seg, _ptr(out, ctypes.c_float)),
        "curvefit_decode",
    )
    return out[:n]


def sigma_unpack(sigma: np.ndarray, n: int) -> np.ndarray:
    """Read the n packed b-bit entries of a reorder map (plain bit loop)."""
    b = sigma_bits(n)
    bits = np.unpackbits(np.ascontiguousarray(sigma, dtype="<u4").view(np.uint8), bitorder="little")
    out = np.zeros(n, dtype=np.uint64)
    for t in range(b):
        out |= bits[np.arange(n, dtype=np.int64) * b + t].astype(np.uint64) << np.uint64(t)
    return out


# --------------------------------------------------------------------------
# index policies
# --------------------------------------------------------------------------


def perm(q: int, N: int, seed: int) -> int:
    """The keyed permutation of the ranks [0, N) that policy P1 uses."""
    return int(_load().drref_perm(q, N, seed))


def policy_slots(npos: int, r: int, policy: int, seed: int) -> tuple[np.ndarray, int]:
    """Value number of each positive rank (NO_SLOT when the policy drops it)
    and the number of values kept."""
    out = np.zeros(max(npos, 1), dtype=np.uint32)
    nc = ctypes.c_uint64()
    _check(_load().drref_policy_slots(npos, r, policy, seed, _ptr(out, ctypes.c_uint32), ctypes.byref(nc)),
           "drref_policy_slots")
    return out[:npos], int(nc.value)


# --------------------------------------------------------------------------
# one round trip over one tensor, in the paper's order
# --------------------------------------------------------------------------


@dataclass
class TensorResult:
    d: int
    S: np.ndarray  # selected indices (sender), ascending
    m: int
    k: int
    bits: np.ndarray  # Bloom filter words
    P: np.ndarray  # sender-side positives, ascending
    V: np.ndarray  # coded values in value order: g at the kept positives (Section 4)
    fit: FitPayload
    P_dec: np.ndarray  # receiver-side positives, from the filter words only
    vals: np.ndarray  # reconstructed value of each P_dec entry (0 where the policy dropped it)
    dense: np.ndarray | None = field(default=None)
    policy: int = 0
    seed: int = 0
    slots: np.ndarray | None = field(default=None)  # value number of each positive rank, or NO_SLOT
    value_source: int = VALUES_DENSE
    layout: int = LAYOUT_STANDARD

    def payload_bits(self) -> dict:
        """Bits that cross the network (Figure 3's container): the filter, the
        fp32 coefficients actually used, and the reorder map."""
        idx = self.m
        val = 32 * self.fit.S_eff * (self.fit.D_eff + 1) if self.fit.n else 0
        if self.fit.seg_mode == SEG_CHORD and self.fit.S_eff > 1:
            val += 32 * (self.fit.S_eff - 1)  # the interior segment starts
        sig = self.fit.n * self.fit.b if self.fit.n else 0
        return {"index": idx, "values": val, "sigma": sig}


def roundtrip_tensor(g: np.ndarray, r, fpr: float, degree: int, n_seg: int, want_dense: bool = True,
                     policy: int = POLICY_P0, seed: int = 0, seg_mode: int = SEG_EQUAL,
                     model: int = FIT_POLY, value_source: int = VALUES_DENSE,
                     layout: int = LAYOUT_STANDARD) -> TensorResult:
    """Sender: top-r (or support) -> Bloom insert -> full-range query (P) ->
    the policy keeps all of P (P0) or r of it -> V = the gradient at the kept
    positives -> curve-fit encode.  Section 4 defines P0's values on the
    sparsified gradient g~ (g on S, 0 elsewhere), so a false positive carries
    0 (``value_source=VALUES_SPARSE``); it also allows reading them from the
    dense g when the sparsifier leaves it accessible (``VALUES_DENSE``).
    Receiver: the same query from the filter words -> the same policy ->
    curve-fit decode -> scatter into a dense gradient that is zero elsewhere
    (Section 4's reconstruction).  ``layout`` is the filter layout (the
    record's hash id tells the receiver).  ``r`` is an int or R_NONZERO."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    d = g.size
    S = nonzero(g) if r == R_NONZERO else topr(g, int(r))
    m, k = bloom_params(S.size, fpr)
    bits = bloom_encode(S, m, k, layout)
    P = bloom_query(bits, m, k, d, layout)
    slots, ncoded = policy_slots(P.size, S.size, policy, seed)
    kept = slots != NO_SLOT
    if value_source == VALUES_SPARSE:
        g_src = np.zeros(d, dtype=np.float32)  # g~: g on the selection, +0 elsewhere
        g_src[S.astype(np.int64)] = g[S.astype(np.int64)]
    elif value_source == VALUES_DENSE:
        g_src = g
    else:
        raise OracleError(f"unknown value source {value_source}")
    V = np.zeros(ncoded, dtype=np.float32)
    V[slots[kept].astype(np.int64)] = g_src[P[kept].astype(np.int64)]
    fit = curvefit_encode(V, degree, n_seg, seg_mode, model)
    # receiver: its own query and the same policy over its own positives
    P_dec = bloom_query(bits, m, k, d, layout)
    slots_dec, nc_dec = policy_slots(P_dec.size, ncoded, policy, seed)
    y = curvefit_decode_seg(fit.coef, fit.sigma, nc_dec, fit.degree, fit.bounds, fit.model)
    vals = np.zeros(P_dec.size, dtype=np.float32)
    keep_dec = slots_dec != NO_SLOT
    vals[keep_dec] = y[slots_dec[keep_dec].astype(np.int64)]
    dense = None
    if want_dense:
        dense = np.zeros(d, dtype=np.float32)
        dense[P_dec.astype(np.int64)] = vals
    return TensorResult(d, S, m, k, bits, P, V, fit, P_dec, vals, dense, policy, seed, slots, value_source, layout)


def roundtrip(g: np.ndarray, offsets, ratio, fpr: float, degree: int, n_seg: int, want_dense: bool = True,
              policy: int = POLICY_P0, seed: int = 0, seg_mode: int = SEG_EQUAL, model: int = FIT_POLY,
              value_source: int = VALUES_DENSE, layout: int = LAYOUT_STANDARD):
    """Code every tensor g[offsets[t]:offsets[t+1]] independently on local
    indices.  ``ratio`` is (num, den) for top-r with r = ceil(d_t num / den),
    or None for the support of an inherently sparse gradient."""
    out = []
    for t in range(len(offsets) - 1):
        gt = g[offsets[t]: offsets[t + 1]]
        r = R_NONZERO if ratio is None else ratio_count(gt.size, ratio[0], ratio[1])
        out.append(roundtrip_tensor(gt, r, fpr, degree, n_seg, want_dense, policy, seed, seg_mode, model,
                                    value_source, layout))
    return out


def decode_sum(results_per_payload, d: int, offsets, scale: float) -> np.ndarray:
    """The receiver of a data-parallel step (Section 2, "Compressed
    distributed training via SGD": the aggregated gradient is the mean of the
    workers' compressed gradients; Section 6.4 gathers the payloads, so every
    worker decodes each of them).  ``results_per_payload[p]`` is the list of
    per-tensor results of ``roundtrip`` for worker p.  Element i of the output
    is scale * (g_0[i] + g_1[i] + ...), the terms added one at a time in fp32
    in payload order starting from +0, then multiplied by scale in fp32.
    Parity pinned by brute force over dictionaries of (index, value) pairs and
    by the one-payload and repeated-payload special cases."""
    acc = np.zeros(d, dtype=np.float32)
    for res in results_per_payload:
        dense = np.zeros(d, dtype=np.float32)
        for t, r in enumerate(res):
            dense[offsets[t]: offsets[t + 1]] = r.dense
        acc = (acc + dense).astype(np.float32)
    return (np.float32(scale) * acc).astype(np.float32)
