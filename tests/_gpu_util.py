"""Helpers shared by the GPU parity tests (not collected by pytest)."""
from __future__ import annotations

import sys

import numpy as np

import oracle
from paper_2102_03112_amd import binding as B


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev_tensor(a: np.ndarray):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def sync():
    import torch

    torch.cuda.synchronize()


def host(t) -> np.ndarray:
    return t.detach().cpu().numpy()


def u64_scalar():
    import torch

    return torch.zeros(1, dtype=torch.int64, device="cuda")


def coef_close(c_gpu: np.ndarray, c_ref64: np.ndarray, rows: int, stride: int, ncoef: int, tol: float = 1e-4):
    """Norm-wise per run: ||c_gpu - c_ref||_inf <= tol ||c_ref||_inf."""
    for s in range(rows):
        a = c_gpu[s * stride: s * stride + ncoef].astype(np.float64)
        b = c_ref64[s * stride: s * stride + ncoef]
        scale = np.max(np.abs(b))
        err = np.max(np.abs(a - b)) if a.size else 0.0
        assert err <= tol * max(scale, 1e-300), f"run {s}: |dc| {err:.3e} > {tol} * {scale:.3e}"


def values_close(y_gpu: np.ndarray, y_ref: np.ndarray, ranks: np.ndarray, n: int, seff: int, tol: float = 1e-5,
                 bounds=None):
    """|dy_q| <= tol * max(|y_ref_q|, max |y_ref| over q's run).  Runs are
    of equal count, or start at `bounds` (chord segmentation)."""
    if n == 0:
        return
    ranks = ranks.astype(np.int64)
    if bounds is None:
        s = ((ranks + 1) * seff - 1) // n
    else:
        s = np.searchsorted(np.asarray(bounds, np.int64), ranks, side="right") - 1
    run_max = np.zeros(seff)
    np.maximum.at(run_max, s, np.abs(y_ref.astype(np.float64)))
    bound = tol * np.maximum(np.abs(y_ref.astype(np.float64)), run_max[s])
    err = np.abs(y_gpu.astype(np.float64) - y_ref.astype(np.float64))
    bad = np.flatnonzero(err > bound)
    assert bad.size == 0, f"{bad.size} values off, first q={bad[0]} gpu={y_gpu[bad[0]]} ref={y_ref[bad[0]]}"


def unpack_sigma(words: np.ndarray, n: int, b: int) -> np.ndarray:
    """The n packed b-bit entries of a reorder map written by the GPU (a numpy
    reader of the LSB-first layout, so that GPU output is never fed to the
    oracle)."""
    bits = np.unpackbits(np.ascontiguousarray(words, dtype="<u4").view(np.uint8), bitorder="little")
    at = np.arange(n, dtype=np.int64)[:, None] * b + np.arange(b, dtype=np.int64)[None, :]
    return (bits[at].astype(np.uint64) << np.arange(b, dtype=np.uint64)[None, :]).sum(axis=1)


def check_record(rec, ref: "oracle.TensorResult", degree: int, n_seg: int):
    """A GPU payload record against the oracle's result for the same tensor:
    bit-exact filter and reorder map, header fields, coefficients within
    1e-4 of the oracle's double-precision solution."""
    assert rec.d == ref.d
    assert rec.n_selected == ref.S.size
    assert (rec.n_positives, rec.n_values) == (ref.P.size, ref.fit.n)
    assert (rec.m_bits, rec.k, rec.hash_id) == (ref.m, ref.k, oracle.HASH_ID[ref.layout])
    assert (rec.policy, rec.seed) == (ref.policy, ref.seed)
    assert rec.seg_mode == ref.fit.seg_mode
    assert rec.model == ref.fit.model
    assert rec.value_source == ref.value_source
    if ref.fit.seg_mode == oracle.SEG_CHORD:
        np.testing.assert_array_equal(rec.knots, ref.fit.bounds[1:-1].astype(np.uint32))
    assert (rec.seg_eff, rec.deg_eff, rec.sigma_b) == (ref.fit.S_eff, ref.fit.D_eff, ref.fit.b)
    np.testing.assert_array_equal(rec.bits, ref.bits)
    np.testing.assert_array_equal(rec.sigma, ref.fit.sigma)
    nc = ref.fit.D_eff + 1
    c_gpu = rec.coef.reshape(rec.seg_eff, nc) if rec.seg_eff else rec.coef
    c_ref = ref.fit.coef64.reshape(n_seg or oracle.MAX_SEG, degree + 1)[: rec.seg_eff, :nc]
    coef_close(np.ascontiguousarray(c_gpu).ravel(), np.ascontiguousarray(c_ref).ravel(), rec.seg_eff, nc, nc)
    words = (ref.fit.n * ref.fit.b + 31) // 32
    assert rec.rec_bytes == 64 + ref.m // 8 + 4 * rec.seg_eff * nc + 4 * rec.knots.size + 4 * words


_WS = {}


def workspace(d, n_tensors=1):
    """A cached device workspace of at least dr_workspace_bytes(d, n_tensors)."""
    need = B.workspace_bytes(d, n_tensors)
    cur = _WS.get("ws")
    if cur is None or cur.numel() < need:
        _WS["ws"] = None
        import torch

        torch.cuda.empty_cache()
        _WS["ws"] = B.workspace(max(d, 1 << 20), n_tensors)
    return _WS["ws"]


def release_workspace():
    _WS.clear()
    import torch

    torch.cuda.empty_cache()


def run_roundtrip(g, cfg: B.Config):
    import torch

    total, rec_off = B.payload_layout(cfg)
    d = cfg.d
    gd = dev_tensor(g) if d else torch.zeros(1, dtype=torch.float32, device="cuda")
    payload = torch.zeros(total, dtype=torch.uint8, device="cuda")
    dense = torch.full((max(d, 1),), 9.0, dtype=torch.float32, device="cuda")
    idx = torch.full((max(d, 1),), -1, dtype=torch.int32, device="cuda")
    val = torch.zeros(max(d, 1), dtype=torch.float32, device="cuda")
    counts = torch.zeros(4 * cfg.n_tensors, dtype=torch.int64, device="cuda")
    ws = workspace(max(d, 1), cfg.n_tensors)
    B.roundtrip(gd, cfg, payload, dense, idx, val, counts, ws)
    sync()
    return dict(payload=host(payload), rec_off=rec_off, dense=host(dense)[:d], idx=host(idx)[:d].view(np.uint32),
                val=host(val)[:d], counts=host(counts).reshape(cfg.n_tensors, 4))


def check_roundtrip(g, cfg: B.Config, out, refs):
    off = cfg.offsets
    for t, ref in enumerate(refs):
        a, b = int(off[t]), int(off[t + 1])
        rec = B.parse_record(out["payload"], out["rec_off"][t])
        check_record(rec, ref, ref.fit.degree, cfg.n_seg)
        n_sel, nv, nv_dec, flags = [int(x) for x in out["counts"][t]]
        assert (n_sel, nv, nv_dec, flags) == (ref.S.size, ref.P.size, ref.P.size, 0)
        np.testing.assert_array_equal(out["idx"][a: a + nv], ref.P_dec)
        # the policy's choice: positives it did not code are received as 0
        vals = out["val"][a: a + nv]
        kept = ref.slots != oracle.NO_SLOT
        assert np.all(vals[~kept] == 0)
        nc = ref.fit.n
        assert int(kept.sum()) == nc
        if nc:
            vn = ref.slots[kept].astype(np.int64)
            y_gpu = np.zeros(nc, np.float32)
            y_gpu[vn] = vals[kept]
            y_ref = np.zeros(nc, np.float32)
            y_ref[vn] = ref.vals[kept]
            # receiver values vs the oracle's own end-to-end reconstruction
            ranks = oracle.sigma_unpack(ref.fit.sigma, nc)
            values_close(y_gpu, y_ref, ranks, nc, ref.fit.S_eff,
                         bounds=ref.fit.bounds if ref.fit.seg_mode == oracle.SEG_CHORD else None)
        dense = out["dense"][a:b]
        pos = ref.P_dec.astype(np.int64)
        np.testing.assert_array_equal(dense[pos], out["val"][a: a + nv])
        offp = np.ones(b - a, bool)
        offp[pos] = False
        assert np.all(dense[offp] == 0)


