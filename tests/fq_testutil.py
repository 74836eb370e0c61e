"""Shared helpers for the device tests: uploads, the oracle replay check, norms."""
from __future__ import annotations

import numpy as np

import oracle as O
from fq_inputs import gen


def need_gpu():
    import pytest
    import torch
    if not torch.cuda.is_available():
        pytest.fail("device tests need a GPU (run them with -m gpu on an MI355X)")
    import paper_2403_06082_amd as fq
    fq.lib()            # fails loudly if libfq.so is missing
    return torch


def upload(arr: np.ndarray, dtype: str):
    """Device tensor from a device-storage numpy array (f32 / f16 / bf16 bits)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(arr))
    if dtype == "bf16":
        t = t.view(torch.bfloat16)
    return t.cuda()


def exact_f64(arr: np.ndarray, dtype: str) -> np.ndarray:
    return gen.storage_to_f32(arr, dtype).astype(np.float64)


def rel_fro(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (den if den > 0 else 1.0))


def unpack_codes(codes_t, K_in: int) -> np.ndarray:
    w = codes_t.cpu().numpy().view(np.uint32)
    return O.unpack2(w, K_in)


def replay_rows(D_gpu: np.ndarray, Ht_gpu: np.ndarray, codes_gpu: np.ndarray, rows=None,
                bits=2, block=128, damp=0.01, clip_sigmas=2.0, codes_are_rows=False):
    """Teacher-forced oracle replay on the device's own D and H~ (stage isolation).

    The oracle runs the clip, grid and OPTQ in float64 on exactly the values the device
    consumed; where its pre-rounding value lies within 1e-6 (code units) of a rounding
    boundary it adopts the device's code, so a legitimate near-tie cannot cascade along a
    row.  rows: optional subset (rows are independent once U is fixed; mu and sigma are
    taken over the whole D).  codes_are_rows: codes_gpu holds only the rows listed."""
    D = np.asarray(D_gpu, dtype=np.float64)
    mu, sigma, lo_b, hi_b = O.clip_bounds(D, clip_sigmas)
    sel = np.arange(D.shape[0]) if rows is None else np.asarray(rows)
    Dc = O.apply_clip(D[sel], lo_b, hi_b)
    scale, zero = O.row_grid(Dc, bits)
    U, dead, _ = O.gptq_prepare(np.asarray(Ht_gpu, dtype=np.float64), damp)
    forced = codes_gpu if codes_are_rows else codes_gpu[sel]
    r = O.gptq(Dc, U, scale, zero, bits, block, dead, forced_codes=forced)
    r.update(scale=scale, zero=zero, rows=sel, mu=mu, sigma=sigma, codes_are_rows=codes_are_rows)
    return r


def check_codes(r, codes_gpu, scale_gpu, zero_gpu, words=None):
    """Codes bit-exact outside the near-tie window; scale/zero equal to the oracle's.
    The device arrays hold every row, or only the replayed rows when the replay was made
    with codes_are_rows.  words: the device's packed 2-bit words (same rows as codes_gpu),
    then compared bit for bit, pad bits included, with the oracle's packing of the
    replayed codes."""
    sel = slice(None) if r.get("codes_are_rows") else r["rows"]
    cg = codes_gpu[sel]
    mism = (r["codes"] != cg) & ~r["tie"]
    np.testing.assert_allclose(scale_gpu[sel], r["scale"], rtol=2e-7, atol=0)
    np.testing.assert_array_equal(zero_gpu[sel], r["zero"])
    assert int(mism.sum()) == 0, f"{int(mism.sum())} code mismatches outside near ties"
    if words is not None:
        np.testing.assert_array_equal(np.asarray(words).view(np.uint32)[sel], O.pack2(r["codes"]))
    return int(r["tie"].sum())


def words_of(codes_t) -> np.ndarray:
    """The device's packed code words as uint32."""
    return codes_t.cpu().numpy().view(np.uint32)
