"""Helpers for GPU parity tests: move a Case to the device, compare results."""
from __future__ import annotations

import numpy as np
import torch

from oracle import layer as OL


def maxrel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = float(np.max(np.abs(ref))) if ref.size else 1.0
    return float(np.max(np.abs(got - ref)) / max(den, 1e-30)) if ref.size else 0.0


def to_f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def per_request_maxrel(got, ref, row_offsets) -> list:
    return [maxrel(got[row_offsets[i]:row_offsets[i + 1]], ref[row_offsets[i]:row_offsets[i + 1]])
            for i in range(len(row_offsets) - 1)]


class DevCase:
    """A test case's tensors on the GPU."""

    def __init__(self, case, device="cuda"):
        self.case = case
        self.w = {k: v.to(device).contiguous() for k, v in case.weights.items()}
        self.k = case.pool.k_cache.to(device).contiguous()
        self.v = case.pool.v_cache.to(device).contiguous()
        self.bt = case.pool.block_tables.to(device).contiguous()
        self.x = case.x.to(device).contiguous()


def cache_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def written_slots(batch, bt: np.ndarray, page=16):
    s = set()
    for i, (c, n) in enumerate(zip(batch.context_lens, batch.chunk_lens)):
        for p in range(int(c), int(c) + int(n)):
            s.add((int(bt[i][p // page]), p % page))
    return s


def check_cache_update(before: np.ndarray, after: np.ndarray, ref_after: np.ndarray, batch, bt, tol=2e-2):
    """Bytes outside the new slots unchanged bit for bit; the set of changed
    slots within the expected set; written values close to the oracle's."""
    slots = written_slots(batch, bt)
    mask = np.zeros(before.shape[0:1] + before.shape[2:3], bool)   # [page, slot]
    for pg, sl in slots:
        mask[pg, sl] = True
    full = np.broadcast_to(mask[:, None, :, None], before.shape)
    assert np.array_equal(before[~full], after[~full]), "cache bytes outside the new slots changed"
    got = OL.bf16_bits_to_f32(after[full])
    ref = OL.bf16_bits_to_f32(ref_after[full])
    assert np.isfinite(got).all(), "a new slot was not written"
    err = maxrel(got, ref)
    assert err <= tol, f"written K/V max-rel {err}"
    return err
