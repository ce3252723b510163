"""The measurement helper fg_mfma_loop (register-only MFMA chains, the
on-chip ceiling the bench reads the convolution rates against) computes
what its header states.

With integer operands every sum is exact, and the sum of a wave's outputs
has a closed form that needs only the MFMA operand layout (lane l holds the
8 reduction elements 8*(l div 32) .. +7 of its row of A and of its column
of B): the sum of C = A B over all (i, j) is sum_k (sum_i A[i,k]) (sum_j
B[k,j]), for each of the 8 (A, B) pairs an iteration issues. Twice the
iterations give exactly twice every output; random operands give finite,
identical bits on every launch."""
import numpy as np
import pytest
import torch

import paper_1909_11150_amd as fg
from gpu_util import host

pytestmark = pytest.mark.gpu

# (A slot, B slot) of the 8 MFMAs of one iteration (B slots are 4..7)
PAIRS = [(0, 0), (1, 1), (2, 2), (3, 3), (1, 2), (2, 3), (3, 0), (0, 1)]
M32 = 0xFFFFFFFF


def _hash(t, slot, e):
    h = (t * 0x9E3779B1 + slot * 0x85EBCA77 + e * 0xC2B2AE3D) & M32
    h ^= h >> 15
    h = (h * 0x2C1B3C6D) & M32
    h ^= h >> 12
    return h


def _int_operand(t, slot):
    """(threads, 8) integer values of the operand in `slot` (mode 1)."""
    e = np.arange(8, dtype=np.uint64)[None, :]
    h = _hash(t.astype(np.uint64)[:, None], np.uint64(slot), e)
    return np.where(h & 1, 0, (h >> 1) % 5).astype(np.int64) - np.where(h & 1, 0, 2)


def _wave_total(wave, iters):
    t = np.arange(64 * wave, 64 * wave + 64)
    half = (np.arange(64) // 32)[:, None]  # lane l holds k = 8 * (l // 32) + e
    tot = 0
    for a, b in PAIRS:
        A, B = _int_operand(t, a), _int_operand(t, 4 + b)
        sa = np.stack([A[half[:, 0] == g].sum(axis=0) for g in (0, 1)]).ravel()
        sb = np.stack([B[half[:, 0] == g].sum(axis=0) for g in (0, 1)]).ravel()
        tot += int((sa * sb).sum())
    return iters * tot


def test_integer_operands_closed_form_and_linearity():
    blocks = 3
    out3 = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    out6 = torch.empty_like(out3)
    fg.mfma_loop(out3, blocks, 3, operands=1)
    fg.mfma_loop(out6, blocks, 6, operands=1)
    g3, g6 = host(out3).astype(np.float64), host(out6).astype(np.float64)
    assert np.array_equal(g6, 2 * g3)
    for wave in range(blocks * 4):
        assert g3[64 * wave:64 * wave + 64].sum() == _wave_total(wave, 3), wave
    assert np.any(g3 != 0)


def test_random_operands_are_finite_and_repeatable():
    out1 = torch.empty(512 * 256, dtype=torch.float32, device="cuda")
    out2 = torch.empty_like(out1)
    fg.mfma_loop(out1, 512, 200)
    fg.mfma_loop(out2, 512, 200)
    a, b = host(out1), host(out2)
    assert np.all(np.isfinite(a)) and np.any(a != 0)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
