"""Helpers for the GPU parity tests: device transfer and the parity metrics.

Parity rule for convolution outputs (fp16 GPU result g against the fp64
oracle o on the same fp16 inputs):
  * where fp16(o) overflows to +-inf, g must be the same infinity, and those
    entries leave the sums below;
  * rel_L2 = ||g - o|| / ||o|| <= 5e-3 and max|g - o| <= 2e-2 * RMS(o).
fp16 output rounding alone gives rel_L2 ~ 2^-11/sqrt(3) ~ 2.8e-4 and a
max error of about 2^-11 * max|o|; fp32 accumulation adds ~sqrt(K)*2^-24
relative. The bound leaves ~18x headroom on the L2 term.
"""
import numpy as np
import torch

REL_L2 = 5e-3
MAX_ABS_RMS = 2e-2


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def empty16(shape):
    return torch.empty(shape, dtype=torch.float16, device="cuda")


def conv_parity(g16, o64, what=""):
    """Assert the parity rule; return (rel_l2, max_abs/rms, n_inf)."""
    g = np.asarray(g16).astype(np.float64).ravel()
    o = np.asarray(o64, dtype=np.float64).ravel()
    assert g.shape == o.shape, (what, g.shape, o.shape)
    with np.errstate(over="ignore"):
        of16 = o.astype(np.float16).astype(np.float64)
    inf = np.isinf(of16)
    if inf.any():
        assert np.array_equal(g[inf], of16[inf]), f"{what}: overflow mismatch"
    fin = ~inf
    assert np.all(np.isfinite(g[fin])), f"{what}: non-finite output"
    d = g[fin] - o[fin]
    on = np.linalg.norm(o[fin])
    rms = np.sqrt(np.mean(o[fin] ** 2)) if fin.any() else 0.0
    rel = np.linalg.norm(d) / on if on > 0 else np.linalg.norm(d)
    mx = np.max(np.abs(d)) if d.size else 0.0
    ratio = mx / rms if rms > 0 else mx
    assert rel <= REL_L2, f"{what}: rel_L2 {rel:.3e} > {REL_L2}"
    assert ratio <= MAX_ABS_RMS, f"{what}: max_abs/RMS {ratio:.3e} > {MAX_ABS_RMS}"
    return rel, ratio, int(inf.sum())


def sample_indices(shape, n, rng, extra=()):
    """Flat indices: n random ones plus the corners and edges of the output."""
    total = int(np.prod(shape))
    idx = set(int(v) for v in rng.choice(total, size=min(n, total), replace=False))
    dims = list(shape)
    # first/last along every axis combination of the leading and trailing axes
    for a in (0, dims[0] - 1):
        for b in (0, dims[1] - 1):
            for c in (0, dims[2] - 1):
                for d in (0, dims[3] - 1):
                    idx.add(int(np.ravel_multi_index((a, b, c, d), dims)))
    idx.update(int(v) for v in extra)
    return np.array(sorted(idx), dtype=np.int64)


def workspace(desc, op):
    """Device workspace the library asks for (at least 16 bytes)."""
    import paper_1909_11150_amd as fg
    return torch.empty(max(16, fg.workspace_bytes(desc, op)), dtype=torch.uint8,
                       device="cuda")
