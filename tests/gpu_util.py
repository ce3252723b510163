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
import pytest
import torch

from oracle import optim as O

REL_L2 = 5e-3
MAX_ABS_RMS = 2e-2

# the optimizer hyperparameters of Section 6.2 (Adam betas, weight decay)
OPT_HP = dict(beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-4)


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


def check_opt_layer(w0, m0, v0, g0, t, lr, w1, m1, v1, h1, hp=OPT_HP):
    """One layer of lars_adam_update from (w0, m0, v0, g0) at step t against
    the fp64 oracle: moments to a few fp32 roundings of each term, the step
    as lr * tau * u of the stored moments, tau within 1e-4 of the oracle's,
    the fp16 copy bit for bit."""
    # the kernel's inputs are the fp32 values of the hyperparameters
    f = lambda x: float(np.float32(x))
    b1, b2, eps, wd = f(hp["beta1"]), f(hp["beta2"]), f(hp["eps"]), f(hp["weight_decay"])
    lr = f(lr)
    rw, rm, rv, tau = O.lars_adam_update(w0, m0, v0, g0, t, lr, b1=b1, b2=b2, eps=eps, wd=wd)
    # moments: a few fp32 roundings of each term (b1 m and (1-b1) g~ may cancel)
    w0d, g0d = w0.astype(np.float64), g0.astype(np.float64)
    gt = g0d + wd * w0d
    ulp = 2.0 ** -24
    mb = 8 * ulp * (b1 * np.abs(m0) + (1 - b1) * np.abs(gt)) + 1e-38
    assert (np.abs(m1 - rm) <= mb).all(), float((np.abs(m1 - rm) / mb).max())
    vb = 8 * ulp * (b2 * v0 + (1 - b2) * gt * gt) + 1e-38
    assert (np.abs(v1 - rv) <= vb).all(), float((np.abs(v1 - rv) / vb).max())
    # the applied step is lr * tau * u of the stored moments, tau = ||w|| / ||u||
    m1d, v1d = m1.astype(np.float64), v1.astype(np.float64)
    u = (m1d / (1 - b1 ** t)) / (np.sqrt(v1d / (1 - b2 ** t)) + eps)
    tg = np.linalg.norm(w0d) / np.linalg.norm(u) if np.linalg.norm(w0d) > 0 else 1.0
    assert tg == pytest.approx(tau, rel=1e-4)
    step = lr * tg * u
    err = np.abs(w1.astype(np.float64) - (w0d - step))
    bound = 1e-5 * np.abs(step) + np.abs(w0d - step) * 2.0 ** -23 + 1e-38
    assert (err <= bound).all(), float((err / bound).max())
    assert np.array_equal(h1.view(np.uint16), O.fp16_copy(w1).view(np.uint16))


def _dist(a, b):
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    d = a - b
    rel = np.linalg.norm(d) / max(np.linalg.norm(b), 1e-30)
    ratio = np.max(np.abs(d)) / max(np.sqrt(np.mean(b ** 2)), 1e-30)
    return rel, ratio


def chain_report(g16, o16, o64, what):
    """A chained output against the oracle chain run from the same seeded
    inputs (O16: fp16 storage at layer boundaries, O64: fp64 throughout).
    Printed only: per-op differences (last bits, a ReLU decision on a value
    within an ulp of zero) propagate down a chain, so chains are reported and
    every op is gated on its own GPU inputs instead."""
    g = np.asarray(g16, np.float64)
    assert np.all(np.isfinite(g)), what
    rel, ratio = _dist(g, o16)
    rel_n, ratio_n = _dist(o16, o64)
    print(f"{what} (chain): rel_L2 {rel:.3e} (fp16 storage {rel_n:.3e}), "
          f"max_abs/RMS {ratio:.3e} (fp16 storage {ratio_n:.3e})")
    return rel, ratio


def chain_parity(g16, o16, o64, t32, what):
    """Chained outputs: rel_L2(GPU, O16) <= max(5e-3, 2 * fp16 noise), the
    noise being the larger of rel_L2(O16, O64) and rel_L2(T32, O16) (t32 may
    be None); the largest single difference is printed, not gated."""
    assert np.all(np.isfinite(np.asarray(g16, np.float64))), what
    rel, ratio = _dist(g16, o16)
    rel_n, ratio_n = _dist(o16, o64)
    if t32 is not None:
        rel_n = max(rel_n, _dist(t32, o16)[0])
    print(f"{what}: rel_L2 {rel:.3e} (fp16 noise {rel_n:.3e}), "
          f"max_abs/RMS {ratio:.3e} (fp16 noise {ratio_n:.3e})")
    assert rel <= max(5e-3, 2 * rel_n), \
        f"{what}: rel_L2 {rel:.3e} (fp16 noise {rel_n:.3e})"
    return rel, ratio
