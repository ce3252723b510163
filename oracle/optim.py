"""Optimizer update and dynamic loss scale, plain NumPy in fp64 — TEST
INFRASTRUCTURE ONLY (tests, the smoke check and the benchmark's CPU leg).

Section 6.2 (Model Implementation) trains with a layer-wise adaptive rate
(LARS: each layer's update is built from L2 norms) together with Adam
(beta1 = 0.9, beta2 = 0.999), and adapts the loss scale so that values stay
inside the float16 range (the OpenSeq2Seq loss scaling it cites). The paper
names these ingredients but not how they combine; the readings taken here:
  * weight decay is added to the gradient: g~ = g + wd * w;
  * Adam moments, bias-corrected with t = the number of applied steps
    including this one:  m = b1 m + (1 - b1) g~,  v = b2 v + (1 - b2) g~^2,
    u = (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps);
  * the layer-wise rate is the trust ratio tau = ||w|| / ||u|| over the
    layer (1 when either norm is 0), and w <- w - lr * tau * u: every
    layer's step then has norm lr * ||w||, its direction Adam's;
  * the fp16 working copy of a layer is its new w rounded to nearest-even
    fp16;
  * a step whose gradients hold a non-finite value (some group flagged by
    the unscale check) is skipped: weights, moments and t stay unchanged;
  * loss-scale backoff: a skipped step halves S (not below s_min) and
    restarts the clean count; `interval` consecutive clean steps double S
    (not above s_max);
  * learning rate: linear warm-up from the initial rate (1e-4 in the paper)
    to the peak (N times it for N ranks), then a staircase decay; the paper
    gives neither the warm-up length nor the decay interval and rate, so
    they are parameters. The step index counts applied updates from 0.
"""
import numpy as np


def lars_adam_update(w, m, v, g, t, lr, b1=0.9, b2=0.999, eps=1e-8, wd=1e-4):
    """One layer's update in fp64. w, m, v, g: arrays of one layer (w the
    fp32 master weights, g the unscaled gradient); t: the 1-based count of
    applied steps including this one. Returns (w_new, m_new, v_new, tau)."""
    w = np.asarray(w, np.float64)
    g = np.asarray(g, np.float64)
    gt = g + wd * w
    m_new = b1 * np.asarray(m, np.float64) + (1.0 - b1) * gt
    v_new = b2 * np.asarray(v, np.float64) + (1.0 - b2) * gt * gt
    u = (m_new / (1.0 - b1 ** t)) / (np.sqrt(v_new / (1.0 - b2 ** t)) + eps)
    wn = np.sqrt(np.sum(w * w))
    un = np.sqrt(np.sum(u * u))
    tau = wn / un if wn > 0 and un > 0 else 1.0
    return w - lr * tau * u, m_new, v_new, tau


def fp16_copy(w):
    """Nearest-even fp16 rounding of the new master weights."""
    with np.errstate(over="ignore"):
        return np.asarray(w, np.float64).astype(np.float32).astype(np.float16)


def loss_scale_next(scale, clean, found, interval=2000, s_min=1.0, s_max=2.0 ** 24):
    """Backoff loss scaling. Returns (new scale, new clean-step count,
    whether this step's update is applied)."""
    if found:
        return max(scale / 2.0, s_min), 0, False
    clean += 1
    if clean >= interval:
        return min(scale * 2.0, s_max), 0, True
    return scale, clean, True


def lr_at(k, base=1e-4, peak=None, warmup=0, every=0, rate=1.0):
    """Learning rate of the k-th applied update (k from 0): linear warm-up
    from base to peak over `warmup` updates, then the peak multiplied by
    rate once per `every` updates (every = 0: no decay)."""
    peak = base if peak is None else peak
    if k < warmup:
        return base + (peak - base) * (k / warmup)
    if every == 0:
        return peak
    return peak * rate ** ((k - warmup) // every)
