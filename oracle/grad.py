"""Gradient grouping path, plain NumPy — TEST INFRASTRUCTURE ONLY.

Covers the paper's grouping of gradient tensors into complete groups that
are fused into one contiguous message each (Section 4.2, Grouping; Figure
grouping) and the mixed-precision loss-scale handling that precedes the
optimizer (Section 6.2, Model Implementation: loss scaling to keep values
inside the float16 range).

Readings where the paper gives no rule (the paper's groups are user
assigned):
  * tensors are taken in backward-completion order, i.e. the reverse of
    the forward layer order for a chain network;
  * a tensor joins the open group unless its aligned end would pass the
    byte cap, in which case the open group is closed first; a tensor larger
    than the cap therefore forms a group of its own;
  * members start at multiples of ``align_bytes``; the gap is zero filled;
    a group ends at its last member's end (no trailing pad);
  * unscale multiplies each fp16 value, as a real number, by ``inv_scale``
    and rounds once to fp32 (nearest-even); the group is flagged when any
    fp16 word has an all-ones exponent field (infinity or NaN).
"""
import numpy as np

FP16_EXP_MASK = 0x7C00


def plan_groups(numels, cap_bytes, align_bytes=256, elem_bytes=2):
    """Return a list of groups, each a dict with members, offsets, numel.

    numels: element counts in completion order. Offsets are in elements.
    """
    if align_bytes % elem_bytes:
        raise ValueError("alignment must be a whole number of elements")
    align = align_bytes // elem_bytes
    groups = []
    members, offsets, end = [], [], 0
    for i, n in enumerate(numels):
        start = -(-end // align) * align  # end rounded up to the alignment
        if members and (start + n) * elem_bytes > cap_bytes:
            groups.append({"members": members, "offsets": offsets,
                           "numel": end})
            members, offsets, end, start = [], [], 0, 0
        members.append(i)
        offsets.append(start)
        end = start + n
    if members:
        groups.append({"members": members, "offsets": offsets, "numel": end})
    return groups


def pack(srcs, group):
    """Copy the members' fp16 bit patterns into one zero-padded buffer."""
    buf = np.zeros(group["numel"], dtype=np.uint16)
    for m, off in zip(group["members"], group["offsets"]):
        s = np.ascontiguousarray(srcs[m]).view(np.uint16).ravel()
        buf[off:off + s.size] = s
    return buf


def found_nonfinite(buf16):
    """True when any fp16 word is an infinity or a NaN (exponent all ones)."""
    b = np.asarray(buf16).view(np.uint16)
    return bool(np.any((b & FP16_EXP_MASK) == FP16_EXP_MASK))


def unscale(buf16, inv_scale):
    """fp32 value of (fp16 value) * inv_scale, rounded once to nearest-even.

    The product of an fp16 and an fp32 number is exact in fp64 (11 + 24
    significand bits), so forming it in fp64 and converting to fp32 is a
    single rounding of the true product.
    """
    v = np.asarray(buf16).view(np.uint16).view(np.float16).astype(np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        return (v * np.float64(np.float32(inv_scale))).astype(np.float32)


def unscale_check(buf16, inv_scale):
    return unscale(buf16, inv_scale), found_nonfinite(buf16)


def unpack(buf32, group, numels):
    """Split an fp32 group buffer back into per-tensor fp32 arrays."""
    out = {}
    for m, off in zip(group["members"], group["offsets"]):
        out[m] = np.array(buf32[off:off + numels[m]], dtype=np.float32)
    return out


def head_grad(y16, target, loss_scale):
    """Gradient of loss_scale * mean((y - t)^2) w.r.t. y, rounded to fp16.

    Computed in fp64 as loss_scale * 2 * (y - t) / numel and rounded once to
    fp16 (nearest-even, overflow to infinity).
    """
    y = np.asarray(y16).astype(np.float64)
    t = np.asarray(target).astype(np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        return (np.float64(loss_scale) * 2.0 * (y - t) / y.size).astype(np.float16)


def relu_backward(dy16, act16):
    """Gradient through a ReLU: dy where the activation is > 0, else +0."""
    a = np.asarray(act16).astype(np.float64)
    d = np.asarray(dy16).astype(np.float64)
    return np.where(a > 0, d, 0.0).astype(np.float16)
