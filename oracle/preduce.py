"""Oracle for one step of the P-Reduce algorithm -- test infrastructure only.

What is computed (paper, Sec. 3.2, and the algorithm of Fig. 4, training
with P-Reduce):

  Step 2 (local update), for every worker i that computes this step:
      x_i <- x_i - eta * grad_i
    With the momentum optimizer the paper uses for ResNet-50 (Sec. 7.1.2,
    momentum 0.9, weight decay 1e-4), the update is the usual heavy-ball form:
      g <- grad_i + wd * x_i   (when weight decay is on)
      v_i <- mu * v_i + g ;  x_i <- x_i - eta * v_i
    or, with Nesterov momentum, x_i <- x_i - eta * (g + mu * v_i).
  Step 4 (P-Reduce of a group G, applied to every member):
      xbar_G = (1/|G|) * sum_{g in G} x_g ;  x_g <- xbar_G for g in G
    which is X <- X F^G with F^G_{ij} = 1/|G| for i, j in G and
    F^G_{uu} = 1 for u outside G (Sec. 3.2).  Disjoint groups commute and are
    applied in one step (end of Sec. 3.2).

Precision.  The paper trains in fp32 (its model sizes are quoted as fp32
bytes, Sec. 7.1.2); replicas are stored as fp32, or as bf16 with fp32
arithmetic.  The oracle therefore computes in fp32, with one fixed order of
operations so that a correct kernel can match it exactly:

  * update:   g' = fl(g + fl(wd*w)) if wd != 0; u = fl(w - fl(eta*g'));
              momentum: v' = fl(fl(mu*v) + g'), u = fl(w - fl(eta*v')), or
              Nesterov u = fl(w - fl(eta*fl(g' + fl(mu*v'))))  -- one rounding
              per operation, never a fused multiply-add;
  * group sum: s = u_{m1}; s = fl(s + u_{mj}) for members in ascending order;
  * mean:     xbar = fl(s * fl32(1/|G|))  -- the sum scaled by 1/|G|, as
              Step 4 writes it; fl32(1/k) is the fp32 rounding of the
              double 1/k;
  * bf16 storage: widen exactly (bits << 16); round once to nearest-even when
              the step stores (fused form), or after the update and again
              after the average (unfused form: a separate update call followed
              by a separate P-Reduce call, each storing its result).

Only x is averaged; momentum buffers stay private to each worker (Step 4
averages parameters only).  Workers outside every group and not updating are
left byte-for-byte unchanged (F^G_{uu} = 1).

The fp32 results are pinned to float64 statements of the same mathematics
(dense X F^G products, closed-form SGD and momentum recurrences) by the CPU
tests, within the rounding-error bounds of the fp32 order above.
"""
from __future__ import annotations

from typing import Iterable, Sequence

import numpy as np

F32 = "f32"
BF16 = "bf16"


# ---------------------------------------------------------------------------
# storage formats
# ---------------------------------------------------------------------------
def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to fp32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even).  NaN stays NaN (quieted)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    out = (b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    is_nan = (b & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    out = np.where(is_nan, (b >> np.uint32(16)) | np.uint32(0x40), out)
    return out.astype(np.uint16)


def load(stored: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == F32:
        return np.array(stored, dtype=np.float32, copy=True)
    if dtype == BF16:
        return bf16_to_f32(stored)
    raise ValueError(dtype)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == F32:
        return np.asarray(x, dtype=np.float32)
    if dtype == BF16:
        return f32_to_bf16(x)
    raise ValueError(dtype)


def inv_k(k: int) -> np.float32:
    """fl32(1/k): the double 1/k rounded once to fp32."""
    return np.float32(1.0 / k)


# ---------------------------------------------------------------------------
# Step 2: local update
# ---------------------------------------------------------------------------
def local_update(w: np.ndarray, g: np.ndarray, v: np.ndarray | None, lr: float,
                 momentum: float | None, weight_decay: float = 0.0, nesterov: bool = False):
    """One worker's update in fp32.  Returns (u, v_new); v_new is None for SGD."""
    lr32 = np.float32(lr)
    if weight_decay:
        g = g + np.float32(weight_decay) * w
    if momentum is None:
        return w - lr32 * g, None
    mu32 = np.float32(momentum)
    v_new = mu32 * v + g
    if nesterov:
        return w - lr32 * (g + mu32 * v_new), v_new
    return w - lr32 * v_new, v_new


# ---------------------------------------------------------------------------
# Step 4: P-Reduce of one group
# ---------------------------------------------------------------------------
def group_mean(values: Sequence[np.ndarray]) -> np.ndarray:
    """(1/k) * sum of the k member vectors, summed in the order given."""
    k = len(values)
    s = np.array(values[0], dtype=np.float32, copy=True)
    for x in values[1:]:
        s = s + x
    return s * inv_k(k)


def _check_schedule(n: int, groups: Sequence[Sequence[int]], active: Iterable[int]):
    seen = set()
    for g in groups:
        if len(g) == 0:
            raise ValueError("empty group")
        if list(g) != sorted(g) or len(set(g)) != len(g):
            raise ValueError(f"group {g} is not strictly ascending")
        for m in g:
            if not 0 <= m < n:
                raise ValueError(f"member {m} out of range")
            if m in seen:
                raise ValueError(f"replica {m} is in two groups of one step")
            seen.add(m)
    act = list(active)
    if len(set(act)) != len(act) or any(not 0 <= r < n for r in act):
        raise ValueError("bad active list")


def step(param: np.ndarray, grad: np.ndarray | None, mom: np.ndarray | None,
         groups: Sequence[Sequence[int]], active: Iterable[int], lr: float = 0.0,
         momentum: float | None = None, dtype: str = F32, fused: bool = True,
         weight_decay: float = 0.0, nesterov: bool = False):
    """One step on all replicas.

    param, grad, mom: arrays of shape (N, P) holding the stored values
    (float32, or uint16 bf16 bit patterns).  ``active`` are the workers that
    apply their local update this step; ``groups`` the disjoint groups whose
    P-Reduce runs in this step.  Returns new (param, mom) arrays; the inputs
    are not modified.

    fused=True: update and average in one pass, rounding to the storage type
    once.  fused=False: the update is stored first, then the P-Reduce reloads.
    """
    n = param.shape[0]
    active = sorted(active)
    _check_schedule(n, groups, active)
    new_param = param.copy()
    new_mom = None if mom is None else mom.copy()

    # Step 2 for every active worker, ascending.
    u = {}
    for r in active:
        w = load(param[r], dtype)
        g = load(grad[r], dtype)
        v = None if momentum is None else load(mom[r], dtype)
        u[r], v_new = local_update(w, g, v, lr, momentum, weight_decay, nesterov)
        if v_new is not None:
            new_mom[r] = store(v_new, dtype)
    if not fused:
        for r in active:
            new_param[r] = store(u[r], dtype)
            u[r] = load(new_param[r], dtype)

    # Step 4 for every scheduled group; members that did not update this step
    # contribute their stored value.
    for g in groups:
        vals = [u[m] if m in u else load(param[m], dtype) for m in g]
        mean = group_mean(vals)
        for m in g:
            u[m] = mean

    for r, x in u.items():
        new_param[r] = store(x, dtype)
    return new_param, new_mom


def preduce(param: np.ndarray, groups: Sequence[Sequence[int]], dtype: str = F32) -> np.ndarray:
    """Pure P-Reduce (no local update) of every group."""
    out, _ = step(param, None, None, groups, [], dtype=dtype)
    return out


def run(param0: np.ndarray, mom0: np.ndarray | None, grad_fn, schedule: Sequence,
        lr: float, momentum: float | None, dtype: str = F32, fused: bool = True,
        weight_decay: float = 0.0, nesterov: bool = False):
    """A trajectory: ``schedule[t] = (active, groups)``; ``grad_fn(t)`` returns
    the (N, P) stored gradients of step t.  Returns final (param, mom)."""
    p, v = param0, mom0
    for t, (active, groups) in enumerate(schedule):
        p, v = step(p, grad_fn(t), v, groups, active, lr, momentum, dtype, fused,
                    weight_decay, nesterov)
    return p, v
