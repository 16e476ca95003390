"""Step-set policies of 0/1 Adam and the communication they cost (host only).

The optimizer takes its variance-update set T_v and synchronisation set T_u
as explicit step lists (``zo_config.tv`` / ``tu``).  This module builds them
with the policies of the paper's experiments (Section 7, "Policy for T_v and
T_u") and counts what a schedule communicates, the accounting behind the
paper's bits-per-parameter and communication-round comparison (Figure 4).

Policies:

* ``tv_kappa``: the j-th variance update at step k_j with
  k_{j+1} - k_j = 2^floor(j / kappa) (kappa = 16 in the paper): the gaps
  double every kappa updates, following the roughly exponential decay of the
  variance change between steps.
* ``tu_doubling``: the sync interval t_{j+1} - t_j is 1 during the
  learning-rate warm-up and doubles each time the learning rate has halved
  (a fixed period for an exponential decay), clipped at H = 16.
* ``tu_inverse_lr``: the same idea for any learning-rate sequence: the
  interval chosen at a sync step is the power of two nearest below
  gamma_ref / gamma_t (gamma_ref the largest rate), clipped to [1, H].
* ``freeze_variance``: the variance is no longer updated inside a sync
  interval longer than one step (the paper stops updating v once
  t_{j+1} - t_j > 1).
"""
import math

__all__ = ["tv_kappa", "tu_doubling", "tu_inverse_lr", "freeze_variance", "communication",
           "one_bit_adam_communication"]


def tv_kappa(T, kappa=16, first=0):
    """Variance-update steps below T: k_0 = first, k_{j+1} = k_j + 2^floor(j/kappa)."""
    if kappa <= 0:
        raise ValueError("kappa must be positive")
    out, k, j = [], first, 0
    while k < T:
        out.append(k)
        k += 2 ** (j // kappa)
        j += 1
    return out


def _sync_steps(T, interval_at):
    out, t = [], 0
    while t < T:
        out.append(t)
        t += interval_at(t)
    return out


def tu_doubling(T, warmup, period, H=16):
    """Sync steps below T: every step while t < warmup; afterwards the
    interval is 2^floor((t - warmup) / period), clipped at H."""
    if warmup < 0 or period <= 0 or H < 1:
        raise ValueError("bad policy parameters")

    def interval(t):
        if t < warmup:
            return 1
        return min(H, 2 ** ((t - warmup) // period))
    return _sync_steps(T, interval)


def tu_inverse_lr(gammas, H=16):
    """Sync steps for the learning rates gammas[0..T-1]: at a sync step t the
    next interval is the largest power of two <= gamma_ref / gamma_t
    (gamma_ref = max gamma), clipped to [1, H]."""
    T = len(gammas)
    if T == 0:
        return []
    ref = max(float(g) for g in gammas)
    if not ref > 0:
        raise ValueError("learning rates must be positive")

    def interval(t):
        r = ref / float(gammas[t])
        p = 2 ** int(math.floor(math.log2(r) + 1e-12)) if r >= 1 else 1
        return max(1, min(H, p))
    return _sync_steps(T, interval)


def freeze_variance(tv, tu, T):
    """T_v restricted to steps whose sync interval is one step long: t is kept
    when the sync steps just before t (or t itself) and just after are at most
    one step apart.  Steps before the first or after the last sync count as
    being in an interval longer than one unless that interval is one step."""
    tu = sorted(set(int(t) for t in tu))
    keep = []
    j = 0
    for t in sorted(set(int(t) for t in tv)):
        if t >= T:
            continue
        while j < len(tu) and tu[j] < t:
            j += 1
        # the interval that ends at step tu[j] (the first sync >= t) started after
        # the sync before it; its length is the gap between the two
        nxt = tu[j] if j < len(tu) else None
        prev = tu[j - 1] if j > 0 else -1
        if nxt is not None and nxt - prev <= 1:
            keep.append(t)
    return keep


def communication(T, tv, tu, n_params, chunk, fp_bits=16, scale_bits=32):
    """What a 0/1 Adam schedule communicates per worker over T steps.

    A step in T_v all-reduces gbar at fp_bits per parameter; a step in T_u runs
    the 1-bit AllReduce of Algorithm 2: one bit per parameter plus one scale
    per chunk (scale_bits) each way of its two phases, counted once as the
    paper counts the 1-bit stage of 1-bit Adam.  Returns a dict with the total
    bits per parameter, its average per step, the number of collective rounds
    (|T_v| + |T_u|) and the number of steps that communicate (|T_v ∪ T_u|)."""
    tv = set(int(t) for t in tv if 0 <= int(t) < T)
    tu = set(int(t) for t in tu if 0 <= int(t) < T)
    nchunks_per_param = 1.0 / chunk
    one_bit = 1.0 + scale_bits * nchunks_per_param
    total = fp_bits * len(tv) + one_bit * len(tu)
    return {"bits_per_param": total, "bits_per_param_per_step": total / T if T else 0.0,
            "rounds": len(tv) + len(tu), "steps_communicating": len(tv | tu),
            "n_params": n_params}


def one_bit_adam_communication(T, T0, n_params, chunk, fp_bits=16, scale_bits=32):
    """1-bit Adam over T steps with a full-precision stage of T0 steps
    (Algorithm 4 with T_v = {0..T0-1}: every step communicates)."""
    T0 = min(T0, T)
    return communication(T, range(T0), range(T0, T), n_params, chunk, fp_bits, scale_bits)
