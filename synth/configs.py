"""Synthetic workloads: shard shapes, schedules and input distributions.

These stand in for the paper's training runs (BERT-Base/Large, ResNet, GPT-2
on their datasets), which are not available: each shard takes a model's
parameter shapes as a per-tensor segment table and draws seeded synthetic
values with the stated distributions.  No optimizer arithmetic lives here;
the schedules T_v / T_u and the learning rates are inputs of the method.

Recipe common to all workloads:
  * x_0 ~ N(0, 0.02) from seed 0, stream X;
  * gradient g_t from seed 0, stream G, step t; the full-precision average
    gbar_t (the AllReduce output, an input on one GPU) from seed 0, stream GBAR,
    with the same distribution;
  * peer w = 1..W-1: packed signs from seed w, stream BITS, step t, indexed by
    the global word; scales from seed w, stream SCALES, step t, indexed by the
    global chunk, uniform in [0.5, 1.5) x base_t with
    base_t = Gamma_t * 0.18 * sigma_g (Gamma_t: learning-rate sum of the
    interval that ends at sync step t; a plausible magnitude of |u|);
  * beta1 = 0.9, beta2 = 0.999, eps = 1e-8.
Schedules follow the shape of the paper's policies: synchronise and update
the variance every step while the learning rate warms up, then freeze the
variance and double the sync interval up to a cap.
"""
from dataclasses import dataclass, field
import math

import numpy as np

STREAM_X, STREAM_G, STREAM_GBAR, STREAM_BITS, STREAM_SCALES = 1, 2, 3, 4, 5
IRWIN_HALL_STD = 65536.0 / math.sqrt(3.0)   # std of the sum of four uniform 16-bit lanes


def ksigma(sigma: float) -> np.float32:
    return np.float32(sigma / IRWIN_HALL_STD)


# ---------------------------------------------------------------------------
# Segment tables (one segment per parameter tensor, in model order)
# ---------------------------------------------------------------------------

def bert_segments(H, F, L, V, P=512, types=2):
    seg = [V * H, P * H, types * H, H, H]
    for _ in range(L):
        seg += [H * H, H, H * H, H, H * H, H, H * H, H, H, H, H * F, F, F * H, H, H, H]
    seg += [H * H, H]
    return seg


def resnet50_segments():
    seg = [64 * 3 * 7 * 7, 64, 64]
    cin = 64
    for width, blocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        for b in range(blocks):
            seg += [cin * width, width, width,
                    9 * width * width, width, width,
                    width * 4 * width, 4 * width, 4 * width]
            if b == 0:
                seg += [cin * 4 * width, 4 * width, 4 * width]
            cin = 4 * width
    seg += [2048 * 1000, 1000]
    return seg


def gpt2_segments(H=1600, F=6400, L=48, V=50257, ctx=1024):
    seg = [V * H, ctx * H]
    for _ in range(L):
        seg += [H, H, H * 3 * H, 3 * H, H * H, H, H, H, H * F, F, F * H, H]
    seg += [H, H]
    return seg


def offsets(lengths):
    return np.concatenate([[0], np.cumsum(np.asarray(lengths, dtype=np.int64))]).astype(np.int64)


# ---------------------------------------------------------------------------
# Workloads
# ---------------------------------------------------------------------------

@dataclass
class Workload:
    name: str
    seg_off: np.ndarray
    world: int
    chunk: int
    steps: int
    tv: list
    tu: list
    gammas: list
    sigma_g: float
    outlier_per_mille: int = 0
    outlier_factor: float = 1.0
    sigma_x: float = 0.02
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    notes: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def n(self):
        return int(self.seg_off[-1])

    @property
    def nseg(self):
        return len(self.seg_off) - 1

    def gamma(self, t):
        return np.float32(self.gammas[t])

    def interval_gamma_sum(self, t):
        """Sum of the learning rates since the previous sync, up to and
        including step t (binary64; only sizes the synthetic peer scales)."""
        tu = set(self.tu)
        s = 0.0
        h = t
        while h >= 0:
            s += float(self.gammas[h])
            h -= 1
            if h in tu:
                break
        return s

    @property
    def algorithm(self):
        return self.extra.get("algorithm", "zero-one")

    def peer_scale_base(self, t):
        if self.algorithm == "frozen-variance":
            # the compressed quantity is the gradient itself: E|g| = 0.8 sigma
            return np.float32(0.8 * self.sigma_g)
        return np.float32(self.interval_gamma_sum(t) * 0.18 * self.sigma_g)


def _bert_gammas(T):
    return [4e-4 * (t + 1) / 16 if t < 16 else 4e-4 * 0.99 ** (t - 15) for t in range(T)]


def tiny(alt=False):
    T = 20
    tv = [1, 2, 4, 8, 16] if alt else [0, 1, 3, 7, 15]
    return Workload(
        name="tiny-alt" if alt else "tiny", seg_off=offsets([1 << 20]), world=4, chunk=2048,
        steps=T, tv=tv, tu=[t for t in range(T) if (t + 1) % 2 == 0], gammas=[1e-4] * T,
        sigma_g=1e-3,
        notes="1,048,576 params, W=4, chunk 2048, 20 steps; variance at 1-based steps "
              "{1,2,4,8,16}, sync every 2 steps" + (" (0-based reading)" if alt else ""))


def bert_base():
    T = 44
    return Workload(
        name="bert-base", seg_off=offsets(bert_segments(768, 3072, 12, 30522)), world=16,
        chunk=4096, steps=T, tv=list(range(16)),
        tu=list(range(16)) + [17, 19, 23, 27, 35, 43], gammas=_bert_gammas(T), sigma_g=1e-3,
        outlier_per_mille=10, outlier_factor=100.0,
        notes="BERT-Base-shaped shard (110M), W=16, chunk 4096")


def bert_large():
    T = 46
    return Workload(
        name="bert-large", seg_off=offsets(bert_segments(1024, 4096, 24, 30522)), world=64,
        chunk=8192, steps=T, tv=list(range(16)), tu=list(range(16)) + [17, 21, 29, 45],
        gammas=_bert_gammas(T), sigma_g=1e-3, outlier_per_mille=10, outlier_factor=100.0,
        notes="BERT-Large-shaped shard (340M), W=64, chunk 8192")


def resnet50():
    T = 46
    return Workload(
        name="resnet50", seg_off=offsets(resnet50_segments()), world=32, chunk=1024, steps=T,
        tv=list(range(16)), tu=list(range(16)) + [17, 21, 29, 45], gammas=[1e-4] * T,
        sigma_g=1e-2, notes="ResNet-50-shaped shard (25.6M), W=32, chunk 1024")


def gpt2_1p5b():
    T = 94
    return Workload(
        name="gpt2-1.5b", seg_off=offsets(gpt2_segments()), world=128, chunk=16384, steps=T,
        tv=list(range(32)), tu=list(range(32)) + [33, 37, 45, 61, 93], gammas=[1e-4] * T,
        sigma_g=1e-4, outlier_per_mille=1, outlier_factor=1000.0,
        notes="GPT-2-1.5B-shaped shard (1.56B), W=128, chunk 16384")


ALL = {"tiny": tiny, "tiny-alt": lambda: tiny(True), "bert-base": bert_base,
       "bert-large": bert_large, "resnet50": resnet50, "gpt2-1.5b": gpt2_1p5b}


def one_bit(base, t0):
    """The same shard run by Algorithm 4 as 1-bit Adam: full-precision steps
    (variance updates) for t < t0, then compressed gradients with the variance
    frozen, no local steps."""
    def make():
        wl = ALL[base]()
        return Workload(name=f"{base}-1bit", seg_off=wl.seg_off, world=wl.world, chunk=wl.chunk,
                        steps=wl.steps, tv=list(range(min(t0, wl.steps))), tu=[],
                        gammas=wl.gammas, sigma_g=wl.sigma_g,
                        outlier_per_mille=wl.outlier_per_mille,
                        outlier_factor=wl.outlier_factor, sigma_x=wl.sigma_x, beta1=wl.beta1,
                        beta2=wl.beta2, eps=wl.eps,
                        notes=f"1-bit Adam on the {base} shard, full-precision stage of {t0} steps",
                        extra={"algorithm": "frozen-variance"})
    return make


for _b, _t0 in (("tiny", 6), ("bert-base", 16), ("bert-large", 16), ("resnet50", 16),
                ("gpt2-1.5b", 32)):
    ALL[f"{_b}-1bit"] = one_bit(_b, _t0)


def get(name):
    return ALL[name]()
