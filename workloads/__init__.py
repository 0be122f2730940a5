"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds none of the method's arithmetic: it only draws data
(features, labels, initial parameters) with torch's seeded generators and
lists the workload shapes.  Both the HIP path and the oracle receive the same
tensors from here.  Straggler masks and the real-valued code's random matrix
are not drawn here: each side generates them from the published SplitMix64
definition, and the tests check that the two agree bit for bit.

Workloads (synthetic stand-ins for the paper's ResNet-18 / CIFAR-10 and
downsampled-ImageNet runs, Sec. III and Sec. VI, whose data and models are not
used here):
  fr_logistic_n4_c2_d64            FR, logistic, N = 4096,      d = 64
  crreal_lsq_n8_c3_d1024           naive real-valued CR, least squares,
                                   N = 262144, d = 1024
  fr_logistic_n32_c4_d4096         FR, logistic, N = 1048576,   d = 4096,
                                   every 10th column scaled by 10
  cr_mlp_n64_c4_784x1024x10        PGC-CR, MLP 784 -> 1024 -> 10, bf16 inputs,
                                   N = 1048576
  cr_logistic_n128_c8_d8192        PGC-CR, logistic, N = 2097152, d = 8192
"""

from dataclasses import dataclass, replace
import math

import torch

# Straggler-mask policies (their definition lives with each generator).
POLICY_EXACT = 0
POLICY_UNIFORM_COUNT = 1
POLICY_BERNOULLI = 2
POLICY_SLOWEST = 3


@dataclass(frozen=True)
class Workload:
    name: str
    scheme: str            # "FR", "CR" or "CR_REAL"
    model: str             # "logistic", "lsq" or "mlp"
    n: int                 # workers = partitions
    c: int                 # partitions per worker = pipeline depth (s = c - 1)
    N: int                 # samples
    d: int                 # features (linear models) or input width (MLP)
    lr: float
    steps: int             # steps t = 0 .. steps-1, t = 0 being the warm-up
    policy: int            # straggler policy
    cap: int               # largest straggler count the policy draws
    p: float = 0.0         # per-worker straggle probability (Bernoulli policy)
    seed: int = 0          # data seed; the mask stream uses seed * 2^32 + 1
    scale_every: int = 0   # multiply columns j % scale_every == 0 by 10
    hidden: int = 0        # MLP hidden width
    classes: int = 0       # MLP classes
    code_seed: int = 0     # seed of the real-valued code's random matrix

    @property
    def s(self):
        return self.c - 1

    @property
    def m(self):
        return self.N // self.n

    @property
    def q(self):
        """Length of the parameter vector."""
        if self.model == "mlp":
            return self.d * self.hidden + self.hidden + self.hidden * self.classes + self.classes
        return self.d

    @property
    def mask_seed(self):
        return (self.seed << 32) | 1

    def resized(self, N=None, d=None, steps=None, **kw):
        """The same workload with fewer samples / features / steps (parity-test sizes)."""
        kw = dict(kw)
        if N is not None:
            kw["N"] = N
        if d is not None:
            kw["d"] = d
        if steps is not None:
            kw["steps"] = steps
        return replace(self, name=self.name + "_resized", **kw)


WORKLOADS = {
    w.name: w for w in [
        Workload("fr_logistic_n4_c2_d64", "FR", "logistic", n=4, c=2, N=4096, d=64,
                 lr=0.1, steps=20, policy=POLICY_EXACT, cap=1, seed=1),
        Workload("crreal_lsq_n8_c3_d1024", "CR_REAL", "lsq", n=8, c=3, N=262144, d=1024,
                 lr=0.01, steps=100, policy=POLICY_UNIFORM_COUNT, cap=2, seed=2, code_seed=2),
        Workload("fr_logistic_n32_c4_d4096", "FR", "logistic", n=32, c=4, N=1048576, d=4096,
                 lr=0.01, steps=50, policy=POLICY_BERNOULLI, cap=3, p=0.05, seed=3,
                 scale_every=10),
        Workload("cr_mlp_n64_c4_784x1024x10", "CR", "mlp", n=64, c=4, N=1048576, d=784,
                 lr=0.01, steps=20, policy=POLICY_BERNOULLI, cap=3, p=0.05, seed=4,
                 hidden=1024, classes=10),
        Workload("cr_logistic_n128_c8_d8192", "CR", "logistic", n=128, c=8, N=2097152, d=8192,
                 lr=0.01, steps=30, policy=POLICY_BERNOULLI, cap=7, p=0.04, seed=5),
    ]
}

# Workload order as the configurations are listed (small case first).
ORDER = list(WORKLOADS)


def make_inputs(w, device="cpu"):
    """Features X, labels y and initial parameters beta0 for workload w.

    Linear models: X ~ N(0, 1) fp32 (N x d, row-major); a planted
    beta* ~ N(0, 1/d); logistic labels y ~ Bernoulli(sigmoid(x . beta*)),
    least-squares labels y = x . beta* + noise of variance 0.01; beta0 = 0.
    MLP: X uniform in [0, 1) stored as bf16; a teacher MLP of the same shape
    with He-normal weights and zero biases labels each row with the argmax of
    its logits (int32); the student starts He-normal with zero biases (a zero
    start would leave the ReLU network without gradient).
    """
    g = torch.Generator(device=device)
    g.manual_seed(w.seed)
    if w.model == "mlp":
        return _make_mlp_inputs(w, g, device)
    X = torch.randn(w.N, w.d, generator=g, device=device, dtype=torch.float32)
    if w.scale_every:
        X[:, ::w.scale_every] *= 10.0
    beta_star = torch.randn(w.d, generator=g, device=device, dtype=torch.float32) / math.sqrt(w.d)
    z = _matvec_chunked(X, beta_star)
    if w.model == "logistic":
        y = torch.bernoulli(torch.sigmoid(z), generator=g)
    elif w.model == "lsq":
        y = z + 0.1 * torch.randn(w.N, generator=g, device=device, dtype=torch.float32)
    else:
        raise ValueError("unknown model %r" % (w.model,))
    beta0 = torch.zeros(w.d, device=device, dtype=torch.float32)
    return X, y.to(torch.float32).contiguous(), beta0


def _matvec_chunked(X, v, rows=1 << 16):
    out = torch.empty(X.shape[0], device=X.device, dtype=torch.float32)
    for r in range(0, X.shape[0], rows):
        out[r:r + rows] = X[r:r + rows] @ v
    return out


def _he_normal(fan_in, shape, g, device):
    return torch.randn(*shape, generator=g, device=device, dtype=torch.float32) * math.sqrt(2.0 / fan_in)


def _make_mlp_inputs(w, g, device):
    X = torch.rand(w.N, w.d, generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)
    t1 = _he_normal(w.d, (w.d, w.hidden), g, device)
    t2 = _he_normal(w.hidden, (w.hidden, w.classes), g, device)
    y = torch.empty(w.N, dtype=torch.int32, device=device)
    rows = 1 << 15
    for r in range(0, w.N, rows):
        h = torch.relu(X[r:r + rows].float() @ t1)
        y[r:r + rows] = torch.argmax(h @ t2, dim=1).to(torch.int32)
    W1 = _he_normal(w.d, (w.d, w.hidden), g, device)
    W2 = _he_normal(w.hidden, (w.hidden, w.classes), g, device)
    beta0 = torch.cat([W1.reshape(-1), torch.zeros(w.hidden, device=device),
                       W2.reshape(-1), torch.zeros(w.classes, device=device)]).contiguous()
    return X.contiguous(), y, beta0
