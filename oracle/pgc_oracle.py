"""fp64 oracle of a pipelined-gradient-coding (PGC) training run.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Plain numpy in
float64; no blocking, fusion or reordering beyond the definitions below.

What it follows (Pipelined Gradient Coding, Su and Li):
  * Sec. III: empirical risk F(beta) = (1/N) sum_i f(beta; x_i, y_i), gradient
    step beta <- beta - eta * g, and the two placements of gradient coding:
    fractional repetition (FR) and cyclic repetition (CR).
  * Sec. IV-A: PGC-FR.  At step t >= 1 worker W_i (group j = i // c) evaluates
    only D_{jc + ((t-1) mod c)} and sends
        ghat_i^(t) = sum_{l<c} g^(t-l)_{jc + ((t-1-l) mod c)};
    the master picks one coded gradient per group and sums across groups.
    Step t = 0 evaluates every partition a worker holds (the warm-up) and is
    plain gradient coding.
  * Sec. V-A: the naive cyclic construction with real encoding coefficients
    c_{j,l}: ghat_j = sum_l c_{j,l} g_{(j+l) mod n}, decoded with weights
    d_m(J) solved from a linear system so the partition sum is recovered.
  * Sec. V-B: PGC-CR.  Worker W_j evaluates D_{(j + (t-1) mod c) mod n} at
    step t, sends ghat_j^(t) = sum_l g^(t-l)_{(j + (t-1-l) mod c) mod n}
    with unit coefficients, and the master forms
        ghat^(t) = (1 / (n mu)) sum_{m} ghat_{j_m}^(t),   mu = |J| c / n.
  * Baselines of Sec. III and VI-A: gradient coding (GC) is the same placement
    and decode with every worker evaluating all c of its partitions at the
    current step (run(..., pipelined=False)); DGD is c = 1; IS-SGD gives each
    worker one partition (c = 1) and averages whatever survivors arrive.

The run keeps the history of iterates beta^(tau) and evaluates each coded
gradient from the formulas above: the copy of slot l used at step t is the
gradient of partition P[i][(t-1-l) mod c] at beta^(t-l).  Gradients are
memoised per (partition, step), which is exact because g_k^(tau) depends only
on k and beta^(tau).  The HIP path keeps per-slot ring buffers instead; the
two bookkeepings agree only if the schedule and the formula agree.

Readings where the paper is silent (each is listed with its reason in the
design notes of the repository):
  R1  Partitions are contiguous equal row blocks, m = N / n rows each.
  R2  g_k is the mean of the per-sample gradients over D_k, so that with c = 1
      the DGD average (1/n) sum_k g_k is exactly grad F.
  R3  Losses: logistic f = log(1 + e^z) - y z with y in {0, 1}; least squares
      f = (z - y)^2 / 2; z = x . beta, no bias, no regulariser.  MLP:
      784 -> hidden (ReLU) -> classes, mean softmax cross-entropy, biases, and
      ReLU'(0) = 0; W1 and W2 enter the layers as bf16-rounded values.
  R4  A copy whose formula step t - l is < 1 is the warm-up value (step 0).
  R5  Stragglers still evaluate and store (stated for CR in Sec. V-B; applied
      to FR too).  J is all non-stragglers in ascending order; more than
      s = c - 1 stragglers is an error.
  R6  FR decodes with the lowest-index survivor of each group.
  R7  CR uses mu_t = |J| c / n, which is the paper's (n - s) c / n when exactly
      s workers straggle and keeps ghat equal to the full average when none do.
  R8  The real-valued code decodes with the minimum-norm solution of
      B_J^T d = 1 (unique also when |J| > n - s) and scale 1/n.
  R9  The real-valued B: row j is supported on {j, ..., j+c-1} mod n with
      B[j, j] = 1 and lies in the null space of a random s x n matrix H whose
      rows sum to zero; then any n - s rows span a space containing 1.

Parity unpinned: the specific entries of B (the paper cites, but does not
print, its construction), and the MLP path beyond its 2e-2 tolerance.
"""

from dataclasses import dataclass, field

import numpy as np

FR = "FR"
CR = "CR"
CR_REAL = "CR_REAL"
IS_SGD = "IS_SGD"
SCHEMES = (FR, CR, CR_REAL, IS_SGD)

LOGISTIC = "logistic"
LSQ = "lsq"
MLP = "mlp"


class StragglerError(ValueError):
    """More stragglers than the scheme tolerates (or an FR group with no survivor)."""


class SingularError(ValueError):
    """The decoding system of the real-valued code has no exact solution."""


# ----------------------------------------------------------------------------
# Placement and schedule (Sec. III, Sec. IV-A, Sec. V-B)
# ----------------------------------------------------------------------------

def placement(scheme, n, c):
    """P[i][l]: the partition worker W_i holds in slot l, l = 0..c-1.

    FR (Sec. III): W_i holds D_{jc}, ..., D_{jc+c-1} with j = floor(i / c); needs c | n.
    CR (Sec. III, Sec. V-B): W_i holds D_{(i+l) mod n}.
    IS-SGD (Sec. VI-A): W_i holds D_i alone (c = 1).
    """
    if scheme not in SCHEMES:
        raise ValueError("unknown scheme %r" % (scheme,))
    if not 1 <= c <= n:
        raise ValueError("need 1 <= c <= n")
    if scheme == IS_SGD and c != 1:
        raise ValueError("IS-SGD gives each worker one partition (c = 1)")
    if scheme == FR:
        if n % c:
            raise ValueError("fractional repetition needs c | n")
        return [[(i // c) * c + l for l in range(c)] for i in range(n)]
    return [[(i + l) % n for l in range(c)] for i in range(n)]


def evaluated_slot(t, c):
    """Slot every worker evaluates at pipelined step t >= 1: (t - 1) mod c."""
    if t < 1:
        raise ValueError("step 0 is the warm-up; every slot is evaluated")
    return (t - 1) % c


def coded_terms(scheme, n, c, i, t, pipelined=True):
    """The c copies worker W_i combines at step t, as (slot, partition, step) triples.

    The copy indexed l = 0..c-1 in the coded-gradient formulas of Sec. IV-A and
    Sec. V-B is partition P[i][(t-1-l) mod c] as evaluated at step t - l; a
    step below 1 means the warm-up evaluation (R4).  At t = 0 the slots
    (-1-l) mod c run over all c slots, all at step 0: the gradient-coding word.
    Without pipelining (gradient coding) every copy is evaluated at step t.
    """
    P = placement(scheme, n, c)
    terms = []
    for l in range(c):
        slot = (t - 1 - l) % c
        if pipelined:
            tau = t - l if t - l >= 1 else 0
        else:
            tau = t
        terms.append((slot, P[i][slot], tau))
    return terms


def encoding_coefficients(scheme, n, c, B=None):
    """E[i][l]: coefficient of slot l in worker i's coded gradient.

    FR and PGC-CR use unit coefficients (Sec. IV-A, Sec. V-B).  The naive
    real-valued cyclic code uses c_{i,l} = B[i, (i+l) mod n] (Sec. V-A).
    """
    if scheme in (FR, CR, IS_SGD):
        return [[1.0] * c for _ in range(n)]
    if B is None:
        raise ValueError("the real-valued cyclic code needs its matrix B")
    return [[float(B[i, (i + l) % n]) for l in range(c)] for i in range(n)]


def cyclic_encoding_matrix(n, c, H):
    """Real-valued cyclic-repetition matrix B (n x n), reading R9.

    Row j is supported on S_j = {j, ..., j+c-1} mod n, has B[j, j] = 1 and
    satisfies H B[j, :]^T = 0: the other c - 1 entries solve the s x s system
    H[:, S_j \\ {j}] x = -H[:, j].  H has s = c - 1 rows.
    """
    s = c - 1
    if H.shape != (s, n):
        raise ValueError("H must be (c-1) x n")
    B = np.zeros((n, n), dtype=np.float64)
    for j in range(n):
        B[j, j] = 1.0
        if s == 0:
            continue
        others = [(j + l) % n for l in range(1, c)]
        x = np.linalg.solve(H[:, others], -H[:, j])
        for col, val in zip(others, x):
            B[j, col] = val
    return B


# ----------------------------------------------------------------------------
# Surviving set and decoding (Sec. IV-A, Sec. V-A, Sec. V-B)
# ----------------------------------------------------------------------------

def survivors(mask):
    """J: the non-straggling workers in ascending order (mask[i] = 1: straggler)."""
    return [i for i, m in enumerate(mask) if int(m) == 0]


def decode_weights(scheme, n, c, J, B=None, tol=1e-9):
    """Decode weights d_m for the survivors J (same order) and the scale.

    The decoded gradient is scale * sum_m d_m * ghat_{J[m]}.
      FR:       d = 1 for the lowest-index survivor of each group (R6), else 0;
                scale = 1/n (the DGD average, Sec. IV-B).
      CR:       d = 1 for every survivor; scale = 1/(n mu) = 1/(|J| c) (R7).
      CR_REAL:  minimum-norm d with B_J^T d = 1 (R8); scale = 1/n.
      IS_SGD:   d = 1 for every survivor, however many straggle; scale = 1/|J|.
    """
    s = c - 1
    J = list(J)
    if scheme == IS_SGD:
        if not J:
            raise StragglerError("every worker straggles")
        return np.ones(len(J)), 1.0 / len(J)
    if len(J) < n - s:
        raise StragglerError("%d stragglers exceed s = %d" % (n - len(J), s))
    if scheme == FR:
        d = [0.0] * len(J)
        for group in range(n // c):
            members = [m for m, j in enumerate(J) if j // c == group]
            if not members:
                raise StragglerError("FR group %d has no survivor" % group)
            d[members[0]] = 1.0
        return np.array(d), 1.0 / n
    if scheme == CR:
        return np.ones(len(J)), 1.0 / (len(J) * c)
    if scheme == CR_REAL:
        A = np.asarray(B, dtype=np.float64)[J, :].T          # n x |J|
        ones = np.ones(n)
        d = np.linalg.lstsq(A, ones, rcond=None)[0]           # minimum-norm solution
        if np.max(np.abs(A @ d - ones)) > tol:
            raise SingularError("B_J^T d = 1 has no solution for J = %r" % (J,))
        return d, 1.0 / n
    raise ValueError("unknown scheme %r" % (scheme,))


def copy_counts(scheme, n, c, J):
    """|N_k|: how many times partition k appears among the received coded gradients (Sec. V-B)."""
    P = placement(scheme, n, c)
    counts = np.zeros(n, dtype=np.int64)
    for j in J:
        for k in P[j]:
            counts[k] += 1
    return counts


def decoding_coefficients(scheme, n, c, J, d, B=None):
    """alpha[m, k] = d_m * c_{j_m, l} with (j_m + l) mod n = k (Sec. V-A)."""
    P = placement(scheme, n, c)
    E = encoding_coefficients(scheme, n, c, B)
    alpha = np.zeros((len(J), n))
    for m, j in enumerate(J):
        for l in range(c):
            alpha[m, P[j][l]] += d[m] * E[j][l]
    return alpha


# ----------------------------------------------------------------------------
# Per-partition gradients (Sec. III with readings R1-R3)
# ----------------------------------------------------------------------------

def round_to_bf16(a):
    """Round float64 values to bf16 (via float32, round-to-nearest-even), returned as float64."""
    f = np.asarray(a, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) >> 16) << 16
    return rounded.astype(np.uint32).view(np.float32).astype(np.float64)


def sigmoid(z):
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-z))


def mlp_unpack(beta, shape):
    d_in, h, k = shape
    o = 0
    W1 = beta[o:o + d_in * h].reshape(d_in, h); o += d_in * h
    b1 = beta[o:o + h]; o += h
    W2 = beta[o:o + h * k].reshape(h, k); o += h * k
    b2 = beta[o:o + k]; o += k
    if o != beta.size:
        raise ValueError("parameter vector does not match the MLP shape")
    return W1, b1, W2, b2


def mlp_param_count(shape):
    d_in, h, k = shape
    return d_in * h + h + h * k + k


def partition_loss(model, Xk, yk, beta, shape=None):
    """Mean loss over the rows of one partition (R3)."""
    if model == LOGISTIC:
        z = Xk @ beta
        return float(np.mean(np.logaddexp(0.0, z) - yk * z))
    if model == LSQ:
        r = Xk @ beta - yk
        return float(np.mean(0.5 * r * r))
    if model == MLP:
        W1, b1, W2, b2 = mlp_unpack(beta, shape)
        W1, W2 = round_to_bf16(W1), round_to_bf16(W2)
        H = np.maximum(Xk @ W1 + b1, 0.0)
        Z2 = H @ W2 + b2
        zmax = Z2.max(axis=1, keepdims=True)
        lse = zmax[:, 0] + np.log(np.exp(Z2 - zmax).sum(axis=1))
        return float(np.mean(lse - Z2[np.arange(len(yk)), yk.astype(np.int64)]))
    raise ValueError("unknown model %r" % (model,))


def partition_gradient(model, Xk, yk, beta, shape=None):
    """g_k: mean per-sample gradient over the rows of one partition (R2, R3)."""
    m = Xk.shape[0]
    if model == LOGISTIC:
        r = sigmoid(Xk @ beta) - yk
        return Xk.T @ r / m
    if model == LSQ:
        r = Xk @ beta - yk
        return Xk.T @ r / m
    if model == MLP:
        W1, b1, W2, b2 = mlp_unpack(beta, shape)
        W1, W2 = round_to_bf16(W1), round_to_bf16(W2)
        Z1 = Xk @ W1 + b1
        H = np.maximum(Z1, 0.0)
        Z2 = H @ W2 + b2
        P = np.exp(Z2 - Z2.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        dZ2 = P
        dZ2[np.arange(m), yk.astype(np.int64)] -= 1.0
        dZ2 /= m
        dW2 = H.T @ dZ2
        db2 = dZ2.sum(axis=0)
        dZ1 = (dZ2 @ W2.T) * (Z1 > 0.0)
        dW1 = Xk.T @ dZ1
        db1 = dZ1.sum(axis=0)
        return np.concatenate([dW1.ravel(), db1, dW2.ravel(), db2])
    raise ValueError("unknown model %r" % (model,))


# ----------------------------------------------------------------------------
# The training run
# ----------------------------------------------------------------------------

@dataclass
class StepRecord:
    t: int
    survivors: list
    d: np.ndarray
    scale: float
    ghat: np.ndarray                 # decoded gradient used by the update
    beta: np.ndarray                 # beta^(t+1)
    evaluated: list                  # partition evaluated by each worker
    staleness: list                  # per worker: the c (partition, step) copies combined
    coded: np.ndarray = None         # n x q coded gradients (when kept)
    copy_counts: np.ndarray = None   # |N_k| over the received coded gradients
    alpha: np.ndarray = None         # decoding coefficients alpha[m, k]
    losses: dict = field(default_factory=dict)


def decode_step(scheme, n, c, E, grad, t, mask, shape, B=None, pipelined=True):
    """Coded gradients and decoded gradient of step t.

    grad(k, tau) is the gradient of partition k at the iterate of step tau;
    E the encoding coefficients.  Each worker's coded gradient combines the
    copies coded_terms lists (Sec. IV-A, V-A, V-B); the master decodes the
    survivors' words with decode_weights.  Returns (coded, staleness,
    survivors, d, scale, ghat).
    """
    coded = []
    stale = []
    for i in range(n):
        terms = coded_terms(scheme, n, c, i, t, pipelined)
        word = np.zeros(shape)
        for slot, k, tau in terms:
            word = word + E[i][slot] * grad(k, tau)
        coded.append(word)
        stale.append([(k, tau) for slot, k, tau in terms])
    J = survivors(mask)
    d, scale = decode_weights(scheme, n, c, J, B)
    acc = np.zeros(shape)
    for dm, j in zip(d, J):
        acc = acc + dm * coded[j]
    return coded, stale, J, d, scale, scale * acc


def teacher_forced_ghat(scheme, model, n, c, X, y, iterates, t, mask, B=None, shape=None,
                        pipelined=True, memo=None):
    """Decoded gradient of step t with every copy evaluated at given iterates.

    iterates[tau] is the parameter vector the step tau started from (taken
    from the run being diagnosed, not from the oracle's own trajectory), so a
    per-step difference separates the error of one step from the drift of two
    independent trajectories.  Same definitions as run().  `memo` (a dict)
    may carry partition gradients from one call to the next when the earlier
    iterates are unchanged.
    """
    X = np.asarray(X, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    m = X.shape[0] // n
    E = encoding_coefficients(scheme, n, c, B)
    memo = {} if memo is None else memo

    def grad(k, tau):
        if (k, tau) not in memo:
            rows = slice(k * m, (k + 1) * m)
            memo[(k, tau)] = partition_gradient(model, X[rows], y[rows],
                                                np.asarray(iterates[tau], dtype=np.float64), shape)
        return memo[(k, tau)]
    return decode_step(scheme, n, c, E, grad, t, mask, np.shape(iterates[t]), B=B, pipelined=pipelined)[-1]


def run(scheme, model, n, c, X, y, beta0, lr, masks, B=None, shape=None,
        keep_coded=True, keep_alpha=True, pipelined=True, on_step=None):
    """Run len(masks) PGC steps t = 0, 1, ... from beta0 and return one StepRecord per step.

    masks[t] is the straggler mask of step t (1 = straggles).  Step 0 is the
    warm-up: every worker evaluates all c of its partitions at beta0
    (Sec. IV-A), so its coded gradient is the gradient-coding word.
    pipelined=False runs gradient coding: every step is such a step.
    on_step(t, record), when given, is called after each step (progress
    reports of long runs); it does not affect the run.
    """
    X = np.asarray(X, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    N = X.shape[0]
    if N == 0 or N % n:
        raise ValueError("N must be a positive multiple of n")
    m = N // n
    P = placement(scheme, n, c)
    E = encoding_coefficients(scheme, n, c, B)
    history = {0: np.array(beta0, dtype=np.float64)}
    memo = {}

    def grad(k, tau):
        key = (k, tau)
        if key not in memo:
            rows = slice(k * m, (k + 1) * m)
            memo[key] = partition_gradient(model, X[rows], y[rows], history[tau], shape)
        return memo[key]

    records = []
    for t, mask in enumerate(masks):
        coded, stale, J, d, scale, ghat = decode_step(scheme, n, c, E, grad, t, mask, history[t].shape,
                                                      B=B, pipelined=pipelined)
        beta_next = history[t] - lr * ghat
        history[t + 1] = beta_next
        evaluated = ([P[i][l] for i in range(n) for l in range(c)] if (t == 0 or not pipelined)
                     else [P[i][evaluated_slot(t, c)] for i in range(n)])
        records.append(StepRecord(
            t=t, survivors=J, d=np.asarray(d), scale=scale, ghat=ghat, beta=beta_next,
            evaluated=evaluated, staleness=stale,
            coded=np.array(coded) if keep_coded else None,
            copy_counts=copy_counts(scheme, n, c, J),
            alpha=decoding_coefficients(scheme, n, c, J, d, B) if keep_alpha else None))
        if on_step is not None:
            on_step(t, records[-1])
        # Step t + 1 combines copies from steps >= t + 2 - c only (with step 0
        # standing in for the steps before the pipeline filled).
        oldest = t + 2 - c
        for key in [key for key in memo if key[1] < oldest]:
            del memo[key]
        for tau in [tau for tau in history if tau < oldest]:
            del history[tau]
    return records


def full_loss(model, X, y, beta, shape=None):
    """F(beta) over the whole dataset (Sec. III)."""
    X = np.asarray(X, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    return partition_loss(model, X, y, beta, shape)
