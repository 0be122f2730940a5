"""Oracle-side random draws: straggler masks and the encoding-matrix seed.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Generator: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014), in its counter form: the i-th output of the
stream seeded with S is mix64(S + (i + 1) * GAMMA) mod 2^64, where mix64 is the
variant-13 finaliser used by that paper's generator.  The HIP library carries
its own implementation of the same definition; tests compare the two bit for
bit.  Nothing here is shared with it.

Indexing of draws.  The j-th draw of step t is stream output i = t * 2^32 + j,
so any step's mask can be produced without replaying earlier steps.

Derived values (all integer-exact or exact in binary64):
  uniform01(z)      = (z >> 11) * 2^-53                      in [0, 1)
  bounded(z, R)     = ((z >> 32) * R) >> 32                  in [0, R), R < 2^32
                      (Lemire's multiply-shift on the top 32 bits)

Straggler policies (the paper simulates stragglers by random delays per
worker, Sec. VI-B; here the straggler set itself is drawn):
  EXACT(k)          k stragglers, chosen uniformly by a partial Fisher-Yates
                    shuffle of [0, n): for i < k, swap(perm[i],
                    perm[i + bounded(draw_i, n - i)]); stragglers = perm[:k].
  UNIFORM_COUNT(cap) count = bounded(draw_0, cap + 1), then EXACT(count) on the
                    following draws.
  BERNOULLI(p, cap) worker i straggles when uniform01(draw_i) < p, i = 0..n-1;
                    if more than cap straggle, a partial Fisher-Yates shuffle
                    of the straggler list (draws n, n+1, ...) keeps the first
                    cap of them.  Each worker is equally likely to straggle,
                    which the unbiasedness argument of Sec. V-B assumes.
  SLOWEST(cap)      worker i draws u_i = uniform01(draw_i); the cap workers with
                    the largest u_i straggle (ties: the lower index straggles).
                    With i.i.d. exponential delays -mean * ln(1 - u_i) on top of
                    equal compute times these are exactly the workers the
                    master does not wait for when it takes the n - cap fastest
                    (the delay model of Sec. VI-B).
"""

import math

import numpy as np

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15

POLICY_EXACT = 0
POLICY_UNIFORM_COUNT = 1
POLICY_BERNOULLI = 2
POLICY_SLOWEST = 3


def mix64(z):
    """SplitMix64 output finaliser (variant 13) on a 64-bit integer."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def splitmix64(seed, index):
    """Output number `index` (0-based) of the SplitMix64 stream seeded with `seed`."""
    return mix64((seed + (index + 1) * GAMMA) & MASK64)


def step_draw(seed, t, j):
    """The j-th draw of step t."""
    return splitmix64(seed, (t << 32) + j)


def uniform01(z):
    return (z >> 11) * (2.0 ** -53)


def bounded(z, r):
    return ((z >> 32) * r) >> 32


def _partial_shuffle(seed, t, first_draw, items, k):
    items = list(items)
    for i in range(k):
        r = bounded(step_draw(seed, t, first_draw + i), len(items) - i)
        items[i], items[i + r] = items[i + r], items[i]
    return items[:k]


def straggler_mask(seed, t, policy, n, cap, p=0.0):
    """Straggler mask of step t: uint8[n], 1 = the worker straggles this step."""
    if policy == POLICY_EXACT:
        chosen = _partial_shuffle(seed, t, 0, range(n), min(cap, n))
    elif policy == POLICY_UNIFORM_COUNT:
        count = bounded(step_draw(seed, t, 0), cap + 1)
        chosen = _partial_shuffle(seed, t, 1, range(n), min(count, n))
    elif policy == POLICY_BERNOULLI:
        chosen = [i for i in range(n) if uniform01(step_draw(seed, t, i)) < p]
        if len(chosen) > cap:
            chosen = _partial_shuffle(seed, t, n, chosen, cap)
    elif policy == POLICY_SLOWEST:
        u = [uniform01(step_draw(seed, t, i)) for i in range(n)]
        order = sorted(range(n), key=lambda i: (-u[i], i))
        chosen = order[:min(cap, n)]
    else:
        raise ValueError("unknown straggler policy %r" % (policy,))
    mask = np.zeros(n, dtype=np.uint8)
    mask[list(chosen)] = 1
    return mask


def delay_draws(seed, t, n):
    """The uniforms u_i behind the SLOWEST policy's delays at step t."""
    return [uniform01(step_draw(seed, t, i)) for i in range(n)]


def delay_step(seed, t, n, s, mean_delay, compute_seconds=0.0):
    """One step of the simulated cluster of Sec. VI-B.

    Every worker adds an independent exponential delay of mean `mean_delay`
    to its compute time; the master continues once n - s workers have
    finished (s = 0: it waits for all of them, as DGD must).  The delay of
    worker i is the inverse exponential CDF at its draw u_i.
    Returns (mask uint8[n] of the s workers not waited for, delays, seconds).
    """
    u = delay_draws(seed, t, n)
    delays = [-mean_delay * math.log1p(-ui) for ui in u]
    finish = [compute_seconds + dl for dl in delays]
    waited = sorted(range(n), key=lambda i: (u[i], -i))[:n - s]
    mask = np.ones(n, dtype=np.uint8)
    mask[waited] = 0
    return mask, np.array(delays), max(finish[i] for i in waited)


def null_space_generator(seed, s, n):
    """The s x n matrix H whose null space the real-valued cyclic code lives in.

    Entries of columns 0..n-2 are uniform in [-1, 1): H[a, k] = 2*uniform01(z) - 1
    with z the draw number a*n + k of step 0.  The last column makes every row
    sum to zero, accumulated left to right: H[a, n-1] = -(H[a,0] + ... + H[a,n-2]),
    so that the all-ones vector lies in null(H).
    """
    H = np.zeros((s, n), dtype=np.float64)
    for a in range(s):
        acc = 0.0
        for k in range(n - 1):
            H[a, k] = 2.0 * uniform01(step_draw(seed, 0, a * n + k)) - 1.0
            acc += H[a, k]
        H[a, n - 1] = -acc
    return H
