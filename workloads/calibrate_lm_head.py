"""Reproduces the lm_head scales used by the 7B-class synthetic workloads.

With the final RMSNorm gain equal to one, a normalised hidden row u has
mean(u^2) = 1 (up to eps), so with lm_head rows drawn i.i.d. N(0, (c*std)^2)
the logits z = W u are i.i.d. N(0, sigma^2) with sigma = c * std * sqrt(d).
The entropy of the last layer is therefore the entropy of V i.i.d. Gaussian
logits; this script finds the sigma whose mean entropy is about 2 nats and
prints the matching scale c for each model shape.

    python workloads/calibrate_lm_head.py
"""
import numpy as np


def _entropy(z):
    m = z.max()
    e = np.exp(z - m)
    s = e.sum()
    return np.log(s) - (e * (z - m)).sum() / s


def mean_entropy(sigma, vocab, samples=64, seed=0):
    rng = np.random.default_rng(seed)
    return float(np.mean([_entropy(sigma * rng.standard_normal(vocab)) for _ in range(samples)]))


def solve_sigma(vocab, target=2.0, lo=4.0, hi=9.0, iters=14):
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        if mean_entropy(mid, vocab) > target:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


if __name__ == "__main__":
    for name, d, V in (("7b", 4096, 128256), ("7b_large_vocab", 3584, 152064), ("10b", 4096, 256000)):
        sigma = solve_sigma(V)
        print(f"{name}: vocab={V} sigma={sigma:.3f} scale={sigma / (0.02 * d ** 0.5):.2f}")
