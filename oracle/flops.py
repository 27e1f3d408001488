"""Analytic prefill-FLOPs accounting (Appendix G, "FLOPs Accounting").

TEST INFRASTRUCTURE ONLY -- see the package docstring.  Pins live in
``tests/test_oracle_flops_pins.py``.

What it computes, in the readings listed below:

1. One decoder layer at sequence length n costs
   phi(n) = 4 n d^2 (the Q, K, V and O projections) + 2 n^2 d (the
   quadratic attention) + 2 n d m (the feed-forward block), with hidden size
   d and feed-forward width m (Appendix G, per-layer equation).
2. Prefill FLOPs sum phi over the length n_i entering each of the T layers;
   the full-token reference is T phi(n_0) (Appendix G, prefill equation).
3. The FLOPs ratio is F_pre / (T phi(n_0)) (Appendix G, ratio equation).
4. A-PACK's length schedule (Algorithm 1, loop over layers from L_mid;
   Section 4.1 implementation details): every layer runs at the length that
   enters it.  A prune at layer l scores with that layer's attention and
   takes effect from layer l + 1 (layers numbered from 0).  Under the
   paper's every-layer schedule each prune keeps ceil((1 - P) |S|) of the
   current candidates S; tokens outside S are never pruned.

All arithmetic is exact: Python integers for phi and its sums, exact
fractions for the ratio, exact decimal ceilings for the keep counts.
"""

from fractions import Fraction

from .prune import keep_count

# Thinker constants (Appendix G): layers T, hidden size d, feed-forward width m.
QWEN_OMNI = {"7B": (28, 3584, 18944), "3B": (36, 2048, 11008)}


def layer_flops(n, d, m):
    """phi(n): prefill cost of one decoder layer at length n (Appendix G)."""
    n, d, m = int(n), int(d), int(m)
    return 4 * n * d * d + 2 * n * n * d + 2 * n * d * m


def prefill_flops(lengths, d, m):
    """F_pre: phi summed over the per-layer lengths n_1..n_T (Appendix G)."""
    return sum(layer_flops(n, d, m) for n in lengths)


def flops_ratio(lengths, n0, d, m):
    """rho = F_pre / (T phi(n0)) as an exact fraction (Appendix G)."""
    return Fraction(prefill_flops(lengths, d, m), len(lengths) * layer_flops(n0, d, m))


def step_schedule(n_layers, n_start, prune_layers, n_after):
    """Lengths entering each of n_layers layers when the sequence starts at
    n_start and the prune at layer prune_layers[j] leaves n_after[j] tokens,
    effective from the next layer."""
    lengths, n, j = [], int(n_start), 0
    for layer in range(n_layers):
        lengths.append(n)
        while j < len(prune_layers) and prune_layers[j] == layer:
            n = int(n_after[j])
            j += 1
    return lengths


def every_layer_counts(n_other, n_cand, first_layer, n_layers, drop):
    """Token counts after each prune of the paper's every-layer schedule:
    from first_layer to the last layer, each prune keeps ceil((1 - drop) |S|)
    of the current candidates (Eq. 6 as written) and every non-candidate."""
    keep = 1.0 - drop
    layers, after, s = [], [], int(n_cand)
    for layer in range(first_layer, n_layers):
        s = keep_count(keep, s)
        layers.append(layer)
        after.append(int(n_other) + s)
    return layers, after
