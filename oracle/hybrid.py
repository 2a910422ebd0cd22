"""Reference of MKOR-H's switching rule (the paper's "Hybrid MKOR"
subsection), in plain Python.

TEST INFRASTRUCTURE ONLY, like the rest of this package: the tests compare
the library's host-side policy with it; it shares no code with the library.

The paper switches from the second-order to the first-order optimizer once
the loss stops falling fast enough, judged by the rate at which the loss
decreases, without giving a formula.  Reading used: the losses are averaged
over consecutive windows of `window` iterations; closed window k >= 1 has the
relative decrease r_k = (m_{k-1} - m_k) / |m_{k-1}| of the window means (0 if
m_{k-1} = 0); windows k >= warmup are evaluated, and after `patience`
consecutive evaluated windows with r_k < threshold the decision turns to
first-order for good.
"""
from __future__ import annotations


def hybrid_decisions(losses, window: int, patience: int, warmup: int, threshold: float):
    """Decision (1 second-order, 0 first-order) after each loss, and the
    1-based iteration at which it turned to 0 (None if it never did)."""
    decisions = []
    means = []
    slow = 0
    decision = 1
    switched = None
    for t in range(1, len(losses) + 1):
        if t % window == 0:
            total = 0.0
            for x in losses[t - window:t]:
                total += float(x)
            mean = total / window
            k = len(means)
            if k >= 1 and k >= warmup:
                prev = means[-1]
                rate = (prev - mean) / abs(prev) if prev != 0.0 else 0.0
                slow = slow + 1 if rate < threshold else 0
                if decision == 1 and slow >= patience:
                    decision = 0
                    switched = t
            means.append(mean)
        decisions.append(decision)
    return decisions, switched
