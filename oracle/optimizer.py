"""Float64 CPU oracle of the backend optimizer step (Algorithm 1, its last
line: the weights take an optimizer step with the rescaled, preconditioned
gradient dW).

TEST INFRASTRUCTURE ONLY: used by the tests, never by the product path;
shares no code with the HIP library.

The paper names the optimizer, not its equations: LAMB for BERT (its
first-order baseline and the backend of the large-language-model runs) and SGD
for the CNN runs.  Readings (listed in the design notes):

* SGD with momentum and L2 weight decay, in the form most frameworks use:
  d = dW + wd W,  m = mu m + d,  W = W - lr m   (m starts at 0).
* LAMB as its authors define it (layer-wise adaptive moments): per layer
  (one weight tensor),
  m = b1 m + (1 - b1) dW,  v = b2 v + (1 - b2) dW^2,
  m_hat = m / (1 - b1^t),  v_hat = v / (1 - b2^t),
  r = m_hat / (sqrt(v_hat) + eps) + wd W,
  phi = ||W||_F / ||r||_F  (1 if either norm is 0),
  W = W - lr phi r.
"""

from __future__ import annotations

import math

import numpy as np


def sgd_step(W, m, g, lr: float, momentum: float, wd: float):
    """One SGD step; returns (W', m')."""
    W = np.asarray(W, np.float64)
    d = np.asarray(g, np.float64) + wd * W
    m = momentum * np.asarray(m, np.float64) + d
    return W - lr * m, m


def lamb_step(W, m, v, g, t: int, lr: float, beta1: float, beta2: float, eps: float, wd: float,
              trust: bool = True):
    """One LAMB step (t >= 1 counts steps from 1); returns (W', m', v', phi).
    trust=False forces phi = 1 (the AdamW-like update, used as a pin)."""
    W = np.asarray(W, np.float64)
    g = np.asarray(g, np.float64)
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    r = m_hat / (np.sqrt(v_hat) + eps) + wd * W
    nW, nr = float(np.linalg.norm(W)), float(np.linalg.norm(r))
    phi = nW / nr if (trust and nW > 0.0 and nr > 0.0) else 1.0
    return W - lr * phi * r, m, v, phi
