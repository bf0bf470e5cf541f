"""Test infrastructure (see the package docstring): the parameter update of the paper's training,
stochastic gradient descent with momentum and weight decay (Sec. 4, training setup: momentum 0.9,
weight decay 5e-4 for VGG and 1e-4 for ResNet, Nesterov momentum), in fp64, one tensor at a time.

Reading: weight decay is the L2 term added to the gradient of every parameter; the momentum buffer
starts at zero, so the first step's buffer equals the decayed gradient.
"""
import numpy as np


def sgd_step(w, g, v, lr, mu, wd, nesterov=True):
    """One update of parameters ``w`` with gradient ``g`` and momentum buffer ``v``:
    d = g + wd w;  v' = mu v + d;  w' = w - lr (d + mu v') (Nesterov) or w - lr v'.
    Returns (w', v') in float64."""
    w = np.asarray(w, dtype=np.float64)
    d = np.asarray(g, dtype=np.float64) + wd * w
    v_new = mu * np.asarray(v, dtype=np.float64) + d
    u = d + mu * v_new if nesterov else v_new
    return w - lr * u, v_new
