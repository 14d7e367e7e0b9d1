"""Training update of the paper on the fp64 oracle -- test infrastructure only.

Section 3, "Training": RMS-prop with momentum.  With a <-rho- b meaning
a = rho a + (1 - rho) b (elementwise), for every parameter tensor theta with
gradient g of the loss:
    MSE <-rho_MSE- g^2                       (Eq. (15), running mean of g^2)
    G    = g / (sqrt(MSE) + eps)             (Eq. (16), normalised gradient)
    M   <-rho_M-  G                          (Eq. (17), smoothed gradient)
    theta = theta - lr M                     (Eq. (18))
with eps = 1e-5 and rho_MSE = rho_M = 0.9, and the decaying learning rate
lr(epoch) = 1e-6 + 1e-2 (1/2)^(epoch / 100).

Reading where the paper is silent: MSE and M start at zero before the first
update.  Plain numpy, one step at a time, in the equations' order.
"""
from __future__ import annotations

import numpy as np

EPS = 1e-5
RHO_MSE = 0.9
RHO_M = 0.9


def learning_rate(epoch: int) -> float:
    """lr = 1e-6 + 1e-2 * (2^(-1/100))^epoch (Section 3, "Training")."""
    return 1e-6 + 1e-2 * (0.5 ** (1.0 / 100.0)) ** epoch


def rmsprop_step(theta, grad, mse, mom, lr, rho_mse=RHO_MSE, rho_m=RHO_M, eps=EPS):
    """One update of Eq. (15)-(18).  Returns new (theta, mse, mom) as fp64
    arrays; the inputs are not modified."""
    theta = np.asarray(theta, dtype=np.float64)
    g = np.asarray(grad, dtype=np.float64)
    mse = rho_mse * np.asarray(mse, dtype=np.float64) + (1.0 - rho_mse) * g * g
    G = g / (np.sqrt(mse) + eps)
    mom = rho_m * np.asarray(mom, dtype=np.float64) + (1.0 - rho_m) * G
    return theta - lr * mom, mse, mom
