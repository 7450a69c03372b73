"""Oracle: AdamW step on the LM-head weight W consuming dW (test infrastructure only; see
oracle/__init__).

The paper trains with AdamW at learning rate 1e-6 and weight decay 1e-2 (Sec. 4.1,
implementation details); the step right after the LM-head backward (Alg. 1, "update
pi_theta on the selected trajectories") applies it to W with g = dW.  The paper gives no
other constant; the readings here are the decoupled weight decay of Loshchilov and Hutter
("Decoupled Weight Decay Regularization", ICLR 2019) with the usual defaults
beta1 = 0.9, beta2 = 0.999, eps = 1e-8 and bias correction, in this order per element:

    theta <- theta - lr * wd * theta
    m     <- beta1 m + (1 - beta1) g
    v     <- beta2 v + (1 - beta2) g^2
    theta <- theta - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)

with t the 1-based step count and g = grad_scale * dW.  float64 throughout.
"""
import numpy as np


def adamw_step(theta, grad, m, v, step, lr=1e-6, beta1=0.9, beta2=0.999, eps=1e-8,
               weight_decay=1e-2, grad_scale=1.0):
    """One step.  Returns new (theta, m, v) as float64 arrays (inputs unchanged)."""
    th = np.array(theta, dtype=np.float64)
    g = np.asarray(grad, dtype=np.float64) * float(grad_scale)
    m1 = np.array(m, dtype=np.float64)
    v1 = np.array(v, dtype=np.float64)
    t = int(step)
    th = th - lr * weight_decay * th
    m1 = beta1 * m1 + (1.0 - beta1) * g
    v1 = beta2 * v1 + (1.0 - beta2) * g * g
    mhat = m1 / (1.0 - beta1 ** t)
    vhat = v1 / (1.0 - beta2 ** t)
    th = th - lr * mhat / (np.sqrt(vhat) + eps)
    return th, m1, v1
