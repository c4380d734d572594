"""Gate g_theta of Eq. 1 (oracle; test infrastructure only).

A dense MLP over the state vector: optional z-scoring of the inputs with
training statistics (Sec. 3.2 and App. A.2 say the inputs are z-scored),
ReLU after every hidden layer, no activation on the output logit z_t.
The decision of Alg. 2 compares sigma(z_t) with tau; sigma is monotone, so
sigma(z) > tau  <=>  z > ln(tau / (1 - tau)), evaluated in float64.

Blob layout (float32): [k, d_0..d_{k-1}, zflag, (mu[d_0], sd[d_0]),
W_1, b_1, ..., W_{k-1}, b_{k-1}] with W_l row-major [d_l, d_{l-1}].
Pinned against torch.nn.Sequential on the same parameters; parameter counts
449 (6-8-8-32-1, App. A.2) and 833 (8-32-16-1) are checked.
"""
import math

import numpy as np


class Gate:
    def __init__(self, widths, layers, mu=None, sd=None):
        self.widths = tuple(widths)
        self.layers = layers          # [(W [out,in] f64, b [out] f64)]
        self.mu = mu
        self.sd = sd

    @property
    def d_in(self):
        return self.widths[0]

    @property
    def n_params(self):
        return sum(W.size + b.size for W, b in self.layers)

    def logit(self, features):
        u = np.asarray(features, np.float64)[: self.d_in]
        if self.mu is not None:
            u = (u - self.mu) / self.sd
        n = len(self.layers)
        for i, (W, b) in enumerate(self.layers):
            u = W @ u + b
            if i < n - 1:
                u = np.maximum(u, 0.0)
        return float(u[0])


def parse_gate_blob(blob) -> Gate:
    a = np.asarray(blob, np.float32).astype(np.float64)
    k = int(a[0])
    if k < 2 or a[0] != k:
        raise ValueError("gate blob: bad layer count")
    widths = [int(v) for v in a[1:1 + k]]
    if widths[-1] != 1:
        raise ValueError("gate blob: output width must be 1")
    p = 1 + k
    zflag = int(a[p]); p += 1
    mu = sd = None
    if zflag:
        d0 = widths[0]
        mu = a[p:p + d0].copy(); p += d0
        sd = a[p:p + d0].copy(); p += d0
    layers = []
    for i in range(1, k):
        o, n_in = widths[i], widths[i - 1]
        W = a[p:p + o * n_in].reshape(o, n_in).copy(); p += o * n_in
        b = a[p:p + o].copy(); p += o
        layers.append((W, b))
    if p != a.size:
        raise ValueError("gate blob: length mismatch")
    return Gate(widths, layers, mu, sd)


def tau_logit(tau: float) -> float:
    return math.log(tau / (1.0 - tau))
