"""Gate g_theta of Eq. 1 (oracle; test infrastructure only).

A dense ReLU network over the state vector: optional z-scoring of the
inputs with training statistics (Sec. 3.2 and App. A.2 say the inputs are
z-scored), ReLU after every hidden layer, no activation on the output
logit z_t.  The decision of Alg. 2 compares sigma(z_t) with tau; sigma is
monotone, so sigma(z) > tau  <=>  z > ln(tau / (1 - tau)), evaluated in
float64.

Two forms, both read from a self-describing float32 blob:

* plain MLP (the FLUX / Qwen gate of App. A.2 and the workloads' gate):
  [k, d_0..d_{k-1}, zflag, (mu[d_0], sd[d_0]), W_1, b_1, ..., W_{k-1}, b_{k-1}]
* branched (the Wan gate of App. A.2: one branch per signal group, fused
  by a trunk): [-n, then per branch (k_j, widths), then the trunk
  (k, widths), zflag, (mu[D], sd[D]), the parameters of branch 1 .. n,
  then of the trunk], D = sum of the branch input widths.  Branch j reads
  the next d_0^(j) features in order (two 3-wide branches: budget state
  f0..f2 and trajectory state f3..f5); every branch layer is followed by
  ReLU (the branch outputs are hidden units of the whole network); the
  trunk reads the concatenated branch outputs.

W_l is row-major [d_l, d_{l-1}] (torch nn.Linear order) in both forms.
Pinned against torch.nn modules on the same parameters; parameter counts
449 (6-8-8-32-1) and 785 (two 3-8-8 branches + 16-32-1) of App. A.2 and
833 (8-32-16-1) are checked.
"""
import math

import numpy as np


def _relu_net(layers, u, last_relu):
    n = len(layers)
    for i, (W, b) in enumerate(layers):
        u = W @ u + b
        if i < n - 1 or last_relu:
            u = np.maximum(u, 0.0)
    return u


class Gate:
    def __init__(self, widths, layers, mu=None, sd=None, branches=()):
        self.widths = tuple(widths)   # trunk widths
        self.layers = layers          # trunk [(W [out,in] f64, b [out] f64)]
        self.mu = mu
        self.sd = sd
        self.branches = list(branches)  # [(widths, layers)]

    @property
    def d_in(self):
        if self.branches:
            return sum(w[0] for w, _ in self.branches)
        return self.widths[0]

    @property
    def n_params(self):
        nets = [self.layers] + [l for _, l in self.branches]
        return sum(W.size + b.size for net in nets for W, b in net)

    def logit(self, features):
        u = np.asarray(features, np.float64)[: self.d_in]
        if self.mu is not None:
            u = (u - self.mu) / self.sd
        if self.branches:
            outs, p = [], 0
            for widths, layers in self.branches:
                outs.append(_relu_net(layers, u[p:p + widths[0]], last_relu=True))
                p += widths[0]
            u = np.concatenate(outs)
        return float(_relu_net(self.layers, u, last_relu=False)[0])


def _widths(a, p):
    k = a[p]
    if k < 2 or k != int(k) or p + 1 + int(k) > a.size:
        raise ValueError("gate blob: bad layer count")
    k = int(k)
    w = a[p + 1:p + 1 + k]
    if np.any(w < 1) or np.any(w != np.floor(w)):
        raise ValueError("gate blob: bad width")
    return [int(v) for v in w], p + 1 + k


def _layers(a, p, widths):
    layers = []
    for i in range(1, len(widths)):
        o, n_in = widths[i], widths[i - 1]
        if p + o * n_in + o > a.size:
            raise ValueError("gate blob: length mismatch")
        W = a[p:p + o * n_in].reshape(o, n_in).copy(); p += o * n_in
        b = a[p:p + o].copy(); p += o
        layers.append((W, b))
    return layers, p


def parse_gate_blob(blob) -> Gate:
    a = np.asarray(blob, np.float32).astype(np.float64)
    if a.size < 4:
        raise ValueError("gate blob too short")
    p = 0
    branch_w = []
    if a[0] < 0:
        nb = -a[0]
        if nb != int(nb) or nb > 8:
            raise ValueError("gate blob: bad branch count")
        p = 1
        for _ in range(int(nb)):
            w, p = _widths(a, p)
            branch_w.append(w)
    widths, p = _widths(a, p)
    if widths[-1] != 1:
        raise ValueError("gate blob: output width must be 1")
    if branch_w and widths[0] != sum(w[-1] for w in branch_w):
        raise ValueError("gate blob: trunk input width != sum of branch outputs")
    d_in = sum(w[0] for w in branch_w) if branch_w else widths[0]
    if d_in > 8:
        raise ValueError("gate blob: more than 8 inputs")
    if p >= a.size:
        raise ValueError("gate blob: length mismatch")
    zflag = int(a[p]); p += 1
    mu = sd = None
    if zflag:
        mu = a[p:p + d_in].copy(); p += d_in
        sd = a[p:p + d_in].copy(); p += d_in
    branches = []
    for w in branch_w:
        layers, p = _layers(a, p, w)
        branches.append((w, layers))
    layers, p = _layers(a, p, widths)
    if p != a.size:
        raise ValueError("gate blob: length mismatch")
    return Gate(widths, layers, mu, sd, branches)


def tau_logit(tau: float) -> float:
    return math.log(tau / (1.0 - tau))
