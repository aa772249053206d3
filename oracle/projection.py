"""Role-routed linear projection (oracle; test infrastructure only).

Sec. 3.1 gives Nexus tokens their own projection matrices (W_Q^N, W_K^N,
W_V^N, W_O^N) and their own MLP branches, while every other token (system
prompt, history text, current query and generated tokens) keeps the model's
standard ones.  Each of those layers is one linear map applied per token with
the weight set its role selects:

    y[t] = W_N x[t]    if role[t] is NEXUS
    y[t] = W   x[t]    otherwise

with x[t] a row of K inputs, W and W_N of shape [N, K] (the output-by-input
layout of a linear layer) and y[t] a row of N outputs.  Inputs and weights are
bf16 bit patterns, widened exactly; the products are summed in float64.
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_bits_to_f64
from .layout import NEXUS


def role_routed_linear(x, role, w_text, w_nexus) -> np.ndarray:
    """y [T, N] float64 for x [T, K] (bf16 bits), role [T], weights [N, K] (bf16 bits)."""
    x = bf16_bits_to_f64(x)
    wt = bf16_bits_to_f64(w_text)
    wn = bf16_bits_to_f64(w_nexus)
    nexus = np.asarray(role) == NEXUS
    y = np.empty((x.shape[0], wt.shape[0]), dtype=np.float64)
    y[~nexus] = x[~nexus] @ wt.T
    y[nexus] = x[nexus] @ wn.T
    return y
