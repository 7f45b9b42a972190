"""GraphSAGE forward on prepared minibatches -- TEST INFRASTRUCTURE ONLY.

Only the tests may import this module; the GPU library never loads it.

Eq. (1) (Sec. 3.1) updates a node's embedding from its own embedding and an
aggregate of its neighbours' embeddings.  The reading used here is GraphSAGE
with the mean aggregator: layer i runs on hop l = L-1-i of a minibatch's
sampled blocks; for every destination node v of that hop

    m_v = mean of h_u over v's sampled neighbours u (zero when there are none)
    z_v = W_i [h_v ; m_v] + b_i,   h'_v = max(z_v, 0) except on the last layer,

with h the layer's input rows in local-id order (layer 0: the node features).
Everything here is float64.  ``forward`` also returns an elementwise bound on
the error of a computation that rounds [h_v ; m_v] to bf16, multiplies with
bf16 weights accumulating in float32, sums the mean in float32, and stores
hidden embeddings as bf16 (the GPU kernels' arithmetic), derived by first-order
forward error analysis:
  - rounding to bf16 (8 significant bits, nearest): relative error <= 2^-8;
  - a float32 sum of n terms, and the division of the mean: <= (n+1) 2^-24
    times the sum of magnitudes;
  - a float32 dot product of K exact products plus the bias: <= (K+2) 2^-24
    times the sum of magnitudes;
  - ReLU does not increase an error.
"""
from __future__ import annotations

import numpy as np

U_BF16 = 2.0 ** -8
U_F32 = 2.0 ** -24


def bf16_bits_to_f64(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def features_f64(features, feat_dtype: str) -> np.ndarray:
    f = np.asarray(features)
    if feat_dtype == "bfloat16":
        return bf16_bits_to_f64(f)
    return f.astype(np.float64)


def forward(mb, X: np.ndarray, weights, biases):
    """One minibatch.  mb: oracle.Minibatch; X: float64 feature rows of all graph
    nodes; weights[i]: bf16 bits [dims[i+1]][2 dims[i]]; biases[i]: float32.
    Returns (out [B][dims[L]], bound [B][dims[L]])."""
    L = len(mb.row_ptr)
    h = X[np.asarray(mb.nodes, dtype=np.int64)]
    E = np.zeros_like(h)
    for i in range(L):
        l = L - 1 - i
        nd = int(mb.layer_sizes[l])
        rp = np.asarray(mb.row_ptr[l], dtype=np.int64)
        col = np.asarray(mb.col[l], dtype=np.int64)
        din = h.shape[1]
        mean = np.zeros((nd, din))
        Em = np.zeros((nd, din))
        for v in range(nd):
            nb = col[rp[v]:rp[v + 1]]
            if len(nb):
                mean[v] = h[nb].sum(axis=0) / len(nb)
                Em[v] = (E[nb].sum(axis=0) + (len(nb) + 1) * U_F32 * (np.abs(h[nb]) + E[nb]).sum(axis=0)) / len(nb)
        A = np.concatenate([h[:nd], mean], axis=1)
        EA = np.concatenate([E[:nd], Em], axis=1)
        EA = EA + U_BF16 * (np.abs(A) + EA)
        W = bf16_bits_to_f64(weights[i])                      # [dout][2 din]
        b = np.asarray(biases[i], dtype=np.float64)
        Z = A @ W.T + b
        Wa = np.abs(W)
        EZ = EA @ Wa.T + (W.shape[1] + 2) * U_F32 * ((np.abs(A) + EA) @ Wa.T + np.abs(b))
        if i + 1 < L:
            h = np.maximum(Z, 0.0)
            E = EZ + U_BF16 * (np.abs(Z) + EZ)
        else:
            h = Z
            E = EZ + U_F32 * (np.abs(Z) + EZ)
    return h, E


def forward_hyperbatch(mbs, X, weights, biases):
    outs, bounds = zip(*[forward(mb, X, weights, biases) for mb in mbs])
    return np.concatenate(outs), np.concatenate(bounds)


def simulate_low_precision(mb, X: np.ndarray, weights, biases) -> np.ndarray:
    """The same forward with the kernels' rounding points emulated on the CPU
    (bf16 operands, float32 sums and products, bf16 hidden storage); used only
    to check that ``forward``'s bound covers that arithmetic."""
    def bf16(x):
        f = np.asarray(x, dtype=np.float32)
        u = f.view(np.uint32).astype(np.uint64)
        u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
        return bf16_bits_to_f64(u.astype(np.uint16)).astype(np.float32)
    L = len(mb.row_ptr)
    h = X[np.asarray(mb.nodes, dtype=np.int64)].astype(np.float32)
    for i in range(L):
        l = L - 1 - i
        nd = int(mb.layer_sizes[l])
        rp = np.asarray(mb.row_ptr[l], dtype=np.int64)
        col = np.asarray(mb.col[l], dtype=np.int64)
        mean = np.zeros((nd, h.shape[1]), np.float32)
        for v in range(nd):
            nb = col[rp[v]:rp[v + 1]]
            if len(nb):
                acc = np.zeros(h.shape[1], np.float32)
                for u in nb:
                    acc = (acc + h[u]).astype(np.float32)
                mean[v] = (acc / np.float32(len(nb))).astype(np.float32)
        A = bf16(np.concatenate([h[:nd], mean], axis=1))
        W = bf16_bits_to_f64(weights[i]).astype(np.float32)
        Z = np.zeros((nd, W.shape[0]), np.float32)
        for k in range(W.shape[1]):                            # float32 accumulation, one product at a time
            Z = (Z + np.outer(A[:, k], W[:, k]).astype(np.float32)).astype(np.float32)
        Z = (Z + np.asarray(biases[i], np.float32)).astype(np.float32)
        h = bf16(np.maximum(Z, 0)) if i + 1 < L else Z
    return h.astype(np.float64)
