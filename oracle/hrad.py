"""Oracle of H-RAD's length predictor (test infrastructure only).

Section "H-RAD" (equations for z_t and s_t): the features of the next
round are the target model's hidden states at the last position t-1 from
its last K layers, concatenated with the embedding of the new token,

    z_t = Concat(h^1_{t-1}, ..., h^K_{t-1}, e_t),

and a small MLP maps them to a class

    s_t = argmax(Softmax(MLP(z_t))) in {0, 1, 2}
          (0: all reject, 1: use the draft's confidence, 2: all accept).

The MLP has two hidden layers of 256 and 64 units with ReLU and a 3-way
output layer (Appendix, "H-RAD Training"; dropout is a training-time
device and is absent at inference).  The trained weights are not
available: the weights are the caller's.

Which form a "hidden state of layer l" takes (the paper names the states,
not their form): h^k, k = 1..K-1, is the residual stream after layer
L - K + k, in the order the layers run, and the last one, h^K, is the output
of the final RMSNorm applied to the residual after layer L.  These are the
last K hidden states a library Llama model reports (its last entry is
normalised), the form a predictor trained on that model's features reads.

Softmax is monotone, so s_t is the argmax of the MLP's logits; ties go to
the lowest class index.  Computed in float64.
"""
from __future__ import annotations

import numpy as np

HIDDEN = (256, 64)
CLASSES = 3


def tapped_states(hidden, final_norm, eps: float, k: int) -> list:
    """The last k hidden states from the residual stream after every layer
    (``hidden``, layer 0 first): the residuals after layers L-k+1..L-1, then
    the final norm's output RMSNorm(h_L) g_f, all in float64."""
    L = len(hidden)
    out = [np.asarray(hidden[l], dtype=np.float64) for l in range(L - k, L - 1)]
    h = np.asarray(hidden[-1], dtype=np.float64)
    r = 1.0 / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)
    out.append(h * r * np.asarray(final_norm, dtype=np.float64))
    return out


def features(hidden_last_k, embed_row) -> np.ndarray:
    """z_t: the K hidden-state rows (layer L-K+1 first) then the embedding."""
    parts = [np.asarray(h, dtype=np.float64).reshape(-1) for h in hidden_last_k]
    parts.append(np.asarray(embed_row, dtype=np.float64).reshape(-1))
    return np.concatenate(parts)


def mlp_logits(z, w1, b1, w2, b2, w3, b3) -> np.ndarray:
    """Two ReLU layers and the output layer, y = W x + b each, float64."""
    x = np.asarray(z, dtype=np.float64)
    x = np.maximum(np.asarray(w1, np.float64) @ x + np.asarray(b1, np.float64), 0.0)
    x = np.maximum(np.asarray(w2, np.float64) @ x + np.asarray(b2, np.float64), 0.0)
    return np.asarray(w3, np.float64) @ x + np.asarray(b3, np.float64)


def predict(z, w1, b1, w2, b2, w3, b3):
    """(logits, s_t): s_t the lowest index of the largest logit."""
    lg = mlp_logits(z, w1, b1, w2, b2, w3, b3)
    return lg, int(np.argmax(lg))
