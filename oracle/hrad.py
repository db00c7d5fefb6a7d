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
available: the weights are the caller's.  h^k is the residual stream after
layer L - K + k (k = 1..K), in the order the layers run.

Softmax is monotone, so s_t is the argmax of the MLP's logits; ties go to
the lowest class index.  Computed in float64.
"""
from __future__ import annotations

import numpy as np

HIDDEN = (256, 64)
CLASSES = 3


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
