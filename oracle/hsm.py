"""CPU oracle of the Hidden State Mapper (Section 4.2; Appendix B, Table S1,
Fig. S1), fp64 numpy.

TEST INFRASTRUCTURE ONLY (see adept_oracle): only the test suite and the
bench's CPU leg may use it; the product path never calls it.

The mapper turns an exiting token's state into an estimate of its final
state from three inputs: the current state s_i, the previous layer's state
s_{i-1} and the inertia of Eq. 7 (the sum of unit states before layer i,
i.e. the inertia the exit test of layer i compared against).  Table S1 lists
the layers; the paper leaves open what is read here as follows:

  * one RMS normalisation with one gain vector g0 [D] is applied to each of
    the three states separately (the table has one Normalization row, the
    text says the three states are normalised separately);
  * the normalised states are stacked in the order (current, previous,
    inertia) into a one-channel 3 x D plane; the convolution is a 3 x 3
    kernel with stride 1 and padding (0, 1), so its output is 1 x D, plus a
    scalar bias;
  * the four fully connected layers carry biases (nn.Linear's default); the
    exact-erf GELU follows FC1 and FC2 (the paper names no activation; an
    MLP without one would be a single linear map);
  * the first Add takes FC1's output as its skip input and the second Add
    the convolution output;
  * the two later Normalization rows are RMS normalisations with their own
    gains g1 [4D] and g2 [D].

Parameter count: 4D^2 + 32D^2 + 32D^2 + 4D^2 = 72 D^2 plus O(D) vectors,
which gives the 42.5M (BERT-base, D = 768) and 184M (GPT2-XL, D = 1600) of
Table 2.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .adept_oracle import F64, gelu_erf, rms_norm


@dataclasses.dataclass
class HSMWeights:
    g0: np.ndarray      # [D] input normalisation gain (shared by the three states)
    conv: np.ndarray    # [3, 3]: row r = state (current, previous, inertia), column t = offset t-1
    conv_b: float
    w1: np.ndarray      # [4D, D]
    b1: np.ndarray
    w2: np.ndarray      # [8D, 4D]
    b2: np.ndarray
    w3: np.ndarray      # [4D, 8D]
    b3: np.ndarray
    g1: np.ndarray      # [4D]
    w4: np.ndarray      # [D, 4D]
    b4: np.ndarray
    g2: np.ndarray      # [D]

    @property
    def d_model(self):
        return self.g0.shape[0]


def n_params(d_model: int) -> int:
    """Trainable parameters of the mapper at width D (Table S1 layers)."""
    D = d_model
    fc = (D * 4 * D + 4 * D) + (4 * D * 8 * D + 8 * D) + (8 * D * 4 * D + 4 * D) + (4 * D * D + D)
    norms = D + 4 * D + D
    return fc + norms + 9 + 1


def conv3x3(x3, kernel, bias):
    """One-channel 3 x D plane, 3 x 3 kernel, stride 1, padding (0, 1):
    out[d] = bias + sum_r sum_t kernel[r, t] * x3[r, d + t - 1], zero outside."""
    x3 = np.asarray(x3, F64)
    D = x3.shape[-1]
    padded = np.zeros(x3.shape[:-1] + (D + 2,))
    padded[..., 1:D + 1] = x3
    out = np.full(x3.shape[:-2] + (D,), float(bias))
    for r in range(3):
        for t in range(3):
            out = out + kernel[r, t] * padded[..., r, t:t + D]
    return out


def hsm_forward(w: HSMWeights, s_cur, s_prev, inertia, eps):
    """Mapped states s~ [n, D] of n exiting tokens (rows of the inputs)."""
    x3 = np.stack([rms_norm(s_cur, w.g0, eps), rms_norm(s_prev, w.g0, eps),
                   rms_norm(inertia, w.g0, eps)], axis=-2)          # [n, 3, D]
    u = conv3x3(x3, np.asarray(w.conv, F64), w.conv_b)              # [n, D]
    a = u @ np.asarray(w.w1, F64).T + w.b1                           # FC1: [n, 4D]
    b = gelu_erf(a) @ np.asarray(w.w2, F64).T + w.b2                 # FC2: [n, 8D]
    c = gelu_erf(b) @ np.asarray(w.w3, F64).T + w.b3                 # FC3: [n, 4D]
    d = rms_norm(c, w.g1, eps) + a                                   # Norm, Add (skip: FC1)
    e = d @ np.asarray(w.w4, F64).T + w.b4                           # FC4: [n, D]
    return rms_norm(e, w.g2, eps) + u                                # Norm, Add (skip: conv)
