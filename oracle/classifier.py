"""The FDCNN classifier head and one training step, in float64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Section 2.5.1 (Fig. 3): after the final inverse transform of the FDCNN a ReLU feeds
the fully connected layers.  Section 3.1: the loss is cross-entropy and the
optimiser Adam with a learning rate and a weight decay.

Readings taken here (listed with their reasons in the design notes):

* The sizes of the fully connected layers are only in Fig. 3, whose numbers the text
  does not carry; the head is one fully connected layer from the flattened ReLU
  output (C * M * M features, channel-major as the tensor is laid out) to the
  classes.
* Cross-entropy is the softmax cross-entropy averaged over the batch.
* Adam is the algorithm of Kingma and Ba with bias correction; the weight decay is
  added to the gradient (L2 form), as the optimiser the paper names applies it.  A
  complex parameter is updated as its (re, im) pairs.
"""

import numpy as np

from . import fdc


def relu(y):
    return np.maximum(y, 0.0)


def head_forward(y, W, bias, labels):
    """y [B][F], W [classes][F], bias [classes], labels [B] ->
    (logits [B][classes], mean cross-entropy)."""
    y = np.asarray(y, np.float64).reshape(len(labels), -1)
    logits = relu(y) @ np.asarray(W, np.float64).T + np.asarray(bias, np.float64)
    B = logits.shape[0]
    loss = 0.0
    for b in range(B):
        row = logits[b]
        m = row.max()
        lse = m + np.log(np.sum(np.exp(row - m)))
        loss += lse - row[labels[b]]
    return logits, loss / B


def head_backward(y, W, logits, labels):
    """(gy [B][F], gW [classes][F], gbias [classes]) of the mean cross-entropy."""
    y = np.asarray(y, np.float64).reshape(len(labels), -1)
    B, classes = logits.shape
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    dl = p.copy()
    dl[np.arange(B), labels] -= 1.0
    dl /= B
    gW = dl.T @ relu(y)
    gbias = dl.sum(axis=0)
    gy = (dl @ np.asarray(W, np.float64)) * (y > 0)
    return gy, gW, gbias


def adam_step(p, g, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0):
    """One Adam step on real arrays (a complex parameter as its (re, im) pairs).
    Returns new (p, m, v)."""
    p, g, m, v = (np.asarray(a, np.float64) for a in (p, g, m, v))
    g = g + weight_decay * p
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** step)
    v_hat = v / (1.0 - beta2 ** step)
    return p - lr * m_hat / (np.sqrt(v_hat) + eps), m, v


def classifier_gradients(x, kernels, W, bias, labels, sizes):
    """Forward and backward of the FDCNN classifier: the spectral chain of section 2.5.1
    (``fdc.cic_chain_forward``), ReLU, the fully connected layer, the mean
    cross-entropy.  Returns (loss, logits, [dL/dK per layer], dL/dW, dL/dbias)."""
    y, saved = fdc.cic_chain_forward(x, kernels, sizes)
    B = y.shape[0]
    logits, loss = head_forward(y.reshape(B, -1), W, bias, labels)
    gy, gW, gbias = head_backward(y.reshape(B, -1), W, logits, labels)
    gks, _ = fdc.cic_chain_backward(gy.reshape(y.shape), saved, kernels, sizes)
    return loss, logits, gks, gW, gbias
