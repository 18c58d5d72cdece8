"""Layer forward/backward definitions in float64 (test infrastructure only).

These are the textbook definitions of the layers the paper's workloads are
built from (Section 4.1: VGG16 and ResNet-152 convolutions, the Transformer
encoder, the residual LSTM, and softmax cross-entropy). Each backward is the
adjoint of its forward written out directly; the gradient tests check them
by central finite differences and against torch CPU.
"""
import numpy as np


# ---------------------------------------------------------------- linear ----

def linear(x, W, b=None):
    """y = x W^T + b, W stored [out, in]."""
    y = x @ W.T
    return y if b is None else y + b


# ------------------------------------------------------- 3x3 convolution ----

def im2col3x3(x):
    """NHWC input [B,H,W,C] -> patches [B*H*W, 3*3*C] for a stride-1, pad-1
    3x3 window, ordered (kh, kw, c) to match a [C_out, kh, kw, C_in] filter."""
    B, H, W, C = x.shape
    xp = np.zeros((B, H + 2, W + 2, C), dtype=np.float64)
    xp[:, 1:H + 1, 1:W + 1, :] = x
    cols = np.empty((B, H, W, 3, 3, C), dtype=np.float64)
    for kh in range(3):
        for kw in range(3):
            cols[:, :, :, kh, kw, :] = xp[:, kh:kh + H, kw:kw + W, :]
    return cols.reshape(B * H * W, 9 * C)


def col2im3x3(dcols, shape):
    """Adjoint of im2col3x3: scatter-add patch gradients back to [B,H,W,C]."""
    B, H, W, C = shape
    d = dcols.reshape(B, H, W, 3, 3, C)
    dxp = np.zeros((B, H + 2, W + 2, C), dtype=np.float64)
    for kh in range(3):
        for kw in range(3):
            dxp[:, kh:kh + H, kw:kw + W, :] += d[:, :, :, kh, kw, :]
    return dxp[:, 1:H + 1, 1:W + 1, :]


def conv3x3_forward(x, Wf):
    """Cross-correlation, stride 1, zero pad 1. x [B,H,W,C_in] NHWC,
    Wf [C_out,3,3,C_in]. Returns [B,H,W,C_out]."""
    B, H, W, _ = x.shape
    cout = Wf.shape[0]
    y = im2col3x3(x) @ Wf.reshape(cout, -1).T
    return y.reshape(B, H, W, cout)


def conv3x3_dgrad(dy, Wf, x_shape):
    cout = Wf.shape[0]
    dcols = dy.reshape(-1, cout) @ Wf.reshape(cout, -1)
    return col2im3x3(dcols, x_shape)


def conv3x3_wgrad(dy, x):
    cout = dy.shape[-1]
    return (dy.reshape(-1, cout).T @ im2col3x3(x)).reshape(cout, 3, 3, x.shape[-1])


def conv1x1_forward(x, Wf):
    """1x1 convolution = per-pixel linear map; Wf [C_out,1,1,C_in]."""
    cout, cin = Wf.shape[0], Wf.shape[-1]
    return (x.reshape(-1, cin) @ Wf.reshape(cout, cin).T).reshape(x.shape[:-1] + (cout,))


def conv1x1_dgrad(dy, Wf):
    cout, cin = Wf.shape[0], Wf.shape[-1]
    return (dy.reshape(-1, cout) @ Wf.reshape(cout, cin)).reshape(dy.shape[:-1] + (cin,))


def conv1x1_wgrad(dy, x):
    cout, cin = dy.shape[-1], x.shape[-1]
    return (dy.reshape(-1, cout).T @ x.reshape(-1, cin)).reshape(cout, 1, 1, cin)


# ------------------------------------------------------------ activations ----

def relu(x):
    return np.maximum(x, 0.0)


def relu_mask(y):
    """Derivative of ReLU read off its output: 1 where y > 0, else 0 (0 at 0)."""
    return (y > 0).astype(np.float64)


def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def softmax_rows(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


# ----------------------------------------------------------- layer norm ----

def layernorm_forward(r, gamma, beta, eps):
    """Normalise each row over the last axis: (r - mean) / sqrt(var + eps),
    var the biased variance, then scale and shift."""
    mu = r.mean(axis=-1, keepdims=True)
    var = ((r - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (r - mu) * rstd
    return gamma * xhat + beta, xhat, rstd


def layernorm_backward(dy, xhat, rstd, gamma):
    """Returns (dr, dgamma, dbeta) for y = gamma * xhat + beta."""
    dgamma = (dy * xhat).reshape(-1, xhat.shape[-1]).sum(axis=0)
    dbeta = dy.reshape(-1, dy.shape[-1]).sum(axis=0)
    dxh = dy * gamma
    dr = rstd * (dxh - dxh.mean(axis=-1, keepdims=True)
                 - xhat * (dxh * xhat).mean(axis=-1, keepdims=True))
    return dr, dgamma, dbeta


# ------------------------------------------------------------- attention ----

def split_heads(t, B, S, H):
    """[B*S, H*dh] -> [B, H, S, dh]."""
    return t.reshape(B, S, H, -1).transpose(0, 2, 1, 3)


def merge_heads(t):
    """[B, H, S, dh] -> [B*S, H*dh]."""
    B, H, S, dh = t.shape
    return t.transpose(0, 2, 1, 3).reshape(B * S, H * dh)


def attention_probs(q, k):
    """P = softmax(q k^T / sqrt(dh)) per (batch, head); q, k [B,H,S,dh]."""
    dh = q.shape[-1]
    return softmax_rows((q @ k.transpose(0, 1, 3, 2)) / np.sqrt(dh))


# -------------------------------------------------------- cross-entropy ----

def softmax_cross_entropy(logits, labels):
    """Mean over rows of -log softmax(logits)[label]; returns (loss, dlogits)
    with dlogits = (softmax - onehot) / rows."""
    n = logits.shape[0]
    m = logits.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(logits - m).sum(axis=1))
    loss = float(np.mean(lse - logits[np.arange(n), labels]))
    p = softmax_rows(logits)
    p[np.arange(n), labels] -= 1.0
    return loss, p / n
