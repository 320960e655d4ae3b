"""Layer-level operations of the UNet, float64, one image at a time.

Images are H x W x C arrays (channels last).  Every function is the plain
textbook definition; see the per-function notes for the source.
"""
import math
import numpy as np
from scipy.special import erf

F = np.float64


def timestep_embedding(t, dim):
    """Sinusoidal timestep embedding (Vaswani et al. 2017, Sec. 3.5 form) in
    the latent-diffusion convention: e = [cos(t f_i) | sin(t f_i)], i < dim/2,
    with f_i = 10000^(-i / (dim/2)) and t taken as a real number."""
    h = dim // 2
    i = np.arange(h, dtype=F)
    f = np.exp(-math.log(10000.0) * i / h)
    a = F(t) * f
    return np.concatenate([np.cos(a), np.sin(a)])


def silu(x):
    """SiLU / swish: x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def gelu(x):
    """Exact GELU: x * Phi(x) with the normal CDF Phi (Hendrycks & Gimpel 2016)."""
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def linear(x, w, b=None):
    """y = x W^T + b with W stored (out, in); x may have leading axes."""
    shp = x.shape
    y = np.ascontiguousarray(x).reshape(-1, shp[-1]) @ np.asarray(w, F).T
    y = y.reshape(shp[:-1] + (y.shape[-1],))
    if b is not None:
        y = y + np.asarray(b, F)
    return y


def conv2d(x, w, b=None, stride=1):
    """2-D cross-correlation with zero padding (k-1)/2, NHWC input.

    x: (H, W, Cin); w: (Cout, Cin, k, k).  Output pixel (y, x) at stride s is
    b[o] + sum over input channels c and taps (ky, kx) of
    xpad[s*y + ky, s*x + kx, c] * w[o, c, ky, kx],
    evaluated as one product of the patch matrix (one row per output pixel,
    columns ordered like w's (c, ky, kx)) with w reshaped to (Cout, Cin*k*k).
    """
    w = np.asarray(w, F)
    cout, cin, k, _ = w.shape
    p = (k - 1) // 2
    H, W, _ = x.shape
    Ho = (H + 2 * p - k) // stride + 1
    Wo = (W + 2 * p - k) // stride + 1
    xp = np.zeros((H + 2 * p, W + 2 * p, cin), F)
    xp[p:p + H, p:p + W] = x
    patches = np.empty((Ho * Wo, cin, k * k), F)
    for ky in range(k):
        for kx in range(k):
            tap = xp[ky:ky + stride * (Ho - 1) + 1:stride, kx:kx + stride * (Wo - 1) + 1:stride]
            patches[:, :, ky * k + kx] = tap.reshape(Ho * Wo, cin)
    out = patches.reshape(Ho * Wo, cin * k * k) @ w.reshape(cout, cin * k * k).T
    if b is not None:
        out += np.asarray(b, F)
    return out.reshape(Ho, Wo, cout)


def upsample_nearest2x(x):
    """Nearest-neighbour 2x upsampling: out[y, x] = in[y // 2, x // 2]."""
    return np.repeat(np.repeat(x, 2, axis=0), 2, axis=1)


def group_norm(x, groups, gamma, beta, eps):
    """GroupNorm (Wu & He 2018): channels split into `groups` runs of
    consecutive channels; each run is normalised with its mean and biased
    variance over all its channels and pixels, then scaled per channel."""
    H, W, C = x.shape
    g = x.reshape(H * W, groups, C // groups)
    mean = g.mean(axis=(0, 2), keepdims=True)
    var = ((g - mean) ** 2).mean(axis=(0, 2), keepdims=True)
    y = ((g - mean) / np.sqrt(var + eps)).reshape(H, W, C)
    return y * np.asarray(gamma, F) + np.asarray(beta, F)


def layer_norm(x, gamma, beta, eps=1e-5):
    """LayerNorm (Ba et al. 2016) over the last axis, biased variance."""
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)
    return (x - mean) / np.sqrt(var + eps) * np.asarray(gamma, F) + np.asarray(beta, F)


def softmax(s, axis=-1):
    m = s.max(axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=axis, keepdims=True)


def attention(q, k, v, heads):
    """Multi-head scaled dot-product attention (Vaswani et al. 2017, Eq. 1).

    q: (Nq, C), k and v: (Nk, C).  Head h uses channels [h*d, (h+1)*d) with
    d = C / heads; O_h = softmax(Q_h K_h^T / sqrt(d)) V_h; heads are
    concatenated back in channel order.
    """
    C = q.shape[1]
    d = C // heads
    out = np.empty((q.shape[0], C), F)

    for h in range(heads):
        sl = slice(h * d, (h + 1) * d)
        p = softmax(np.ascontiguousarray(q[:, sl]) @ np.ascontiguousarray(k[:, sl]).T / math.sqrt(d))
        out[:, sl] = p @ np.ascontiguousarray(v[:, sl])
    return out
