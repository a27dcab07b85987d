"""Winograd F(2x2, 3x3) in numpy fp64 (the transforms the comparison path
uses, written from their definition) and the magnitude sum its rounding-error
bound is stated in.  Test infrastructure, not the HIP path."""
import numpy as np

G = np.array([[1, 0, 0], [0.5, 0.5, 0.5], [0.5, -0.5, 0.5], [0, 0, 1]], dtype=np.float64)
BT = np.array([[1, 0, -1, 0], [0, 1, 1, 0], [0, -1, 1, 0], [0, 1, 0, -1]], dtype=np.float64)
AT = np.array([[1, 1, 1, 0], [0, 1, -1, -1]], dtype=np.float64)


def _patches(x, pad, ho, wo):
    """[C_in, tiles_h, tiles_w, 4, 4] input patches (zero outside the image)."""
    _, c, h, w = x.shape
    th, tw = -(-ho // 2), -(-wo // 2)
    xp = np.zeros((c, 2 * th + 2, 2 * tw + 2), dtype=x.dtype)
    hh, ww = min(h, 2 * th + 2 - pad), min(w, 2 * tw + 2 - pad)
    xp[:, pad:pad + hh, pad:pad + ww] = x[0, :, :hh, :ww]
    idx_r = (2 * np.arange(th))[:, None] + np.arange(4)[None, :]
    idx_c = (2 * np.arange(tw))[:, None] + np.arange(4)[None, :]
    return xp[:, idx_r[:, None, :, None], idx_c[None, :, None, :]]


def winograd_conv(x, w, b, pad, absolute=False, dtype=np.float64):
    """[1, C_out, H_out, W_out]: the F(2x2,3x3) result in fp64, or with
    absolute=True the sum |A^T| (sum_ci (|G||g||G^T|) (.) (|B^T||d||B|)) |A|."""
    x = np.asarray(x, dtype)
    w = np.asarray(w, dtype)
    _, c_in, h, wd = x.shape
    c_out = w.shape[0]
    ho, wo = h + 2 * pad - 2, wd + 2 * pad - 2
    g, bt, at = ((np.abs(G), np.abs(BT), np.abs(AT)) if absolute else (G, BT, AT))
    g, bt, at = g.astype(dtype), bt.astype(dtype), at.astype(dtype)
    ww = np.abs(w) if absolute else w
    d = _patches(x, pad, ho, wo)
    if absolute:
        d = np.abs(d)
    u = np.einsum("ij,ocjk,lk->ocil", g, ww, g)              # [C_out, C_in, 4, 4]
    v = np.einsum("ij,ctujk,lk->ctuil", bt, d, bt)           # [C_in, th, tw, 4, 4]
    m = np.einsum("ocil,ctuil->otuil", u, v)                 # [C_out, th, tw, 4, 4]
    y = np.einsum("ij,otujk,lk->otuil", at, m, at)           # [C_out, th, tw, 2, 2]
    th, tw = y.shape[1], y.shape[2]
    out = y.transpose(0, 1, 3, 2, 4).reshape(c_out, 2 * th, 2 * tw)[:, :ho, :wo]
    if b is not None and not absolute:
        out = out + np.asarray(b, dtype)[:, None, None]
    return out[None]


def error_bound(x, w, pad):
    """Bound on |fp32 Winograd - exact| per output: gamma_{C_in+10} times the
    absolute-value Winograd sum (transform sums of at most 3 + 3 terms on the
    filter, 2 + 2 on the input, 3 + 3 on the output, C_in products)."""
    c_in = x.shape[1]
    u = 2.0 ** -24
    n = c_in + 10
    return n * u / (1 - n * u) * winograd_conv(x, w, None, pad, absolute=True)
