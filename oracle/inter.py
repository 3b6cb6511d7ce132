"""Inter-channel CG convolution with a per-degree channel reduction, for the
oracle (test infrastructure only).

Paper §4.1: features with m and m' channels give a tensor product with
(2J+1) m m' components per output degree J (every channel of the query meets
every channel of the key), heads do not interact in the product, and the
multiplicity is reduced again by a learned equivariant map.  Read here with
C = H m channels in H heads of m (channel c = h m + c'), and the reduction as
one real matrix per head and output degree (a linear map on multiplicities
commutes with rotations only if it acts alike on the 2J+1 components of a
degree):

    u[b,i,(J,M),h,c1,c2] = sum_{paths} sum_{m1,m2} R^{(l1 l2 J)}[M,m1,m2]
                           sum_j q[b,j,(l1,m1),h m+c1] k[b,(i-j) mod N,(l2,m2),h m+c2]
    out[b,i,(J,M),h m_o+o] = sum_{c1,c2} W[h,J,o,c1 m+c2] u[b,i,(J,M),h,c1,c2]

W has shape (H, L+1, m_o, m*m).  ``interchannel_products`` is the unreduced
product u (H m^2 channels, channel h m^2 + c1 m + c2): the depthwise
convolution of the oracle applied to every channel pair of a head.
``cgconv_interchannel`` applies W to it degree by degree.  ``mode`` selects
the depthwise oracle's direct (definition) or FFT mode.  float64 throughout.
"""

from __future__ import annotations

import numpy as np

from .cg import n_comp
from .conv import cgconv_direct, cgconv_fft


def pair_channels(q, k, heads: int):
    """The query and key channels of every pair (h, c1, c2): arrays of
    shape (B, N, K, H*m*m) with channel h m^2 + c1 m + c2 holding q channel
    h m + c1 and k channel h m + c2."""
    q = np.asarray(q)
    k = np.asarray(k)
    B, N, K, C = q.shape
    if C % heads:
        raise ValueError("C must be a multiple of heads")
    m = C // heads
    qh = q.reshape(B, N, K, heads, m, 1)
    kh = k.reshape(B, N, K, heads, 1, m)
    qe = np.broadcast_to(qh, (B, N, K, heads, m, m)).reshape(B, N, K, heads * m * m)
    ke = np.broadcast_to(kh, (B, N, K, heads, m, m)).reshape(B, N, K, heads * m * m)
    return qe, ke


def interchannel_products(q, k, L: int, heads: int, mode: str = "direct") -> np.ndarray:
    """Unreduced inter-channel convolution, (B, N, K, H*m*m) float64."""
    qe, ke = pair_channels(q, k, heads)
    if mode == "direct":
        return cgconv_direct(qe, ke, L)
    if mode == "fft":
        return cgconv_fft(qe, ke, L)
    raise ValueError("mode must be 'direct' or 'fft'")


def reduce_degrees(u, L: int, heads: int, W) -> np.ndarray:
    """out[..., (J,M), h m_o + o] = sum_pair W[h, J, o, pair] u[..., (J,M), h m^2 + pair]."""
    u = np.asarray(u, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    B, N, K, P = u.shape
    if K != n_comp(L) or W.ndim != 4 or W.shape[0] != heads or W.shape[1] != L + 1:
        raise ValueError("W must have shape (heads, L+1, m_o, m*m)")
    mo, pairs = W.shape[2], W.shape[3]
    if P != heads * pairs:
        raise ValueError("u has the wrong channel count for W")
    out = np.zeros((B, N, K, heads * mo))
    uh = u.reshape(B, N, K, heads, pairs)
    for J in range(L + 1):
        sl = slice(J * J, (J + 1) ** 2)
        # (B, N, 2J+1, H, pairs) x (H, m_o, pairs) -> (B, N, 2J+1, H, m_o)
        out[:, :, sl, :] = np.einsum("bnkhp,hop->bnkho", uh[:, :, sl], W[:, J]).reshape(B, N, 2 * J + 1, heads * mo)
    return out


def cgconv_interchannel(q, k, L: int, heads: int, W, mode: str = "direct") -> np.ndarray:
    """Inter-channel convolution reduced per degree: (B, N, K, H*m_o) float64."""
    return reduce_degrees(interchannel_products(q, k, L, heads, mode), L, heads, W)
