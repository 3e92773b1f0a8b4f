"""Second, independent float64 formulation of PnP-Nystra for tiny N.

Test infrastructure.  Where the C oracle walks Algorithm 1 step by step with
loops, this module builds the explicit matrices of Sec. 2: the extended
query/key stacks, the extended kernel of Eq. (3) and its blocks, the full
N x N normalised Nystrom kernel of Eq. (8), and divides row-wise.  It is only
used at sizes where N x N matrices are cheap, to catch association,
transposition and normalisation mistakes in the C oracle.
"""
import numpy as np


def pool_indicator(landmark_of_token, m):
    """N x m averaging matrix: column l averages the tokens mapped to l."""
    N = landmark_of_token.shape[0]
    E = np.zeros((N, m))
    E[np.arange(N), landmark_of_token] = 1.0
    return E / E.sum(axis=0, keepdims=True)


def landmarks(Q, K, landmark_of_token, m):
    """Step 1 as a matrix product: Qbar = E^T Q, Kbar = E^T K."""
    E = pool_indicator(landmark_of_token, m)
    return E.T @ Q, E.T @ K


def extended_kernel(Q, K, Qbar, Kbar, scale):
    """Eq. (3): exp of the scaled extended Gram matrix, split in blocks."""
    m = Qbar.shape[0]
    Qt = np.vstack([Qbar, Q])
    Kt = np.vstack([Kbar, K])
    Gt = np.exp(scale * Qt @ Kt.T)
    return Gt, Gt[:m, :m], Gt[:m, m:], Gt[m:, :m], Gt[m:, m:]


def razavi_pinv(A, iters):
    """Step 4 iteration, written in matrix form with numpy operators."""
    m = A.shape[0]
    eye = np.eye(m)
    Z = A.T / (np.abs(A).sum(axis=0).max() * np.abs(A).sum(axis=1).max())
    for _ in range(iters):
        AZ = A @ Z
        Z = 0.25 * Z @ (13 * eye - AZ @ (15 * eye - AZ @ (7 * eye - AZ)))
    return Z


def stabilised_output(Q, K, V, landmark_of_token, m, scale, iters=None, pinv=None):
    """Eq. (8): O = (Ghat^n V) / (Ghat^n 1) with Ghat^n = G_L^n (G_A^n)^+ G_U^n.

    The pseudo-inverse is the Step 4 iteration when ``iters`` is given, else
    ``pinv`` (e.g. numpy.linalg.pinv).
    """
    Qbar, Kbar = landmarks(Q, K, landmark_of_token, m)
    SL = scale * Q @ Kbar.T
    SU = scale * Qbar @ K.T
    SA = scale * Qbar @ Kbar.T
    ML = SL.max(axis=1, keepdims=True)
    MU = SU.max(axis=1, keepdims=True)
    GLn = np.exp(SL - ML)
    GUn = np.exp(SU - MU)
    GAn = np.exp(SA - MU)
    Z = razavi_pinv(GAn, iters) if iters is not None else pinv(GAn)
    Gn = GLn @ Z @ GUn
    return (Gn @ V) / (Gn @ np.ones((Gn.shape[1], 1)))


def unstabilised_output(Q, K, V, landmark_of_token, m, scale, pinv=np.linalg.pinv):
    """Eqs. (6)-(7) without any row-max shift, with a library pseudo-inverse."""
    Qbar, Kbar = landmarks(Q, K, landmark_of_token, m)
    _, GA, GU, GL, _ = extended_kernel(Q, K, Qbar, Kbar, scale)
    Ghat = GL @ pinv(GA) @ GU
    return (Ghat @ V) / (Ghat @ np.ones((Ghat.shape[1], 1)))
