"""Newton-Schulz orthogonalisation, unquantised and NVFP4 (oracle; test infrastructure only).

Section 2 ("Root optimizer") gives the quintic iteration
    X_{k+1} = a X_k + b X_k (X_k^T X_k) + c X_k (X_k^T X_k)^2,
typically five steps.  Section 3.4 gives its NVFP4 form, written with the Gram
matrix on the left (the same polynomial, applied on the short side):
    qX_k = Q_1x16(X_k H),           A_k = qX_k qX_k^T
    qA_k = Q_1x16(A_k H),           qA_k^16x1 = Q_16x1(H^T A_k)
    B_k  = b A_k + c qA_k qA_k^16x1
    qB_k = Q_1x16(B_k H),           qX_k^16x1 = Q_16x1(H^T X_k)
    X_{k+1} = a X_k + qB_k qX_k^16x1
Readings taken where the paper is silent:
* the first line's X is X_k;
* tall matrices (rows > cols) are transposed so that the Gram matrix is the
  short side's (m = min(rows, cols) square);
* X_k, A_k and B_k are binary32 between products; each product's sums are
  exact, rounded once to binary64 (``block_dot64``), then combined in binary64
  as the formulas read and rounded once to binary32 (B_k after its binary64
  combination with b A_k);
* A_k is exactly symmetric, so qA_k^16x1 is qA_k transposed bit for bit and
  B_k's product is the Gram matrix of qA_k;
* before the iteration the momentum is clipped at its p99 magnitude and
  divided by its Frobenius norm plus eps (the Muon convention): X_0 =
  fl32(X' * fl32(1 / (||X'||_F + eps))), the norm summed in binary64.
"""
from __future__ import annotations

import math
import time

import numpy as np
from scipy.linalg.blas import dsyrk

from .formats import E2M1_GRID

from .quantile import clip, clip_threshold
from .quantize import quantize
from .rht import sylvester16, step_signs

MUON_COEFFS = (3.4445, -4.7750, 2.0315)


def gram64(d: np.ndarray) -> np.ndarray:
    """d d^T in binary64, computed on the upper triangle and mirrored (exactly symmetric)."""
    d = np.asarray(d, dtype=np.float64)
    if d.shape[0] == 0:
        return np.zeros((0, 0))
    u = dsyrk(1.0, d, lower=0)
    return np.triu(u) + np.triu(u, 1).T


def _integer_rows(q):
    """Decoded NVFP4 values of every row as (I, e): value = I * 2^(e - 11) per element.

    q * s with q = k / 2 (|k| <= 12) and the E4M3 scale s = M 2^(e - 10) (normal:
    M = 8 + mantissa, e = the exponent field; subnormal: M = mantissa, e = 1), so
    I = k M is an integer with |I| <= 180.  Returns I (float64, exact) and e per
    element (int64), plus each row's largest e over its non-zero elements.
    """
    codes = np.asarray(q.codes)
    sc = np.asarray(q.scales).astype(np.int64)
    rows, cols = codes.shape
    k = np.rint(E2M1_GRID[codes & 7] * 2.0)
    k = np.where(codes & 8, -k, k)
    ef = (sc >> 3) & 15
    mant = sc & 7
    M = np.where(ef == 0, mant, 8 + mant).astype(np.float64)
    e = np.where(ef == 0, 1, ef)
    I = (k.reshape(rows, cols // 16, 16) * M[..., None]).reshape(rows, cols)
    E = np.repeat(e, 16, axis=1)
    emax = np.where(I != 0, E, -1).max(axis=1) if cols else np.full(rows, -1)
    return I, E, emax


def block_dot64(qa, qb=None) -> np.ndarray:
    """binary64 rounding of the exact sums  sum_k D(qa)_ik D(qb)_jk  (D = q * s, no
    tensor scale) for every i, j; qb = None gives the Gram matrix of qa, exactly symmetric.

    Each row is scaled by 2^(-its largest exponent), which leaves integers times powers of
    two no smaller than 2^-(spread); a binary64 BLAS product of such rows is exact in any
    summation order whenever every partial sum fits 53 bits, i.e. when
    K * 180^2 * 2^(spread_a(i) + spread_b(j)) < 2^53.  Entries whose rows fail that
    condition are summed with math.fsum, which is correctly rounded.
    """
    Ia, Ea, ma = _integer_rows(qa)
    if qb is None:
        Ib, Eb, mb = Ia, Ea, ma
    else:
        Ib, Eb, mb = _integer_rows(qb)
    K = Ia.shape[1]
    if K == 0 or Ia.shape[0] == 0 or Ib.shape[0] == 0:
        return np.zeros((Ia.shape[0], Ib.shape[0]))
    sa = np.where(Ia != 0, np.ldexp(1.0, Ea - np.maximum(ma, 0)[:, None]), 0.0)
    sb = np.where(Ib != 0, np.ldexp(1.0, Eb - np.maximum(mb, 0)[:, None]), 0.0)
    ta, tb = Ia * sa, Ib * sb                     # exact: |I| <= 180 times a power of two
    if qb is None:
        u = dsyrk(1.0, ta, lower=0)
        d = np.triu(u) + np.triu(u, 1).T
    else:
        d = ta @ tb.T
    # spread of each row: its largest minus its smallest exponent over non-zero elements
    spa = ma - np.where(Ia != 0, Ea, 99).min(axis=1)
    spb = mb - np.where(Ib != 0, Eb, 99).min(axis=1)
    spa = np.where(ma < 0, 0, spa)
    spb = np.where(mb < 0, 0, spb)
    bits = np.log2(K * 180.0 * 180.0) + spa[:, None] + spb[None, :]
    out = np.ldexp(d, (np.maximum(ma, 0)[:, None] + np.maximum(mb, 0)[None, :]) - 22)
    bad = np.argwhere(bits >= 53.0)
    if len(bad):
        va = Ia * np.ldexp(1.0, Ea - 11)
        vb = Ib * np.ldexp(1.0, Eb - 11)
        for i, j in bad:
            out[i, j] = math.fsum(va[i] * vb[j])   # each product exact (at most 16 bits)
    return out


def f32(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def normalise(x: np.ndarray, eps: float = 1e-7) -> np.ndarray:
    """X_0 = fl32(X * fl32(1 / (||X||_F + eps))) with the norm summed in binary64."""
    x = np.asarray(x, dtype=np.float32)
    nu = np.sqrt(np.sum(np.square(x.astype(np.float64))))
    inv = np.float32(1.0 / (nu + np.float64(np.float32(eps))))
    return (x * inv).astype(np.float32)


class _Clock:
    """Optional wall-clock accounting of the oracle's parts (for a CPU baseline):
    seconds spent quantising and in products, added to the dict it is given."""

    def __init__(self, sink):
        self.sink = sink

    def __call__(self, part, fn, *args):
        if self.sink is None:
            return fn(*args)
        t0 = time.perf_counter()
        out = fn(*args)
        self.sink[part] = self.sink.get(part, 0.0) + time.perf_counter() - t0
        return out


def ns_step_nvfp4(x, a, b, c, signs=None, adaptive46=True, trace=None, timing=None):
    """One NVFP4 NS step on a binary32 m x n matrix (Section 3.4 display equation)."""
    clk = _Clock(timing)
    x = np.asarray(x, dtype=np.float32)
    a64, b64, c64 = (np.float64(np.float32(t)) for t in (a, b, c))
    qx = clk("quantize", quantize, x, 1, signs, adaptive46)
    qxt = clk("quantize", quantize, x, 0, signs, adaptive46)
    A = f32((np.float64(qx.sg) * np.float64(qx.sg)) * clk("products", block_dot64, qx))
    qa = clk("quantize", quantize, A, 1, signs, adaptive46)
    P = (np.float64(qa.sg) * np.float64(qa.sg)) * clk("products", block_dot64, qa)
    B = f32(b64 * A.astype(np.float64) + c64 * P)
    qb = clk("quantize", quantize, B, 1, signs, adaptive46)
    prod = clk("products", block_dot64, qb, qxt)
    x1 = f32(a64 * x.astype(np.float64) + (np.float64(qb.sg) * np.float64(qxt.sg)) * prod)
    if trace is not None:
        trace.update(qx=qx, qxt=qxt, A=A, qa=qa, B=B, qb=qb)
    return x1


def rotate64(x: np.ndarray, signs: np.ndarray, axis: int) -> np.ndarray:
    """Exact binary64 rotation X H (axis=1) or H^T X (axis=0) with H = diag(d) H_16 / 4."""
    h = np.diag(signs.astype(np.float64)) @ sylvester16() / 4.0
    x = np.asarray(x, dtype=np.float64)
    if axis == 1:
        r, c = x.shape
        return (x.reshape(r, c // 16, 16) @ h).reshape(r, c)
    r, c = x.shape
    return np.einsum("ij,bjc->bic", h.T, x.reshape(r // 16, 16, c)).reshape(r, c)


def ns_step_exact(x, a, b, c, signs=None):
    """One unquantised binary64 NS step in the Section 3.4 arrangement.

    With ``signs`` the rotations of Section 3.4 are applied on both sides of
    every product (quantisation replaced by the identity); they cancel exactly
    in exact arithmetic, which is what the placement of H must achieve.
    """
    x = np.asarray(x, dtype=np.float64)
    if signs is None:
        A = x @ x.T
        B = b * A + c * (A @ A)
        return a * x + B @ x
    xh = rotate64(x, signs, 1)
    A = xh @ xh.T
    B = b * A + c * (rotate64(A, signs, 1) @ rotate64(A, signs, 0))
    return a * x + rotate64(B, signs, 1) @ rotate64(x, signs, 0)


def to_bf16(x) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits, ties to even) of each finite input, as float64."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                      # x = m * 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0), e - 8)


def ns_step_bf16(x, a, b, c):
    """One step of the plain BF16 comparison path: X_k binary32 master, bf16 operands.

    Xb = bf16(X_k); A = bf16(Xb Xb^T); B = bf16(b A + c A A); X_{k+1} = fl32(a X_k + B Xb),
    each product exact in binary64 before its single rounding.
    """
    x = np.asarray(x, dtype=np.float32)
    xb = to_bf16(x)
    A = to_bf16(gram64(xb))
    B = to_bf16(np.float64(np.float32(b)) * A + np.float64(np.float32(c)) * gram64(A))
    return f32(np.float64(np.float32(a)) * x.astype(np.float64) + B @ xb)


def canonical(m: np.ndarray):
    m = np.asarray(m, dtype=np.float32)
    tall = m.shape[0] > m.shape[1]
    return (np.ascontiguousarray(m.T) if tall else m), tall


def prepare(m, clip_on=True, q=0.99, eps=1e-7):
    """Clip (optional), orient (short side first) and normalise: returns (X_0, tall, tau)."""
    m = np.asarray(m, dtype=np.float32)
    tau = clip_threshold(m, q) if clip_on else np.float32(np.inf)
    mc = clip(m, tau) if clip_on else m
    x, tall = canonical(mc)
    return normalise(x, eps), tall, tau


def orthogonalize(m, coeffs, clip_on=True, q=0.99, eps=1e-7, hadamard=True,
                  adaptive46=True, seed=0, mode="nvfp4", timing=None):
    """Clip, normalise and run len(coeffs) NS steps; returns binary32 in the input's orientation.

    mode: "nvfp4" (Section 3.4), "bf16" (plain BF16 comparison path) or "exact"
    (binary64, no quantisation; returns float64).  timing: optional dict that
    receives the seconds spent in "prepare", "quantize" and "products".
    """
    x, tall, _ = _Clock(timing)("prepare", prepare, m, clip_on, q, eps)
    if mode == "exact":
        x = x.astype(np.float64)
    for k, (a, b, c) in enumerate(coeffs):
        if mode == "nvfp4":
            signs = step_signs(seed, k) if hadamard else None
            x = ns_step_nvfp4(x, a, b, c, signs, adaptive46, timing=timing)
        elif mode == "bf16":
            x = ns_step_bf16(x, a, b, c)
        elif mode == "exact":
            x = ns_step_exact(x, a, b, c)
        else:
            raise ValueError(mode)
    return np.ascontiguousarray(x.T) if tall else x


def poly(sig, a, b, c):
    """The scalar map one NS step applies to each singular value: a s + b s^3 + c s^5."""
    return a * sig + b * sig ** 3 + c * sig ** 5


def closed_form(x, coeffs):
    """U diag(p_S(...p_1(sigma))) V^T from a binary64 SVD: what exact NS must return."""
    u, s, vt = np.linalg.svd(np.asarray(x, dtype=np.float64), full_matrices=False)
    for (a, b, c) in coeffs:
        s = poly(s, a, b, c)
    return (u * s) @ vt
