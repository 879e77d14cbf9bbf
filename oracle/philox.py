"""Philox4x64-10 and the random streams of the ORF draw (oracle side).

Test infrastructure only (see ``oracle/__init__``).

The paper draws omega_i from a Gaussian and b_i uniformly on (0, 2 pi)
(Sec. 2.3) but does not say how. Both the oracle and the GPU library therefore
implement one counter-based generator from its published definition:
Philox4x64 with 10 rounds (J. Salmon, M. Moraes, R. Dror, D. Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC'11). A round maps counter (c0,c1,c2,c3)
and key (k0,k1) to (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1,
lo(M0 c0)); the key is bumped by the Weyl constants between rounds.

Stream definition (shared contract with the library, restated in its header):
  key      = (seed, 0)
  counter  = (index, head, purpose, 0)      purpose: 0 ORF Gaussian blocks,
                                                     1 chi row-norm Gaussians,
                                                     2 phases b,
                                                     3 Hadamard-block signs,
                                                     4 Givens rotations
  one call -> four 64-bit words w0..w3 -> eight 32-bit words
              x[2j] = low half of wj, x[2j+1] = high half of wj
  element n of a stream is word n % 8 of the call with index n // 8.
  uniform   u = (x + 0.5) * 2^-32, strictly inside (0, 1)
  Gaussian  pairs (u[2p], u[2p+1]) -> r = sqrt(-2 ln u[2p]),
            z[2p] = r cos(2 pi u[2p+1]), z[2p+1] = r sin(2 pi u[2p+1])  (Box-Muller)
"""
import numpy as np

# Philox4x64 multipliers and Weyl key increments as published by Salmon et al.
_M0 = 0xD2E7470EE14C6C93
_M1 = 0xCA5A826395121157
_W0 = 0x9E3779B97F4A7C15
_W1 = 0xBB67AE8584CAA73B
_ROUNDS = 10

PURPOSE_ORF = 0
PURPOSE_CHI = 1
PURPOSE_PHASE = 2
PURPOSE_SIGNS = 3       # Rademacher diagonals of Hadamard ORF blocks
PURPOSE_GIVENS = 4      # coordinate pairs and angles of Givens ORF blocks

_LO32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo64(a, m):
    """Full 128-bit product of uint64 arrays a and the constant m: (hi, lo)."""
    a = a.astype(np.uint64)
    a0 = a & _LO32
    a1 = a >> _S32
    m0 = np.uint64(m & 0xFFFFFFFF)
    m1 = np.uint64(m >> 32)
    p00 = a0 * m0
    p01 = a0 * m1
    p10 = a1 * m0
    p11 = a1 * m1
    mid = (p00 >> _S32) + (p01 & _LO32) + (p10 & _LO32)  # < 3 * 2^32, no overflow
    lo = (p00 & _LO32) | ((mid & _LO32) << _S32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    return hi, lo


def philox4x64(c0, c1, c2, c3, k0, k1):
    """Philox4x64-10 on arrays of counters (broadcast), returns four uint64 arrays."""
    with np.errstate(over="ignore"):
        c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) for c in (c0, c1, c2, c3))
        c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
        k0 = np.uint64(k0)
        k1 = np.uint64(k1)
        for r in range(_ROUNDS):
            hi0, lo0 = _mulhilo64(c0, _M0)
            hi1, lo1 = _mulhilo64(c2, _M1)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
            if r + 1 < _ROUNDS:
                k0 = k0 + np.uint64(_W0)
                k1 = k1 + np.uint64(_W1)
    return c0, c1, c2, c3


def philox4x64_int(counter, key):
    """Same generator on Python integers for one counter; used to cross-check."""
    mask = (1 << 64) - 1
    c = [int(v) & mask for v in counter]
    k = [int(v) & mask for v in key]
    for r in range(_ROUNDS):
        p0 = _M0 * c[0]
        p1 = _M1 * c[2]
        c = [(p1 >> 64) ^ c[1] ^ k[0], p1 & mask, (p0 >> 64) ^ c[3] ^ k[1], p0 & mask]
        if r + 1 < _ROUNDS:
            k = [(k[0] + _W0) & mask, (k[1] + _W1) & mask]
    return c


def words32(seed, head, purpose, n):
    """First n 32-bit words of stream (seed, head, purpose), as uint64 values."""
    n_calls = (n + 7) // 8
    idx = np.arange(n_calls, dtype=np.uint64)
    w = philox4x64(idx, np.uint64(head), np.uint64(purpose), np.uint64(0),
                   np.uint64(seed), np.uint64(0))
    out = np.empty((n_calls, 8), dtype=np.uint64)
    for j in range(4):
        out[:, 2 * j] = w[j] & _LO32
        out[:, 2 * j + 1] = w[j] >> _S32
    return out.reshape(-1)[:n]


def uniforms(seed, head, purpose, n):
    """u = (x + 0.5) 2^-32 in fp64 (exact), strictly inside (0, 1)."""
    x = words32(seed, head, purpose, n).astype(np.float64)
    return (x + 0.5) * 2.0 ** -32


def gaussians(seed, head, purpose, n):
    """Box-Muller normals: element 2p, 2p+1 from uniforms 2p, 2p+1."""
    n_even = n + (n & 1)
    u = uniforms(seed, head, purpose, n_even).reshape(-1, 2)
    r = np.sqrt(-2.0 * np.log(u[:, 0]))
    t = 2.0 * np.pi * u[:, 1]
    z = np.empty((u.shape[0], 2), dtype=np.float64)
    z[:, 0] = r * np.cos(t)
    z[:, 1] = r * np.sin(t)
    return z.reshape(-1)[:n]
