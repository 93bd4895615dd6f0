"""The method's random parameters, drawn from the seed (oracle side).

TEST INFRASTRUCTURE (CPU oracle); see oracle/__init__.py for who may import it.

Paper: section 3.2 (Eq. 2-3) draws the projection entries i.i.d. Gaussian with
variance 1/sqrt(d) and the phases uniform on [0, 2 pi); Algorithm 2 starts Lanczos
from a random unit vector; Eq. 5 draws the hyperplanes i.i.d. standard normal.
Readings (the paper gives no generator, dtype or layout for them):
  * W is D x m (row k = input coordinate, column j = feature); entry
    W[k, j] = bf16(float32(n_e * std)) with std = 1 / sqrt(sqrt(D)) and
    n_e the e-th normal of the W stream, e = k * m + j.  bf16 rounding is
    round-to-nearest-even from float32 (the feature-map GEMM runs in bf16).
  * psi[j] = float32(2 pi * u_j), u_j the j-th uniform of the psi stream.
  * q1 for window w: the first N_w normals of the q1 stream with window = w,
    scaled to unit length (fp64).
  * R is r x b (row = Ritz coordinate, column = hyperplane), entry
    R[c, l] = n_e with e = c * b + l, kept in fp64.
"""
import math
import numpy as np

from .philox import normals, uniforms, STREAM_W, STREAM_PSI, STREAM_Q1, STREAM_R


def _f32_to_bf16_f64(x32):
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def projection(seed, D, m):
    """W (D x m) as float64 holding bf16 values."""
    std = 1.0 / math.sqrt(math.sqrt(float(D)))
    n = normals(seed, STREAM_W, 0, D * m).reshape(D, m)
    return _f32_to_bf16_f64((n * std).astype(np.float32))


def phases(seed, m):
    """psi (m) as float64 holding float32 values."""
    u = uniforms(seed, STREAM_PSI, 0, m)
    return ((2.0 * math.pi) * u).astype(np.float32).astype(np.float64)


def start_vector(seed, n, window=0):
    """Unit-norm Lanczos start vector q1 (fp64) for one window."""
    g = normals(seed, STREAM_Q1, window, n)
    return g / np.linalg.norm(g)


def hyperplanes(seed, r, b):
    """R (r x b) standard normal hyperplanes, fp64."""
    return normals(seed, STREAM_R, 0, r * b).reshape(r, b)
