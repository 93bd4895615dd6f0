"""Plain fp64 CPU oracle of the Spectral-LSH hot path.

TEST INFRASTRUCTURE (CPU oracle); see oracle/__init__.py for who may import it.

Each function follows one step of the paper (arXiv 2607.19368, "Spectral-LSH:
Sub-Quadratic Prompt Compression via Krylov-Projected Locality-Sensitive
Hashing") in its order and notation.  Notation used here: N tokens, embedding
width D (the paper's d), m random features (the paper's D), n_it Lanczos steps
(the paper's r in Algorithm 2), r kept Ritz vectors (the paper's k), b hash bits.
Library primitives serve as steps (BLAS matmul, LAPACK eigh); there is no
blocking, fusion or reordering beyond what the paper states.

Readings of the paper that this file takes (where it is silent or ambiguous):
  R1 (Eq. 2-3) The random-feature map is sqrt(2/m) cos(x W + psi) times the
     per-token factor s(x) = exp(||x||^2 / (2 sqrt(D))). Without s the map
     estimates the Gaussian kernel exp(-||x-y||^2 / (2 sqrt(D))); with it the
     estimate is unbiased for the unnormalised kernel exp(x.y / sqrt(D)) that
     Eq. 2 names, since that kernel equals s(x) s(y) times the Gaussian one.
     kernel="gauss" gives the map exactly as Eq. 3 prints it.
  R2 The feature map consumes X rounded to bf16; the merge uses X as given.
  R3 (Algorithm 2) "Full re-orthogonalization" is classical Gram-Schmidt applied
     twice against q_1..q_j after the three-term subtraction; alpha_j is taken
     before the subtraction and beta_j after the re-orthogonalization; the
     corrections are not folded into T.
  R4 (Algorithm 2) Breakdown: stop when beta_j <= 1e-10 * max_{i<=j} |alpha_i|.
  R5 (Algorithm 1) Ritz columns are the top-r eigenvectors of T in ascending
     eigenvalue order (the slice V[:, n-r:n]); each eigenvector's sign makes its
     first nonzero component positive; Z is not rescaled.  If Lanczos stopped
     after n_eff < r steps, Z gets r - n_eff leading zero columns (and the
     corresponding Ritz values are reported as 0).
  R6 (Eq. 5) Hash bit l is 1 iff r_l . z_i > 0 (a tie gives 0); the code is
     sum_l bit_l 2^l.
  R7 (Eq. 7, section 3.4, section 3.6) Positions are 0-based token indices; a
     bucket's position is the max of its members' positions; macro-tokens are
     ordered by that position; a bucket whose mean is the zero vector yields the
     zero vector.
  R8 (Eq. 8) The centroid is the normalised sum of the raw rows; zero rows
     contribute 0 to the score.
  R9 (section 3.6) tau(rho) is piecewise linear in log2(rho) through (2, 0.70),
     (8, 0.60), (16, 0.55), 0.70 below 2; rho >= 16 routes every window to the
     spectral path.
  R10 (section 3.5) Chunk size k = max(1, round(rho)) with round-half-to-even;
     the last chunk may be partial; chunks are renormalised like Eq. 7 and take
     the max position of their members.
  R17 (section 3.4 position schemes) Median is the lower median of the member
     positions; mean is their average rounded half to even; macro-tokens are
     ordered by the representative position, ties (possible only for the mean)
     by the group's max position.  Chunk groups use the same scheme.
  R18 (section 5 kill test on bucket purity) Purity counts token pairs i < j of
     one bucket (one window) whose embeddings, as given, have cosine
     similarity strictly above the threshold (0.7); a zero row has cosine 0.
  R19 (section 3.5, section 5.1) A preserved suffix of K tokens is not part of
     any window or bucket: compression runs on the first N - K tokens and the
     K tail tokens follow as singleton macro-tokens at their own positions.
  R20 (section 3.3 adjustment to the target length; no algorithm given, parity
     unpinned) See adjust_to_target: per spectral window, budget
     floor(B / n) (+1 for the first B mod n windows) of B target macro-tokens;
     merges join runs of consecutive macro-tokens, splits cut groups into
     contiguous member runs apportioned by size.
  R16 (section 3.2 remark on row normalisation; appendix, softmax normalisation
     gap) The normalised variant estimates the row sums s = Phi (Phi^T 1) and
     uses diag(s)^-1 Phi Phi^T.  That operator is not symmetric; it is similar to
     S = diag(s)^-1/2 Phi Phi^T diag(s)^-1/2 = Phi~ Phi~^T with Phi~ the rows of
     Phi scaled by s_i^-1/2, so Lanczos runs unchanged on Phi~.  Its Ritz vectors
     Z relate to those of the normalised operator by diag(s)^-1/2 Z, a positive
     row scaling that leaves every SimHash bit unchanged; Z is reported.  A row
     whose estimated sum is not positive gets weight 0 (it leaves the operator).
     Row sums are per window.
"""
import math
from dataclasses import dataclass, field

import numpy as np


# --------------------------------------------------------------------------
# bf16 rounding of the feature-map input (reading R2)
# --------------------------------------------------------------------------
def bf16_round(a):
    """Round to bfloat16 (nearest-even) after rounding to float32; fp64 out."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Step 1: random-feature map (section 3.2, Eq. 2-3; Algorithm 1 first step)
# --------------------------------------------------------------------------
def unnormalised_kernel(X, Y=None):
    """kappa(x, y) = exp(x.y / sqrt(D)) (section 3.2), explicit, for checks."""
    Y = X if Y is None else Y
    D = X.shape[1]
    return np.exp((X @ Y.T) / math.sqrt(D))


def feature_map(X, W, psi, kernel="softmax"):
    """Phi[i, j] = s_i sqrt(2/m) cos(x_i . W[:, j] + psi_j)   (Eq. 3, reading R1).

    X: N x D (any float type; rounded to bf16 first, reading R2).
    W: D x m, psi: m.  Returns N x m fp64.
    """
    Xh = bf16_round(X)
    D = Xh.shape[1]
    m = W.shape[1]
    Phi = math.sqrt(2.0 / m) * np.cos(Xh @ W + psi[None, :])
    if kernel == "softmax":
        s = np.exp(np.sum(Xh * Xh, axis=1) / (2.0 * math.sqrt(D)))
        Phi *= s[:, None]
    elif kernel != "gauss":
        raise ValueError(kernel)
    return Phi


def normalised_features(Phi):
    """Phi~ = diag(w) Phi with w_i = s_i^-1/2, s = Phi (Phi^T 1) (reading R16).

    Returns (Phi~, s).  w_i = 0 where s_i <= 0."""
    s_hat = Phi @ (Phi.T @ np.ones(Phi.shape[0]))
    w = np.zeros_like(s_hat)
    pos = s_hat > 0
    w[pos] = 1.0 / np.sqrt(s_hat[pos])
    return Phi * w[:, None], s_hat


# --------------------------------------------------------------------------
# Step 2: implicit Lanczos (Eq. 4, Algorithm 2)
# --------------------------------------------------------------------------
@dataclass
class LanczosResult:
    alpha: np.ndarray          # n_eff diagonal entries of T
    beta: np.ndarray           # n_eff entries: beta[:n_eff-1] off-diagonal, beta[-1] the residual norm
    Q: np.ndarray              # N x n_eff orthonormal basis
    q_next: np.ndarray         # q_{n_eff+1} (zeros if the run broke down)
    n_eff: int
    broke_down: bool


def implicit_matvec(Phi, v):
    """A v ~ Phi (Phi^T v), never forming the N x N kernel (Eq. 4)."""
    return Phi @ (Phi.T @ v)


def lanczos(Phi, q1, n_it, breakdown_rel=1e-10, matvec=None):
    """Algorithm 2 with full re-orthogonalization (readings R3, R4)."""
    mv = (lambda v: implicit_matvec(Phi, v)) if matvec is None else matvec
    N = q1.shape[0]
    Q = np.zeros((N, n_it + 1))
    alpha = np.zeros(n_it)
    beta = np.zeros(n_it)
    Q[:, 0] = q1 / np.linalg.norm(q1)
    amax = 0.0
    n_eff = n_it
    broke = False
    for j in range(n_it):
        z = mv(Q[:, j])
        alpha[j] = Q[:, j] @ z
        z = z - alpha[j] * Q[:, j]
        if j > 0:
            z = z - beta[j - 1] * Q[:, j - 1]
        for _ in range(2):                       # full re-orthogonalization
            h = Q[:, :j + 1].T @ z
            z = z - Q[:, :j + 1] @ h
        beta[j] = np.linalg.norm(z)
        amax = max(amax, abs(alpha[j]))
        if beta[j] <= breakdown_rel * amax:
            n_eff = j + 1
            broke = True
            break
        Q[:, j + 1] = z / beta[j]
    q_next = np.zeros(N) if broke else Q[:, n_eff].copy()
    return LanczosResult(alpha[:n_eff].copy(), beta[:n_eff].copy(),
                         Q[:, :n_eff].copy(), q_next, n_eff, broke)


def tridiagonal(alpha, beta_off):
    """T = tridiag(beta; alpha; beta) (Algorithm 2, last step)."""
    n = len(alpha)
    T = np.diag(np.asarray(alpha, dtype=np.float64))
    if n > 1:
        T += np.diag(beta_off[:n - 1], 1) + np.diag(beta_off[:n - 1], -1)
    return T


# --------------------------------------------------------------------------
# Step 3: Eigh(T) and Ritz coordinates (Algorithm 1, reading R5)
# --------------------------------------------------------------------------
def eigh_tridiagonal(alpha, beta_off):
    """Eigenpairs of T, ascending, with each vector's first nonzero entry > 0."""
    theta, S = np.linalg.eigh(tridiagonal(alpha, beta_off))
    for c in range(S.shape[1]):
        nz = np.flatnonzero(S[:, c] != 0.0)
        if nz.size and S[nz[0], c] < 0:
            S[:, c] = -S[:, c]
    return theta, S


def ritz(lz, r):
    """Top-r Ritz values (ascending) and coordinates Z = Q S[:, n-r:]."""
    n = lz.n_eff
    theta, S = eigh_tridiagonal(lz.alpha, lz.beta)
    r_eff = min(r, n)
    N = lz.Q.shape[0]
    Z = np.zeros((N, r))
    Z[:, r - r_eff:] = lz.Q @ S[:, n - r_eff:]
    vals = np.zeros(r)
    vals[r - r_eff:] = theta[n - r_eff:]
    return vals, Z, theta, S


def spectral_energy(ritz_values, Phi):
    """Fraction of the operator's spectral energy captured by the kept Ritz
    values: sum(theta) / tr(Phi Phi^T), with tr(Phi Phi^T) = ||Phi||_F^2 (the
    quantity of the section 5 kill test on spectral energy and of the rank
    ablation); 0 for an all-zero Phi."""
    tr = float(np.sum(Phi * Phi))
    return float(np.sum(ritz_values)) / tr if tr > 0 else 0.0


def bucket_purity(X, codes, thresh=0.7, L=None):
    """Bucket purity (section 5 kill test on buckets): over token pairs i < j
    that share a bucket (the same code, within the same window of L tokens when
    L is given), the number whose embeddings have cosine similarity > thresh,
    and the number of such pairs.  cos is taken as 0 when either row is zero
    (reading R18).  Returns (similar_pairs, pairs)."""
    X = np.asarray(X, dtype=np.float64)
    N = len(codes)
    L = L or N
    nrm = np.linalg.norm(X, axis=1)
    sim = tot = 0
    for w in range(N // L):
        groups = {}
        for i in range(w * L, (w + 1) * L):
            groups.setdefault(int(codes[i]), []).append(i)
        for idx in groups.values():
            n = len(idx)
            if n < 2:
                continue
            G = X[idx] @ X[idx].T
            den = np.outer(nrm[idx], nrm[idx])
            C = np.divide(G, den, out=np.zeros_like(G), where=den > 0)
            iu = np.triu_indices(n, 1)
            sim += int(np.count_nonzero(C[iu] > thresh))
            tot += n * (n - 1) // 2
    return sim, tot


# --------------------------------------------------------------------------
# Step 4: SimHash in the spectral subspace (Eq. 5, reading R6)
# --------------------------------------------------------------------------
def projections(Z, R):
    return Z @ R


def simhash(Z, R):
    """codes[i] = sum_l [r_l . z_i > 0] 2^l  (Eq. 5)."""
    P = projections(Z, R)
    bits = (P > 0.0).astype(np.int64)
    return (bits << np.arange(R.shape[1], dtype=np.int64)[None, :]).sum(axis=1)


# --------------------------------------------------------------------------
# Step 5: macro-tokens (Eq. 7, section 3.4 max positions, section 3.6 order)
# --------------------------------------------------------------------------
@dataclass
class MergeResult:
    E: np.ndarray              # M x D macro-token embeddings (fp64)
    P: np.ndarray              # M positions (int64), ascending
    tok2macro: np.ndarray      # N macro index per token
    members: list = field(default_factory=list)   # member token indices per macro (ascending)
    codes_of_macro: np.ndarray = None


def renormalised_mean(rows):
    """Eq. 7: mean of the rows rescaled to the mean row norm (zero stays zero)."""
    rows = np.asarray(rows, dtype=np.float64)
    mean = rows.mean(axis=0)
    eta = np.linalg.norm(rows, axis=1).mean()
    nrm = np.linalg.norm(mean)
    if nrm == 0.0:
        return np.zeros_like(mean)
    return mean * (eta / nrm)


def group_position(p, scheme="max"):
    """Representative position of a group with member positions p (section 3.4):
    max (default), lower median, or mean rounded half to even (reading R17)."""
    p = sorted(int(v) for v in p)
    if scheme == "max":
        return p[-1]
    if scheme == "median":
        return p[(len(p) - 1) // 2]
    if scheme == "mean":
        q, rem = divmod(sum(p), len(p))
        if 2 * rem > len(p) or (2 * rem == len(p) and q % 2 == 1):
            q += 1
        return q
    raise ValueError(scheme)


def merge(X, codes, positions=None, compact=False, scheme="max"):
    """Group tokens by code; one renormalised mean per group; the group's
    representative position (max by default); groups ordered by that position,
    ties (possible for the mean) by the max position (readings R7, R17)."""
    X = np.asarray(X)
    N = len(codes)
    pos = np.arange(N, dtype=np.int64) if positions is None else np.asarray(positions, np.int64)
    groups = {}
    for i in range(N):
        groups.setdefault(int(codes[i]), []).append(i)
    entries = sorted(((group_position(pos[idx], scheme), max(pos[idx]), c, idx)
                      for c, idx in groups.items()), key=lambda e: (e[0], e[1]))
    entries = [(p, c, idx) for p, _, c, idx in entries]
    M = len(entries)
    E = np.zeros((M, X.shape[1]))
    P = np.zeros(M, dtype=np.int64)
    t2m = np.zeros(N, dtype=np.int64)
    members = []
    cm = np.zeros(M, dtype=np.int64)
    for k, (p, c, idx) in enumerate(entries):
        E[k] = renormalised_mean(X[idx].astype(np.float64))
        P[k] = p
        t2m[idx] = k
        members.append(np.asarray(idx, dtype=np.int64))
        cm[k] = c
    if compact:
        P = np.arange(M, dtype=np.int64)
    return MergeResult(E, P, t2m, members, cm)


# --------------------------------------------------------------------------
# Adaptive backend pieces (section 3.5 chunk, section 3.6 Eq. 8 and routing)
# --------------------------------------------------------------------------
def redundancy_score(Xw):
    """Eq. 8: mean cosine of each row to the normalised centroid (reading R8)."""
    Xw = np.asarray(Xw, dtype=np.float64)
    S = Xw.sum(axis=0)
    sn = np.linalg.norm(S)
    if sn == 0.0:
        return 0.0
    xbar = S / sn
    norms = np.linalg.norm(Xw, axis=1)
    dots = Xw @ xbar
    cos = np.where(norms > 0, dots / np.where(norms > 0, norms, 1.0), 0.0)
    return float(cos.mean())


def tau_of_rho(rho):
    """Routing threshold schedule (section 3.6, reading R9)."""
    if rho <= 2.0:
        return 0.70
    if rho <= 8.0:
        return 0.70 + (0.60 - 0.70) * (math.log2(rho) - 1.0) / 2.0
    if rho < 16.0:
        return 0.60 + (0.55 - 0.60) * (math.log2(rho) - 3.0)
    return 0.55


def route_window(L, score, rho, tau=None):
    """True = spectral path, False = chunk (section 3.6)."""
    if rho >= 16.0:
        return True
    if L <= 4:
        return False
    t = tau_of_rho(rho) if tau is None else tau
    return score >= t


def adjust_to_target(groups, T):
    """Exact target length (section 3.3: an adjustment step merges or splits
    clusters until their number matches the target; the paper gives no
    algorithm, reading R20, parity unpinned).  groups: member index arrays
    (ascending) in macro order (ascending position).  Returns T groups in the
    same form.

    Merge (more groups than T): group k joins new group floor(k T / M), so runs
    of consecutive groups in position order are merged into T near-equal runs.
    Split (fewer): E = T - M extra pieces are apportioned to the groups in
    proportion to s_k - 1 (the cuts a group of s_k members admits): floor of the
    quota, then one more for the E - sum largest remainders (ties: earlier
    group); a group of s members in n pieces is cut, in member order, into
    pieces of ceil(s/n) (the first s mod n) and floor(s/n) members; pieces are
    ordered by their last member."""
    M = len(groups)
    if T < 1 or T > sum(len(g) for g in groups):
        raise ValueError("target out of range")
    if M == T:
        return [np.asarray(g) for g in groups]
    if M > T:
        out = [[] for _ in range(T)]
        for k, g in enumerate(groups):
            out[k * T // M].extend(int(v) for v in g)
        return [np.array(sorted(g), dtype=np.int64) for g in out]
    sizes = [len(g) for g in groups]
    E, den = T - M, sum(sizes) - M
    extra = [E * (s - 1) // den for s in sizes]
    rem = [E * (s - 1) % den for s in sizes]
    R = E - sum(extra)
    order = sorted(range(M), key=lambda k: (-rem[k], k))
    for k in order[:R]:
        extra[k] += 1
    pieces = []
    for g, e in zip(groups, extra):
        g = np.asarray(g, dtype=np.int64)
        n, s_ = e + 1, len(g)
        q, rr = divmod(s_, n)
        cut = 0
        for j in range(n):
            sz = q + 1 if j < rr else q
            pieces.append(g[cut:cut + sz])
            cut += sz
    pieces.sort(key=lambda p: int(p[-1]))
    return pieces


def target_budgets(T, spectral, L, k, keep_last=0):
    """Per-window output budgets for an exact total length T over windows of L
    tokens (section 3.3 adjustment to the target; the appendix's per-window
    exact budgets for the adaptive backend; reading R20, parity unpinned).

    spectral: one flag per window (True = spectral path, False = chunk
    pooling).  A chunk window yields ceil(L / k) macro-tokens of its own and the
    keep_last preserved tokens one each; the spectral windows share the rest,
    B = T - (chunk macro-tokens) - keep_last, as floor(B / n) each plus one for
    the first B mod n spectral windows in window order.  Chunk windows get 0.
    Raises ValueError when some spectral budget would leave [1, L], or when
    there is no spectral window and B != 0."""
    flags = [bool(f) for f in spectral]
    n = sum(flags)
    chunk = sum(-(-L // k) for f in flags if not f)
    B = T - chunk - keep_last
    if n == 0:
        if B != 0:
            raise ValueError("target unreachable without spectral windows")
        return [0] * len(flags)
    if B < n or B > n * L:
        raise ValueError("target unreachable with this routing")
    q, rem = divmod(B, n)
    out, a = [], 0
    for f in flags:
        if f:
            out.append(q + (1 if a < rem else 0))
            a += 1
        else:
            out.append(0)
    return out


def merge_groups(X, groups, positions=None, compact=False):
    """Eq. 7 and max positions for given member groups (in macro order)."""
    X = np.asarray(X)
    N = X.shape[0]
    pos = np.arange(N, dtype=np.int64) if positions is None else np.asarray(positions, np.int64)
    M = len(groups)
    E = np.zeros((M, X.shape[1]))
    P = np.zeros(M, dtype=np.int64)
    t2m = np.full(N, -1, dtype=np.int64)
    for k, g in enumerate(groups):
        E[k] = renormalised_mean(X[g].astype(np.float64))
        P[k] = int(pos[g].max())
        t2m[g] = k
    if compact:
        P = np.arange(M, dtype=np.int64)
    return E, P, t2m


def preserve_suffix(E, P, tok2macro, X_tail, pos0, compact=False):
    """Section 3.5 (every backend can keep a fixed number of final tokens as
    they are; section 5.1: the last 12 by default): each of the K tail rows
    becomes a macro-token of its own (Eq. 7 on a single row gives the row) at its
    own position pos0 + t, after the macro-tokens of the compressed tokens, whose
    positions are all smaller (reading R19).  Returns (E, P, tok2macro) of the
    whole prompt."""
    X_tail = np.asarray(X_tail, dtype=np.float64)
    K = X_tail.shape[0]
    M = len(P)
    E2 = np.concatenate([E, np.stack([renormalised_mean(X_tail[t:t + 1]) for t in range(K)])
                         if K else np.zeros((0, E.shape[1]))])
    P_tail = np.arange(M, M + K) if compact else pos0 + np.arange(K)
    P2 = np.concatenate([np.asarray(P, np.int64), P_tail.astype(np.int64)])
    t2m = np.concatenate([np.asarray(tok2macro, np.int64), np.arange(M, M + K, dtype=np.int64)])
    return E2, P2, t2m


def chunk_size(rho):
    return max(1, int(round(rho)))          # Python round: half to even (reading R10)


def chunk_pool(Xw, k, pos0=0, scheme="max"):
    """Section 3.5: consecutive groups of k rows, renormalised mean, the group's
    representative position (max by default, reading R17)."""
    L = Xw.shape[0]
    starts = list(range(0, L, k))
    E = np.stack([renormalised_mean(Xw[s:min(s + k, L)]) for s in starts])
    P = np.array([group_position(range(pos0 + s, pos0 + min(s + k, L)), scheme) for s in starts],
                 dtype=np.int64)
    return E, P


# --------------------------------------------------------------------------
# End to end (Algorithm 1)
# --------------------------------------------------------------------------
@dataclass
class CompressResult:
    Phi: np.ndarray
    lz: LanczosResult
    ritz_values: np.ndarray
    Z: np.ndarray
    proj: np.ndarray
    codes: np.ndarray
    merge: MergeResult


def compress(X, W, psi, q1, R, n_it, r, kernel="softmax", positions=None, keep_phi=True,
             normalise=False, scheme="max"):
    """One global Spectral-LSH pass over X (Algorithm 1); normalise=True runs
    it on the normalised operator (reading R16)."""
    Phi = feature_map(X, W, psi, kernel)
    if normalise:
        Phi, _ = normalised_features(Phi)
    lz = lanczos(Phi, q1, n_it)
    vals, Z, _, _ = ritz(lz, r)
    proj = projections(Z, R)
    codes = simhash(Z, R)
    mg = merge(X, codes, positions, scheme=scheme)
    return CompressResult(Phi if keep_phi else None, lz, vals, Z, proj, codes, mg)
