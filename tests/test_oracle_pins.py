"""Pins for the CPU oracle: each check ties an oracle function to something
other than itself (published vectors, hand-worked examples, closed forms,
dense linear algebra, Monte-Carlo laws, invariants)."""
import math
import os

import numpy as np
import pytest

from oracle import params as OP
from oracle import philox as PH
from oracle import spectral_lsh as O
from workloads import make_inputs

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rows(path, tag):
    out = []
    with open(os.path.join(GOLD, path)) as f:
        for line in f:
            if line.startswith(tag + " "):
                out.append([float(v) for v in line.split()[1:]])
    return np.array(out)


# ---------------------------------------------------------------- Philox
def test_philox_known_answers():
    with open(os.path.join(GOLD, "philox4x32_10_kat.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    assert len(rows) == 3
    for row in rows:
        v = [int(x, 16) for x in row]
        out = PH.philox4x32_10(*[np.array([x], np.uint64) for x in v[:4]], v[4], v[5])
        assert [int(o[0]) for o in out] == v[6:10]


def test_philox_streams_are_distinct_and_uniform():
    a = PH.uniforms(0, PH.STREAM_W, 0, 20000)
    b = PH.uniforms(0, PH.STREAM_PSI, 0, 20000)
    c = PH.uniforms(1, PH.STREAM_W, 0, 20000)
    assert a.min() >= 0.0 and a.max() < 1.0
    assert abs(a.mean() - 0.5) < 0.01 and abs(a.var() - 1 / 12) < 0.005
    assert not np.array_equal(a, b) and not np.array_equal(a, c)
    n = PH.normals(0, PH.STREAM_R, 0, 40001)
    assert abs(n.mean()) < 0.02 and abs(n.std() - 1.0) < 0.02
    # odd count is a prefix of the even count (block n -> elements 2n, 2n+1)
    assert np.array_equal(PH.normals(0, PH.STREAM_R, 0, 7), PH.normals(0, PH.STREAM_R, 0, 8)[:7])


def test_params_shapes_and_distributions():
    D, m = 64, 4096
    W = OP.projection(3, D, m)
    assert W.shape == (D, m)
    # bf16 values: low 16 bits of the float32 pattern are zero
    assert np.all(W.astype(np.float32).view(np.uint32) & 0xFFFF == 0)
    # variance 1/sqrt(D) (section 3.2)
    assert abs(W.var() / (1 / math.sqrt(D)) - 1.0) < 0.02
    psi = OP.phases(3, m)
    assert psi.min() >= 0 and psi.max() < 2 * math.pi + 1e-6
    # Uniform(0, 2 pi): mean pi, variance (2 pi)^2 / 12
    assert abs(psi.mean() / math.pi - 1.0) < 0.03
    assert abs(psi.var() / (math.pi ** 2 / 3) - 1.0) < 0.05
    q = OP.start_vector(3, 1000, window=5)
    assert abs(np.linalg.norm(q) - 1.0) < 1e-14
    assert not np.allclose(q, OP.start_vector(3, 1000, window=6))


# ---------------------------------------------------------------- feature map
def _small_points(n=48, D=16, seed=7):
    X, _ = make_inputs("tiny").X[:n, :D], None
    X = O.bf16_round(X * 0.8)        # bf16-representable, norms about 0.9
    return X


def _kernel_rms(X, m, seed, kernel="softmax"):
    W = OP.projection(seed, X.shape[1], m)
    psi = OP.phases(seed, m)
    Phi = O.feature_map(X, W, psi, kernel)
    if kernel == "softmax":
        K = O.unnormalised_kernel(X)
    else:
        sq = np.sum(X * X, 1)
        K = np.exp(-(sq[:, None] + sq[None, :] - 2 * X @ X.T) / (2 * math.sqrt(X.shape[1])))
    return np.sqrt(np.mean((Phi @ Phi.T - K) ** 2))


@pytest.mark.parametrize("kernel", ["softmax", "gauss"])
def test_feature_map_converges_to_kernel(kernel):
    """Bochner (Eq. 2): Phi Phi^T -> kernel with Monte-Carlo error ~ m^-1/2."""
    X = _small_points()
    ms = [256, 1024, 4096, 16384]
    err = [np.mean([_kernel_rms(X, m, s, kernel) for s in range(3)]) for m in ms]
    slope = np.polyfit(np.log(ms), np.log(err), 1)[0]
    assert -0.62 < slope < -0.38, (err, slope)
    assert err[-1] < 0.02


def test_feature_map_diagonal_limit():
    """phi(x).phi(x) -> kappa(x, x) = exp(||x||^2 / sqrt(D))."""
    X = _small_points()
    m = 65536
    Phi = O.feature_map(X, OP.projection(11, X.shape[1], m), OP.phases(11, m))
    diag = np.sum(Phi * Phi, 1)
    want = np.exp(np.sum(X * X, 1) / math.sqrt(X.shape[1]))
    assert np.max(np.abs(diag / want - 1)) < 0.03


def test_feature_map_gauss_is_softmax_without_prefactor():
    X = _small_points()
    W, psi = OP.projection(2, X.shape[1], 64), OP.phases(2, 64)
    a = O.feature_map(X, W, psi, "softmax")
    g = O.feature_map(X, W, psi, "gauss")
    s = a[:, 0] / g[:, 0]
    assert np.allclose(a, g * s[:, None], rtol=1e-13, atol=0)
    assert np.all(s >= 1.0)


# ---------------------------------------------------------------- Lanczos + Ritz
@pytest.fixture(scope="module")
def tiny_run():
    inp = make_inputs("tiny")
    wl = inp.workload
    X = inp.x_float()
    W, psi = OP.projection(0, wl.D, wl.m), OP.phases(0, wl.m)
    Phi = O.feature_map(X, W, psi)
    lz = O.lanczos(Phi, OP.start_vector(0, wl.N), wl.n_it)
    return wl, X, Phi, lz


def test_lanczos_orthonormal_and_relation(tiny_run):
    wl, X, Phi, lz = tiny_run
    Q = lz.Q
    assert np.max(np.abs(Q.T @ Q - np.eye(lz.n_eff))) < 1e-12
    T = O.tridiagonal(lz.alpha, lz.beta)
    AQ = Phi @ (Phi.T @ Q)
    res = AQ - Q @ T
    res[:, -1] -= lz.beta[-1] * lz.q_next
    normA = np.linalg.norm(Phi, 2) ** 2
    assert np.max(np.abs(res)) < 1e-11 * normA


def test_lanczos_matches_dense_eigendecomposition(tiny_run):
    """Converged Ritz pairs equal eigenpairs of the explicit Phi Phi^T."""
    wl, X, Phi, lz = tiny_run
    A = Phi @ Phi.T
    lam, V = np.linalg.eigh(A)
    lam, V = lam[::-1], V[:, ::-1]
    vals, Z, theta, S = O.ritz(lz, wl.r)
    n = lz.n_eff
    resid = np.abs(lz.beta[-1] * S[-1, :])          # ||A y - theta y|| for each Ritz pair
    top = theta[::-1]
    conv = 0
    for c in range(wl.r):
        col = n - 1 - c
        if resid[col] < 1e-7 * top[0]:
            conv += 1
            assert abs(top[c] - lam[c]) <= 1e-8 * lam[0]
            y = Z[:, wl.r - 1 - c]
            assert abs(abs(y @ V[:, c]) - 1.0) < 1e-6
    assert conv >= 3
    # interlacing / Kaniel-Paige-Saad upper side: theta_c <= lambda_c
    assert np.all(top[:wl.r] <= lam[:wl.r] + 1e-9 * lam[0])


def test_lanczos_exact_spectrum_and_breakdown():
    """Low-rank operator with known eigenvalues: the Krylov space is exhausted
    after rank+1 steps, Lanczos breaks down, and the Ritz values are exact."""
    rng = np.random.default_rng(5)
    N, m, rank = 300, 40, 12
    U, _ = np.linalg.qr(rng.standard_normal((N, rank)))
    Vt, _ = np.linalg.qr(rng.standard_normal((m, rank)))
    sig = np.linspace(1.0, 6.0, rank)
    Phi = U @ np.diag(sig) @ Vt.T
    lz = O.lanczos(Phi, rng.standard_normal(N), 30)
    assert lz.broke_down and lz.n_eff == rank + 1
    vals, Z, theta, S = O.ritz(lz, rank)
    assert np.allclose(np.sort(theta)[1:], np.sort(sig ** 2), rtol=0, atol=1e-10)
    assert abs(np.sort(theta)[0]) < 1e-10
    assert np.allclose(vals, np.sort(sig ** 2), atol=1e-10)


def test_lanczos_identical_rows_rank_one():
    """Identical rows: Phi Phi^T has rank one, breakdown after two steps, and
    the unused leading Ritz columns are zero."""
    X = np.tile(make_inputs("tiny").X[:1], (64, 1)).astype(np.float64)
    W, psi = OP.projection(0, X.shape[1], 32), OP.phases(0, 32)
    Phi = O.feature_map(X, W, psi)
    lz = O.lanczos(Phi, OP.start_vector(0, 64), 10)
    assert lz.broke_down and lz.n_eff == 2
    vals, Z, theta, S = O.ritz(lz, 4)
    assert np.all(Z[:, :2] == 0) and np.all(vals[:2] == 0)
    assert abs(vals[-1] - np.sum(Phi[0] ** 2) * 64) < 1e-9 * vals[-1]


# ---------------------------------------------------------------- spectral energy
def test_spectral_energy_exact_and_bounded(tiny_run):
    """sum(theta)/||Phi||_F^2: 1 when the Krylov space holds the whole spectrum
    (sum of all eigenvalues = trace = squared Frobenius norm); within (0, 1] and
    non-decreasing in r otherwise (Ritz values of a PSD operator are >= 0 and,
    by interlacing, the top r of them sum to at most the top r eigenvalues)."""
    rng = np.random.default_rng(7)
    N, m, rank = 200, 30, 9
    Phi = rng.standard_normal((N, rank)) @ rng.standard_normal((rank, m))
    lz = O.lanczos(Phi, rng.standard_normal(N), 20)
    vals, _, _, _ = O.ritz(lz, rank)
    assert abs(O.spectral_energy(vals, Phi) - 1.0) < 1e-12
    wl, X, Phi, lz = tiny_run
    lam = np.linalg.eigvalsh(Phi @ Phi.T)[::-1]
    prev = 0.0
    for r in (1, 2, 4, 8):
        vals, _, _, _ = O.ritz(lz, r)
        e = O.spectral_energy(vals, Phi)
        assert prev <= e <= lam[:r].sum() / lam.sum() + 1e-12 and e <= 1.0
        prev = e
    assert O.spectral_energy(np.ones(3), np.zeros((4, 5))) == 0.0


# ---------------------------------------------------------------- normalised operator
def test_normalised_operator_closed_forms(tiny_run):
    """Reading R16: the normalised matvec diag(s)^-1 Phi Phi^T with s = Phi Phi^T 1
    maps 1 to 1 (rows sum to one), so S = Phi~ Phi~^T has sqrt(s) as an exact
    eigenvector with eigenvalue 1; S and the non-symmetric normalised matrix
    share their spectrum; the right eigenvectors of the latter are
    diag(s)^-1/2 times those of S."""
    wl, X, Phi, lz = tiny_run
    Pn, s_hat = O.normalised_features(Phi)
    A = Phi @ Phi.T
    assert np.allclose(s_hat, A.sum(axis=1), rtol=1e-12, atol=0)
    assert np.all(s_hat > 0)
    P = A / s_hat[:, None]                        # the paper's normalised matrix
    assert np.allclose(P.sum(axis=1), 1.0, rtol=0, atol=1e-12)
    u = np.sqrt(s_hat)
    assert np.allclose(Pn @ (Pn.T @ u), u, rtol=0, atol=1e-11 * np.abs(u).max())
    S = Pn @ Pn.T
    ev_S = np.sort(np.linalg.eigvalsh(S))
    ev_P = np.sort(np.linalg.eigvals(P).real)
    assert np.allclose(ev_S[-40:], ev_P[-40:], rtol=0, atol=1e-10)
    # Lanczos on Phi~ (the unchanged algorithm): converged Ritz pairs of S give
    # right eigenvectors diag(s)^-1/2 z of P
    lzn = O.lanczos(Pn, OP.start_vector(0, wl.N), wl.n_it)
    vals, Z, theta, Sv = O.ritz(lzn, wl.r)
    resid = np.abs(lzn.beta[-1] * Sv[-1, :])
    checked = 0
    for c in range(wl.r):
        k = lzn.n_eff - wl.r + c
        if resid[k] < 1e-9 * theta[-1]:
            v = Z[:, c] / np.sqrt(s_hat)
            assert np.allclose(P @ v, vals[c] * v, rtol=0, atol=1e-7 * np.abs(v).max())
            checked += 1
    assert checked >= 3
    assert abs(vals[-1] - 1.0) < 1e-9           # the top of the spectrum is 1 here
    # SimHash of the right eigenvectors equals SimHash of Z (positive row scaling)
    R = OP.hyperplanes(0, wl.r, wl.bits)
    assert np.array_equal(O.simhash(Z, R), O.simhash(Z / np.sqrt(s_hat)[:, None], R))


def test_normalised_operator_nonpositive_row_sum():
    """Reading R16: a row whose estimated sum is not positive leaves the operator."""
    Phi = np.array([[1.0, 0.0, 0.5], [-1.0, 0.2, 0.0], [0.0, 0.3, -0.5]])
    Pn, s_hat = O.normalised_features(Phi)
    c = Phi.sum(axis=0)                            # Phi^T 1 = [0, 0.5, 0]
    assert np.allclose(s_hat, Phi @ c)             # [0, 0.1, 0.15]
    assert s_hat[0] == 0.0 and np.all(Pn[0] == 0.0)
    assert np.allclose(Pn[1:], Phi[1:] / np.sqrt(s_hat[1:, None]))


def test_tridiagonal_eigensolve_toeplitz_closed_form():
    """tridiag(b; a; b) of order n: eigenvalues a + 2b cos(k pi/(n+1)),
    eigenvectors sin(j k pi/(n+1)) (first entry positive)."""
    n, a, b = 17, 2.5, -0.75
    theta, S = O.eigh_tridiagonal(np.full(n, a), np.full(n, b))
    k = np.arange(1, n + 1)
    want = np.sort(a + 2 * b * np.cos(k * np.pi / (n + 1)))
    assert np.allclose(theta, want, atol=1e-13)
    j = np.arange(1, n + 1)
    for c in range(n):
        # eigenvalue theta[c] = a + 2b cos(kk pi/(n+1)) for the matching kk
        kk = k[np.argmin(np.abs(a + 2 * b * np.cos(k * np.pi / (n + 1)) - theta[c]))]
        v = np.sin(j * kk * np.pi / (n + 1))
        v /= np.linalg.norm(v)
        v *= np.sign(v[0])
        assert S[0, c] > 0
        assert np.allclose(S[:, c], v, atol=1e-12)


# ---------------------------------------------------------------- SimHash
def test_simhash_hand_example():
    Z = _rows("simhash_hand.txt", "Z")
    R = _rows("simhash_hand.txt", "R")
    codes = _rows("simhash_hand.txt", "CODES")[0].astype(int)
    assert list(O.simhash(Z, R)) == list(codes)


def test_simhash_scale_invariance_and_code_range():
    rng = np.random.default_rng(1)
    Z = rng.standard_normal((500, 8))
    R = rng.standard_normal((8, 6))
    c = O.simhash(Z, R)
    s = rng.uniform(0.01, 100, size=(500, 1))
    assert np.array_equal(c, O.simhash(Z * s, R))
    assert c.min() >= 0 and c.max() < 2 ** 6
    # negating a row flips every (non-tied) bit
    assert np.array_equal(O.simhash(-Z, R), (2 ** 6 - 1) - c)


def test_simhash_collision_law():
    """Eq. 6: P[h_i = h_j] = (1 - angle/pi)^b, by Monte Carlo over hyperplanes."""
    rng = np.random.default_rng(2)
    k, b, trials = 6, 4, 20000
    for ang in (0.3, 0.9, 1.6):
        zi = np.zeros(k); zi[0] = 1.0
        zj = np.zeros(k); zj[0] = math.cos(ang); zj[1] = math.sin(ang)
        Z = np.stack([zi, zj])
        same = 0
        for _ in range(trials // 500):
            R = rng.standard_normal((500, k, b))
            P = np.einsum("nk,tkb->tnb", Z, R) > 0
            codes = (P.astype(np.int64) << np.arange(b)).sum(-1)
            same += int(np.sum(codes[:, 0] == codes[:, 1]))
        p = (1 - ang / math.pi) ** b
        sd = math.sqrt(p * (1 - p) / trials)
        assert abs(same / trials - p) < 4.5 * sd, (ang, same / trials, p)
        # and the oracle's own simhash agrees with the vectorised bits here
        R = rng.standard_normal((k, b))
        assert O.simhash(Z, R)[0] == int(((Z[0] @ R) > 0) @ (1 << np.arange(b)))


# ---------------------------------------------------------------- bf16 rounding
def _bf16_cases():
    rows = []
    with open(os.path.join(GOLD, "bf16_round_hand.txt")) as f:
        for line in f:
            if line.startswith("F32 "):
                t = line.split()
                rows.append((int(t[1], 16), int(t[3], 16)))
    return rows


@pytest.mark.parametrize("fn", ["bf16_round", "projection_rounding"])
def test_bf16_round_hand_ties_and_library_cast(fn):
    """Reading R2: round-to-nearest-even from float32.  Pinned by hand-worked
    ties (tests/golden/bf16_round_hand.txt) and by torch's float32 -> bfloat16
    conversion (round to nearest even) on random bit patterns of every finite
    magnitude; both rounding routines of the oracle are checked (the feature
    map's input rounding and the W draw's)."""
    import torch
    rnd = O.bf16_round if fn == "bf16_round" else OP._f32_to_bf16_f64
    cases = _bf16_cases()
    assert len(cases) >= 10
    x = np.array([c[0] for c in cases], np.uint32).view(np.float32)
    want = (np.array([c[1] for c in cases], np.uint32) << 16).view(np.float32).astype(np.float64)
    got = rnd(x)
    assert np.array_equal(got, want), [hex(int(v)) for v in np.asarray(got, np.float32).view(np.uint32)]
    rng = np.random.default_rng(17)
    bits = rng.integers(0, 2**32, 200000, dtype=np.uint64).astype(np.uint32)
    bits = bits[(bits & 0x7F800000) != 0x7F800000]           # finite only
    ties = (rng.integers(0, 2**16, 5000, dtype=np.uint64).astype(np.uint32) << 16) | 0x8000
    vals = np.concatenate([bits, ties & 0xFF7FFFFF]).view(np.float32)
    ref = torch.from_numpy(vals.copy()).to(torch.bfloat16).to(torch.float64).numpy()
    out = rnd(vals)
    fin = np.isfinite(ref)
    assert np.array_equal(out[fin], ref[fin])
    assert np.all(np.isinf(out[~fin]) & (np.sign(out[~fin]) == np.sign(ref[~fin])))


# ---------------------------------------------------------------- merge
def test_merge_hand_example():
    X = _rows("merge_hand.txt", "X")
    codes = _rows("merge_hand.txt", "CODES")[0].astype(int)
    mg = O.merge(X, codes)
    assert list(mg.P) == list(_rows("merge_hand.txt", "P")[0].astype(int))
    assert list(mg.tok2macro) == list(_rows("merge_hand.txt", "MAP")[0].astype(int))
    assert np.allclose(mg.E, _rows("merge_hand.txt", "E"), rtol=0, atol=1e-15)
    # a bucket whose mean is zero yields the zero vector
    z = O.merge(np.array([[1.0, 0.0], [-1.0, 0.0]]), np.array([4, 4]))
    assert np.all(z.E == 0) and list(z.P) == [1]


def test_merge_groups_hand_example_and_agreement_with_merge():
    """merge_groups (Eq. 7 on given member groups, max positions): the hand
    example of tests/golden/merge_hand.txt given as groups in macro order, at
    positions offset by 10 (each position is the group's largest member
    position, not its smallest), and on random codes the same E, P and token
    map as merge() when handed merge()'s own groups."""
    X = _rows("merge_hand.txt", "X")
    groups = [np.array([0, 2]), np.array([3]), np.array([1, 4])]
    E, P, t2m = O.merge_groups(X, groups)
    assert list(P) == list(_rows("merge_hand.txt", "P")[0].astype(int))
    assert list(t2m) == list(_rows("merge_hand.txt", "MAP")[0].astype(int))
    assert np.allclose(E, _rows("merge_hand.txt", "E"), rtol=0, atol=1e-15)
    _, P10, _ = O.merge_groups(X, groups, positions=10 + np.arange(5))
    assert list(P10) == [12, 13, 14]
    _, Pc, _ = O.merge_groups(X, groups, compact=True)
    assert list(Pc) == [0, 1, 2]
    rng = np.random.default_rng(23)
    for trial in range(5):
        N = int(rng.integers(30, 300))
        Xr = rng.standard_normal((N, 6))
        codes = rng.integers(0, int(rng.integers(2, 50)), N)
        pos = 100 * trial + np.arange(N)
        mg = O.merge(Xr, codes, positions=pos)
        E2, P2, t2 = O.merge_groups(Xr, mg.members, positions=pos)
        assert np.array_equal(E2, mg.E) and np.array_equal(P2, mg.P)
        assert np.array_equal(t2, mg.tok2macro)


def test_target_budgets_hand_and_invariants():
    """Reading R20 (parity unpinned: the paper states per-window exact budgets
    but no rule).  Hand example: 5 windows of 256, windows 1 and 4 routed to
    chunk pooling with k = 8 (32 macro-tokens each), 12 preserved tokens,
    T = 140: B = 140 - 64 - 12 = 64 over 3 spectral windows = 21 each and one
    more for the first (64 mod 3 = 1).  Then the exact-fit and unreachable
    cases, and invariants on random routings."""
    assert O.target_budgets(140, [1, 0, 1, 1, 0], 256, 8, 12) == [22, 0, 21, 21, 0]
    assert O.target_budgets(512, [1], 8192, 1) == [512]
    assert O.target_budgets(3, [1, 1, 1], 16, 4) == [1, 1, 1]
    assert O.target_budgets(64, [0, 0], 256, 8) == [0, 0]
    # a chunk window of 10 tokens with k = 4 yields ceil(10 / 4) = 3
    assert O.target_budgets(3 + 5, [0, 1], 10, 4) == [0, 5]
    for T, sp in ((2, [1, 1, 1]), (49, [1, 1, 1]), (63, [0, 0])):
        with pytest.raises(ValueError):
            O.target_budgets(T, sp, 16, 8)
    rng = np.random.default_rng(29)
    for trial in range(50):
        nw = int(rng.integers(1, 20))
        L = int(rng.choice([16, 64, 256]))
        k = int(rng.integers(1, 9))
        K = int(rng.integers(0, 13))
        sp = rng.random(nw) < 0.6
        n = int(sp.sum())
        chunk = int((~sp).sum()) * (-(-L // k))
        if n == 0:
            continue
        T = chunk + K + int(rng.integers(n, n * L + 1))
        b = O.target_budgets(T, sp, L, k, K)
        assert sum(b) == T - chunk - K
        sb = [v for v, f in zip(b, sp) if f]
        assert all(1 <= v <= L for v in sb) and max(sb) - min(sb) <= 1
        assert sb == sorted(sb, reverse=True)
        assert all(v == 0 for v, f in zip(b, sp) if not f)


def test_position_schemes_hand_example():
    """Section 3.4 position schemes worked by hand (tests/golden/positions_hand.txt)."""
    f = "positions_hand.txt"
    X = np.arange(16, dtype=np.float64).reshape(8, 2) + 1.0
    codes = _rows(f, "CODES")[0].astype(int)
    for scheme, tag in (("max", "MAX"), ("median", "MEDIAN"), ("mean", "MEAN")):
        mg = O.merge(X, codes, scheme=scheme)
        assert list(mg.P) == list(_rows(f, tag + "_P")[0].astype(int)), scheme
        assert list(mg.tok2macro) == list(_rows(f, tag + "_MAP")[0].astype(int)), scheme
    tie = O.merge(X[:4], _rows(f, "TIE_CODES")[0].astype(int), scheme="mean")
    assert list(tie.P) == list(_rows(f, "TIE_P")[0].astype(int))
    assert list(tie.tok2macro) == list(_rows(f, "TIE_MAP")[0].astype(int))
    for scheme, tag in (("max", "CHUNK_MAX"), ("median", "CHUNK_MEDIAN"), ("mean", "CHUNK_MEAN")):
        _, P = O.chunk_pool(X, 3, scheme=scheme)
        assert list(P) == list(_rows(f, tag)[0].astype(int)), scheme


def test_position_schemes_invariants():
    """Every scheme keeps the same groups and embeddings; median positions are
    member positions; mean positions lie within [min, max]; max positions are
    causal; positions are non-decreasing along the macro order."""
    rng = np.random.default_rng(11)
    N = 500
    X = rng.standard_normal((N, 4))
    codes = rng.integers(0, 40, N)
    pos = 1000 + np.arange(N)
    ref = O.merge(X, codes, positions=pos)
    for scheme in ("max", "median", "mean"):
        mg = O.merge(X, codes, positions=pos, scheme=scheme)
        assert np.all(np.diff(mg.P) >= 0)
        assert sorted(map(tuple, mg.members)) == sorted(map(tuple, ref.members))
        for k, idx in enumerate(mg.members):
            p = pos[idx]
            if scheme == "median":
                assert mg.P[k] in p
            assert p.min() <= mg.P[k] <= p.max()
            kr = ref.tok2macro[idx[0]]
            assert np.array_equal(mg.E[k], ref.E[kr])
        assert np.all(mg.tok2macro[np.arange(N)] >= 0)


def test_bucket_purity_hand_and_brute_force():
    """Reading R18.  Hand example: rows (1,0), (1,0.1), (0,1), (-1,0), (0,0) with
    codes 1 1 1 1 1 -> 10 pairs; cos > 0.7 only for rows 0-1 (0.995); the zero
    row pairs count as cos 0.  Then a brute-force double loop on random data
    with windows, and the closed forms for identical and orthogonal rows."""
    X = np.array([[1.0, 0.0], [1.0, 0.1], [0.0, 1.0], [-1.0, 0.0], [0.0, 0.0]])
    assert O.bucket_purity(X, np.ones(5, int)) == (1, 10)
    assert O.bucket_purity(X, np.arange(5)) == (0, 0)
    rng = np.random.default_rng(9)
    N, L = 96, 32
    Xr = rng.standard_normal((N, 3))
    Xr[5] = 0.0
    codes = rng.integers(0, 4, N)
    sim = tot = 0
    for i in range(N):
        for j in range(i + 1, N):
            if i // L == j // L and codes[i] == codes[j]:
                tot += 1
                ni, nj = np.linalg.norm(Xr[i]), np.linalg.norm(Xr[j])
                c = Xr[i] @ Xr[j] / (ni * nj) if ni > 0 and nj > 0 else 0.0
                sim += c > 0.7
    assert O.bucket_purity(Xr, codes, L=L) == (sim, tot)
    assert O.bucket_purity(np.tile(Xr[:1], (7, 1)), np.zeros(7, int)) == (21, 21)
    assert O.bucket_purity(np.eye(6), np.zeros(6, int)) == (0, 15)


def test_preserve_suffix_hand_example():
    """Reading R19: two compressed macro-tokens then a kept tail of 2 rows."""
    X = np.array([[3.0, 4.0], [1.0, 0.0], [0.0, 2.0], [-2.0, 0.0], [0.5, 0.5]])
    mg = O.merge(X[:3], np.array([5, 3, 5]))          # {0, 2} at 2, {1} at 1 -> order {1}, {0, 2}
    E, P, t2m = O.preserve_suffix(mg.E, mg.P, mg.tok2macro, X[3:], 3)
    assert list(P) == [1, 2, 3, 4] and list(t2m) == [1, 0, 1, 2, 3]
    assert np.array_equal(E[2:], X[3:]) and np.all(np.diff(P) > 0)
    _, Pc, _ = O.preserve_suffix(mg.E, np.arange(2), mg.tok2macro, X[3:], 3, compact=True)
    assert list(Pc) == [0, 1, 2, 3]


def test_adjust_to_target_hand_and_invariants():
    """Reading R20 (parity unpinned: the paper gives no algorithm).  Hand
    examples of both directions, then invariants on random groupings: exactly
    T groups, a partition of the members, ascending last members, merges join
    runs of consecutive groups, splits are contiguous member runs."""
    g = [np.array([0, 4]), np.array([1, 2, 5]), np.array([3, 6]), np.array([7])]
    # merge 4 -> 2: groups 0,1 -> new 0; groups 2,3 -> new 1
    m = O.adjust_to_target(g, 2)
    assert [list(x) for x in m] == [[0, 1, 2, 4, 5], [3, 6, 7]]
    # split 4 -> 6: E = 2, sizes 2 3 2 1, s-1 = 1 2 1 0, den = 8 - 4 = 4:
    # quotas 2*1/4, 2*2/4 = 1, 2*1/4, 0 -> extra 0 1 0 0, remainders 2 0 2 0 ->
    # R = 1 extra piece to group 0 (largest remainder, earliest)
    sp = O.adjust_to_target(g, 6)
    assert [list(x) for x in sp] == [[0], [1, 2], [4], [5], [3, 6], [7]]
    assert [list(x) for x in O.adjust_to_target(g, 4)] == [list(x) for x in g]
    rng = np.random.default_rng(13)
    for trial in range(30):
        N = int(rng.integers(20, 200))
        codes = rng.integers(0, int(rng.integers(2, 40)), N)
        mg = O.merge(np.zeros((N, 1)), codes)
        M = len(mg.members)
        for T in sorted({1, M, max(1, M // 3), min(N, 2 * M + 3), N}):
            out = O.adjust_to_target(mg.members, T)
            assert len(out) == T
            assert np.array_equal(np.sort(np.concatenate(out)), np.arange(N))
            last = [int(x[-1]) for x in out]
            assert last == sorted(last)
            if T < M:
                for gg in out:   # a merged group is a union of consecutive groups
                    ks = sorted({int(mg.tok2macro[v]) for v in gg})
                    assert ks == list(range(ks[0], ks[-1] + 1))
            if T > M:
                for gg in out:   # a piece lies inside one group, as a contiguous run
                    k = {int(mg.tok2macro[v]) for v in gg}
                    assert len(k) == 1
                    mem = list(mg.members[k.pop()])
                    i0 = mem.index(int(gg[0]))
                    assert mem[i0:i0 + len(gg)] == list(gg)


def test_merge_invariants():
    rng = np.random.default_rng(3)
    N, D = 700, 5
    X = rng.standard_normal((N, D))
    codes = rng.integers(0, 40, N)
    mg = O.merge(X, codes)
    M = len(mg.P)
    sizes = np.bincount(mg.tok2macro, minlength=M)
    assert sizes.sum() == N and np.all(sizes > 0)
    assert np.all(np.diff(mg.P) > 0)                      # strictly increasing
    assert np.all(np.arange(N) <= mg.P[mg.tok2macro])     # causal: never before a member
    for k in range(M):
        mem = mg.members[k]
        assert mg.P[k] == mem.max()
        assert np.all(codes[mem] == codes[mem[0]])
        eta = np.linalg.norm(X[mem], axis=1).mean()
        assert abs(np.linalg.norm(mg.E[k]) - eta) < 1e-12 * eta
        if len(mem) == 1:
            assert np.allclose(mg.E[k], X[mem[0]], rtol=1e-15, atol=0)
    # tokens with equal codes share a macro; different codes never do
    same = codes[:, None] == codes[None, :]
    assert np.array_equal(same, mg.tok2macro[:, None] == mg.tok2macro[None, :])
    cm = O.merge(X, codes, compact=True)
    assert list(cm.P) == list(range(M))


# ---------------------------------------------------------------- adaptive pieces
def test_redundancy_score_closed_forms():
    x = np.array([0.3, -1.2, 2.0])
    assert abs(O.redundancy_score(np.tile(x, (9, 1))) - 1.0) < 1e-14
    L = 16
    Q, _ = np.linalg.qr(np.random.default_rng(4).standard_normal((32, L)))
    assert abs(O.redundancy_score(2.5 * Q.T) - 1 / math.sqrt(L)) < 1e-12
    Xz = np.vstack([np.tile(x, (3, 1)), np.zeros((3, 3))])
    assert abs(O.redundancy_score(Xz) - 0.5) < 1e-14
    assert O.redundancy_score(np.zeros((4, 3))) == 0.0


def test_tau_schedule_and_routing():
    assert O.tau_of_rho(2) == pytest.approx(0.70)
    assert O.tau_of_rho(8) == pytest.approx(0.60)
    assert O.tau_of_rho(16) == pytest.approx(0.55)
    assert O.tau_of_rho(4) == pytest.approx(0.65)
    assert O.tau_of_rho(1.5) == pytest.approx(0.70)
    assert O.route_window(2048, 0.61, 8.0) and not O.route_window(2048, 0.59, 8.0)
    assert not O.route_window(4, 0.99, 8.0)
    assert O.route_window(2048, 0.0, 16.0)
    assert O.chunk_size(2.5) == 2 and O.chunk_size(3.5) == 4 and O.chunk_size(0.3) == 1


def test_chunk_pool_brute_force():
    rng = np.random.default_rng(6)
    Xw = rng.standard_normal((21, 4))
    E, P = O.chunk_pool(Xw, 8, pos0=100)
    assert list(P) == [107, 115, 120]
    for g, (s, e) in enumerate([(0, 8), (8, 16), (16, 21)]):
        acc = np.zeros(4)
        nsum = 0.0
        for i in range(s, e):
            acc += Xw[i]
            nsum += math.sqrt(sum(v * v for v in Xw[i]))
        acc /= (e - s)
        want = acc * (nsum / (e - s)) / math.sqrt(sum(v * v for v in acc))
        assert np.allclose(E[g], want, rtol=1e-13, atol=0)


# ---------------------------------------------------------------- end to end on the tiny workload
def test_tiny_end_to_end_invariants():
    inp = make_inputs("tiny")
    wl = inp.workload
    X = inp.x_float()
    res = O.compress(X, OP.projection(0, wl.D, wl.m), OP.phases(0, wl.m),
                     OP.start_vector(0, wl.N), OP.hyperplanes(0, wl.r, wl.bits), wl.n_it, wl.r)
    mg = res.merge
    assert np.bincount(mg.tok2macro).sum() == wl.N
    assert np.all(np.diff(mg.P) > 0)
    assert np.all(np.arange(wl.N) <= mg.P[mg.tok2macro])
    assert len(mg.P) <= 2 ** wl.bits
    assert res.lz.n_eff == wl.n_it
    # the top Ritz value is the dominant eigenvalue of Phi Phi^T (= that of Phi^T Phi)
    lam = np.linalg.eigvalsh(res.Phi.T @ res.Phi)
    assert abs(res.ritz_values[-1] - lam[-1]) < 1e-10 * lam[-1]
