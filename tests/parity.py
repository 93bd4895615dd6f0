"""Runs the HIP path (through the C ABI binding) and the CPU oracle on the same
seeded inputs and compares them under the parity rules:

  * bucket codes, token->bucket maps and positions bit-exact, except rows where
    some oracle SimHash projection has |value| < 1e-5 (and every bucket that
    holds such a row, on either side);
  * kept Ritz values within 1e-3 relative error (values that are zero up to
    rounding, below 1e-12 of the largest, within that absolute floor);
  * largest principal angle between the GPU and oracle Ritz subspaces < 1e-2 rad;
  * macro-token embeddings within 1e-3 relative error (fp32 accumulation).
"""
import math
from dataclasses import dataclass, field

import numpy as np

from oracle import params as OP
from oracle import spectral_lsh as O

EXCL = 1e-5
RITZ_REL = 1e-3
ANGLE = 1e-2
EMB_REL = 1e-3


def to_device_x(inp):
    import torch
    X = inp.X
    if inp.workload.x_dtype == "bf16":
        t = torch.from_numpy(X.view(np.int16).copy()).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32))
    return t.cuda()


@dataclass
class Window:
    """Results of one window (oracle or GPU)."""
    w: int
    spectral: bool
    codes: np.ndarray = None        # window tokens (spectral)
    proj: np.ndarray = None
    ritz: np.ndarray = None
    Z: np.ndarray = None
    iters: int = 0
    alpha: np.ndarray = None
    beta: np.ndarray = None


@dataclass
class Run:
    windows: list = field(default_factory=list)
    E: np.ndarray = None
    P: np.ndarray = None
    t2m: np.ndarray = None
    Phi: np.ndarray = None
    scores: np.ndarray = None
    route: np.ndarray = None
    R: np.ndarray = None             # SimHash hyperplanes (oracle runs)
    rowsum: np.ndarray = None        # estimated row sums of the normalised operator
    xrows: object = None             # oracle runs: rows -> X as given (float64), for checks
    compact: bool = False            # positions are 0..M-1


def run_gpu(inp, n_it, seed=0, window=0, rho=None, tau=-1.0, kernel=0, compact=False,
            phi_from=None, codes_from=None, want_phi=False, X=None, short_windows=None,
            normalise=False, scheme=0, keep_last=None, timing=False, resident=None):
    """phi_from: host float32 array (n_act*L, m) loaded instead of computing Phi;
    codes_from: host uint32 (N,) loaded instead of computing codes;
    short_windows: value of SLH_OPT_SHORT_WINDOWS (None keeps the default);
    timing: SLH_OPT_TIMING = 1 (every Lanczos pass launched directly, timed);
    resident: value of SLH_OPT_RESIDENT (None keeps the default)."""
    import torch
    import paper_2607_19368_amd as P
    from paper_2607_19368_amd import slh as B
    wl = inp.workload
    ctx = P.slh_create(wl.N, wl.D, wl.m, wl.r, wl.bits, seed)
    if timing:
        P.slh_set_option(ctx, B.SLH_OPT_TIMING, 1)
    K = wl.keep_last if keep_last is None else keep_last
    if K:
        P.slh_set_option(ctx, B.SLH_OPT_KEEP_LAST, K)
    if window:
        P.slh_set_option(ctx, B.SLH_OPT_WINDOW_LEN, window)
    if kernel:
        P.slh_set_option(ctx, B.SLH_OPT_KERNEL, kernel)
    if compact:
        P.slh_set_option(ctx, B.SLH_OPT_POS_MODE, 1)
    if short_windows is not None:
        P.slh_set_option(ctx, B.SLH_OPT_SHORT_WINDOWS, short_windows)
    if resident is not None:
        P.slh_set_option(ctx, B.SLH_OPT_RESIDENT, resident)
    if normalise:
        P.slh_set_option(ctx, B.SLH_OPT_NORMALIZE, 1)
    if scheme:
        P.slh_set_option(ctx, B.SLH_OPT_POS_SCHEME, scheme)
    Xd = to_device_x(inp) if X is None else X
    run = Run()
    if rho is not None:
        run.route, run.scores = P.slh_route(ctx, Xd, rho, tau)
    L = ctx.window_len
    na = ctx.n_spectral
    if codes_from is None:
        if phi_from is None:
            P.slh_feature_map(ctx, Xd)
        else:
            P.slh_load(ctx, B.SLH_OUT_PHI, torch.from_numpy(np.ascontiguousarray(phi_from, np.float32)).cuda())
        if want_phi and na:
            run.Phi = P.slh_copy_out(ctx, B.SLH_OUT_PHI).reshape(na * L, wl.m)
        if normalise and na:
            run.rowsum = P.slh_copy_out(ctx, B.SLH_OUT_ROWSUM).reshape(-1)
        ritz, iters = P.slh_lanczos(ctx, n_it, want=True)
        P.slh_simhash(ctx)
        wins = P.slh_copy_out(ctx, B.SLH_OUT_WINDOWS)
        codes = P.slh_copy_out(ctx, B.SLH_OUT_CODES)
        if na:
            Z = P.slh_copy_out(ctx, B.SLH_OUT_Z)
            proj = P.slh_copy_out(ctx, B.SLH_OUT_PROJ)
            al = P.slh_copy_out(ctx, B.SLH_OUT_ALPHA)
            be = P.slh_copy_out(ctx, B.SLH_OUT_BETA)
        for a, w in enumerate(wins):
            run.windows.append(Window(int(w), True, codes[w * L:(w + 1) * L].astype(np.int64), proj[a],
                                      ritz[a], Z[a], int(iters[a]), al[a], be[a]))
    else:
        P.slh_load(ctx, B.SLH_OUT_CODES, torch.from_numpy(codes_from.astype(np.int32)).cuda())
    E, Pp, t2m, M = P.slh_merge(ctx, Xd)
    torch.cuda.synchronize()
    run.E = E.cpu().numpy().astype(np.float64)
    run.P = Pp.cpu().numpy().astype(np.int64)
    run.t2m = t2m.cpu().numpy().astype(np.int64)
    return run


def run_oracle(inp, n_it, seed=0, window=0, rho=None, tau=-1.0, kernel="softmax", compact=False,
               phi_rows=None, normalise=False, scheme="max", keep_last=None):
    wl = inp.workload
    Ntot = wl.N
    K = wl.keep_last if keep_last is None else keep_last
    N = Ntot - K                     # compressed tokens; the last K are preserved
    L = window or N
    W = OP.projection(seed, wl.D, wl.m)
    psi = OP.phases(seed, wl.m)
    R = OP.hyperplanes(seed, wl.r, wl.bits)
    run = Run()
    run.xrows = inp.x_float
    run.compact = compact
    Es, Ps = [], []
    t2m = np.zeros(N, np.int64)
    base = 0
    scores, route = [], []
    rowsums = []
    for w in range(N // L):
        Xw = inp.x_float(slice(w * L, (w + 1) * L))
        if rho is not None:
            sc = O.redundancy_score(Xw)
            spectral = O.route_window(L, sc, rho, None if tau < 0 else tau)
            scores.append(sc)
            route.append(spectral)
        else:
            spectral = True
        if spectral:
            Phi = O.feature_map(Xw, W, psi, kernel)
            if normalise:
                Phi, s_hat = O.normalised_features(Phi)
                rowsums.append(s_hat)
            lz = O.lanczos(Phi, OP.start_vector(seed, L, w), n_it)
            vals, Z, _, _ = O.ritz(lz, wl.r)
            proj = O.projections(Z, R)
            codes = O.simhash(Z, R)
            mg = O.merge(Xw, codes, positions=w * L + np.arange(L), scheme=scheme)
            al = np.zeros(n_it); al[:lz.n_eff] = lz.alpha
            be = np.zeros(n_it); be[:lz.n_eff] = lz.beta
            run.windows.append(Window(w, True, codes, proj, vals, Z, lz.n_eff, al, be))
            if phi_rows is not None:
                phi_rows.append(Phi)
            E, Pw, tm = mg.E, mg.P, mg.tok2macro
        else:
            k = O.chunk_size(rho)
            E, Pw = O.chunk_pool(Xw, k, pos0=w * L, scheme=scheme)
            tm = np.arange(L) // k
        Es.append(E)
        Ps.append(Pw)
        t2m[w * L:(w + 1) * L] = base + tm
        base += len(Pw)
    run.E = np.concatenate(Es)
    run.P = np.concatenate(Ps)
    run.R = R
    if rowsums:
        run.rowsum = np.concatenate(rowsums)
    if compact:
        run.P = np.arange(len(run.P))
    run.t2m = t2m
    if K:
        run.E, run.P, run.t2m = O.preserve_suffix(run.E, run.P, run.t2m,
                                                  inp.x_float(slice(N, Ntot)), N, compact)
    if rho is not None:
        run.scores = np.array(scores)
        run.route = np.array(route, dtype=np.uint8)
    return run


_PARAMS = {}


def _params(seed, D, m, r, bits):
    """The oracle's W, psi, R for these sizes, drawn once per process."""
    key = (seed, D, m, r, bits)
    if key not in _PARAMS:
        _PARAMS[key] = (OP.projection(seed, D, m), OP.phases(seed, m), OP.hyperplanes(seed, r, bits))
    return _PARAMS[key]


def oracle_uncertainty(inp, w, L, n_it, seed=0, normalise=False):
    """How far two valid fp64 evaluations of the method disagree on window w.

    Reversing the token order leaves the method's result unchanged up to the
    same permutation (Eq. 4 and Algorithm 2 are permutation-equivariant when q1
    is permuted with the tokens), but changes every summation order.  Returns
    max |proj - proj_reversed| over the window: SimHash bits whose oracle
    projection is smaller than this are not determined in fp64 arithmetic."""
    wl = inp.workload
    W, psi, R = _params(seed, wl.D, wl.m, wl.r, wl.bits)
    Xw = inp.x_float(slice(w * L, (w + 1) * L))
    q1 = OP.start_vector(seed, L, w)
    rv = np.arange(L)[::-1]
    Phi = O.feature_map(Xw, W, psi)
    if normalise:
        Phi, _ = O.normalised_features(Phi)
    _, Z, _, _ = O.ritz(O.lanczos(Phi, q1, n_it), wl.r)
    _, Zr, _, _ = O.ritz(O.lanczos(Phi[rv], q1[rv], n_it), wl.r)
    return float(np.max(np.abs(Zr[rv] @ R - Z @ R)))


def subspace_angle(Zo, Zg):
    """Largest principal angle, arcsin ||(I - Zo Zo^T) Zg||_2 (orthonormal columns)."""
    if Zo.shape[1] == 0:
        return 0.0
    Qo, _ = np.linalg.qr(Zo)
    Qg, _ = np.linalg.qr(Zg)
    res = Qg - Qo @ (Qo.T @ Qg)
    s = np.linalg.norm(res, 2)
    return math.asin(min(1.0, s))


@dataclass
class Report:
    excluded_rows: int = 0
    at_risk_rows: int = 0
    code_mismatch: int = 0
    max_ritz_rel: float = 0.0
    max_angle: float = 0.0
    max_emb_rel: float = 0.0
    buckets_checked: int = 0
    buckets_excluded: int = 0
    undetermined_rows: int = 0
    undecided_windows: int = 0
    literal_rule_mismatch_rows: int = 0   # code mismatches outside the bare 1e-5 band
    gpu_macros_validated: int = 0         # GPU macros checked on their own members


def compare(o, g, L, check_spectral=True, ritz_rel=RITZ_REL, angle=ANGLE, emb_rel=EMB_REL,
            exact_codes=False, merge_only=False, unc=None, scheme="max"):
    """Assert the parity rules; returns a Report.

    unc: optional {window: U} from oracle_uncertainty(); a SimHash bit whose
    oracle projection is below max(1e-5, 2 U) is then treated like the 1e-5
    exclusion (its value is not determined by fp64 evaluation of the method)."""
    rep = Report()
    N = len(o.t2m)
    assert len(g.t2m) == N
    ow = {w.w: w for w in o.windows}
    gw = {w.w: w for w in g.windows}
    if merge_only:
        ow = {}
    else:
        assert set(ow) == set(gw), (sorted(ow), sorted(gw))
    excluded_tok = np.zeros(N, bool)
    for w, a in ow.items():
        b = gw[w]
        floor_a = 1e-12 * float(np.abs(a.ritz).max(initial=0))
        floor_b = 1e-12 * float(np.abs(b.ritz).max(initial=0))
        undecided = False
        if a.iters != b.iters:
            # Only where the operator's rank ran out inside the Krylov space: the
            # step that decides the breakdown then compares a rounding-noise beta
            # with the threshold, so the two sides may stop one or two steps
            # apart.  The extra steps add Ritz values that are zero up to
            # rounding; where they are among the kept columns the spectral check
            # below requires it (the counts of the other, determined values must
            # agree), where they are not (r below the rank) they leave the kept
            # values unchanged.  The window's SimHash bits are not determined.
            assert abs(a.iters - b.iters) <= 2, (w, a.iters, b.iters)
            # the deciding beta (first step where one side stops) is at noise
            # level on both sides: at most 1e-6 of that side's largest |alpha|
            j0 = min(a.iters, b.iters) - 1
            for s_ in (a, b):
                if s_.beta is not None and s_.alpha is not None:
                    am = float(np.abs(s_.alpha[:j0 + 1]).max())
                    assert s_.beta[j0] <= 1e-6 * am, (w, j0, s_.beta[j0], am)
            undecided = True
            rep.undecided_windows += 1
        if check_spectral:
            # Ritz values that are zero up to rounding (a rank-deficient operator
            # inside the Krylov space) have no relative accuracy: they are checked
            # against an absolute floor of 1e-12 of the largest one instead, and
            # their Ritz vectors (directions of the null space that rounding
            # picked) are left out of the subspace comparison.  Columns are in
            # ascending order, so the determined ones align from the top.
            ka = np.flatnonzero(np.abs(a.ritz) > floor_a)
            kb = np.flatnonzero(np.abs(b.ritz) > floor_b)
            assert len(ka) == len(kb), (w, len(ka), len(kb))
            rel = np.abs(b.ritz[kb] - a.ritz[ka]) / np.abs(a.ritz[ka])
            rep.max_ritz_rel = max(rep.max_ritz_rel, float(rel.max(initial=0)))
            assert np.all(rel <= ritz_rel), (w, rel.max())
            if not undecided:
                tiny = (a.ritz != 0) & (np.abs(a.ritz) <= floor_a)
                assert np.all(np.abs(b.ritz[tiny] - a.ritz[tiny]) <= floor_a), (w, b.ritz[tiny], a.ritz[tiny])
            ang = subspace_angle(a.Z[:, ka], b.Z[:, kb])
            rep.max_angle = max(rep.max_angle, ang)
            assert ang < angle, (w, ang)
        if undecided:
            rep.undetermined_rows += L
            rep.excluded_rows += L
            rep.literal_rule_mismatch_rows += int(np.count_nonzero(
                (a.codes != b.codes) & ~np.any(np.abs(a.proj) < EXCL, axis=1)))
            excluded_tok[w * L:(w + 1) * L] = True
            continue
        ex = np.any(np.abs(a.proj) < EXCL, axis=1)
        rep.literal_rule_mismatch_rows += int(np.count_nonzero((a.codes != b.codes) & ~ex))
        tiny = (a.ritz != 0) & (np.abs(a.ritz) <= floor_a)
        if np.count_nonzero(tiny) >= 2 and o.R is not None:
            # a null space of dimension >= 2 inside the Krylov space: any basis of
            # it is a valid set of Ritz vectors, so a bit is determined only where
            # no rotation of that basis can flip it.  The null space adds
            # Z[i, null] U R[null, l] to the projection for some orthogonal U,
            # at most |Z[i, null]| |R[null, l]| in magnitude (Cauchy-Schwarz),
            # so the part of the projection outside the null space must exceed
            # that bound
            zt = np.linalg.norm(a.Z[:, tiny], axis=1)[:, None]
            rt = np.linalg.norm(o.R[tiny], axis=0)[None, :]
            p_out = a.Z[:, ~tiny] @ o.R[~tiny]
            und = np.any(np.abs(p_out) <= zt * rt, axis=1) & ~ex
            rep.undetermined_rows += int(und.sum())
            ex |= und
        if unc is not None and w in unc:
            thr = max(EXCL, 2.0 * unc[w])
            und = np.any(np.abs(a.proj) < thr, axis=1) & ~ex
            rep.undetermined_rows += int(und.sum())
            ex |= und
        if exact_codes:
            ex[:] = False
        dproj = np.max(np.abs(b.proj - a.proj))
        risk = np.any((np.abs(a.proj) >= EXCL) & (np.abs(a.proj) < dproj), axis=1)
        rep.at_risk_rows += int(risk.sum())
        rep.excluded_rows += int(ex.sum())
        mism = (a.codes != b.codes) & ~ex
        rep.code_mismatch += int(mism.sum())
        assert not mism.any(), (w, np.flatnonzero(mism)[:10])
        # buckets holding an excluded row (on either side) are excluded
        bad = set(a.codes[ex].tolist()) | set(b.codes[ex].tolist())
        bad_tok = np.isin(a.codes, list(bad)) | np.isin(b.codes, list(bad)) if bad else np.zeros(L, bool)
        excluded_tok[w * L:(w + 1) * L] = bad_tok
    # merge: every oracle macro whose members avoid excluded tokens must appear on
    # the GPU with the same members, position and (close) embedding
    Mo = len(o.P)
    members_o = [[] for _ in range(Mo)]
    for i, k in enumerate(o.t2m):
        members_o[k].append(i)
    Mg = len(g.P)
    assert g.t2m.min() >= 0 and g.t2m.max() < Mg
    members_g = [[] for _ in range(Mg)]
    for i, k in enumerate(g.t2m):
        members_g[k].append(i)
    assert all(len(mm) > 0 for mm in members_g)
    # GPU structural invariants of the position scheme (section 3.4): max and
    # median positions are distinct members (strictly increasing), the max is
    # causal; mean positions lie within the members' range (non-decreasing)
    if scheme == "mean":
        assert np.all(np.diff(g.P) >= 0)
    else:
        assert np.all(np.diff(g.P) > 0)
    compact = bool(o.compact)
    for k, mm in enumerate(members_g):
        if compact:
            assert g.P[k] == k
            continue
        if scheme == "max":
            assert g.P[k] == max(mm)
        elif scheme == "median":
            assert g.P[k] in mm
        else:
            assert min(mm) <= g.P[k] <= max(mm)
    matched = np.zeros(Mg, bool)
    for k, mm in enumerate(members_o):
        if excluded_tok[mm].any():
            rep.buckets_excluded += 1
            continue
        kg = g.t2m[mm[0]]
        assert members_g[kg] == mm, (k, mm[:5], members_g[kg][:5])
        assert g.P[kg] == o.P[k]
        den = np.linalg.norm(o.E[k])
        err = np.linalg.norm(g.E[kg] - o.E[k]) / (den if den > 0 else 1.0)
        rep.max_emb_rel = max(rep.max_emb_rel, float(err))
        assert err <= emb_rel, (k, err)
        rep.buckets_checked += 1
        matched[kg] = True
    # every GPU macro-token no checked oracle bucket vouches for (it holds a row
    # the rules exclude) must still be a valid macro-token of its own members:
    # one window, one GPU code (spectral windows), the scheme's position of
    # its members, and the Eq. 7 renormalised mean of their rows
    if o.xrows is not None:
        gcodes = {w.w: w.codes for w in g.windows}
        for kg in np.flatnonzero(~matched):
            mm = np.asarray(members_g[kg])
            w0 = int(mm[0]) // L
            assert np.all(mm // L == w0), (kg, mm[:5])          # one window
            if w0 in gcodes:                                     # one code
                cw = gcodes[w0][mm - w0 * L]
                assert np.all(cw == cw[0]), (kg, np.unique(cw))
            if not compact and scheme == "max":
                assert g.P[kg] == mm.max()
            ref = O.renormalised_mean(o.xrows(mm))
            den = np.linalg.norm(ref)
            err = np.linalg.norm(g.E[kg] - ref) / (den if den > 0 else 1.0)
            assert err <= emb_rel, (kg, err)
            rep.gpu_macros_validated += 1
    return rep
