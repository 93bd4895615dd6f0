"""The allocation-free merge (slh_merge_noalloc) against the context path
(slh_load of the same codes, then slh_merge) on two calls in a row, the second
smaller than the first: positions, token maps and M bit for bit, embeddings
to the parity rule's 1e-3 (the kernels are the same, so they are expected
bit-identical), plus the size limits it rejects before any GPU work."""
import sys

import numpy as np
import pytest

from workloads import Workload, Inputs, zipf_ids, embed, mixture
import parity as PR

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _inputs(N, D, x, seed):
    wl = Workload("na", N, D, 256, 8, 4, 8, 8.0, 32768, 0, x)
    if x == "f32":
        X, lab = mixture(seed, N, D)
        return Inputs(wl, X, lab)
    rng = np.random.default_rng(np.random.SeedSequence([seed, 0x1D5]))
    ids = zipf_ids(rng, 32768, N)
    return Inputs(wl, embed(seed, ids, D), ids)


def _context_merge(inp, codes, bits):
    import torch
    import paper_2607_19368_amd as P
    from paper_2607_19368_amd import slh as B
    wl = inp.workload
    ctx = P.slh_create(wl.N, wl.D, 256, 1, bits, 0)
    Xd = PR.to_device_x(inp)
    P.slh_load(ctx, B.SLH_OUT_CODES, torch.from_numpy(codes.astype(np.int32)).cuda())
    E, Pp, t2m, M = P.slh_merge(ctx, Xd)
    torch.cuda.synchronize()
    return E.cpu().numpy(), Pp.cpu().numpy(), t2m.cpu().numpy(), M


def test_merge_noalloc_matches_context_merge_twice():
    import torch
    import paper_2607_19368_amd as P
    P.load()
    cases = [(8192, 4096, "bf16", 12, 1), (1000, 264, "f32", 6, 2)]
    for N, D, x, bits, seed in cases:
        inp = _inputs(N, D, x, seed)
        rng = np.random.default_rng(seed)
        codes = np.minimum(rng.zipf(1.3, N) - 1, (1 << bits) - 1).astype(np.uint32)
        _say(f"[noalloc] N={N} D={D} x={x} bits={bits}")
        Xd = PR.to_device_x(inp)
        cd = torch.from_numpy(codes.astype(np.int32)).cuda()
        cap = min(N, 1 << bits)
        E = torch.empty((cap, D), dtype=torch.float32, device="cuda")
        Pp = torch.empty(cap, dtype=torch.int32, device="cuda")
        T = torch.empty(N, dtype=torch.int32, device="cuda")
        En, Pn, Tn, Mn = P.slh_merge_noalloc(Xd, cd, bits, E, Pp, T)
        torch.cuda.synchronize()
        Ec, Pc, Tc, Mc = _context_merge(inp, codes, bits)
        En, Pn, Tn = En.cpu().numpy(), Pn.cpu().numpy(), Tn.cpu().numpy()
        rel = np.linalg.norm(En - Ec, axis=1) / np.maximum(np.linalg.norm(Ec, axis=1), 1e-30)
        _say(f"   M={Mn} (context {Mc}) max emb rel {rel.max():.2e} identical={np.array_equal(En, Ec)}")
        assert Mn == Mc and np.array_equal(Pn, Pc) and np.array_equal(Tn, Tc)
        assert rel.max() <= 1e-3


def test_merge_noalloc_rejects_sizes_beyond_its_limits():
    import torch
    import paper_2607_19368_amd as P
    from paper_2607_19368_amd import slh as B
    lib = P.load()
    X = torch.zeros((8200, 16), dtype=torch.bfloat16, device="cuda")
    c = torch.zeros(8200, dtype=torch.int32, device="cuda")
    E = torch.empty((64, 16), dtype=torch.float32, device="cuda")
    Pp = torch.empty(64, dtype=torch.int32, device="cuda")
    with pytest.raises(B.SLHError, match=r"\(-1\)"):
        P.slh_merge_noalloc(X, c, 6, E, Pp)                    # N > 8192
    X2 = torch.zeros((64, 4104), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(B.SLHError, match=r"\(-1\)"):
        P.slh_merge_noalloc(X2, c[:64], 6, torch.empty((64, 4104), device="cuda"), Pp)   # D > 4096
    with pytest.raises(B.SLHError, match=r"\(-1\)"):
        P.slh_merge_noalloc(X[:200], c[:200], 7, E, Pp)        # cap 64 < min(200, 2^7)
