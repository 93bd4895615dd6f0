"""CPU checks of the C ABI: the library loads, exports every declared symbol,
draws the method's parameters bit-identically to the oracle's independent
generator, and rejects bad arguments before touching a GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import params as OP
import paper_2607_19368_amd.slh as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "slh.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(slh_\w+)\s*\(", src)))


def test_library_exports_every_declared_function():
    lib = B.load()
    names = header_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.EXPORTS)


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", "/nonexistent/libslh.so")
    with pytest.raises(B.SLHError):
        B.load()


@pytest.mark.parametrize("seed,D,m,r,bits", [(0, 256, 256, 8, 6), (5, 64, 512, 3, 16), (2**40 + 7, 24, 256, 1, 1)])
def test_parameters_match_oracle_generator(seed, D, m, r, bits):
    W, psi, R = B.slh_gen_params(seed, D, m, r, bits)
    Wv = (W.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert np.array_equal(Wv, OP.projection(seed, D, m))
    assert np.array_equal(psi.astype(np.float64), OP.phases(seed, m))
    Ro = OP.hyperplanes(seed, r, bits)
    # both sides evaluate Box-Muller with their own libm; allow 2 ulp
    assert np.all(np.abs(R - Ro) <= 4.5e-16 * np.maximum(np.abs(Ro), 1e-300))


@pytest.mark.parametrize("window,n", [(0, 512), (7, 2048), (3, 33)])
def test_start_vector_matches_oracle(window, n):
    q = B.slh_gen_start(11, window, n)
    qo = OP.start_vector(11, n, window)
    assert np.max(np.abs(q - qo)) < 1e-15
    assert abs(np.linalg.norm(q) - 1.0) < 1e-14


@pytest.mark.parametrize("args", [
    (1, 256, 256, 8, 6),        # N < 2
    (0, 256, 256, 8, 6),
    (512, 250, 256, 8, 6),      # D % 8
    (512, 0, 256, 8, 6),
    (512, 256, 300, 8, 6),      # m % 256
    (512, 256, 4096, 8, 6),     # m > 2048
    (512, 256, 256, 0, 6),      # r
    (512, 256, 256, 129, 6),
    (512, 256, 256, 8, 0),      # bits
    (512, 256, 256, 8, 17),
])
def test_create_rejects_bad_sizes_without_gpu(args):
    lib = B.load()
    h = ctypes.c_void_p(1234)
    rc = lib.slh_create(ctypes.byref(h), *args, 0)
    assert rc == B.SLH_EINVAL
    assert not h.value


def test_host_calls_reject_bad_arguments():
    lib = B.load()
    assert lib.slh_gen_params(0, 0, 256, 1, 1, None, None, None) == B.SLH_EINVAL
    assert lib.slh_gen_start(0, 0, 0, None) == B.SLH_EINVAL
    assert lib.slh_set_option(None, B.SLH_OPT_KERNEL, 0.0) == B.SLH_EINVAL
    assert lib.slh_feature_map(None, None, 0, 0) == B.SLH_EINVAL
    assert lib.slh_lanczos(None, 4, None, None) == B.SLH_EINVAL
    assert lib.slh_copy_out(None, B.SLH_OUT_PHI, None, 0) == B.SLH_EINVAL
    assert lib.slh_merge_capacity(None) == 0


def test_header_constants_match_binding():
    src = open(os.path.join(ROOT, "include", "slh.h")).read()
    defs = dict(re.findall(r"#define\s+(SLH_[A-Z0-9_]+)\s+\(?(-?\d+)\)?", src))
    assert len(defs) >= 20
    for name, val in defs.items():
        assert getattr(B, name) == int(val), name


@pytest.mark.parametrize("rho", [1.0, 0.5])
def test_identity_path_returns_prompt_unchanged(rho):
    """rho <= 1: the wrapper returns X itself with positions 0..N-1 and the
    identity token map, without calling the library (no GPU involved)."""
    import torch
    X = torch.randn(37, 16, dtype=torch.float32)
    E, P, t2m, M, lz = B.compress(None, X, 8, rho=rho)
    assert E is X and M == 37 and lz is None
    assert torch.equal(P, torch.arange(37, dtype=torch.int32)) and torch.equal(t2m, P)


def test_destroy_frees_every_context_buffer():
    """Every grow-only device buffer that the context declares is on the list
    slh_destroy frees (a buffer missing from it leaks once per context)."""
    src = open(os.path.join(ROOT, "paper_2607_19368_amd", "csrc", "slh_api.cpp")).read()
    declared = set()
    for m in re.finditer(r"^\s*DevBuf ([^;]+);", src, re.M):
        declared.update(n.strip() for n in m.group(1).split(","))
    i = src.index("DevBuf* bufs[] = {")
    freed = set(re.findall(r"&c->(\w+)", src[i:src.index("};", i)]))
    assert declared, "no DevBuf members found"
    assert declared - freed == set(), "not freed by slh_destroy"
    assert freed - declared == set()
