"""Python binding of libslh.so (include/slh.h): argument marshalling only.

Every function keeps the C name and takes torch tensors for device buffers
(PyTorch supplies device memory and the stream); all computation runs in the
library's HIP kernels.  There is no fallback: if the library is not built or
cannot be loaded, every call raises.
"""
import collections
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libslh.so")

SLH_OK, SLH_EINVAL, SLH_ENOMEM, SLH_EHIP, SLH_ESTATE = 0, -1, -2, -3, -4
SLH_BF16, SLH_F32 = 0, 1
SLH_OPT_KERNEL, SLH_OPT_WINDOW_LEN, SLH_OPT_POS_MODE, SLH_OPT_BREAKDOWN_TOL, SLH_OPT_TIMING = 1, 2, 3, 4, 5
SLH_OPT_SHORT_WINDOWS, SLH_OPT_NORMALIZE, SLH_OPT_POS_SCHEME, SLH_OPT_KEEP_LAST = 6, 7, 8, 9
SLH_OPT_TARGET_LEN, SLH_OPT_RESIDENT, SLH_OPT_WAIT_POLLS = 10, 11, 12
SLH_OUT_PHI, SLH_OUT_ALPHA, SLH_OUT_BETA, SLH_OUT_Z = 1, 2, 3, 4
SLH_OUT_PROJ, SLH_OUT_CODES, SLH_OUT_THETA, SLH_OUT_Q, SLH_OUT_WINDOWS = 5, 6, 7, 8, 9
SLH_OUT_ROWSUM = 10
SLH_NOALLOC_BYTES = 17355008

EXPORTS = [
    "slh_gen_params", "slh_gen_start", "slh_create", "slh_destroy", "slh_last_error",
    "slh_set_option", "slh_set_stream", "slh_route", "slh_feature_map", "slh_lanczos",
    "slh_simhash", "slh_merge", "slh_merge_capacity", "slh_copy_out", "slh_num_windows",
    "slh_num_spectral", "slh_load", "slh_stage_times", "slh_time_passes", "slh_spectral_energy",
    "slh_bucket_purity", "slh_eigh_ritz", "slh_peak_read", "slh_peak_mfma", "slh_merge_noalloc",
    "slh_merge_async", "slh_merge_wait",
]

_lib = None


class SLHError(RuntimeError):
    pass


def load():
    """Load libslh.so (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise SLHError(f"{LIB_PATH} is not built; run `python -m paper_2607_19368_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u64, dp = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p
    sig = {
        "slh_gen_params": (i32, [u64, i64, i64, i32, i32, vp, vp, vp]),
        "slh_gen_start": (i32, [u64, i64, i64, vp]),
        "slh_create": (i32, [ctypes.POINTER(vp), i64, i64, i64, i32, i32, u64]),
        "slh_destroy": (None, [vp]),
        "slh_last_error": (ctypes.c_char_p, [vp]),
        "slh_set_option": (i32, [vp, i32, ctypes.c_double]),
        "slh_set_stream": (i32, [vp, vp]),
        "slh_route": (i32, [vp, vp, i32, i64, ctypes.c_double, ctypes.c_double, vp, vp]),
        "slh_feature_map": (i32, [vp, vp, i32, i64]),
        "slh_lanczos": (i32, [vp, i32, vp, vp]),
        "slh_eigh_ritz": (i32, [vp, i32, vp, vp]),
        "slh_peak_read": (i32, [vp, i64, i32, vp, vp]),
        "slh_peak_mfma": (i32, [i32, vp, vp, vp]),
        "slh_merge_noalloc": (i32, [vp, i32, i64, i64, i64, vp, i32, vp, vp, vp, i64, vp, vp]),
        "slh_simhash": (i32, [vp, vp]),
        "slh_merge": (i32, [vp, vp, i32, i64, vp, vp, vp, i64, vp]),
        "slh_merge_async": (i32, [vp, vp, i32, i64, vp, vp, vp, i64]),
        "slh_merge_wait": (i32, [vp, vp]),
        "slh_merge_capacity": (i64, [vp]),
        "slh_copy_out": (i32, [vp, i32, vp, i64]),
        "slh_num_windows": (i64, [vp]),
        "slh_num_spectral": (i64, [vp]),
        "slh_load": (i32, [vp, i32, vp, i64]),
        "slh_spectral_energy": (i32, [vp, vp]),
        "slh_bucket_purity": (i32, [vp, vp, i32, i64, ctypes.c_double, vp]),
        "slh_stage_times": (i32, [vp, vp, i32]),
        "slh_time_passes": (i32, [vp, i32, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(ctx, rc, what):
    if rc != SLH_OK:
        msg = load().slh_last_error(ctx.handle if ctx is not None else None)
        raise SLHError(f"{what} failed ({rc}): {msg.decode() if msg else ''}")


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if isinstance(a, np.ndarray) else ctypes.c_void_p(a)


def _xinfo(X):
    import torch
    if X.dim() != 2 or X.stride(1) != 1:
        raise SLHError("X must be a 2-D tensor with unit column stride")
    if X.dtype == torch.bfloat16:
        dt = SLH_BF16
    elif X.dtype == torch.float32:
        dt = SLH_F32
    else:
        raise SLHError(f"unsupported X dtype {X.dtype}")
    if not X.is_cuda:
        raise SLHError("X must be a device tensor")
    return ctypes.c_void_p(X.data_ptr()), dt, X.stride(0)


class Ctx:
    """Owns one slh_ctx handle."""

    def __init__(self, handle, N, D, m, r, bits):
        self.handle = handle
        self.N, self.D, self.m, self.r, self.bits = N, D, m, r, bits
        self.n_it = 0
        self.keep_last = 0          # preserved suffix (tokens N - keep_last .. N - 1)
        self.in_flight = collections.deque()   # tensors of merges not yet waited for

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.slh_destroy(self.handle)
            self.handle = None

    @property
    def n_windows(self):
        return int(load().slh_num_windows(self.handle))

    @property
    def n_spectral(self):
        return int(load().slh_num_spectral(self.handle))

    @property
    def window_len(self):
        return (self.N - self.keep_last) // self.n_windows


# ---------------------------------------------------------------- host-only calls
def slh_gen_params(seed, D, m, r, bits):
    """(W bf16 bits [D, m] uint16, psi [m] float32, R [r, bits] float64)."""
    W = np.empty((D, m), np.uint16)
    psi = np.empty(m, np.float32)
    R = np.empty((r, bits), np.float64)
    rc = load().slh_gen_params(seed, D, m, r, bits, _ptr(W), _ptr(psi), _ptr(R))
    if rc != SLH_OK:
        raise SLHError(f"slh_gen_params failed ({rc})")
    return W, psi, R


def slh_gen_start(seed, window, n):
    q = np.empty(n, np.float64)
    rc = load().slh_gen_start(seed, window, n, _ptr(q))
    if rc != SLH_OK:
        raise SLHError(f"slh_gen_start failed ({rc})")
    return q


# ---------------------------------------------------------------- context calls
def slh_create(N, D, m, r, bits, seed=0):
    h = ctypes.c_void_p()
    rc = load().slh_create(ctypes.byref(h), N, D, m, r, bits, seed)
    if rc != SLH_OK:
        raise SLHError(f"slh_create(N={N}, D={D}, m={m}, r={r}, bits={bits}) failed ({rc})")
    ctx = Ctx(h, N, D, m, r, bits)
    slh_set_stream(ctx)
    return ctx


def slh_set_option(ctx, key, value):
    _check(ctx, load().slh_set_option(ctx.handle, key, float(value)), "slh_set_option")
    if key == SLH_OPT_KEEP_LAST:
        ctx.keep_last = int(value)


def slh_set_stream(ctx, stream=None):
    """Use `stream` (a torch.cuda.Stream; default: torch's current stream)."""
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    _check(ctx, load().slh_set_stream(ctx.handle, ctypes.c_void_p(stream.cuda_stream)), "slh_set_stream")


def slh_route(ctx, X, rho, tau=-1.0):
    p, dt, ld = _xinfo(X)
    nw = ctx.n_windows
    route = np.empty(nw, np.uint8)
    scores = np.empty(nw, np.float64)
    _check(ctx, load().slh_route(ctx.handle, p, dt, ld, float(rho), float(tau), _ptr(route), _ptr(scores)),
           "slh_route")
    return route, scores


def slh_feature_map(ctx, X):
    p, dt, ld = _xinfo(X)
    _check(ctx, load().slh_feature_map(ctx.handle, p, dt, ld), "slh_feature_map")


def slh_lanczos(ctx, n_it, want=True):
    """Runs n_it steps; returns (ritz [n_spectral, r], iters [n_spectral]) or None."""
    ctx.n_it = n_it
    na = ctx.n_spectral
    if want:
        ritz = np.zeros((na, ctx.r), np.float64)
        iters = np.zeros(na, np.int32)
        _check(ctx, load().slh_lanczos(ctx.handle, n_it, _ptr(ritz), _ptr(iters)), "slh_lanczos")
        return ritz, iters
    _check(ctx, load().slh_lanczos(ctx.handle, n_it, None, None), "slh_lanczos")
    return None


def slh_eigh_ritz(ctx, n_it, want=True):
    """Eigh(T) and Z = Q S on the context's T and Q (after slh_lanczos, or after
    slh_load of SLH_OUT_ALPHA, SLH_OUT_BETA and SLH_OUT_Q); returns (ritz, iters)
    as slh_lanczos does, or None."""
    ctx.n_it = n_it
    na = ctx.n_spectral
    if want:
        ritz = np.zeros((na, ctx.r), np.float64)
        iters = np.zeros(na, np.int32)
        _check(ctx, load().slh_eigh_ritz(ctx.handle, n_it, _ptr(ritz), _ptr(iters)), "slh_eigh_ritz")
        return ritz, iters
    _check(ctx, load().slh_eigh_ritz(ctx.handle, n_it, None, None), "slh_eigh_ritz")
    return None


def slh_simhash(ctx, codes_out=None):
    if codes_out is not None:
        import torch
        _device_tensor("codes_out", codes_out, (torch.int32, torch.uint32), (ctx.N,))
    p = ctypes.c_void_p(codes_out.data_ptr()) if codes_out is not None else None
    _check(ctx, load().slh_simhash(ctx.handle, p), "slh_simhash")
    return codes_out


def slh_merge_capacity(ctx):
    return int(load().slh_merge_capacity(ctx.handle))


def _device_tensor(name, t, dtypes=None, shape=None, device=None):
    """The library reads or writes t through a raw device pointer: it must be a
    contiguous device tensor (of one of `dtypes`, of `shape` where an entry
    None is free, on `device`)."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda or (device is not None and t.device != device):
        raise SLHError(f"{name} must be a device tensor" + (f" on {device}" if device is not None else ""))
    if (dtypes is not None and t.dtype not in dtypes) or not t.is_contiguous():
        kinds = " or ".join(str(d) for d in dtypes) if dtypes is not None else "any type"
        raise SLHError(f"{name} must be a contiguous tensor of {kinds}")
    if shape is not None and (t.dim() != len(shape)
                              or any(w is not None and w != d for w, d in zip(shape, t.shape))):
        want = ", ".join("*" if w is None else str(w) for w in shape)
        raise SLHError(f"{name} must have shape ({want})")


def _check_merge_outputs(D, N, device, emb_out, pos_out, tok2macro_out):
    """Merge outputs: E [cap, D] float32, P [>= cap] int32, tok2macro [N] int32."""
    import torch
    _device_tensor("emb_out", emb_out, (torch.float32,), (None, D), device)
    _device_tensor("pos_out", pos_out, (torch.int32,), (None,), device)
    if tok2macro_out is not None:
        _device_tensor("tok2macro_out", tok2macro_out, (torch.int32,), (N,), device)
    if pos_out.shape[0] < emb_out.shape[0]:
        raise SLHError("pos_out must hold at least as many entries as emb_out")


def slh_merge(ctx, X, emb_out=None, pos_out=None, tok2macro_out=None):
    """Returns (E [M, D] float32, P [M] int32, tok2macro [N] int32, M) as device tensors
    (views of the given or newly allocated outputs)."""
    import torch
    p, dt, ld = _xinfo(X)
    cap = slh_merge_capacity(ctx)
    if emb_out is None:
        emb_out = torch.empty((cap, ctx.D), dtype=torch.float32, device=X.device)
    if pos_out is None:
        pos_out = torch.empty(cap, dtype=torch.int32, device=X.device)
    if tok2macro_out is None:
        tok2macro_out = torch.empty(ctx.N, dtype=torch.int32, device=X.device)
    _check_merge_outputs(ctx.D, ctx.N, X.device, emb_out, pos_out, tok2macro_out)
    M = ctypes.c_int64(0)
    _check(ctx, load().slh_merge(ctx.handle, p, dt, ld, ctypes.c_void_p(emb_out.data_ptr()),
                                 ctypes.c_void_p(pos_out.data_ptr()),
                                 ctypes.c_void_p(tok2macro_out.data_ptr()), emb_out.shape[0],
                                 ctypes.byref(M)), "slh_merge")
    m = int(M.value)
    return emb_out[:m], pos_out[:m], tok2macro_out, m


def slh_merge_async(ctx, X, emb_out, pos_out, tok2macro_out=None):
    """Enqueues the merge into the given device outputs and returns at once; the
    outputs hold the result once slh_merge_wait has returned its M.  X and the
    outputs are kept referenced until that wait, since the GPU still reads and
    writes them."""
    p, dt, ld = _xinfo(X)
    _check_merge_outputs(ctx.D, ctx.N, X.device, emb_out, pos_out, tok2macro_out)
    _check(ctx, load().slh_merge_async(ctx.handle, p, dt, ld, ctypes.c_void_p(emb_out.data_ptr()),
                                       ctypes.c_void_p(pos_out.data_ptr()),
                                       ctypes.c_void_p(tok2macro_out.data_ptr())
                                       if tok2macro_out is not None else None,
                                       emb_out.shape[0]), "slh_merge_async")
    ctx.in_flight.append((X, emb_out, pos_out, tok2macro_out))


def slh_merge_wait(ctx):
    """M of the oldest merge from slh_merge_async not yet waited for."""
    M = ctypes.c_int64(0)
    rc = load().slh_merge_wait(ctx.handle, ctypes.byref(M))
    if rc != SLH_ESTATE and ctx.in_flight:
        ctx.in_flight.popleft()          # that merge has left the GPU
    _check(ctx, rc, "slh_merge_wait")
    return int(M.value)


_OUT = {
    SLH_OUT_PHI: (np.float32, lambda c: (c.n_spectral, c.window_len, c.m)),
    SLH_OUT_ALPHA: (np.float64, lambda c: (c.n_spectral, c.n_it)),
    SLH_OUT_BETA: (np.float64, lambda c: (c.n_spectral, c.n_it)),
    SLH_OUT_Z: (np.float64, lambda c: (c.n_spectral, c.window_len, c.r)),
    SLH_OUT_PROJ: (np.float64, lambda c: (c.n_spectral, c.window_len, c.bits)),
    SLH_OUT_CODES: (np.uint32, lambda c: (c.N,)),
    SLH_OUT_THETA: (np.float64, lambda c: (c.n_spectral, c.r)),
    SLH_OUT_Q: (np.float64, lambda c: (c.n_spectral, c.n_it + 1, c.window_len)),
    SLH_OUT_WINDOWS: (np.int32, lambda c: (c.n_spectral,)),
    SLH_OUT_ROWSUM: (np.float64, lambda c: (c.n_spectral, c.window_len)),
}


STAGE_NAMES = ["featmap_ms", "lanczos_ms", "phi_pass_ms_sum", "phi_pass_count", "eig_ritz_ms",
               "simhash_ms", "merge_ms", "normalise_ms", "lanczos_resident"]


def slh_stage_times(ctx):
    """Dict of the stage timings recorded with SLH_OPT_TIMING = 1."""
    out = np.zeros(len(STAGE_NAMES), np.float64)
    _check(ctx, load().slh_stage_times(ctx.handle, _ptr(out), len(out)), "slh_stage_times")
    return dict(zip(STAGE_NAMES, out.tolist()))


def slh_time_passes(ctx, reps=96):
    """Microseconds per pass over Phi, from a graph replay of the last Lanczos step's passes."""
    out = np.zeros(1, np.float64)
    _check(ctx, load().slh_time_passes(ctx.handle, int(reps), _ptr(out)), "slh_time_passes")
    return float(out[0])


def slh_load(ctx, which, src):
    """Replace a stage result (SLH_OUT_PHI, SLH_OUT_ALPHA, SLH_OUT_BETA, SLH_OUT_Q or
    SLH_OUT_CODES) with a device tensor."""
    import torch
    kinds = {SLH_OUT_PHI: (torch.float32,), SLH_OUT_ALPHA: (torch.float64,),
             SLH_OUT_BETA: (torch.float64,), SLH_OUT_Q: (torch.float64,),
             SLH_OUT_CODES: (torch.int32, torch.uint32)}
    _device_tensor("src", src, kinds.get(which))
    nbytes = src.numel() * src.element_size()
    _check(ctx, load().slh_load(ctx.handle, which, ctypes.c_void_p(src.data_ptr()), nbytes), "slh_load")
    if which == SLH_OUT_ALPHA:
        ctx.n_it = nbytes // (8 * max(1, ctx.n_spectral))


def slh_copy_out(ctx, which):
    dt, shape = _OUT[which]
    a = np.empty(shape(ctx), dt)
    _check(ctx, load().slh_copy_out(ctx.handle, which, _ptr(a), a.nbytes), "slh_copy_out")
    return a


def compress(ctx, X, n_it, rho=None, tau=-1.0, want_ritz=False):
    """The whole path on one prompt: [route] -> feature map -> Lanczos -> SimHash -> merge.

    rho <= 1 is the identity path (the paper's appendix on backends: at a
    compression ratio of at most one the prompt is returned as it is): X itself,
    positions 0..N-1 and the identity token map, with M = N and no library call
    (ctx may then be None)."""
    if rho is not None and rho <= 1.0:
        import torch
        N = X.shape[0]
        pos = torch.arange(N, dtype=torch.int32, device=X.device)
        return X, pos, pos.clone(), N, None
    if rho is not None:
        slh_route(ctx, X, rho, tau)
    slh_feature_map(ctx, X)
    lz = slh_lanczos(ctx, n_it, want=want_ritz)
    slh_simhash(ctx)
    E, P, t2m, M = slh_merge(ctx, X)
    return E, P, t2m, M, lz


def slh_spectral_energy(ctx):
    """Per spectral window: sum of the kept Ritz values / ||Phi_w||_F^2."""
    out = np.empty(ctx.n_spectral, np.float64)
    _check(ctx, load().slh_spectral_energy(ctx.handle, _ptr(out)), "slh_spectral_energy")
    return out


def slh_bucket_purity(ctx, X, thresh=0.7):
    """(pairs with cosine > thresh, pairs) over same-bucket token pairs; X as
    passed to slh_merge."""
    p, dt, ld = _xinfo(X)
    out = np.zeros(2, np.int64)
    _check(ctx, load().slh_bucket_purity(ctx.handle, p, dt, ld, float(thresh), _ptr(out)),
           "slh_bucket_purity")
    return int(out[0]), int(out[1])


def slh_peak_read(buf, reps=20, stream=None):
    """GB/s of a plain streaming read of the device tensor `buf` (measurement aid)."""
    import torch
    _device_tensor("buf", buf)
    st = torch.cuda.current_stream() if stream is None else stream
    out = np.zeros(1, np.float64)
    rc = load().slh_peak_read(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
                              int(reps), ctypes.c_void_p(st.cuda_stream), _ptr(out))
    if rc != SLH_OK:
        raise SLHError(f"slh_peak_read failed ({rc})")
    return float(out[0])


def slh_peak_mfma(reps=10, stream=None):
    """TFLOP/s of independent dense bf16 MFMA chains (measurement aid)."""
    import torch
    st = torch.cuda.current_stream() if stream is None else stream
    sink = torch.empty(4, dtype=torch.float32, device="cuda")
    out = np.zeros(1, np.float64)
    rc = load().slh_peak_mfma(int(reps), ctypes.c_void_p(sink.data_ptr()),
                              ctypes.c_void_p(st.cuda_stream), _ptr(out))
    if rc != SLH_OK:
        raise SLHError(f"slh_peak_mfma failed ({rc})")
    return float(out[0])


def slh_merge_noalloc(X, codes, bits, emb_out, pos_out, tok2macro_out=None, stream=None):
    """The allocation-free merge of one window from given codes (device tensors
    throughout; outputs allocated by the caller).  Returns (E [M, D], P [M],
    tok2macro, M) as views of the given outputs."""
    import torch
    p, dt, ld = _xinfo(X)
    _device_tensor("codes", codes, (torch.int32, torch.uint32), (X.shape[0],), X.device)
    _check_merge_outputs(X.shape[1], X.shape[0], X.device, emb_out, pos_out, tok2macro_out)
    st = torch.cuda.current_stream() if stream is None else stream
    M = ctypes.c_int64(0)
    rc = load().slh_merge_noalloc(p, dt, ld, X.shape[0], X.shape[1], ctypes.c_void_p(codes.data_ptr()),
                                  int(bits), ctypes.c_void_p(emb_out.data_ptr()),
                                  ctypes.c_void_p(pos_out.data_ptr()),
                                  ctypes.c_void_p(tok2macro_out.data_ptr()) if tok2macro_out is not None
                                  else None, emb_out.shape[0], ctypes.byref(M),
                                  ctypes.c_void_p(st.cuda_stream))
    if rc != SLH_OK:
        raise SLHError(f"slh_merge_noalloc failed ({rc})")
    m = int(M.value)
    return emb_out[:m], pos_out[:m], tok2macro_out, m
