"""Thin ctypes binding of libmca (the C ABI in include/mca.h).

Argument marshalling only: torch tensors become device pointers and the
current HIP stream; every step of the forward pass runs in the library's HIP
kernels. There is no fallback: if libmca.so is missing or cannot be loaded,
every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmca.so")

MCA_OK = 0
MCA_ERR_INVALID_ARGUMENT = 1
MCA_ERR_UNSUPPORTED = 2
MCA_ERR_WORKSPACE_TOO_SMALL = 3
MCA_ERR_HIP = 4
MCA_F32 = 0
MCA_BF16 = 1
MCA_SAMPLING_TOKEN = 0   # Eq. 4 per token
MCA_SAMPLING_WEIGHT = 1  # Eq. 6, input independent
SAMPLING = {"token": MCA_SAMPLING_TOKEN, "weight": MCA_SAMPLING_WEIGHT}
MCA_IMPORTANCE_MAX, MCA_IMPORTANCE_MEAN, MCA_IMPORTANCE_MEDIAN = 0, 1, 2
IMPORTANCE = {"max": MCA_IMPORTANCE_MAX, "mean": MCA_IMPORTANCE_MEAN, "median": MCA_IMPORTANCE_MEDIAN}


def _importance_code(rule) -> int:
    if rule not in IMPORTANCE:
        raise ValueError(f"importance must be one of {sorted(IMPORTANCE)} (got {rule!r})")
    return IMPORTANCE[rule]


def _sampling_code(sampling) -> int:
    if sampling not in SAMPLING:
        raise ValueError(f"sampling must be one of {sorted(SAMPLING)} (got {sampling!r})")
    return SAMPLING[sampling]
NUM_STAGES = 5
STAGES = ("scores_colmax", "sample", "gather", "attn_out", "saturated")


class ForwardDesc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int64),
        ("seq", ctypes.c_int64),
        ("heads", ctypes.c_int64),
        ("d_head", ctypes.c_int64),
        ("d_in", ctypes.c_int64),
        ("dtype", ctypes.c_int32),
        ("sampling", ctypes.c_int32),
        ("alpha", ctypes.c_double),
        ("seed", ctypes.c_uint64),
        ("seq_lens", ctypes.c_void_p),
        ("r_in", ctypes.c_void_p),
        ("colmax_out", ctypes.c_void_p),
        ("sample_idx_out", ctypes.c_void_p),
        ("sample_coef_out", ctypes.c_void_p),
        ("encoded_out", ctypes.c_void_p),
        ("profiler", ctypes.c_void_p),
        ("window", ctypes.c_int64),
        ("importance", ctypes.c_int32),
        ("exact_from", ctypes.c_int32),
    ]


class MCAError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)}: {detail}")


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libmca.so (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run paper_2201_12854_amd.build_lib.build() first")
    # torch first: its HIP runtime (same soname as the one libmca.so was linked against)
    # then serves the library too. Loaded the other way round, the process would end up
    # with two HIP runtimes, and the second finds no device.
    import torch  # noqa: F401

    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.mca_prepared_size.argtypes = [i32, i64, i64, ctypes.POINTER(sz)]
    lib.mca_prepared_size.restype = ctypes.c_int
    lib.mca_prepare_weights.argtypes = [vp, i32, i64, i64, vp, sz, vp]
    lib.mca_prepare_weights.restype = ctypes.c_int
    lib.mca_workspace_size.argtypes = [ctypes.POINTER(ForwardDesc), ctypes.POINTER(sz)]
    lib.mca_workspace_size.restype = ctypes.c_int
    lib.mca_attention_forward.argtypes = [ctypes.POINTER(ForwardDesc), vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.mca_attention_forward.restype = ctypes.c_int
    lib.mca_attention_forward_noalloc.argtypes = [ctypes.POINTER(ForwardDesc), vp, vp, vp, vp, vp, vp, vp, vp]
    lib.mca_attention_forward_noalloc.restype = ctypes.c_int
    lib.mca_status_string.argtypes = [ctypes.c_int]
    lib.mca_status_string.restype = ctypes.c_char_p
    lib.mca_last_error.argtypes = []
    lib.mca_last_error.restype = ctypes.c_char_p
    lib.mca_num_stages.argtypes = []
    lib.mca_num_stages.restype = ctypes.c_int
    lib.mca_stage_name.argtypes = [ctypes.c_int]
    lib.mca_stage_name.restype = ctypes.c_char_p
    lib.mca_profiler_create.argtypes = [ctypes.POINTER(vp)]
    lib.mca_profiler_create.restype = ctypes.c_int
    lib.mca_profiler_collect.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64), ctypes.c_int]
    lib.mca_profiler_collect.restype = ctypes.c_int
    lib.mca_profiler_destroy.argtypes = [vp]
    lib.mca_profiler_destroy.restype = ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().mca_status_string(status).decode()


def _check(status: int, where: str):
    if status != MCA_OK:
        raise MCAError(status, where, load_library().mca_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dtype_code(t) -> int:
    import torch

    if t.dtype == torch.float32:
        return MCA_F32
    if t.dtype == torch.bfloat16:
        return MCA_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _stream_handle(device) -> int:
    import torch

    return torch.cuda.current_stream(device).cuda_stream


def make_desc(batch, seq, heads, d_in, dtype_code, alpha, seed, *, seq_lens=None, r_in=None,
              colmax_out=None, sample_idx_out=None, sample_coef_out=None, encoded_out=None,
              profiler=None, sampling=0, window=0, importance=0, exact_from=0) -> ForwardDesc:
    d = ForwardDesc()
    d.batch, d.seq, d.heads, d.d_head, d.d_in = batch, seq, heads, 64, d_in
    d.dtype, d.sampling = dtype_code, sampling
    d.alpha, d.seed = float(alpha), int(seed) & 0xFFFFFFFFFFFFFFFF
    d.seq_lens, d.r_in = _ptr(seq_lens), _ptr(r_in)
    d.colmax_out, d.sample_idx_out = _ptr(colmax_out), _ptr(sample_idx_out)
    d.sample_coef_out, d.encoded_out = _ptr(sample_coef_out), _ptr(encoded_out)
    d.profiler = None if profiler is None else profiler.handle
    d.window = int(window)
    d.importance = int(importance)
    d.exact_from = int(exact_from)
    return d


def workspace_size(desc: ForwardDesc) -> int:
    lib = load_library()
    out = ctypes.c_size_t(0)
    _check(lib.mca_workspace_size(ctypes.byref(desc), ctypes.byref(out)), "mca_workspace_size")
    return out.value


def prepared_size(dtype_code: int, d_in: int, d_out: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().mca_prepared_size(dtype_code, d_in, d_out, ctypes.byref(out)), "mca_prepared_size")
    return out.value


def prepare_weights(W_v, prepared=None):
    """Prepared weights of W_v [d_in, d_out] (a uint8 device buffer): the row norms
    float32 [d_in] at offset 0 (see ``rownorm``) and a transposed copy for the MFMA path."""
    import torch

    lib = load_library()
    if W_v.dim() != 2 or not W_v.is_cuda or not W_v.is_contiguous():
        raise ValueError("W_v must be a contiguous 2-D device tensor [d_in, d_out]")
    nbytes = prepared_size(_dtype_code(W_v), W_v.shape[0], W_v.shape[1])
    if prepared is None:
        prepared = torch.empty(nbytes, dtype=torch.uint8, device=W_v.device)
    _check(lib.mca_prepare_weights(_ptr(W_v), _dtype_code(W_v), W_v.shape[0], W_v.shape[1], _ptr(prepared),
                                   prepared.numel(), _stream_handle(W_v.device)), "mca_prepare_weights")
    return prepared


def rownorm(prepared, d_in: int):
    """The float32 row norms held at the start of a prepared-weights buffer."""
    return prepared[: 4 * d_in].view(dtype=__import__("torch").float32)


@dataclass
class ForwardResult:
    Y: object
    r: object
    colmax: object = None
    sample_idx: object = None
    sample_coef: object = None
    encoded: object = None


MCA_NOALLOC_SCRATCH_BYTES = 64 << 20  # the no-allocation entry's scratch array per device


def attention_forward(Q, K, X, W_v, prepared, alpha: float, seed: int = 0, *, heads: int,
                      seq_lens=None, r_in=None, export: bool = False, export_samples: bool = False,
                      workspace=None, out=None, profiler=None, sampling: str = "token",
                      window: int = 0, importance: str = "max", exact_from: int = 0,
                      noalloc: bool = False) -> ForwardResult:
    """One MCA forward pass through libmca on the current HIP stream.

    Q, K: [B, n, heads*64]; X: [B, n, d_in]; W_v: [d_in, heads*64]; all float32 or
    all bfloat16, contiguous, on one device. ``prepared`` from ``prepare_weights(W_v)``.
    seq_lens: optional int32 [B]. r_in: optional int32 [B, n] overriding the count
    rule. ``export`` also returns the column max and H~ (float32); ``export_samples``
    the per-draw indices and coefficients ([B, n, d_in], first r_j entries valid).
    ``out`` may pass preallocated (Y, r). ``noalloc``: call mca_attention_forward_noalloc,
    whose scratch memory is the library's own device array (no workspace; the outputs are
    still allocated here unless ``out`` passes them). ``sampling``: "token" (Eq. 4, per token) or
    "weight" (Eq. 6, the paper's input-independent probability). ``window``: 0 for full
    attention, or an even local window (keys within window / 2 of each query, plus a
    global first token). ``importance``: "max" (Eq. 8-9), "mean" or "median", the per-key
    statistic of the count rule (full attention). ``exact_from`` > 0: tokens with
    r_j >= exact_from are encoded exactly on MFMA too.
    """
    import torch

    lib = load_library()
    B, n, d_in = X.shape
    d_out = W_v.shape[1]
    dt = _dtype_code(X)
    dev = X.device
    for name, t in (("Q", Q), ("K", K), ("X", X), ("W_v", W_v)):
        if not t.is_cuda or not t.is_contiguous() or t.dtype != X.dtype or t.device != dev:
            raise ValueError(f"{name} must be a contiguous {X.dtype} tensor on {dev}")
    if Q.shape != (B, n, heads * 64) or K.shape != Q.shape or W_v.shape[0] != d_in or d_out != heads * 64:
        raise ValueError("shape mismatch: Q, K [B, n, heads*64], X [B, n, d_in], W_v [d_in, heads*64]")
    if prepared.dtype != torch.uint8 or prepared.device != dev or \
            prepared.numel() < prepared_size(dt, d_in, d_out):
        raise ValueError("prepared must be the uint8 buffer prepare_weights(W_v) returns")
    if seq_lens is not None and (seq_lens.dtype != torch.int32 or seq_lens.shape != (B,)):
        raise ValueError("seq_lens must be int32 [B]")
    if r_in is not None and (r_in.dtype != torch.int32 or r_in.numel() != B * n or not r_in.is_contiguous()):
        raise ValueError("r_in must be a contiguous int32 [B, n]")
    res = ForwardResult(None, None)
    if export:
        res.colmax = torch.empty((B, n), dtype=torch.float32, device=dev)
        res.encoded = torch.empty((B, n, d_out), dtype=torch.float32, device=dev)
    if export_samples:
        res.sample_idx = torch.full((B, n, d_in), -1, dtype=torch.int32, device=dev)
        res.sample_coef = torch.zeros((B, n, d_in), dtype=torch.float32, device=dev)
    desc = make_desc(B, n, heads, d_in, dt, alpha, seed, seq_lens=seq_lens, r_in=r_in,
                     colmax_out=res.colmax, sample_idx_out=res.sample_idx,
                     sample_coef_out=res.sample_coef, encoded_out=res.encoded, profiler=profiler,
                     sampling=_sampling_code(sampling), window=window,
                     importance=_importance_code(importance), exact_from=exact_from)
    if out is None:
        Y = torch.empty((B, n, d_out), dtype=torch.float32, device=dev)
        r = torch.empty((B, n), dtype=torch.int32, device=dev)
    else:
        Y, r = out
    if noalloc:
        _check(lib.mca_attention_forward_noalloc(ctypes.byref(desc), _ptr(Q), _ptr(K), _ptr(X), _ptr(W_v),
                                                 _ptr(prepared), _ptr(Y), _ptr(r), _stream_handle(dev)),
               "mca_attention_forward_noalloc")
    else:
        ws_bytes = workspace_size(desc)
        if workspace is None or workspace.numel() < ws_bytes:
            workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
        _check(lib.mca_attention_forward(ctypes.byref(desc), _ptr(Q), _ptr(K), _ptr(X), _ptr(W_v), _ptr(prepared),
                                         _ptr(Y), _ptr(r), _ptr(workspace), workspace.numel(),
                                         _stream_handle(dev)), "mca_attention_forward")
    res.Y, res.r = Y, r
    return res


class Profiler:
    """Per-stage HIP-event timing of mca_attention_forward calls."""

    def __init__(self):
        lib = load_library()
        h = ctypes.c_void_p()
        _check(lib.mca_profiler_create(ctypes.byref(h)), "mca_profiler_create")
        self.handle = h.value

    def collect(self) -> dict:
        lib = load_library()
        ms = (ctypes.c_double * NUM_STAGES)()
        cnt = (ctypes.c_int64 * NUM_STAGES)()
        _check(lib.mca_profiler_collect(self.handle, ms, cnt, NUM_STAGES), "mca_profiler_collect")
        return {STAGES[i]: (ms[i], cnt[i]) for i in range(NUM_STAGES)}

    def close(self):
        if self.handle:
            load_library().mca_profiler_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class ForwardPlan:
    """A forward call with every argument bound once (tensors, workspace, outputs,
    stream), so that ``run()`` is a single C call: for timing loops and serving."""

    def __init__(self, Q, K, X, W_v, prepared, alpha: float, seed: int = 0, *, heads: int, seq_lens=None,
                 r_in=None, profiler=None, sampling: str = "token", window: int = 0, importance: str = "max",
                 exact_from: int = 0):
        import torch

        lib = load_library()
        B, n, d_in = X.shape
        d_out = W_v.shape[1]
        dev = X.device
        self._keep = (Q, K, X, W_v, prepared, seq_lens, r_in)
        self.desc = make_desc(B, n, heads, d_in, _dtype_code(X), alpha, seed, seq_lens=seq_lens, r_in=r_in,
                              profiler=profiler, sampling=_sampling_code(sampling), window=window,
                              importance=_importance_code(importance), exact_from=exact_from)
        ws = workspace_size(self.desc)
        self.workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=dev)
        self.Y = torch.empty((B, n, d_out), dtype=torch.float32, device=dev)
        self.r = torch.empty((B, n), dtype=torch.int32, device=dev)
        self._fn = lib.mca_attention_forward
        self._args = (ctypes.byref(self.desc), _ptr(Q), _ptr(K), _ptr(X), _ptr(W_v), _ptr(prepared), _ptr(self.Y),
                      _ptr(self.r), _ptr(self.workspace), self.workspace.numel())
        self._stream = _stream_handle(dev)

    def run(self):
        st = self._fn(*self._args, self._stream)
        if st != MCA_OK:
            _check(st, "mca_attention_forward")
