"""Python binding of libgspar (gradient sparsification on MI355X).

Argument marshalling only: every step of the sparsifier runs in the HIP kernels of
``csrc/gspar.hip`` behind the C ABI declared in ``include/gspar.h``; PyTorch provides device
memory and the current stream. There is no CPU fallback: every entry point raises if the
library has not been built (``__graft_entry__.build()`` or ``python -m paper_1710_09854_amd.build``).

Entry points mirror the C ABI:

* ``sparsify_probs(g, rho, solver, iters)``                  -> Probs(p, lam, k, flags)
* ``sparsify_sample_compact(g, rho, seed, solver, iters)``   -> Sparse(idx, val, nnz, lam, k, flags)
* ``sparsify_probs_batched(g2d, rho, solver, iters)``
* ``sparsify_sample_compact_batched(g2d, rho, seeds, ...)``
* ``sparsify_sample_hybrid(g, rho, seed, ...)`` / ``sparsify_sample_hybrid_batched(g2d, rho, seeds, ...)``
  -> Hybrid(idx_a, val_a, n_a, code_b, n_b, inv_lam, q, lam, flags): the Q_A / Q_B coding
* ``coding_bits(d, n_a, n_b, n_b_neg, float_bits)`` -> (sparse lists, ternary entropy, paper formula)
* ``aggregate(idx2d, val2d, nnz, d)`` -> the workers' average (1/M) sum_m Q(g^m) as a dense fp32 vector
* ``Plan``: a preallocated batched sample/compact call for timing loops.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgspar.so")

GREEDY = 0
EXACT = 1
VARIANCE = 2  # the rho arguments then carry the variance budget eps
FLAG_NONFINITE = 1
FLAG_OVERFLOW = 2
FLAG_ALLZERO = 4
FLAG_BADRHO = 8
FLAG_INTERNAL = 16
FLAG_BADSEG = 32

OK = 0
ERR_ARG = -1
ERR_WORKSPACE = -2
ERR_HIP = -3
ERR_TOO_LARGE = -4

INSTR_LIB_PATH = os.path.join(_HERE, "libgspar_instr.so")

_lib = None
_instr = None


def _bind(L):
    """Argument types of the C ABI of include/gspar.h on a loaded library."""
    vp, i64, u64, f64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_int
    L.gspar_workspace_bytes.argtypes = [i64, i64, i32]
    L.gspar_workspace_bytes.restype = ctypes.c_size_t
    L.gspar_capacity_hint.argtypes = [i64, f64]
    L.gspar_capacity_hint.restype = i64
    L.sparsify_probs.argtypes = [vp, i64, f64, i32, i32, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.sparsify_probs.restype = i32
    L.sparsify_sample_compact.argtypes = [vp, i64, f64, i32, i32, u64, vp, vp, i64, vp, vp, vp, vp, vp,
                                          ctypes.c_size_t, vp]
    L.sparsify_sample_compact.restype = i32
    L.sparsify_probs_batched.argtypes = [vp, i64, i64, i64, vp, i32, i32, vp, vp, vp, vp, vp,
                                         ctypes.c_size_t, vp]
    L.sparsify_probs_batched.restype = i32
    L.sparsify_sample_compact_batched.argtypes = [vp, i64, i64, i64, vp, i32, i32, vp, vp, vp, i64, vp, vp,
                                                  vp, vp, vp, ctypes.c_size_t, vp]
    L.sparsify_sample_compact_batched.restype = i32
    L.sparsify_sample_hybrid_batched.argtypes = [vp, i64, i64, i64, vp, i32, i32, vp, vp, vp, i64, vp, vp, i64,
                                                 vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.sparsify_sample_hybrid_batched.restype = i32
    L.sparsify_sample_hybrid.argtypes = [vp, i64, f64, i32, i32, u64, vp, vp, i64, vp, vp, i64, vp, vp, vp, vp, vp,
                                         vp, ctypes.c_size_t, vp]
    L.sparsify_sample_hybrid.restype = i32
    L.gspar_coding_bits.argtypes = [i64, i64, i64, i64, i32, ctypes.POINTER(f64)]
    L.gspar_coding_bits.restype = i32
    L.sparsify_sample_compact_segmented.argtypes = [vp, i64, vp, vp, vp, i32, i32, vp, vp, vp, i64, vp, vp, vp,
                                                    vp, vp, ctypes.c_size_t, vp]
    L.sparsify_sample_compact_segmented.restype = i32
    L.sparsify_probs_segmented.argtypes = [vp, i64, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.sparsify_probs_segmented.restype = i32
    L.sparsify_sample_hybrid_segmented.argtypes = [vp, i64, vp, vp, vp, i32, i32, vp, vp, vp, i64, vp, vp, i64,
                                                   vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.sparsify_sample_hybrid_segmented.restype = i32
    L.sparsify_sample_compact_batched_noalloc.argtypes = [vp, i64, i64, i64, vp, i32, i32, vp, vp, vp, i64, vp,
                                                          vp, vp, vp, vp]
    L.sparsify_sample_compact_batched_noalloc.restype = i32
    L.gspar_aggregate.argtypes = [vp, vp, i64, vp, i64, i64, vp, vp]
    L.gspar_aggregate.restype = i32
    L.gspar_status_string.argtypes = [i32]
    L.gspar_status_string.restype = ctypes.c_char_p
    L.gspar_version.argtypes = []
    L.gspar_version.restype = i32
    return L


def _open(path):
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build the HIP library first "
                           "(python -m paper_1710_09854_amd.build)")
    return _bind(ctypes.CDLL(path))


def lib():
    """The loaded product library (libgspar.so); raises if it was never built."""
    global _lib
    if _lib is None:
        _lib = _open(LIB_PATH)
    return _lib


PROF_CLASSES = ("k_sample", "k_stats", "k_probs", "k_solve", "k_refine", "k_init", "k_aggregate", "k_probs_out",
                "k_presample")


def instr_lib():
    """The measurement build (libgspar_instr.so: the same kernels, plus the launch timer and the
    host-compiled arithmetic checks of include/gspar_instr.h). For the benchmark and the tests."""
    global _instr
    if _instr is None:
        L = _open(INSTR_LIB_PATH)
        i32, f64 = ctypes.c_int, ctypes.c_double
        L.gspar_prof_arm.argtypes = [i32]
        L.gspar_prof_arm.restype = i32
        L.gspar_prof_read.argtypes = [ctypes.POINTER(f64), ctypes.POINTER(i32)]
        L.gspar_prof_read.restype = i32
        L.gspar_prof_disarm.argtypes = []
        L.gspar_prof_disarm.restype = i32
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        L.gspar_probe_stream.argtypes = [vp, vp, i64, vp, vp]
        L.gspar_probe_stream.restype = i32
        _instr = L
    return _instr


def probe_stream(src, dst=None, sink=None, stream=None):
    """The measurement build's stream probe on the current stream: reads src (fp32, contiguous,
    on the device) and adds its sum into sink (a one-element float64 device tensor), or copies it
    into dst. For bandwidth comparisons only."""
    import torch

    L = instr_lib()
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    rc = L.gspar_probe_stream(src.data_ptr(), dst.data_ptr() if dst is not None else None, src.numel(),
                              sink.data_ptr() if sink is not None else None, s)
    _check(rc, "gspar_probe_stream")


def _solver_id(solver) -> int:
    if solver in ("greedy", GREEDY):
        return GREEDY
    if solver in ("exact", EXACT):
        return EXACT
    if solver in ("variance", VARIANCE):
        return VARIANCE
    raise ValueError(f"unknown solver {solver!r}")


def _check(rc: int, what: str):
    if rc != OK:
        msg = lib().gspar_status_string(rc).decode()
        raise RuntimeError(f"{what} failed: {msg} ({rc})")


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def workspace_bytes(rows: int, d: int, solver="greedy") -> int:
    return int(lib().gspar_workspace_bytes(rows, d, _solver_id(solver)))


def capacity_hint(d: int, rho: float) -> int:
    return int(lib().gspar_capacity_hint(d, rho))


def _default_cap(d: int, rho: float, solver) -> int:
    """Output capacity per row when the caller gives none: from the density, or every coordinate
    for the variance budget (its survivor count is not known before the solve)."""
    if _solver_id(solver) == VARIANCE:
        return int(d)
    return capacity_hint(d, min(max(float(rho), 0.0), 1.0))


class Workspace:
    """Grow-only device workspace (the library itself never allocates). Calls that share one must
    be ordered on one stream; the buffer is allocated on that stream, so a buffer dropped when the
    workspace grows is reused by the caching allocator only after the stream's earlier work."""

    def __init__(self, device=None, stream=None):
        self.device = torch.device("cuda" if device is None else device)
        self.stream = stream
        self.buf = None

    def get(self, nbytes: int) -> torch.Tensor:
        if self.buf is None or self.buf.numel() < nbytes:
            if self.stream is None:
                self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
            else:
                with torch.cuda.stream(self.stream):
                    self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        return self.buf


_default_ws: dict = {}


def _ws(ws, device, nbytes, stream=None):
    """The caller's workspace, or the default one of (device, stream): calls on different streams
    never share a default workspace."""
    if ws is None:
        dev = torch.device(device)
        idx = dev.index if dev.index is not None else torch.cuda.current_device()
        s = torch.cuda.current_stream(idx) if stream is None else stream
        key = (idx, s.cuda_stream)
        if key not in _default_ws:
            _default_ws[key] = Workspace(torch.device("cuda", idx), s)
        ws = _default_ws[key]
    buf = ws.get(nbytes)
    return buf, buf.numel()


def _as_row(g):
    if not (isinstance(g, torch.Tensor) and g.is_cuda and g.dtype == torch.float32):
        raise TypeError("g must be a float32 CUDA tensor")
    if g.dim() != 1 or not g.is_contiguous():
        raise ValueError("g must be a contiguous 1-D tensor")
    return g


def _as_rows(g):
    if not (isinstance(g, torch.Tensor) and g.is_cuda and g.dtype == torch.float32):
        raise TypeError("g must be a float32 CUDA tensor")
    if g.dim() != 2 or (g.stride(1) != 1 and g.shape[1] > 1):
        raise ValueError("g must be 2-D with unit stride along a row")
    return g


def _leading_dim(g) -> int:
    """Row pitch in elements; a single row's stride is irrelevant (size-1 dimensions may report
    any stride, including 0)."""
    rows, d = g.shape
    return d if rows == 1 else g.stride(0)


@dataclass
class Probs:
    p: torch.Tensor | None
    lam: torch.Tensor
    k: torch.Tensor
    flags: torch.Tensor


@dataclass
class Sparse:
    idx: torch.Tensor
    val: torch.Tensor
    nnz: torch.Tensor
    lam: torch.Tensor
    k: torch.Tensor
    flags: torch.Tensor


def sparsify_probs(g, rho: float, solver="greedy", iters: int = 2, want_p: bool = True, workspace=None,
                   stream=None) -> Probs:
    g = _as_row(g)
    d = g.numel()
    dev = g.device
    p = torch.empty(d, dtype=torch.float32, device=dev) if want_p else None
    lam = torch.empty(1, dtype=torch.float64, device=dev)
    k = torch.empty(1, dtype=torch.int64, device=dev)
    fl = torch.empty(1, dtype=torch.int32, device=dev)
    sid = _solver_id(solver)
    buf, nb = _ws(workspace, dev, workspace_bytes(1, d, sid), stream)
    rc = lib().sparsify_probs(g.data_ptr(), d, float(rho), sid, int(iters), _ptr(p), lam.data_ptr(),
                              k.data_ptr(), fl.data_ptr(), buf.data_ptr(), nb, _stream(stream))
    _check(rc, "sparsify_probs")
    return Probs(p, lam, k, fl)


def sparsify_sample_compact(g, rho: float, seed: int = 0, solver="greedy", iters: int = 2,
                            capacity: int | None = None, workspace=None, stream=None) -> Sparse:
    g = _as_row(g)
    d = g.numel()
    dev = g.device
    cap = _default_cap(d, rho, solver) if capacity is None else int(capacity)
    idx = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    val = torch.empty(max(cap, 1), dtype=torch.float32, device=dev)
    nnz = torch.empty(1, dtype=torch.int64, device=dev)
    lam = torch.empty(1, dtype=torch.float64, device=dev)
    k = torch.empty(1, dtype=torch.int64, device=dev)
    fl = torch.empty(1, dtype=torch.int32, device=dev)
    sid = _solver_id(solver)
    buf, nb = _ws(workspace, dev, workspace_bytes(1, d, sid), stream)
    rc = lib().sparsify_sample_compact(g.data_ptr(), d, float(rho), sid, int(iters),
                                       int(seed) & 0xFFFFFFFFFFFFFFFF, idx.data_ptr(), val.data_ptr(), cap,
                                       nnz.data_ptr(), lam.data_ptr(), k.data_ptr(), fl.data_ptr(),
                                       buf.data_ptr(), nb, _stream(stream))
    _check(rc, "sparsify_sample_compact")
    return Sparse(idx[:cap], val[:cap], nnz, lam, k, fl)


@dataclass
class Hybrid:
    """Section 3.3's coding: Q_A = (idx_a, val_a) for the capped survivors (n_a of them), Q_B =
    code_b words (index | sign << 31) for the others (n_b), whose value is sign / lambda; inv_lam
    is the fp32 1/lambda they share; q the optional dense ternary vector (2, +-1 or 0)."""
    idx_a: torch.Tensor
    val_a: torch.Tensor
    n_a: torch.Tensor
    code_b: torch.Tensor
    n_b: torch.Tensor
    inv_lam: torch.Tensor
    q: torch.Tensor | None
    lam: torch.Tensor
    flags: torch.Tensor


def sparsify_sample_hybrid(g, rho: float, seed: int = 0, solver="greedy", iters: int = 2,
                           cap_a: int | None = None, cap_b: int | None = None, dense_q: bool = False,
                           workspace=None, stream=None) -> Hybrid:
    g = _as_row(g)
    d = g.numel()
    dev = g.device
    cap_b = _default_cap(d, rho, solver) if cap_b is None else int(cap_b)
    cap_a = cap_b if cap_a is None else int(cap_a)
    idx_a = torch.empty(max(cap_a, 1), dtype=torch.int32, device=dev)
    val_a = torch.empty(max(cap_a, 1), dtype=torch.float32, device=dev)
    code_b = torch.empty(max(cap_b, 1), dtype=torch.int32, device=dev)
    n_a = torch.empty(1, dtype=torch.int64, device=dev)
    n_b = torch.empty(1, dtype=torch.int64, device=dev)
    inv = torch.empty(1, dtype=torch.float32, device=dev)
    q = torch.empty(d, dtype=torch.int8, device=dev) if dense_q else None
    lam = torch.empty(1, dtype=torch.float64, device=dev)
    fl = torch.empty(1, dtype=torch.int32, device=dev)
    sid = _solver_id(solver)
    buf, nb = _ws(workspace, dev, workspace_bytes(1, d, sid), stream)
    rc = lib().sparsify_sample_hybrid(g.data_ptr(), d, float(rho), sid, int(iters), int(seed) & 0xFFFFFFFFFFFFFFFF,
                                      idx_a.data_ptr(), val_a.data_ptr(), cap_a, n_a.data_ptr(), code_b.data_ptr(),
                                      cap_b, n_b.data_ptr(), inv.data_ptr(), _ptr(q), lam.data_ptr(), fl.data_ptr(),
                                      buf.data_ptr(), nb, _stream(stream))
    _check(rc, "sparsify_sample_hybrid")
    return Hybrid(idx_a[:cap_a], val_a[:cap_a], n_a, code_b[:cap_b], n_b, inv, q, lam, fl)


def sparsify_sample_hybrid_batched(g, rho, seeds, solver="greedy", iters: int = 2, cap_a: int | None = None,
                                   cap_b: int | None = None, dense_q: bool = False, workspace=None,
                                   stream=None) -> Hybrid:
    g = _as_rows(g)
    rows, d = g.shape
    ld = _leading_dim(g)
    dev = g.device
    r = _rho_dev(rho, rows, dev)
    s = _seeds_dev(seeds, rows, dev)
    if cap_b is None:
        rmax = float(r.max().item()) if rows else 0.0
        cap_b = _default_cap(d, rmax, solver)
    cap_b = int(cap_b)
    cap_a = cap_b if cap_a is None else int(cap_a)
    idx_a = torch.empty((rows, max(cap_a, 1)), dtype=torch.int32, device=dev)
    val_a = torch.empty((rows, max(cap_a, 1)), dtype=torch.float32, device=dev)
    code_b = torch.empty((rows, max(cap_b, 1)), dtype=torch.int32, device=dev)
    n_a = torch.empty(rows, dtype=torch.int64, device=dev)
    n_b = torch.empty(rows, dtype=torch.int64, device=dev)
    inv = torch.empty(rows, dtype=torch.float32, device=dev)
    q = torch.empty((rows, ld), dtype=torch.int8, device=dev) if dense_q else None
    lam = torch.empty(rows, dtype=torch.float64, device=dev)
    fl = torch.empty(rows, dtype=torch.int32, device=dev)
    sid = _solver_id(solver)
    buf, nb = _ws(workspace, dev, workspace_bytes(rows, d, sid), stream)
    rc = lib().sparsify_sample_hybrid_batched(g.data_ptr(), rows, d, ld, r.data_ptr(), sid, int(iters), s.data_ptr(),
                                              idx_a.data_ptr(), val_a.data_ptr(), cap_a, n_a.data_ptr(),
                                              code_b.data_ptr(), cap_b, n_b.data_ptr(), inv.data_ptr(), _ptr(q),
                                              lam.data_ptr(), fl.data_ptr(), buf.data_ptr(), nb, _stream(stream))
    _check(rc, "sparsify_sample_hybrid_batched")
    return Hybrid(idx_a[:, :cap_a], val_a[:, :cap_a], n_a, code_b[:, :cap_b], n_b, inv,
                  None if q is None else q[:, :d], lam, fl)


def coding_bits(d: int, n_a: int, n_b: int, n_b_neg: int, float_bits: int = 32):
    """(sparse lists, entropy-coded ternary vector, the experiments' formula) in bits for one hybrid
    message; see gspar_coding_bits in include/gspar.h."""
    out = (ctypes.c_double * 3)()
    rc = lib().gspar_coding_bits(int(d), int(n_a), int(n_b), int(n_b_neg), int(float_bits), out)
    _check(rc, "gspar_coding_bits")
    return out[0], out[1], out[2]


def aggregate(idx, val, nnz, d: int, out=None, stream=None, library=None) -> torch.Tensor:
    """Algorithm 1, step 6: v = (1/M) sum_m Q(g^m), dense fp32 [d], from M workers' ascending
    (index, value) lists (rows of idx / val, the first nnz[m] entries of row m)."""
    if idx.dim() != 2 or val.shape != idx.shape or idx.dtype != torch.int32 or val.dtype != torch.float32:
        raise ValueError("idx / val must be [workers, cap] int32 / float32")
    if not (idx.is_contiguous() and val.is_contiguous()):
        raise ValueError("idx / val must be contiguous")
    workers, cap = idx.shape
    dev = idx.device
    n = nnz.to(device=dev, dtype=torch.int64).contiguous()
    v = torch.empty(d, dtype=torch.float32, device=dev) if out is None else out
    L = lib() if library is None else library
    rc = L.gspar_aggregate(idx.data_ptr(), val.data_ptr(), cap, n.data_ptr(), workers, int(d), v.data_ptr(),
                               _stream(stream))
    _check(rc, "gspar_aggregate")
    return v


def _rho_dev(rho, rows, dev):
    if isinstance(rho, torch.Tensor):
        r = rho.to(device=dev, dtype=torch.float64).contiguous()
    else:
        if isinstance(rho, (int, float)):
            rho = [float(rho)] * rows
        r = torch.tensor(list(rho), dtype=torch.float64, device=dev)
    if r.numel() != rows:
        raise ValueError("rho needs one value per row")
    return r


def _seeds_dev(seeds, rows, dev):
    if isinstance(seeds, torch.Tensor):
        s = seeds.to(device=dev, dtype=torch.int64).contiguous()
    else:
        vals = [int(x) & 0xFFFFFFFFFFFFFFFF for x in seeds]
        vals = [v - (1 << 64) if v >= (1 << 63) else v for v in vals]  # same 64 bits, signed view
        s = torch.tensor(vals, dtype=torch.int64, device=dev)
    if s.numel() != rows:
        raise ValueError("seeds need one value per row")
    return s


def sparsify_probs_batched(g, rho, solver="greedy", iters: int = 2, want_p: bool = True, workspace=None,
                           stream=None) -> Probs:
    g = _as_rows(g)
    rows, d = g.shape
    ld = _leading_dim(g)
    dev = g.device
    r = _rho_dev(rho, rows, dev)
    p = torch.empty((rows, ld), dtype=torch.float32, device=dev) if want_p else None
    lam = torch.empty(rows, dtype=torch.float64, device=dev)
    k = torch.empty(rows, dtype=torch.int64, device=dev)
    fl = torch.empty(rows, dtype=torch.int32, device=dev)
    sid = _solver_id(solver)
    buf, nb = _ws(workspace, dev, workspace_bytes(rows, d, sid), stream)
    rc = lib().sparsify_probs_batched(g.data_ptr(), rows, d, ld, r.data_ptr(), sid, int(iters), _ptr(p),
                                      lam.data_ptr(), k.data_ptr(), fl.data_ptr(), buf.data_ptr(), nb,
                                      _stream(stream))
    _check(rc, "sparsify_probs_batched")
    return Probs(None if p is None else p[:, :d], lam, k, fl)


class Plan:
    """Preallocated batched solve + sample + compact (or, with probs=True, the probabilities
    entry point): inputs, outputs and workspace stay resident, so a timing loop measures only the
    library's kernels."""

    def __init__(self, rows: int, d: int, ld: int | None = None, solver="greedy", iters: int = 2,
                 cap_per_row: int | None = None, rho_for_cap: float = 1.0, device="cuda", hybrid: bool = False,
                 dense_q: bool = False, segments: "Segments | None" = None, library=None, probs: bool = False):
        # with segments: one output row per segment (rows and d are then the segment count and the
        # longest segment); `library`: the loaded library to call (default the product library;
        # the benchmark's timing loop passes the measurement build)
        self.L = lib() if library is None else library
        self.seg = segments
        if segments is not None:
            if hybrid:
                raise ValueError("segmented calls write the compaction output")
            rows, d = segments.segs, segments.max_len
        self.rows, self.d = rows, d
        self.ld = d if ld is None else ld
        self.sid = _solver_id(solver)
        self.iters = int(iters)
        self.cap = _default_cap(d, rho_for_cap, solver) if cap_per_row is None else int(cap_per_row)
        self.hybrid = bool(hybrid)
        self.probs = bool(probs)
        dev = torch.device(device)
        if self.probs:
            if hybrid:
                raise ValueError("the probabilities entry point has no hybrid output")
            self.cap = 0
            self.p = torch.empty(segments.total if segments is not None else (rows, self.ld), dtype=torch.float32,
                                 device=dev)
        # compaction: (idx, val) per survivor; hybrid coding: Q_A in (idx, val), Q_B in code_b
        self.idx = torch.empty((rows, max(self.cap, 1)), dtype=torch.int32, device=dev)
        self.val = torch.empty((rows, max(self.cap, 1)), dtype=torch.float32, device=dev)
        self.nnz = torch.empty(rows, dtype=torch.int64, device=dev)
        self.lam = torch.empty(rows, dtype=torch.float64, device=dev)
        self.k = torch.empty(rows, dtype=torch.int64, device=dev)
        self.flags = torch.empty(rows, dtype=torch.int32, device=dev)
        self.ws = torch.empty(workspace_bytes(rows, d, self.sid), dtype=torch.uint8, device=dev)
        if self.hybrid:
            self.code_b = torch.empty((rows, max(self.cap, 1)), dtype=torch.int32, device=dev)
            self.nnz_b = torch.empty(rows, dtype=torch.int64, device=dev)
            self.inv = torch.empty(rows, dtype=torch.float32, device=dev)
            self.q = torch.empty((rows, self.ld), dtype=torch.int8, device=dev) if dense_q else None

    def run(self, g, rho_dev, seeds_dev, stream=None):
        if self.probs:
            if self.seg is not None:
                rc = self.L.sparsify_probs_segmented(
                    g.data_ptr(), self.rows, self.seg.host.data_ptr(), self.seg.dev.data_ptr(), rho_dev.data_ptr(),
                    self.sid, self.iters, self.p.data_ptr(), self.lam.data_ptr(), self.k.data_ptr(),
                    self.flags.data_ptr(), self.ws.data_ptr(), self.ws.numel(), _stream(stream))
            else:
                rc = self.L.sparsify_probs_batched(
                    g.data_ptr(), self.rows, self.d, self.ld, rho_dev.data_ptr(), self.sid, self.iters,
                    self.p.data_ptr(), self.lam.data_ptr(), self.k.data_ptr(), self.flags.data_ptr(),
                    self.ws.data_ptr(), self.ws.numel(), _stream(stream))
            _check(rc, "sparsify_probs")
            return
        if self.seg is not None:
            rc = self.L.sparsify_sample_compact_segmented(
                g.data_ptr(), self.rows, self.seg.host.data_ptr(), self.seg.dev.data_ptr(), rho_dev.data_ptr(),
                self.sid, self.iters, seeds_dev.data_ptr(), self.idx.data_ptr(), self.val.data_ptr(), self.cap,
                self.nnz.data_ptr(), self.lam.data_ptr(), self.k.data_ptr(), self.flags.data_ptr(),
                self.ws.data_ptr(), self.ws.numel(), _stream(stream))
            _check(rc, "sparsify_sample_compact_segmented")
            return
        if self.hybrid:
            rc = self.L.sparsify_sample_hybrid_batched(
                g.data_ptr(), self.rows, self.d, self.ld, rho_dev.data_ptr(), self.sid, self.iters,
                seeds_dev.data_ptr(), self.idx.data_ptr(), self.val.data_ptr(), self.cap, self.nnz.data_ptr(),
                self.code_b.data_ptr(), self.cap, self.nnz_b.data_ptr(), self.inv.data_ptr(), _ptr(self.q),
                self.lam.data_ptr(), self.flags.data_ptr(), self.ws.data_ptr(), self.ws.numel(), _stream(stream))
            _check(rc, "sparsify_sample_hybrid_batched")
            return
        rc = self.L.sparsify_sample_compact_batched(
            g.data_ptr(), self.rows, self.d, self.ld, rho_dev.data_ptr(), self.sid, self.iters,
            seeds_dev.data_ptr(), self.idx.data_ptr(), self.val.data_ptr(), self.cap, self.nnz.data_ptr(),
            self.lam.data_ptr(), self.k.data_ptr(), self.flags.data_ptr(), self.ws.data_ptr(),
            self.ws.numel(), _stream(stream))
        _check(rc, "sparsify_sample_compact_batched")

    def survivors_and_bytes(self):
        """(survivors, output bytes) of the last run, summed over rows (host sync); for the
        probabilities entry point (capped coordinates, the 4 B per coordinate of p)."""
        if self.probs:
            n = self.seg.total if self.seg is not None else self.rows * self.d
            return int(self.k.sum().item()), 4 * n
        if self.hybrid:
            na, nb = int(self.nnz.sum().item()), int(self.nnz_b.sum().item())
            qb = self.rows * self.d if self.q is not None else 0
            return na + nb, 8 * na + 4 * nb + qb
        n = int(self.nnz.sum().item())
        return n, 8 * n


def sparsify_sample_compact_batched(g, rho, seeds, solver="greedy", iters: int = 2,
                                    cap_per_row: int | None = None, workspace=None, stream=None) -> Sparse:
    g = _as_rows(g)
    rows, d = g.shape
    ld = _leading_dim(g)
    dev = g.device
    r = _rho_dev(rho, rows, dev)
    s = _seeds_dev(seeds, rows, dev)
    if cap_per_row is None:
        rmax = float(r.max().item()) if rows else 0.0
        cap_per_row = _default_cap(d, rmax, solver)
    cap = int(cap_per_row)
    idx = torch.empty((rows, max(cap, 1)), dtype=torch.int32, device=dev)
    val = torch.empty((rows, max(cap, 1)), dtype=torch.float32, device=dev)
    nnz = torch.empty(rows, dtype=torch.int64, device=dev)
    lam = torch.empty(rows, dtype=torch.float64, device=dev)
    k = torch.empty(rows, dtype=torch.int64, device=dev)
    fl = torch.empty(rows, dtype=torch.int32, device=dev)
    sid = _solver_id(solver)
    buf, nb = _ws(workspace, dev, workspace_bytes(rows, d, sid), stream)
    rc = lib().sparsify_sample_compact_batched(g.data_ptr(), rows, d, ld, r.data_ptr(), sid, int(iters),
                                               s.data_ptr(), idx.data_ptr(), val.data_ptr(), cap, nnz.data_ptr(),
                                               lam.data_ptr(), k.data_ptr(), fl.data_ptr(), buf.data_ptr(), nb,
                                               _stream(stream))
    _check(rc, "sparsify_sample_compact_batched")
    return Sparse(idx[:, :cap], val[:, :cap], nnz, lam, k, fl)


def sparsify_sample_compact_batched_noalloc(g, rho_dev, seeds_dev, idx, val, nnz, lam=None, k=None, flags=None,
                                            solver="greedy", iters: int = 2, stream=None):
    """The no-allocation entry point: every argument is a preallocated device tensor (rho_dev
    [rows] float64, seeds_dev [rows] int64, idx / val [rows, cap], nnz [rows], optional lam, k,
    flags [rows]); the library uses its own fixed scratch array instead of a workspace and
    allocates nothing. Returns the status code (OK, or ERR_TOO_LARGE when the call does not fit
    the array)."""
    g = _as_rows(g)
    rows, d = g.shape
    cap = idx.shape[1]
    if val.shape != idx.shape or idx.dtype != torch.int32 or val.dtype != torch.float32:
        raise ValueError("idx / val must be [rows, cap] int32 / float32")
    if rho_dev.dtype != torch.float64 or seeds_dev.dtype != torch.int64:
        raise ValueError("rho_dev must be float64 and seeds_dev int64 device tensors")
    return int(lib().sparsify_sample_compact_batched_noalloc(
        g.data_ptr(), rows, d, _leading_dim(g), rho_dev.data_ptr(), _solver_id(solver), int(iters),
        seeds_dev.data_ptr(), idx.data_ptr(), val.data_ptr(), cap, nnz.data_ptr(), _ptr(lam), _ptr(k), _ptr(flags),
        _stream(stream)))


class Segments:
    """Offsets of the segments (layers) of a flat gradient, kept on the host and on the device:
    segment s is g[off[s]:off[s+1]]."""

    def __init__(self, offsets, device="cuda"):
        self.host = torch.as_tensor(offsets, dtype=torch.int64, device="cpu").contiguous().clone()
        if self.host.dim() != 1 or self.host.numel() < 2:
            raise ValueError("offsets need at least two entries")
        self.dev = self.host.to(torch.device(device))
        self.segs = self.host.numel() - 1
        self.max_len = max(1, int((self.host[1:] - self.host[:-1]).max().item()))
        self.total = int(self.host[-1].item())

    @classmethod
    def from_lengths(cls, lengths, device="cuda"):
        lens = torch.as_tensor(lengths, dtype=torch.int64, device="cpu")
        return cls(torch.cat([torch.zeros(1, dtype=torch.int64), torch.cumsum(lens, 0)]), device)


def _flat(g, seg: Segments):
    g = _as_row(g)
    if g.numel() < seg.total:
        raise ValueError("g is shorter than the last segment offset")
    return g


def sparsify_sample_compact_segmented(g, seg: Segments, rho, seeds, solver="greedy", iters: int = 2,
                                      cap_per_seg: int | None = None, workspace=None, stream=None) -> Sparse:
    """Per-layer sparsification: every segment of the flat gradient g gets its own lambda, density
    and Philox key; row s of the outputs holds segment s's survivors, indexed within the segment."""
    g = _flat(g, seg)
    dev = g.device
    rows = seg.segs
    r = _rho_dev(rho, rows, dev)
    s = _seeds_dev(seeds, rows, dev)
    if cap_per_seg is None:
        rmax = float(r.max().item())
        cap_per_seg = _default_cap(seg.max_len, rmax, solver)
    cap = int(cap_per_seg)
    idx = torch.empty((rows, max(cap, 1)), dtype=torch.int32, device=dev)
    val = torch.empty((rows, max(cap, 1)), dtype=torch.float32, device=dev)
    nnz = torch.empty(rows, dtype=torch.int64, device=dev)
    lam = torch.empty(rows, dtype=torch.float64, device=dev)
    k = torch.empty(rows, dtype=torch.int64, device=dev)
    fl = torch.empty(rows, dtype=torch.int32, device=dev)
    sid = _solver_id(solver)
    buf, nb = _ws(workspace, dev, workspace_bytes(rows, seg.max_len, sid), stream)
    rc = lib().sparsify_sample_compact_segmented(g.data_ptr(), rows, seg.host.data_ptr(), seg.dev.data_ptr(),
                                                 r.data_ptr(), sid, int(iters), s.data_ptr(), idx.data_ptr(),
                                                 val.data_ptr(), cap, nnz.data_ptr(), lam.data_ptr(), k.data_ptr(),
                                                 fl.data_ptr(), buf.data_ptr(), nb, _stream(stream))
    _check(rc, "sparsify_sample_compact_segmented")
    return Sparse(idx[:, :cap], val[:, :cap], nnz, lam, k, fl)


def sparsify_sample_hybrid_segmented(g, seg: Segments, rho, seeds, solver="greedy", iters: int = 2,
                                     cap_a: int | None = None, cap_b: int | None = None, dense_q: bool = False,
                                     workspace=None, stream=None) -> Hybrid:
    """Per-layer hybrid coding: row s of the outputs holds segment s's Q_A and Q_B; q (optional)
    has g's flat layout."""
    g = _flat(g, seg)
    dev = g.device
    rows = seg.segs
    r = _rho_dev(rho, rows, dev)
    s = _seeds_dev(seeds, rows, dev)
    if cap_b is None:
        rmax = float(r.max().item())
        cap_b = _default_cap(seg.max_len, rmax, solver)
    cap_b = int(cap_b)
    cap_a = cap_b if cap_a is None else int(cap_a)
    idx_a = torch.empty((rows, max(cap_a, 1)), dtype=torch.int32, device=dev)
    val_a = torch.empty((rows, max(cap_a, 1)), dtype=torch.float32, device=dev)
    code_b = torch.empty((rows, max(cap_b, 1)), dtype=torch.int32, device=dev)
    n_a = torch.empty(rows, dtype=torch.int64, device=dev)
    n_b = torch.empty(rows, dtype=torch.int64, device=dev)
    inv = torch.empty(rows, dtype=torch.float32, device=dev)
    q = torch.zeros(seg.total, dtype=torch.int8, device=dev) if dense_q else None
    lam = torch.empty(rows, dtype=torch.float64, device=dev)
    fl = torch.empty(rows, dtype=torch.int32, device=dev)
    sid = _solver_id(solver)
    buf, nb = _ws(workspace, dev, workspace_bytes(rows, seg.max_len, sid), stream)
    rc = lib().sparsify_sample_hybrid_segmented(g.data_ptr(), rows, seg.host.data_ptr(), seg.dev.data_ptr(),
                                                r.data_ptr(), sid, int(iters), s.data_ptr(), idx_a.data_ptr(),
                                                val_a.data_ptr(), cap_a, n_a.data_ptr(), code_b.data_ptr(), cap_b,
                                                n_b.data_ptr(), inv.data_ptr(), _ptr(q), lam.data_ptr(),
                                                fl.data_ptr(), buf.data_ptr(), nb, _stream(stream))
    _check(rc, "sparsify_sample_hybrid_segmented")
    return Hybrid(idx_a[:, :cap_a], val_a[:, :cap_a], n_a, code_b[:, :cap_b], n_b, inv, q, lam, fl)


def sparsify_probs_segmented(g, seg: Segments, rho, solver="greedy", iters: int = 2, want_p: bool = True,
                             workspace=None, stream=None) -> Probs:
    """Per-layer probabilities: p in g's flat layout, lambda / k / flags per segment."""
    g = _flat(g, seg)
    dev = g.device
    rows = seg.segs
    r = _rho_dev(rho, rows, dev)
    p = torch.zeros(seg.total, dtype=torch.float32, device=dev) if want_p else None
    lam = torch.empty(rows, dtype=torch.float64, device=dev)
    k = torch.empty(rows, dtype=torch.int64, device=dev)
    fl = torch.empty(rows, dtype=torch.int32, device=dev)
    sid = _solver_id(solver)
    buf, nb = _ws(workspace, dev, workspace_bytes(rows, seg.max_len, sid), stream)
    rc = lib().sparsify_probs_segmented(g.data_ptr(), rows, seg.host.data_ptr(), seg.dev.data_ptr(), r.data_ptr(),
                                        sid, int(iters), _ptr(p), lam.data_ptr(), k.data_ptr(), fl.data_ptr(),
                                        buf.data_ptr(), nb, _stream(stream))
    _check(rc, "sparsify_probs_segmented")
    return Probs(p, lam, k, fl)


class KernelProfiler:
    """Kernel times per class from the measurement build (libgspar_instr.so): every launch made
    through that library while armed carries HIP start / stop events stamped by its dispatch.
    ``read()`` returns {class name: (total ms, launches)}; ``close()`` disarms."""

    def __init__(self, max_launches: int):
        self.L = instr_lib()
        _check(self.L.gspar_prof_arm(int(max_launches)), "gspar_prof_arm")

    def read(self):
        n = len(PROF_CLASSES)
        ms = (ctypes.c_double * n)()
        cnt = (ctypes.c_int * n)()
        _check(self.L.gspar_prof_read(ms, cnt), "gspar_prof_read")
        return {name: (ms[i], cnt[i]) for i, name in enumerate(PROF_CLASSES)}

    def close(self):
        self.L.gspar_prof_disarm()
