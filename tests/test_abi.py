"""CPU checks of the C-ABI library: it loads, exports every declared symbol, rejects bad
arguments before enqueuing anything, and its host-compiled arithmetic building blocks (exact
accumulator rounding, capped-threshold search, Philox) are right. No GPU is touched: every
sparsify_* call here carries an argument error, which the library reports before any HIP call."""
import fractions
import math
import os
import re

import numpy as np
import pytest

import ctypes
import shutil
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gspar.h")


@pytest.fixture(scope="module")
def L():
    import paper_1710_09854_amd as gs

    if not (os.path.exists(gs.LIB_PATH) and os.path.exists(gs.INSTR_LIB_PATH)):
        from paper_1710_09854_amd import build

        build.build()
    return gs.lib()


@pytest.fixture(scope="module")
def LI(L):
    """The measurement build: the same source with the host-compiled arithmetic checks."""
    import paper_1710_09854_amd as gs

    return gs.instr_lib()


def declared_functions(header=HEADER):
    src = open(header).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = "\n".join(l for l in src.splitlines() if not l.lstrip().startswith("#"))  # preprocessor lines
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", src)))


def exported_functions(path):
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True, check=True).stdout
    return sorted(line.split()[-1] for line in out.splitlines() if line.strip())


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert "sparsify_probs" in names and "sparsify_sample_compact_batched" in names
    for n in names:
        assert hasattr(L, n), f"symbol {n} declared in gspar.h is not exported"


@pytest.mark.skipif(not shutil.which("nm"), reason="needs nm")
def test_exports_are_exactly_the_header(L):
    """The product library exports the functions of gspar.h and nothing else (no kernel handles,
    no measurement hooks); the measurement build adds exactly gspar_instr.h's."""
    import paper_1710_09854_amd as gs

    assert exported_functions(gs.LIB_PATH) == declared_functions()
    instr = sorted(declared_functions() + declared_functions(os.path.join(ROOT, "include", "gspar_instr.h")))
    assert exported_functions(gs.INSTR_LIB_PATH) == instr


def test_workspace_and_capacity(L):
    assert L.gspar_workspace_bytes(0, 10, 0) == 0
    a = L.gspar_workspace_bytes(1, 65536, 0)
    b = L.gspar_workspace_bytes(16, 1 << 20, 0)
    assert a > 0 and b > a and b % 256 == 0
    assert L.gspar_capacity_hint(1000, 0.1) == min(1000, math.ceil(100 + 8 * 10 + 64))
    assert L.gspar_capacity_hint(100, 0.9) == 100
    assert L.gspar_capacity_hint(100, 1.5) == 0
    assert L.gspar_version() >= 100


FAKE = 0x10000  # a non-null, 256-aligned address that is never dereferenced


def _sc(L, g=FAKE, d=1000, rho=0.1, solver=0, iters=2, idx=FAKE, val=FAKE, cap=10, nnz=FAKE, ws=FAKE, wsb=None):
    if wsb is None:
        wsb = L.gspar_workspace_bytes(1, max(d, 1), 0)
    return L.sparsify_sample_compact(g, d, rho, solver, iters, 0, idx, val, cap, nnz, None, None, None, ws, wsb, None)


def test_argument_errors(L):
    import paper_1710_09854_amd as gs

    assert _sc(L, g=None) == gs.ERR_ARG
    assert _sc(L, d=0) == gs.ERR_ARG
    assert _sc(L, d=(1 << 31)) == gs.ERR_ARG
    assert _sc(L, rho=-0.1) == gs.ERR_ARG
    assert _sc(L, rho=1.5) == gs.ERR_ARG
    assert _sc(L, rho=float("nan")) == gs.ERR_ARG
    assert _sc(L, solver=3) == gs.ERR_ARG
    # the variance-budget solver takes any finite eps >= 0 in place of rho
    assert _sc(L, solver=2, rho=-0.1) == gs.ERR_ARG
    assert _sc(L, solver=2, rho=float("inf")) == gs.ERR_ARG
    assert _sc(L, solver=2, rho=float("nan")) == gs.ERR_ARG
    assert _sc(L, solver=2, rho=5.0, ws=FAKE + 8) == gs.ERR_WORKSPACE  # eps = 5 passes the eps check
    assert _sc(L, iters=-1) == gs.ERR_ARG
    assert _sc(L, iters=65) == gs.ERR_ARG
    assert _sc(L, cap=-1) == gs.ERR_ARG
    assert _sc(L, idx=None) == gs.ERR_ARG
    assert _sc(L, nnz=None) == gs.ERR_ARG
    assert _sc(L, ws=None) == gs.ERR_WORKSPACE
    assert _sc(L, ws=FAKE + 8) == gs.ERR_WORKSPACE
    assert _sc(L, wsb=100) == gs.ERR_WORKSPACE
    # probabilities
    wsb = L.gspar_workspace_bytes(1, 1000, 1)
    assert L.sparsify_probs(FAKE, 1000, 0.1, 1, 2, None, None, None, None, FAKE, wsb, None) == gs.ERR_ARG
    assert L.sparsify_probs(FAKE, 1000, 2.0, 1, 2, None, FAKE, None, None, FAKE, wsb, None) == gs.ERR_ARG
    # batched
    wsb = L.gspar_workspace_bytes(4, 1000, 0)
    assert L.sparsify_sample_compact_batched(FAKE, 4, 1000, 999, FAKE, 0, 2, FAKE, FAKE, FAKE, 10, FAKE,
                                             None, None, None, FAKE, wsb, None) == gs.ERR_ARG  # ld < d
    assert L.sparsify_sample_compact_batched(FAKE, 0, 1000, 1000, FAKE, 0, 2, FAKE, FAKE, FAKE, 10, FAKE,
                                             None, None, None, FAKE, wsb, None) == gs.ERR_ARG
    assert L.sparsify_sample_compact_batched(FAKE, 4, 1000, 1000, None, 0, 2, FAKE, FAKE, FAKE, 10, FAKE,
                                             None, None, None, FAKE, wsb, None) == gs.ERR_ARG
    assert L.sparsify_sample_compact_batched(FAKE, 4, 1000, 1000, FAKE, 0, 2, None, FAKE, FAKE, 10, FAKE,
                                             None, None, None, FAKE, wsb, None) == gs.ERR_ARG
    assert L.sparsify_probs_batched(FAKE, 4, 1000, 1000, FAKE, 0, 2, None, FAKE, None, None, FAKE, 10, None) \
        == gs.ERR_WORKSPACE
    assert L.gspar_status_string(gs.ERR_ARG) == b"invalid argument"


def test_hybrid_argument_errors(L):
    import paper_1710_09854_amd as gs

    wsb = L.gspar_workspace_bytes(1, 1000, 0)

    def one(**kw):
        a = dict(g=FAKE, d=1000, rho=0.1, idx_a=FAKE, val_a=FAKE, cap_a=10, n_a=FAKE, code_b=FAKE, cap_b=10,
                 n_b=FAKE, ws=FAKE)
        a.update(kw)
        return L.sparsify_sample_hybrid(a["g"], a["d"], a["rho"], 0, 2, 0, a["idx_a"], a["val_a"], a["cap_a"],
                                        a["n_a"], a["code_b"], a["cap_b"], a["n_b"], None, None, None, None,
                                        a["ws"], wsb, None)

    assert one(code_b=None) == gs.ERR_ARG
    assert one(n_a=None) == gs.ERR_ARG
    assert one(n_b=None) == gs.ERR_ARG
    assert one(cap_b=-1) == gs.ERR_ARG
    assert one(idx_a=None) == gs.ERR_ARG
    assert one(rho=2.0) == gs.ERR_ARG
    assert one(ws=FAKE + 8) == gs.ERR_WORKSPACE
    assert L.sparsify_sample_hybrid_batched(FAKE, 2, 1000, 1000, None, 0, 2, FAKE, FAKE, FAKE, 10, FAKE, FAKE, 10,
                                            FAKE, None, None, None, None, FAKE, wsb, None) == gs.ERR_ARG


def test_segmented_argument_errors(L):
    import paper_1710_09854_amd as gs

    good = np.array([0, 400, 400, 1000], np.int64)
    wsb = L.gspar_workspace_bytes(3, 600, 0)

    def one(off=good, segs=3, off_dev=FAKE, rho=FAKE, ws=FAKE, wsb_=wsb, g=FAKE):
        offp = None if off is None else np.ascontiguousarray(off, np.int64).ctypes.data
        a = L.sparsify_sample_compact_segmented(g, segs, offp, off_dev, rho, 0, 2, FAKE, FAKE, FAKE, 10, FAKE,
                                                None, None, None, ws, wsb_, None)
        b = L.sparsify_probs_segmented(g, segs, offp, off_dev, rho, 0, 2, FAKE, FAKE, None, None, ws, wsb_, None)
        assert a == b
        return a

    assert one(off=None) == gs.ERR_ARG
    assert one(off_dev=None) == gs.ERR_ARG
    assert one(g=None) == gs.ERR_ARG
    assert one(rho=None) == gs.ERR_ARG
    assert one(segs=0) == gs.ERR_ARG
    assert one(off=[5, 3, 7, 9]) == gs.ERR_ARG           # decreasing
    assert one(off=[-4, 0, 4, 8]) == gs.ERR_ARG          # negative start
    assert one(off=[0, 1 << 31, 1 << 31, 1 << 31]) == gs.ERR_ARG  # a segment of 2^31 floats
    assert one(ws=FAKE + 8) == gs.ERR_WORKSPACE
    assert one(wsb_=wsb - 1) == gs.ERR_WORKSPACE         # sized for the longest segment (600)

    def hyb(code_b=FAKE, n_a=FAKE, n_b=FAKE, cap_a=10, idx_a=FAKE, off=good, ws=FAKE):
        offp = np.ascontiguousarray(off, np.int64).ctypes.data
        return L.sparsify_sample_hybrid_segmented(FAKE, 3, offp, FAKE, FAKE, 0, 2, FAKE, idx_a, FAKE, cap_a, n_a,
                                                  code_b, 10, n_b, None, None, None, None, ws, wsb, None)

    assert hyb(code_b=None) == gs.ERR_ARG
    assert hyb(n_a=None) == gs.ERR_ARG
    assert hyb(n_b=None) == gs.ERR_ARG
    assert hyb(cap_a=-1) == gs.ERR_ARG
    assert hyb(idx_a=None) == gs.ERR_ARG
    assert hyb(off=[0, 8, 4, 12]) == gs.ERR_ARG
    assert hyb(ws=FAKE + 8) == gs.ERR_WORKSPACE


def test_aggregate_argument_errors(L):
    import paper_1710_09854_amd as gs

    def one(**kw):
        a = dict(idx=FAKE, val=FAKE, cap=10, nnz=FAKE, workers=4, d=1000, v=FAKE)
        a.update(kw)
        return L.gspar_aggregate(a["idx"], a["val"], a["cap"], a["nnz"], a["workers"], a["d"], a["v"], None)

    assert one(nnz=None) == gs.ERR_ARG
    assert one(v=None) == gs.ERR_ARG
    assert one(idx=None) == gs.ERR_ARG
    assert one(val=None) == gs.ERR_ARG
    assert one(cap=-1) == gs.ERR_ARG
    assert one(workers=0) == gs.ERR_ARG
    assert one(workers=(1 << 20) + 1) == gs.ERR_ARG
    assert one(d=0) == gs.ERR_ARG
    assert one(d=1 << 31) == gs.ERR_ARG


def test_coding_bits_match_oracle(L):
    """The library's host-side coding-length helper against the oracle's own statement."""
    import oracle
    import paper_1710_09854_amd as gs

    rng = np.random.default_rng(3)
    for _ in range(200):
        d = int(rng.integers(1, 1 << 28))
        n_a = int(rng.integers(0, min(d, 100000) + 1))
        n_b = int(rng.integers(0, min(d - n_a, 1000000) + 1))
        n_neg = int(rng.integers(0, n_b + 1))
        bits = int(rng.choice([16, 32, 64]))
        got = gs.coding_bits(d, n_a, n_b, n_neg, bits)
        want = oracle.coding_bits(d, n_a, n_b, n_neg, bits)
        for x, y in zip(got, want):
            assert abs(x - y) <= 1e-12 * max(1.0, abs(y))
    out = (ctypes.c_double * 3)()
    assert L.gspar_coding_bits(10, 6, 5, 0, 32, out) == gs.ERR_ARG   # n_a + n_b > d
    assert L.gspar_coding_bits(10, 1, 2, 3, 32, out) == gs.ERR_ARG   # more negatives than Q_B entries
    assert L.gspar_coding_bits(10, 1, 2, 1, 0, out) == gs.ERR_ARG
    assert L.gspar_coding_bits(10, 1, 2, 1, 32, None) == gs.ERR_ARG


def _fx_limbs(v: int):
    return (ctypes.c_uint64 * 5)(*[(v >> (64 * i)) & 0xFFFFFFFFFFFFFFFF for i in range(5)])


def test_fixed_point_rounding_is_correct(LI):
    L = LI
    L.gspar_check_fx_round.argtypes = [ctypes.c_uint64 * 5]
    L.gspar_check_fx_round.restype = ctypes.c_double
    rng = np.random.default_rng(3)
    cases = [0, 1, (1 << 53) - 1, 1 << 53, (1 << 53) + 1, (1 << 54) + 2, (1 << 54) + 6, (1 << 300) - 1]
    for _ in range(3000):
        bits = int(rng.integers(1, 310))
        v = int(rng.integers(0, 1 << 62)) << max(0, bits - 62)
        v |= int(rng.integers(0, 1 << 20))
        cases.append(v & ((1 << 310) - 1))
    # ties: exactly half an ulp above a representable value
    for sh in (0, 7, 100):
        m = (1 << 52) + int(rng.integers(0, 1 << 52))
        cases.append(((2 * m + 1) << sh))
    for v in cases:
        want = float(fractions.Fraction(v, 1 << 149))
        assert L.gspar_check_fx_round(_fx_limbs(v)) == want, hex(v)


def test_exact_sum_matches_fsum(LI):
    L = LI
    L.gspar_check_exact_sum.argtypes = [np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS"), ctypes.c_int64]
    L.gspar_check_exact_sum.restype = ctypes.c_double
    rng = np.random.default_rng(4)
    for t in range(20):
        x = (rng.standard_normal(5000) * np.exp2(rng.uniform(-150, 120, 5000))).astype(np.float32)
        x[:10] = 0
        assert L.gspar_check_exact_sum(x, x.size) == math.fsum(np.abs(x.astype(np.float64)))


def test_cap_key_is_smallest_capped_pattern(LI):
    L = LI
    L.gspar_check_cap_key.argtypes = [ctypes.c_double]
    L.gspar_check_cap_key.restype = ctypes.c_uint32
    rng = np.random.default_rng(5)
    lams = list(np.exp(rng.uniform(-90, 100, 3000))) + [1.0, 0.5, 3.0, 1e-45, 1e40, 2.0 ** -126]

    def val(k):
        return float(np.array([k], np.uint32).view(np.float32)[0])

    for lam in lams:
        lam = float(lam)
        k = L.gspar_check_cap_key(lam)
        assert 1 <= k <= 0x7F800000
        if k < 0x7F800000:
            assert lam * val(k) >= 1.0
        if k > 1:
            assert lam * val(k - 1) < 1.0
    assert L.gspar_check_cap_key(0.0) == 0x7F800000
    assert L.gspar_check_cap_key(float("inf")) == 1
    assert L.gspar_check_cap_key(float("nan")) == 0x7F800000


def test_device_philox_known_answers(LI):
    L = LI
    u32p = np.ctypeslib.ndpointer(np.uint32, flags="C_CONTIGUOUS")
    L.gspar_check_philox.argtypes = [u32p, u32p, u32p]
    L.gspar_check_philox.restype = None
    path = os.path.join(ROOT, "tests", "golden", "philox4x32_10_kat.txt")
    n = 0
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        v = [int(t, 16) for t in line.split()]
        out = np.zeros(4, np.uint32)
        L.gspar_check_philox(np.array(v[0:4], np.uint32), np.array(v[4:6], np.uint32), out)
        assert out.tolist() == v[6:10]
        n += 1
    assert n == 3


def test_shift_out_of_range_is_flagged(LI):
    """The exact accumulators' shifts: in range they place v * 2^s exactly; out of range (a broken
    invariant of the solver) they report the internal flag (16) and give zero, never a clamped
    shift."""
    L = LI
    L.gspar_check_fx_shifted.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.c_uint64 * 5]
    L.gspar_check_fx_shifted.restype = ctypes.c_uint32
    L.gspar_check_fq_squares.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int, ctypes.c_uint64 * 10]
    L.gspar_check_fq_squares.restype = ctypes.c_uint32

    def fx(v, sh):
        out = (ctypes.c_uint64 * 5)()
        err = L.gspar_check_fx_shifted(v, sh, out)
        return err, sum(int(out[i]) << (64 * i) for i in range(5))

    def fq(qh, ql, sh):
        out = (ctypes.c_uint64 * 10)()
        err = L.gspar_check_fq_squares(qh, ql, sh, out)
        return err, sum(int(out[i]) << (64 * i) for i in range(10))

    v = 0xFEDCBA9876543210
    for sh in (0, 1, 63, 64, 65, 127, 200, 254, 255):
        assert fx(v, sh) == (0, v << sh), sh
    for sh in (-1, -64, 256, 300, 1 << 20):
        assert fx(v, sh) == (16, 0), sh
    qh, ql = (1 << 55) - 3, (1 << 55) - 5
    for sh in (0, 1, 100, 254, 255):
        assert fq(qh, ql, sh) == (0, ((qh << 24) + ql) << (2 * sh)), sh
    for sh in (-1, 256, 1000):
        assert fq(qh, ql, sh) == (16, 0), sh


def test_no_cpu_fallback_in_binding():
    """The binding must not compute anything itself: its only numeric dependency is torch for
    allocation; it never imports the oracle or numpy."""
    src = open(os.path.join(ROOT, "paper_1710_09854_amd", "__init__.py")).read()
    assert "import oracle" not in src and "from oracle" not in src
    assert "import numpy" not in src
