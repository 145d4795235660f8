"""The C-ABI library loads, exports every declared entry point, and rejects
bad arguments on the host before any device work (CPU only: no call here
reaches a kernel)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "stagefrontier.h")


def declared_functions():
    with open(HEADER) as fh:
        text = fh.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sf_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def sf():
    import torch  # noqa: F401  (binding order: torch's HIP runtime first)
    from paper_2606_06751_amd import stagefrontier
    return stagefrontier


def test_header_declares_the_boundary():
    assert declared_functions() == ["sf_exposure_gain", "sf_frontier", "sf_frontier_checked",
                                    "sf_frontier_evidence",
                                    "sf_frontier_lag", "sf_frontier_summary", "sf_ingest",
                                    "sf_num_windows",
                                    "sf_rank_spread", "sf_read_xor", "sf_read_xor_pieces", "sf_route",
                                    "sf_strerror", "sf_version",
                                    "sf_window_lead_exposed", "sf_window_leader_switches",
                                    "sf_window_median",
                                    "sf_window_summary"]


def test_header_is_plain_c(tmp_path):
    """The boundary is usable from C: the header alone compiles as strict C99."""
    import shutil
    import subprocess

    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use.c"
    src.write_text('#include "stagefrontier.h"\n'
                   "int use(void) { return SF_OK + (int)sizeof(sf_stream_t); }\n")
    proc = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                           "-I", os.path.join(ROOT, "include"), "-c", str(src),
                           "-o", str(tmp_path / "use.o")], capture_output=True, text=True)
    assert proc.returncode == 0, proc.stderr


def test_every_declared_symbol_is_exported(sf):
    lib = sf.raw_library()
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert hasattr(sf, name), "binding lacks %s" % name


def test_constants_match_header(sf):
    with open(HEADER) as fh:
        text = fh.read()
    assert "#define SF_MAX_R %d" % sf.SF_MAX_R in text
    for gone in ("SF_MAX_WINDOW_MEDIAN", "#define SF_MAX_S ", "SF_MAX_S_GAIN", "SF_MAX_R_LAG",
                 "SF_MAX_S_EVIDENCE", "SF_MAX_S_INGEST"):
        assert gone not in text, gone
    assert "#define SF_XOR_PIECE_BYTES %d" % sf.SF_XOR_PIECE_BYTES in text
    for name in ("SF_OK", "SF_EINVAL", "SF_ERANGE", "SF_EHIP"):
        assert re.search(r"%s = %d" % (name, getattr(sf, name)), text), name


def test_host_only_calls(sf):
    assert sf.sf_version().startswith("libstagefrontier")
    assert sf.sf_strerror(sf.SF_OK) == "success"
    assert sf.sf_strerror(sf.SF_EINVAL) == "invalid argument"
    assert sf.sf_strerror(12345) == "unknown status"
    assert sf.sf_num_windows(0, 10) == 0
    assert sf.sf_num_windows(1000, 100) == 10
    assert sf.sf_num_windows(1001, 100) == 11
    assert sf.sf_num_windows(5, 1) == 5
    assert sf.sf_num_windows(-1, 1) == -1
    assert sf.sf_num_windows(10, 0) == -1


# fake, never-dereferenced device addresses for host-side validation
A = 1 << 40
B = 2 << 40
C = 3 << 40


def test_frontier_argument_checks(sf):
    lib = sf.raw_library()
    ok_args = dict(d=A, T=10, R=8, S=6, inc=B, lead=C)

    def call(**kw):
        a = dict(ok_args, **kw)
        return lib.sf_frontier(a["d"], a["T"], a["R"], a["S"], a["inc"], a["lead"], None)

    assert call(T=0, d=None, inc=None, lead=None) == sf.SF_OK   # empty input: no-op
    assert call(T=-1) == sf.SF_EINVAL
    assert call(R=0) == sf.SF_EINVAL
    assert call(R=sf.SF_MAX_R + 1) == sf.SF_EINVAL
    assert call(S=0) == sf.SF_EINVAL
    assert call(d=None) == sf.SF_EINVAL
    assert call(inc=None) == sf.SF_EINVAL
    assert call(lead=None) == sf.SF_EINVAL
    assert call(d=A + 4) == sf.SF_EINVAL          # misaligned int64
    assert call(inc=B + 4) == sf.SF_EINVAL
    assert call(lead=C + 2) == sf.SF_EINVAL
    assert call(inc=A + 8) == sf.SF_EINVAL        # output overlaps input
    assert call(lead=B + 16) == sf.SF_EINVAL      # outputs overlap
    assert call(T=1 << 50, R=sf.SF_MAX_R, S=512) == sf.SF_EINVAL  # size overflow
    assert call(T=1 << 20, R=sf.SF_MAX_R, S=1 << 20) == sf.SF_EINVAL  # size overflow at large S


def test_checked_argument_checks(sf):
    lib = sf.raw_library()
    D = 4 << 40

    def call(**kw):
        a = dict(dict(d=A, T=10, R=8, S=6, inc=B, lead=C, st=D), **kw)
        return lib.sf_frontier_checked(a["d"], a["T"], a["R"], a["S"], a["inc"], a["lead"],
                                       a["st"], None)

    assert call(T=0, d=None, inc=None, lead=None) == sf.SF_OK
    assert call(st=None) == sf.SF_EINVAL          # the status word is required
    assert call(st=D + 2) == sf.SF_EINVAL         # misaligned
    assert call(st=B + 8) == sf.SF_EINVAL         # inside an output
    assert call(st=A + 16) == sf.SF_EINVAL        # inside the input
    assert call(R=0) == sf.SF_EINVAL
    assert call(inc=A + 8) == sf.SF_EINVAL        # output overlaps input


def test_evidence_argument_checks(sf):
    lib = sf.raw_library()
    names = ["d", "inc", "lead", "gap", "ties", "smax", "ssum"]
    base = {n: (i + 1) << 40 for i, n in enumerate(names)}
    ok_args = dict(base, T=10, R=8, S=6)

    def call(**kw):
        a = dict(ok_args, **kw)
        return lib.sf_frontier_evidence(a["d"], a["T"], a["R"], a["S"],
                                        *(a[n] for n in names[1:]), None)

    assert call(T=0, **{n: None for n in names}) == sf.SF_OK
    assert call(R=0) == sf.SF_EINVAL
    assert call(S=0) == sf.SF_EINVAL
    for n in names:
        assert call(**{n: None}) == sf.SF_EINVAL, n
    assert call(ties=base["ties"] + 2) == sf.SF_EINVAL       # misaligned int32
    assert call(gap=base["gap"] + 4) == sf.SF_EINVAL         # misaligned int64
    assert call(ssum=base["d"] + 64) == sf.SF_EINVAL         # output overlaps input
    assert call(ties=base["gap"] + 8) == sf.SF_EINVAL        # outputs overlap
    assert call(T=1 << 33, R=1, S=1) == sf.SF_EINVAL         # one workgroup per step


def test_ingest_and_route_argument_checks(sf):
    lib = sf.raw_library()
    X, Wl, D, O = 1 << 40, 2 << 40, 3 << 40, 4 << 40

    def ingest(**kw):
        a = dict(dict(x=X, w=Wl, T=10, R=8, K=5, d=D, o=O), **kw)
        return lib.sf_ingest(a["x"], a["w"], a["T"], a["R"], a["K"], a["d"], a["o"], None)

    assert ingest(T=0, x=None, w=None, d=None, o=None) == sf.SF_OK
    assert ingest(K=-1) == sf.SF_EINVAL
    assert ingest(K=(1 << 31) - 2) == sf.SF_EINVAL           # K + 2 overflows int32
    assert ingest(R=0) == sf.SF_EINVAL
    assert ingest(w=None) == sf.SF_EINVAL
    assert ingest(d=X + 8) == sf.SF_EINVAL                  # output overlaps input
    assert ingest(o=D + 16) == sf.SF_EINVAL                 # outputs overlap
    assert ingest(o=O + 4) == sf.SF_EINVAL                  # misaligned

    def route(**kw):
        a = dict(dict(e=X, W=10, S=6, num=4, den=5, order=D, size=O), **kw)
        return lib.sf_route(a["e"], a["W"], a["S"], a["num"], a["den"], a["order"], a["size"], None)

    assert route(W=0, e=None, order=None, size=None) == sf.SF_OK
    assert route(den=0) == sf.SF_EINVAL
    assert route(num=6) == sf.SF_EINVAL                     # tau > 1
    assert route(num=-1) == sf.SF_EINVAL
    assert route(S=0) == sf.SF_EINVAL
    assert route(order=X + 8) == sf.SF_EINVAL
    assert route(size=D + 4) == sf.SF_EINVAL


def test_gain_argument_checks(sf):
    lib = sf.raw_library()
    names = ["d", "b", "g", "m", "wg", "wm"]
    base = {n: (i + 1) << 40 for i, n in enumerate(names)}

    def call(**kw):
        a = dict(dict(base, T=100, R=8, S=6, window=10), **kw)
        return lib.sf_exposure_gain(a["d"], a["b"], a["T"], a["R"], a["S"], a["window"],
                                    *(a[n] for n in names[2:]), None)

    assert call(T=0) == sf.SF_OK
    assert call(window=0) == sf.SF_EINVAL
    for n in names:
        assert call(**{n: None}) == sf.SF_EINVAL, n
    assert call(b=base["b"] + 4) == sf.SF_EINVAL            # misaligned
    assert call(g=base["d"] + 8) == sf.SF_EINVAL            # output overlaps input
    assert call(wm=base["wg"] + 8) == sf.SF_EINVAL          # outputs overlap


def test_lag_argument_checks(sf):
    lib = sf.raw_library()

    def call(**kw):
        a = dict(dict(d=A, T=10, R=8, S=6, lag=B, inc=C), **kw)
        return lib.sf_frontier_lag(a["d"], a["T"], a["R"], a["S"], a["lag"], a["inc"], None)

    assert call(T=0, d=None, lag=None, inc=None) == sf.SF_OK
    assert call(R=sf.SF_MAX_R + 1) == sf.SF_EINVAL
    assert call(S=0) == sf.SF_EINVAL
    assert call(inc=None) == sf.SF_EINVAL
    assert call(lag=B + 4) == sf.SF_EINVAL
    assert call(lag=A + 8) == sf.SF_EINVAL                  # output overlaps input
    assert call(inc=B + 8) == sf.SF_EINVAL                  # outputs overlap
    assert call(T=1 << 32, R=1, S=1) == sf.SF_EINVAL        # one workgroup per step


def test_spread_argument_checks(sf):
    lib = sf.raw_library()

    def call(**kw):
        a = dict(dict(d=A, T=10, R=8, S=6, window=4, sp=B, wsp=C), **kw)
        return lib.sf_rank_spread(a["d"], a["T"], a["R"], a["S"], a["window"], a["sp"], a["wsp"],
                                  None)

    assert call(T=0, d=None, sp=None, wsp=None) == sf.SF_OK
    assert call(R=sf.SF_MAX_R + 1) == sf.SF_EINVAL
    assert call(S=0) == sf.SF_EINVAL
    assert call(window=0) == sf.SF_EINVAL
    assert call(wsp=None) == sf.SF_EINVAL
    assert call(sp=B + 4) == sf.SF_EINVAL                   # misaligned
    assert call(sp=A + 8) == sf.SF_EINVAL                   # output overlaps input
    assert call(wsp=B + 8) == sf.SF_EINVAL                  # outputs overlap
    assert call(T=1 << 32, R=1, S=1) == sf.SF_EINVAL        # one workgroup per step


def test_window_median_argument_checks(sf):
    lib = sf.raw_library()

    def call(**kw):
        a = dict(dict(d=A, T=100, R=8, S=6, window=10, m=B), **kw)
        return lib.sf_window_median(a["d"], a["T"], a["R"], a["S"], a["window"], a["m"], None)

    assert call(T=0, d=None, m=None) == sf.SF_OK
    assert call(R=0) == sf.SF_EINVAL
    assert call(R=sf.SF_MAX_R + 1) == sf.SF_EINVAL
    assert call(window=0) == sf.SF_EINVAL
    assert call(m=None) == sf.SF_EINVAL
    assert call(m=B + 4) == sf.SF_EINVAL                    # misaligned
    assert call(m=A + 8) == sf.SF_EINVAL                    # output overlaps input


def test_read_xor_argument_checks(sf):
    lib = sf.raw_library()
    P = sf.SF_XOR_PIECE_BYTES

    def call(**kw):
        a = dict(dict(buf=A, n=3 * P + 8, out=B), **kw)
        return lib.sf_read_xor(a["buf"], a["n"], a["out"], None)

    assert call(n=0, buf=None, out=None) == sf.SF_OK       # empty: nothing to do
    assert call(n=-8) == sf.SF_EINVAL
    assert call(n=4100) == sf.SF_EINVAL                    # not a multiple of 8
    assert call(out=None) == sf.SF_EINVAL
    assert call(out=B + 4) == sf.SF_EINVAL                 # misaligned result words
    assert call(buf=A + 8) == sf.SF_EINVAL                 # buffer not 16-byte aligned
    assert call(buf=None) == sf.SF_EINVAL
    assert call(out=A + 1024) == sf.SF_EINVAL              # result words inside the buffer
    assert call(out=A - 16) == sf.SF_EINVAL                # 4 result words run into the buffer
    assert call(n=(1 << 31) * P) == sf.SF_EINVAL           # more than 2^31 - 1 pieces
    assert sf.sf_read_xor_pieces(0) == 0
    assert sf.sf_read_xor_pieces(8) == 1
    assert sf.sf_read_xor_pieces(P) == 1
    assert sf.sf_read_xor_pieces(P + 8) == 2
    assert sf.sf_read_xor_pieces(-8) == -1


def test_summary_argument_checks(sf):
    lib = sf.raw_library()
    D = 4 << 40
    E = 5 << 40
    ok_args = dict(inc=A, lead=B, T=100, R=8, S=6, window=10, ex=C, cnt=D, top=E)

    def call(**kw):
        a = dict(ok_args, **kw)
        return lib.sf_window_summary(a["inc"], a["lead"], a["T"], a["R"], a["S"], a["window"],
                                     a["ex"], a["cnt"], a["top"], None)

    assert call(T=0, inc=None, lead=None, ex=None, cnt=None, top=None) == sf.SF_OK
    assert call(window=0) == sf.SF_EINVAL
    assert call(T=-5) == sf.SF_EINVAL
    assert call(R=0) == sf.SF_EINVAL
    assert call(cnt=None) == sf.SF_EINVAL
    assert call(top=E + 2) == sf.SF_EINVAL
    assert call(ex=A + 8) == sf.SF_EINVAL         # output overlaps input
    assert call(top=D + 4) == sf.SF_EINVAL        # outputs overlap


def test_lead_exposed_argument_checks(sf):
    lib = sf.raw_library()
    D = 4 << 40
    ok_args = dict(inc=A, lead=B, T=100, R=8, S=6, window=10, le=C, top=D)

    def call(**kw):
        a = dict(ok_args, **kw)
        return lib.sf_window_lead_exposed(a["inc"], a["lead"], a["T"], a["R"], a["S"],
                                          a["window"], a["le"], a["top"], None)

    assert call(T=0, inc=None, lead=None, le=None, top=None) == sf.SF_OK
    assert call(window=0) == sf.SF_EINVAL
    assert call(T=-5) == sf.SF_EINVAL
    assert call(R=0) == sf.SF_EINVAL
    assert call(R=sf.SF_MAX_R + 1) == sf.SF_EINVAL
    assert call(le=None) == sf.SF_EINVAL
    assert call(top=None) == sf.SF_EINVAL
    assert call(le=C + 4) == sf.SF_EINVAL         # misaligned int64 output
    assert call(top=D + 2) == sf.SF_EINVAL
    assert call(le=B + 8) == sf.SF_EINVAL         # output overlaps input
    assert call(top=C + 8) == sf.SF_EINVAL        # outputs overlap
    assert call(T=1 << 40, R=65536, S=512, window=1) == sf.SF_EINVAL  # W*S*R*8 overflows


def test_leader_switches_argument_checks(sf):
    lib = sf.raw_library()
    D = 4 << 40
    E = 5 << 40
    ok_args = dict(lead=A, gap=B, ties=C, T=100, S=6, window=10, g=0, sw=D, el=E)

    def call(**kw):
        a = dict(ok_args, **kw)
        return lib.sf_window_leader_switches(a["lead"], a["gap"], a["ties"], a["T"], a["S"],
                                             a["window"], a["g"], a["sw"], a["el"], None)

    assert call(T=0, lead=None, gap=None, ties=None, sw=None, el=None) == sf.SF_OK
    assert call(window=0) == sf.SF_EINVAL
    assert call(T=-1) == sf.SF_EINVAL
    assert call(S=0) == sf.SF_EINVAL
    assert call(ties=None) == sf.SF_EINVAL
    assert call(el=None) == sf.SF_EINVAL
    assert call(gap=B + 4) == sf.SF_EINVAL        # misaligned int64 input
    assert call(sw=D + 2) == sf.SF_EINVAL
    assert call(sw=C + 8) == sf.SF_EINVAL         # output overlaps an input
    assert call(el=D + 8) == sf.SF_EINVAL         # outputs overlap
    assert call(T=1 << 32, S=1, window=1 << 32) == sf.SF_EINVAL  # counts past int32


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    """The binding has no CPU fallback: a missing library is an ImportError."""
    import importlib

    import torch  # noqa: F401
    from paper_2606_06751_amd import build as b
    monkeypatch.setattr(b, "LIB", str(tmp_path / "missing.so"))
    import paper_2606_06751_amd.stagefrontier as mod
    try:
        with pytest.raises(ImportError):
            importlib.reload(mod)
    finally:
        monkeypatch.undo()
        importlib.reload(mod)


def test_ctypes_argtypes_cover_header(sf):
    lib = sf.raw_library()
    assert len(lib.sf_frontier.argtypes) == 7
    assert len(lib.sf_frontier_evidence.argtypes) == 11
    assert len(lib.sf_frontier_checked.argtypes) == 8
    assert len(lib.sf_ingest.argtypes) == 8
    assert len(lib.sf_exposure_gain.argtypes) == 11
    assert len(lib.sf_frontier_lag.argtypes) == 7
    assert len(lib.sf_rank_spread.argtypes) == 8
    assert len(lib.sf_window_median.argtypes) == 7
    assert len(lib.sf_route.argtypes) == 8
    assert len(lib.sf_window_summary.argtypes) == 10
    assert len(lib.sf_window_lead_exposed.argtypes) == 9
    assert len(lib.sf_window_leader_switches.argtypes) == 10
    assert len(lib.sf_read_xor.argtypes) == 4
    assert lib.sf_num_windows.restype is ctypes.c_int64


def test_frontier_summary_argument_checks(sf):
    lib = sf.raw_library()
    names = ["d", "inc", "lead", "ex", "cnt", "top"]
    base = {n: (i + 1) << 40 for i, n in enumerate(names)}

    def call(**kw):
        a = dict(dict(base, T=100, R=8, S=6, window=10), **kw)
        return lib.sf_frontier_summary(a["d"], a["T"], a["R"], a["S"], a["window"],
                                       *(a[n] for n in names[1:]), None)

    assert call(T=0, **{n: None for n in names}) == sf.SF_OK
    assert call(T=-1) == sf.SF_EINVAL
    assert call(R=0) == sf.SF_EINVAL
    assert call(R=sf.SF_MAX_R + 1) == sf.SF_EINVAL
    assert call(S=0) == sf.SF_EINVAL
    assert call(window=0) == sf.SF_EINVAL
    for n in names:
        assert call(**{n: None}) == sf.SF_EINVAL, n
    assert call(inc=base["inc"] + 4) == sf.SF_EINVAL      # misaligned int64
    assert call(lead=base["lead"] + 2) == sf.SF_EINVAL    # misaligned int32
    assert call(ex=base["d"] + 8) == sf.SF_EINVAL         # output overlaps input
    assert call(cnt=base["inc"] + 8) == sf.SF_EINVAL      # outputs overlap
    assert call(T=1 << 50, R=sf.SF_MAX_R, S=512) == sf.SF_EINVAL  # size overflow
