"""The C ABI: the library loads, exports every function include/specverify.h
declares, the ctypes prototypes agree with the header, and host-checkable
argument errors come back synchronously (no GPU work is enqueued by any
call in this file)."""

import ctypes
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_12370_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "specverify.h")


def _header_text():
    with open(HEADER) as f:
        return f.read()


def header_prototypes():
    src = _header_text()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    protos = {}
    for m in re.finditer(r"\b(?:spec_status|size_t|int|const char\*)\s+(spec_\w+)\s*\(([^;]*?)\)\s*;", src, re.S):
        args = [a.strip() for a in m.group(2).split(",") if a.strip() and a.strip() != "void"]
        protos[m.group(1)] = args
    return protos


@pytest.fixture(scope="module")
def lib():
    return binding.load_library()


def test_exports_every_declared_function(lib):
    protos = header_prototypes()
    assert set(protos) == {"spec_verify_workspace_size", "spec_verify", "spec_tv_workspace_size",
                           "spec_tv_loss_fwd_bwd", "spec_status_string", "spec_version",
                           "spec_verify_target_only_workspace_size", "spec_verify_target_only",
                           "spec_sample_workspace_size", "spec_sample",
                           "spec_diagnostics_workspace_size", "spec_diagnostics",
                           "spec_verify_gumbel_workspace_size", "spec_verify_gumbel",
                           "spec_sample_gumbel_workspace_size", "spec_sample_gumbel",
                           "spec_kl_workspace_size", "spec_kl_loss_fwd_bwd", "spec_verify_ex",
                           "spec_verify_noalloc", "spec_verify_noalloc_max_workspace"}
    for name in protos:
        assert hasattr(lib, name), name


def test_ctypes_prototypes_match_header():
    protos = header_prototypes()
    assert len(protos["spec_verify"]) == len(binding.VERIFY_ARGTYPES)
    assert len(protos["spec_tv_loss_fwd_bwd"]) == len(binding.TV_ARGTYPES)
    assert len(protos["spec_verify_target_only"]) == len(binding.TO_ARGTYPES)
    assert len(protos["spec_sample"]) == len(binding.SAMPLE_ARGTYPES)
    assert len(protos["spec_diagnostics"]) == len(binding.DIAG_ARGTYPES)
    assert len(protos["spec_verify_gumbel"]) == len(binding.VERIFY_ARGTYPES)
    assert protos["spec_verify_gumbel"] == protos["spec_verify"]
    assert len(protos["spec_sample_gumbel"]) == len(binding.SAMPLE_GUMBEL_ARGTYPES)
    assert len(protos["spec_kl_loss_fwd_bwd"]) == len(binding.KL_ARGTYPES)
    assert len(protos["spec_verify_ex"]) == len(binding.VERIFY_EX_ARGTYPES)
    assert protos["spec_verify_ex"][:-1] == protos["spec_verify"]
    assert len(protos["spec_verify_noalloc"]) == len(binding.VERIFY_NOALLOC_ARGTYPES)
    assert protos["spec_verify_noalloc"][:-1] == protos["spec_verify"][:-3]


def test_diag_columns_match_header():
    src = _header_text()
    cols = re.findall(r"SPEC_DIAG_(\w+) = (\d+)", src)
    named = {name.lower(): int(v) for name, v in cols}
    assert named.pop("ncols") == len(binding.DIAG_COLUMNS)
    assert sorted(named.values()) == list(range(len(binding.DIAG_COLUMNS)))
    for name, v in named.items():
        assert binding.DIAG_COLUMNS[v] == name, (name, v)


def test_version_and_status_strings(lib):
    ver = int(re.search(r"#define SPEC_VERSION (\d+)", _header_text()).group(1))
    assert lib.spec_version() == ver
    for code in (0, 1, 2, 4, 5):
        assert lib.spec_status_string(code)
    assert lib.spec_status_string(99) == b"unknown status"


def test_workspace_sizes(lib):
    assert lib.spec_verify_workspace_size(0, 3, 100, 1) == 0
    assert lib.spec_verify_workspace_size(4, 0, 100, 1) == 0
    assert lib.spec_verify_workspace_size(4, 9, 100, 1) == 0
    assert lib.spec_verify_workspace_size(4, 3, 0, 1) == 0
    assert lib.spec_verify_workspace_size(4, 3, 100, 7) == 0
    a = lib.spec_verify_workspace_size(64, 3, 151936, 1)
    b = lib.spec_verify_workspace_size(256, 3, 151936, 1)
    assert 0 < a < b and a % 256 == 0
    assert lib.spec_tv_workspace_size(16384, 3, 151936, 1) > 0
    assert lib.spec_tv_workspace_size(16384, 0, 151936, 1) == 0
    # target-only: statistics of the K+1 target rows only, one 16-byte record
    # per 8192-element sub-chunk (19 per bf16 row of 151936)
    to = lib.spec_verify_target_only_workspace_size(256, 3, 151936, 1)
    assert to == 256 * 4 * 19 * 16
    assert lib.spec_verify_target_only_workspace_size(256, 9, 151936, 1) == 0
    assert lib.spec_sample_workspace_size(768, 151936, 1) == 768 * 19 * 16
    assert lib.spec_sample_workspace_size(0, 151936, 1) == 0
    assert lib.spec_sample_workspace_size(4, 0, 0) == 0
    assert lib.spec_diagnostics_workspace_size(256, 3, 151936, 1) > 0
    assert lib.spec_diagnostics_workspace_size(256, 0, 151936, 1) == 0
    # multinomial verification keeps statistics per 8192-element sub-chunk (19 per bf16 row
    # at V=151936); Gumbel-max verification per 16384-element chunk (10 per row) plus one
    # 16-byte best key per (batch row, chunk)
    assert b >= 256 * 7 * 19 * 16 + 256 * 3 * 19 * 16
    g = lib.spec_verify_gumbel_workspace_size(256, 3, 151936, 1)
    assert 256 * 7 * 10 * 16 + 256 * 3 * 10 * 16 + 256 * 10 * 16 <= g < b
    assert lib.spec_verify_gumbel_workspace_size(256, 9, 151936, 1) == 0
    assert lib.spec_sample_gumbel_workspace_size(768, 151936, 1) == 768 * 10 * 16
    assert lib.spec_sample_gumbel_workspace_size(0, 151936, 1) == 0
    assert lib.spec_kl_workspace_size(16384, 3, 151936, 1) > 0
    assert lib.spec_kl_workspace_size(16384, 9, 151936, 1) == 0


def test_vocabulary_limit(lib):
    """V up to SPEC_MAX_V = 2^31 - 2^16 is accepted (element indices, 32-bit,
    run one 16384-element chunk past V); one more is rejected everywhere."""
    max_v = int(re.search(r"#define SPEC_MAX_V (\d+)", _header_text()).group(1))
    assert max_v == (1 << 31) - (1 << 16)
    for V, ok in ((max_v, True), (max_v + 1, False)):
        for dt in (0, 1):
            sizes = [lib.spec_verify_workspace_size(1, 1, V, dt), lib.spec_tv_workspace_size(1, 1, V, dt),
                     lib.spec_verify_gumbel_workspace_size(1, 1, V, dt), lib.spec_sample_gumbel_workspace_size(1, V, dt),
                     lib.spec_verify_target_only_workspace_size(1, 1, V, dt), lib.spec_sample_workspace_size(1, V, dt),
                     lib.spec_diagnostics_workspace_size(1, 1, V, dt), lib.spec_kl_workspace_size(1, 1, V, dt)]
            assert all((x > 0) == ok for x in sizes), (V, dt, sizes)


FAKE = 0x10000  # never dereferenced: every call below fails validation first


def call_verify(lib, **kw):
    args = dict(t=FAKE, tsb=400, tsk=100, d=FAKE, dsb=300, dsk=100, dtype=1, B=4, K=3, V=100, ids=FAKE,
                temp=None, temp_s=1.0, seed=0, off=0, acc=FAKE, em=FAKE, ov=None, p=None, q=None,
                lzt=None, lzd=None, ws=FAKE, wsb=1 << 30, stream=None)
    args.update(kw)
    return lib.spec_verify(*[args[k] for k in ("t", "tsb", "tsk", "d", "dsb", "dsk", "dtype", "B", "K", "V", "ids",
                                               "temp", "temp_s", "seed", "off", "acc", "em", "ov", "p", "q", "lzt",
                                               "lzd", "ws", "wsb", "stream")])


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), 2),
    (dict(K=9), 2),
    (dict(B=0), 1),
    (dict(V=0), 1),
    (dict(K=0), 1),
    (dict(t=None), 1),
    (dict(d=None), 1),
    (dict(ids=None), 1),
    (dict(acc=None), 1),
    (dict(em=None), 1),
    (dict(tsb=-1), 1),
    (dict(dsk=-100), 1),
    (dict(temp_s=0.0), 1),
    (dict(temp_s=float("nan")), 1),
    (dict(temp_s=float("inf")), 1),
    (dict(temp_s=-1.0), 1),
    (dict(ws=None), 4),
    (dict(wsb=64), 4),
    (dict(ws=FAKE + 4), 1),
    (dict(V=(1 << 31) - (1 << 16) + 1, tsk=1 << 31, tsb=1 << 33, dsk=1 << 31, dsb=1 << 33), 1),
])
def test_verify_argument_errors(lib, kw, status):
    assert call_verify(lib, **kw) == status


def call_verify_ex(lib, path, groups, shape=0, **kw):
    args = dict(t=FAKE, tsb=400, tsk=100, d=FAKE, dsb=300, dsk=100, dtype=1, B=4, K=3, V=100, ids=FAKE,
                temp=None, temp_s=1.0, seed=0, off=0, acc=FAKE, em=FAKE, ov=None, p=None, q=None,
                lzt=None, lzd=None, ws=FAKE, wsb=1 << 30, stream=None)
    args.update(kw)
    lc = binding.SpecLaunch(path, groups, shape)
    return lib.spec_verify_ex(*[args[k] for k in ("t", "tsb", "tsk", "d", "dsb", "dsk", "dtype", "B", "K", "V", "ids",
                                                  "temp", "temp_s", "seed", "off", "acc", "em", "ov", "p", "q", "lzt",
                                                  "lzd", "ws", "wsb", "stream")], ctypes.byref(lc))


@pytest.mark.parametrize("path,groups,kw,status", [
    (3, 0, {}, 1),
    (-1, 0, {}, 1),
    (0, -2, {}, 1),
    (2, 0, dict(K=9), 2),
    (1, 0, dict(B=0), 1),
    (2, 4, dict(ws=None), 4),
    (0, 0, dict(temp_s=0.0), 1),
    (1, 0, dict(shape=3), 1),
    (1, 0, dict(shape=-1), 1),
])
def test_verify_ex_argument_errors(lib, path, groups, kw, status):
    assert call_verify_ex(lib, path, groups, **kw) == status


def call_tv(lib, **kw):
    args = dict(t=FAKE, tsn=300, tsk=100, d=FAKE, dsn=300, dsk=100, dtype=1, N=4, K=3, V=100, T=1.0, mode=0,
                scale=1.0, loss=FAKE, ov=None, grad=None, ws=FAKE, wsb=1 << 30, stream=None)
    args.update(kw)
    return lib.spec_tv_loss_fwd_bwd(*[args[k] for k in ("t", "tsn", "tsk", "d", "dsn", "dsk", "dtype", "N", "K", "V",
                                                        "T", "mode", "scale", "loss", "ov", "grad", "ws", "wsb",
                                                        "stream")])


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=3), 2),
    (dict(K=9), 2),
    (dict(N=0), 1),
    (dict(V=-5), 1),
    (dict(t=None), 1),
    (dict(loss=None), 1),
    (dict(T=0.0), 1),
    (dict(T=float("nan")), 1),
    (dict(mode=3), 1),
    (dict(scale=float("inf")), 1),
    (dict(tsk=-1), 1),
    (dict(ws=None), 4),
    (dict(wsb=100), 4),
    (dict(V=(1 << 31) - (1 << 16) + 1, tsk=1 << 31, tsn=1 << 33, dsk=1 << 31, dsn=1 << 33), 1),
])
def test_tv_argument_errors(lib, kw, status):
    assert call_tv(lib, **kw) == status


def call_to(lib, **kw):
    args = dict(t=FAKE, tsb=400, tsk=100, dtype=1, B=4, K=3, V=100, ids=FAKE, temp=None, temp_s=1.0, seed=0,
                off=0, acc=FAKE, em=FAKE, p=None, lzt=None, ws=FAKE, wsb=1 << 30, stream=None)
    args.update(kw)
    return lib.spec_verify_target_only(*[args[k] for k in ("t", "tsb", "tsk", "dtype", "B", "K", "V", "ids", "temp",
                                                           "temp_s", "seed", "off", "acc", "em", "p", "lzt", "ws",
                                                           "wsb", "stream")])


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), 2),
    (dict(K=9), 2),
    (dict(B=0), 1),
    (dict(K=0), 1),
    (dict(V=0), 1),
    (dict(t=None), 1),
    (dict(ids=None), 1),
    (dict(acc=None), 1),
    (dict(em=None), 1),
    (dict(tsk=-1), 1),
    (dict(temp_s=0.0), 1),
    (dict(temp_s=float("nan")), 1),
    (dict(ws=None), 4),
    (dict(wsb=64), 4),
    (dict(ws=FAKE + 8), 1),
])
def test_target_only_argument_errors(lib, kw, status):
    assert call_to(lib, **kw) == status


def call_sample(lib, **kw):
    args = dict(z=FAKE, sr=100, dtype=1, R=4, V=100, temp=None, temp_s=1.0, seed=0, off=0, tok=FAKE, lz=None,
                ws=FAKE, wsb=1 << 30, stream=None)
    args.update(kw)
    return lib.spec_sample(*[args[k] for k in ("z", "sr", "dtype", "R", "V", "temp", "temp_s", "seed", "off", "tok",
                                               "lz", "ws", "wsb", "stream")])


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=5), 2),
    (dict(R=0), 1),
    (dict(V=0), 1),
    (dict(z=None), 1),
    (dict(tok=None), 1),
    (dict(sr=-1), 1),
    (dict(temp_s=-0.5), 1),
    (dict(temp_s=float("inf")), 1),
    (dict(temp_s=float("nan")), 1),
    (dict(ws=None), 4),
    (dict(wsb=8), 4),
    (dict(ws=FAKE + 4), 1),
])
def test_sample_argument_errors(lib, kw, status):
    assert call_sample(lib, **kw) == status


def call_diag(lib, **kw):
    args = dict(t=FAKE, tsb=400, tsk=100, d=FAKE, dsb=300, dsk=100, dtype=1, B=4, K=3, V=100, temp=None,
                temp_s=1.0, out=FAKE, g=None, pr=None, ws=FAKE, wsb=1 << 30, stream=None)
    args.update(kw)
    return lib.spec_diagnostics(*[args[k] for k in ("t", "tsb", "tsk", "d", "dsb", "dsk", "dtype", "B", "K", "V",
                                                    "temp", "temp_s", "out", "g", "pr", "ws", "wsb", "stream")])


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=2), 2),
    (dict(K=9), 2),
    (dict(B=0), 1),
    (dict(K=0), 1),
    (dict(V=0), 1),
    (dict(t=None), 1),
    (dict(d=None), 1),
    (dict(out=None), 1),
    (dict(dsb=-3), 1),
    (dict(temp_s=0.0), 1),
    (dict(ws=None), 4),
    (dict(wsb=16), 4),
])
def test_diagnostics_argument_errors(lib, kw, status):
    assert call_diag(lib, **kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), 2),
    (dict(K=9), 2),
    (dict(B=0), 1),
    (dict(t=None), 1),
    (dict(ids=None), 1),
    (dict(temp_s=0.0), 1),
    (dict(ws=None), 4),
    (dict(wsb=64), 4),
])
def test_verify_gumbel_argument_errors(lib, kw, status):
    args = dict(t=FAKE, tsb=400, tsk=100, d=FAKE, dsb=300, dsk=100, dtype=1, B=4, K=3, V=100, ids=FAKE,
                temp=None, temp_s=1.0, seed=0, off=0, acc=FAKE, em=FAKE, ov=None, p=None, q=None,
                lzt=None, lzd=None, ws=FAKE, wsb=1 << 30, stream=None)
    args.update(kw)
    assert lib.spec_verify_gumbel(*[args[k] for k in ("t", "tsb", "tsk", "d", "dsb", "dsk", "dtype", "B", "K", "V",
                                                      "ids", "temp", "temp_s", "seed", "off", "acc", "em", "ov", "p",
                                                      "q", "lzt", "lzd", "ws", "wsb", "stream")]) == status


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=5), 2),
    (dict(R=0), 1),
    (dict(V=0), 1),
    (dict(z=None), 1),
    (dict(tok=None), 1),
    (dict(temp_s=-0.5), 1),
    (dict(ws=None), 4),
    (dict(wsb=8), 4),
    (dict(ws=FAKE + 4), 1),
])
def test_sample_gumbel_argument_errors(lib, kw, status):
    args = dict(z=FAKE, sr=100, dtype=1, R=4, V=100, temp=None, temp_s=1.0, seed=0, off=0, tok=FAKE,
                ws=FAKE, wsb=1 << 30, stream=None)
    args.update(kw)
    assert lib.spec_sample_gumbel(*[args[k] for k in ("z", "sr", "dtype", "R", "V", "temp", "temp_s", "seed", "off",
                                                      "tok", "ws", "wsb", "stream")]) == status


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=3), 2),
    (dict(K=9), 2),
    (dict(N=0), 1),
    (dict(V=-5), 1),
    (dict(t=None), 1),
    (dict(loss=None), 1),
    (dict(T=0.0), 1),
    (dict(T=float("inf")), 1),
    (dict(kind=3), 1),
    (dict(kind=-1), 1),
    (dict(scale=float("nan")), 1),
    (dict(dsk=-1), 1),
    (dict(ws=None), 4),
    (dict(wsb=100), 4),
])
def test_kl_argument_errors(lib, kw, status):
    args = dict(t=FAKE, tsn=300, tsk=100, d=FAKE, dsn=300, dsk=100, dtype=1, N=4, K=3, V=100, T=1.0, kind=0,
                scale=1.0, loss=FAKE, ps=None, grad=None, ws=FAKE, wsb=1 << 30, stream=None)
    args.update(kw)
    assert lib.spec_kl_loss_fwd_bwd(*[args[k] for k in ("t", "tsn", "tsk", "d", "dsn", "dsk", "dtype", "N", "K", "V",
                                                        "T", "kind", "scale", "loss", "ps", "grad", "ws", "wsb",
                                                        "stream")]) == status


C_CLIENT = r"""
#include <stdio.h>
#include "specverify.h"
int main(void) {
  const int32_t ids[1] = {0};
  printf("%d\n", spec_version());
  printf("%s\n", spec_status_string(SPEC_EINVAL));
  printf("%zu\n", spec_verify_workspace_size(256, 3, 151936, SPEC_BF16));
  printf("%zu\n", spec_tv_workspace_size(16384, 3, 151936, SPEC_BF16));
  /* rejected before any GPU work: no logits */
  printf("%d\n", (int)spec_verify(NULL, 0, 0, NULL, 0, 0, SPEC_BF16, 1, 1, 8, ids, NULL, 1.0f, 0u, 0u,
                                  NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL));
  return 0;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs a C compiler")
def test_c99_client_links_and_calls(lib, tmp_path):
    """A C99 program (no C++, no torch) compiled against include/specverify.h
    with -pedantic -Werror, linked to the built library, sees the same
    version, status strings and workspace sizes as the Python binding and
    gets the synchronous argument error."""
    src = tmp_path / "client.c"
    src.write_text(C_CLIENT)
    exe = tmp_path / "client"
    libdir = os.path.dirname(os.path.abspath(lib._name))
    cmd = ["gcc", "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror", "-I" + os.path.join(ROOT, "include"),
           str(src), "-o", str(exe), "-L" + libdir, "-lspecverify", "-Wl,-rpath," + libdir]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    out = r.stdout.split("\n")
    lib.spec_status_string.restype = ctypes.c_char_p
    assert int(out[0]) == lib.spec_version()
    assert out[1] == lib.spec_status_string(1).decode()
    assert int(out[2]) == lib.spec_verify_workspace_size(256, 3, 151936, 1)
    assert int(out[3]) == lib.spec_tv_workspace_size(16384, 3, 151936, 1)
    assert int(out[4]) == 1  # SPEC_EINVAL


def test_verify_noalloc_limits_without_a_gpu(lib):
    """The scratch array's size is reported, a shape beyond it is refused and
    argument errors are returned, all before the GPU is touched."""
    assert lib.spec_verify_noalloc_max_workspace() == 32 << 20
    big = lib.spec_verify_noalloc(FAKE, 1 << 22, 1 << 18, FAKE, 1 << 22, 1 << 18, 1, 4096, 8, 262144, FAKE, None,
                                  1.0, 0, 0, FAKE, FAKE, None, None, None, None, None, None)
    assert big == 4  # SPEC_EWORKSPACE
    assert lib.spec_verify_noalloc(None, 400, 100, FAKE, 300, 100, 1, 4, 3, 100, FAKE, None, 1.0, 0, 0, FAKE, FAKE,
                                   None, None, None, None, None, None) == 1
    assert lib.spec_verify_noalloc(FAKE, 400, 100, FAKE, 300, 100, 1, 4, 9, 100, FAKE, None, 1.0, 0, 0, FAKE, FAKE,
                                   None, None, None, None, None, None) == 2
