"""The C-ABI library: it loads, exports every symbol include/snn_lif.h declares, and its
host-side logic (sizes, argument validation, empty problems) behaves as documented.
CPU only: nothing here launches a kernel (every call is rejected, or is empty, before
any HIP call)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "snn_lif.h")


@pytest.fixture(scope="module")
def nat():
    from paper_2408_00280_amd import native
    return native


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(snn_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(nat):
    declared = declared_functions()
    assert declared == sorted(nat.EXPORTS)
    for name in declared:
        assert hasattr(nat.lib, name), name
    out = os.popen(f"nm -D --defined-only {nat.LIB_PATH}").read()
    for name in declared:
        assert re.search(rf"\bT {name}\b", out), name


def test_library_has_gfx950_code(nat):
    data = open(nat.LIB_PATH, "rb").read()
    assert b"gfx950" in data


def test_status_strings(nat):
    for s in range(-6, 1):
        assert nat.snn_status_str(s) != "unknown status"
    assert nat.snn_status_str(-99) == "unknown status"


def test_size_formulas(nat):
    cfg8 = nat.make_cfg(0.5, 1.0, spk="u8")
    cfgb = nat.make_cfg(0.5, 1.0, spk="bits")
    for N in (0, 1, 63, 64, 65, 1000, 8388608):
        assert nat.snn_spike_row_bytes(cfg8, N) == N
        assert nat.snn_spike_row_bytes(cfgb, N) == 8 * ((N + 63) // 64)
    # checkpoints: one fp32 row of N per chunk boundary; chunks hold 8 to 32 steps depending
    # on the lane plan, so short layers need none and the size grows with T
    for io in ("f32", "bf16"):
        c = nat.make_cfg(0.5, 1.0, io=io)
        for N in (1, 4097, 4096, 131072, 524288, 1 << 24):
            sizes = [nat.snn_lif_saved_bytes(c, T, N) for T in range(0, 300, 7)]
            assert all(sz % (4 * N) == 0 for sz in sizes)
            assert sizes == sorted(sizes)
            for T in (1, 8, 16):
                assert nat.snn_lif_saved_bytes(c, T, N) == 0
            for T in (33, 100, 256):
                chunks = nat.snn_lif_saved_bytes(c, T, N) // (4 * N) + 1
                assert -(-T // 32) <= chunks <= -(-T // 8)
        # large layers use 16-step chunks (fp32) or 32-step chunks (bf16)
        K = 16 if io == "f32" else 32
        assert nat.snn_lif_saved_bytes(c, 256, 1 << 24) == (256 // K - 1) * (1 << 24) * 4
        assert nat.snn_lif_saved_bytes(c, 0, 4096) == 0
        assert nat.snn_lif_saved_bytes(c, 100, 0) == 0


BAD_CFGS = [
    dict(decay=-0.1), dict(decay=1.5), dict(decay=float("nan")), dict(v_th=float("inf")),
    dict(v_th=float("nan")), dict(v_reset=float("-inf")), dict(alpha=0.0), dict(alpha=-1.0),
    dict(alpha=float("inf")), dict(reset=2), dict(io=7), dict(spk=-1),
]


@pytest.mark.parametrize("bad", BAD_CFGS, ids=lambda d: ",".join(f"{k}={v}" for k, v in d.items()))
def test_bad_params_rejected(nat, bad):
    args = dict(decay=0.5, v_th=1.0, v_reset=0.0, alpha=4.0, reset=0, io=0, spk=0)
    args.update(bad)
    cfg = nat.snn_lif_cfg(args["decay"], args["v_th"], args["v_reset"], args["alpha"], args["reset"],
                          args["io"], args["spk"])
    fake = 0x10000   # never dereferenced: validation fails before any launch
    for call in (lambda: nat.snn_lif_forward(cfg, 4, 64, fake, fake, None, None, 0),
                 lambda: nat.snn_lif_backward(cfg, 4, 64, fake, None, fake, fake, 0),
                 lambda: nat.snn_lif_saved_bytes(cfg, 4, 64),
                 lambda: nat.snn_spike_row_bytes(cfg, 64),
                 lambda: nat.snn_gain_spikes_forward(cfg, 4, 2, 32, fake, fake, fake, 0),
                 lambda: nat.snn_gain_grad_backward(cfg, 4, 2, 32, fake, fake, fake, 0)):
        with pytest.raises(nat.SnnError) as e:
            call()
        assert e.value.status == -3


def test_null_cfg(nat):
    st = nat.lib.snn_lif_forward(None, 4, 64, 0x10000, 0x10000, None, None, None)
    assert st == -1
    sz = ctypes.c_size_t(0)
    assert nat.lib.snn_lif_saved_bytes(None, 4, 64, ctypes.byref(sz)) == -1
    cfg = nat.make_cfg(0.5, 1.0)
    assert nat.lib.snn_lif_saved_bytes(ctypes.byref(cfg), 4, 64, None) == -1


def test_shape_errors(nat):
    cfg = nat.make_cfg(0.5, 1.0)
    fake = 0x10000
    for T, N in ((-1, 64), (4, -1), (2 ** 31, 64), (4, 2 ** 31 + 1), (2 ** 20, 2 ** 30)):
        with pytest.raises(nat.SnnError) as e:
            nat.snn_lif_forward(cfg, T, N, fake, fake, fake, None, 0)
        assert e.value.status == -2
        with pytest.raises(nat.SnnError) as e:
            nat.snn_lif_backward(cfg, T, N, fake, fake, fake, fake, 0)
        assert e.value.status == -2
    with pytest.raises(nat.SnnError) as e:
        nat.snn_gain_spikes_forward(cfg, 4, -2, 32, fake, fake, fake, 0)
    assert e.value.status == -2


def test_null_and_alignment_errors(nat):
    cfg = nat.make_cfg(0.5, 1.0)
    a = 0x10000
    cases = [
        (lambda: nat.snn_lif_forward(cfg, 4, 64, None, a, None, None, 0), -1),
        (lambda: nat.snn_lif_forward(cfg, 4, 64, a, None, None, None, 0), -1),
        (lambda: nat.snn_lif_forward(cfg, 40, 64, a, a, None, None, 0), -1),   # checkpoints needed
        (lambda: nat.snn_lif_forward(cfg, 4, 64, a + 4, a, None, None, 0), -4),
        (lambda: nat.snn_lif_forward(cfg, 4, 64, a, a + 8, None, None, 0), -4),
        (lambda: nat.snn_lif_forward(cfg, 4, 64, a, a, None, a + 2, 0), -4),
        (lambda: nat.snn_lif_backward(cfg, 4, 64, a, None, None, a, 0), -1),
        (lambda: nat.snn_lif_backward(cfg, 4, 64, a, None, a, None, 0), -1),
        (lambda: nat.snn_lif_backward(cfg, 40, 64, a, None, a, a, 0), -1),
        (lambda: nat.snn_lif_backward(cfg, 4, 64, a, None, a, a + 4, 0), -4),
        (lambda: nat.snn_gain_spikes_forward(cfg, 4, 2, 32, a, None, a, 0), -1),
        (lambda: nat.snn_gain_grad_backward(cfg, 4, 2, 32, a, a, a + 1, 0), -4),
    ]
    for call, status in cases:
        with pytest.raises(nat.SnnError) as e:
            call()
        assert e.value.status == status


def test_empty_problems_are_noops(nat):
    """T == 0 or N == 0: OK without launching anything, pointers unused."""
    cfg = nat.make_cfg(0.5, 1.0)
    nat.snn_lif_forward(cfg, 0, 64, None, None, None, None, 0)
    nat.snn_lif_forward(cfg, 8, 0, None, None, None, None, 0)
    nat.snn_lif_backward(cfg, 0, 64, None, None, None, None, 0)
    nat.snn_lif_backward(cfg, 8, 0, None, None, None, None, 0)
    nat.snn_gain_spikes_forward(cfg, 8, 0, 32, None, None, None, 0)
    nat.snn_gain_grad_backward(cfg, 0, 2, 32, None, None, None, 0)


def test_c_client_links():
    """The plain-C client builds against the header and links the library, the oracle, the
    generator and the HIP runtime (running it needs the GPU)."""
    import subprocess

    from tests import c_abi
    c_abi.build()
    out = subprocess.run(["ldd", c_abi.BIN], capture_output=True, text=True).stdout
    assert "not found" not in out
    for lib in ("libsnnlif.so", "liboracle.so", "libsynth.so", "libamdhip64"):
        assert lib in out, lib


@pytest.mark.parametrize("compiler,flags,ext", [("gcc", ["-std=c99"], "c"), ("g++", ["-std=c++11"], "cc")])
def test_header_is_plain_c_and_cxx(tmp_path, compiler, flags, ext):
    """include/snn_lif.h compiles on its own, warning-free and pedantic, as C99 and as C++11
    (no HIP or torch types in the interface)."""
    import shutil
    import subprocess
    if shutil.which(compiler) is None:
        pytest.skip(f"{compiler} not available")
    src = tmp_path / f"use.{ext}"
    src.write_text('#include "snn_lif.h"\n'
                   "snn_status probe(const snn_lif_cfg *c, size_t *b) { return snn_lif_saved_bytes(c, 4, 64, b); }\n")
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    r = subprocess.run([compiler, *flags, "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only", "-I", inc, str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
