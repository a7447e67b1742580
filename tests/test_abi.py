"""The C-ABI library loads, exports what include/fdllm.h declares, and its
host-side argument checks reject bad calls without touching a GPU."""
import ctypes
import os
import re

import pytest

import paper_2606_02955_amd as fd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fdllm.h")


BENCH_HEADER = os.path.join(ROOT, "include", "fdllm_bench.h")


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fdllm_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fd.LIB_PATH):
        from paper_2606_02955_amd import build
        build.build()
    return fd.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(fd.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for st in (0, -1, -2, -3, -4, -5, -6, -7, -8, -9):
        assert len(fd.status_string(st)) > 0
        assert "unknown" not in fd.status_string(st)
    assert fd.status_string(0) == "ok"
    assert "unknown" in fd.status_string(99)


def test_workspace_size_host_only(lib):
    n = ctypes.c_size_t(123)
    assert lib.fdllm_workspace_size(1024, 32, 126464, 0, ctypes.byref(n)) == 0
    assert n.value == 0                      # large batches run fused: no workspace
    assert lib.fdllm_workspace_size(8, 32, 126464, 0, ctypes.byref(n)) == 0
    assert n.value >= 3 * 8 * 32 * 4
    assert lib.fdllm_workspace_size(8, 32, 126464, 7, ctypes.byref(n)) == fd.ERR_UNSUPPORTED_DTYPE
    assert lib.fdllm_workspace_size(8, 32, 0, 0, ctypes.byref(n)) == fd.ERR_SIZE
    assert lib.fdllm_workspace_size(-1, 32, 10, 0, ctypes.byref(n)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_workspace_size(8, 32, 10, 0, None) == fd.ERR_INVALID_ARG


def test_error_paths_enqueue_nothing(lib):
    p = ctypes.c_void_p(0x1000)            # never dereferenced: checks fail first
    null = None
    # confidence: null logits / tokens / conf, bad dtype, bad sizes
    assert lib.fdllm_confidence(null, 0, 2, 4, 16, p, p, p, p, p, null, null, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_confidence(p, 0, 2, 4, 16, p, p, p, null, p, null, null, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_confidence(p, 0, 2, 4, 16, p, p, p, p, null, null, null, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_confidence(p, 5, 2, 4, 16, p, p, p, p, p, null, null, null) == fd.ERR_UNSUPPORTED_DTYPE
    assert lib.fdllm_confidence(p, 0, 2, 4, 0, p, p, p, p, p, null, null, null) == fd.ERR_SIZE
    assert lib.fdllm_confidence(p, 0, -2, 4, 16, p, p, p, p, p, null, null, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_confidence(p, 0, 2, 0, 16, p, p, p, p, p, null, null, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_confidence(p, 0, 1 << 30, 1 << 30, 1 << 30, p, p, p, p, p, null, null, null) == fd.ERR_SIZE
    # B == 0 is a no-op
    assert lib.fdllm_confidence(null, 0, 0, 4, 16, null, null, null, null, null, null, null, null) == 0
    # selectors: conf, mask, bounds and commit are required
    for name in ("fdllm_select_profile", "fdllm_select_factor", "fdllm_select_threshold"):
        f = getattr(lib, name)
        assert f(null, null, p, p, p, 2, 4, 1.0, p, null, null) == fd.ERR_INVALID_ARG
        assert f(p, null, p, p, p, 2, 4, 1.0, null, null, null) == fd.ERR_INVALID_ARG
        assert f(p, null, null, p, p, 2, 4, 1.0, p, null, null) == fd.ERR_INVALID_ARG
        assert f(p, null, p, p, p, 2, 0, 1.0, p, null, null) == fd.ERR_INVALID_ARG
        assert f(null, null, null, null, null, 0, 4, 1.0, null, null, null) == 0
    f = lib.fdllm_select_robust
    assert f(null, null, null, 0.0, p, p, p, 2, 4, 1.0, p, null, null) == fd.ERR_INVALID_ARG
    assert f(p, null, null, 0.0, p, p, p, 2, 4, 1.0, null, null, null) == fd.ERR_INVALID_ARG
    assert f(p, null, null, float("nan"), p, p, p, 2, 4, 1.0, p, null, null) == fd.ERR_INVALID_ARG
    assert f(null, null, null, 0.1, null, null, null, 0, 4, 1.0, null, null, null) == 0
    assert lib.fdllm_reveal(null, p, p, p, 2, 4, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_reveal(p, p, p, p, -1, 4, null) == fd.ERR_INVALID_ARG
    # decode step: bad selector, dtype, null in/out arrays, missing workspace
    args = lambda **kw: [kw.get("logits", p), kw.get("dt", 0), kw.get("B", 8), 32, kw.get("V", 64),
                         kw.get("mask", p), p, p, kw.get("x", p), kw.get("sel", 2), 1.0,
                         null, kw.get("eta_u", 0.0),
                         null, null, null, null, null, null, kw.get("ws", null), kw.get("wsb", 0), null]
    assert lib.fdllm_decode_step(*args(sel=4)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_decode_step(*args(sel=-1)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_decode_step(*args(sel=3, eta_u=float("nan"))) == fd.ERR_INVALID_ARG
    assert lib.fdllm_decode_step(*args(dt=9)) == fd.ERR_UNSUPPORTED_DTYPE
    assert lib.fdllm_decode_step(*args(logits=null)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_decode_step(*args(mask=null)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_decode_step(*args(x=null)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_decode_step(*args(V=0)) == fd.ERR_SIZE
    assert lib.fdllm_decode_step(*args()) == fd.ERR_WORKSPACE            # B=8: two-kernel plan
    assert lib.fdllm_decode_step(*args(ws=p, wsb=16)) == fd.ERR_WORKSPACE


def test_check_inputs_error_paths(lib):
    p = ctypes.c_void_p(0x1000)
    null = None
    f = lib.fdllm_check_inputs
    assert f(p, 0, 2, 4, 16, p, p, p, null, null) == fd.ERR_INVALID_ARG        # counts required
    assert f(null, 0, 2, 4, 16, p, p, p, p, null) == fd.ERR_INVALID_ARG
    assert f(p, 0, 2, 4, 16, null, p, p, p, null) == fd.ERR_INVALID_ARG
    assert f(p, 3, 2, 4, 16, p, p, p, p, null) == fd.ERR_UNSUPPORTED_DTYPE
    assert f(p, 0, 2, 4, 0, p, p, p, p, null) == fd.ERR_SIZE
    assert f(p, 0, -1, 4, 16, p, p, p, p, null) == fd.ERR_INVALID_ARG


def test_static_decode_step_error_paths(lib):
    p = ctypes.c_void_p(0x1000)
    null = None
    args = lambda **kw: [kw.get("logits", p), kw.get("dt", 0), kw.get("B", 8), kw.get("L", 32),
                         kw.get("V", 64), kw.get("mask", p), p, p, kw.get("x", p), kw.get("sel", 2),
                         1.0, null, kw.get("eta_u", 0.0), null, null, null, null, null, null, null]
    f = lib.fdllm_decode_step_static
    assert f(*args(sel=7)) == fd.ERR_INVALID_ARG
    assert f(*args(sel=3, eta_u=float("nan"))) == fd.ERR_INVALID_ARG
    assert f(*args(dt=9)) == fd.ERR_UNSUPPORTED_DTYPE
    assert f(*args(logits=null)) == fd.ERR_INVALID_ARG
    assert f(*args(x=null)) == fd.ERR_INVALID_ARG
    assert f(*args(V=0)) == fd.ERR_SIZE
    # a small batch over a long span needs 12 B per slot of scratch: beyond the static array
    assert f(*args(B=64, L=100000)) == fd.ERR_SCRATCH
    assert f(*args(B=0)) == 0


def test_constants_agree_with_header():
    text = open(HEADER).read()
    m = re.search(r"#define FDLLM_MAX_ABS_LOGIT ([0-9.e]+)f", text)
    assert m and float(m.group(1)) == fd.MAX_ABS_LOGIT
    m = re.search(r"#define FDLLM_STATIC_SCRATCH_BYTES \(8u << 20\)", text)
    assert m and fd.STATIC_SCRATCH_BYTES == 8 << 20
    for name, val in (("BOUNDS", fd.ERR_BOUNDS), ("BLOCK_TOO_LARGE", fd.ERR_BLOCK_TOO_LARGE),
                      ("NONFINITE", fd.ERR_NONFINITE), ("SCRATCH", fd.ERR_SCRATCH)):
        assert re.search(rf"#define FDLLM_ERR_{name} \({val}\)", text), name


def test_binding_refuses_cpu_tensors(lib):
    import torch
    lg = torch.zeros(1, 2, 8, dtype=torch.bfloat16)
    m = torch.ones(1, 2, dtype=torch.uint8)
    b = torch.zeros(1, dtype=torch.int32)
    with pytest.raises(ValueError):
        fd.fdllm_confidence(lg, m, b, b + 2, torch.zeros(1, 2, dtype=torch.int32),
                            torch.zeros(1, 2))


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(FileNotFoundError):
        fd.load(str(tmp_path / "libfdllm.so"))


def test_block_limit_agrees_with_header():
    text = open(HEADER).read()
    m = re.search(r"#define\s+FDLLM_MAX_BLOCK\s+(\d+)", text)
    import parity
    assert m and int(m.group(1)) == fd.MAX_BLOCK == parity.MAX_BLOCK


def test_bench_library_exports_and_checks(lib):
    blib = fd.load_bench()
    names = declared_functions(BENCH_HEADER)
    assert set(names) == set(fd.BENCH_EXPORTS), names
    p = ctypes.c_void_p(0x1000)
    assert blib.fdllm_stream_read(None, 0, None, None) == 0          # empty: no-op
    assert blib.fdllm_stream_read(None, 32, p, None) == -1
    assert blib.fdllm_stream_read(p, 32, None, None) == -1
    assert blib.fdllm_stream_read(p, 24, p, None) == -1              # not a multiple of 16
    assert blib.fdllm_stream_read(ctypes.c_void_p(0x1008), 32, p, None) == -1   # misaligned


def test_generation_desc_layout_matches_header(tmp_path):
    """The ctypes mirror of fdllm_generation_desc has the C compiler's layout."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    names = [f for f, _ in fd.GenerationDesc._fields_]
    src = tmp_path / "layout.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "fdllm.h"\nint main(void) {\n'
                   + f'  printf("%zu\\n", sizeof(fdllm_generation_desc));\n'
                   + "".join(f'  printf("%zu\\n", offsetof(fdllm_generation_desc, {n}));\n' for n in names)
                   + "  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    out = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    assert out[0] == ctypes.sizeof(fd.GenerationDesc)
    assert out[1:] == [getattr(fd.GenerationDesc, n).offset for n in names]


def test_loop_entry_points_check_arguments(lib):
    p = ctypes.c_void_p(0x1000)
    null = None
    assert lib.fdllm_synth_logits(null, 2, 8, 16, 4, p, p, 1, 0, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_synth_logits(p, 2, 8, 16, 0, p, p, 1, 0, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_synth_logits(p, 2, 8, 16, 2000, p, p, 1, 0, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_synth_logits(p, 2, 8, 16, 4, p, p, 1, -1, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_synth_logits(null, 0, 8, 16, 4, null, null, 1, 0, null) == 0
    assert lib.fdllm_advance_blocks(null, p, p, 2, 8, 4, null, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_advance_blocks(p, p, p, 2, 0, 4, null, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_advance_blocks(null, null, null, 0, 8, 4, null, null) == 0
    d = fd.GenerationDesc()
    d.B, d.G, d.blk, d.V, d.seed, d.sel, d.param = 4, 64, 16, 100, 1, fd.SEL_PROFILE, 1.0
    d.max_steps, d.chunk, d.use_graph = 64, 4, 1
    n = ctypes.c_size_t(0)
    assert lib.fdllm_generation_workspace_size(ctypes.byref(d), ctypes.byref(n)) == fd.ERR_INVALID_ARG
    for f in ("logits", "mask", "x", "block_start", "block_end"):
        setattr(d, f, 0x1000)
    assert lib.fdllm_generation_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    assert n.value >= 3 * 4 * 64 * 4                 # B=4 < 256: decode scratch included
    h = ctypes.c_void_p(0)
    assert lib.fdllm_generation_create(ctypes.byref(d), ctypes.byref(h)) == fd.ERR_WORKSPACE
    assert not h.value
    d.sel = 7
    assert lib.fdllm_generation_create(ctypes.byref(d), ctypes.byref(h)) == fd.ERR_INVALID_ARG
    d.sel, d.blk = fd.SEL_PROFILE, 2048
    assert lib.fdllm_generation_workspace_size(ctypes.byref(d), ctypes.byref(n)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_generation_run(null, null, null) == fd.ERR_INVALID_ARG
    assert lib.fdllm_generation_destroy(null) == 0


def test_lmhead_entry_points_check_arguments(lib):
    p = ctypes.c_void_p(0x1000)
    null = None
    n = ctypes.c_size_t(0)
    assert lib.fdllm_lmhead_workspace_size(4, 32, 4096, 126464, ctypes.byref(n)) == 0
    assert n.value >= 4 * 32 * 4                     # row list at least
    assert lib.fdllm_lmhead_workspace_size(4, 32, 100, 1000, ctypes.byref(n)) == fd.ERR_SIZE   # d % 64
    assert lib.fdllm_lmhead_workspace_size(4, 32, 0, 1000, ctypes.byref(n)) == fd.ERR_SIZE
    assert lib.fdllm_lmhead_workspace_size(4, 32, 64, 0, ctypes.byref(n)) == fd.ERR_SIZE
    assert lib.fdllm_lmhead_workspace_size(4, 32, 64, 10, None) == fd.ERR_INVALID_ARG
    # hidden states beyond 32-bit byte offsets (2^16 * 64 * 512 * 2 bytes = 4 GiB)
    assert lib.fdllm_lmhead_workspace_size(1 << 16, 64, 512, 1000, ctypes.byref(n)) == fd.ERR_SIZE
    assert lib.fdllm_lmhead_workspace_size((1 << 16) - 1, 64, 512, 1000, ctypes.byref(n)) == 0
    args = lambda **kw: [kw.get("h", p), kw.get("w", p), 2, 8, kw.get("d", 64), 100, kw.get("m", p), p, p,
                         kw.get("tok", p), kw.get("conf", p), null, null, kw.get("ws", p),
                         kw.get("wsb", 1 << 30), null]
    assert lib.fdllm_lmhead_confidence(*args(h=null)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_lmhead_confidence(*args(w=null)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_lmhead_confidence(*args(m=null)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_lmhead_confidence(*args(tok=null)) == fd.ERR_INVALID_ARG
    assert lib.fdllm_lmhead_confidence(*args(d=96)) == fd.ERR_SIZE
    assert lib.fdllm_lmhead_confidence(*args(h=ctypes.c_void_p(0x1008))) == fd.ERR_INVALID_ARG  # alignment
    assert lib.fdllm_lmhead_confidence(*args(ws=null, wsb=0)) == fd.ERR_WORKSPACE
    assert lib.fdllm_lmhead_confidence(*args(wsb=64)) == fd.ERR_WORKSPACE
    dargs = [p, p, 2, 8, 64, 100, p, p, p, p, 9, 1.0, null, 0.0, null, null, null, null, null, null,
             p, 1 << 30, null]
    assert lib.fdllm_lmhead_decode_step(*dargs) == fd.ERR_INVALID_ARG          # selector 9
    dargs[10] = 2
    dargs[9] = None
    assert lib.fdllm_lmhead_decode_step(*dargs) == fd.ERR_INVALID_ARG          # x missing


def _ws(fn, *args):
    n = ctypes.c_size_t(0)
    assert fn(*args, ctypes.byref(n)) == 0
    return n.value


def test_workspace_sizes_follow_the_plans(lib):
    """Host planning, seen through the workspace queries: small batches with
    blocks of at most one wavefront reserve room for the rows' wave partials
    (24 bytes each); the LM head's two-part plan (33..64 positions, d a
    multiple of 1024) reserves the two halves' partial logits."""
    V = 126464
    # decode step: B=1, L=32 bf16 rows split 16 ways -> 32 x 16 partials
    small = _ws(lib.fdllm_workspace_size, 1, 32, V, 0)
    assert small >= 3 * 32 * 4 + 32 * 16 * 24
    # a long span (L > 64) keeps single-workgroup rows: outputs only
    assert _ws(lib.fdllm_workspace_size, 8, 256, V, 0) < 3 * 8 * 256 * 4 + 1024 * 3
    # one workgroup per sequence (no workspace) from 256 sequences on
    assert _ws(lib.fdllm_workspace_size, 255, 32, V, 0) >= 3 * 255 * 32 * 4
    assert _ws(lib.fdllm_workspace_size, 256, 32, V, 0) == 0
    # LM head: up to 32 positions need no partial logits
    s32 = _ws(lib.fdllm_lmhead_workspace_size, 1, 32, 4096, V)
    assert s32 < 4 << 20
    # 64 positions: 2 halves x V x 64 float32 partial logits
    s64 = _ws(lib.fdllm_lmhead_workspace_size, 2, 32, 4096, V)
    assert s64 >= 2 * V * 64 * 4
    # 64 positions with d not a multiple of 1024: the tiled plan, no partial logits
    assert _ws(lib.fdllm_lmhead_workspace_size, 2, 32, 4032, V) < 2 * V * 64 * 4
    # 65 positions: the tiled plan
    assert _ws(lib.fdllm_lmhead_workspace_size, 1, 65, 4096, V) < 2 * V * 64 * 4
