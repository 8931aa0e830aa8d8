"""The C-ABI library loads, exports what include/turnkl.h declares, and rejects
bad arguments on the host before anything is enqueued (no GPU needed: every
call here returns before the first HIP runtime call)."""
import ctypes
import os
import re

import pytest

from paper_2607_05804_amd import turnkl as T

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "turnkl.h")
TESTING_HEADER = os.path.join(ROOT, "include", "turnkl_testing.h")


def declared_functions(path=HEADER):
    src = open(path).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(turnkl_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert set(names) == set(T.EXPORTS), names
    testing = declared_functions(TESTING_HEADER)
    assert set(testing) == set(T.TESTING_EXPORTS), testing
    assert not set(names) & set(testing)  # the product header declares no test hook
    lib = ctypes.CDLL(T.LIB_PATH)
    for n in names + testing:
        assert hasattr(lib, n), n


def test_status_strings_and_alpha_schedule():
    assert T.status_string(T.OK) == "ok"
    for code in range(-11, 0):
        assert T.status_string(code) != "unknown status"
    assert T.status_string(-99) == "unknown status"
    assert T.alpha_schedule(0, 100) == 0.0
    assert T.alpha_schedule(50, 100) == 0.5
    assert T.alpha_schedule(150, 100) == 1.0
    assert T.alpha_schedule(3, 10, 0.2, 0.6) == pytest.approx(0.25)
    assert T.alpha_schedule(5, 10, 0.6, 0.6) == 0.0 and T.alpha_schedule(6, 10, 0.6, 0.6) == 1.0
    import math
    assert math.isnan(T.alpha_schedule(1, 0))


def _ws(n, v, dtype, max_turns, aligned):
    return int(T.lib().turnkl_workspace_bytes(n, v, dtype, max_turns, aligned))


def test_workspace_bytes_sized_for_the_path_the_call_takes():
    """With aligned rows the workspace holds the 16-byte vector path's
    exchange slots only (4 words of 8 bytes per chunk, 3 chunks per row at
    V = 151,936 in bf16); without, also the element-wise path's (19 chunks).
    The size is a pure function of the arguments: a tiling override of the
    calling thread changes only turnkl_testing_workspace_bytes."""
    n, v = 65536, 151936
    aligned, unaligned = _ws(n, v, T.BF16, 50, 1), _ws(n, v, T.BF16, 50, 0)
    assert aligned <= 15_000_000  # the long-horizon batch's workspace
    assert unaligned - aligned == n * (19 - 3) * 32
    # a vocabulary without whole 16-byte vectors only ever takes the element-wise path
    assert _ws(n, v + 1, T.BF16, 50, 1) == _ws(n, v + 1, T.BF16, 50, 0)
    # one chunk per row: no slots on either path
    assert _ws(1000, 1024, T.BF16, 8, 1) == _ws(1000, 1024, T.BF16, 8, 0)
    lib = T.lib()
    T.set_row_tiling(3)
    try:
        assert _ws(n, v, T.BF16, 50, 1) == aligned
        t = int(lib.turnkl_testing_workspace_bytes(n, v, T.BF16, 50, 1, 3))
        assert t == aligned + n * (25 - 3) * 32  # 3 packs per thread: 25 chunks per row
        assert T.workspace_bytes(n, v, T.BF16, 50) == t  # the binding follows the override
    finally:
        T.set_row_tiling(0)
    assert int(lib.turnkl_testing_workspace_bytes(n, v, T.BF16, 50, 1, 0)) == aligned
    assert int(lib.turnkl_testing_workspace_bytes(n, v, T.BF16, 50, 1, 26)) == 0
    # the stress batch fits the no-allocation entry point's scratch
    assert _ws(131072, v, T.BF16, 200, 1) <= T.NOALLOC_SCRATCH_BYTES


def test_workspace_bytes():
    assert T.workspace_bytes(-1, 10, T.BF16, 4) == 0
    assert T.workspace_bytes(10, 0, T.BF16, 4) == 0
    assert T.workspace_bytes(10, 10, 7, 4) == 0
    assert T.workspace_bytes(10, 10, T.BF16, 0) == 0
    assert T.workspace_bytes(10, 10, T.BF16, (2**31 - 2) // 3 + 1) == 0
    # the per-turn survivor counts of the support floor grow with max_turns
    assert T.workspace_bytes(10, 10, T.BF16, 4096) > T.workspace_bytes(10, 10, T.BF16, 4)
    a = T.workspace_bytes(1000, 151936, T.BF16, 50)
    b = T.workspace_bytes(2000, 151936, T.BF16, 50)
    assert 0 < a < b and a % 256 == 0
    assert T.workspace_bytes(0, 10, T.F32, 1) > 0
    # smaller per-thread tiles mean more chunks per row and more exchange slots
    T.set_row_tiling(1)
    try:
        c = T.workspace_bytes(1000, 151936, T.BF16, 50)
    finally:
        T.set_row_tiling(0)
    assert c > a
    with pytest.raises(T.TurnKLError):
        T.set_row_tiling(26)
    with pytest.raises(T.TurnKLError):
        T.set_row_tiling(-1)
    with pytest.raises(T.TurnKLError):
        T.set_spin_limit(-1)
    T.set_spin_limit(5)
    T.set_spin_limit(0)


def _call(**kw):
    """turnkl_fwd_bwd with fake (never dereferenced) addresses unless overridden."""
    n, v = kw.get("n", 64), kw.get("v", 1024)
    es = 2 if kw.get("dtype", T.BF16) == T.BF16 else 4
    zs = kw.get("zs", 0x100000000)
    zt = kw.get("zt", 0x200000000)
    ws_bytes = T.workspace_bytes(n, v, kw.get("dtype", T.BF16), kw.get("max_turns", 8),
                                 kw.pop("aligned", True))
    args = dict(zs=zs, ld_s=v, zt=zt, ld_t=v, dtype=T.BF16, n=n, v=v, turn=0x300000000,
                traj=0x300100000, mask=0x300200000, alpha=0.5, scale=1.0, loss=0x300300000,
                grad=0x400000000, ld_g=v, stats=0, max_turns=8, acc=0, kl=0,
                ws=0x500000000, ws_bytes=ws_bytes, opts=None)
    args.update(kw)
    p = lambda x: ctypes.c_void_p(x) if x else None
    return T.lib().turnkl_fwd_bwd(
        p(args["zs"]), args["ld_s"], p(args["zt"]), args["ld_t"], args["dtype"], args["n"],
        args["v"], p(args["turn"]), p(args["traj"]), p(args["mask"]), args["alpha"],
        args["scale"], p(args["loss"]), p(args["grad"]), args["ld_g"], p(args["stats"]),
        args["max_turns"], args["acc"], p(args["kl"]), _opts(args["opts"]), p(args["ws"]),
        args["ws_bytes"], None)


def _opts(o):
    """(support_floor, support_frac, success, outcome_stats_out[, token_weight_out,
    token_lse_out]) -> turnkl_options*."""
    if o is None:
        return None
    o = tuple(o) + (0,) * (6 - len(o))
    return ctypes.byref(T.Options(o[0], o[1], o[2] or None, o[3] or None, o[4] or None,
                                  o[5] or None))


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=5), T.ERR_INVALID_ARG),
    (dict(n=-1), T.ERR_INVALID_ARG),
    (dict(v=0), T.ERR_INVALID_ARG),
    (dict(max_turns=0), T.ERR_INVALID_ARG),
    (dict(alpha=-0.1), T.ERR_INVALID_ARG),
    (dict(alpha=1.5), T.ERR_INVALID_ARG),
    (dict(alpha=float("nan")), T.ERR_INVALID_ARG),
    (dict(scale=float("inf")), T.ERR_INVALID_ARG),
    (dict(scale=float("nan")), T.ERR_INVALID_ARG),
    (dict(loss=0), T.ERR_INVALID_ARG),
    (dict(ws=0), T.ERR_INVALID_ARG),
    (dict(zs=0), T.ERR_INVALID_ARG),
    (dict(zt=0), T.ERR_INVALID_ARG),
    (dict(turn=0), T.ERR_INVALID_ARG),
    (dict(traj=0), T.ERR_INVALID_ARG),
    (dict(mask=0), T.ERR_INVALID_ARG),
    (dict(ld_s=1023), T.ERR_INVALID_ARG),
    (dict(ld_t=1000), T.ERR_INVALID_ARG),
    (dict(ld_g=1), T.ERR_INVALID_ARG),
    # gradient overlapping the teacher, or the student other than exactly in place
    (dict(grad=0x200000000), T.ERR_ALIAS),
    (dict(grad=0x200000000 + 64 * 1024), T.ERR_ALIAS),
    (dict(grad=0x100000000 + 2), T.ERR_ALIAS),
    (dict(grad=0x100000000, ld_g=2048), T.ERR_ALIAS),
    (dict(grad=0x100000000 - 2 * 1024), T.ERR_ALIAS),
    # workspace too small or misaligned; sized for aligned rows but given a
    # row stride that is not a whole number of 16-byte vectors (the
    # element-wise path, 19 chunks per row instead of 3)
    (dict(ws_bytes=1024), T.ERR_WORKSPACE),
    (dict(ws=0x500000010), T.ERR_WORKSPACE),
    (dict(v=151936, ld_s=151937, ld_t=151936, ld_g=151936), T.ERR_WORKSPACE),
    (dict(v=151936, ld_s=151936, ld_t=151936, ld_g=151936, zt=0x200000002), T.ERR_WORKSPACE),
    (dict(max_turns=(2**31 - 2) // 3 + 1), T.ERR_INVALID_ARG),
    # size limits: 128 chunks per row on the vector path (25 packs of 8 bf16 per
    # thread) and on the scalar path (32 elements per thread), 32-bit row
    # strides, token counts and task counts
    (dict(v=6553600 + 8, ld_s=6553608, ld_t=6553608, ld_g=6553608), T.ERR_INVALID_ARG),
    (dict(v=1048577, ld_s=1048577, ld_t=1048577, ld_g=1048577), T.ERR_INVALID_ARG),
    (dict(ld_s=2**31, grad=0), T.ERR_INVALID_ARG),
    (dict(n=2**31, grad=0), T.ERR_INVALID_ARG),
    (dict(n=2**24, v=6553600, ld_s=6553600, ld_t=6553600, grad=0), T.ERR_INVALID_ARG),
    # options: floor and fraction ranges; success flags and outcome statistics
    # go together; the outcome statistics must not overlap the turn statistics
    (dict(opts=(-1, 0.0, 0, 0)), T.ERR_INVALID_ARG),
    (dict(opts=(8, -0.1, 0, 0)), T.ERR_INVALID_ARG),
    (dict(opts=(8, 1.5, 0, 0)), T.ERR_INVALID_ARG),
    (dict(opts=(8, float("nan"), 0, 0)), T.ERR_INVALID_ARG),
    (dict(opts=(0, 0.0, 0x700000000, 0)), T.ERR_INVALID_ARG),
    (dict(opts=(0, 0.0, 0, 0x710000000)), T.ERR_INVALID_ARG),
    (dict(stats=0x710000000, opts=(0, 0.0, 0x700000000, 0x710000000 + 48 * 7)), T.ERR_ALIAS),
    (dict(stats=0x710000000 + 48 * 15, opts=(0, 0.0, 0x700000000, 0x710000000)), T.ERR_ALIAS),
    # per-token outputs: 4-byte aligned, overlapping no input, no other output
    # and not each other
    (dict(opts=(0, 0.0, 0, 0, 0x720000002, 0)), T.ERR_INVALID_ARG),
    (dict(opts=(0, 0.0, 0, 0, 0, 0x730000001)), T.ERR_INVALID_ARG),
    (dict(opts=(0, 0.0, 0, 0, 0x100000000 + 4096, 0)), T.ERR_ALIAS),
    (dict(opts=(0, 0.0, 0, 0, 0, 0x200000000 + 8)), T.ERR_ALIAS),
    (dict(opts=(0, 0.0, 0, 0, 0x400000000, 0)), T.ERR_ALIAS),
    (dict(kl=0x720000000, opts=(0, 0.0, 0, 0, 0, 0x720000000 + 4 * 63)), T.ERR_ALIAS),
    (dict(opts=(0, 0.0, 0, 0, 0x720000000, 0x720000000 + 4 * 63)), T.ERR_ALIAS),
    (dict(opts=(0, 0.0, 0, 0, 0x300300000 + 8, 0)), T.ERR_ALIAS),
    (dict(stats=0x710000000, opts=(0, 0.0, 0, 0, 0, 0x710000000 + 48 * 7)), T.ERR_ALIAS),
    (dict(opts=(0, 0.0, 0x700000000, 0x710000000, 0x710000000 + 48 * 15, 0)), T.ERR_ALIAS),
])
def test_host_rejects_bad_arguments_before_launch(kw, code):
    assert _call(**kw) == code


def test_unaligned_rows_run_with_a_workspace_sized_for_them():
    """The same unaligned call is accepted by the host checks once the
    workspace is sized with aligned_rows = 0 (it then fails only at the first
    HIP call: a launch error, since the fake addresses are never reached on a
    machine without a GPU)."""
    kw = dict(v=151936, ld_s=151937, ld_t=151936, ld_g=151936)
    assert _call(**kw) == T.ERR_WORKSPACE
    assert _call(aligned=False, **kw) not in (T.ERR_WORKSPACE, T.ERR_INVALID_ARG, T.ERR_ALIAS)


def _call_noalloc(**kw):
    """turnkl_fwd_bwd_noalloc with fake (never dereferenced) addresses."""
    n, v = kw.get("n", 64), kw.get("v", 1024)
    args = dict(zs=0x100000000, ld_s=v, zt=0x200000000, ld_t=v, dtype=T.BF16, n=n, v=v,
                turn=0x300000000, traj=0x300100000, mask=0x300200000, alpha=0.5, scale=1.0,
                loss=0x300300000, grad=0x400000000, ld_g=v, stats=0, max_turns=8, acc=0, kl=0,
                opts=None, status=0x300400000)
    args.update(kw)
    p = lambda x: ctypes.c_void_p(x) if x else None
    return T.lib().turnkl_fwd_bwd_noalloc(
        p(args["zs"]), args["ld_s"], p(args["zt"]), args["ld_t"], args["dtype"], args["n"],
        args["v"], p(args["turn"]), p(args["traj"]), p(args["mask"]), args["alpha"],
        args["scale"], p(args["loss"]), p(args["grad"]), args["ld_g"], p(args["stats"]),
        args["max_turns"], args["acc"], p(args["kl"]), _opts(args["opts"]), p(args["status"]),
        None)


@pytest.mark.parametrize("kw,code", [
    (dict(alpha=2.0), T.ERR_INVALID_ARG),
    (dict(loss=0), T.ERR_INVALID_ARG),
    (dict(zs=0), T.ERR_INVALID_ARG),
    (dict(grad=0x200000000), T.ERR_ALIAS),
    (dict(status=0x300400002), T.ERR_INVALID_ARG),  # status_out not 4-byte aligned
    (dict(status=0x300300004), T.ERR_ALIAS),        # inside loss_out
    (dict(status=0x100000000 + 64), T.ERR_ALIAS),   # inside the student logits
    (dict(opts=(-1, 0.0, 0, 0)), T.ERR_INVALID_ARG),
    # larger than the 32 MiB scratch: 212 bytes per token at V = 151,936 with
    # aligned rows, 724 on the element-wise path
    (dict(n=160000, v=151936, ld_s=151936, ld_t=151936, ld_g=151936, zs=0x1000000000,
          zt=0x3000000000, grad=0x5000000000), T.ERR_SCRATCH),
    (dict(n=50000, v=151936, ld_s=151937, ld_t=151937, ld_g=151937, zs=0x1000000000,
          zt=0x3000000000, grad=0x5000000000), T.ERR_SCRATCH),
])
def test_noalloc_host_rejects_before_launch(kw, code):
    assert _call_noalloc(**kw) == code


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(T, "_lib", None)
    monkeypatch.setattr(T, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        T.lib()


def _call_topk(**kw):
    """turnkl_fwd_bwd_topk with fake (never dereferenced) addresses."""
    n, v, k = kw.get("n", 64), kw.get("v", 1024), kw.get("k", 50)
    ws_bytes = T.lib().turnkl_topk_workspace_bytes(n, k, kw.get("max_turns", 8))
    args = dict(zs=0x100000000, ld_s=v, dtype=T.BF16, n=n, v=v, ids=0x200000000,
                vals=0x210000000, ld_k=k, k=k, turn=0x300000000, traj=0x300100000,
                mask=0x300200000, alpha=0.5, scale=1.0, loss=0x300300000, grad=0x400000000,
                ld_g=v, gk=0x600000000, ld_gk=k, stats=0, max_turns=8, acc=0, kl=0,
                ws=0x500000000, ws_bytes=ws_bytes, opts=None)
    args.update(kw)
    p = lambda x: ctypes.c_void_p(x) if x else None
    return T.lib().turnkl_fwd_bwd_topk(
        p(args["zs"]), args["ld_s"], args["dtype"], args["n"], args["v"], p(args["ids"]),
        p(args["vals"]), args["ld_k"], args["k"], p(args["turn"]), p(args["traj"]), p(args["mask"]),
        args["alpha"], args["scale"], p(args["loss"]), p(args["grad"]), args["ld_g"], p(args["gk"]),
        args["ld_gk"], p(args["stats"]), args["max_turns"], args["acc"], p(args["kl"]),
        _opts(args["opts"]), p(args["ws"]), args["ws_bytes"], None)


def test_topk_workspace_bytes():
    a = T.lib().turnkl_topk_workspace_bytes(1000, 50, 8)
    b = T.lib().turnkl_topk_workspace_bytes(1000, 100, 8)
    assert 0 < a < b and a % 256 == 0
    assert T.lib().turnkl_topk_workspace_bytes(1000, 0, 8) == 0
    assert T.lib().turnkl_topk_workspace_bytes(1000, 1025, 8) == 0
    assert T.lib().turnkl_topk_workspace_bytes(-1, 50, 8) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=3), T.ERR_INVALID_ARG),
    (dict(k=0), T.ERR_INVALID_ARG),
    (dict(k=1025, ld_k=1025, ld_gk=1025), T.ERR_INVALID_ARG),
    (dict(k=64, v=32, ld_s=32, ld_g=32, ld_k=64, ld_gk=64), T.ERR_INVALID_ARG),  # K > V
    (dict(ld_k=49), T.ERR_INVALID_ARG),
    (dict(ld_gk=10), T.ERR_INVALID_ARG),
    (dict(ld_s=1000), T.ERR_INVALID_ARG),
    (dict(ids=0), T.ERR_INVALID_ARG),
    (dict(vals=0), T.ERR_INVALID_ARG),
    (dict(alpha=2.0), T.ERR_INVALID_ARG),
    # outputs overlapping inputs or each other (exact in-place dense is allowed)
    (dict(grad=0x200000000), T.ERR_ALIAS),
    (dict(grad=0x100000000 + 2), T.ERR_ALIAS),
    (dict(gk=0x210000000), T.ERR_ALIAS),
    (dict(gk=0x100000000), T.ERR_ALIAS),
    (dict(gk=0x400000000 + 4096), T.ERR_ALIAS),
    (dict(ws_bytes=1024), T.ERR_WORKSPACE),
    (dict(opts=(-3, 0.0, 0, 0)), T.ERR_INVALID_ARG),
    (dict(opts=(0, 0.0, 0x700000000, 0)), T.ERR_INVALID_ARG),
    # per-token outputs overlapping the support, the sparse gradient or each other
    (dict(opts=(0, 0.0, 0, 0, 0x200000000 + 64, 0)), T.ERR_ALIAS),
    (dict(opts=(0, 0.0, 0, 0, 0, 0x210000000 + 8)), T.ERR_ALIAS),
    (dict(opts=(0, 0.0, 0, 0, 0x600000000 + 200, 0)), T.ERR_ALIAS),
    (dict(opts=(0, 0.0, 0, 0, 0x720000000, 0x720000000 + 4 * 63)), T.ERR_ALIAS),
    (dict(opts=(0, 0.0, 0, 0, 0x720000001, 0)), T.ERR_INVALID_ARG),
])
def test_topk_host_rejects_bad_arguments_before_launch(kw, code):
    assert _call_topk(**kw) == code


def test_header_is_plain_c_and_links(tmp_path):
    """include/turnkl.h (and turnkl_testing.h) compile as C11 with warnings as errors, and a C
    program linked against the library calls its host entry points (no GPU
    is touched)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "abi.c"
    src.write_text(r'''
#include <stdio.h>
#include "turnkl.h"
#include "turnkl_testing.h"
int main(void) {
  size_t b = turnkl_workspace_bytes(1000, 151936, TURNKL_BF16, 50, 1);
  if (turnkl_testing_workspace_bytes(1000, 151936, TURNKL_BF16, 50, 1, 0) != b) return 3;
  if (TURNKL_NOALLOC_SCRATCH_BYTES < b) return 4;
  turnkl_depth_config c;
  turnkl_depth_default_config(&c);
  if (b == 0 || c.h_max < c.h_min) return 1;
  if (turnkl_alpha_schedule(5, 10, 0.0, 1.0) != 0.5) return 2;
  printf("%s\n", turnkl_status_string(TURNKL_ERR_SYNC_TIMEOUT));
  return 0;
}
''')
    exe = tmp_path / "abi"
    libdir = os.path.dirname(T.LIB_PATH)
    cmd = [gcc, "-std=c11", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", str(src),
           "-L", libdir, "-lturnkl", f"-Wl,-rpath,{libdir}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, (r.returncode, r.stderr)
    assert r.stdout.strip() == T.status_string(T.ERR_SYNC_TIMEOUT)
