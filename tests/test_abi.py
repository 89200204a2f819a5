"""The C ABI library loads, exports every entry point include/ultraep.h
declares, and rejects bad host-visible arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

import paper_2606_04101_amd as uep

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "ultraep.h")


def declared_symbols():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ultraep_[a-z_]+)\s*\(", src)))


def test_header_declares_the_entry_points():
    names = declared_symbols()
    for n in ("ultraep_count", "ultraep_plan", "ultraep_dispatch",
              "ultraep_plan_replicate", "ultraep_plan_reroute", "ultraep_reroute_and_pack",
              "ultraep_dispatch_layout", "ultraep_dispatch_scatter",
              "ultraep_pack_replicas", "ultraep_plan_sizes",
              "ultraep_dispatch_ws_bytes", "ultraep_strerror",
              "ultraep_relay_plan", "ultraep_pack_relay"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(uep.LIB_PATH)
    missing = [n for n in declared_symbols() if not hasattr(lib, n)]
    assert not missing, missing


def test_plan_sizes():
    g = uep.Group(64, 256, 1, 1024)
    assert uep.ultraep_plan_sizes(g) == (64, 256 * 64, 257, 320, 320, 64 * 320, 8)
    for bad in [uep.Group(3, 8, 1, 1), uep.Group(65, 65, 1, 1),
                uep.Group(4, 2048, 1, 1), uep.Group(4, 8, -1, 1),
                uep.Group(4, 8, 65, 1), uep.Group(4, 8, 1, 0),
                uep.Group(4, 8, 1, 1, 99, 100), uep.Group(4, 8, 1, 1, 1, 0)]:
        with pytest.raises(uep.UltraEPError):
            uep.ultraep_plan_sizes(bad)


def test_plan_ws_bytes():
    g = uep.Group(64, 256, 1, 1024)
    n = uep.ultraep_plan_ws_bytes(g)
    assert n >= 2 * 1023 * (1 + 2 * 64) * 4
    assert uep.ultraep_plan_ws_bytes(uep.Group(3, 8, 1, 1)) == 0


def test_noalloc_planner_array_covers_every_supported_group():
    """The fixed workspace of ultraep_plan_noalloc holds the planner
    workspace of the largest supported group."""
    m = re.search(r"#define ULTRAEP_PLAN_STATIC_WS_BYTES \(\(size_t\)(\d+) << (\d+)\)",
                  open(HEADER).read())
    cap = int(m.group(1)) << int(m.group(2))
    worst = max(uep.ultraep_plan_ws_bytes(uep.Group(R, E, ns, 1))
                for R, E, ns in [(64, 1024, 4), (64, 64, 4), (32, 1024, 8), (16, 1024, 16),
                                 (1, 1024, 256), (2, 1024, 128)])
    assert 0 < worst <= cap < worst + (1 << 20)


def test_ws_bytes():
    g = uep.Group(64, 256, 1, 1024)
    n = uep.ultraep_dispatch_ws_bytes(4096, 8, g)
    assert n >= 4 * (16 * 256 + 2 * 320 + 256) and n % 256 == 0
    assert uep.ultraep_dispatch_ws_bytes(-1, 8, g) == 0
    assert uep.ultraep_dispatch_ws_bytes(10, 0, g) == 0
    assert uep.ultraep_dispatch_ws_bytes(10, 300, g) == 0


def test_invalid_arguments_return_einval_without_launch():
    L = uep.lib()
    g = uep.Group(4, 16, 2, 32)
    pb = uep.PlanBuf(*([None] * 7))
    fake = ctypes.c_void_p(4096)  # never dereferenced: validation fails first
    E = uep.ULTRAEP_EINVAL
    assert L.ultraep_count(fake, 8, 2, 16, 1, None, fake, None) == E      # no counts
    assert L.ultraep_count(fake, 8, 0, 16, 1, fake, fake, None) == E      # k = 0
    assert L.ultraep_count(fake, 8, 17, 16, 1, fake, fake, None) == E     # k > E
    assert L.ultraep_count(fake, 8, 2, 16, 0, fake, fake, None) == E      # no groups
    assert L.ultraep_count(fake, 8, 2, 16, 65536, fake, fake, None) == E  # too many groups
    assert L.ultraep_count(fake, 8, 2, 16, 1, fake, None, None) == E      # no status
    assert L.ultraep_plan(fake, ctypes.byref(g), ctypes.byref(pb), fake, 1 << 30, None) == E
    bad = uep.Group(4, 15, 2, 32)
    full = uep.PlanBuf(*([4096] * 7))
    assert L.ultraep_plan(fake, ctypes.byref(bad), ctypes.byref(full), fake, 1 << 30, None) == E
    assert L.ultraep_plan(fake, ctypes.byref(g), ctypes.byref(full), fake, 16, None) == E  # ws
    assert L.ultraep_plan(fake, ctypes.byref(g), ctypes.byref(full), None, 1 << 30, None) == E
    assert L.ultraep_plan_replicate(fake, ctypes.byref(g), ctypes.byref(full), fake, 16,
                                    None) == E
    assert L.ultraep_plan_replicate(None, ctypes.byref(g), ctypes.byref(full), fake,
                                    1 << 30, None) == E
    assert L.ultraep_plan_reroute(fake, ctypes.byref(bad), ctypes.byref(full), None) == E
    assert L.ultraep_plan_reroute(fake, ctypes.byref(g), ctypes.byref(pb), None) == E
    assert L.ultraep_dispatch(fake, fake, 8, 2, 12, 0, ctypes.byref(g),  # H % 8
                              ctypes.byref(full), fake, fake, fake, fake, 1 << 20,
                              fake, None) == E
    assert L.ultraep_dispatch(fake, fake, 8, 2, 16, 4, ctypes.byref(g),  # rank >= R
                              ctypes.byref(full), fake, fake, fake, fake, 1 << 20,
                              fake, None) == E
    assert L.ultraep_dispatch(fake, fake, 8, 2, 16, 0, ctypes.byref(g),  # small ws
                              ctypes.byref(full), fake, fake, fake, fake, 16,
                              fake, None) == E
    for args in [(None, g, full, fake, 16, 0), (fake, bad, full, fake, 16, 0),   # load, group
                 (fake, g, full, fake, 12, 0), (fake, g, full, fake, 16, 4),     # W % 8, rank
                 (fake, g, pb, fake, 16, 0)]:                                     # plan
        ld, gg, pl, w, W, rank = args
        assert L.ultraep_reroute_and_pack(ld, ctypes.byref(gg), ctypes.byref(pl), w, W, rank,
                                          fake, 4, fake, fake, None) == E
    odd = ctypes.c_void_p(4096 + 4)
    assert L.ultraep_dispatch_scatter(odd, 8, 2, 16, fake, fake, fake, None) == E
    assert L.ultraep_pack_replicas(fake, 12, 0, ctypes.byref(g), ctypes.byref(full),
                                   fake, 4, fake, fake, None) == E     # W % 8
    assert L.ultraep_pack_replicas(fake, 16, 0, ctypes.byref(g), ctypes.byref(full),
                                   fake, -1, fake, fake, None) == E    # cap < 0
    assert L.ultraep_pack_replicas(fake, 16, 0, ctypes.byref(g), ctypes.byref(full),
                                   odd, 4, fake, fake, None) == E      # misaligned

    # relay trees: negative threshold, missing outputs, bad group or plan
    for gg, pl, thr, src, vol, st in [(g, full, -1, fake, fake, fake), (bad, full, 4, fake, fake, fake),
                                      (g, pb, 4, fake, fake, fake), (g, full, 4, None, fake, fake),
                                      (g, full, 4, fake, None, fake), (g, full, 4, fake, fake, None)]:
        assert L.ultraep_relay_plan(ctypes.byref(gg), ctypes.byref(pl), thr, src, vol, fake, st,
                                    None) == E
    for w, rs, W, rank, src, stg in [(fake, None, 16, 0, fake, fake),   # no relay source
                                     (fake, odd, 16, 0, fake, fake),    # misaligned relay source
                                     (fake, fake, 12, 0, fake, fake),   # W % 8
                                     (fake, fake, 16, 4, fake, fake),   # rank >= R
                                     (fake, fake, 16, 0, None, fake),   # no slot senders
                                     (None, fake, 16, 0, fake, fake)]:  # no blobs
        assert L.ultraep_pack_relay(w, rs, W, rank, ctypes.byref(g), ctypes.byref(full), src,
                                    stg, 4, fake, fake, None) == E


def test_strerror():
    assert uep.ultraep_strerror(0) == "ok"
    assert "capacity" in uep.ultraep_strerror(uep.ULTRAEP_ENOSPC)


def test_header_compiles_as_c_and_links():
    """include/ultraep.h is a C header: a plain C11 caller of every path entry
    point (tests/native/abi_consumer.c) compiles with gcc -Wall -Wextra
    -Werror and links against the library."""
    import shutil
    import subprocess
    import tempfile
    if not shutil.which("gcc") or not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"):
        pytest.skip("gcc or the HIP headers are not installed")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    with tempfile.TemporaryDirectory() as d:
        r = subprocess.run(
            ["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
             "-I", os.path.join(root, "include"), "-I", "/opt/rocm/include",
             os.path.join(root, "tests", "native", "abi_consumer.c"),
             "-L", os.path.dirname(uep.LIB_PATH), "-lultraep", "-L", "/opt/rocm/lib", "-lamdhip64",
             "-o", os.path.join(d, "abi_consumer")], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_binding_has_every_entry_point_by_name():
    """The Python binding names each function after the C entry point it
    calls: every symbol the header declares has a same-named function."""
    missing = [n for n in declared_symbols() if not callable(getattr(uep, n, None))]
    assert not missing, missing
