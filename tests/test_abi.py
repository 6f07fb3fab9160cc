"""The C ABI without a GPU: the library loads, exports every entry point that
include/adept.h declares, its struct layouts match the ctypes mirror, and
bad arguments are rejected on the host before anything is launched."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2601_03700_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "adept.h")


def declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(adept_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    names = declared()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), f"{n} declared in adept.h but not exported"
    assert set(names) == set(B.EXPORTED), "binding signatures and header differ"
    assert lib.adept_abi_version() == 6


@pytest.mark.parametrize("cname,pyname", [("adept_layer_args", "LayerArgs"),
                                           ("adept_encoder_args", "EncoderArgs")])
def test_struct_layout_matches_header(tmp_path, cname, pyname):
    S = getattr(B, pyname)
    fields = [f for f, _ in S._fields_]
    src = ['#include <stdio.h>', '#include <stddef.h>', f'#include "{HEADER}"', 'int main(void){',
           f'printf("%zu\\n", sizeof({cname}));']
    for f in fields:
        src.append(f'printf("%zu\\n", offsetof({cname}, {f}));')
    src.append('printf("%zu\\n", sizeof(adept_exit_cfg)); return 0; }')
    c = tmp_path / "layout.c"
    c.write_text("\n".join(src))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-o", str(exe), str(c)], check=True)
    vals = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(S)
    for f, off in zip(fields, vals[1:-1]):
        assert getattr(S, f).offset == off, f
    assert vals[-1] == ctypes.sizeof(B.ExitCfg)


def _expect_invalid(status):
    assert status == -1, status
    assert B.lib().adept_last_error()


def test_host_validation_rejects_bad_arguments():
    L = B.lib()
    cfg = B.exit_cfg(0.9, 4)
    # NULL cfg, bad layer, bad dtype, bad d_model
    _expect_invalid(L.adept_exit_test(1, 256, 1, None, 16, 16, 4, 16, 16, 16, None, 16, None, None))
    _expect_invalid(L.adept_exit_test(1, 256, 5, ctypes.byref(cfg), 16, 16, 4, 16, 16, 16, None,
                                      16, None, None))
    _expect_invalid(L.adept_exit_test(7, 256, 1, ctypes.byref(cfg), 16, 16, 4, 16, 16, 16, None,
                                      16, None, None))
    _expect_invalid(L.adept_exit_test(1, 250, 1, ctypes.byref(cfg), 16, 16, 4, 16, 16, 16, None,
                                      16, None, None))
    # d_model beyond the largest row one wavefront holds (8192 for GLOBAL)
    assert L.adept_exit_test(1, 8196, 1, ctypes.byref(cfg), 16, 16, 4, 16, 16, 16, None, 16,
                             None, None) == -2
    assert L.adept_last_error()
    # GLOBAL without inertia
    _expect_invalid(L.adept_exit_test(1, 256, 1, ctypes.byref(cfg), 16, 16, 4, 16, 16, None, None,
                                      16, None, None))
    # BOTH needs h_prev and the inertia, and holds rows up to 4096 wide; unknown metric
    both = B.exit_cfg(0.9, 4, "both")
    _expect_invalid(L.adept_exit_test(1, 256, 1, ctypes.byref(both), 16, 16, 4, 16, None, 16,
                                      None, 16, None, None))
    _expect_invalid(L.adept_exit_test(1, 256, 1, ctypes.byref(both), 16, 16, 4, 16, 16, None,
                                      None, 16, None, None))
    assert L.adept_exit_test(1, 4100, 1, ctypes.byref(both), 16, 16, 4, 16, 16, 16, None, 16,
                             None, None) == -2
    bad = B.exit_cfg(0.9, 4)
    bad.metric = 3
    _expect_invalid(L.adept_exit_test(1, 256, 1, ctypes.byref(bad), 16, 16, 4, 16, 16, 16, None,
                                      16, None, None))
    # compaction output aliasing its input
    _expect_invalid(L.adept_compact(1, 4, 16, 32, 16, 8, 32, 16, 48, 16, 64, None, 0, None))
    # compaction at a layer outside 1..n_layers
    _expect_invalid(L.adept_compact(5, 4, 16, 32, 16, 8, 48, 16, 64, 16, 80, None, 0, None))
    # KV generation: layer stride smaller than one [2*H*hd][D] block
    _expect_invalid(L.adept_kv_generate(1, 4, 256, 2, 128, 1e-6, 16, 16, 16, 8, 16, 16, 16, 16,
                                        100, 16, 16, 16, 8, 16, 16, 8, None, 0, None))
    # attention: head_dim that does not divide 256
    _expect_invalid(L.adept_attend(1, 2, 96, 0.1, 1, 16, 16, 16, 8, 16, 16, 1, 16, 16, 8, None,
                                   None, 16, None, 0, None))
    # bidirectional attention without key lengths
    _expect_invalid(L.adept_attend(1, 2, 64, 0.1, 0, 16, 16, 16, 8, 16, 16, 1, 16, 16, 8, None,
                                   None, 16, None, 0, None))
    # layer step: NULL args, then empty args
    _expect_invalid(L.adept_layer_step(None, 1, None))
    a = B.LayerArgs()
    _expect_invalid(L.adept_layer_step(ctypes.byref(a), 1, None))


def test_workspace_queries_are_host_only():
    assert B.compact_workspace_bytes(1000) == 0          # one workgroup
    assert B.compact_workspace_bytes(1 << 20) > 0        # multi-pass tiles
    assert B.kv_generate_workspace_bytes(32, 4096) >= 4096 * 8
    assert B.attend_workspace_bytes(16384, 8, 32, 128, 2048) >= (16384 // 128 + 8) * 8  # query tiles
    # decode: 64 queries x 32 heads, sized for 4 key chunks each (about 8192
    # workgroups) of (max, sum, 128 partial outputs) in f32; fewer active
    # queries on the device take more chunks within the same capacity
    assert B.attend_workspace_bytes(64, 64, 32, 128, 4352) == 64 * 32 * 4 * 130 * 4
    # one query: at most one chunk per 256 keys of s_max (17 for 4352)
    assert B.attend_workspace_bytes(1, 1, 32, 128, 4352) == 1 * 32 * 17 * 130 * 4
    assert B.attend_workspace_bytes(1 << 20, 1, 32, 128, 16384) < 64 << 20   # bounded
