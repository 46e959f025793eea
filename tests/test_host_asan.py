"""Host code under AddressSanitizer (CPU only).

The library's host side (argument checks, the plan, the workspace layout,
the checked-mode validator: art_api.cpp, compiled by g++ with
-fsanitize=address into libart_asan.so, with the same device code) and the
oracles (gcc with -fsanitize=address) run a CPU subset of the suite in a
child process that preloads gcc's libasan.  Any heap, stack or global
overflow, use after free or double free in that code ends the child with
an AddressSanitizer report.  A planted out-of-bounds write (an output array
one element short, handed to the oracle) shows that the sanitizer is live.
"""
from __future__ import annotations

import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SUBSET = ["tests/test_abi_host.py", "tests/test_parity_rule.py", "tests/test_oracle_pins.py",
          "tests/test_oracle_lists.py", "tests/test_oracle_per_head.py"]


@pytest.fixture(scope="module")
def asan_env():
    import oracle
    from oracle import lists
    from paper_2606_00024_amd import build
    if not os.path.exists(build.ASAN_LIB):
        build.build()
    oracle.build_asan()
    libasan = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    if not os.path.exists(libasan):
        pytest.skip("gcc's libasan is not installed")
    env = dict(os.environ, LD_PRELOAD=libasan,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:exitcode=23",
               ART_LIBRARY=build.ASAN_LIB, ART_ORACLE_LIBRARY=oracle.ASAN_LIB,
               ART_LIST_ORACLE_LIBRARY=lists.ASAN_LIB)
    return env


def test_the_child_loads_the_sanitized_builds(asan_env):
    code = textwrap.dedent("""
        import ctypes, oracle
        from oracle import lists
        from paper_2606_00024_amd import _lib
        _lib.load(); oracle._load(); lists._load()
        maps = open('/proc/self/maps').read()
        for name in ('libasan', 'libart_asan.so', 'libart_oracle_asan.so', 'libart_list_oracle_asan.so'):
            assert name in maps, name
        print('sanitized builds loaded')
    """)
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=asan_env, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0 and "sanitized builds loaded" in r.stdout, r.stdout + r.stderr[-3000:]


def test_planted_overflow_is_caught(asan_env):
    code = textwrap.dedent("""
        import ctypes, numpy as np, oracle
        lib = oracle._load()
        B, Hq, Hkv, D, Bk, Ps = 1, 1, 1, 128, 64, 64
        q = np.zeros((B, Hq, D), np.uint16); k = np.zeros((1, Hkv, Ps, D), np.uint16); v = k.copy()
        pt = np.zeros((B, 1), np.int32); sl = np.full(B, 64, np.int32)
        sh = oracle.Shape(batch=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, block_size=Bk,
                          page_size=Ps, num_pages=1, max_pages_per_seq=1, max_blocks_per_list=0,
                          list_per_head=1, k_stride_page=Hkv * Ps * D, k_stride_head=Ps * D,
                          k_stride_token=D, v_stride_page=Hkv * Ps * D, v_stride_head=Ps * D,
                          v_stride_token=D)
        op = oracle.Opts(scale=0.088, tau=0.0, phi=0.0, patience=1, dense_order=0, probe_stride=1,
                         scale_of_accumulator=0, per_head_stop=0)
        out = np.zeros(B * Hq * D - 1)          # one element short: a planted mistake
        lse = np.zeros(B * Hq); stop = np.zeros(B * Hkv, np.int32); err = ctypes.c_int32()
        P = lambda a, t: a.ctypes.data_as(ctypes.POINTER(t))
        lib.artref_decode(ctypes.byref(sh), ctypes.byref(op), P(q, ctypes.c_uint16),
                          P(k, ctypes.c_uint16), P(v, ctypes.c_uint16), P(pt, ctypes.c_int32),
                          P(sl, ctypes.c_int32), None, None, None, None, P(out, ctypes.c_double),
                          P(lse, ctypes.c_double), P(stop, ctypes.c_int32), None, None, 0, 1,
                          ctypes.byref(err))
        print('no report')
    """)
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=asan_env, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 23 and "heap-buffer-overflow" in r.stderr, r.stdout + r.stderr[-3000:]


def test_cpu_subset_is_clean_under_address_sanitizer(asan_env):
    r = subprocess.run([sys.executable, "-m", "pytest", *SUBSET, "-q", "-x", "-m", "not gpu",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=asan_env, capture_output=True,
                       text=True, timeout=1200)
    tail = (r.stdout[-3000:] + r.stderr[-3000:])
    assert "AddressSanitizer" not in r.stdout + r.stderr, tail
    assert r.returncode == 0, tail
