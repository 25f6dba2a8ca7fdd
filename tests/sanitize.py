#!/usr/bin/env python3
"""CPU sanitizer runs of the host code (no GPU needed).

1. The oracle (oracle/oracle.c) and the input generators (synth/synth.c),
   built by gcc with AddressSanitizer and UndefinedBehaviorSanitizer, under the
   whole CPU test suite (gcc's ASan runtime preloaded into Python).
2. The library's host code (argument checks, workspace planning, the host
   side of every entry point, the subgraph matching in graph.hip), built by
   hipcc with both sanitizers on the host compilation only, under the CPU
   tests that drive it (the ABI checks and the subgraph matching; clang's ASan
   runtime preloaded).

Undefined behaviour aborts the run (-fno-sanitize-recover); leak checking is
off (Python's own allocations are not ours).  Usage:
    python tests/sanitize.py            # both runs, exit status 0 when clean
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

GCC_SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer", "-g"]


def run(cmd, env):
    print("[sanitize] " + " ".join(cmd), flush=True)
    return subprocess.call(cmd, env=env, cwd=ROOT)


def base_env(preload: str) -> dict:
    env = dict(os.environ)
    env["LD_PRELOAD"] = preload
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["PYTHONPATH"] = ROOT
    return env


def gcc_runtime() -> str:
    return subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()


def clang_runtime() -> str:
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise SystemExit("clang's AddressSanitizer runtime was not found under /opt/rocm")
    return hits[-1]


def main() -> int:
    import oracle
    import synth
    from paper_2512_08365_amd import _build

    rc = 0
    with tempfile.TemporaryDirectory(prefix="mag_san_") as tmp:
        # 1. oracle + generators
        orc = oracle.build(out=os.path.join(tmp, "_oracle_san.so"), extra_flags=GCC_SAN)
        syn = synth.build(out=os.path.join(tmp, "_synth_san.so"), extra_flags=GCC_SAN)
        env = base_env(gcc_runtime())
        env["MAG_ORACLE_SO"] = orc
        env["MAG_SYNTH_SO"] = syn
        rc |= run([sys.executable, "-m", "pytest", "tests", "-q", "-x", "-m", "not gpu",
                   "--ignore=tests/test_sanitize.py", "-p", "no:cacheprovider"], env)
        # 2. the library's host code
        lib = _build.build(out=os.path.join(tmp, "libmagneton_san.so"), host_sanitize=True)
        env = base_env(clang_runtime())
        env["MAG_LIBRARY_SO"] = lib
        rc |= run([sys.executable, "-m", "pytest", "tests/test_abi.py", "tests/test_graph_match.py",
                   "-q", "-x", "-p", "no:cacheprovider"], env)
    print(f"[sanitize] {'clean' if rc == 0 else 'FAILED'}", flush=True)
    return rc


if __name__ == "__main__":
    sys.exit(main())
