"""A build of libpced whose host code (the C ABI and the kernels' launch code)
carries AddressSanitizer and UndefinedBehaviorSanitizer; the gfx950 device code
is the same as in the product build. For running the host-only ABI tests under
the sanitizers (the library then needs the ASan runtime preloaded into the
process: `runtime()`). Not used by the product path."""
from __future__ import annotations

import os
import subprocess

from .build import COMMON, CSRC, HIPCC, LINK, _run

# each host-only sanitizer flag follows its own -Xarch_host (device code is not instrumented)
SANITIZE = ("-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined "
            "-Xarch_host -fno-sanitize-recover=undefined -Xarch_host -fno-omit-frame-pointer").split()


def build(out_dir: str, verbose: bool = False) -> str:
    os.makedirs(out_dir, exist_ok=True)
    objs = []
    for src in ("pced_kernels.hip", "pced_api.cpp"):
        obj = os.path.join(out_dir, src.replace(".", "_") + ".san.o")
        cmd = [HIPCC, *COMMON, "-g", *SANITIZE, "-c", os.path.join(CSRC, src), "-o", obj]
        if src.endswith(".cpp"):
            cmd.insert(1, "-xhip")
        _run(cmd, verbose)
        objs.append(obj)
    lib = os.path.join(out_dir, "libpced_sanitized.so")
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", lib, *LINK,
          "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan"], verbose)
    return lib


def runtime() -> str:
    """Path of the shared ASan runtime (it carries the UBSan handlers too)."""
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return r.stdout.strip()
