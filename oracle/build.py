"""Compile the C oracle (oracle.c) into liboracle.so with gcc and OpenMP.

Test infrastructure only.  Run as ``python -m oracle.build`` or call build().
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


SANITIZE = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
            "-fno-omit-frame-pointer"]


def build(verbose: bool = False, sanitize: bool = False, out: str = LIB) -> str:
    """Compile oracle.c to `out` (always recompiles); return the path.  With
    sanitize, an AddressSanitizer + UndefinedBehaviorSanitizer build (host
    code only: the oracle is plain C), loaded with the sanitizer runtimes
    preloaded (sanitizer_preload())."""
    tmp = out + ".tmp"
    opt = SANITIZE if sanitize else ["-O2"]
    cmd = ["gcc", *opt, "-std=c99", "-fPIC", "-shared", "-fopenmp",
           "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def sanitizer_preload() -> str:
    """LD_PRELOAD entries of the sanitizer runtimes a sanitized build needs."""
    libs = [subprocess.run(["gcc", f"-print-file-name={n}"], capture_output=True, text=True,
                           check=True).stdout.strip() for n in ("libasan.so", "libubsan.so")]
    return ":".join(libs)


if __name__ == "__main__":
    print(build(verbose=True))
