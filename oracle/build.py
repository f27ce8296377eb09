"""Build the CPU oracle (test infrastructure) into oracle/liboctoref.so with gcc.

build(sanitize=True) builds oracle/liboctoref_san.so instead, with AddressSanitizer and
UndefinedBehaviorSanitizer (host code only), for the sanitizer check in
tests/test_oracle_sanitizers.py: a Python process loads it when started with the gcc ASan runtime
preloaded and OCTOREF_LIB naming it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboctoref.so")
SAN_LIB = os.path.join(HERE, "liboctoref_san.so")


def build(verbose: bool = False, sanitize: bool = False) -> str:
    src = os.path.join(HERE, "octoref.c")
    out = SAN_LIB if sanitize else LIB
    opt = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined"] if sanitize else ["-O2"]
    cmd = ["gcc", *opt, "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
           "-o", out + ".tmp", src, "-lpthread"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
