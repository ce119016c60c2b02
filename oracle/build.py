"""Compile the plain-C oracle into ``oracle/_build/liborc.so`` (gcc, host only).

The oracle is test infrastructure: only the tests, the smoke check and the
benchmark's CPU-baseline leg load it."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "orc.c")
OUT = os.path.join(HERE, "_build", "liborc.so")


def build(force: bool = True) -> str:
    if not force and os.path.exists(OUT) and os.path.getmtime(OUT) >= os.path.getmtime(SRC):
        return OUT
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    tmp = OUT + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                           "-o", tmp, SRC])
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build())
