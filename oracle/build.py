"""Build the DAF CPU oracle (test infrastructure only).

Compiles ``daf_oracle.c`` with gcc into ``liboracle.so`` beside this file.
``build(mutant=k, out=path)`` compiles a copy with planted mistake ``k``; the
test suite uses those copies to show that the oracle's pins catch mistakes.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "daf_oracle.c")
DEFAULT_LIB = os.path.join(HERE, "liboracle.so")


def build(mutant: int = 0, out: str = DEFAULT_LIB, quiet: bool = True) -> str:
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-Wno-unused-parameter",
           f"-DDAF_ORACLE_MUTANT={int(mutant)}", SRC, "-o", out + ".tmp", "-lm"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("oracle build failed:\n" + res.stdout + res.stderr)
    if not quiet and (res.stdout or res.stderr):
        sys.stderr.write(res.stdout + res.stderr)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(quiet=False))
