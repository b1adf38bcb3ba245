"""Build the oracle's shared library (test infrastructure only).

The oracle is plain C compiled with gcc and OpenMP.  Only the tests, the smoke
check and the CPU-baseline leg of the benchmark load it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "sparse_attn_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False, src: str = SRC, lib: str = LIB) -> str:
    """Compile the oracle source into a shared library; returns its path."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", src, "-o", lib + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


def ensure_built() -> str:
    """Build only when the library is missing or older than its source.

    SPARSE_ATTN_ORACLE_LIB names another build of the same source to load
    instead (used by the mutation test, which plants mistakes in a copy)."""
    override = os.environ.get("SPARSE_ATTN_ORACLE_LIB")
    if override:
        return override
    if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        build()
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
