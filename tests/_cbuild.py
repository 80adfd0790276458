"""Compiles the small C helpers under tests/csrc with gcc (test side only)."""
import ctypes
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
OUT = os.path.join(HERE, "csrc", "_build")


def helper(name, link_oracle=False, extra=()):
    """Build tests/csrc/<name>.c into a shared object and load it."""
    os.makedirs(OUT, exist_ok=True)
    src = os.path.join(HERE, "csrc", name + ".c")
    so = os.path.join(OUT, "lib%s.so" % name)
    cmd = ["gcc", "-std=gnu11", "-O2", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-pthread", "-o", so + ".tmp", src]
    if link_oracle:
        import oracle
        lib = oracle.build(force=False)
        cmd += ["-L", os.path.dirname(lib), "-loracle",
                "-Wl,-rpath," + os.path.dirname(lib)]
    cmd += list(extra) + ["-lm"]
    subprocess.check_call(cmd)
    os.replace(so + ".tmp", so)
    if link_oracle:
        import oracle
        oracle.lib()  # load liboracle first so the dependency resolves
    return ctypes.CDLL(so)
