"""Build the CPU oracle (test infrastructure) into oracle/libhco.so with gcc."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


SANITIZED = os.path.join(HERE, "libhco_san.so")


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """sanitize: an AddressSanitizer + UndefinedBehaviorSanitizer build in
    libhco_san.so (host code only; load it with the ASan runtime preloaded and
    HCO_LIB pointing at it)."""
    src = os.path.join(HERE, "hco.c")
    out = SANITIZED if sanitize else os.path.join(HERE, "libhco.so")
    tmp = out + ".tmp"
    flags = (["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
              "-fno-sanitize-recover=undefined"] if sanitize else ["-O2"])
    cmd = ["gcc", "-std=c99", *flags, "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, src, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
