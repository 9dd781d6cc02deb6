"""Build tests/c_abi_consumer (test infrastructure): a plain C program that
uses libposeidon.so through include/poseidon.h and checks it against the CPU
oracle (liboracle.so).  Run by ``__graft_entry__.build()`` after both
libraries are built; the GPU test that runs it never compiles anything."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "c_abi_consumer.c")
EXE = os.path.join(HERE, "c_abi_consumer")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(verbose: bool = False) -> str:
    lib_dir = os.path.join(ROOT, "paper_1706_03292_amd")
    oracle_dir = os.path.join(ROOT, "oracle")
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           SRC, "-o", EXE + ".tmp",
           "-L", lib_dir, "-lposeidon", "-L", oracle_dir, "-loracle",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           f"-Wl,-rpath,{lib_dir}:{oracle_dir}:{os.path.join(ROCM, 'lib')}",
           # the repository moves between machines: also look beside the executable
           "-Wl,-rpath,$ORIGIN/../paper_1706_03292_amd:$ORIGIN/../oracle"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"gcc failed for {SRC}:\n{r.stdout}\n{r.stderr}")
    os.replace(EXE + ".tmp", EXE)
    return EXE


if __name__ == "__main__":
    print(build(verbose=True))
