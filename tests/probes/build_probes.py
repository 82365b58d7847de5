"""Build the test-only HIP probes under tests/probes (gfx950) next to their sources."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
PROBES = {"dot2_probe.hip": "libdot2probe.so"}


def build() -> None:
    for src, lib in PROBES.items():
        out = os.path.join(HERE, lib)
        cmd = ["/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else "hipcc", "-O3", "-std=c++17",
               "-fPIC", "-shared", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
               "-packed-fp32-ops", "-x", "hip", os.path.join(HERE, src), "-o", out + ".tmp"]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
        os.replace(out + ".tmp", out)


if __name__ == "__main__":
    build()
