"""The C ABI driven by a plain C program (tests/c_consumer/gpu_consumer.c):
device memory from hipMalloc, the three convolution passes of Section 5.2
called from C on the null stream, no Python binding or PyTorch in between.
The program is built with gcc and run as a child process on seeded inputs;
its outputs meet the single-op rule against the fp64 oracle."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
import paper_1909_11150_amd as fg
import synth
from gpu_util import conv_parity

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# n, h, w, c, k, r, stride, pad: a register-staged, a 128-tile and a
# 256-tile shape with a split kernel gradient
SHAPES = [(2, 19, 23, 24, 40, 3, 1, 1), (2, 33, 31, 64, 128, 3, 2, 1),
          (1, 64, 64, 256, 256, 3, 1, 1)]


@pytest.fixture(scope="module")
def exe(tmp_path_factory):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    out = str(tmp_path_factory.mktemp("c") / "gpu_consumer")
    libdir = os.path.dirname(fg.LIB_PATH)
    subprocess.run([gcc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                    os.path.join(ROOT, "tests", "c_consumer", "gpu_consumer.c"),
                    "-L", libdir, "-lfcngrad", "-L", "/opt/rocm/lib", "-lamdhip64",
                    f"-Wl,-rpath,{libdir}", "-Wl,-rpath,/opt/rocm/lib", "-o", out],
                   check=True, timeout=120)
    return out


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_c_program_runs_the_passes(exe, tmp_path, shape):
    n, h, w, c, k, r, st, pd = shape
    p, q = (h + 2 * pd - r) // st + 1, (w + 2 * pd - r) // st + 1
    rng = np.random.default_rng(sum(shape))
    x = synth.uniform(rng, (n, h, w, c))
    W = synth.normal(rng, (k, r, r, c), np.sqrt(2.0 / (r * r * c)))
    dy = synth.uniform(rng, (n, p, q, k))
    fin, fout = tmp_path / "in.bin", tmp_path / "out.bin"
    np.concatenate([a.ravel().view(np.uint16) for a in (x, W, dy)]).tofile(fin)
    d = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
    print(f"{shape}: {fg.kernel_name(d, fg.OP_FWD)}, {fg.kernel_name(d, fg.OP_BWD_DATA)}, "
          f"{fg.kernel_name(d, fg.OP_BWD_WEIGHT)}", flush=True)
    r_ = subprocess.run([exe, str(fin), str(fout), *map(str, shape)], capture_output=True,
                        text=True, timeout=120)
    assert r_.returncode == 0, r_.stderr
    out = np.fromfile(fout, dtype=np.uint16).view(np.float16)
    ny, nx = n * p * q * k, x.size
    y, dx, dw = out[:ny], out[ny:ny + nx], out[ny + nx:]
    assert dw.size == W.size
    conv_parity(y, oracle.conv2d_fwd(x, W, st, pd), f"C fwd {shape}")
    conv_parity(dx, oracle.conv2d_bwd_data(dy, W, x.shape, st, pd), f"C dx {shape}")
    conv_parity(dw, oracle.conv2d_bwd_weight(x, dy, r, r, st, pd), f"C dW {shape}")
