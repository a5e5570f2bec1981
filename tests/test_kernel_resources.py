"""Register budgets of the kernels the benchmark's pass launches, checked on
the compiler's own resource report (the device assembly's .num_vgpr and
.private_seg_size symbols): none of them may spill to scratch memory, whose
reloads wait for every outstanding load, and each must fit the VGPR budget of
the occupancy it is designed for.  Runs on the CPU (hipcc cross-compiles
gfx950); skipped where hipcc is missing."""
import concurrent.futures
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_2608_21541_amd import build as B

# (source, kernel symbol prefix, largest VGPR count)
KERNELS = [
    ("score.hip", "_ZN6certkv17score_mfma_kernelILi128ELi8ELi0E", 128),       # pass 1
    ("score.hip", "_ZN6certkv22score_pass2_w16_kernelILi128ELi8ELb1E", 128),  # pass 2, key sums
    ("score.hip", "_ZN6certkv22score_pass2_w16_kernelILi128ELi8ELb0E", 128),  # pass 2
    ("sort.hip", "_ZN6certkv15seg_sort_kernel", 128),
    ("curves.hip", "_ZN6certkv13curves_kernelILi128ELb1ELi0E", 128),         # centered
    ("curves.hip", "_ZN6certkv13curves_kernelILi128ELb1ELi1E", 128),         # uncentered
    ("curves.hip", "_ZN6certkv13curves_kernelILi128ELb1ELi2E", 128),         # tail mass
    ("curves.hip", "_ZN6certkv13curves_kernelILi64ELb0ELi0E", 128),          # fp32, d = 64
    ("allocate.hip", "_ZN6certkv15allocate_kernel", 128),
    ("select.hip", "_ZN6certkv13select_kernel", 128),
    ("tail.hip", "_ZN6certkv18tail_gather_kernelILi128EtLb1ELb1E", 128),
    ("clusters.hip", "_ZN6certkv19cluster_tail_kernelILi128EtE", 102),       # five waves per SIMD
    ("decode.hip", "_ZN6certkv13decode_kernelILi128ELi4EE", 256),
]


def _device_asm(src, out_dir):
    path = os.path.join(out_dir, src + ".s")
    cmd = [B.HIPCC, *[f for f in B.FLAGS if f != "-fPIC"], "--cuda-device-only", "-S",
           os.path.join(B.CSRC, src), "-o", path]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    with open(path) as fh:
        return fh.read()


@pytest.fixture(scope="module")
def asm():
    if not (os.path.exists(B.HIPCC) or shutil.which(B.HIPCC)):
        pytest.skip("hipcc not available")
    srcs = sorted({s for s, _, _ in KERNELS})
    with tempfile.TemporaryDirectory() as d:
        with concurrent.futures.ThreadPoolExecutor(min(len(srcs), 8)) as ex:
            texts = dict(zip(srcs, ex.map(lambda s: _device_asm(s, d), srcs)))
    return texts


def _symbols(text, prefix, field):
    pat = re.compile(r"\.set (" + re.escape(prefix) + r"\w*)\." + field + r", (\d+)")
    return {m.group(1): int(m.group(2)) for m in pat.finditer(text)}


@pytest.mark.parametrize("src,prefix,vmax", KERNELS, ids=[k[1][-40:] for k in KERNELS])
def test_hot_kernels_do_not_spill(asm, src, prefix, vmax):
    scratch = _symbols(asm[src], prefix, "private_seg_size")
    vgprs = _symbols(asm[src], prefix, "num_vgpr")
    assert scratch, f"no kernel {prefix} in {src}"
    for name, n in scratch.items():
        assert n == 0, f"{name} spills {n} bytes per lane"
        assert vgprs[name] <= vmax, f"{name} uses {vgprs[name]} VGPRs (budget {vmax})"
