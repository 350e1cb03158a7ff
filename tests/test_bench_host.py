"""Host-side checks of bench.py (no GPU): the source digest that guards the
committed HBM-traffic counters covers every file a kernel is built from."""
import os
import re

import bench

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2605_30359_amd", "csrc")


def _includes(name, seen):
    if name in seen or not os.path.exists(os.path.join(CSRC, name)):
        return
    seen.add(name)
    for inc in re.findall(r'#include "([^"]+)"', open(os.path.join(CSRC, name)).read()):
        _includes(inc, seen)


def test_kernel_digest_covers_included_sources():
    shared = {"kf_device.hpp", "kf_internal.hpp"}
    for kernel, files in bench.KERNEL_FILES.items():
        for f in files:
            assert os.path.exists(os.path.join(CSRC, f)), (kernel, f)
        closure = set()
        for f in files:
            _includes(f, closure)
        # kf_launch.hpp only declares the launchers
        missing = closure - set(files) - shared - {"kf_launch.hpp"}
        assert not missing, f"{kernel}: digest misses {sorted(missing)}"


def test_digest_differs_between_kernels():
    a = bench._source_digest(bench.KERNEL_FILES["kf_gemm_f32_8x8"])
    b = bench._source_digest(bench.KERNEL_FILES["kf_conv3x3_bf16_256x128"])
    assert a != b and len(a) == 16
