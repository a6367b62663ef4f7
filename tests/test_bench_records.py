"""Host-only checks of the benchmark's recorded counter figures.

The traffic and matrix-core busy figures that the bench line reports next to
its own timing are taken from rocprofv3 counter runs summarised under
profiles/, keyed by a hash of the kernel's sources.  These tests check that
each hashed source list covers every device header the kernel's source
includes (so an edit of any of them invalidates the record), and that the
two workloads the default bench line reports carry records for the current
sources.
"""
import os
import re
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1906_11786_amd", "csrc")
sys.path.insert(0, ROOT)

import bench  # noqa: E402

# Launch declarations only: no device code.
HOST_ONLY = {"kernels.h"}


def local_includes(name, seen=None):
    seen = set() if seen is None else seen
    with open(os.path.join(CSRC, name)) as f:
        for inc in re.findall(r'^#include "([^"/]+)"', f.read(), flags=re.M):
            if inc not in seen and inc not in HOST_ONLY:
                seen.add(inc)
                local_includes(inc, seen)
    return seen


@pytest.mark.parametrize("kernel", sorted(bench.KERNELS))
def test_hashed_sources_cover_device_includes(kernel):
    srcs = bench.KERNELS[kernel][1]
    missing = local_includes(srcs[0]) - set(srcs)
    assert not missing, f"{kernel}: {sorted(missing)} included by {srcs[0]} but not hashed"


@pytest.mark.parametrize("kernel,workload", [
    ("step_wide_fwd", "stress_n1048576_B256_E10_H256"),
    ("step_wide_rev", "stress_n1048576_B256_E10_H256"),
    ("step_bits_gru", "program_graph_n20000_B128_E10_H64"),
    ("step_bits_gru_bwd", "program_graph_n20000_B128_E10_H64"),
])
def test_default_workloads_have_current_records(kernel, workload):
    traffic, src = bench.recorded_traffic(kernel, workload, "bits")
    assert traffic is not None and traffic > 0, f"no traffic record of {kernel} for the current sources"
    busy, _ = bench.recorded_busy(kernel, workload, "bits")
    assert busy is not None and 0.0 < busy < 1.0, f"no matrix-core busy record of {kernel} for the current sources"
