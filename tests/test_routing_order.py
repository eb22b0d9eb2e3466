"""The routing order of the HIP kernels, run on the CPU.

tests/host/route_order.cpp compiles the device header's routing helpers
(route_select of the multi-kernel path, logit_key and the 16-lane rank of the
single-pass kernel) for the host.  Over logit patterns with NaN, +-Inf, +-0
and ties, both paths must pick the same streams, every routed slot must get
exactly one distinct stream (the ranks of the candidates are a permutation),
and the choice must equal the oracle's routing (eq:router_topk: descending
logit, ties to the lower index; NaN, which no order of the paper ranks, is
placed below every number)."""

import math
import os
import shutil
import struct
import subprocess

import pytest
import torch

from oracle import xhc_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("route") / "route_order")
    cmd = [HIPCC, "-std=c++17", "-O1", "--offload-host-only", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2607_14530_amd", "csrc"),
           os.path.join(ROOT, "tests", "host", "route_order.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def _bits(v):
    return struct.unpack("<I", struct.pack("<f", v))[0]


def _patterns():
    g = torch.Generator().manual_seed(5)
    pool = [float("nan"), float("inf"), -float("inf"), 0.0, -0.0, 1.0, -1.0, 2.0, 1e-30, -1e-30, 3.4e38]
    pats = []
    for m in range(0, 5):
        for k in range(max(m, 1), 9):
            pats.append((m, k, torch.randn(16, generator=g).tolist()))
            pats.append((m, k, [1.0] * 16))                                  # all tied
            pats.append((m, k, [float("nan")] * 16))                         # all NaN
            pats.append((m, k, [0.0 if i % 2 else -0.0 for i in range(16)])) # signed zeros tie
            for _ in range(12):
                sel = torch.randint(0, len(pool), (16,), generator=g).tolist()
                pats.append((m, k, [pool[s] for s in sel]))
            z = torch.randn(16, generator=g).tolist()
            for i in torch.randint(0, 16, (3,), generator=g).tolist():
                z[i] = float("nan")
            pats.append((m, k, z))
    return pats


def _brute(z, m, k):
    """First k - m candidates by (is a number, value, lower index)."""
    def key(i):
        v = z[i]
        return (0, 0.0, -i) if math.isnan(v) else (1, v + 0.0, -i)
    return list(range(m)) + sorted(range(m, 16), key=key, reverse=True)[: k - m]


def test_routing_order_paths_agree_with_oracle(harness):
    pats = _patterns()
    text = "".join(f"{m} {k} " + " ".join(f"{_bits(v):08x}" for v in z) + "\n" for m, k, z in pats)
    r = subprocess.run([harness], input=text, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    lines = r.stdout.strip().splitlines()
    assert len(lines) == len(pats)
    for (m, k, z), line in zip(pats, lines):
        vals = [int(x) for x in line.split()]
        sel, fused, ranks = vals[:k], vals[k:2 * k], vals[2 * k:]
        assert sorted(ranks) == list(range(16 - m)), (m, k, z, ranks)
        assert sel == fused, (m, k, z, sel, fused)
        assert sel[:m] == list(range(m)) and len(set(sel)) == k and all(0 <= s < 16 for s in sel)
        zt = torch.tensor([z], dtype=torch.float32).to(torch.float64)
        idx, _, _ = O.route(zt, m, k)
        assert sel == idx[0].tolist(), (m, k, z, sel, idx[0].tolist())
        assert sel == _brute(z, m, k), (m, k, z, sel)
