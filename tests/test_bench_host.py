"""bench.py on a host without a GPU: the multi-GPU refusal and the lookup of recorded HBM
traffic in profiles/ (a record counts only for its kernel, its workload, its algorithmic
bytes and the current hash of its kernel source)."""
import hashlib
import os
import re

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _records():
    out = []
    for name in sorted(os.listdir(os.path.join(ROOT, "profiles"))):
        if name.endswith(".md"):
            out += bench._TRAFFIC_RECORD.findall(open(os.path.join(ROOT, "profiles", name)).read())
    return out


def test_refuses_more_than_one_gpu(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU" in capsys.readouterr().err


def test_traffic_records_resolve_only_on_their_source():
    """A record whose kernel source still hashes as recorded is returned; one taken on an
    earlier source is ignored (the bench then reports null traffic)."""
    recs = _records()
    assert {r[0] for r in recs} >= {"repack_direct_kernel", "repack_inplace_pipe_kernel",
                                    "vtoken_paged_decode"}
    for kernel, workload, src, sha, alg, traffic in recs:
        assert 0.99 < int(traffic) / int(alg) < 1.2
        digest = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()
        expect = int(traffic) if digest == sha else None
        assert bench.recorded_traffic(kernel, workload, int(alg)) == expect


def test_traffic_lookup_needs_the_same_workload_and_bytes():
    kernel, workload, _, _, alg, _ = _records()[0]
    assert bench.recorded_traffic(kernel, workload, int(alg) + 1) is None
    assert bench.recorded_traffic(kernel, workload + "_other", int(alg)) is None
    assert bench.recorded_traffic("another_kernel", workload, int(alg)) is None


@pytest.mark.parametrize("name", sorted(n for n in os.listdir(os.path.join(ROOT, "profiles"))
                                        if n.endswith(".md")))
def test_profiles_state_their_command(name):
    text = open(os.path.join(ROOT, "profiles", name)).read()
    assert re.search(r"rocprofv3 --(kernel-trace|pmc) ", text), name
