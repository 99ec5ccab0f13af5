"""The stored oracle digests (tests/golden/oracle_digests.json) are those of
the oracle as it stands: the first block of instances of each workload and
policy is simulated again here and hashed (format: tests/digests.py).  The
100000-request instance is left out (about a minute of CPU per policy)."""
import json
import os

import pytest

import digests as D
from oracle import oracle as O
from paper_2508_14544_amd import workloads as W

PATH = os.path.join(os.path.dirname(__file__), "golden", "oracle_digests.json")
DIG = json.load(open(PATH))
CASES = [(w, a) for w, e in DIG["workloads"].items() for a in e["algos"]
         if w != "single_n100000_m1048576" and not (w.startswith("online") and a != "amin")]


def test_digest_file_covers_every_configuration():
    want = {"single_n200_m512": {"amin", "amax", "hsf"},
            "batch4096_n1000_m16384": {"amin", "amax", "hsf"},
            "online1024_n10000_m65536": {"amin", "amax"},
            "single_n100000_m1048576": {"amin", "amax"},
            "sweep65536_n2000_m32768": {"amin", "hsf"}}
    for w, algos in want.items():
        assert algos <= set(DIG["workloads"][w]["algos"]), w
        for a in DIG["workloads"][w]["algos"].values():
            assert a["totals"]["status_counts"] == {"0": W.WORKLOADS[w].num_instances}
            assert len(a["blocks"]) == -(-W.WORKLOADS[w].num_instances // D.BLOCK)


@pytest.mark.parametrize("workload,algo", CASES, ids=[f"{w}-{a}" for w, a in CASES])
def test_first_block_matches_current_oracle(workload, algo):
    entry = DIG["workloads"][workload]
    k1 = min(D.BLOCK, W.WORKLOADS[workload].num_instances)
    batch = W.generate(workload, 0, instance_ids=range(k1), with_upper=entry["with_upper"])
    out = O.simulate_batch(batch, O.ALGOS[algo])
    assert D.block_digests(batch.offsets, out)[0] == entry["algos"][algo]["blocks"][0]
