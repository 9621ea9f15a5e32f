"""Workload shapes pinned to Table II (2-byte weights, three d x f matrices per expert)."""
import json
import os

import synth


def test_expert_size_matches_table2(golden_dir):
    t2 = json.load(open(os.path.join(golden_dir, "paper_table2.json")))["models"]
    for name in ("mixtral", "phi"):
        wl = synth.WORKLOADS[name]
        row = t2[name]
        assert (wl.L, wl.n, wl.k) == (row["layers"], row["experts_per_layer"], row["top_k"])
        mib = synth.slab_bytes(wl.d, wl.f) / 2**20
        assert abs(mib - row["size_per_expert_MB"]) / row["size_per_expert_MB"] < 0.02, (name, mib)
        # parameters x 2 bytes ~ model size (GiB), the 2-byte weight reading
        gib = row["params_billion"] * 1e9 * 2 / 2**30
        assert abs(gib - row["model_size_GB"]) / row["model_size_GB"] < 0.02, (name, gib)


def test_exact_slab_sizes():
    assert synth.slab_bytes(4096, 14336) == 352_321_536
    assert synth.slab_bytes(4096, 6400) == 157_286_400
