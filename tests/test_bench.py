"""The benchmark's command-line contract that needs no GPU: it runs on one GPU
only, and says so (one JSON line, exit status 2) when asked for more."""

import json
import os
import subprocess
import sys

import numpy as np

from conftest import ROOT

BENCH = os.path.join(ROOT, "bench.py")


def _run(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, BENCH, *args], capture_output=True, text=True, env=env, timeout=120,
                          cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run(["--gpus", "2"])
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"]


def test_a_multi_rank_launch_is_refused_too():
    r = _run(["--gpus", "1"], {"WORLD_SIZE": "4"})
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def test_help_lists_the_contract_flags():
    r = _run(["--help"])
    assert r.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup", "--config", "--weights", "--update"):
        assert flag in r.stdout


def test_default_launch_leaves_the_knobs_to_the_library():
    # the measured launch lives in the library (automatic kernel, tile size
    # and tiles per workgroup from N and the storage type): the benchmark
    # passes no knob, except kernel 1 for the unfused comparator built on it
    sys.path.insert(0, ROOT)
    import bench
    from synth import CONFIGS
    for argv, cfg_key, kernel, storage in ((["--config", "4"], 4, 0, 0), (["--weights", "f16"], 4, 0, 1),
                                           (["--config", "3"], 3, 0, 0), (["--config", "5"], 5, 0, 0),
                                           (["--config", "2"], 2, 0, 0), (["--config", "5", "--weights", "f16"], 5, 0, 1),
                                           (["--unfused"], 4, 1, 0)):
        knobs = bench.launch_knobs(bench.parse(argv), CONFIGS[cfg_key])
        assert knobs.pop("kernel") == kernel and knobs.pop("storage") == storage, argv
        assert not any(knobs.values()), (argv, knobs)


def test_counter_entries_belong_to_the_current_kernels():
    # fabric traffic is reported only from counters taken on the current kernel
    # sources: any edit to them must come with new counters
    sys.path.insert(0, ROOT)
    import bench
    digest = bench.csrc_digest()
    for key, entry in bench.MEASURED_TRAFFIC.items():
        assert entry["csrc"] == digest, (key, "kernel sources changed since these counters were taken")
        assert len(entry["fetch_kib"]) == len(entry["write_kib"]) == len(json.loads(key)[1])
    # the default run (the whole 512^2 pass, automatic launch) has its counters
    from synth import CONFIGS
    knobs = bench.launch_knobs(bench.parse([]), CONFIGS[4])
    key = json.dumps([CONFIGS[4].name, [0, 1], 0, 262208, "f32", False, False, False, False,
                      {k: v for k, v in sorted(knobs.items())}])
    assert key in bench.MEASURED_TRAFFIC


def test_oracle_sample_plan():
    sys.path.insert(0, ROOT)
    import bench
    from synth import CONFIGS, batch_sizes
    for cfg_key in (3, 4, 5):
        sizes = batch_sizes(CONFIGS[cfg_key])
        batches = list(range(len(sizes)))
        s = bench.sample_docs(sizes, cfg_key, batches, 2048)
        assert sorted(s) == batches
        total = sum(len(v) for v in s.values())
        assert 0.9 * 2048 <= total <= 2048 + 2 * len(batches), (cfg_key, total)
        for b, B in zip(batches, sizes):
            assert s[b][0] == 0 and s[b][-1] == B - 1 and len(np.unique(s[b])) == len(s[b])
    # every document of the 32^2 workload and of the first 128^2 batch
    s = bench.sample_docs([10000], 1, [0], 2048)
    assert np.array_equal(s[0], np.arange(10000))
    s = bench.sample_docs([65536, 65536], 2, [0, 1], 2048)
    assert len(s[0]) == 65536 and len(s[1]) == 1024
