"""The benchmark's command-line contract that needs no GPU: it runs on one GPU
only, and says so (one JSON line, exit status 2) when asked for more."""

import json
import os
import subprocess
import sys

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


def test_default_launches_match_their_counter_entries():
    # the fabric-traffic figure is reported only when the timed launch is the
    # one the counters were taken on; a change of launch knobs must come with
    # new counters, not with a silently missing figure
    sys.path.insert(0, ROOT)
    import bench
    from synth import CONFIGS, batch_sizes
    for argv, cfg_key, weights in ((["--config", "4"], 4, "f32"), (["--weights", "f16"], 4, "f16"),
                                   (["--config", "5"], 5, "f32")):
        args = bench.parse(argv)
        kernel_arg, _, knobs = bench.launch_knobs(args)
        cfg = CONFIGS[cfg_key]
        keys = [k for k in bench.MEASURED_TRAFFIC if k[0] == cfg.name and k[4] == weights]
        assert keys, argv
        for k in keys:
            assert k[1] == 0 and k[2] == batch_sizes(cfg)[0], argv
            assert k[5] == (kernel_arg or 1), argv
            assert k[6] == json.dumps(knobs, sort_keys=True), argv
