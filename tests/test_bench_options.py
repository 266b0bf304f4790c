"""bench.py's option handling, on the CPU: the workload each mode runs and
the combinations it refuses (no GPU needed)."""

import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from workloads import get_config  # noqa: E402


def _cfg(*argv):
    return bench.workload_config(bench.parser().parse_args(list(argv)), get_config)


def test_default_workload_is_the_largest_single_gpu_share():
    cfg, problem = _cfg()
    assert problem is None
    assert cfg.name == "llama70b_share" and cfg.gamma == get_config("llama70b_share").gamma


def test_counter_digest_covers_included_headers():
    files = bench.source_files("attention.hip")
    assert files[0] == "attention.hip"
    assert {"common.h", "launch.h", "combine.h"} <= set(files)
    assert len(files) == len(set(files))
    assert bench.source_digest("attention.hip") != bench.source_digest("vocab.hip")


def test_cpu_baseline_is_bounded_and_reports_stages():
    from workloads import make_inputs

    x = make_inputs(get_config("vicuna7b").replace(batch=3, n_q_heads=4, n_kv_heads=2, hidden=512, vocab=3000,
                                                   lengths=("explicit", (40, 90, 70))))
    out = bench.cpu_baseline(x, budget_s=0.0)          # stops after the first request
    assert out["requests"] == 1 and out["kind"] == "oracle"
    assert out["cores"] == len(os.sched_getaffinity(0))
    assert set(out["stage_s"]) == {"attention", "logits_softmax", "accept"}
    assert out["value"] > 0 and out["cpu_model"]
    full = bench.cpu_baseline(x, budget_s=1e9)         # the whole batch
    assert full["requests"] == 3


@pytest.mark.parametrize("nodes", [15, 31, 63])
def test_tree_nodes_set_the_node_count(nodes):
    cfg, problem = _cfg("--workload", "llama3_8b", "--tree-nodes", str(nodes))
    assert problem is None
    assert cfg.gamma == nodes and cfg.batch == get_config("llama3_8b").batch


@pytest.mark.parametrize("argv", [
    ("--tree-nodes", "15", "--sampling", "0.8,40,0.9"),
    ("--paged", "64", "--tree-nodes", "15"),
    ("--paged", "64", "--sampling", "1.0,0,0.9"),
    ("--starsd", "1.46,0.5", "--tree-nodes", "15"),
    ("--starsd", "1.46,0.5", "--sampling", "0.8,40,0.9"),
])
def test_modes_that_do_not_combine_are_refused(argv):
    cfg, problem = _cfg(*argv)
    assert cfg is None and problem


def test_more_than_one_gpu_is_refused(monkeypatch, capsys):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--gpus", "2"])
    assert bench.main() == 2
    assert "one GPU" in capsys.readouterr().err


def test_warmup_has_a_time_floor_besides_the_step_count():
    """--warmup steps always run; --warmup-ms (default 200 ms) keeps the
    warm-up going until the GPU has been busy that long, so that a short
    --warmup does not time steps run at idle clocks."""
    args = bench.parser().parse_args(["--steps", "20", "--warmup", "5"])
    assert args.warmup == 5 and args.steps == 20 and args.warmup_ms == 200.0
    assert bench.parser().parse_args(["--warmup-ms", "0"]).warmup_ms == 0.0
