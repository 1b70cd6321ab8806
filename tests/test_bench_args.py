"""Host-side checks of bench.py's command line: the schedule each workload
gets by default, and explicit flags taking precedence (no GPU, no torch)."""

import os
import sys

import pytest

import bench


def parsed(*argv):
    old = sys.argv
    sys.argv = ["bench.py", *argv]
    try:
        return bench.parse()
    finally:
        sys.argv = old


@pytest.mark.parametrize("argv,streams,assign,queues", [
    ((), 6, "balance", 8),                         # Llama-600M set, input side
    (("--sides", "both"), 6, "balance", 8),
    (("--ef",), 8, "balance", 8),                  # error feedback: eight streams
    (("--config", "4"), 4, "round-robin", 4),      # Llama-300M set keeps the four-stream deal
    (("--config", "2"), 4, "round-robin", 4),
    (("--hw-queues", "4", "--streams", "4", "--assign", "round-robin"), 4, "round-robin", 4),
    (("--streams", "3"), 3, "balance", 8),
    (("--config", "4", "--hw-queues", "0"), 4, "round-robin", 0),
])
def test_schedule_defaults(argv, streams, assign, queues):
    a = parsed(*argv)
    assert (a.streams, a.assign, a.hw_queues) == (streams, assign, queues)


def test_more_than_one_gpu_is_refused(capsys, monkeypatch):
    monkeypatch.delenv("GPU_MAX_HW_QUEUES", raising=False)
    old = sys.argv
    sys.argv = ["bench.py", "--gpus", "2"]
    try:
        with pytest.raises(SystemExit) as e:
            bench.main()
    finally:
        sys.argv = old
    assert e.value.code == 2
    assert "one GPU" in capsys.readouterr().err
    assert "GPU_MAX_HW_QUEUES" not in os.environ   # refused before touching it
