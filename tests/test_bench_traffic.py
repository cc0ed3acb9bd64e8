"""The HBM traffic that bench.py reports beside its roofline comes from a
stored counter record (profiles/traffic_<workload>.json).  It may be reported
only for the kernels the counters saw: the same kernel sources and, for a
conv layer, the same tile configuration in the current tuning table (CPU)."""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_1511_07376_amd import workloads as wl  # noqa: E402

TUNE = "64 3 227 227 96 11 11 4 4 0 0 1 6\n64 96 31 31 256 5 5 1 1 0 0 2 0\n64 384 13 13 384 3 3 1 1 1 1 2 9"


def _layers(net, kind):
    return [layer for layer in net.layers if layer.kind == kind]


def test_conv_configs_of_matches_channels_filter_stride_groups():
    conv1, conv2, _, conv4, conv5 = _layers(wl.alexnet, "conv")
    assert bench.conv_configs_of(TUNE, conv1) == [6]
    assert bench.conv_configs_of(TUNE, conv2) == [0]   # bordered 31x31 input, no padding
    assert bench.conv_configs_of(TUNE, conv4) == [9]
    assert bench.conv_configs_of(TUNE, conv5) == []    # 256 output channels: no line
    assert bench.conv_configs_of("", conv1) == []


def _record(d, name, digest, tuning, conv2_bytes=123):
    rec = {"source_digest": digest, "tuning": tuning.splitlines(),
           "layers": {"conv2": {"hbm_bytes_per_launch": conv2_bytes}, "pool3": {"hbm_bytes_per_launch": 7}}}
    (d / name).write_text(json.dumps(rec))


def test_traffic_needs_the_same_sources_and_tiles(tmp_path):
    conv2 = _layers(wl.alexnet, "conv")[1]
    pool3 = _layers(wl.alexnet, "pool")[2]
    d = str(tmp_path)
    _record(tmp_path, "traffic_w.json", bench.source_digest(), TUNE)
    assert bench.stored_traffic("w", "conv2", conv2, TUNE, prof_dir=d) == 123
    # conv2 tuned to another configuration, or not tuned at all (the heuristic's pick)
    other = TUNE.replace(" 2 0\n", " 2 2\n")
    assert bench.stored_traffic("w", "conv2", conv2, other, prof_dir=d) is None
    assert bench.stored_traffic("w", "conv2", conv2, "", prof_dir=d) is None
    # a pooling layer has no tiles: the sources decide alone
    assert bench.stored_traffic("w", "pool3", pool3, "", prof_dir=d) == 7
    assert bench.stored_traffic("w", "fc9", None, TUNE, prof_dir=d) is None
    # a record taken with the other configuration applies to it, not to the first
    _record(tmp_path, "traffic_w_conv2cfg2.json", bench.source_digest(), other, conv2_bytes=456)
    assert bench.stored_traffic("w", "conv2", conv2, other, prof_dir=d) == 456
    assert bench.stored_traffic("w", "conv2", conv2, TUNE, prof_dir=d) == 123
    # records of other kernel sources never apply
    _record(tmp_path, "traffic_w.json", "0" * 16, TUNE)
    _record(tmp_path, "traffic_w_conv2cfg2.json", "0" * 16, other)
    assert bench.stored_traffic("w", "conv2", conv2, TUNE, prof_dir=d) is None
    assert bench.stored_traffic("w", "pool3", pool3, TUNE, prof_dir=d) is None


def test_no_records_at_all(tmp_path):
    conv2 = _layers(wl.alexnet, "conv")[1]
    assert bench.stored_traffic("w", "conv2", conv2, TUNE, prof_dir=str(tmp_path)) is None
    assert bench.stored_traffic("w", "conv2", conv2, TUNE, prof_dir=str(tmp_path / "missing")) is None


def test_committed_records_carry_their_tuning_table():
    for name in os.listdir(os.path.join(ROOT, "profiles")):
        if name.startswith("traffic_") and name.endswith(".json"):
            with open(os.path.join(ROOT, "profiles", name)) as f:
                rec = json.load(f)
            assert rec.get("tuning"), name
            assert all(len(line.split()) == 13 for line in rec["tuning"]), name
