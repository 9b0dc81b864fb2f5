"""Host-side checks of bench.py: the one-GPU rule and the counter-traffic record."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.fixture
def bench(monkeypatch):
    import bench as b

    monkeypatch.setattr(b, "PLAN_OPTIONS", {"u_ranges": 0, "pace_windows": 0})
    return b


def test_traffic_record_matches_kernel_source(bench):
    """Every workload has a counter record; the bench uses it (bytes = read +
    written) only while the library sources still hash to the recorded
    values, and reports null traffic otherwise."""
    for c in (1, 2, 3, 4, 5, 6):
        text = open(os.path.join(ROOT, "profiles", bench.TRAFFIC_RECORDS[c])).read()
        raw = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
        assert raw["traffic_bytes_per_launch"] == raw["read_bytes_per_launch"] + raw["write_bytes_per_launch"]
        rec = bench.traffic_record(c)
        fresh = raw.get("library_sha256") == bench.library_sha256(ROOT)
        assert (rec is not None) == fresh, c
        if rec is not None:
            assert rec["bytes"] == rec["read_bytes"] + rec["write_bytes"]
    # only for the launch configuration the counters were taken on
    assert bench.traffic_record(4, "binary") is None
    assert bench.traffic_record(6, "binary") is None
    bench.PLAN_OPTIONS["u_ranges"] = 8
    assert bench.traffic_record(2) is None


def test_traffic_record_null_after_kernel_change(bench, tmp_path, monkeypatch):
    name = bench.TRAFFIC_RECORDS[2]
    text = open(os.path.join(ROOT, "profiles", name)).read()
    rec = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    rec["kernel_source_sha256"] = "0" * 64
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / name).write_text("```json\n" + json.dumps(rec) + "\n```\n")
    src_dir = tmp_path / os.path.dirname(rec["kernel_source"])
    src_dir.mkdir(parents=True)
    (tmp_path / rec["kernel_source"]).write_bytes(open(os.path.join(ROOT, rec["kernel_source"]), "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.traffic_record(2) is None


def test_traffic_record_null_after_library_change(bench, tmp_path, monkeypatch):
    """A change anywhere in the library (unit building, join order, launch
    choice) voids the counters even when the kernel's own file is unchanged."""
    import shutil

    import hashlib

    name = bench.TRAFFIC_RECORDS[3]
    shutil.copytree(os.path.join(ROOT, "profiles"), tmp_path / "profiles")
    shutil.copytree(os.path.join(ROOT, "paper_2603_08957_amd", "csrc"), tmp_path / "paper_2603_08957_amd" / "csrc")
    # a record taken on exactly these sources
    path = tmp_path / "profiles" / name
    text = path.read_text()
    rec = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    rec["kernel_source_sha256"] = hashlib.sha256((tmp_path / rec["kernel_source"]).read_bytes()).hexdigest()
    rec["library_sha256"] = bench.library_sha256(str(tmp_path))
    path.write_text("```json\n" + json.dumps(rec) + "\n```\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.traffic_record(3) is not None, name
    with open(tmp_path / "paper_2603_08957_amd" / "csrc" / "api.cpp", "a") as f:
        f.write("\n")
    assert bench.traffic_record(3) is None


def test_relation_from_dense_matches_the_generator(bench):
    """The planner check lays out dense arrays as relations: for the
    adjacency of the 4096-vertex graph in 64 x 64 tiles' promoted form (here
    both labels promoted with tiles of 1) the keys are the edges and the
    tiles their values; with nothing promoted one tuple holds the array."""
    import numpy as np

    import workloads

    w = workloads.config(1, "small", y_layout="jk")
    n = w["n"]
    Y = np.zeros((n, n), np.float32)
    Y[w["Y"]["coo"][0][:, 0], w["Y"]["coo"][0][:, 1]] = w["Y"]["coo"][1]
    rel = bench.relation_from_dense(Y, "jk", {"j", "k"})
    assert np.array_equal(rel["keys"], w["Y"]["coo"][0].astype(np.int32))
    assert np.array_equal(rel["tiles"][:, 0], w["Y"]["coo"][1].astype(np.float32))
    rows = bench.relation_from_dense(Y, "jk", {"k"})
    assert np.array_equal(rows["keys"][:, 0], np.unique(w["Y"]["coo"][0][:, 1]))
    assert np.array_equal(rows["tiles"], Y.T[rows["keys"][:, 0]])
    one = bench.relation_from_dense(Y, "jk", set())
    assert one["keys"].shape == (1, 0) and np.array_equal(one["tiles"][0], Y.reshape(-1))
    # with tiles: the generator's own 64 x 64 relation
    tiled = bench.relation_from_dense(Y, "jk", {"j": 64, "k": 64})
    assert np.array_equal(tiled["keys"], w["Y"]["keys"]) and np.array_equal(tiled["tiles"], w["Y"]["tiles"])
    coo = bench.relation_from_coo(w["Y"]["coo"][0], w["Y"]["values"], "jk", {"j": 64, "k": 64}, {"j": n, "k": n},
                                  1 << 30, "f32")
    assert np.array_equal(coo["keys"], w["Y"]["keys"]) and np.array_equal(coo["tiles"], w["Y"]["tiles"])
    emb = w["emb"]
    X = np.ascontiguousarray(w["X"]["tiles"].reshape(n // 64, emb, 64).transpose(1, 0, 2).reshape(emb, n))
    xr = bench.relation_from_dense(X, "ij", {"j": 64})
    assert np.array_equal(xr["keys"], w["X"]["keys"]) and np.array_equal(xr["tiles"], w["X"]["tiles"])


def test_relation_from_coo(bench):
    """Entries of a sparse tensor laid out under a promoted set: keys are the
    distinct promoted coordinates, tiles dense over the demoted labels; too
    large a layout is refused."""
    import numpy as np

    coords = np.array([[0, 2], [0, 5], [3, 1], [3, 2]], np.int64)
    vals = np.array([1.0, 2.0, 3.0, 4.0], np.float32)
    ext = {"j": 4, "k": 6}
    r = bench.relation_from_coo(coords, vals, "jk", {"j", "k"}, ext, 1 << 20, "f32")
    assert np.array_equal(r["keys"], coords.astype(np.int32)) and np.array_equal(r["tiles"][:, 0], vals)
    r = bench.relation_from_coo(coords, vals, "jk", {"j"}, ext, 1 << 20, "f32")
    assert r["keys"].reshape(-1).tolist() == [0, 3]
    assert r["tiles"].tolist() == [[0, 0, 1, 0, 0, 2], [0, 3, 4, 0, 0, 0]]
    r = bench.relation_from_coo(coords, vals, "jk", {"k"}, ext, 1 << 20, "f32")
    assert r["keys"].reshape(-1).tolist() == [1, 2, 5]
    assert r["tiles"].tolist() == [[0, 0, 0, 3], [1, 0, 0, 4], [2, 0, 0, 0]]
    r = bench.relation_from_coo(coords, vals, "jk", set(), ext, 1 << 20, "f32")
    assert r["keys"].shape == (1, 0) and r["tiles"].reshape(4, 6)[3, 2] == 4.0
    assert bench.relation_from_coo(coords, vals, "jk", set(), ext, 64, "f32") is None
