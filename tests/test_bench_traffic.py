"""bench.py on the CPU: it reports a kernel's HBM traffic from a committed
counter summary only while that summary was taken from the current sources
(every file the entry point's kernels are built from must match the
recorded hash), and it refuses to measure more than one GPU."""
import os

import bench


def _setup(tmp_path, monkeypatch, sources):
    for rel, text in sources.items():
        path = tmp_path / rel
        path.parent.mkdir(parents=True, exist_ok=True)
        path.write_text(text)
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", {"cluster": list(sources)})


def _write_summary(tmp_path, digest, nbytes=12345):
    (tmp_path / "profiles" / "cluster_w_counters.md").write_text(
        f"HBM bytes per launch (scaled): {nbytes}\n\nsource sha256[:16]: `{digest}` (files)\n")


def test_traffic_needs_every_source_to_match(tmp_path, monkeypatch):
    sources = {"a.hip": "kernel a", "b.hip": "kernel b", "c.h": "common"}
    _setup(tmp_path, monkeypatch, sources)
    digest = bench.source_hash(list(sources))
    _write_summary(tmp_path, digest)
    assert bench.committed_traffic("cluster", "w") == 12345.0
    # a change in any one of the files voids the summary
    (tmp_path / "b.hip").write_text("kernel b, changed")
    assert bench.committed_traffic("cluster", "w") is None


def test_traffic_absent_or_unhashed(tmp_path, monkeypatch):
    _setup(tmp_path, monkeypatch, {"a.hip": "kernel a"})
    assert bench.committed_traffic("cluster", "w") is None  # no summary
    (tmp_path / "profiles" / "cluster_w_counters.md").write_text("HBM bytes per launch (scaled): 5\n")
    assert bench.committed_traffic("cluster", "w") is None  # no hash line


def test_source_hash_is_order_sensitive(tmp_path, monkeypatch):
    _setup(tmp_path, monkeypatch, {"a.hip": "x", "b.hip": "y"})
    assert bench.source_hash(["a.hip", "b.hip"]) != bench.source_hash(["b.hip", "a.hip"])
    assert len(bench.source_hash(["a.hip"])) == 16
    assert os.path.isabs(bench.ROOT)


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: --gpus above 1 (or a multi-rank launch)
    exits with status 2 and says why, before touching torch or the GPU."""
    import subprocess
    import sys
    env = dict(os.environ, WORLD_SIZE="1")
    r = subprocess.run([sys.executable, os.path.join(bench.ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, env=env, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr
    env["WORLD_SIZE"] = "4"
    r = subprocess.run([sys.executable, os.path.join(bench.ROOT, "bench.py")], capture_output=True, text=True,
                       env=env, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr
