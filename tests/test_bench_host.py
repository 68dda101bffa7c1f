"""Host-side pieces of bench.py that need no GPU."""
import importlib.util
import os

import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _summary(digest, shapes):
    lines = [f"kernel sources digest: `{digest}`", ""]
    lines += [f"HBM bytes per launch (scaled), block {b}, LDS {l}, row chunks {r}: {v:.6e}"
              for (b, l, r), v in shapes.items()]
    return "\n".join(lines) + "\n"


def test_traffic_is_read_for_the_launch_shape_and_current_sources(bench, tmp_path, monkeypatch):
    w = W.full_workloads()["vgg16_adaptive"]
    assert (w.K, w.P) == (8, 138_000_000)
    f = tmp_path / "traffic.md"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    shapes = {(64, 0, 1): 1.8768e10, (64, 8192, 1): 1.8769e10, (128, 0, 1): 1.877e10, (64, 8192, 32): 1.8771e10}
    f.write_text(_summary(bench.kernel_source_digest(), shapes))
    for (b, l, r), v in shapes.items():
        assert bench.measured_traffic(w, b, l, r) == pytest.approx(v, rel=1e-6)
    assert bench.measured_traffic(w, 256, 0, 1) is None       # shape not profiled
    assert bench.measured_traffic(w, 64, 8192, 3) is None     # no prefix match of a figure
    assert bench.measured_traffic(w, 64, 819, 1) is None
    f.write_text(_summary("0" * 16, shapes))                  # counters from other sources
    assert bench.measured_traffic(w, 64, 0, 1) is None
    assert bench.measured_traffic(W.parity_workloads()["resnet18_like"], 64, 0, 1) is None


def test_more_than_one_gpu_is_refused(bench, monkeypatch, capsys):
    monkeypatch.setattr("sys.argv", ["bench.py", "--gpus", "2"])
    with pytest.raises(SystemExit) as e:
        bench.main()
    assert e.value.code == 2
    assert "one GPU" in capsys.readouterr().err


def test_source_digest_ignores_comments_not_code(bench):
    """The counter figures describe compiled kernels: comment and whitespace
    edits leave the digest alone, a change of code does not."""
    code = 'int f(int a) {  // the sum\n  /* twice */ return a + a; }\nconst char *s = "// kept";\n'
    same = 'int f(int a) {\n  return a + a;   // another comment\n}\nconst char *s = "// kept";\n'
    other = 'int f(int a) { return a * 2; }\nconst char *s = "// kept";\n'
    assert bench.code_tokens(code) == bench.code_tokens(same)
    assert bench.code_tokens(code) != bench.code_tokens(other)
    assert '"// kept"' in bench.code_tokens(code)
