"""Host-side helpers of bench.py (no GPU): the staleness rule of the committed counters and the
pricing of the kernel's product mix at measured rates."""
import importlib.util
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_module", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_kernel_hash_ignores_comments_only(tmp_path):
    b = _bench()
    base = "// header\n__global__ void k(int* p) {\n  p[0] = 1;  // store\n  /* block\n comment */ p[1] = 2;\n}\n"
    recomment = "// another header\n\n__global__ void k(int* p) {\n  p[0] = 1;\n  p[1] = 2;   /* moved */\n}\n"
    changed = "// header\n__global__ void k(int* p) {\n  p[0] = 1;\n  p[1] = 3;\n}\n"
    paths = []
    for i, src in enumerate((base, recomment, changed)):
        f = tmp_path / f"k{i}.hip"
        f.write_text(src)
        paths.append(str(f))
    h = [b.kernel_source_hash(p) for p in paths]
    assert h[0] == h[1] and h[0] != h[2]


def test_committed_counters_record_their_source():
    """The committed HBM counters name the attention source they were taken on (a 16-digit hash
    under the rule of kernel_source_hash); bench.py reports their traffic only while it matches."""
    import json
    import re
    b = _bench()
    c = json.load(open(b.COUNTERS))
    assert re.fullmatch(r"[0-9a-f]{16}", c["kernel_source_sha256_16"])
    assert c["hbm_bytes_per_launch"] > 0
    assert (b.measured_traffic() is not None) == (c["kernel_source_sha256_16"] == b.kernel_source_hash())


def test_mix_ceiling_arithmetic(monkeypatch):
    b = _bench()
    rates = {"int8_32x32x32_random": {"tops": 3000.0}, "fp8_32x32x64_random": {"tops": 4000.0},
             "fp4_32x32x64_random": {"tops": 6000.0}}

    class R:
        returncode = 0
        stdout = '{"rate": %s}' % __import__("json").dumps(rates)
        stderr = ""

    monkeypatch.setattr(b.os.path, "exists", lambda p: True)
    import subprocess
    monkeypatch.setattr(subprocess, "run", lambda *a, **k: R())
    c = b.measured_ceiling(1500.0, 2000.0)
    # time per 2 score ops: 1/3000 (scores) + (1 + 1/8 + 1/16)/4000 (values, row sums, means)
    t = 1 / 3000 + (1 + 1 / 8 + 1 / 16) / 4000
    assert abs(c["attention_mix_ceiling_tops"] - 2 / t) < 1e-9
    assert abs(c["attention_frac_of_mix_ceiling"] - 1500.0 * t / 2) < 1e-12
    t4 = 1 / 6000 + (1 + 1 / 8 + 1 / 16) / 4000
    assert abs(c["mxfp4_mix_ceiling_tops"] - 2 / t4) < 1e-9
