"""Host-side parts of bench.py's contract: one GPU only, and the HBM traffic
figure read from the committed counter summary only while the kernel source
it was taken from is unchanged."""
import hashlib
import importlib.util
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_contract_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode != 0
    assert "one GPU" in p.stderr
    assert p.stdout.strip() == ""


def _traffic_block(name):
    text = open(os.path.join(ROOT, "profiles", name)).read()
    block = re.search(r"```traffic\n(.*?)```", text, re.S).group(1)
    return dict(line.split("=", 1) for line in block.strip().splitlines())


def test_traffic_follows_the_kernel_source_hash(tmp_path):
    b = _bench()
    name = "lm_head_8b_layer_p8192_traffic.md"
    kv = _traffic_block(name)
    src = open(os.path.join(ROOT, kv["source"]), "rb").read()
    current = hashlib.sha256(src).hexdigest() == kv["sha256"]
    got = b.measured_traffic(name)
    if current:
        assert got == int(kv["bytes_per_launch"]) and got > 0
    else:
        assert got is None
    # a summary whose recorded hash does not match its source gives null
    text = open(os.path.join(ROOT, "profiles", name)).read().replace(kv["sha256"], "0" * 64)
    os.makedirs(tmp_path / "profiles")
    (tmp_path / "profiles" / name).write_text(text)
    copied = tmp_path / kv["source"]
    os.makedirs(copied.parent)
    copied.write_bytes(src)
    b.ROOT = str(tmp_path)
    assert b.measured_traffic(name) is None
    # and the untouched summary beside the same source reads as before
    (tmp_path / "profiles" / name).write_text(open(os.path.join(ROOT, "profiles", name)).read())
    assert b.measured_traffic(name) == got
