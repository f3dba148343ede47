"""Host-side logic of bench.py (CPU only): the one-GPU guard, the work per
unit its roofline divides by, and the counter-reading lookup that reports
`roofline.traffic` only for the kernels the reading was taken on."""
import os
import subprocess
import sys

import pytest

import bench
from paper_2112_15317_amd import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# VGG-16 on 32x32 inputs: (input channels, output channels, image side) per
# conv layer, written out from the architecture (13 convs, pools after 2, 4,
# 7, 10, 13).
VGG16_CIFAR = [(3, 64, 32), (64, 64, 32), (64, 128, 16), (128, 128, 16), (128, 256, 8),
               (256, 256, 8), (256, 256, 8), (256, 512, 4), (512, 512, 4), (512, 512, 4),
               (512, 512, 2), (512, 512, 2), (512, 512, 2)]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout.strip()


def test_stack_flops_closed_form():
    """Three passes per layer; a 3x3 tap with padding 1 is inside an n-pixel
    axis for 3n - 2 of its 3n (position, offset) pairs."""
    n = 128
    layers = configs.conv_layers(configs.VGG16, 3, 32)
    assert [(L.c, L.k, L.h) for L in layers] == VGG16_CIFAR
    nominal = sum(3 * 2 * n * k * c * 9 * s * s for c, k, s in VGG16_CIFAR)
    valid = sum(3 * 2 * n * k * c * (3 * s - 2) ** 2 for c, k, s in VGG16_CIFAR)
    f = configs.stack_flops(layers, n)
    assert f == {"nominal": nominal, "valid": valid}
    assert round(nominal / 1e9, 2) == 240.53 and round(valid / 1e9, 2) == 189.93
    for L, (c, k, s) in zip(layers, VGG16_CIFAR):
        assert bench.layer_flops(L, n) == (2 * n * k * c * (3 * s - 2) ** 2,
                                           2 * n * k * c * 9 * s * s)


def test_pool_bytes_per_window():
    L = configs.conv_layers(configs.VGG16, 3, 32)[1]           # 64 channels, 32x32
    for es in (4, 2):
        assert bench.pool_bytes(L, 8, es) == 8 * 64 * 16 * 16 * (5 * es + 1)


def _fake_tree(tmp_path, digest_line):
    (tmp_path / "paper_2112_15317_amd" / "csrc").mkdir(parents=True)
    (tmp_path / "paper_2112_15317_amd" / "csrc" / "k.hip").write_text("// kernel\n")
    (tmp_path / "profiles").mkdir()
    body = ("# HBM traffic\n\nworkload: wl-a\n%s\n\n"
            "| kernel | launches | traffic_bytes_per_launch |\n|---|---:|---:|\n"
            "| `sb::k<1>` | 3 | 1234 |\n" % digest_line)
    (tmp_path / "profiles" / "x_hbm_traffic.md").write_text(body)


def test_stored_traffic_needs_the_current_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    _fake_tree(tmp_path, "csrc_sha256: 0")
    digest = bench.csrc_digest()
    assert bench.stored_traffic("sb::k<1>", "wl-a") is None          # stale reading
    text = (tmp_path / "profiles" / "x_hbm_traffic.md").read_text()
    (tmp_path / "profiles" / "x_hbm_traffic.md").write_text(
        text.replace("csrc_sha256: 0", "csrc_sha256: " + digest))
    assert bench.stored_traffic("sb::k<1>", "wl-a") == 1234
    assert bench.stored_traffic("sb::k<2>", "wl-a") is None          # no such kernel
    assert bench.stored_traffic("sb::k<1>", "wl-b") is None          # another workload
    (tmp_path / "paper_2112_15317_amd" / "csrc" / "k.hip").write_text("// changed\n")
    assert bench.stored_traffic("sb::k<1>", "wl-a") is None          # sources changed


def test_committed_profiles_name_their_sources():
    """Every committed HBM-traffic summary records the workload and the
    source digest it was taken on (bench.py reports it only while they
    match)."""
    import glob
    import re
    paths = glob.glob(os.path.join(ROOT, "profiles", "*hbm_traffic*.md"))
    assert paths
    for p in paths:
        text = open(p).read()
        assert re.search(r"^csrc_sha256: *[0-9a-f]{64}$", text, re.M), p
        assert re.search(r"^workload: *\S+", text, re.M), p
