"""Host-side parts of bench.py (no GPU): the algorithmic work model against
a brute-force count, the one-GPU contract, and the rule that a committed
profile's traffic figure applies only to the kernel sources it was taken
from."""
import os
import shutil
import subprocess
import sys
import types

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _batch(prefix, qlen, page):
    return types.SimpleNamespace(prefix_lens=np.array(prefix, dtype=np.int32), q_lens=np.array(qlen, dtype=np.int32),
                                 page_size=page, num_reqs=len(prefix))


def test_algorithmic_work_matches_a_brute_force_count():
    prefix, qlen, page = [10, 5, 0, 63], [1, 3, 2, 1], 4
    w = bench.algorithmic_work(_batch(prefix, qlen, page))
    pairs, pages, rows, cached = 0, 0, 0, 0
    for p, c in zip(prefix, qlen):
        for i in range(c):  # query token i of the request sees keys 0 .. p + i (causal)
            pairs += sum(1 for _ in range(p + i + 1))
        pages += len({k // page for k in range(p + c)})  # block-table entries the request uses
        rows += c
        cached += p
    assert w["pairs"] == pairs and w["rows"] == rows and w["keys"] == sum(prefix) + sum(qlen)
    assert w["flops"] == pairs * 2 * 16 * (576 + 512)
    q_bytes, out_bytes = rows * 16 * 576 * 2, rows * 16 * 512 * 4
    common = q_bytes + out_bytes + 4 * pages + 8 * len(prefix)
    # fused step: cached latents read once, new latents read and written once
    assert w["step_bytes"] == cached * 1152 + 2 * rows * 1152 + common
    # attention alone: every key (cached or new) read once from the cache
    assert w["attn_bytes"] == (cached + rows) * 1152 + common


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stdout and "--gpus 2" in r.stdout


def _tree(tmp_path):
    src = os.path.join(ROOT, "paper_2607_02043_amd", "csrc")
    dst = tmp_path / "paper_2607_02043_amd" / "csrc"
    dst.mkdir(parents=True)
    for f in ("mla_kernels.hip", "mla_api.cpp", "mla_kernels.h"):
        shutil.copy(os.path.join(src, f), dst / f)
    return dst


def test_kernel_hash_ignores_comments_and_follows_code(tmp_path):
    dst = _tree(tmp_path)
    h0 = bench.kernel_source_hash(str(tmp_path))
    assert h0 == bench.kernel_source_hash()
    f = dst / "mla_api.cpp"
    text = f.read_text()
    f.write_text("// a new comment\n\n/* and a block\n   comment */\n" + text.replace("\n", "  // trailing\n", 3))
    assert bench.kernel_source_hash(str(tmp_path)) == h0
    f.write_text(text.replace("constexpr", "constexpr ", 1) + "\nstatic int changed_code = 1;\n")
    assert bench.kernel_source_hash(str(tmp_path)) != h0


def test_profile_traffic_applies_only_to_its_sources(tmp_path):
    _tree(tmp_path)
    (tmp_path / "profiles").mkdir()
    h = bench.kernel_source_hash(str(tmp_path))
    prof = tmp_path / "profiles" / "mixed_step_config2.md"
    prof.write_text(f"# summary\n\n    kernel_source_sha256_16: {h}\n    traffic_bytes_per_call: 123456\n")
    assert bench.profiled_traffic(2, str(tmp_path)) == 123456
    prof.write_text("# summary\n\n    kernel_source_sha256_16: 0000000000000000\n    traffic_bytes_per_call: 123456\n")
    assert bench.profiled_traffic(2, str(tmp_path)) is None
    assert bench.profiled_traffic(3, str(tmp_path)) is None  # no profile for that workload
