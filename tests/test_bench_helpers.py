"""Host logic of bench.py (no GPU): the kernel-code hash that keys the stored
counter figures, the lookup of those figures, and the refusal of more than
one GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

CODE = """// a kernel
__global__ void k(float* p)   // the body
{
    /* one
       comment */
    p[0] = 1.0f;
}
"""


def _tree(tmp_path, src, profile_lines):
    csrc = tmp_path / "paper_1706_03292_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "k.hip").write_text(src)
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "k_workload.md").write_text("\n".join(profile_lines) + "\n")
    return str(tmp_path)


def test_code_hash_ignores_comments_and_blank_lines_only(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", _tree(tmp_path, CODE, []))
    h = bench._kernel_source_hash("k.hip")
    edited = CODE.replace("// the body", "// another comment").replace("/* one", "/* two") + "\n\n// trailing\n"
    (tmp_path / "paper_1706_03292_amd" / "csrc" / "k.hip").write_text(edited)
    assert bench._kernel_source_hash("k.hip") == h
    (tmp_path / "paper_1706_03292_amd" / "csrc" / "k.hip").write_text(CODE.replace("1.0f", "2.0f"))
    assert bench._kernel_source_hash("k.hip") != h


def test_stored_traffic_only_for_the_current_code(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", _tree(tmp_path, CODE, []))
    h = bench._kernel_source_hash("k.hip")
    lines = [f"`traffic: kernel=k source_sha256={h} bytes_per_launch=1234`",
             "`traffic: kernel=k source_sha256=0000000000000000 bytes_per_launch=999`",
             f"`traffic: kernel=other source_sha256={h} bytes_per_step=5`"]
    (tmp_path / "profiles" / "k_workload.md").write_text("\n".join(lines) + "\n")
    assert bench._stored_traffic("k", "k.hip") == 1234.0
    assert bench._stored_traffic("other", "k.hip") == 5.0
    (tmp_path / "paper_1706_03292_amd" / "csrc" / "k.hip").write_text(CODE.replace("1.0f", "2.0f"))
    assert bench._stored_traffic("k", "k.hip") is None


def test_committed_profiles_match_the_current_kernels():
    # the figures bench.py reports as `traffic` come from these summaries
    assert bench._stored_traffic("sf_apply", "sf_apply.hip") is not None
    assert bench._stored_traffic("ps_apply_largest", "ps_apply.hip") is not None


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       env={**os.environ, **env}, timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "error" in line and "one GPU" in r.stderr
