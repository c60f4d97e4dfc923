"""Host-side pieces of bench.py, on the CPU: the refusal of a multi-GPU run, and the visible-pair
counts behind its causal-adjusted FLOP figures (14 d Hq A per fwd+bwd), checked against a
brute-force count of the mask and against the work of the context-parallel shares."""
import os
import subprocess
import sys

import numpy as np
import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def brute_pairs(lq, lk, diag):
    """Visible (query, key) pairs counted element by element: key j is visible to query i iff
    j <= i + diag (global positions k_off + j <= q_off + i with diag = q_off - k_off)."""
    i = np.arange(lq)[:, None]
    j = np.arange(lk)[None, :]
    return int(np.count_nonzero(j <= i + diag))


@pytest.mark.parametrize("lq,lk", [(0, 5), (5, 0), (1, 1), (7, 3), (3, 7), (64, 64), (65, 129)])
def test_chunk_pair_counts_match_brute_force(lq, lk):
    for diag in (-lq - lk - 3, -lq, -1, 0, 1, lk - 1, lk, lk + lq + 5):
        want = brute_pairs(lq, lk, diag)
        assert bench.visible_pairs_chunk(lq, lk, diag) == want, (lq, lk, diag)
        assert bench.visible_pairs_chunk_closed(lq, lk, diag) == want, (lq, lk, diag)


def test_context_parallel_share_areas():
    """A of the two chunk workloads: 8 steps of a 32K Q chunk at 1,015,808 against KV chunks at
    24..31 x 32K (seven fully in the past, one diagonal), and the zig-zag share's four part pairs
    (parts 0 and 7 of a 256K sequence, one pair entirely in the future)."""
    c = 32768
    _, _, cc, q_offs, kv_offs, pairs = bench.chunk_workload("cp7b")
    assert cc == c and len(pairs) == 8
    a = sum(bench.visible_pairs_chunk_closed(c, c, q_offs[i] - kv_offs[j]) for i, j in pairs)
    assert a == 7 * c * c + c * (c + 1) // 2 == 8_053_080_064
    _, _, _, q_offs, kv_offs, pairs = bench.chunk_workload("zigzag141b")
    per = [bench.visible_pairs_chunk_closed(c, c, q_offs[i] - kv_offs[j]) for i, j in pairs]
    assert sorted(per) == [0, c * (c + 1) // 2, c * (c + 1) // 2, c * c]
    assert sum(per) == 2_147_516_416


def test_more_than_one_gpu_is_refused_before_any_device_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2, (r.returncode, r.stderr[-500:])
    assert "--gpus 2 is not supported" in r.stderr
    assert r.stdout.strip() == ""


def test_counter_records_survive_comment_edits_only(tmp_path, monkeypatch):
    """A counter record is matched to the kernel's sources without their comments and blank
    lines: editing a comment keeps it, editing code drops it."""
    import shutil
    csrc = os.path.join(ROOT, "paper_2502_21231_amd", "csrc")
    dst = tmp_path / "paper_2502_21231_amd" / "csrc"
    dst.mkdir(parents=True)
    for f in set(sum(bench.KERNEL_SOURCES.values(), [])):
        shutil.copy(os.path.join(csrc, f), dst / f)
    monkeypatch.setattr(bench, "REPO", str(tmp_path))
    before = {k: bench.kernel_source_hash(k) for k in bench.KERNEL_SOURCES}
    p = dst / "dkdv_bf16.hip"
    text = p.read_text()
    p.write_text("// a new first line\n\n" + text.replace("\n", "\n\n", 3) + "/* and a block\n comment */\n")
    assert {k: bench.kernel_source_hash(k) for k in bench.KERNEL_SOURCES} == before
    p.write_text(text.replace("n_vis - 1 - s", "n_vis - s", 1))
    after = {k: bench.kernel_source_hash(k) for k in bench.KERNEL_SOURCES}
    assert after["bwd_dkdv"] != before["bwd_dkdv"]
    assert after["fwd"] == before["fwd"] and after["bwd_dq"] == before["bwd_dq"]
