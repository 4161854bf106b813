"""The descriptor-table cache policy of the multi-tensor step, on the host
(no GPU): the policy header the HIP library compiles is built with g++
against a fake backend that logs allocations and uploads
(tests/table_cache_test.cpp).  Checked: a repeated list uploads nothing; a
table is recycled only by a call on the stream of its latest use (so the
rewrite is queued behind every launch that read it), the least recently
used idle table of that stream with enough room; a table used while a
stream captures a graph is pinned and survives 40 further lists; a list
first seen during a capture is refused with no allocation or upload;
tables whose launches are not yet enqueued are never recycled; devices keep
separate caches; nothing is ever freed or waited for."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_table_cache_policy(tmp_path):
    exe = tmp_path / "table_cache_test"
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", "-fsanitize=address,undefined",
                    "-I", os.path.join(ROOT, "paper_2607_10611_amd", "csrc"),
                    os.path.join(ROOT, "tests", "table_cache_test.cpp"), "-o", str(exe)],
                   check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stderr
