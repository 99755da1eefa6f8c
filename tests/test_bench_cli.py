"""bench.py contract checks that need no GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_rows_listed_in_help():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--help"], capture_output=True, text=True,
                       timeout=60)
    assert r.returncode == 0 and "kv_vmm" in r.stdout and "file" in r.stdout


def test_traffic_digest_ignores_comments_but_not_code(tmp_path, monkeypatch):
    """The stored traffic counts stay valid across comment edits and lapse on code edits."""
    import shutil

    import bench

    for rel in bench.KERNEL_SOURCES + [bench.HEADER, bench.CHUNKING[0]]:
        dst = tmp_path / rel
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copy(os.path.join(bench.ROOT, rel), dst)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    base = bench.kernel_source_digest()
    k = tmp_path / bench.KERNEL_SOURCES[0]
    src = k.read_text()
    k.write_text("// a new comment line\n" + src.replace("namespace gms {", "namespace gms {  /* x */", 1))
    assert bench.kernel_source_digest() == base
    k.write_text(src.replace("constexpr uint32_t kXcds = 8;", "constexpr uint32_t kXcds = 4;", 1))
    assert "constexpr uint32_t kXcds = 8;" in src and bench.kernel_source_digest() != base
    k.write_text(src)
    c = tmp_path / bench.CHUNKING[0]
    cs = c.read_text()
    c.write_text(cs.replace("constexpr uint64_t kSplitUnits = 16384;", "constexpr uint64_t kSplitUnits = 8192;", 1))
    assert "constexpr uint64_t kSplitUnits = 16384;" in cs and bench.kernel_source_digest() != base
    c.write_text(cs)
    h = tmp_path / bench.HEADER
    hs = h.read_text()
    h.write_text(hs.replace("#define GMS_DEFAULT_CHUNK_BYTES (64u * 1024u)", "#define GMS_DEFAULT_CHUNK_BYTES (256u * 1024u)"))
    assert bench.kernel_source_digest() != base
