"""The C-ABI from plain C, and the oracle and host code under sanitizers (CPU only)."""
import os
import subprocess

import pytest

import oracle
import paper_2609_25451_amd as gms

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))


def _run(cmd, **kw):
    return subprocess.run(cmd, capture_output=True, text=True, timeout=300, **kw)


def test_header_is_c99_and_abi_works_from_c(tmp_path):
    exe = tmp_path / "abi_host"
    libdir = os.path.dirname(gms.LIB_PATH)
    r = _run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
              os.path.join(HERE, "c", "abi_host.c"), "-L", libdir, "-lgms", f"-Wl,-rpath,{libdir}",
              "-o", str(exe)])
    assert r.returncode == 0, r.stderr
    r = _run([str(exe)])
    assert r.returncode == 0 and "abi_host ok" in r.stdout, r.stdout + r.stderr


def test_oracle_under_address_and_ub_sanitizers(tmp_path):
    """Brute-force round trips and hashes of ragged inputs through an ASan/UBSan build of the oracle."""
    drv = tmp_path / "drv.c"
    drv.write_text(r'''
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include "oracle.h"
int main(void) {
    uint64_t state = 12345;
    for (int rep = 0; rep < 300; ++rep) {
        uint64_t n = 1 + rep % 7, sz[8], total = 0;
        uint8_t *src[8], *dst[8];
        for (uint64_t i = 0; i < n; ++i) {
            state = state * 6364136223846793005ull + 1442695040888963407ull;
            sz[i] = (state >> 33) % 9000;
            src[i] = malloc(sz[i] + 1); dst[i] = malloc(sz[i] + 1);
            for (uint64_t k = 0; k < sz[i]; ++k) src[i][k] = (uint8_t)(k * 31 + i);
            total += sz[i];
        }
        uint64_t off[8], base[8], ib, nb;
        oracle_layout(sz, n, off, base, &ib, &nb);
        uint8_t *img = malloc(ib + 1);
        oracle_pack((const uint8_t *const *)src, sz, n, img);
        oracle_unpack(img, dst, sz, n);
        for (uint64_t i = 0; i < n; ++i) if (sz[i] && memcmp(src[i], dst[i], sz[i])) return 2;
        uint64_t *blk = malloc((nb + 1) * 8), ten[8], list[4];
        oracle_hash((const uint8_t *const *)src, sz, n, blk, ten);
        if (oracle_verify((const uint8_t *const *)dst, sz, n, blk, list, 4) != 0) return 3;
        for (uint64_t i = 0; i < n; ++i)
            for (uint64_t b = 0; b * 4096 < sz[i]; ++b)
                if (oracle_block_hash_at(src[i] + 4096 * b, sz[i], b) != blk[base[i] + b]) return 4;
        free(blk); free(img);
        for (uint64_t i = 0; i < n; ++i) { free(src[i]); free(dst[i]); }
        (void)total;
    }
    puts("oracle sanitized ok");
    return 0;
}
''')
    exe = tmp_path / "drv"
    r = _run(["gcc", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-I", oracle.HERE,
              str(drv), oracle.SOURCE, "-o", str(exe)])
    if r.returncode != 0 and "asan" in r.stderr.lower():
        pytest.skip("sanitizer runtime not available: " + r.stderr[:200])
    assert r.returncode == 0, r.stderr
    r = _run([str(exe)])
    assert r.returncode == 0 and "oracle sanitized ok" in r.stdout, r.stdout + r.stderr


def test_host_code_under_sanitizers(tmp_path):
    """The library's host code under ASan/UBSan: validation, overlap sort, layout and chunking
    (a fuzzed manifest builder), and the owner process's message handling (a fuzzed peer)."""
    lib = tmp_path / "libgms_san.so"
    srcs = sorted(os.path.join(ROOT, "paper_2609_25451_amd", "csrc", f)
                  for f in os.listdir(os.path.join(ROOT, "paper_2609_25451_amd", "csrc")) if f.endswith(".hip"))
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    r = _run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
              "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
              "-Xarch_host", "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"), *srcs, "-o", str(lib)])
    assert r.returncode == 0, r.stderr[-2000:]
    exe = tmp_path / "fuzz"
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc)), "..", "lib", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    # the sanitized library carries clang's sanitizer runtime, so the driver is linked by clang too
    r = _run([clang, "-std=c99", "-O1", "-g", "-fsanitize=address,undefined", "-I", os.path.join(ROOT, "include"),
              os.path.join(HERE, "c", "manifest_fuzz.c"), str(lib), f"-Wl,-rpath,{tmp_path}", "-o", str(exe)])
    if r.returncode != 0 and "asan" in r.stderr.lower():
        pytest.skip("sanitizer runtime not available: " + r.stderr[:200])
    assert r.returncode == 0, r.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="halt_on_error=1")
    r = _run([str(exe)], env=env)
    assert r.returncode == 0 and "manifest fuzz ok" in r.stdout, (r.stdout + r.stderr)[-3000:]
    # the owner process's message handling against hostile peers, in the same sanitized build
    exe = tmp_path / "owner_fuzz"
    r = _run([clang, "-std=c99", "-O1", "-g", "-pthread", "-fsanitize=address,undefined", "-I",
              os.path.join(ROOT, "include"), os.path.join(HERE, "c", "owner_fuzz.c"), str(lib),
              f"-Wl,-rpath,{tmp_path}", "-o", str(exe)])
    assert r.returncode == 0, r.stderr[-2000:]
    r = _run([str(exe), str(tmp_path / "owner.sock")], env=env)
    assert r.returncode == 0 and "owner fuzz ok" in r.stdout, (r.stdout + r.stderr)[-3000:]
