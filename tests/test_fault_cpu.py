"""Failure injection on the CPU: a forced host-allocation failure returns
BOOST_ENOMEM and leaves nothing allocated (plan-only contexts)."""
import glob
import os
import subprocess

import pytest

from paper_2609_13592_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_13592_amd")
SAN_LIB = os.path.join(PKG, "_lib_sanitize", "libboostcap.so")
CLANG = "/opt/rocm/llvm/bin/clang"


def test_forced_host_alloc_failure_plan_only(monkeypatch):
    ctx = bd.boost_init(-1)
    try:
        monkeypatch.setenv("BOOST_FAULT_HOST_ALLOC", "1")
        with pytest.raises(bd.BoostError) as e:
            bd.boost_kv_pool_create(ctx, 2, 8, 128, 4096, 12, q_heads=32)
        assert e.value.code == bd.ENOMEM
        monkeypatch.setenv("BOOST_FAULT_HOST_ALLOC", "0")     # 0: no fault
        pool = bd.boost_kv_pool_create(ctx, 2, 8, 128, 4096, 12, q_heads=32)
        bd.boost_kv_pool_destroy(pool)
        monkeypatch.delenv("BOOST_FAULT_HOST_ALLOC")
        pool = bd.boost_kv_pool_create(ctx, 2, 8, 128, 4096, 12, q_heads=32)
        assert bd.boost_kv_alloc(pool, 1, 3) != bd.EAGAIN
        bd.boost_kv_pool_destroy(pool)
    finally:
        bd.boost_shutdown(ctx)


def _sanitize_build_current():
    if not os.path.exists(SAN_LIB):
        return False
    built = os.path.getmtime(SAN_LIB)
    srcs = glob.glob(os.path.join(PKG, "csrc", "*")) + glob.glob(os.path.join(ROOT, "include", "*.h"))
    return all(os.path.getmtime(s) <= built for s in srcs)


@pytest.mark.skipif(not os.path.exists(CLANG) or not _sanitize_build_current(),
                    reason="needs the current host-sanitizer build "
                           "(python -m paper_2609_13592_amd.build --sanitize)")
def test_forced_failure_releases_everything_under_asan(tmp_path):
    """The failing calls leak nothing: a C program linked against the
    AddressSanitizer build runs them with leak checking on."""
    exe = str(tmp_path / "fault_host_alloc")
    src = os.path.join(ROOT, "tests", "native", "fault_host_alloc.c")
    lib_dir = os.path.dirname(SAN_LIB)
    subprocess.run([CLANG, "-fsanitize=address", "-g", f"-I{ROOT}/include", src, "-o", exe,
                    f"-L{lib_dir}", "-lboostcap", "-lubsan", f"-Wl,-rpath,{lib_dir}"],
                   check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1")
    env.pop("BOOST_FAULT_HOST_ALLOC", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "fault-injection ok" in r.stdout
    assert "LeakSanitizer" not in r.stderr
