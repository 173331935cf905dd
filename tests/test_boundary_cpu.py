"""The C boundary helper (paper_2608_14575_amd/csrc/c_boundary.hpp): every
exported function of the library runs its body through it, so a host
exception becomes a status instead of unwinding into a C caller.  Built with
g++ from the header alone (no device, no HIP): a failed allocation, a thread
that cannot start and a non-standard throw each give HWR_ERR_OOM with the
message recorded; a normal return passes through; a note that itself throws
is contained."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PROGRAM = r'''
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <system_error>

#include "c_boundary.hpp"

static std::string noted;
static int check(bool ok, const char *what) {
    if (!ok) std::printf("FAIL %s\n", what);
    return ok ? 0 : 1;
}
int main() {
    auto note = [](const char *m) { noted = m; };
    int bad = 0;
    bad += check(hwr::c_boundary([] { return HWR_ERR_STATE; }, note) == HWR_ERR_STATE, "pass-through");
    bad += check(noted.empty(), "no note on a normal return");
    bad += check(hwr::c_boundary([]() -> hwr_status { throw std::bad_alloc(); }, note) == HWR_ERR_OOM, "bad_alloc");
    bad += check(!noted.empty(), "bad_alloc noted");
    noted.clear();
    bad += check(hwr::c_boundary([]() -> hwr_status {
                     throw std::system_error(std::make_error_code(std::errc::resource_unavailable_try_again),
                                             "thread");
                 }, note) == HWR_ERR_OOM, "system_error");
    bad += check(noted.find("thread") != std::string::npos, "system_error message");
    bad += check(hwr::c_boundary([]() -> hwr_status { throw 7; }, note) == HWR_ERR_OOM, "non-standard throw");
    bad += check(noted == "unknown host exception", "non-standard note");
    bad += check(hwr::c_boundary([]() -> hwr_status { throw std::bad_alloc(); },
                                 [](const char *) { throw std::bad_alloc(); }) == HWR_ERR_OOM, "throwing note");
    std::printf(bad ? "failures: %d\n" : "ok\n", bad);
    return bad;
}
'''


def test_c_boundary_turns_exceptions_into_status(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    src = tmp_path / "boundary.cpp"
    src.write_text(PROGRAM)
    exe = tmp_path / "boundary"
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", "-I",
                    os.path.join(ROOT, "paper_2608_14575_amd", "csrc"), "-I", os.path.join(ROOT, "include"),
                    str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.strip() == "ok", out.stdout
