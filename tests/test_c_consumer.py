"""The boundary is a C ABI: include/dart.h compiles as C11 (and C++17) with
warnings as errors, and a C program linked against libdart.so takes the
address of every function the header declares (the link fails if one is not
exported) and calls the host-only helpers and a host-side argument check from
C. No GPU work: every call made here returns before any launch."""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dart.h")
LIBDIR = os.path.join(ROOT, "paper_2509_23866_amd")
ROCM = "/opt/rocm"


def declared_functions():
    with open(HEADER) as fh:
        text = fh.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dart_\w+)\s*\(", text)))


PROGRAM = r'''
#include <stdio.h>
#include <string.h>
#include "dart.h"

int main(void) {
    void* const fns[] = { %(fns)s };
    size_t n = 0;
    for (size_t i = 0; i < sizeof fns / sizeof fns[0]; ++i) n += fns[i] != NULL;
    if (n != %(nfns)d) return 10;
    if (dart_kept_steps(240, 0.8) != 192) return 11;
    if (dart_kept_steps(10, 1.5) != -1) return 12;
    if (strcmp(dart_status_string(DART_ERR_INVALID_ARG), "DART_ERR_INVALID_ARG") != 0) return 13;
    if (dart_lmhead_backward_workspace_bytes(2, 300) != 2u * 304u * 2u) return 14;
    if (dart_lmhead_backward_ex_workspace_bytes(2, 16, 300, 2, 300, 0) != 2u * 304u * 2u) return 15;
    if (dart_lmhead_backward_ex_workspace_bytes(2, 16, 300, 2, 300, 8u) != 0) return 16;
    /* a null logits pointer is rejected on the host, before anything is enqueued */
    if (dart_tok_stats(NULL, DART_BF16, 4, 8, 8, NULL, NULL, NULL, NULL, 0) != DART_ERR_INVALID_ARG)
        return 17;
    printf("ok %%zu\n", n);
    return 0;
}
'''


def _compiler(name):
    path = shutil.which(name)
    if path is None:
        pytest.skip(f"{name} not available")
    return path


def test_header_compiles_as_c_and_cpp(tmp_path):
    src = tmp_path / "h.c"
    src.write_text('#include "dart.h"\nint main(void) { return (int)DART_OK; }\n')
    for cc, std, lang in ((_compiler("gcc"), "-std=c11", "c"), (_compiler("g++"), "-std=c++17", "c++")):
        r = subprocess.run([cc, std, "-x", lang, "-Wall", "-Wextra", "-Werror",
                            "-D__HIP_PLATFORM_AMD__", "-isystem", f"{ROCM}/include",
                            "-I", os.path.join(ROOT, "include"), "-fsyntax-only", str(src)],
                           capture_output=True, text=True, timeout=120)
        assert r.returncode == 0, r.stderr


def test_c_program_links_every_declared_function(tmp_path):
    if not os.path.exists(os.path.join(LIBDIR, "libdart.so")):
        pytest.skip("libdart.so is not built")
    fns = declared_functions()
    assert len(fns) >= 20 and "dart_lmhead_backward_ex" in fns
    src = tmp_path / "consumer.c"
    src.write_text(PROGRAM % {"fns": ", ".join(f"(void*){f}" for f in fns), "nfns": len(fns)})
    exe = tmp_path / "consumer"
    r = subprocess.run([_compiler("gcc"), "-std=c11", "-Wall", "-Wextra", "-Werror",
                        "-Wno-pedantic", "-D__HIP_PLATFORM_AMD__", "-isystem", f"{ROCM}/include",
                        "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                        "-L", LIBDIR, "-ldart", f"-Wl,-rpath,{LIBDIR}", "-L", f"{ROCM}/lib",
                        "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120,
                         env=dict(os.environ, HIP_VISIBLE_DEVICES=""))
    assert run.returncode == 0, (run.returncode, run.stdout, run.stderr)
    assert run.stdout.strip() == f"ok {len(fns)}"
