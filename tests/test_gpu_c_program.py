"""A plain C program, with no Python or torch, uses the library through the C
ABI: it allocates with HIP, runs the token statistics on bf16 logits with a
ragged vocabulary, and checks them against the C oracle it also links (the
tolerances of the parity tests)."""

import os
import shutil
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = "/opt/rocm"

PROGRAM = r'''
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dart.h"

/* the float64 C oracle (test infrastructure) */
void oracle_token_stats(const void* z, int dtype, int64_t nrows, int64_t V, int64_t ld,
                        const int32_t* target, double* logp, double* H, double* lse,
                        int nthreads);

static uint64_t state = 12345u;
static uint32_t next32(void) {
    state = state * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(state >> 32);
}

#define CK(x) do { if ((x) != hipSuccess) { printf("hip error line %d\n", __LINE__); return 2; } } while (0)

int main(void) {
    const int64_t T = 257, V = 5003;
    uint16_t* z = malloc((size_t)T * V * 2);
    int32_t* y = malloc((size_t)T * 4);
    for (int64_t i = 0; i < T * V; ++i) {
        /* a float in [-6, 6), kept to its top 16 bits: an exact bf16 value */
        float f = ((float)(next32() >> 8) / 16777216.0f - 0.5f) * 12.0f;
        uint32_t u;
        memcpy(&u, &f, 4);
        z[i] = (uint16_t)(u >> 16);
    }
    for (int64_t t = 0; t < T; ++t) y[t] = (int32_t)(next32() % (uint32_t)V);

    void *dz, *dy, *dlogp, *dent, *dlse;
    CK(hipMalloc(&dz, (size_t)T * V * 2));
    CK(hipMalloc(&dy, (size_t)T * 4));
    CK(hipMalloc(&dlogp, (size_t)T * 4));
    CK(hipMalloc(&dent, (size_t)T * 4));
    CK(hipMalloc(&dlse, (size_t)T * 4));
    CK(hipMemcpy(dz, z, (size_t)T * V * 2, hipMemcpyHostToDevice));
    CK(hipMemcpy(dy, y, (size_t)T * 4, hipMemcpyHostToDevice));
    dart_status_t st = dart_tok_stats(dz, DART_BF16, T, V, V, (const int32_t*)dy, (float*)dlogp,
                                      (float*)dent, (float*)dlse, 0);
    if (st != DART_OK) { printf("dart_tok_stats: %s\n", dart_status_string(st)); return 3; }
    CK(hipDeviceSynchronize());
    float* logp = malloc((size_t)T * 4);
    float* ent = malloc((size_t)T * 4);
    CK(hipMemcpy(logp, dlogp, (size_t)T * 4, hipMemcpyDeviceToHost));
    CK(hipMemcpy(ent, dent, (size_t)T * 4, hipMemcpyDeviceToHost));

    double* rl = malloc((size_t)T * 8);
    double* rH = malloc((size_t)T * 8);
    double* rlse = malloc((size_t)T * 8);
    oracle_token_stats(z, 1 /* bf16 bit patterns */, T, V, V, y, rl, rH, rlse, 1);
    double el = 0.0, eh = 0.0;
    for (int64_t t = 0; t < T; ++t) {
        el = fmax(el, fabs((double)logp[t] - rl[t]));
        eh = fmax(eh, fabs((double)ent[t] - rH[t]));
    }
    printf("max |logp - oracle| %.3e, max |H - oracle| %.3e\n", el, eh);
    return (el <= 2e-4 && eh <= 2e-4) ? 0 : 1;
}
'''


def test_c_program_token_stats_against_c_oracle(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    pkg, ora = os.path.join(ROOT, "paper_2509_23866_amd"), os.path.join(ROOT, "oracle")
    for lib in (os.path.join(pkg, "libdart.so"), os.path.join(ora, "liboracle.so")):
        if not os.path.exists(lib):
            pytest.fail(f"{lib} is not built")
    src = tmp_path / "consumer.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "consumer"
    r = subprocess.run([gcc, "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror",
                        "-D__HIP_PLATFORM_AMD__", "-isystem", f"{ROCM}/include",
                        "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                        "-L", pkg, "-ldart", f"-Wl,-rpath,{pkg}", "-L", ora, "-loracle",
                        f"-Wl,-rpath,{ora}", "-L", f"{ROCM}/lib", "-lamdhip64",
                        f"-Wl,-rpath,{ROCM}/lib", "-lm"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    print(run.stdout, flush=True)
    assert run.returncode == 0, (run.returncode, run.stdout, run.stderr)
