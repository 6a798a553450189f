"""Plain C programs, with no Python or torch, use the library through the C
ABI: they allocate with HIP, run the token statistics on bf16 logits with a
ragged vocabulary, or the fused LM head (statistics at an inverse temperature
and the blocked backward), and check the results against the C oracle they
also link (the tolerances of the parity tests)."""

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


LMHEAD_PROGRAM = r'''
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dart.h"

/* the float64 C oracle (test infrastructure) */
void oracle_token_stats_ex(const void* z, int dtype, int64_t nrows, int64_t V, int64_t ld,
                           const int32_t* target, double inv_temp, double* logp, double* H,
                           double* lse, int nthreads);
void oracle_dlogits_ex(const void* z, int dtype, int64_t nrows, int64_t V, int64_t ld,
                       const int32_t* target, const double* lse, const double* logp,
                       const double* g, double inv_temp, double* out, int nthreads);

static uint64_t state = 777u;
static uint32_t next32(void) {
    state = state * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(state >> 32);
}
static double uniform(void) { return (double)(next32() >> 8) / 16777216.0 - 0.5; }
/* the top 16 bits of a float: an exact bf16 value */
static uint16_t bf16_bits(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}
static double widen(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

#define CK(x) do { if ((x) != hipSuccess) { printf("hip error line %d\n", __LINE__); return 2; } } while (0)

/* got [n, m] float32 against the exact product ref within (3 U + A) B, with
 * B the product of the absolute values; returns the largest error over B, or
 * a negative value when an element is out of tolerance */
static double check(const float* got, const double* ref, const double* bound, int64_t n) {
    const double U = 1.0 / 256.0, A = 1.0 / 8192.0;
    double worst = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const double err = fabs((double)got[i] - ref[i]);
        if (err > (3.0 * U + A) * bound[i] + 1e-30) return -1.0;
        if (bound[i] > 0.0) worst = fmax(worst, err / bound[i]);
    }
    return worst;
}

int main(void) {
    const int64_t T = 130, d = 64, V = 1000, R = 64, C = 384;
    const float inv_temp = 0.8f;
    uint16_t* h = malloc((size_t)(T * d) * 2);
    uint16_t* w = malloc((size_t)(V * d) * 2);
    int32_t* y = malloc((size_t)T * 4);
    float* g = malloc((size_t)T * 4);
    double* g64 = malloc((size_t)T * 8);
    for (int64_t i = 0; i < T * d; ++i) h[i] = bf16_bits((float)(2.0 * uniform()));
    for (int64_t i = 0; i < V * d; ++i) w[i] = bf16_bits((float)(0.8 * uniform()));
    for (int64_t t = 0; t < T; ++t) {
        y[t] = (int32_t)(next32() % (uint32_t)V);
        g[t] = t % 4 == 3 ? 0.0f : (float)(0.02 * uniform());
        g64[t] = (double)g[t];
    }
    /* the logits h W^T of the exact bf16 inputs, in float64 */
    double* z = malloc((size_t)(T * V) * 8);
    for (int64_t t = 0; t < T; ++t)
        for (int64_t v = 0; v < V; ++v) {
            double acc = 0.0;
            for (int64_t k = 0; k < d; ++k) acc += widen(h[t * d + k]) * widen(w[v * d + k]);
            z[t * V + v] = acc;
        }

    const size_t ws_stats = dart_lmhead_stats_workspace_bytes(T, V);
    const size_t ws_bwd = dart_lmhead_backward_ex_workspace_bytes(T, d, V, R, C, 0u);
    if (ws_stats == 0 || ws_bwd == 0) { printf("workspace size 0\n"); return 4; }
    const size_t ws_bytes = ws_stats > ws_bwd ? ws_stats : ws_bwd;
    void *dh, *dw, *dy, *dg, *dlogp, *dent, *dlse, *ddh, *ddw, *dws;
    CK(hipMalloc(&dh, (size_t)(T * d) * 2));
    CK(hipMalloc(&dw, (size_t)(V * d) * 2));
    CK(hipMalloc(&dy, (size_t)T * 4));
    CK(hipMalloc(&dg, (size_t)T * 4));
    CK(hipMalloc(&dlogp, (size_t)T * 4));
    CK(hipMalloc(&dent, (size_t)T * 4));
    CK(hipMalloc(&dlse, (size_t)T * 4));
    CK(hipMalloc(&ddh, (size_t)(T * d) * 4));
    CK(hipMalloc(&ddw, (size_t)(V * d) * 4));
    CK(hipMalloc(&dws, ws_bytes));
    CK(hipMemcpy(dh, h, (size_t)(T * d) * 2, hipMemcpyHostToDevice));
    CK(hipMemcpy(dw, w, (size_t)(V * d) * 2, hipMemcpyHostToDevice));
    CK(hipMemcpy(dy, y, (size_t)T * 4, hipMemcpyHostToDevice));
    CK(hipMemcpy(dg, g, (size_t)T * 4, hipMemcpyHostToDevice));

    dart_status_t st = dart_lmhead_tok_stats_ex(dh, T, d, d, dw, V, d, (const int32_t*)dy,
                                                inv_temp, (float*)dlogp, (float*)dent,
                                                (float*)dlse, dws, ws_stats, 0);
    if (st != DART_OK) { printf("dart_lmhead_tok_stats_ex: %s\n", dart_status_string(st)); return 3; }
    st = dart_lmhead_backward_ex(dh, T, d, d, dw, V, d, (const int32_t*)dy, (const float*)dlse,
                                 (const float*)dlogp, (const float*)dg, inv_temp, ddh, d, ddw, d,
                                 R, C, 0u, dws, ws_bwd, 0);
    if (st != DART_OK) { printf("dart_lmhead_backward_ex: %s\n", dart_status_string(st)); return 3; }
    CK(hipDeviceSynchronize());
    float* logp = malloc((size_t)T * 4);
    float* ent = malloc((size_t)T * 4);
    float* lse = malloc((size_t)T * 4);
    float* gh = malloc((size_t)(T * d) * 4);
    float* gw = malloc((size_t)(V * d) * 4);
    CK(hipMemcpy(logp, dlogp, (size_t)T * 4, hipMemcpyDeviceToHost));
    CK(hipMemcpy(ent, dent, (size_t)T * 4, hipMemcpyDeviceToHost));
    CK(hipMemcpy(lse, dlse, (size_t)T * 4, hipMemcpyDeviceToHost));
    CK(hipMemcpy(gh, ddh, (size_t)(T * d) * 4, hipMemcpyDeviceToHost));
    CK(hipMemcpy(gw, ddw, (size_t)(V * d) * 4, hipMemcpyDeviceToHost));

    double* rl = malloc((size_t)T * 8);
    double* rH = malloc((size_t)T * 8);
    double* rlse = malloc((size_t)T * 8);
    oracle_token_stats_ex(z, 2 /* float64 */, T, V, V, y, inv_temp, rl, rH, rlse, 1);
    double el = 0.0, eh = 0.0, es = 0.0;
    for (int64_t t = 0; t < T; ++t) {
        el = fmax(el, fabs((double)logp[t] - rl[t]));
        eh = fmax(eh, fabs((double)ent[t] - rH[t]));
        es = fmax(es, fabs((double)lse[t] - rlse[t]));
    }
    printf("max |logp - oracle| %.3e, |H - oracle| %.3e, |lse - oracle| %.3e\n", el, eh, es);
    if (!(el <= 2e-4 && eh <= 2e-4 && es <= 2e-4)) return 1;

    /* dh = dz W and dW = dz^T h from the oracle's dz, exactly, with the sums
     * of the absolute terms */
    double* dz = malloc((size_t)(T * V) * 8);
    oracle_dlogits_ex(z, 2, T, V, V, y, rlse, rl, g64, inv_temp, dz, 1);
    double* rh = calloc((size_t)(T * d), 8);
    double* bh = calloc((size_t)(T * d), 8);
    double* rw = calloc((size_t)(V * d), 8);
    double* bw = calloc((size_t)(V * d), 8);
    for (int64_t t = 0; t < T; ++t)
        for (int64_t v = 0; v < V; ++v) {
            const double q = dz[t * V + v];
            for (int64_t k = 0; k < d; ++k) {
                const double wv = widen(w[v * d + k]), hv = widen(h[t * d + k]);
                rh[t * d + k] += q * wv;
                bh[t * d + k] += fabs(q) * fabs(wv);
                rw[v * d + k] += q * hv;
                bw[v * d + k] += fabs(q) * fabs(hv);
            }
        }
    const double xh = check(gh, rh, bh, T * d), xw = check(gw, rw, bw, V * d);
    printf("dhidden %.3e, dweight %.3e (largest error over B; negative: out of tolerance)\n", xh, xw);
    return (xh >= 0.0 && xw >= 0.0) ? 0 : 1;
}
'''


def _build_and_run(tmp_path, source, name):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    pkg, ora = os.path.join(ROOT, "paper_2509_23866_amd"), os.path.join(ROOT, "oracle")
    for lib in (os.path.join(pkg, "libdart.so"), os.path.join(ora, "liboracle.so")):
        if not os.path.exists(lib):
            pytest.fail(f"{lib} is not built")
    src = tmp_path / f"{name}.c"
    src.write_text(source)
    exe = tmp_path / name
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


def test_c_program_token_stats_against_c_oracle(tmp_path):
    _build_and_run(tmp_path, PROGRAM, "consumer")


def test_c_program_lmhead_against_c_oracle(tmp_path):
    """The fused LM head from C at inverse temperature 0.8: statistics, then
    the backward in blocks of 64 rows x 384 entries (ragged in both), fp32
    gradients against the oracle's dz times the exact inputs within
    (3 U + A) B."""
    _build_and_run(tmp_path, LMHEAD_PROGRAM, "lmhead_consumer")
