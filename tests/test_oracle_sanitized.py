"""The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

A small driver is compiled with the oracle's source, with
``-fsanitize=address,undefined`` and without OpenMP (so the sanitizers see one
thread).  It runs every entry point on ragged shapes: attention rows, pack and
unpack for every element size, and the backward.  It also checks a few results
against values it can derive by itself: pack then unpack restores the input,
a single key gives O = V, and dv sums to the summed output gradient.  Any
out-of-bounds access or undefined operation aborts the process with a report.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

DRIVER = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_attention_rows(const double *, const double *, const double *, int64_t, int64_t, double,
                          const int64_t *, int64_t, double *);
int oracle_pack(const void *, void *, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t);
int oracle_unpack(const void *, void *, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t);
int oracle_attention_backward(const double *, const double *, const double *, const double *,
                              int64_t, int64_t, double, const int64_t *, int64_t, const int64_t *,
                              int64_t, double *, double *, double *);

static double rnd(unsigned *s) { *s = *s * 1103515245u + 12345u; return ((*s >> 8) & 0xffff) / 32768.0 - 1.0; }

int main(void) {
    unsigned seed = 7;
    /* attention rows on ragged shapes, every row */
    for (int64_t S = 1; S <= 37; S += 9)
        for (int64_t d = 1; d <= 9; d += 4) {
            double *q = malloc(sizeof(double) * S * d), *k = malloc(sizeof(double) * S * d);
            double *v = malloc(sizeof(double) * S * d), *o = malloc(sizeof(double) * S * d);
            int64_t *rows = malloc(sizeof(int64_t) * S);
            for (int64_t i = 0; i < S * d; ++i) { q[i] = rnd(&seed); k[i] = rnd(&seed); v[i] = rnd(&seed); }
            for (int64_t i = 0; i < S; ++i) rows[i] = i;
            if (oracle_attention_rows(q, k, v, S, d, 0.3, rows, S, o)) return 1;
            if (S == 1)
                for (int64_t t = 0; t < d; ++t) if (fabs(o[t] - v[t]) > 1e-15) return 2;
            double *g = malloc(sizeof(double) * S * d), *dq = malloc(sizeof(double) * S * d);
            double *dk = malloc(sizeof(double) * S * d), *dv = malloc(sizeof(double) * S * d);
            for (int64_t i = 0; i < S * d; ++i) g[i] = rnd(&seed);
            if (oracle_attention_backward(q, k, v, g, S, d, 0.3, rows, S, rows, S, dq, dk, dv)) return 3;
            for (int64_t t = 0; t < d; ++t) {          /* sum_j dv_j = sum_i g_i */
                double a = 0, b = 0;
                for (int64_t j = 0; j < S; ++j) { a += dv[j * d + t]; b += g[j * d + t]; }
                if (fabs(a - b) > 1e-10) return 4;
            }
            free(q); free(k); free(v); free(o); free(rows); free(g); free(dq); free(dk); free(dv);
        }
    /* pack / unpack roundtrip for every element size and head range */
    const int64_t P = 3, S = 12, H = 5, d = 3;
    for (int64_t es = 1; es <= 8; es *= 2)
        for (int64_t h0 = 0; h0 < H; ++h0)
            for (int64_t hc = 1; h0 + hc <= H; ++hc) {
                unsigned char *src = malloc(S * H * d * es), *hm = malloc(S * hc * d * es);
                unsigned char *back = malloc(S * H * d * es);
                for (int64_t i = 0; i < S * H * d * es; ++i) { src[i] = (unsigned char)(i * 31 + 7); back[i] = src[i]; }
                if (oracle_pack(src, hm, P, S, H, d, h0, hc, es)) return 5;
                memset(back, 0, S * H * d * es);
                if (oracle_unpack(hm, back, P, S, H, d, h0, hc, es)) return 6;
                for (int64_t t = 0; t < S; ++t)
                    for (int64_t h = h0; h < h0 + hc; ++h)
                        if (memcmp(back + (t * H + h) * d * es, src + (t * H + h) * d * es, d * es)) return 7;
                free(src); free(hm); free(back);
            }
    /* rejected shapes return an error instead of touching memory */
    if (oracle_pack(NULL, NULL, 5, 12, 5, 3, 0, 1, 2) != -1) return 8;
    if (oracle_unpack(NULL, NULL, 3, 12, 5, 3, 4, 2, 2) != -1) return 9;
    puts("sanitized oracle ok");
    return 0;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_address_and_undefined_sanitizers(tmp_path):
    drv = tmp_path / "driver.c"
    drv.write_text(DRIVER)
    exe = tmp_path / "driver"
    src = os.path.join(ROOT, "oracle", "hcms_oracle.c")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-Wno-unknown-pragmas", str(drv), src, "-lm", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, f"exit {r.returncode}\n{r.stdout[-1000:]}\n{r.stderr[-3000:]}"
    assert "sanitized oracle ok" in r.stdout
