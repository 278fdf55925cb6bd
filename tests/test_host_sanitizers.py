"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The oracle's C half (codecs, absmax initialisation, weight and activation fake quantisation,
  packing and decoding) is built with gcc -fsanitize=address,undefined and driven over special
  values (zeros, subnormals, infinities, NaNs, saturating magnitudes), every format, sub-block size
  and E8M0 rule, with and without the optional outputs.
* The C ABI's host side (argument checks, workspace sizing, the GEMM planners) is built with the
  sanitizers on the host pass only (the device code is compiled as usual and never launched) and
  driven through calls that each fail a host check, and through focus_workspace_size over many shapes.
Any sanitizer report fails the run (-fno-sanitize-recover=all).
"""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

import pytest

REPO = Path(__file__).resolve().parents[1]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]

ORACLE_DRIVER = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
void oracle_e2m1_array(const float *u, int64_t n, float *q, uint8_t *code);
void oracle_e2m1_decode_array(const uint8_t *code, int64_t n, float *v);
int oracle_e8m0_ceil_array(const float *s, int64_t n, uint8_t *byte);
int oracle_e8m0_floor_array(const float *s, int64_t n, uint8_t *byte);
int oracle_e4m3_array(const float *x, int64_t n, uint8_t *byte);
void oracle_e4m3_decode_array(const uint8_t *byte, int64_t n, float *v);
void oracle_bf16_round_array(const float *x, int64_t n, float *y);
int oracle_init_scales(int fmt, int sb, int e8m0_floor, const float *W, int64_t rows, int64_t K, float *s_fp,
                       float *c, float *alpha_out);
int oracle_fq_weight(int fmt, int sb, int ste_clip, int e8m0_floor, const float *W, int64_t rows, int64_t K,
                     const float *s_fp, const float *c, float alpha, float *w_hat, uint8_t *codes,
                     uint8_t *scale_bytes, float *u_out, uint8_t *m_out, float *sdq_out, float *sq_out);
int oracle_fq_act(int fmt, int e8m0_floor, const float *X, int64_t rows, int64_t K, float *x_hat, uint8_t *codes,
                  uint8_t *scale_bytes, float *alpha_out);
void oracle_pack_codes(const uint8_t *codes, int64_t rows, int64_t K, uint8_t *packed);
void oracle_unpack_codes(const uint8_t *packed, int64_t rows, int64_t K, uint8_t *codes);
void oracle_decode_packed(int fmt, const uint8_t *packed, const uint8_t *scale_bytes, float alpha, int64_t rows,
                          int64_t K, float *out);

static float f_of(uint32_t b) { float f; memcpy(&f, &b, 4); return f; }
static uint64_t st = 0x9E3779B97F4A7C15ULL;
static uint32_t rnd(void) { st ^= st << 13; st ^= st >> 7; st ^= st << 17; return (uint32_t)st; }

int main(void) {
    /* codecs over every bf16 pattern and random fp32 patterns */
    const int64_t n = 65536 + 65536;
    float *x = malloc(n * sizeof(float)), *y = malloc(n * sizeof(float));
    uint8_t *b = malloc(n);
    for (int64_t i = 0; i < 65536; i++) x[i] = f_of((uint32_t)i << 16);
    for (int64_t i = 65536; i < n; i++) x[i] = f_of(rnd());
    oracle_e2m1_array(x, n, y, b);
    oracle_e2m1_decode_array(b, n, y);
    oracle_e8m0_ceil_array(x, n, b);
    oracle_e8m0_floor_array(x, n, b);
    oracle_e4m3_array(x, n, b);
    for (int64_t i = 0; i < 256; i++) b[i] = (uint8_t)i;
    oracle_e4m3_decode_array(b, 256, y);
    oracle_bf16_round_array(x, n, y);
    /* fake quantisation of tensors holding specials */
    const int64_t rows = 9, K = 128;
    float *W = malloc(rows * K * sizeof(float)), *wh = malloc(rows * K * sizeof(float));
    float *u = malloc(rows * K * sizeof(float)), *s = malloc(rows * K * sizeof(float));
    float *c = malloc(rows * K * sizeof(float)), *sdq = malloc(rows * K * sizeof(float));
    float *sq = malloc(rows * K * sizeof(float)), alpha = 1.0f, dec[9 * 128];
    uint8_t *codes = malloc(rows * K), *m = malloc(rows * K), *sb = malloc(rows * K), *pk = malloc(rows * K / 2);
    for (int64_t i = 0; i < rows * K; i++) W[i] = (float)((int)(rnd() % 2001) - 1000) * 1e-3f;
    const uint32_t special[] = {0x00000000u, 0x80000000u, 0x00000001u, 0x7F800000u, 0xFF800000u, 0x7FC00000u,
                                0x7F7FFFFFu, 0x3E800000u, 0x40C00000u, 0x00800000u};
    for (int i = 0; i < 10; i++) W[i * 37] = f_of(special[i]);
    for (int j = 0; j < 32; j++) W[5 * K + j] = 0.0f; /* an all-zero block */
    const int sbs[] = {2, 4, 8, 16, 32};
    for (int fmt = 0; fmt < 2; fmt++)
        for (int fl = 0; fl < 2 - fmt; fl++)
            for (int k = 0; k < 5; k++) {
                const int sbk = sbs[k];
                if (fmt == 1 && sbk == 32) continue;
                oracle_init_scales(fmt, sbk, fl, W, rows, K, s, c, &alpha);
                for (int64_t i = 0; i < rows * K / sbk; i++) c[i] = 0.75f + (float)(rnd() % 1000) * 5e-4f;
                c[3] = 0.0f; /* a domain error */
                oracle_fq_weight(fmt, sbk, 1, fl, W, rows, K, s, c, alpha, wh, codes, sb, u, m, sdq, sq);
                oracle_fq_weight(fmt, sbk, 0, fl, W, rows, K, s, NULL, alpha, wh, NULL, NULL, NULL, NULL, NULL, NULL);
                oracle_fq_act(fmt, fl, W, rows, K, wh, codes, sb, &alpha);
                oracle_fq_act(fmt, fl, W, rows, K, NULL, NULL, NULL, NULL);
                oracle_pack_codes(codes, rows, K, pk);
                oracle_unpack_codes(pk, rows, K, codes);
                oracle_decode_packed(fmt, pk, sb, alpha, rows, K, dec);
            }
    free(x); free(y); free(b); free(W); free(wh); free(u); free(s); free(c); free(sdq); free(sq);
    free(codes); free(m); free(sb); free(pk);
    printf("oracle ok\n");
    return 0;
}
"""

ABI_DRIVER = r"""
#include "focus.h"
#include <cstdint>
#include <cstdio>

static int fails = 0;
static void expect(int got, int want, const char *what) {
    if (got != want) { std::printf("%s: got %d want %d\n", what, got, want); fails++; }
}

int main() {
    void *B = reinterpret_cast<void *>(uintptr_t(1) << 20);  // never dereferenced
    const uint8_t *B8 = static_cast<const uint8_t *>(B);
    focus_qconfig mx = {FOCUS_MXFP4, 8, 1, 0, 0}, nv = {FOCUS_NVFP4, 8, 1, 0, 0};
    focus_qconfig bad_fmt = {7, 8, 1, 0, 0}, bad_sb = {FOCUS_MXFP4, 3, 1, 0, 0}, nv32 = {FOCUS_NVFP4, 32, 1, 0, 0};
    focus_qconfig nv_floor = {FOCUS_NVFP4, 8, 1, 0, 1}, bad_layout = {FOCUS_MXFP4, 8, 1, 5, 0};
    // workspace sizing over many shapes (the planners' host arithmetic)
    for (int call = 0; call < 12; call++)
        for (int64_t M : {0LL, 1LL, 4LL, 255LL, 4096LL, 65536LL, 131072LL, 262144LL, 2147483647LL})
            for (int64_t N : {0LL, 8LL, 1024LL, 28672LL})
                for (int64_t K : {0LL, 32LL, 8192LL, 28672LL}) {
                    (void)focus_workspace_size(call, &mx, M, N, K);
                    (void)focus_workspace_size(call, &nv, M, N, K);
                    (void)focus_workspace_size(call, nullptr, M, N, K);
                }
    expect((int)(focus_workspace_size(FOCUS_CALL_RECON_GEMM_BWD, &nv32, 1, 1, 16) == 0), 1, "nv sb32 sizes to 0");
    for (int s = -1; s < 12; s++) (void)focus_status_string(s);
    // fake quantisation
    auto fq = [&](const focus_qconfig *q, int64_t rows, int64_t K, void *ws, size_t wsb) {
        return focus_fakequant_fwd(q, B, 1, rows, K, nullptr, nullptr, nullptr, B, 1, nullptr, nullptr, nullptr, ws,
                                   wsb, nullptr);
    };
    expect(fq(&bad_fmt, 4, 64, B, 1 << 20), FOCUS_ERR_CONFIG, "format");
    expect(fq(&bad_sb, 4, 64, B, 1 << 20), FOCUS_ERR_CONFIG, "sub-block");
    expect(fq(&nv32, 4, 64, B, 1 << 20), FOCUS_ERR_CONFIG, "nv sub-block 32");
    expect(fq(&nv_floor, 4, 64, B, 1 << 20), FOCUS_ERR_CONFIG, "nv floor");
    expect(fq(&bad_layout, 4, 64, B, 1 << 20), FOCUS_ERR_CONFIG, "layout");
    expect(fq(nullptr, 4, 64, B, 1 << 20), FOCUS_ERR_NULL, "null q");
    expect(fq(&mx, 4, 48, B, 1 << 20), FOCUS_ERR_SHAPE, "K % 32");
    expect(fq(&mx, -1, 64, B, 1 << 20), FOCUS_ERR_SHAPE, "negative rows");
    expect(fq(&mx, int64_t(1) << 40, 1 << 20, B, 1 << 20), FOCUS_ERR_SHAPE, "too many elements");
    expect(fq(&mx, 4, 64, nullptr, 1 << 20), FOCUS_ERR_WORKSPACE, "null workspace");
    expect(fq(&mx, 4, 64, B, 16), FOCUS_ERR_WORKSPACE, "small workspace");
    expect(fq(&mx, 4, 64, reinterpret_cast<void *>((uintptr_t(1) << 20) + 8), 1 << 20), FOCUS_ERR_WORKSPACE,
           "misaligned workspace");
    expect(focus_fakequant_fwd(&mx, B, 9, 4, 64, nullptr, nullptr, nullptr, B, 1, nullptr, nullptr, nullptr, B,
                               1 << 20, nullptr), FOCUS_ERR_DTYPE, "dtype");
    expect(focus_fakequant_fwd(&mx, B, 1, 4, 64, nullptr, nullptr, nullptr, nullptr, 1, nullptr, nullptr, nullptr,
                               B, 1 << 20, nullptr), FOCUS_ERR_NULL, "no output");
    expect(focus_scales_init(&nv, B, 1, 4, 64, static_cast<float *>(B), static_cast<float *>(B), nullptr, B,
                             1 << 20, nullptr), FOCUS_ERR_NULL, "nv init needs alpha");
    expect(focus_export_packed(&mx, B, 1, 4, 64, static_cast<float *>(B), nullptr, nullptr, nullptr,
                               static_cast<uint8_t *>(B), B, 1 << 20, nullptr), FOCUS_ERR_NULL, "export codes");
    // reconstruction GEMMs
    expect(focus_recon_gemm_fwd(B, B, 1, 8, 8, 24, nullptr, B, nullptr, nullptr, B, 1 << 30, nullptr),
           FOCUS_ERR_SHAPE, "fwd K % 16");
    expect(focus_recon_gemm_fwd(B, B, 1, 8, 8, 32, B, B, nullptr, nullptr, B, 1 << 30, nullptr), FOCUS_ERR_NULL,
           "fwd loss");
    expect(focus_recon_gemm_fwd(B, B, 3, 8, 8, 32, nullptr, B, nullptr, nullptr, B, 1 << 30, nullptr),
           FOCUS_ERR_DTYPE, "fwd dtype");
    expect(focus_recon_gemm_fwd_mxfp4(B8, B8, B8, B8, 8, 8, 64, nullptr, B, nullptr, nullptr, B, 1 << 30, nullptr),
           FOCUS_ERR_SHAPE, "mx fwd K % 128");
    expect(focus_recon_gemm_fwd_mxfp4(B8, B8, B8, B8, 8, 8, 128, nullptr, B, nullptr, nullptr, B, 16, nullptr),
           FOCUS_ERR_WORKSPACE, "mx fwd workspace");
    expect(focus_recon_gemm_fwd_mxfp4_noalloc(B8, B8, B8, B8, 65536, 28672, 8192, B, B, static_cast<double *>(B),
                                              nullptr, nullptr), FOCUS_ERR_SCRATCH, "noalloc scratch");
    expect(focus_recon_gemm_bwd(&mx, B, B, 1, 64, 4, 64, B, 1, static_cast<float *>(B), nullptr, nullptr,
                                static_cast<float *>(B), static_cast<float *>(B), nullptr, B, 16, nullptr),
           FOCUS_ERR_WORKSPACE, "bwd workspace");
    expect(focus_recon_gemm_bwd(&nv, B, B, 1, 64, 4, 64, B, 1, static_cast<float *>(B), nullptr, nullptr,
                                static_cast<float *>(B), static_cast<float *>(B), nullptr, B, 1 << 30, nullptr),
           FOCUS_ERR_NULL, "bwd nv alpha");
    expect(focus_recon_gemm_bwd_mxfp4(&nv, B, B8, B8, 8, 8, 64, B, 1, static_cast<float *>(B), nullptr,
                                      static_cast<float *>(B), static_cast<float *>(B), B, 1 << 30, nullptr),
           FOCUS_ERR_CONFIG, "bwd mx nv");
    expect(focus_recon_gemm_bwd_mxfp4(&mx, B, B8, B8, 6, 8, 64, B, 1, static_cast<float *>(B), nullptr,
                                      static_cast<float *>(B), static_cast<float *>(B), B, 1 << 30, nullptr),
           FOCUS_ERR_SHAPE, "bwd mx M % 4");
    expect(focus_recon_gemm_dx(B, B, 1, 8, 12, 32, B, B, 1 << 30, nullptr), FOCUS_ERR_SHAPE, "dx N % 16");
    expect(focus_kl_top(B, B, 1, 4, 16, 0, B, static_cast<double *>(B), B, 1 << 20, nullptr), FOCUS_ERR_CONFIG,
           "kl k");
    focus_adamw_config ok = {1e-2f, 0.9f, 0.999f, 1e-8f, 0.0f, 1}, bad = {1e-2f, 1.0f, 0.999f, 1e-8f, 0.0f, 0};
    float *P = static_cast<float *>(B);
    expect(focus_adamw_step(&ok, 0, 16, P, P, P, P, B, 256, nullptr), FOCUS_ERR_CONFIG, "adamw t");
    expect(focus_adamw_step(&bad, 1, 16, P, P, P, P, B, 256, nullptr), FOCUS_ERR_CONFIG, "adamw beta");
    expect(focus_adamw_step(&ok, 1, -1, P, P, P, P, B, 256, nullptr), FOCUS_ERR_SHAPE, "adamw n");
    expect(focus_check_flags(nullptr, nullptr), FOCUS_ERR_WORKSPACE, "flags");
    // grouped weight fake quantisation: the host copies the layer table; every layer is checked
    focus_weight_layer lay[FOCUS_MAX_WEIGHT_LAYERS + 1];
    for (int i = 0; i <= FOCUS_MAX_WEIGHT_LAYERS; i++)
        lay[i] = focus_weight_layer{B, 4, 64, P, nullptr, nullptr, nullptr, static_cast<uint8_t *>(B), static_cast<uint8_t *>(B)};
    expect(focus_fakequant_weights(&mx, 1, 1, lay, FOCUS_MAX_WEIGHT_LAYERS + 1, B, 256, nullptr), FOCUS_ERR_SHAPE,
           "group too many layers");
    expect(focus_fakequant_weights(&mx, 1, 1, nullptr, 2, B, 256, nullptr), FOCUS_ERR_NULL, "group table");
    lay[FOCUS_MAX_WEIGHT_LAYERS - 1].K = 48;
    expect(focus_fakequant_weights(&mx, 1, 1, lay, FOCUS_MAX_WEIGHT_LAYERS, B, 256, nullptr), FOCUS_ERR_SHAPE,
           "group last layer K");
    lay[FOCUS_MAX_WEIGHT_LAYERS - 1].K = 64;
    expect(focus_fakequant_weights(&nv, 1, 1, lay, 3, B, 256, nullptr), FOCUS_ERR_NULL, "group nv alpha");
    expect(focus_fakequant_weights(&mx, 1, 1, lay, 3, B, 16, nullptr), FOCUS_ERR_WORKSPACE, "group ws");
    expect(focus_fakequant_weights(&mx, 1, 1, lay, 0, B, 256, nullptr), FOCUS_OK, "group empty");
    std::printf("abi %s (%d failures)\n", fails ? "FAILED" : "ok", fails);
    return fails != 0;
}
"""


def test_oracle_under_sanitizers(tmp_path):
    drv = tmp_path / "oracle_driver.c"
    drv.write_text(ORACLE_DRIVER)
    exe = tmp_path / "oracle_san"
    cmd = ["gcc", "-O1", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", *SAN,
           str(REPO / "oracle" / "focus_oracle.c"), str(drv), "-o", str(exe), "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, OMP_NUM_THREADS="2", ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert out.returncode == 0 and "oracle ok" in out.stdout, (out.stdout + out.stderr)[-4000:]


def test_abi_host_checks_under_sanitizers(tmp_path):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    if not Path(hipcc).exists():
        pytest.skip("hipcc is not available")
    host_san = [f for s in SAN for f in ("-Xarch_host", s)]
    common = ["--offload-arch=gfx950", "-O1", "-std=c++17", "-fPIC", "-ffp-contract=off",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *host_san, "-I", str(REPO / "include")]
    srcs = sorted((REPO / "paper_2608_01847_amd" / "csrc").glob("*.hip"))
    drv = tmp_path / "abi_driver.cpp"
    drv.write_text(ABI_DRIVER)

    def compile_one(src):
        obj = tmp_path / (src.stem + ".o")
        r = subprocess.run([hipcc, *common, "-c", str(src), "-o", str(obj)], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        return obj

    with ThreadPoolExecutor(max_workers=min(8, len(srcs) + 1)) as ex:
        objs = list(ex.map(compile_one, [*srcs, drv]))
    exe = tmp_path / "abi_san"
    r = subprocess.run([hipcc, "--offload-arch=gfx950", *host_san, *map(str, objs), "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert out.returncode == 0 and "abi ok" in out.stdout, (out.stdout + out.stderr)[-4000:]
    shutil.rmtree(tmp_path, ignore_errors=True)
