/* A plain C11 caller of the Jorge C ABI (include/jorge.h) and the HIP runtime:
 * no Python, no PyTorch. It creates a context over the layers named on the
 * command line, takes a number of Jorge steps on seeded inputs on the null
 * stream, and writes every layer's parameters and state to a file, so a test
 * can compare them with the same steps taken through the Python binding.
 *
 * Usage: jorge_c_driver OUT SEED STEPS m1 n1 [m2 n2 ...]
 *
 * Inputs: element i of layer l's initial parameters is u(SEED, 0, l, i) and
 * of its gradient at step t (1-based) 1e-2 * u(SEED, t, l, i), where
 * u(s, t, l, i) = (int)(z >> 40) / 2^23 - 1, in [-1, 1) and exact in fp32,
 * z = splitmix64(splitmix64(s * 2^32 + t * 2^16 + l) + i) (splitmix64 as
 * published by Steele, Lea and Flood, 2014). Hyperparameters: lr 0.1,
 * beta2 0.9, beta1 0.9, weight decay 5e-4; every other option at its
 * default.
 *
 * Output, per layer in order, raw little-endian float32, row-major: theta
 * (m x n), L_hat (m x m), R_hat (n x n), m (m x n), m_SGD (m x n). Stdout:
 * the step counter and the non-finite flag count. Exit status 0 on success;
 * on any failed call, 1 with the call and its message on stderr. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "jorge.h"

static uint64_t splitmix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

static void fill(float* out, size_t count, uint64_t seed, uint64_t t, uint64_t layer, float scale) {
    const uint64_t base = splitmix64((seed << 32) + (t << 16) + layer);
    for (size_t i = 0; i < count; ++i) {
        const int32_t q = (int32_t)(splitmix64(base + i) >> 40);  /* 24 bits */
        out[i] = scale * ((float)q / 8388608.0f - 1.0f);
    }
}

static jorge_ctx* g_ctx = NULL;

static void die(const char* what, const char* detail) {
    fprintf(stderr, "jorge_c_driver: %s failed: %s\n", what, detail ? detail : "");
    if (g_ctx) jorge_destroy(g_ctx);
    exit(1);
}

#define HIP_CHECK(call)                                                \
    do {                                                               \
        hipError_t e_ = (call);                                        \
        if (e_ != hipSuccess) die(#call, hipGetErrorString(e_));       \
    } while (0)

#define JORGE_CHECK(call)                                                           \
    do {                                                                            \
        jorge_status s_ = (call);                                                   \
        if (s_ != JORGE_OK) {                                                       \
            char m_[512];                                                           \
            snprintf(m_, sizeof m_, "%s (%s)", jorge_status_string(s_), jorge_last_error(g_ctx)); \
            die(#call, m_);                                                         \
        }                                                                           \
    } while (0)

int main(int argc, char** argv) {
    if (argc < 6 || (argc - 4) % 2 != 0) {
        fprintf(stderr, "usage: %s OUT SEED STEPS m1 n1 [m2 n2 ...]\n", argv[0]);
        return 2;
    }
    const char* out_path = argv[1];
    const uint64_t seed = strtoull(argv[2], NULL, 10);
    const int steps = atoi(argv[3]);
    const int nl = (argc - 4) / 2;
    jorge_shape* shapes = calloc((size_t)nl, sizeof *shapes);
    float** params = calloc((size_t)nl, sizeof *params);
    float** grads = calloc((size_t)nl, sizeof *grads);
    size_t max_elems = 0;
    if (!shapes || !params || !grads) die("calloc", "out of host memory");
    for (int l = 0; l < nl; ++l) {
        shapes[l].rows = atoll(argv[4 + 2 * l]);
        shapes[l].cols = atoll(argv[5 + 2 * l]);
        if (shapes[l].rows <= 0 || shapes[l].cols <= 0) die("argument parsing", "layer sizes must be positive");
        const size_t e = (size_t)(shapes[l].rows * shapes[l].cols);
        const size_t f = (size_t)(shapes[l].rows > shapes[l].cols ? shapes[l].rows : shapes[l].cols);
        if (e > max_elems) max_elems = e;
        if (f * f > max_elems) max_elems = f * f;
    }
    float* host = malloc(max_elems * sizeof(float));
    float* dev_state = NULL;
    if (!host) die("malloc", "out of host memory");

    /* Device buffers owned by the caller: parameters and gradients. */
    for (int l = 0; l < nl; ++l) {
        const size_t e = (size_t)(shapes[l].rows * shapes[l].cols);
        HIP_CHECK(hipMalloc((void**)&params[l], e * sizeof(float)));
        HIP_CHECK(hipMalloc((void**)&grads[l], e * sizeof(float)));
        fill(host, e, seed, 0, (uint64_t)l, 1.0f);
        HIP_CHECK(hipMemcpy(params[l], host, e * sizeof(float), hipMemcpyHostToDevice));
    }
    HIP_CHECK(hipMalloc((void**)&dev_state, max_elems * sizeof(float)));

    JORGE_CHECK(jorge_create(shapes, nl, NULL, NULL, &g_ctx));
    for (int t = 1; t <= steps; ++t) {
        for (int l = 0; l < nl; ++l) {
            const size_t e = (size_t)(shapes[l].rows * shapes[l].cols);
            fill(host, e, seed, (uint64_t)t, (uint64_t)l, 1e-2f);
            /* Synchronous copy: the previous step has read this buffer by the time it returns. */
            HIP_CHECK(hipMemcpy(grads[l], host, e * sizeof(float), hipMemcpyHostToDevice));
        }
        JORGE_CHECK(jorge_step(g_ctx, params, (const float* const*)grads, 0.1, 0.9, 0.9, 5e-4));
    }
    JORGE_CHECK(jorge_synchronize(g_ctx));

    FILE* f = fopen(out_path, "wb");
    if (!f) die("fopen", out_path);
    for (int l = 0; l < nl; ++l) {
        const int64_t m = shapes[l].rows, n = shapes[l].cols;
        const int32_t kinds[4] = {JORGE_STATE_L, JORGE_STATE_R, JORGE_STATE_MOM, JORGE_STATE_MOM_SGD};
        const int64_t rows[4] = {m, n, m, m}, cols[4] = {m, n, n, n};
        HIP_CHECK(hipMemcpy(host, params[l], (size_t)(m * n) * sizeof(float), hipMemcpyDeviceToHost));
        if (fwrite(host, sizeof(float), (size_t)(m * n), f) != (size_t)(m * n)) die("fwrite", out_path);
        for (int k = 0; k < 4; ++k) {
            const size_t e = (size_t)(rows[k] * cols[k]);
            JORGE_CHECK(jorge_get_state(g_ctx, l, kinds[k], dev_state, cols[k]));
            JORGE_CHECK(jorge_synchronize(g_ctx));
            HIP_CHECK(hipMemcpy(host, dev_state, e * sizeof(float), hipMemcpyDeviceToHost));
            if (fwrite(host, sizeof(float), e, f) != e) die("fwrite", out_path);
        }
    }
    if (fclose(f) != 0) die("fclose", out_path);

    int64_t t_now = 0;
    int32_t bad = 0, first = -1;
    JORGE_CHECK(jorge_get_step(g_ctx, &t_now));
    JORGE_CHECK(jorge_nonfinite(g_ctx, &bad, &first));
    printf("steps %lld nonfinite %d\n", (long long)t_now, (int)bad);

    jorge_destroy(g_ctx);
    g_ctx = NULL;
    for (int l = 0; l < nl; ++l) {
        HIP_CHECK(hipFree(params[l]));
        HIP_CHECK(hipFree(grads[l]));
    }
    HIP_CHECK(hipFree(dev_state));
    free(host);
    free(grads);
    free(params);
    free(shapes);
    return 0;
}
