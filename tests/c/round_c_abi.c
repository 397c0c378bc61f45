/*
 * A plain C11 consumer of libdedloc: include/dedloc.h and the HIP runtime's C
 * API only (no Python, no torch).  Test infrastructure: it also links the CPU
 * oracle and checks the library against it on the same seeded inputs.
 *
 *   round_c_abi --host   host-only entry points and argument validation
 *                        (no device is touched)
 *   round_c_abi          the above, then whole fp16 and int8 rounds on
 *                        device 0, each with and without the local peer's
 *                        fp32 gradient; exits 77 when no device is present
 *
 * Bars as in the Python parity tests: bounds, weights, codes, scales, the
 * fp32 average and m', v' identical; x' within 1e-5 of max|x|; trust ratios
 * within 1e-6 relative.  Exit status 0 = pass, 1 = mismatch, 77 = skipped.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dedloc.h"

/* The oracle's entry points (oracle/dedloc_oracle.c). */
typedef struct {
    float lr, beta1, beta2, eps, weight_decay;
    uint64_t step;
    int32_t bias_correction;
    int32_t force_unit_trust;
} oracle_lamb_cfg;
int oracle_partition(uint64_t P, uint32_t n, const uint64_t *beta, uint32_t align, uint64_t *bounds);
int oracle_weights(const uint32_t *counts, uint32_t n, float *w);
void oracle_encode_fp16(const float *x, size_t n, uint16_t *codes);
void oracle_encode_i8(const float *x, size_t n, uint32_t block, int8_t *codes, float *scales);
int oracle_round(const void *const *peer_codes, const float *const *peer_scales, const uint32_t *counts,
                 uint32_t n_peers, const uint64_t *bounds, uint32_t n_shards, int codec, uint32_t block,
                 void *out_codes, float *out_scales, float *x, float *m, float *v, uint64_t P,
                 const uint64_t *off, const uint8_t *flags, uint32_t T, const oracle_lamb_cfg *cfg,
                 float *trust, float *out_mean, float *scratch);

static int failures = 0;

#define CHECK(cond, ...)                                    \
    do {                                                    \
        if (!(cond)) {                                      \
            fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            fprintf(stderr, __VA_ARGS__);                   \
            fprintf(stderr, "\n");                          \
            failures++;                                     \
        }                                                   \
    } while (0)

#define HIP(call)                                                              \
    do {                                                                       \
        hipError_t e_ = (call);                                                \
        if (e_ != hipSuccess) {                                                \
            fprintf(stderr, "HIP error %s at %s:%d\n", hipGetErrorString(e_), __FILE__, __LINE__); \
            exit(1);                                                           \
        }                                                                      \
    } while (0)

/* xorshift64*: the seeded input generator (no part of the method). */
static uint64_t rng_state;
static double uniform(void) {
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (double)((rng_state * 2685821657736338717ull) >> 11) * 0x1p-53;
}
static float gauss(float sigma) {  /* Box-Muller */
    double u1 = uniform(), u2 = uniform();
    if (u1 < 1e-300) u1 = 1e-300;
    return (float)(sigma * sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2));
}

static int same_bits(const void *a, const void *b, size_t bytes) { return memcmp(a, b, bytes) == 0; }

/* ------------------------------------------------------------------ host */

static void host_checks(void) {
    /* shard bounds and weights: integer-exact, identical to the oracle */
    const uint64_t P = 17683968, beta[5] = {100, 10, 0, 250, 40};
    uint64_t b[6], ob[6];
    CHECK(dedloc_partition(P, 5, beta, 64, b) == DEDLOC_OK, "partition: %s", dedloc_last_error());
    CHECK(oracle_partition(P, 5, beta, 64, ob) == 0, "oracle partition");
    CHECK(same_bits(b, ob, sizeof b), "partition differs from the oracle");
    const uint32_t counts[6] = {3, 0, 7, 1, 12, 255};
    float w[6], ow[6];
    CHECK(dedloc_weights(counts, 6, w) == DEDLOC_OK, "weights: %s", dedloc_last_error());
    CHECK(oracle_weights(counts, 6, ow) == 0, "oracle weights");
    CHECK(same_bits(w, ow, sizeof w), "weights differ from the oracle");

    /* encoded sizes */
    uint64_t ns = 7;
    CHECK(dedloc_encoded_bytes(DEDLOC_CODEC_FP16, 0, 1000, &ns) == 2000 && ns == 0, "fp16 encoded size");
    CHECK(dedloc_encoded_bytes(DEDLOC_CODEC_I8, DEDLOC_I8_BLOCK, 2049, &ns) == 2049 && ns == 3, "int8 encoded size");

    /* validation happens on the host, before anything is enqueued */
    const uint32_t zero[2] = {0, 0};
    CHECK(dedloc_weights(zero, 2, w) == DEDLOC_ERR_ZERO_WEIGHT, "all-zero counts");
    CHECK(strlen(dedloc_last_error()) > 0, "no error message");
    CHECK(dedloc_partition(P, 0, NULL, 64, b) == DEDLOC_ERR_INVALID_ARG, "zero shards");
    const uint64_t off[3] = {0, 12, 24};  /* 12 is not a multiple of 8 */
    const uint8_t flags[2] = {3, 3};
    CHECK(dedloc_lamb_workspace_bytes(24, off, 2) == 0, "bad tensor table accepted");
    const uint64_t off_ok[3] = {0, 16, 24};
    CHECK(dedloc_lamb_workspace_bytes(24, off_ok, 2) > 0, "good tensor table rejected");
    dedloc_lamb_cfg cfg = {1e-3f, 0.9f, 0.999f, 1e-6f, 0.01f, 1, 1, 0};
    float fake[64];
    float *mis = (float *)((char *)fake + 4);  /* not 16-byte aligned */
    char ws[4096];
    int rc = dedloc_lamb_step(mis, mis, mis, mis, NULL, DEDLOC_CODEC_F32, 0, 24, off_ok, flags, 2, &cfg, NULL,
                              ws, sizeof ws, NULL);
    CHECK(rc == DEDLOC_ERR_ALIGN, "misaligned buffers: got %d", rc);
    const void *pc[2] = {fake, fake};
    rc = dedloc_reduce_shard(pc, NULL, zero, 2, 8, DEDLOC_CODEC_FP16, 0, fake, NULL, NULL, NULL);
    CHECK(rc == DEDLOC_ERR_ZERO_WEIGHT, "reduce with no samples: got %d", rc);
    rc = dedloc_reduce_shard(pc, NULL, counts, 0, 8, DEDLOC_CODEC_FP16, 0, fake, NULL, NULL, NULL);
    CHECK(rc == DEDLOC_ERR_INVALID_ARG, "reduce with no peers: got %d", rc);
}

/* ---------------------------------------------------------------- device */

static void *dev_copy(const void *h, size_t bytes) {
    void *d = NULL;
    HIP(hipMalloc(&d, bytes ? bytes : 16));
    if (h && bytes) HIP(hipMemcpy(d, h, bytes, hipMemcpyHostToDevice));
    return d;
}

static void host_copy(void *h, const void *d, size_t bytes) {
    if (bytes) HIP(hipMemcpy(h, d, bytes, hipMemcpyDeviceToHost));
}

/* One round of codec `codec` on device 0 against the oracle.  local >= 0:
 * that peer hands the round its fp32 gradient (the round writes its message). */
static void device_round(int32_t codec, int local) {
    enum { N = 5, T = 3 };
    const uint64_t sizes[T] = {2 * 2048, 1024 + 520, 2048 * 2 + 5};
    uint64_t off[T + 1] = {0};
    for (int t = 0; t < T; t++) off[t + 1] = off[t] + sizes[t];
    const uint64_t P = off[T];
    const uint8_t flags[T] = {3, 2, 3};
    const uint32_t counts[N] = {3, 0, 7, 1, 12};
    const uint32_t block = DEDLOC_I8_BLOCK;
    const size_t cb = codec == DEDLOC_CODEC_FP16 ? 2 : 1;
    const size_t nsc = (P + block - 1) / block;
    rng_state = 0x9E3779B97F4A7C15ull ^ (uint64_t)(codec * 131 + local + 7);

    float *grad[N], *x = malloc(P * 4), *m = malloc(P * 4), *v = malloc(P * 4);
    void *codes[N];
    float *scales[N];
    for (int p = 0; p < N; p++) {
        grad[p] = malloc(P * 4);
        for (uint64_t e = 0; e < P; e++) grad[p][e] = gauss(1e-3f) * (uniform() < 0.01 ? 100.0f : 1.0f);
        codes[p] = malloc(P * cb);
        scales[p] = malloc(nsc * 4);
        if (codec == DEDLOC_CODEC_FP16) oracle_encode_fp16(grad[p], P, codes[p]);
        else oracle_encode_i8(grad[p], P, block, codes[p], scales[p]);
    }
    for (uint64_t e = 0; e < P; e++) {
        x[e] = gauss(0.02f);
        m[e] = gauss(1e-4f);
        const float s = gauss(1e-3f);
        v[e] = s * s;
    }
    const uint64_t beta[3] = {5, 1, 3};
    uint64_t bounds[4];
    CHECK(dedloc_partition(P, 3, beta, codec == DEDLOC_CODEC_FP16 ? 64 : block, bounds) == DEDLOC_OK, "bounds");

    /* device buffers: hipMalloc, no other allocator */
    void *d_codes[N];
    float *d_scales[N], *d_grad_local = NULL;
    for (int p = 0; p < N; p++) {
        d_codes[p] = dev_copy(codes[p], P * cb);
        d_scales[p] = dev_copy(scales[p], nsc * 4);
    }
    HIP(hipMemset(d_codes[1], 0xff, P * cb));  /* peer 1 holds no samples: never read */
    HIP(hipMemset(d_scales[1], 0xff, nsc * 4));
    if (local >= 0) {
        d_grad_local = dev_copy(grad[local], P * 4);
        HIP(hipMemset(d_codes[local], 0x7e, P * cb));  /* the round must write it */
        HIP(hipMemset(d_scales[local], 0xff, nsc * 4));
    }
    /* the library's encode of one peer's gradient equals the oracle's */
    float *d_g0 = dev_copy(grad[0], P * 4);
    void *d_enc = dev_copy(NULL, P * cb);
    float *d_enc_sc = dev_copy(NULL, nsc * 4);
    CHECK(dedloc_encode(d_g0, P, codec, block, d_enc, d_enc_sc, NULL) == DEDLOC_OK, "encode: %s", dedloc_last_error());

    float *d_x = dev_copy(x, P * 4), *d_m = dev_copy(m, P * 4), *d_v = dev_copy(v, P * 4);
    void *d_out = dev_copy(NULL, P * cb);
    float *d_out_sc = dev_copy(NULL, nsc * 4), *d_mean = dev_copy(NULL, P * 4), *d_trust = dev_copy(NULL, T * 4);
    const size_t ws_bytes = dedloc_lamb_workspace_bytes(P, off, T);
    CHECK(ws_bytes > 0, "workspace size");
    void *d_ws = dev_copy(NULL, ws_bytes);
    CHECK(dedloc_workspace_clear(d_ws, ws_bytes, NULL) == DEDLOC_OK, "workspace clear");

    const dedloc_lamb_cfg cfg = {2e-3f, 0.9f, 0.999f, 1e-6f, 0.01f, 3, 1, 0};
    const dedloc_local_peer lp = {(uint32_t)(local >= 0 ? local : 0), d_grad_local};
    const float *const *psc = codec == DEDLOC_CODEC_I8 ? (const float *const *)d_scales : NULL;
    int rc = dedloc_round((const void *const *)d_codes, psc, counts, N, bounds, 3, codec, block, d_out,
                          codec == DEDLOC_CODEC_I8 ? d_out_sc : NULL, d_x, d_m, d_v, P, off, flags, T, &cfg,
                          d_trust, d_mean, local >= 0 ? &lp : NULL, d_ws, ws_bytes, NULL);
    CHECK(rc == DEDLOC_OK, "round: %d %s", rc, dedloc_last_error());
    HIP(hipDeviceSynchronize());

    /* the oracle on the host, from the same messages and state */
    const oracle_lamb_cfg ocfg = {2e-3f, 0.9f, 0.999f, 1e-6f, 0.01f, 3, 1, 0};
    void *o_out = malloc(P * cb);
    float *o_sc = malloc(nsc * 4), *o_mean = malloc(P * 4), *o_trust = malloc(T * 4), *scratch = malloc(3 * P * 4);
    float *ox = malloc(P * 4), *om = malloc(P * 4), *ov = malloc(P * 4);
    memcpy(ox, x, P * 4);
    memcpy(om, m, P * 4);
    memcpy(ov, v, P * 4);
    CHECK(oracle_round((const void *const *)codes, (const float *const *)scales, counts, N, bounds, 3, codec,
                       block, o_out, o_sc, ox, om, ov, P, off, flags, T, &ocfg, o_trust, o_mean, scratch) == 0,
          "oracle round");

    void *g_out = malloc(P * cb), *g_enc = malloc(P * cb), *g_local = malloc(P * cb);
    float *g_sc = malloc(nsc * 4), *g_enc_sc = malloc(nsc * 4), *g_mean = malloc(P * 4), *g_trust = malloc(T * 4);
    float *gx = malloc(P * 4), *gm = malloc(P * 4), *gv = malloc(P * 4);
    host_copy(g_out, d_out, P * cb);
    host_copy(g_enc, d_enc, P * cb);
    host_copy(g_enc_sc, d_enc_sc, nsc * 4);
    host_copy(g_mean, d_mean, P * 4);
    host_copy(g_trust, d_trust, T * 4);
    host_copy(gx, d_x, P * 4);
    host_copy(gm, d_m, P * 4);
    host_copy(gv, d_v, P * 4);
    if (codec == DEDLOC_CODEC_I8) host_copy(g_sc, d_out_sc, nsc * 4);

    CHECK(same_bits(g_enc, codes[0], P * cb), "encode codes differ from the oracle");
    if (codec == DEDLOC_CODEC_I8) CHECK(same_bits(g_enc_sc, scales[0], nsc * 4), "encode scales differ");
    if (local >= 0) {
        host_copy(g_local, d_codes[local], P * cb);
        CHECK(same_bits(g_local, codes[local], P * cb), "the local peer's message differs from the oracle's encode");
        if (codec == DEDLOC_CODEC_I8) {
            host_copy(g_enc_sc, d_scales[local], nsc * 4);
            CHECK(same_bits(g_enc_sc, scales[local], nsc * 4), "the local peer's scales differ from the oracle's");
        }
    }
    CHECK(same_bits(g_out, o_out, P * cb), "gathered codes differ from the oracle");
    if (codec == DEDLOC_CODEC_I8) CHECK(same_bits(g_sc, o_sc, nsc * 4), "gathered scales differ");
    CHECK(same_bits(g_mean, o_mean, P * 4), "average differs from the oracle");
    CHECK(same_bits(gm, om, P * 4), "m' differs from the oracle");
    CHECK(same_bits(gv, ov, P * 4), "v' differs from the oracle");
    double xmax = 0.0, err = 0.0;
    for (uint64_t e = 0; e < P; e++) {
        xmax = fmax(xmax, fabs((double)x[e]));
        err = fmax(err, fabs((double)gx[e] - (double)ox[e]));
    }
    CHECK(err <= 1e-5 * xmax, "x' differs from the oracle by %g (bar %g)", err, 1e-5 * xmax);
    for (int t = 0; t < T; t++)
        CHECK(fabs((double)g_trust[t] - (double)o_trust[t]) <= 1e-6 * fabs((double)o_trust[t]),
              "trust ratio %d: %g vs %g", t, g_trust[t], o_trust[t]);
    printf("c-abi %s round%s: P=%llu, %d tensors, %d peers: %s\n", codec == DEDLOC_CODEC_FP16 ? "fp16" : "int8",
           local >= 0 ? " (local peer)" : "", (unsigned long long)P, T, N, failures ? "MISMATCH" : "ok");

    /* the same round from the same state through the entry point without a
     * workspace argument: the same bits */
    HIP(hipMemcpy(d_x, x, P * 4, hipMemcpyHostToDevice));
    HIP(hipMemcpy(d_m, m, P * 4, hipMemcpyHostToDevice));
    HIP(hipMemcpy(d_v, v, P * 4, hipMemcpyHostToDevice));
    if (local >= 0) HIP(hipMemset(d_codes[local], 0x7e, P * cb));
    rc = dedloc_round_noalloc((const void *const *)d_codes, psc, counts, N, bounds, 3, codec, block, d_out,
                              codec == DEDLOC_CODEC_I8 ? d_out_sc : NULL, d_x, d_m, d_v, P, off, flags, T, &cfg,
                              d_trust, d_mean, local >= 0 ? &lp : NULL, NULL);
    CHECK(rc == DEDLOC_OK, "round_noalloc: %d %s", rc, dedloc_last_error());
    HIP(hipDeviceSynchronize());
    {
        void *n_out = malloc(P * cb);
        float *n_x = malloc(P * 4), *n_m = malloc(P * 4), *n_v = malloc(P * 4), *n_trust = malloc(T * 4);
        host_copy(n_out, d_out, P * cb);
        host_copy(n_x, d_x, P * 4);
        host_copy(n_m, d_m, P * 4);
        host_copy(n_v, d_v, P * 4);
        host_copy(n_trust, d_trust, T * 4);
        CHECK(same_bits(n_out, g_out, P * cb) && same_bits(n_x, gx, P * 4) && same_bits(n_m, gm, P * 4) &&
                  same_bits(n_v, gv, P * 4) && same_bits(n_trust, g_trust, T * 4),
              "dedloc_round_noalloc differs from dedloc_round");
        printf("c-abi %s round%s without a workspace argument: %s\n", codec == DEDLOC_CODEC_FP16 ? "fp16" : "int8",
               local >= 0 ? " (local peer)" : "", failures ? "MISMATCH" : "ok");
        free(n_out);
        free(n_x);
        free(n_m);
        free(n_v);
        free(n_trust);
    }

    for (int p = 0; p < N; p++) {
        HIP(hipFree(d_codes[p]));
        HIP(hipFree(d_scales[p]));
        free(grad[p]);
        free(codes[p]);
        free(scales[p]);
    }
    if (d_grad_local) HIP(hipFree(d_grad_local));
    void *dev_bufs[] = {d_g0, d_enc, d_enc_sc, d_x, d_m, d_v, d_out, d_out_sc, d_mean, d_trust, d_ws};
    for (size_t i = 0; i < sizeof dev_bufs / sizeof dev_bufs[0]; i++) HIP(hipFree(dev_bufs[i]));
    void *host_bufs[] = {x, m, v, o_out, o_sc, o_mean, o_trust, scratch, ox, om, ov,
                         g_out, g_enc, g_local, g_sc, g_enc_sc, g_mean, g_trust, gx, gm, gv};
    for (size_t i = 0; i < sizeof host_bufs / sizeof host_bufs[0]; i++) free(host_bufs[i]);
}

int main(int argc, char **argv) {
    const int host_only = argc > 1 && strcmp(argv[1], "--host") == 0;
    host_checks();
    printf("c-abi host checks: %s\n", failures ? "MISMATCH" : "ok");
    if (host_only || failures) return failures ? 1 : 0;
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || n == 0) {
        printf("c-abi: no device, device checks skipped\n");
        return 77;
    }
    HIP(hipSetDevice(0));
    device_round(DEDLOC_CODEC_FP16, -1);
    device_round(DEDLOC_CODEC_FP16, 2);
    device_round(DEDLOC_CODEC_I8, -1);
    device_round(DEDLOC_CODEC_I8, 3);
    return failures ? 1 : 0;
}
