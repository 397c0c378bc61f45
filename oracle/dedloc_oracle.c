/*
 * CPU oracle for one DeDLOC averaging round: TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg load
 * this file's library.  It is the plain, slow, sequential definition of what
 * the GPU library computes, written from the paper and the codec/optimizer
 * definitions stated below.  It shares no source with the GPU library.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math (no contraction: every fused
 * multiply-add below is an explicit fmaf, every other operation rounds once).
 * The CPU baseline's build adds -O3 -march=native -fopenmp: loops marked
 * OR_PARALLEL_FOR, whose iterations are independent, are then split
 * statically over threads.  Every element is still computed by the same
 * operations and every sum over elements stays sequential in element order,
 * so the results are the same bits for any thread count.
 *
 * Pins (the checks that tie each function to something other than itself)
 * live in tests/test_oracle_*.py; the whole composed round is "parity
 * unpinned" against the paper, which prints no numeric example for it.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#define OR_PARALLEL_FOR _Pragma("omp parallel for schedule(static)")
#else
#define OR_PARALLEL_FOR
#endif

#define OR_OK 0
#define OR_EINVAL (-1)
#define OR_EZERO (-3)

/* Threads the parallel loops use (n > 0 sets it); 1 in the plain build. */
int oracle_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
    return omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Shard partition.  Section 3.2 / Appendix B: after solving the load-
 * balancing problem, peer i aggregates a share of the gradient vector that is
 * proportional to its effective throughput.  The paper does not say how a
 * fractional share becomes whole elements; the reading used here floors the
 * cumulative share to a multiple of `align` elements:
 *     C_k = sum_{i<k} beta_i,   B_k = align * floor(P * C_k / (C_n * align)),
 *     B_0 = 0, B_n = P.
 * beta = NULL means equal shares.  Returns OR_EINVAL when n == 0, align == 0
 * or all shares are zero. */
int oracle_partition(uint64_t P, uint32_t n, const uint64_t *beta,
                     uint32_t align, uint64_t *bounds)
{
    if (n == 0 || align == 0) return OR_EINVAL;
    unsigned __int128 total = 0;
    for (uint32_t i = 0; i < n; i++) total += beta ? beta[i] : 1u;
    if (total == 0) return OR_EINVAL;
    unsigned __int128 cum = 0;
    bounds[0] = 0;
    for (uint32_t k = 1; k < n; k++) {
        cum += beta ? beta[k - 1] : 1u;
        unsigned __int128 q = ((unsigned __int128)P * cum) / (total * align);
        bounds[k] = (uint64_t)(q * align);
    }
    bounds[n] = P;
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Peer weights.  The global gradient is the mean over every accumulated
 * sample (appendix "Convergence analysis", the definition of g^k), so a peer
 * whose mean gradient covers n_p samples enters with weight n_p / sum_q n_q.
 * Each weight is one correctly rounded fp32 division of exactly converted
 * integers; the total must stay below 2^24 so the conversion is exact.
 * Returns OR_EZERO if every count is zero. */
int oracle_weights(const uint32_t *counts, uint32_t n, float *w)
{
    uint64_t W = 0;
    for (uint32_t p = 0; p < n; p++) W += counts[p];
    if (W == 0) return OR_EZERO;
    if (W > (1u << 24)) return OR_EINVAL;
    for (uint32_t p = 0; p < n; p++) w[p] = (float)counts[p] / (float)W;
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* fp16 wire codec (the build's codec: the paper trains GPU peers in fp16 but
 * does not specify a wire format).  Encode = IEEE-754 binary16 round to
 * nearest, ties to even, gradual underflow kept, overflow to infinity, NaN to
 * a quiet NaN of the same sign.  Written out from the format definition. */

/* v / 2^s rounded to nearest, ties to even (s >= 0). */
static uint64_t shift_rne(uint64_t v, int s)
{
    if (s == 0) return v;
    if (s >= 64) return 0;
    uint64_t q = v >> s;
    uint64_t rem = v & ((1ull << s) - 1);
    uint64_t half = 1ull << (s - 1);
    if (rem > half || (rem == half && (q & 1))) q++;
    return q;
}

static uint16_t f32_to_f16(float f)
{
    uint32_t b;
    memcpy(&b, &f, 4);
    uint16_t sign = (uint16_t)((b >> 16) & 0x8000u);
    uint32_t e8 = (b >> 23) & 0xffu;
    uint32_t m23 = b & 0x7fffffu;
    if (e8 == 0xff) return (uint16_t)(sign | (m23 ? 0x7e00u : 0x7c00u));
    if (e8 == 0) return sign; /* fp32 zero or subnormal: below 2^-126, rounds to 0 */
    int e = (int)e8 - 127;           /* value = sig * 2^(e-23), sig in [2^23, 2^24) */
    uint64_t sig = m23 | 0x800000u;
    if (e > 15) return (uint16_t)(sign | 0x7c00u);
    if (e >= -14) {
        /* normal range: keep 11 significant bits; a carry moves the exponent */
        uint64_t r = shift_rne(sig, 13);           /* in [2^10, 2^11] */
        uint32_t h = (uint32_t)((e + 14) << 10) + (uint32_t)r;
        if (h >= 0x7c00u) h = 0x7c00u;
        return (uint16_t)(sign | h);
    }
    /* subnormal range: count units of 2^-24 */
    uint64_t r = shift_rne(sig, -e - 1);           /* sig*2^(e-23) / 2^-24 */
    return (uint16_t)(sign | (uint32_t)r);          /* r == 2^10 is the smallest normal */
}

static float f16_to_f32(uint16_t h)
{
    float s = (h & 0x8000u) ? -1.0f : 1.0f;
    uint32_t e5 = (h >> 10) & 0x1fu;
    uint32_t m10 = h & 0x3ffu;
    if (e5 == 0x1f) return m10 ? s * NAN : s * INFINITY;
    if (e5 == 0) return s * ldexpf((float)m10, -24);
    return s * ldexpf((float)(m10 | 0x400u), (int)e5 - 25);
}

void oracle_encode_fp16(const float *x, size_t n, uint16_t *codes)
{
    OR_PARALLEL_FOR
    for (size_t i = 0; i < n; i++) codes[i] = f32_to_f16(x[i]);
}

void oracle_decode_fp16(const uint16_t *codes, size_t n, float *out)
{
    OR_PARALLEL_FOR
    for (size_t i = 0; i < n; i++) out[i] = f16_to_f32(codes[i]);
}

/* ------------------------------------------------------------------------ */
/* 8-bit absmax codec (the build's stress codec).  The message is cut into
 * blocks of `block` elements from its first element; the last block may be
 * partial.  Per block: a = max |x|, s = a / 127 (fp32, correctly rounded);
 * if s == 0 (a == 0, or a so small that a / 127 underflows: a <= 63 *
 * 2^-149) every code is 0; otherwise q = clamp(rint(x / s), -127, 127) with
 * ties to even.  Decode: x = q * s.  Inputs must be finite. */
void oracle_encode_i8(const float *x, size_t n, uint32_t block, int8_t *codes,
                      float *scales)
{
    size_t nb = (n + block - 1) / block;
    OR_PARALLEL_FOR
    for (size_t bi = 0; bi < nb; bi++) {
        size_t b0 = bi * block;
        size_t b1 = b0 + block < n ? b0 + block : n;
        float a = 0.0f;
        for (size_t i = b0; i < b1; i++) {
            float ax = fabsf(x[i]);
            if (ax > a) a = ax;
        }
        float s = a / 127.0f;
        scales[bi] = s;
        for (size_t i = b0; i < b1; i++) {
            float q = 0.0f;
            if (s != 0.0f) {
                q = rintf(x[i] / s);
                if (q > 127.0f) q = 127.0f;
                if (q < -127.0f) q = -127.0f;
            }
            codes[i] = (int8_t)q;
        }
    }
}

void oracle_decode_i8(const int8_t *codes, const float *scales, size_t n,
                      uint32_t block, float *out)
{
    OR_PARALLEL_FOR
    for (size_t i = 0; i < n; i++) out[i] = (float)codes[i] * scales[i / block];
}

/* codec ids: 1 = fp16, 2 = int8 absmax */
static void decode_any(int codec, const void *codes, const float *scales,
                       size_t n, uint32_t block, float *out)
{
    if (codec == 1) oracle_decode_fp16((const uint16_t *)codes, n, out);
    else oracle_decode_i8((const int8_t *)codes, scales, n, block, out);
}

static void encode_any(int codec, const float *x, size_t n, uint32_t block,
                       void *codes, float *scales)
{
    if (codec == 1) oracle_encode_fp16(x, n, (uint16_t *)codes);
    else oracle_encode_i8(x, n, block, (int8_t *)codes, scales);
}

static size_t code_bytes(int codec) { return codec == 1 ? 2 : 1; }

/* ------------------------------------------------------------------------ */
/* Reducer step (Section 3.2: the peer that owns a share of the vector sums
 * what every sender sent for that share and sends the mean back).  Peers with zero
 * samples have weight 0 and are not read at all (Appendix B: a peer with
 * c_i != 1 disregards its local gradient but still aggregates).
 *     mean[e] = sum over active p, ascending, of w_p * dec_p[e]
 * accumulated from +0 with one fused multiply-add per peer.  The mean is then
 * re-encoded with the wire codec.  `scratch` holds 2*len floats. */
int oracle_reduce(const void *const *peer_codes, const float *const *peer_scales,
                  const uint32_t *counts, uint32_t n_peers, size_t len,
                  int codec, uint32_t block, void *out_codes, float *out_scales,
                  float *out_mean, float *scratch)
{
    float w[1024];
    if (n_peers == 0 || n_peers > 1024) return OR_EINVAL;
    int rc = oracle_weights(counts, n_peers, w);
    if (rc != OR_OK) return rc;
    float *acc = scratch, *dec = scratch + len;
    OR_PARALLEL_FOR
    for (size_t e = 0; e < len; e++) acc[e] = 0.0f;
    for (uint32_t p = 0; p < n_peers; p++) {
        if (counts[p] == 0) continue;
        decode_any(codec, peer_codes[p], peer_scales ? peer_scales[p] : NULL,
                   len, block, dec);
        OR_PARALLEL_FOR
        for (size_t e = 0; e < len; e++) acc[e] = fmaf(w[p], dec[e], acc[e]);
    }
    if (out_mean) memcpy(out_mean, acc, len * sizeof(float));
    encode_any(codec, acc, len, block, out_codes, out_scales);
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* LAMB step on the averaged gradient (Section 3.1 trains with large batches
 * and LAMB; the sahajBERT-XL appendix keeps LAMB statistics).  The update is
 * the published LAMB algorithm with Adam moments and a layer-wise trust ratio:
 *   m' = b1*m + (1-b1)*g,  v' = b2*v + (1-b2)*g^2
 *   u  = (m'/c1) / (sqrt(v'/c2) + eps) + lambda_t * x,  c_i = 1 - b_i^step
 *   r  = ||x_t|| / ||u_t|| per tensor t (1 if either norm is 0 or the tensor
 *        is not adaptive),   x' = x - (lr*r) * u.
 * Roundings: m' = fmaf(b1, m, (1-b1)*g); v' = fmaf(b2, v, (1-b2)*(g*g));
 * c_i computed in double and rounded to fp32; the norms accumulate exact
 * double squares in double, in element order; r = (float)(X/U).
 * flags: bit 0 weight decay (lambda_t = wd, else 0), bit 1 adaptive.
 * trust (nullable) receives r per tensor. */
typedef struct {
    float lr, beta1, beta2, eps, weight_decay;
    uint64_t step;
    int32_t bias_correction;
    int32_t force_unit_trust;
} oracle_lamb_cfg;

int oracle_lamb(float *x, float *m, float *v, const float *g, uint64_t P,
                const uint64_t *off, const uint8_t *flags, uint32_t T,
                const oracle_lamb_cfg *cfg, float *trust, float *u)
{
    if (T == 0 || off[0] != 0 || off[T] != P || cfg->step == 0) return OR_EINVAL;
    for (uint32_t t = 0; t < T; t++)
        if (off[t + 1] < off[t]) return OR_EINVAL;
    float c1 = 1.0f, c2 = 1.0f;
    if (cfg->bias_correction) {
        c1 = (float)(1.0 - pow((double)cfg->beta1, (double)cfg->step));
        c2 = (float)(1.0 - pow((double)cfg->beta2, (double)cfg->step));
    }
    float omb1 = 1.0f - cfg->beta1, omb2 = 1.0f - cfg->beta2;
    for (uint32_t t = 0; t < T; t++) {
        float lam = (flags[t] & 1) ? cfg->weight_decay : 0.0f;
        const uint64_t e0 = off[t], e1 = off[t + 1];
        OR_PARALLEL_FOR
        for (uint64_t e = e0; e < e1; e++) {
            float gg = g[e];
            float mn = fmaf(cfg->beta1, m[e], omb1 * gg);
            float vn = fmaf(cfg->beta2, v[e], omb2 * (gg * gg));
            float mh = mn / c1;
            float vh = vn / c2;
            float ue = mh / (sqrtf(vh) + cfg->eps) + lam * x[e];
            m[e] = mn;
            v[e] = vn;
            u[e] = ue;
        }
        double sx = 0.0, su = 0.0;
        for (uint64_t e = e0; e < e1; e++) {
            sx += (double)x[e] * (double)x[e];
            su += (double)u[e] * (double)u[e];
        }
        double X = sqrt(sx), U = sqrt(su);
        float r = 1.0f;
        if (!cfg->force_unit_trust && (flags[t] & 2) && X > 0.0 && U > 0.0)
            r = (float)(X / U);
        if (trust) trust[t] = r;
        float lrr = cfg->lr * r;
        OR_PARALLEL_FOR
        for (uint64_t e = e0; e < e1; e++) x[e] = x[e] - lrr * u[e];
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* LARS step (Section 4.1 trains SwAV with LARS).  The update is the published
 * LARS algorithm (layer-wise adaptive rate scaling with momentum, learning
 * rate folded into the momentum buffer):
 *   r = eta*||x_t|| / (||g_t|| + lambda_t*||x_t||) per tensor t (1 if either
 *       norm is 0, the tensor is not adaptive, or force_unit_trust)
 *   v' = mu*v + (lr*r) * (g + lambda_t*x),   x' = x - v'
 * Roundings: d = g + lambda*x (product then sum), s = lr*r (fp32),
 * v' = fmaf(mu, v, s*d), x' = x - v'; the norms accumulate exact double
 * squares in double in element order; r is evaluated in double from the
 * norms and rounded once to fp32. */
typedef struct {
    float lr, momentum, trust_coef, weight_decay;
    int32_t force_unit_trust;
} oracle_lars_cfg;

int oracle_lars(float *x, float *v, const float *g, uint64_t P, const uint64_t *off,
                const uint8_t *flags, uint32_t T, const oracle_lars_cfg *cfg, float *trust)
{
    if (T == 0 || off[0] != 0 || off[T] != P) return OR_EINVAL;
    for (uint32_t t = 0; t < T; t++)
        if (off[t + 1] < off[t]) return OR_EINVAL;
    for (uint32_t t = 0; t < T; t++) {
        float lam = (flags[t] & 1) ? cfg->weight_decay : 0.0f;
        double sx = 0.0, sg = 0.0;
        for (uint64_t e = off[t]; e < off[t + 1]; e++) {
            sx += (double)x[e] * (double)x[e];
            sg += (double)g[e] * (double)g[e];
        }
        double X = sqrt(sx), G = sqrt(sg);
        float r = 1.0f;
        if (!cfg->force_unit_trust && (flags[t] & 2) && X > 0.0 && G > 0.0)
            r = (float)((double)cfg->trust_coef * X / (G + (double)lam * X));
        if (trust) trust[t] = r;
        float s = cfg->lr * r;
        const uint64_t e0 = off[t], e1 = off[t + 1];
        OR_PARALLEL_FOR
        for (uint64_t e = e0; e < e1; e++) {
            float d = g[e] + lam * x[e];
            float vn = fmaf(cfg->momentum, v[e], s * d);
            v[e] = vn;
            x[e] = x[e] - vn;
        }
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* One whole round as a peer sees it (Section 3.1: accumulate, exchange,
 * one optimizer step; Section 3.2: reduce-scatter by shards, then gather).
 * Every shard k of `bounds` is reduced from the N peers' full-vector
 * messages, the encoded means are gathered into out_codes/out_scales, every
 * peer decodes the same gathered message and applies one LAMB step.
 * For the int8 codec interior shard bounds must be multiples of `block`, so
 * a message's blocks are the same whether counted from the vector start or
 * from the shard start.  `scratch` holds 3*P floats. */
int oracle_round(const void *const *peer_codes, const float *const *peer_scales,
                 const uint32_t *counts, uint32_t n_peers, const uint64_t *bounds,
                 uint32_t n_shards, int codec, uint32_t block, void *out_codes,
                 float *out_scales, float *x, float *m, float *v, uint64_t P,
                 const uint64_t *off, const uint8_t *flags, uint32_t T,
                 const oracle_lamb_cfg *cfg, float *trust, float *out_mean,
                 float *scratch)
{
    if (n_peers == 0 || n_peers > 1024 || n_shards == 0) return OR_EINVAL;
    if (bounds[0] != 0 || bounds[n_shards] != P) return OR_EINVAL;
    const void *pc[1024];
    const float *ps[1024];
    size_t cb = code_bytes(codec);
    uint32_t blk = codec == 1 ? 1 : block;
    for (uint32_t k = 0; k < n_shards; k++) {
        uint64_t b0 = bounds[k], b1 = bounds[k + 1];
        if (b1 < b0) return OR_EINVAL;
        if (codec == 2 && k > 0 && b0 % blk) return OR_EINVAL;
        for (uint32_t p = 0; p < n_peers; p++) {
            pc[p] = (const char *)peer_codes[p] + b0 * cb;
            ps[p] = codec == 2 ? peer_scales[p] + b0 / blk : NULL;
        }
        int rc = oracle_reduce(pc, codec == 2 ? ps : NULL, counts, n_peers, b1 - b0,
                               codec, blk, (char *)out_codes + b0 * cb,
                               codec == 2 ? out_scales + b0 / blk : NULL,
                               out_mean ? out_mean + b0 : NULL, scratch);
        if (rc != OR_OK) return rc;
    }
    float *ghat = scratch + 2 * P;
    for (uint32_t k = 0; k < n_shards; k++) {
        uint64_t b0 = bounds[k], b1 = bounds[k + 1];
        decode_any(codec, (const char *)out_codes + b0 * cb,
                   codec == 2 ? out_scales + b0 / blk : NULL, b1 - b0, blk, ghat + b0);
    }
    if (!cfg) return OR_OK; /* reduce-scatter and gather only: ghat = scratch + 2P */
    return oracle_lamb(x, m, v, ghat, P, off, flags, T, cfg, trust, scratch);
}

/* The same round with the LARS step in place of LAMB (SwAV, Section 4.1);
 * v is the momentum buffer.  `scratch` holds 3*P floats. */
int oracle_round_lars(const void *const *peer_codes, const float *const *peer_scales,
                      const uint32_t *counts, uint32_t n_peers, const uint64_t *bounds,
                      uint32_t n_shards, int codec, uint32_t block, void *out_codes,
                      float *out_scales, float *x, float *v, uint64_t P,
                      const uint64_t *off, const uint8_t *flags, uint32_t T,
                      const oracle_lars_cfg *cfg, float *trust, float *out_mean,
                      float *scratch)
{
    int rc = oracle_round(peer_codes, peer_scales, counts, n_peers, bounds, n_shards, codec,
                          block, out_codes, out_scales, x, NULL, v, P, off, flags, T, NULL,
                          trust, out_mean, scratch);
    if (rc != OR_OK) return rc;
    return oracle_lars(x, v, scratch + 2 * P, P, off, flags, T, cfg, trust);
}

/* ------------------------------------------------------------------------ */
/* Group (Moshpit) all-reduce (Section 3.2 "Node failures", Appendix C
 * "Fault tolerance"): instead of one global average, peers average in
 * groups of m, in consecutive iterations with alternating groups, so that
 * every peer holds the global average after ceil(log_m n) iterations.
 *
 * The grid used here: d = max(1, ceil(log_m n)) iterations over m^d slots;
 * slot i holds peer i (i < n), the others are empty (zero samples).  In
 * iteration k the groups are the sets of slots whose base-m digits agree
 * except digit k; group id = slot with digit k removed.  Each member carries
 * a sample count (initially its own); a group whose members carry zero
 * samples in total produces nothing, otherwise it computes the weighted
 * average of its members' messages exactly as oracle_reduce does (members
 * with zero samples are not read), and every member takes the encoded group
 * average and the group's total count.
 *
 * `iters` = 0 runs the d iterations; a positive value runs that many (to
 * observe the intermediate state).  Outputs: the messages of the last
 * iteration's groups, group g at out_codes + g*len codes (and, for int8,
 * out_scales + g*ceil(len/block)); peer_out[i] = the group whose message
 * peer i holds (UINT32_MAX if it holds none); *n_out = number of groups of
 * the last iteration.  `work` holds 2*m^(d-1)*len codes (plus scales) and
 * `scratch` 2*len floats. */
static uint32_t ipow(uint32_t m, uint32_t d)
{
    uint32_t r = 1;
    for (uint32_t i = 0; i < d; i++) r *= m;
    return r;
}

int oracle_group_allreduce(const void *const *peer_codes, const float *const *peer_scales,
                           const uint32_t *counts, uint32_t n, uint32_t m, size_t len, int codec,
                           uint32_t block, uint32_t iters, void *out_codes, float *out_scales,
                           uint32_t *peer_out, uint32_t *n_out, void *work, float *work_scales,
                           float *scratch)
{
    if (n == 0 || n > 1024 || m < 2) return OR_EINVAL;
    uint64_t total = 0;
    for (uint32_t i = 0; i < n; i++) total += counts[i];
    if (total == 0) return OR_EZERO;
    uint32_t d = 1;
    while (ipow(m, d) < n) d++;
    if (iters == 0) iters = d;
    if (iters > d) return OR_EINVAL;
    const uint32_t slots = ipow(m, d);
    const uint32_t groups = slots / m;
    const size_t cb = code_bytes(codec);
    const uint32_t blk = codec == 1 ? 1 : block;
    const size_t nsc = codec == 1 ? 0 : (len + blk - 1) / blk;

    /* per slot: where its message is (-1: original peer message; else the
     * group index in the previous iteration's buffer) and its count */
    int64_t src[1024 * 16];
    uint64_t cnt[1024 * 16];
    if (slots > 1024 * 16) return OR_EINVAL;
    for (uint32_t i = 0; i < slots; i++) {
        src[i] = -1;
        cnt[i] = i < n ? counts[i] : 0;
    }
    const void *mem_codes[1024];
    const float *mem_scales[1024];
    uint32_t mem_counts[1024];
    for (uint32_t k = 0; k < iters; k++) {
        const uint32_t lo = ipow(m, k); /* weight of digit k */
        const int last = (k + 1 == iters);
        char *dst_codes = last ? (char *)out_codes : (char *)work + (size_t)(k % 2) * groups * len * cb;
        float *dst_scales = last ? out_scales : work_scales + (size_t)(k % 2) * groups * nsc;
        const char *prev_codes = (const char *)work + (size_t)((k + 1) % 2) * groups * len * cb;
        const float *prev_scales = work_scales + (size_t)((k + 1) % 2) * groups * nsc;
        int64_t nsrc[1024 * 16];
        uint64_t ncnt[1024 * 16];
        for (uint32_t g = 0; g < groups; g++) {
            /* members: slots with digit k = 0..m-1, other digits from g */
            const uint32_t base = (g / lo) * lo * m + (g % lo);
            uint64_t gt = 0;
            uint32_t nm = 0;
            for (uint32_t j = 0; j < m; j++) {
                const uint32_t s = base + j * lo;
                gt += cnt[s];
            }
            for (uint32_t j = 0; j < m; j++) {
                const uint32_t s = base + j * lo;
                if (cnt[s] == 0) continue;
                if (src[s] < 0) {
                    mem_codes[nm] = peer_codes[s];
                    mem_scales[nm] = codec == 2 ? peer_scales[s] : NULL;
                } else {
                    mem_codes[nm] = prev_codes + (size_t)src[s] * len * cb;
                    mem_scales[nm] = codec == 2 ? prev_scales + (size_t)src[s] * nsc : NULL;
                }
                if (cnt[s] > 0xffffffffull) return OR_EINVAL;
                mem_counts[nm] = (uint32_t)cnt[s];
                nm++;
            }
            if (gt > 0) {
                int rc = oracle_reduce(mem_codes, codec == 2 ? mem_scales : NULL, mem_counts, nm, len,
                                       codec, blk, dst_codes + (size_t)g * len * cb,
                                       codec == 2 ? dst_scales + (size_t)g * nsc : NULL, NULL, scratch);
                if (rc != OR_OK) return rc;
            }
            for (uint32_t j = 0; j < m; j++) {
                const uint32_t s = base + j * lo;
                nsrc[s] = gt > 0 ? (int64_t)g : -2;
                ncnt[s] = gt;
            }
        }
        for (uint32_t i = 0; i < slots; i++) {
            src[i] = nsrc[i];
            cnt[i] = ncnt[i];
        }
    }
    for (uint32_t i = 0; i < n; i++) peer_out[i] = src[i] >= 0 ? (uint32_t)src[i] : 0xffffffffu;
    *n_out = groups;
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Local accumulation (Section 3.1: a peer keeps summing micro-batch
 * gradients, however fast it runs, until the whole group's sample total
 * hits the global batch size).  A micro-batch
 * of b samples whose mean gradient is g adds b*g to the running sum:
 *     acc = fmaf(b, g, acc)          (one rounding per element per batch)
 * When the round starts the peer's mean gradient is acc / count (one
 * correctly rounded division, count = samples accumulated), encoded with the
 * wire codec; reset != 0 then zeroes acc for the next round.  g is fp32
 * (codec 0) or fp16 codes (codec 1). */
void oracle_accumulate(float *acc, const void *g, int g_codec, size_t n, float b)
{
    for (size_t i = 0; i < n; i++) {
        float gi = g_codec == 0 ? ((const float *)g)[i] : f16_to_f32(((const uint16_t *)g)[i]);
        acc[i] = fmaf(b, gi, acc[i]);
    }
}

int oracle_finalize(float *acc, size_t n, uint32_t count, int codec, uint32_t block,
                    void *codes, float *scales, int reset, float *scratch)
{
    if (count == 0 || count > (1u << 24)) return count == 0 ? OR_EZERO : OR_EINVAL;
    float c = (float)count;
    for (size_t i = 0; i < n; i++) scratch[i] = acc[i] / c;
    encode_any(codec, scratch, n, codec == 1 ? 1 : block, codes, scales);
    if (reset)
        for (size_t i = 0; i < n; i++) acc[i] = 0.0f;
    return OR_OK;
}
