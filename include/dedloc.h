/*
 * dedloc.h - C ABI of the MI355X (gfx950) library for one DeDLOC averaging
 * round: wire codecs, the per-reducer shard average, and the LAMB step.
 *
 * The paper (Distributed Deep Learning In Open Collaborations) averages
 * gradients by reduce-scatter then all-gather (Section 3.2): every peer is
 * assigned a share of the flat gradient vector proportional to its
 * throughput (Appendix B), receives that share from every sender, averages
 * it and returns the average; after the exchange every peer applies one
 * optimizer step (Section 3.1), LAMB in the paper's transformer runs.
 * Here the N peers' messages are N regions of one GPU's memory.
 *
 * Conventions for every call below
 *  - Pointers are DEVICE pointers unless the argument says "host".
 *  - The caller owns every buffer; the library allocates no device memory.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream): they validate their arguments on the host, enqueue kernels and
 *    return.  Invalid arguments are rejected before anything is enqueued and
 *    leave every output untouched.
 *  - Return value: DEDLOC_OK (0) or a negative dedloc_status;
 *    dedloc_last_error() gives a message for the calling thread's last
 *    failure.  No C++ exception crosses the ABI.
 *  - fp32 and fp16 buffers are read and written in 16-byte vectors: their
 *    pointers must be 16-byte aligned (DEDLOC_ERR_ALIGN otherwise), int8
 *    code buffers too; scale buffers 4-byte aligned.
 *  - Codec ids: DEDLOC_CODEC_F32 (raw fp32; only as the LAMB gradient),
 *    DEDLOC_CODEC_FP16, DEDLOC_CODEC_I8 (8-bit absmax; `block` = 1024).
 *    For fp16 and f32 the `block` argument is ignored.
 */
#ifndef DEDLOC_H
#define DEDLOC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DEDLOC_OK = 0,
    DEDLOC_ERR_INVALID_ARG = -1,
    DEDLOC_ERR_ALIGN = -2,
    DEDLOC_ERR_ZERO_WEIGHT = -3,
    DEDLOC_ERR_WORKSPACE = -4,
    DEDLOC_ERR_HIP = -5
} dedloc_status;

enum { DEDLOC_CODEC_F32 = 0, DEDLOC_CODEC_FP16 = 1, DEDLOC_CODEC_I8 = 2 };

/* Maximum number of peers in one reduce or round call.  Up to 64 peers with
 * samples are reduced in one launch; more are reduced in launches of 64
 * chained through the fp32 average buffer (out_mean, then required). */
#define DEDLOC_MAX_PEERS 1024
/* Maximum number of peers in one group all-reduce, and in one of its groups. */
#define DEDLOC_MAX_GROUP_PEERS 1024
#define DEDLOC_MAX_GROUP_SIZE 64
/* The only supported int8 block length. */
#define DEDLOC_I8_BLOCK 1024

/* Per-tensor flag bits for the LAMB step. */
#define DEDLOC_TENSOR_DECAY 1u /* apply weight decay to this tensor */
#define DEDLOC_TENSOR_ADAPT 2u /* apply the layer-wise trust ratio */

/* LAMB hyper-parameters (host struct). step >= 1 is the 1-based step index
 * used for bias correction.  force_unit_trust != 0 replaces every trust ratio
 * by 1 (the step is then AdamW with decoupled weight decay). */
typedef struct {
    float lr, beta1, beta2, eps, weight_decay;
    uint64_t step;
    int32_t bias_correction;
    int32_t force_unit_trust;
} dedloc_lamb_cfg;

/* LARS hyper-parameters (host struct).  force_unit_trust != 0 replaces every
 * rate ratio by 1 (the step is then SGD with momentum). */
typedef struct {
    float lr, momentum, trust_coef, weight_decay;
    int32_t force_unit_trust;
} dedloc_lars_cfg;

/* Library version (major*10000 + minor*100 + patch). */
int dedloc_version(void);

/* Message for the calling thread's last failed call ("" if none). */
const char *dedloc_last_error(void);

/* Size of one encoded message of n elements: returns the code bytes and
 * stores the number of fp32 scales in *n_scales (host, nullable): 0 for
 * fp16, ceil(n / block) for int8.  Returns 0 for an unknown codec. */
size_t dedloc_encoded_bytes(int32_t codec, uint32_t block, uint64_t n, uint64_t *n_scales);

/* Shard bounds (host only, integer).  Section 3.2 / Appendix B assign each
 * aggregating peer a share of the vector proportional to its effective
 * throughput.  With C_k the sum of the first k weights (weights = NULL means
 * equal weights):
 *     bounds[0] = 0, bounds[k] = align * floor(P * C_k / (C_n * align)),
 *     bounds[n_shards] = P,
 * so the shards tile [0, P), interior bounds are multiples of `align`, and
 * the last shard keeps the remainder.  bounds (host) has n_shards+1 entries.
 * Errors: n_shards == 0, align == 0, all weights zero -> INVALID_ARG. */
int dedloc_partition(uint64_t P, uint32_t n_shards, const uint64_t *weights,
                     uint32_t align, uint64_t *bounds);

/* Peer weights (host only).  The averaged gradient is the mean over all
 * accumulated samples (appendix "Convergence analysis"): peer p, whose mean
 * gradient covers counts[p] samples, gets w[p] = counts[p] / sum(counts),
 * one correctly rounded fp32 division.  sum(counts) must be in [1, 2^24].
 * counts and w are host arrays of n entries.
 * Errors: counts or w NULL, n == 0 -> INVALID_ARG; all counts zero ->
 * ZERO_WEIGHT; sum above 2^24 -> INVALID_ARG. */
int dedloc_weights(const uint32_t *counts, uint32_t n, float *w);

/* Encode n fp32 values (the sender's side of the exchange).
 *   fp16: IEEE binary16, round to nearest even, subnormals kept, overflow
 *         to infinity, NaN to a NaN of the same sign (payload unspecified).
 *         codes: uint16[n].  scales unused (may be NULL).
 *   int8: blocks of `block` elements from x[0] (last block partial):
 *         s = max|x| / 127 (fp32), q = clamp(rint(x/s), -127, 127), ties to
 *         even; a block with s = 0 (all zero, or max|x| <= 63 * 2^-149 so
 *         that the division underflows) has every q = 0.  codes: int8[n],
 *         scales: float[ceil(n/block)].  Inputs must be finite.
 * x, codes, scales: device, caller-owned.  n == 0 is a no-op.
 * Errors: unknown codec or an int8 block other than DEDLOC_I8_BLOCK ->
 * INVALID_ARG; x or codes NULL (n > 0), or int8 scales NULL -> INVALID_ARG;
 * x or codes not 16-byte aligned, scales not 4-byte aligned -> ALIGN. */
int dedloc_encode(const float *x, uint64_t n, int32_t codec, uint32_t block,
                  void *codes, float *scales, void *stream);

/* Decode n elements: fp16 -> fp32 exactly; int8 -> q * s (one rounding).
 * codes, scales, out: device, caller-owned, laid out as dedloc_encode
 * writes them; out is fp32[n].  n == 0 is a no-op.  Errors as for
 * dedloc_encode (out in place of x). */
int dedloc_decode(const void *codes, const float *scales, uint64_t n,
                  int32_t codec, uint32_t block, float *out, void *stream);

/* The reducer's step (Section 3.2): average one shard of shard_len
 * elements as sent by n_peers peers and re-encode the average.
 *   peer_codes  (host array of n_peers device pointers) - each peer's
 *               message for this shard, already offset to the shard start;
 *   peer_scales (host array, int8 only; NULL for fp16) - each peer's block
 *               scales for this shard (blocks counted from the shard start);
 *   counts      (host, n_peers) - accumulated samples per peer.
 * mean[e] = sum over peers with counts > 0, in ascending order, of
 * w_p * decode_p[e], accumulated from +0 with one fused multiply-add per
 * peer (w_p as in dedloc_weights).  Peers with zero samples are never read
 * (Appendix B: a peer that does not compute still aggregates, and its local
 * gradient is disregarded); their pointers may be NULL.
 * Outputs: out_codes / out_scales - the encoded average (as dedloc_encode);
 * out_mean - the fp32 average before encoding; nullable with at most 64
 * peers holding samples, required with more (it then carries the running
 * sum between launches, stored exactly, so the result is the same as one
 * pass).
 * Non-finite fp16 codes (a sender whose gradient overflowed) are averaged
 * like any other value: an element with an infinity from one peer averages
 * to that infinity, +inf meeting -inf or a NaN code gives NaN, and the NaN
 * is encoded with either sign.  int8 scales must be finite.
 * Errors: n_peers == 0 or > DEDLOC_MAX_PEERS -> INVALID_ARG; all counts
 * zero -> ZERO_WEIGHT; more than 64 peers with samples and out_mean NULL ->
 * INVALID_ARG.  shard_len == 0 is a no-op (after validation). */
int dedloc_reduce_shard(const void *const *peer_codes, const float *const *peer_scales,
                        const uint32_t *counts, uint32_t n_peers, uint64_t shard_len,
                        int32_t codec, uint32_t block, void *out_codes,
                        float *out_scales, float *out_mean, void *stream);

/* Workspace for dedloc_lamb_step / dedloc_round (and the LARS
 * counterparts dedloc_lars_step / dedloc_round_lars) with this tensor table
 * (offsets: host, n_tensors+1): two fp64 partial sums per 2048-element tile,
 * one 8-byte word per tensor (its trust ratio, tagged for the call that
 * wrote it) and a counter that advances the tag on every call, graph
 * replays included.  Returns 0 for an invalid table.  Its contents need no
 * initialisation: a word left by an earlier call on the workspace never
 * carries the current tag, and other contents match it only by a 2^-32
 * chance per tensor.  Calls that share one workspace must not overlap in
 * time. */
size_t dedloc_lamb_workspace_bytes(uint64_t P, const uint64_t *offsets, uint32_t n_tensors);

/* Zero-fill a device buffer (for example a workspace) with a kernel: no
 * memset node, so the call may be captured into a graph.  ws must be
 * 4-byte aligned and ws_bytes a multiple of 4 (INVALID_ARG otherwise;
 * ws_bytes == 0 is a no-op). */
int dedloc_workspace_clear(void *ws, size_t ws_bytes, void *stream);

/* One LAMB step over a flat parameter buffer (Section 3.1 trains with LAMB;
 * the sahajBERT-XL appendix keeps its statistics), with the published LAMB
 * update and a trust ratio per tensor:
 *   m' = fma(b1, m, (1-b1)*g);  v' = fma(b2, v, (1-b2)*(g*g))
 *   u  = (m'/c1) / (sqrt(v'/c2) + eps) + lambda_t * x,  c_i = 1 - b_i^step
 *        (c_i computed in double, rounded to fp32; 1 without bias correction)
 *   r_t = ||x_t|| / ||u_t||, or 1 if either norm is 0, the tensor lacks
 *         DEDLOC_TENSOR_ADAPT, or force_unit_trust is set
 *   x' = x - (lr * r_t) * u
 * lambda_t = weight_decay if the tensor has DEDLOC_TENSOR_DECAY, else 0.
 *   x, m, v    fp32[P], updated in place;
 *   grad       the gradient: fp32[P] (grad_codec = DEDLOC_CODEC_F32) or an
 *              encoded message of P elements (fp16, or int8 with grad_scales);
 *   offsets    host uint64[n_tensors+1]: offsets[0] = 0, offsets[T] = P,
 *              non-decreasing, every offset except P a multiple of 8;
 *   flags      host uint8[n_tensors];
 *   trust_out  device float[n_tensors] (nullable): r_t.
 * The norms are accumulated in fp64 in a fixed order, so results are
 * deterministic run to run.  Non-finite gradient values are neither skipped
 * nor clamped: they go through the formulas above.  r_t is the quotient
 * only when both norms compare greater than 0, so a NaN norm gives r_t = 1;
 * an infinite norm gives 0 or infinity by the division.
 * P = 0 (every tensor empty) is valid: no element is read or written, x,
 * m, v and grad may be NULL, and trust_out receives r = 1 for every tensor.
 * Errors: cfg NULL or step 0 -> INVALID_ARG; offsets NULL, n_tensors 0,
 * offsets not tiling [0, P), a tensor of 2^32 or more elements, flags NULL
 * -> INVALID_ARG; an offset (other than P) not a multiple of 8 -> ALIGN;
 * x, m, v or grad NULL (P > 0) -> INVALID_ARG (grad: ALIGN); a buffer not
 * 16-byte aligned -> ALIGN; int8 grad without 4-byte aligned grad_scales
 * -> INVALID_ARG; ws NULL or smaller than dedloc_lamb_workspace_bytes ->
 * WORKSPACE; ws not 256-byte aligned -> ALIGN. */
int dedloc_lamb_step(float *x, float *m, float *v, const void *grad,
                     const float *grad_scales, int32_t grad_codec, uint32_t block,
                     uint64_t P, const uint64_t *offsets, const uint8_t *flags,
                     uint32_t n_tensors, const dedloc_lamb_cfg *cfg, float *trust_out,
                     void *ws, size_t ws_bytes, void *stream);

/* One LARS step over a flat parameter buffer (Section 4.1 trains SwAV with
 * LARS), with the published LARS update (layer-wise rate, momentum buffer
 * holding the learning rate):
 *   r_t = eta*||x_t|| / (||g_t|| + lambda_t*||x_t||), or 1 if either norm is
 *         0, the tensor lacks DEDLOC_TENSOR_ADAPT, or force_unit_trust is set
 *         (evaluated in double from fp64 norms, rounded once to fp32)
 *   d = g + lambda_t*x;  v' = fma(mu, v, (lr*r_t)*d);  x' = x - v'
 * eta = trust_coef, mu = momentum, lambda_t as for LAMB.
 *   x, v  fp32[P] (v is the momentum buffer), updated in place;
 *   grad, grad_scales, grad_codec, offsets, flags, trust_out, workspace: as
 *   for dedloc_lamb_step (the workspace size is the same). */
int dedloc_lars_step(float *x, float *v, const void *grad, const float *grad_scales,
                     int32_t grad_codec, uint32_t block, uint64_t P, const uint64_t *offsets,
                     const uint8_t *flags, uint32_t n_tensors, const dedloc_lars_cfg *cfg,
                     float *trust_out, void *ws, size_t ws_bytes, void *stream);

/* The local peer of a round (optional argument of dedloc_round and
 * dedloc_round_lars).  Every peer encodes its own gradient before sending
 * it (Section 3.1: peers exchange their accumulated gradients).  Instead of a
 * message encoded beforehand, peer `index` hands the round its fp32 mean
 * gradient; the round encodes it into that peer's message buffers
 * (peer_codes[index] and, for int8, peer_scales[index], which are outputs
 * here): the fp16 round inside the pass that averages it (the message is
 * written but never read back), the int8 round in a launch of its own before
 * the reduce.  Every output, that message included, is bit-identical to
 * dedloc_encode followed by the round.
 *   index  in [0, n_peers), with counts[index] > 0;
 *   grad   device fp32[P], 16-byte aligned, not overlapping any output. */
typedef struct {
    uint32_t index;
    const float *grad;
} dedloc_local_peer;

/* One whole averaging round as seen by one GPU holding every reducer
 * (Sections 3.1-3.2): each shard [bounds[k], bounds[k+1]) of the vector is
 * averaged from the n_peers messages (as dedloc_reduce_shard), the encoded
 * averages are gathered into out_codes / out_scales (full-vector messages),
 * and every element is decoded from that gathered message and updated by
 * one LAMB step (as dedloc_lamb_step).  Fused: the fp16 path reads each
 * peer byte once and re-reads only x, m and v for the trust ratio.
 *   peer_codes  host array of n_peers device pointers to full-vector
 *               messages (P elements); peer_scales likewise for int8;
 *   bounds      host uint64[n_shards+1] tiling [0, P); for int8 every
 *               interior bound must be a multiple of `block`;
 *   out_mean    fp32[P]: the average before encoding; nullable with at
 *               most 64 peers holding samples, required with more (as in
 *               dedloc_reduce_shard);
 *   local       host, nullable: the local peer (dedloc_local_peer).
 * Workspace as dedloc_lamb_workspace_bytes.  P = 0 is valid as for
 * dedloc_lamb_step: the messages, outputs and state may then be NULL.
 * Errors: the peers and counts as for dedloc_reduce_shard; the tensor table,
 * state, cfg and workspace as for dedloc_lamb_step; bounds NULL, n_shards 0,
 * bounds not tiling [0, P) -> INVALID_ARG; an int8 interior bound not a
 * multiple of `block` -> INVALID_ARG; out_codes NULL or misaligned, out_mean
 * misaligned -> ALIGN; int8 out_scales NULL or misaligned -> INVALID_ARG;
 * a local peer out of range or without samples -> INVALID_ARG, its
 * gradient NULL or misaligned -> ALIGN. */
int dedloc_round(const void *const *peer_codes, const float *const *peer_scales,
                 const uint32_t *counts, uint32_t n_peers, const uint64_t *bounds,
                 uint32_t n_shards, int32_t codec, uint32_t block, void *out_codes,
                 float *out_scales, float *x, float *m, float *v, uint64_t P,
                 const uint64_t *offsets, const uint8_t *flags, uint32_t n_tensors,
                 const dedloc_lamb_cfg *cfg, float *trust_out, float *out_mean,
                 const dedloc_local_peer *local, void *ws, size_t ws_bytes, void *stream);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * round as dedloc_round (same arguments, kernels, results and errors) but
 * without the workspace argument: the LAMB workspace is a static device
 * array of DEDLOC_NOALLOC_SCRATCH_BYTES held by every GPU the library runs
 * on until the process ends.  The call allocates no device memory.
 *   - the round's workspace (dedloc_lamb_workspace_bytes of the tensor table,
 *     about 16 bytes per 2048 elements) must fit the array: at most about
 *     2^31 elements; larger tables -> DEDLOC_ERR_WORKSPACE before anything
 *     is launched (use dedloc_round with a workspace of its own);
 *   - `stream` must belong to the current device (INVALID_ARG otherwise);
 *     the array's address on that device is looked up at the first call
 *     there (a failed lookup -> DEDLOC_ERR_HIP);
 *   - every call on one GPU shares that GPU's array, and the array needs no
 *     initialisation: calls that overlap in time on one GPU (two streams,
 *     two threads) race on it and must not be issued. */
#define DEDLOC_NOALLOC_SCRATCH_BYTES (16u << 20)
int dedloc_round_noalloc(const void *const *peer_codes, const float *const *peer_scales,
                         const uint32_t *counts, uint32_t n_peers, const uint64_t *bounds,
                         uint32_t n_shards, int32_t codec, uint32_t block, void *out_codes,
                         float *out_scales, float *x, float *m, float *v, uint64_t P,
                         const uint64_t *offsets, const uint8_t *flags, uint32_t n_tensors,
                         const dedloc_lamb_cfg *cfg, float *trust_out, float *out_mean,
                         const dedloc_local_peer *local, void *stream);

/* The same round with the LARS step (dedloc_lars_step) in place of LAMB;
 * v is the momentum buffer.  The fp16 path reads each peer byte once; pass B
 * reads the gathered message, x and v again. */
int dedloc_round_lars(const void *const *peer_codes, const float *const *peer_scales,
                      const uint32_t *counts, uint32_t n_peers, const uint64_t *bounds,
                      uint32_t n_shards, int32_t codec, uint32_t block, void *out_codes,
                      float *out_scales, float *x, float *v, uint64_t P,
                      const uint64_t *offsets, const uint8_t *flags, uint32_t n_tensors,
                      const dedloc_lars_cfg *cfg, float *trust_out, float *out_mean,
                      const dedloc_local_peer *local, void *ws, size_t ws_bytes, void *stream);

/* Group (Moshpit) all-reduce (Section 3.2 "Node failures"; Appendix C):
 * instead of one global average, peers average in groups of m = group_size
 * over d = max(1, ceil(log_m n)) consecutive iterations, so that one failing
 * peer only affects its group, and every peer holds the global average after
 * d iterations.  Grid: m^d slots, slot i holds peer i (i < n) and the others
 * are empty; in iteration k the groups are the slots whose base-m digits
 * agree except digit k (group id = slot with digit k removed).  Each member
 * carries a sample count (initially counts[i]); a group whose members carry
 * zero samples produces nothing, otherwise it computes the weighted average
 * of its members' messages exactly as dedloc_reduce_shard does (members with
 * zero samples are not read) and every member takes the encoded group
 * average and the group's total count.
 *   peer_codes / peer_scales  host arrays of n_peers device messages of len
 *                             elements (16-byte aligned);
 *   out_codes   device, n_out messages at a stride of
 *               round_up(len * code_bytes, 256) bytes (256-byte aligned);
 *   out_scales  int8 only: n_out * ceil(len/1024) floats;
 *   peer_out    host uint32[n_peers]: the output message peer i holds
 *               (0xffffffff if it holds none);  n_out (host): m^(d-1);
 *   ws          dedloc_group_allreduce_workspace_bytes() bytes, 256-byte
 *               aligned (two sets of intermediate group messages).
 * n_peers <= DEDLOC_MAX_GROUP_PEERS, 2 <= group_size <= DEDLOC_MAX_GROUP_SIZE;
 * errors as for dedloc_reduce_shard.  Each iteration takes one launch per
 * batch of up to 64 groups holding up to 64 members with samples. */
size_t dedloc_group_allreduce_workspace_bytes(uint32_t n_peers, uint32_t group_size, uint64_t len,
                                              int32_t codec, uint32_t block);
int dedloc_group_allreduce(const void *const *peer_codes, const float *const *peer_scales,
                           const uint32_t *counts, uint32_t n_peers, uint32_t group_size,
                           uint64_t len, int32_t codec, uint32_t block, void *out_codes,
                           float *out_scales, uint32_t *peer_out, uint32_t *n_out, void *ws,
                           size_t ws_bytes, void *stream);

/* Local accumulation (Section 3.1: a peer keeps summing micro-batch
 * gradients, however fast it runs, until the whole group's sample total
 * hits the global batch size).  A micro-batch
 * of batch_samples samples whose mean gradient is grad (fp32, or fp16 codes
 * with grad_codec = DEDLOC_CODEC_FP16) is added as
 *     acc[e] = fma(batch_samples, grad[e], acc[e]).
 * acc, grad: device, n elements, 16-byte aligned. */
int dedloc_accumulate(float *acc, const void *grad, int32_t grad_codec, uint64_t n,
                      float batch_samples, void *stream);

/* The sender's message at the start of a round: the peer's mean gradient
 * acc[e] / count (one correctly rounded division; count = samples
 * accumulated, in [1, 2^24]) encoded as by dedloc_encode; reset != 0 zeroes
 * acc afterwards for the next round.  count == 0 -> ZERO_WEIGHT. */
int dedloc_finalize(float *acc, uint64_t n, uint32_t count, int32_t codec, uint32_t block,
                    void *codes, float *scales, int32_t reset, void *stream);

/* Load balancer (Section 3.2, Appendix B): the relaxed linear program
 * (Eq. main_problem_appendix_relaxed) that maximises training steps per
 * second xi over the send rates a_ij (peer i -> reducer j), the return rates
 * g_ij (reducer i -> peer j) and the compute indicators c_i in [0, 1]:
 *   xi <= sum_i s_i c_i / B;   xi <= sum_j g_ji / P            (every i)
 *   g_ij <= a_ki + (1 - c_k) d_i                               (every i, j, k)
 *   sum_{j != i} (a_ji + g_ji) <= d_i;  sum_{j != i} (a_ij + g_ij) <= u_i
 *   a_ij + g_ij <= t_ij (where finite);  a, g >= 0;  0 <= c <= 1
 * solved on the host by a deterministic primal-dual interior-point method
 * (the appendix also solves it with one).  The n^3 aggregation constraints
 * are replaced by an exactly equivalent O(n^2) set with a rate variable per
 * reducer; each Newton system is reduced to a dense symmetric system of
 * about 5n unknowns (Bunch-Kaufman LDL^T).  Converged to a relative duality
 * gap of 1e-12 (an iterate within 1e-9 on every measure is accepted if
 * rounding stalls it earlier).  Equal inputs give equal outputs bit for bit.
 * Reducer i's share is proportional to min_{j != i} g_ij (the appendix's
 * "fraction" equation; the rate to itself is free).
 * Units: s in samples/s, d, u, t in parameters/s, B samples, P parameters.
 * Peers with can_aggregate[i] == 0 receive nothing to aggregate (a_ji = g_ij
 * = 0).  c_fixed (nullable, n entries): c_i is fixed to c_fixed[i] in [0, 1]
 * where it is not NaN (1 and 0 give the paper's binary choice before the
 * relaxation: the parameter-server and BytePS special cases of Section 3.2).
 * All arrays are host memory; t (n*n, row-major, INFINITY = no limit),
 * can_aggregate and c_fixed may be NULL.
 * Outputs: xi, c[n], frac[n] (sums to 1), weights[n] (nullable): frac scaled
 * to integers summing to about 2^24, ready for dedloc_partition; a[n*n] and
 * g[n*n] (nullable) in parameters/s.  n <= DEDLOC_BALANCE_MAX_PEERS.
 * Errors: NULL required arrays, n out of range, B or P not positive, a
 * negative or non-finite s, d, u, a negative or NaN t, c_fixed outside
 * [0, 1] -> INVALID_ARG; no convergence -> INVALID_ARG. */
#define DEDLOC_BALANCE_MAX_PEERS 128
typedef struct {
    uint32_t n;
    const double *s, *d, *u, *t;
    const uint8_t *can_aggregate;
    double B, P;
    const double *c_fixed;
} dedloc_balance_problem;
int dedloc_balance(const dedloc_balance_problem *pr, double *xi, double *c, double *frac,
                   uint64_t *weights, double *a, double *g);

/* Group size for dedloc_group_allreduce (Appendix C "Fault tolerance"):
 * the m in [2, min(n_peers, max_group)] that minimises the expected number
 * of iterations to the global average, counting restarts after failures:
 *     E(m) = ceil(log_m n_peers) / (1 - failure_rate)^m,
 * with failure_rate the probability that one peer fails during one group
 * attempt (a group of m succeeds only if none of its members fails, and
 * restarts otherwise).  The paper states the objective but no formula; this
 * reading reaches the two limits it does state: m = n when failures are
 * rare, m = 2 (pairs, as in decentralized SGD; Section 3.2) when they are
 * frequent.  Ties go to the smaller m.  Host-only.
 *   n_peers in [2, DEDLOC_MAX_GROUP_PEERS], 0 <= failure_rate < 1,
 *   max_group = 0 (no cap) or >= 2; otherwise INVALID_ARG.
 *   m_out: host, required; expected_out: host, nullable (E of the chosen m).
 * dedloc_group_allreduce takes groups of at most DEDLOC_MAX_GROUP_SIZE:
 * pass that as max_group to get a size it accepts. */
int dedloc_group_size(uint32_t n_peers, double failure_rate, uint32_t max_group, uint32_t *m_out,
                      double *expected_out);

/* Per-kernel timing (tracing support for benchmarks).  Between
 * dedloc_profile_begin() and dedloc_profile_end() every kernel the library
 * enqueues is bracketed by a pair of HIP events on its stream; at most
 * max_launches launches are recorded (later ones are not timed).
 * dedloc_profile_end waits for the recorded events and writes, for every
 * kernel kind k < n_kinds, the summed duration total_ms[k] (host) and the
 * launch count launches[k] (host).  Kinds are named by
 * dedloc_kernel_name(k); dedloc_kernel_kinds() gives their number.
 * Profiling is process-wide; calls from several threads are serialised. */
int dedloc_profile_begin(uint32_t max_launches);
int dedloc_profile_end(uint32_t n_kinds, double *total_ms, uint64_t *launches);
int dedloc_kernel_kinds(void);
const char *dedloc_kernel_name(int kind);

/* Test hook of the LAMB and LARS steps and rounds.  Inside the pass that
 * applies the update, one workgroup per tensor computes the tensor's trust
 * ratio and publishes it; the others poll for it at most `polls` times
 * (default 4096), then compute it themselves, in the same order, so the
 * results are the same bits for every value (0: every workgroup computes
 * it).  Process-wide, read when a call is made; returns the previous value. */
uint32_t dedloc_test_trust_polls(uint32_t polls);

#ifdef __cplusplus
}
#endif

#endif /* DEDLOC_H */
