// C ABI of libdedloc (declared in include/dedloc.h): argument validation,
// host-side integer work (shard bounds, peer weights, LAMB tile tables) and
// the launch sequence of each call.  All arithmetic on vector data runs in
// the kernels of kernels.hip.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/dedloc.h"
#include "dedloc_internal.h"

using namespace dedloc;

// The workspace of dedloc_round_noalloc.  In host code `scratch` names a
// host-side stand-in, not device memory: its device address (one per GPU)
// comes from hipGetSymbolAddress and only that address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[DEDLOC_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(DEDLOC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// ------------------------------------------------------------ profiling
enum Kind {
    K_ENCODE_FP16, K_DECODE_FP16, K_ENCODE_I8, K_DECODE_I8, K_REDUCE_FP16, K_REDUCE_I8,
    K_LAMB_A_F32, K_LAMB_A_FP16, K_LAMB_A_I8, K_LAMB_A_FUSED_FP16, K_LAMB_B,
    K_LARS_A_F32, K_LARS_A_FP16, K_LARS_A_I8, K_LARS_A_FUSED_FP16, K_LARS_B,
    K_ACCUMULATE, K_FINALIZE_FP16, K_FINALIZE_I8, K_FILL, K_COUNT
};
const char *const kKindNames[K_COUNT] = {
    "encode_fp16", "decode_fp16", "encode_i8", "decode_i8", "reduce_fp16", "reduce_i8",
    "lamb_a_f32", "lamb_a_fp16", "lamb_a_i8", "lamb_a_fused_fp16", "lamb_b",
    "lars_a_f32", "lars_a_fp16", "lars_a_i8", "lars_a_fused_fp16", "lars_b",
    "accumulate", "finalize_fp16", "finalize_i8", "fill_zero"};

struct Profiler {
    std::mutex mu;
    bool on = false;
    uint32_t cap = 0;
    std::vector<hipEvent_t> ev;     // 2 per recorded launch
    std::vector<int> kind;
    size_t used = 0;
} g_prof;

// Run `launch` (returning hipError_t), bracketed by events when profiling.
template <typename F>
hipError_t timed(int kind, hipStream_t s, F launch) {
    std::unique_lock<std::mutex> lk(g_prof.mu);
    if (!g_prof.on || g_prof.used >= g_prof.cap) {
        lk.unlock();
        return launch();
    }
    const size_t i = g_prof.used++;
    while (g_prof.ev.size() < 2 * g_prof.used) {
        hipEvent_t e;
        hipError_t r = hipEventCreate(&e);
        if (r != hipSuccess) return r;
        g_prof.ev.push_back(e);
    }
    g_prof.kind.resize(g_prof.used);
    g_prof.kind[i] = kind;
    hipError_t r = hipEventRecord(g_prof.ev[2 * i], s);
    if (r != hipSuccess) return r;
    r = launch();
    if (r != hipSuccess) return r;
    return hipEventRecord(g_prof.ev[2 * i + 1], s);
}

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Host copy of dedloc_weights' definition: exact integer total, exactly
// converted, one fp32 division per peer.
int compute_weights(const uint32_t *counts, uint32_t n, float *w) {
    uint64_t W = 0;
    for (uint32_t p = 0; p < n; p++) W += counts[p];
    if (W == 0) return fail(DEDLOC_ERR_ZERO_WEIGHT, "every peer has zero samples");
    if (W > (1u << 24)) return fail(DEDLOC_ERR_INVALID_ARG, "total sample count %llu exceeds 2^24",
                                    (unsigned long long)W);
    for (uint32_t p = 0; p < n; p++) w[p] = (float)counts[p] / (float)W;
    return DEDLOC_OK;
}

int check_codec(int32_t codec, uint32_t block, bool allow_f32) {
    if (codec == DEDLOC_CODEC_FP16) return DEDLOC_OK;
    if (codec == DEDLOC_CODEC_F32 && allow_f32) return DEDLOC_OK;
    if (codec == DEDLOC_CODEC_I8) {
        if (block != DEDLOC_I8_BLOCK)
            return fail(DEDLOC_ERR_INVALID_ARG, "int8 block must be %d (got %u)", DEDLOC_I8_BLOCK, block);
        return DEDLOC_OK;
    }
    return fail(DEDLOC_ERR_INVALID_ARG, "unknown codec %d", codec);
}

static_assert(DEDLOC_MAX_GROUP_SIZE <= kMaxPeers, "a group must fit one launch's peer table");

// Active peers: those with counts > 0, in ascending order, with weights.
struct PeerList {
    std::vector<const void *> codes;
    std::vector<const float *> scales;
    std::vector<float> w;
    std::vector<uint32_t> index;  // the caller's peer index
    uint32_t n() const { return (uint32_t)w.size(); }
};

int build_peers(const void *const *codes, const float *const *scales, const uint32_t *counts,
                uint32_t n, int32_t codec, PeerList &pl, bool check_ptrs = true) {
    if (!codes || !counts) return fail(DEDLOC_ERR_INVALID_ARG, "peer_codes and counts must not be NULL");
    if (n == 0 || n > DEDLOC_MAX_PEERS)
        return fail(DEDLOC_ERR_INVALID_ARG, "n_peers must be in [1, %d] (got %u)", DEDLOC_MAX_PEERS, n);
    if (codec == DEDLOC_CODEC_I8 && !scales)
        return fail(DEDLOC_ERR_INVALID_ARG, "int8 messages need peer_scales");
    std::vector<float> w(n);
    int rc = compute_weights(counts, n, w.data());
    if (rc) return rc;
    pl = PeerList();
    if (!check_ptrs) return DEDLOC_OK;  // nothing will be read at all
    for (uint32_t p = 0; p < n; p++) {
        if (counts[p] == 0) continue;  // weight 0: never read
        if (!codes[p]) return fail(DEDLOC_ERR_INVALID_ARG, "peer %u has samples but a NULL message", p);
        if (!aligned(codes[p], 16)) return fail(DEDLOC_ERR_ALIGN, "peer %u message is not 16-byte aligned", p);
        const float *sc = nullptr;
        if (codec == DEDLOC_CODEC_I8) {
            if (!scales[p]) return fail(DEDLOC_ERR_INVALID_ARG, "peer %u has samples but NULL scales", p);
            if (!aligned(scales[p], 4)) return fail(DEDLOC_ERR_ALIGN, "peer %u scales not 4-byte aligned", p);
            sc = scales[p];
        }
        pl.codes.push_back(codes[p]);
        pl.scales.push_back(sc);
        pl.w.push_back(w[p]);
        pl.index.push_back(p);
    }
    return DEDLOC_OK;
}

// Active peers [lo, hi) as one launch's table (hi - lo <= kMaxPeers).
PeerTable table_of(const PeerList &pl, uint32_t lo, uint32_t hi) {
    PeerTable pt;
    memset(&pt, 0, sizeof pt);
    for (uint32_t p = lo; p < hi; p++) {
        pt.codes[pt.n] = pl.codes[p];
        pt.scales[pt.n] = pl.scales[p];
        pt.w[pt.n] = pl.w[p];
        pt.n++;
    }
    return pt;
}

// A plain reduce: every peer of the table in one group writing `out`.
GroupTable single_group(const PeerTable &pt, void *out, float *out_scales) {
    GroupTable gt;
    memset(&gt, 0, sizeof gt);
    gt.pt = pt;
    gt.gbegin[0] = 0;
    gt.gbegin[1] = pt.n;
    gt.out[0] = out;
    gt.out_scales[0] = out_scales;
    gt.n_groups = 1;
    return gt;
}

// More active peers than one launch's table holds need the fp32 mean buffer
// to carry the running sum between launches.
int check_chain(const PeerList &pl, const float *mean) {
    if (pl.n() > (uint32_t)kMaxPeers && !mean)
        return fail(DEDLOC_ERR_INVALID_ARG, "%u peers with samples (more than %d) need out_mean", pl.n(), kMaxPeers);
    return DEDLOC_OK;
}

// Start of the last launch's peers when peers [0, n) are reduced in
// launches of kMaxPeers.
uint32_t last_batch(uint32_t n) { return n == 0 ? 0 : (n - 1) / kMaxPeers * kMaxPeers; }

// The local peer as seen by a launch of active peers [a, b): its position
// relative to a, or -1 if the launch does not hold it.
LocalArgs local_in(const LocalArgs &la, uint32_t a, uint32_t b) {
    LocalArgs r = la;
    r.pos = (la.pos >= 0 && (uint32_t)la.pos >= a && (uint32_t)la.pos < b) ? la.pos - (int32_t)a : -1;
    return r;
}

// Reduce peers [lo, hi) of the list in launches of kMaxPeers, chained through
// `mean`; the launch holding peer hi - 1 encodes into out / out_scales when
// `encode` is set.  Peers before lo must already be summed into `mean`.
// la.pos: the local peer's position in the list (-1: none; fp16 only).
int run_reduce(int32_t codec, const PeerList &pl, uint32_t lo, uint32_t hi, bool encode, uint64_t len,
               void *out, float *out_scales, float *mean, const LocalArgs &la, hipStream_t s) {
    for (uint32_t a = lo; a < hi; a += kMaxPeers) {
        const uint32_t b = std::min(hi, a + (uint32_t)kMaxPeers);
        const GroupTable gt = single_group(table_of(pl, a, b), out, out_scales);
        const ChainArgs ca = {a > 0 ? mean : nullptr, mean, encode && b == hi, local_in(la, a, b)};
        const hipError_t e = codec == DEDLOC_CODEC_FP16
                                 ? timed(K_REDUCE_FP16, s, [&] { return launch_reduce_fp16(gt, len, ca, s); })
                                 : timed(K_REDUCE_I8, s, [&] { return launch_reduce_i8(gt, len, ca, s); });
        if (e != hipSuccess) return hip_fail(e, "reduce launch");
    }
    return DEDLOC_OK;
}

// LAMB tile table: tensors in launch chunks of at most kChunkTensors.
struct Plan {
    std::vector<Chunk> chunks;
    std::vector<uint32_t> chunk_tiles;
    uint32_t n_tiles = 0;
    size_t ws_partials = 0, ws_trust = 0, ws_epoch = 0, ws_total = 0;
};

int check_tensors(uint64_t P, const uint64_t *off, uint32_t T) {
    if (!off) return fail(DEDLOC_ERR_INVALID_ARG, "offsets must not be NULL");
    if (T == 0) return fail(DEDLOC_ERR_INVALID_ARG, "n_tensors must be >= 1");
    if (off[0] != 0 || off[T] != P)
        return fail(DEDLOC_ERR_INVALID_ARG, "tensor offsets must start at 0 and end at P");
    for (uint32_t t = 0; t < T; t++) {
        if (off[t + 1] < off[t]) return fail(DEDLOC_ERR_INVALID_ARG, "tensor offsets decrease at %u", t);
        if (off[t] % kVec) return fail(DEDLOC_ERR_ALIGN, "tensor offset %u is not a multiple of 8", t);
        if (off[t + 1] - off[t] >= (1ull << 32))
            return fail(DEDLOC_ERR_INVALID_ARG, "tensor %u has 2^32 or more elements", t);
    }
    return DEDLOC_OK;
}

void make_plan(uint64_t P, const uint64_t *off, const uint8_t *flags, uint32_t T, Plan &pl) {
    (void)P;
    pl.chunks.clear();
    pl.chunk_tiles.clear();
    uint32_t base_tile = 0;
    uint32_t t0 = 0;
    while (t0 < T) {
        Chunk c;
        memset(&c, 0, sizeof c);
        c.base = off[t0];
        c.t0 = t0;
        c.tile_base = base_tile;
        uint32_t tiles = 0, k = 0;
        // take tensors while they fit the table and the chunk spans < 2^32 elements
        while (k < (uint32_t)kChunkTensors && t0 + k < T && off[t0 + k + 1] - c.base < (1ull << 32)) {
            c.start[k] = (uint32_t)(off[t0 + k] - c.base);
            c.tile_begin[k] = tiles;
            c.flags[k] = flags ? flags[t0 + k] : 0;
            const uint64_t len = off[t0 + k + 1] - off[t0 + k];
            tiles += (uint32_t)((len + kTile - 1) / kTile);
            k++;
        }
        if (k == 0) k = 1;  // unreachable: every tensor was checked to span < 2^32 elements
        c.nt = k;
        c.start[k] = (uint32_t)(off[t0 + k] - c.base);
        c.tile_begin[k] = tiles;
        pl.chunks.push_back(c);
        pl.chunk_tiles.push_back(tiles);
        base_tile += tiles;
        t0 += k;
    }
    pl.n_tiles = base_tile;
    pl.ws_partials = round_up((size_t)base_tile * 2 * sizeof(double), 256);
    pl.ws_trust = round_up((size_t)T * sizeof(unsigned long long), 256);
    pl.ws_epoch = 256;
    pl.ws_total = pl.ws_partials + pl.ws_trust + pl.ws_epoch;
}

LambWs carve(const Plan &pl, void *ws) {
    char *b = (char *)ws;
    LambWs w;
    w.partials = (double *)b;
    w.trust = (unsigned long long *)(b + pl.ws_partials);
    w.epoch = (uint32_t *)(b + pl.ws_partials + pl.ws_trust);
    return w;
}

// Polls of a tensor's published trust ratio in pass B before a workgroup
// computes it itself (dedloc_test_trust_polls).
std::atomic<uint32_t> g_trust_polls{4096};

int lamb_params(const dedloc_lamb_cfg *cfg, OptParams &op) {
    if (!cfg) return fail(DEDLOC_ERR_INVALID_ARG, "cfg must not be NULL");
    if (cfg->step == 0) return fail(DEDLOC_ERR_INVALID_ARG, "step must be >= 1");
    memset(&op, 0, sizeof op);
    op.lr = cfg->lr;
    op.wd = cfg->weight_decay;
    op.beta1 = cfg->beta1;
    op.beta2 = cfg->beta2;
    op.omb1 = 1.0f - cfg->beta1;
    op.omb2 = 1.0f - cfg->beta2;
    op.c1 = 1.0f;
    op.c2 = 1.0f;
    if (cfg->bias_correction) {
        op.c1 = (float)(1.0 - pow((double)cfg->beta1, (double)cfg->step));
        op.c2 = (float)(1.0 - pow((double)cfg->beta2, (double)cfg->step));
    }
    op.eps = cfg->eps;
    op.unit_trust = cfg->force_unit_trust ? 1 : 0;
    op.trust_polls = g_trust_polls.load(std::memory_order_relaxed);
    return DEDLOC_OK;
}

int lars_params(const dedloc_lars_cfg *cfg, OptParams &op) {
    if (!cfg) return fail(DEDLOC_ERR_INVALID_ARG, "cfg must not be NULL");
    memset(&op, 0, sizeof op);
    op.lr = cfg->lr;
    op.wd = cfg->weight_decay;
    op.momentum = cfg->momentum;
    op.trust_coef = cfg->trust_coef;
    op.unit_trust = cfg->force_unit_trust ? 1 : 0;
    op.trust_polls = g_trust_polls.load(std::memory_order_relaxed);
    return DEDLOC_OK;
}

// x and the optimizer state (m and v for LAMB, the momentum v for LARS).
// An empty vector (P == 0) reads and writes no element: its buffers may be
// NULL; only the workspace (the per-tensor ratios) is used.
// ws == kNoWs: the caller brings no workspace (the static array is used;
// its size is checked by the caller of this function).
void *const kNoWs = nullptr;

int check_state(int opt, float *x, float *m, float *v, uint64_t P, void *ws, size_t ws_bytes, const Plan &pl,
                bool check_ws = true) {
    if (P > 0 && (!x || !v || (opt == kOptLamb && !m)))
        return fail(DEDLOC_ERR_INVALID_ARG, "parameter and state buffers must not be NULL");
    if (!aligned(x, 16) || !aligned(v, 16) || (m && !aligned(m, 16)))
        return fail(DEDLOC_ERR_ALIGN, "parameter and state buffers must be 16-byte aligned");
    if (!check_ws) return DEDLOC_OK;
    if (!ws || ws_bytes < pl.ws_total)
        return fail(DEDLOC_ERR_WORKSPACE, "workspace of %zu bytes needed (got %zu)", pl.ws_total,
                    ws ? ws_bytes : (size_t)0);
    if (!aligned(ws, 256)) return fail(DEDLOC_ERR_ALIGN, "workspace must be 256-byte aligned");
    return DEDLOC_OK;
}

int grad_src(int32_t codec) {
    return codec == DEDLOC_CODEC_F32 ? kSrcF32 : codec == DEDLOC_CODEC_FP16 ? kSrcFP16 : kSrcI8;
}

// The host's part of the tag of a call's published trust ratios (pass B
// adds the workspace counter that pass A advances): a process-wide
// sequence with a start drawn from the clock and the process id, so that
// workspace contents left by anything else are unlikely to carry it.
uint32_t next_nonce() {
    static std::atomic<uint32_t> ctr{(uint32_t)std::chrono::steady_clock::now().time_since_epoch().count() * 2654435761u ^
                                     (uint32_t)getpid()};
    return ctr.fetch_add(0x9E3779B9u, std::memory_order_relaxed);
}

// Per chunk of tensors: pass A (gradient from src_a) and pass B, which
// computes the trust ratios (LARS reads the gradient again from src_b).
int run_opt(int opt, int src_a, int src_b, const Plan &pl, const PeerTable *pt, const GradArgs &ga_a,
            const GradArgs &ga_b, const OptParams &op, float *x, float *m, float *v, void *ws,
            float *trust_out, hipStream_t s) {
    const LambWs w = carve(pl, ws);
    const int k_a = (opt == kOptLamb ? K_LAMB_A_F32 : K_LARS_A_F32) + std::min(src_a, (int)kSrcPeersFP16);
    const int k_b = opt == kOptLamb ? K_LAMB_B : K_LARS_B;
    const uint32_t nonce = next_nonce();
    for (size_t c = 0; c < pl.chunks.size(); c++) {
        const Chunk &ch = pl.chunks[c];
        const uint32_t tiles = pl.chunk_tiles[c];
        hipError_t e = timed(k_a, s, [&] { return launch_opt_a(opt, src_a, ch, tiles, pt, ga_a, op, x, m, v, w, s); });
        if (e != hipSuccess) return hip_fail(e, "optimizer pass A launch");
        e = timed(k_b, s, [&] {
            return launch_opt_b(opt, src_b, ch, tiles, ga_b, op, x, m, v, w, nonce, trust_out, s);
        });
        if (e != hipSuccess) return hip_fail(e, "optimizer pass B launch");
    }
    return DEDLOC_OK;
}

// Validation shared by the LAMB and LARS steps.
int prepare_step(int opt, float *x, float *m, float *v, const void *grad, const float *grad_scales,
                 int32_t grad_codec, uint32_t block, uint64_t P, const uint64_t *offsets,
                 const uint8_t *flags, uint32_t n_tensors, void *ws, size_t ws_bytes, Plan &pl) {
    int rc = check_codec(grad_codec, block, true);
    if (rc) return rc;
    rc = check_tensors(P, offsets, n_tensors);
    if (rc) return rc;
    if (!flags) return fail(DEDLOC_ERR_INVALID_ARG, "flags must not be NULL");
    make_plan(P, offsets, flags, n_tensors, pl);
    rc = check_state(opt, x, m, v, P, ws, ws_bytes, pl);
    if (rc) return rc;
    if (P == 0) return DEDLOC_OK;
    if (!grad || !aligned(grad, 16)) return fail(DEDLOC_ERR_ALIGN, "grad must be non-NULL and 16-byte aligned");
    if (grad_codec == DEDLOC_CODEC_I8 && (!grad_scales || !aligned(grad_scales, 4)))
        return fail(DEDLOC_ERR_INVALID_ARG, "int8 gradient needs aligned grad_scales");
    return DEDLOC_OK;
}

// Validation shared by the LAMB and LARS rounds.
int prepare_round(int opt, const void *const *peer_codes, const float *const *peer_scales,
                  const uint32_t *counts, uint32_t n_peers, const uint64_t *bounds, uint32_t n_shards,
                  int32_t codec, uint32_t block, void *out_codes, float *out_scales, float *x, float *m,
                  float *v, uint64_t P, const uint64_t *offsets, const uint8_t *flags, uint32_t n_tensors,
                  float *out_mean, const dedloc_local_peer *local, void *ws, size_t ws_bytes,
                  PeerList &peers, Plan &pl, LocalArgs &la, bool check_ws = true) {
    int rc = check_codec(codec, block, false);
    if (rc) return rc;
    rc = build_peers(peer_codes, peer_scales, counts, n_peers, codec, peers, P > 0);
    if (rc) return rc;
    la = LocalArgs{-1, nullptr, nullptr, nullptr};
    if (local) {
        if (local->index >= n_peers || counts[local->index] == 0)
            return fail(DEDLOC_ERR_INVALID_ARG, "the local peer must be one of the peers and hold samples");
        if (P > 0 && (!local->grad || !aligned(local->grad, 16)))
            return fail(DEDLOC_ERR_ALIGN, "the local gradient must be non-NULL and 16-byte aligned");
        for (uint32_t k = 0; k < peers.n(); k++)
            if (peers.index[k] == local->index) la.pos = (int32_t)k;
        la.grad = local->grad;
        la.codes = const_cast<void *>(peer_codes[local->index]);
        la.scales = codec == DEDLOC_CODEC_I8 ? const_cast<float *>(peer_scales[local->index]) : nullptr;
    }
    if (!bounds || n_shards == 0) return fail(DEDLOC_ERR_INVALID_ARG, "bounds must list n_shards >= 1 shards");
    if (bounds[0] != 0 || bounds[n_shards] != P) return fail(DEDLOC_ERR_INVALID_ARG, "shard bounds must tile [0, P)");
    for (uint32_t k = 0; k < n_shards; k++) {
        if (bounds[k + 1] < bounds[k]) return fail(DEDLOC_ERR_INVALID_ARG, "shard bounds decrease at %u", k);
        if (codec == DEDLOC_CODEC_I8 && k > 0 && bounds[k] % block)
            return fail(DEDLOC_ERR_INVALID_ARG, "int8 shard bound %u is not a multiple of the block", k);
    }
    rc = check_tensors(P, offsets, n_tensors);
    if (rc) return rc;
    if (!flags) return fail(DEDLOC_ERR_INVALID_ARG, "flags must not be NULL");
    make_plan(P, offsets, flags, n_tensors, pl);
    rc = check_state(opt, x, m, v, P, ws, ws_bytes, pl, check_ws);
    if (rc) return rc;
    if (P == 0) return DEDLOC_OK;
    if (!out_codes || !aligned(out_codes, 16)) return fail(DEDLOC_ERR_ALIGN, "out_codes must be non-NULL and 16-byte aligned");
    if (out_mean && !aligned(out_mean, 16)) return fail(DEDLOC_ERR_ALIGN, "out_mean must be 16-byte aligned");
    if (codec == DEDLOC_CODEC_I8 && (!out_scales || !aligned(out_scales, 4)))
        return fail(DEDLOC_ERR_INVALID_ARG, "int8 round needs aligned out_scales");
    return check_chain(peers, out_mean);
}

// The round after validation: the reduce-scatter and gather, then the
// optimizer.  fp16: the codec is elementwise, so every shard's average is the
// same function of the element index and pass A fuses the average of all
// shards (of the last launch's peers, after the earlier ones are summed into
// out_mean).  int8: interior shard bounds sit on block boundaries, so every
// shard's blocks are the vector's blocks and one reduce covers all shards
// before the optimizer reads the gathered message.
int run_round(int opt, const PeerList &peers, int32_t codec, void *out_codes, float *out_scales, float *x,
              float *m, float *v, uint64_t P, const Plan &pl, const OptParams &op, float *trust_out,
              float *out_mean, const LocalArgs &la, void *ws, hipStream_t s) {
    const LocalArgs none = {-1, nullptr, nullptr, nullptr};
    const GradArgs gathered = {out_codes, out_scales, nullptr, nullptr, nullptr, none};
    if (codec == DEDLOC_CODEC_FP16) {
        const uint32_t n = peers.n(), f = last_batch(n);
        int rc = run_reduce(codec, peers, 0, f, false, P, out_codes, nullptr, out_mean, la, s);
        if (rc) return rc;
        const PeerTable pt = table_of(peers, f, n);
        const GradArgs fused = {nullptr, nullptr, (uint16_t *)out_codes, out_mean, out_mean, local_in(la, f, n)};
        const int src = f > 0 ? kSrcPeersFP16Chain : fused.local.pos >= 0 ? kSrcPeersFP16Local : kSrcPeersFP16;
        return run_opt(opt, src, kSrcFP16, pl, &pt, fused, gathered, op, x, m, v, ws, trust_out, s);
    }
    // int8: the local peer's encode stays a launch of its own (folded into
    // the reduce it costs more than it saves: the block encode's wave-wide
    // maximum and divisions lengthen every wave of the reduce)
    if (la.pos >= 0) {
        const hipError_t e = timed(K_ENCODE_I8, s, [&] {
            return launch_encode_i8(la.grad, P, (int8_t *)la.codes, la.scales, s);
        });
        if (e != hipSuccess) return hip_fail(e, "encode launch");
    }
    int rc = run_reduce(codec, peers, 0, peers.n(), true, P, out_codes, out_scales, out_mean, none, s);
    if (rc) return rc;
    return run_opt(opt, kSrcI8, kSrcI8, pl, nullptr, gathered, gathered, op, x, m, v, ws, trust_out, s);
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // device address of `scratch` per device (null: not looked up yet)

// The address of this GPU's static scratch array: the current device, which
// `stream` must belong to.  Looked up once per device.
int noalloc_scratch(hipStream_t stream, void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(DEDLOC_ERR_INVALID_ARG, "device %d is beyond %d", dev, kMaxDevices);
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
    if (sdev != dev)
        return fail(DEDLOC_ERR_INVALID_ARG, "the stream belongs to device %d, the current device is %d", (int)sdev, dev);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p || !aligned(p, 256)) return fail(DEDLOC_ERR_HIP, "the static scratch array has no usable address");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return DEDLOC_OK;
}

// Group all-reduce layout: m^d slots, m^(d-1) groups per iteration, every
// group message at a 256-byte stride.
struct GroupPlan {
    uint32_t d = 0, slots = 0, groups = 0;
    size_t code_stride = 0, scale_stride = 0;   // bytes, floats
    size_t ws_codes = 0, ws_total = 0;          // two ping-pong sets of group messages
};

int group_plan(uint32_t n, uint32_t m, uint64_t len, int32_t codec, GroupPlan &gp) {
    if (n == 0 || n > DEDLOC_MAX_GROUP_PEERS)
        return fail(DEDLOC_ERR_INVALID_ARG, "n_peers must be in [1, %d]", DEDLOC_MAX_GROUP_PEERS);
    if (m < 2 || m > DEDLOC_MAX_GROUP_SIZE) return fail(DEDLOC_ERR_INVALID_ARG, "group_size must be in [2, %d]", DEDLOC_MAX_GROUP_SIZE);
    uint32_t d = 1;
    uint64_t slots = m;
    while (slots < n) {
        slots *= m;
        d++;
    }
    gp.d = d;
    gp.slots = (uint32_t)slots;
    gp.groups = (uint32_t)(slots / m);
    const size_t cb = codec == DEDLOC_CODEC_FP16 ? 2 : 1;
    gp.code_stride = round_up((size_t)len * cb, 256);
    gp.scale_stride = codec == DEDLOC_CODEC_I8 ? (size_t)((len + DEDLOC_I8_BLOCK - 1) / DEDLOC_I8_BLOCK) : 0;
    const size_t d_prev = d > 1 ? 2 : 0;  // iterations before the last ping-pong between two sets
    gp.ws_codes = d_prev * gp.groups * gp.code_stride;
    gp.ws_total = gp.ws_codes + round_up(d_prev * gp.groups * gp.scale_stride * sizeof(float), 256);
    return DEDLOC_OK;
}

}  // namespace

extern "C" {

int dedloc_version(void) { return 100; }

const char *dedloc_last_error(void) { return g_err.c_str(); }

size_t dedloc_encoded_bytes(int32_t codec, uint32_t block, uint64_t n, uint64_t *n_scales) {
    if (n_scales) *n_scales = 0;
    if (codec == DEDLOC_CODEC_FP16) return (size_t)n * 2;
    if (codec == DEDLOC_CODEC_I8 && block > 0) {
        if (n_scales) *n_scales = (n + block - 1) / block;
        return (size_t)n;
    }
    if (codec == DEDLOC_CODEC_F32) return (size_t)n * 4;
    return 0;
}

int dedloc_partition(uint64_t P, uint32_t n_shards, const uint64_t *weights, uint32_t align,
                     uint64_t *bounds) {
    if (!bounds) return fail(DEDLOC_ERR_INVALID_ARG, "bounds must not be NULL");
    if (n_shards == 0 || align == 0) return fail(DEDLOC_ERR_INVALID_ARG, "n_shards and align must be > 0");
    unsigned __int128 total = 0;
    for (uint32_t k = 0; k < n_shards; k++) total += weights ? weights[k] : 1;
    if (total == 0) return fail(DEDLOC_ERR_INVALID_ARG, "all shard weights are zero");
    const unsigned __int128 denom = total * align;
    unsigned __int128 c = 0;
    bounds[0] = 0;
    for (uint32_t k = 1; k < n_shards; k++) {
        c += weights ? weights[k - 1] : 1;
        bounds[k] = (uint64_t)(((unsigned __int128)P * c / denom) * align);
    }
    bounds[n_shards] = P;
    return DEDLOC_OK;
}

int dedloc_weights(const uint32_t *counts, uint32_t n, float *w) {
    if (!counts || !w || n == 0) return fail(DEDLOC_ERR_INVALID_ARG, "counts/w must be non-NULL, n > 0");
    return compute_weights(counts, n, w);
}

int dedloc_encode(const float *x, uint64_t n, int32_t codec, uint32_t block, void *codes,
                  float *scales, void *stream) {
    int rc = check_codec(codec, block, false);
    if (rc) return rc;
    if (n == 0) return DEDLOC_OK;
    if (!x || !codes) return fail(DEDLOC_ERR_INVALID_ARG, "x and codes must not be NULL");
    if (!aligned(x, 16) || !aligned(codes, 16)) return fail(DEDLOC_ERR_ALIGN, "x and codes must be 16-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (codec == DEDLOC_CODEC_FP16) {
        e = timed(K_ENCODE_FP16, s, [&] { return launch_encode_fp16(x, n, (uint16_t *)codes, s); });
    } else {
        if (!scales) return fail(DEDLOC_ERR_INVALID_ARG, "int8 encode needs scales");
        if (!aligned(scales, 4)) return fail(DEDLOC_ERR_ALIGN, "scales must be 4-byte aligned");
        e = timed(K_ENCODE_I8, s, [&] { return launch_encode_i8(x, n, (int8_t *)codes, scales, s); });
    }
    return e == hipSuccess ? DEDLOC_OK : hip_fail(e, "encode launch");
}

int dedloc_decode(const void *codes, const float *scales, uint64_t n, int32_t codec, uint32_t block,
                  float *out, void *stream) {
    int rc = check_codec(codec, block, false);
    if (rc) return rc;
    if (n == 0) return DEDLOC_OK;
    if (!codes || !out) return fail(DEDLOC_ERR_INVALID_ARG, "codes and out must not be NULL");
    if (!aligned(out, 16) || !aligned(codes, 16)) return fail(DEDLOC_ERR_ALIGN, "codes and out must be 16-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (codec == DEDLOC_CODEC_FP16) {
        e = timed(K_DECODE_FP16, s, [&] { return launch_decode_fp16((const uint16_t *)codes, n, out, s); });
    } else {
        if (!scales) return fail(DEDLOC_ERR_INVALID_ARG, "int8 decode needs scales");
        if (!aligned(scales, 4)) return fail(DEDLOC_ERR_ALIGN, "scales must be 4-byte aligned");
        e = timed(K_DECODE_I8, s, [&] { return launch_decode_i8((const int8_t *)codes, scales, n, out, s); });
    }
    return e == hipSuccess ? DEDLOC_OK : hip_fail(e, "decode launch");
}

int dedloc_reduce_shard(const void *const *peer_codes, const float *const *peer_scales,
                        const uint32_t *counts, uint32_t n_peers, uint64_t shard_len, int32_t codec,
                        uint32_t block, void *out_codes, float *out_scales, float *out_mean,
                        void *stream) {
    int rc = check_codec(codec, block, false);
    if (rc) return rc;
    PeerList peers;
    rc = build_peers(peer_codes, peer_scales, counts, n_peers, codec, peers, shard_len > 0);
    if (rc) return rc;
    if (shard_len == 0) return DEDLOC_OK;
    if (!out_codes || !aligned(out_codes, 16)) return fail(DEDLOC_ERR_ALIGN, "out_codes must be non-NULL and 16-byte aligned");
    if (out_mean && !aligned(out_mean, 16)) return fail(DEDLOC_ERR_ALIGN, "out_mean must be 16-byte aligned");
    if (codec == DEDLOC_CODEC_I8 && (!out_scales || !aligned(out_scales, 4)))
        return fail(DEDLOC_ERR_INVALID_ARG, "int8 reduce needs aligned out_scales");
    rc = check_chain(peers, out_mean);
    if (rc) return rc;
    const LocalArgs none = {-1, nullptr, nullptr, nullptr};
    return run_reduce(codec, peers, 0, peers.n(), true, shard_len, out_codes, out_scales, out_mean, none,
                      (hipStream_t)stream);
}

size_t dedloc_lamb_workspace_bytes(uint64_t P, const uint64_t *offsets, uint32_t n_tensors) {
    if (check_tensors(P, offsets, n_tensors)) return 0;
    Plan pl;
    make_plan(P, offsets, nullptr, n_tensors, pl);
    return pl.ws_total;
}

int dedloc_workspace_clear(void *ws, size_t ws_bytes, void *stream) {
    if (!ws || !aligned(ws, 4)) return fail(DEDLOC_ERR_INVALID_ARG, "workspace must be non-NULL and 4-byte aligned");
    if (ws_bytes % 4) return fail(DEDLOC_ERR_INVALID_ARG, "ws_bytes must be a multiple of 4 (got %zu)", ws_bytes);
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = timed(K_FILL, s, [&] { return launch_fill_zero(ws, ws_bytes, s); });
    return e == hipSuccess ? DEDLOC_OK : hip_fail(e, "workspace clear launch");
}

int dedloc_lamb_step(float *x, float *m, float *v, const void *grad, const float *grad_scales,
                     int32_t grad_codec, uint32_t block, uint64_t P, const uint64_t *offsets,
                     const uint8_t *flags, uint32_t n_tensors, const dedloc_lamb_cfg *cfg,
                     float *trust_out, void *ws, size_t ws_bytes, void *stream) {
    OptParams op;
    int rc = lamb_params(cfg, op);
    if (rc) return rc;
    Plan pl;
    rc = prepare_step(kOptLamb, x, m, v, grad, grad_scales, grad_codec, block, P, offsets, flags, n_tensors,
                      ws, ws_bytes, pl);
    if (rc) return rc;
    const GradArgs ga = {grad, grad_scales, nullptr, nullptr, nullptr, {-1, nullptr, nullptr, nullptr}};
    const int src = grad_src(grad_codec);
    return run_opt(kOptLamb, src, src, pl, nullptr, ga, ga, op, x, m, v, ws, trust_out, (hipStream_t)stream);
}

int dedloc_lars_step(float *x, float *v, const void *grad, const float *grad_scales, int32_t grad_codec,
                     uint32_t block, uint64_t P, const uint64_t *offsets, const uint8_t *flags,
                     uint32_t n_tensors, const dedloc_lars_cfg *cfg, float *trust_out, void *ws,
                     size_t ws_bytes, void *stream) {
    OptParams op;
    int rc = lars_params(cfg, op);
    if (rc) return rc;
    Plan pl;
    rc = prepare_step(kOptLars, x, nullptr, v, grad, grad_scales, grad_codec, block, P, offsets, flags,
                      n_tensors, ws, ws_bytes, pl);
    if (rc) return rc;
    const GradArgs ga = {grad, grad_scales, nullptr, nullptr, nullptr, {-1, nullptr, nullptr, nullptr}};
    const int src = grad_src(grad_codec);
    return run_opt(kOptLars, src, src, pl, nullptr, ga, ga, op, x, nullptr, v, ws, trust_out, (hipStream_t)stream);
}

int dedloc_round(const void *const *peer_codes, const float *const *peer_scales, const uint32_t *counts,
                 uint32_t n_peers, const uint64_t *bounds, uint32_t n_shards, int32_t codec, uint32_t block,
                 void *out_codes, float *out_scales, float *x, float *m, float *v, uint64_t P,
                 const uint64_t *offsets, const uint8_t *flags, uint32_t n_tensors,
                 const dedloc_lamb_cfg *cfg, float *trust_out, float *out_mean, const dedloc_local_peer *local,
                 void *ws, size_t ws_bytes, void *stream) {
    OptParams op;
    int rc = lamb_params(cfg, op);
    if (rc) return rc;
    PeerList peers;
    Plan pl;
    LocalArgs la;
    rc = prepare_round(kOptLamb, peer_codes, peer_scales, counts, n_peers, bounds, n_shards, codec, block,
                       out_codes, out_scales, x, m, v, P, offsets, flags, n_tensors, out_mean, local, ws, ws_bytes,
                       peers, pl, la);
    if (rc) return rc;
    return run_round(kOptLamb, peers, codec, out_codes, out_scales, x, m, v, P, pl, op, trust_out, out_mean, la,
                     ws, (hipStream_t)stream);
}

int dedloc_round_noalloc(const void *const *peer_codes, const float *const *peer_scales, const uint32_t *counts,
                         uint32_t n_peers, const uint64_t *bounds, uint32_t n_shards, int32_t codec, uint32_t block,
                         void *out_codes, float *out_scales, float *x, float *m, float *v, uint64_t P,
                         const uint64_t *offsets, const uint8_t *flags, uint32_t n_tensors,
                         const dedloc_lamb_cfg *cfg, float *trust_out, float *out_mean,
                         const dedloc_local_peer *local, void *stream) {
    OptParams op;
    int rc = lamb_params(cfg, op);
    if (rc) return rc;
    PeerList peers;
    Plan pl;
    LocalArgs la;
    rc = prepare_round(kOptLamb, peer_codes, peer_scales, counts, n_peers, bounds, n_shards, codec, block,
                       out_codes, out_scales, x, m, v, P, offsets, flags, n_tensors, out_mean, local, kNoWs, 0,
                       peers, pl, la, /*check_ws=*/false);
    if (rc) return rc;
    if (pl.ws_total > DEDLOC_NOALLOC_SCRATCH_BYTES)
        return fail(DEDLOC_ERR_WORKSPACE,
                    "this tensor table needs %zu bytes of workspace, more than the %u of the static scratch array "
                    "(call dedloc_round with a workspace)", pl.ws_total, (unsigned)DEDLOC_NOALLOC_SCRATCH_BYTES);
    void *ws = nullptr;
    rc = noalloc_scratch((hipStream_t)stream, &ws);
    if (rc) return rc;
    return run_round(kOptLamb, peers, codec, out_codes, out_scales, x, m, v, P, pl, op, trust_out, out_mean, la,
                     ws, (hipStream_t)stream);
}

int dedloc_round_lars(const void *const *peer_codes, const float *const *peer_scales, const uint32_t *counts,
                      uint32_t n_peers, const uint64_t *bounds, uint32_t n_shards, int32_t codec,
                      uint32_t block, void *out_codes, float *out_scales, float *x, float *v, uint64_t P,
                      const uint64_t *offsets, const uint8_t *flags, uint32_t n_tensors,
                      const dedloc_lars_cfg *cfg, float *trust_out, float *out_mean,
                      const dedloc_local_peer *local, void *ws, size_t ws_bytes, void *stream) {
    OptParams op;
    int rc = lars_params(cfg, op);
    if (rc) return rc;
    PeerList peers;
    Plan pl;
    LocalArgs la;
    rc = prepare_round(kOptLars, peer_codes, peer_scales, counts, n_peers, bounds, n_shards, codec, block,
                       out_codes, out_scales, x, nullptr, v, P, offsets, flags, n_tensors, out_mean, local, ws,
                       ws_bytes, peers, pl, la);
    if (rc) return rc;
    return run_round(kOptLars, peers, codec, out_codes, out_scales, x, nullptr, v, P, pl, op, trust_out, out_mean,
                     la, ws, (hipStream_t)stream);
}

size_t dedloc_group_allreduce_workspace_bytes(uint32_t n_peers, uint32_t group_size, uint64_t len,
                                              int32_t codec, uint32_t block) {
    if (check_codec(codec, block, false)) return 0;
    GroupPlan gp;
    if (group_plan(n_peers, group_size, len, codec, gp)) return 0;
    return gp.ws_total > 0 ? gp.ws_total : 256;
}

int dedloc_group_allreduce(const void *const *peer_codes, const float *const *peer_scales,
                           const uint32_t *counts, uint32_t n_peers, uint32_t group_size, uint64_t len,
                           int32_t codec, uint32_t block, void *out_codes, float *out_scales,
                           uint32_t *peer_out, uint32_t *n_out, void *ws, size_t ws_bytes, void *stream) {
    int rc = check_codec(codec, block, false);
    if (rc) return rc;
    GroupPlan gp;
    rc = group_plan(n_peers, group_size, len, codec, gp);
    if (rc) return rc;
    if (!peer_codes || !counts) return fail(DEDLOC_ERR_INVALID_ARG, "peer_codes and counts must not be NULL");
    if (codec == DEDLOC_CODEC_I8 && !peer_scales) return fail(DEDLOC_ERR_INVALID_ARG, "int8 messages need peer_scales");
    uint64_t total = 0;
    for (uint32_t i = 0; i < n_peers; i++) total += counts[i];
    if (total == 0) return fail(DEDLOC_ERR_ZERO_WEIGHT, "every peer has zero samples");
    if (total > (1u << 24)) return fail(DEDLOC_ERR_INVALID_ARG, "total sample count exceeds 2^24");
    if (len > 0) {
        for (uint32_t i = 0; i < n_peers; i++) {
            if (counts[i] == 0) continue;  // never read
            if (!peer_codes[i] || !aligned(peer_codes[i], 16))
                return fail(DEDLOC_ERR_ALIGN, "peer %u message must be non-NULL and 16-byte aligned", i);
            if (codec == DEDLOC_CODEC_I8 && (!peer_scales[i] || !aligned(peer_scales[i], 4)))
                return fail(DEDLOC_ERR_ALIGN, "peer %u scales must be non-NULL and 4-byte aligned", i);
        }
    }
    if (!peer_out || !n_out) return fail(DEDLOC_ERR_INVALID_ARG, "peer_out and n_out must not be NULL");
    if (len > 0) {
        if (!out_codes || !aligned(out_codes, 256)) return fail(DEDLOC_ERR_ALIGN, "out_codes must be non-NULL and 256-byte aligned");
        if (codec == DEDLOC_CODEC_I8 && (!out_scales || !aligned(out_scales, 4)))
            return fail(DEDLOC_ERR_INVALID_ARG, "int8 group all-reduce needs aligned out_scales");
        if (gp.ws_total > 0 && (!ws || ws_bytes < gp.ws_total))
            return fail(DEDLOC_ERR_WORKSPACE, "workspace of %zu bytes needed (got %zu)", gp.ws_total, ws ? ws_bytes : (size_t)0);
        if (gp.ws_total > 0 && !aligned(ws, 256)) return fail(DEDLOC_ERR_ALIGN, "workspace must be 256-byte aligned");
    }
    const uint32_t m = group_size;
    std::vector<int64_t> src(gp.slots, -1), nsrc(gp.slots);
    std::vector<uint64_t> cnt(gp.slots, 0), ncnt(gp.slots);
    for (uint32_t i = 0; i < n_peers; i++) cnt[i] = counts[i];
    hipStream_t s = (hipStream_t)stream;
    char *wsc = (char *)ws;
    float *wss = (float *)(wsc + gp.ws_codes);
    GroupTable gt;
    // launch the groups gathered in gt (one grid row each)
    auto flush = [&]() -> int {
        if (gt.n_groups == 0) return DEDLOC_OK;
        gt.gbegin[gt.n_groups] = gt.pt.n;
        if (len > 0) {
            const ChainArgs ca = {nullptr, nullptr, 1, {-1, nullptr, nullptr, nullptr}};
            hipError_t e = codec == DEDLOC_CODEC_FP16
                               ? timed(K_REDUCE_FP16, s, [&] { return launch_reduce_fp16(gt, len, ca, s); })
                               : timed(K_REDUCE_I8, s, [&] { return launch_reduce_i8(gt, len, ca, s); });
            if (e != hipSuccess) return hip_fail(e, "group reduce launch");
        }
        memset(&gt, 0, sizeof gt);
        return DEDLOC_OK;
    };
    uint64_t lo = 1;  // m^k, the weight of digit k
    for (uint32_t k = 0; k < gp.d; k++, lo *= m) {
        const bool last = k + 1 == gp.d;
        char *dst_c = last ? (char *)out_codes : wsc + (size_t)(k % 2) * gp.groups * gp.code_stride;
        float *dst_s = last ? out_scales : wss + (size_t)(k % 2) * gp.groups * gp.scale_stride;
        const char *prev_c = wsc + (size_t)((k + 1) % 2) * gp.groups * gp.code_stride;
        const float *prev_s = wss + (size_t)((k + 1) % 2) * gp.groups * gp.scale_stride;
        memset(&gt, 0, sizeof gt);
        for (uint32_t g = 0; g < gp.groups; g++) {
            const uint64_t base = (g / lo) * lo * m + (g % lo);
            uint32_t members = 0;
            uint64_t gtotal = 0;
            for (uint32_t j = 0; j < m; j++) {
                gtotal += cnt[base + j * lo];
                members += cnt[base + j * lo] > 0;
            }
            // a launch describes at most kMaxPeers members and kMaxGroups groups
            if (gt.pt.n + members > (uint32_t)kMaxPeers || gt.n_groups == (uint32_t)kMaxGroups) {
                rc = flush();
                if (rc) return rc;
            }
            const uint32_t first = gt.pt.n;
            uint32_t mc[DEDLOC_MAX_GROUP_SIZE];
            uint32_t nm = 0;
            for (uint32_t j = 0; j < m; j++) {
                const uint64_t sl = base + j * lo;
                if (cnt[sl] == 0) continue;
                if (src[sl] < 0) {
                    gt.pt.codes[gt.pt.n] = peer_codes[sl];
                    gt.pt.scales[gt.pt.n] = codec == DEDLOC_CODEC_I8 ? peer_scales[sl] : nullptr;
                } else {
                    gt.pt.codes[gt.pt.n] = prev_c + (size_t)src[sl] * gp.code_stride;
                    gt.pt.scales[gt.pt.n] = codec == DEDLOC_CODEC_I8 ? prev_s + (size_t)src[sl] * gp.scale_stride : nullptr;
                }
                mc[nm++] = (uint32_t)cnt[sl];
                gt.pt.n++;
            }
            if (nm > 0) {
                float w[DEDLOC_MAX_GROUP_SIZE];
                rc = compute_weights(mc, nm, w);
                if (rc) return rc;
                for (uint32_t j = 0; j < nm; j++) gt.pt.w[first + j] = w[j];
            }
            const uint32_t lg = gt.n_groups++;
            gt.gbegin[lg] = first;
            gt.out[lg] = dst_c + (size_t)g * gp.code_stride;
            gt.out_scales[lg] = codec == DEDLOC_CODEC_I8 ? dst_s + (size_t)g * gp.scale_stride : nullptr;
            for (uint32_t j = 0; j < m; j++) {
                const uint64_t sl = base + j * lo;
                nsrc[sl] = gtotal > 0 ? (int64_t)g : -2;
                ncnt[sl] = gtotal;
            }
        }
        rc = flush();
        if (rc) return rc;
        src.swap(nsrc);
        cnt.swap(ncnt);
    }
    for (uint32_t i = 0; i < n_peers; i++) peer_out[i] = src[i] >= 0 ? (uint32_t)src[i] : 0xffffffffu;
    *n_out = gp.groups;
    return DEDLOC_OK;
}

int dedloc_accumulate(float *acc, const void *grad, int32_t grad_codec, uint64_t n, float batch_samples,
                      void *stream) {
    if (grad_codec != DEDLOC_CODEC_F32 && grad_codec != DEDLOC_CODEC_FP16)
        return fail(DEDLOC_ERR_INVALID_ARG, "accumulate takes fp32 or fp16 gradients");
    if (n == 0) return DEDLOC_OK;
    if (!acc || !grad) return fail(DEDLOC_ERR_INVALID_ARG, "acc and grad must not be NULL");
    if (!aligned(acc, 16) || !aligned(grad, 16)) return fail(DEDLOC_ERR_ALIGN, "acc and grad must be 16-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = timed(K_ACCUMULATE, s, [&] {
        return launch_accumulate(acc, grad, grad_codec == DEDLOC_CODEC_FP16, n, batch_samples, s);
    });
    return e == hipSuccess ? DEDLOC_OK : hip_fail(e, "accumulate launch");
}

int dedloc_finalize(float *acc, uint64_t n, uint32_t count, int32_t codec, uint32_t block, void *codes,
                    float *scales, int32_t reset, void *stream) {
    int rc = check_codec(codec, block, false);
    if (rc) return rc;
    if (count == 0) return fail(DEDLOC_ERR_ZERO_WEIGHT, "no samples were accumulated");
    if (count > (1u << 24)) return fail(DEDLOC_ERR_INVALID_ARG, "count %u exceeds 2^24", count);
    if (n == 0) return DEDLOC_OK;
    if (!acc || !codes) return fail(DEDLOC_ERR_INVALID_ARG, "acc and codes must not be NULL");
    if (!aligned(acc, 16) || !aligned(codes, 16)) return fail(DEDLOC_ERR_ALIGN, "acc and codes must be 16-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (codec == DEDLOC_CODEC_FP16) {
        e = timed(K_FINALIZE_FP16, s, [&] { return launch_finalize_fp16(acc, n, (float)count, (uint16_t *)codes, reset, s); });
    } else {
        if (!scales || !aligned(scales, 4)) return fail(DEDLOC_ERR_INVALID_ARG, "int8 finalize needs aligned scales");
        e = timed(K_FINALIZE_I8, s, [&] {
            return launch_finalize_i8(acc, n, (float)count, (int8_t *)codes, scales, reset, s);
        });
    }
    return e == hipSuccess ? DEDLOC_OK : hip_fail(e, "finalize launch");
}

int dedloc_profile_begin(uint32_t max_launches) {
    std::lock_guard<std::mutex> lk(g_prof.mu);
    g_prof.on = true;
    g_prof.cap = max_launches;
    g_prof.used = 0;
    g_prof.kind.clear();
    return DEDLOC_OK;
}

int dedloc_profile_end(uint32_t n_kinds, double *total_ms, uint64_t *launches) {
    std::lock_guard<std::mutex> lk(g_prof.mu);
    if (!g_prof.on) return fail(DEDLOC_ERR_INVALID_ARG, "profiling was not started");
    g_prof.on = false;
    for (uint32_t k = 0; k < n_kinds; k++) {
        if (total_ms) total_ms[k] = 0.0;
        if (launches) launches[k] = 0;
    }
    for (size_t i = 0; i < g_prof.used; i++) {
        hipError_t r = hipEventSynchronize(g_prof.ev[2 * i + 1]);
        if (r != hipSuccess) return hip_fail(r, "profile event wait");
        float ms = 0.0f;
        r = hipEventElapsedTime(&ms, g_prof.ev[2 * i], g_prof.ev[2 * i + 1]);
        if (r != hipSuccess) return hip_fail(r, "profile event time");
        const int k = g_prof.kind[i];
        if ((uint32_t)k < n_kinds) {
            if (total_ms) total_ms[k] += ms;
            if (launches) launches[k] += 1;
        }
    }
    g_prof.used = 0;
    return DEDLOC_OK;
}

uint32_t dedloc_test_trust_polls(uint32_t polls) { return g_trust_polls.exchange(polls); }

int dedloc_kernel_kinds(void) { return K_COUNT; }

const char *dedloc_kernel_name(int kind) {
    return (kind >= 0 && kind < K_COUNT) ? kKindNames[kind] : "";
}

}  // extern "C"
