// Internal declarations shared by the kernels and the C-ABI layer of
// libdedloc.  Not part of the public interface (include/dedloc.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dedloc {

// Launch-shape tuning (set from measurements on MI355X).
#ifndef DEDLOC_VPL
#define DEDLOC_VPL 1          // 8-element vectors per lane in a LAMB tile
#endif
#ifndef DEDLOC_PEER_BATCH
#define DEDLOC_PEER_BATCH 16  // peer loads issued before the first fma
#endif
#ifndef DEDLOC_NT_PEERS
#define DEDLOC_NT_PEERS 1     // non-temporal hint on loads of data read once
#endif
#ifndef DEDLOC_NT_STORES
#define DEDLOC_NT_STORES 0    // non-temporal hint on streamed stores
#endif
#ifndef DEDLOC_NT_MSG_STORES
#define DEDLOC_NT_MSG_STORES 1  // non-temporal hint on stores of encoded messages
#endif
#ifndef DEDLOC_TRUST_UNROLL
#define DEDLOC_TRUST_UNROLL 8   // tile partials loaded per lane before summing
#endif
#ifndef DEDLOC_I8_BATCH
#define DEDLOC_I8_BATCH 16    // int8 peer messages loaded per batch in the reduce
#endif
#ifndef DEDLOC_B_REVERSE
#define DEDLOC_B_REVERSE 1    // pass B visits tiles last-to-first (its re-reads
                              // start with what pass A touched last)
#endif

constexpr int kWG = 256;               // threads per workgroup: 4 wave64
constexpr int kVec = 8;                // fp32/fp16 elements per lane (16 B of fp16, 2x16 B of fp32)
constexpr int kVPL = DEDLOC_VPL;
constexpr int kPeerBatch = DEDLOC_PEER_BATCH;
constexpr int kTile = kWG * kVec * kVPL;  // LAMB tile: elements of one tensor per workgroup
constexpr int kMaxPeers = 64;          // peer table lives in the kernel arguments
constexpr int kI8Block = 1024;         // int8 codec block = one wave64 x 16 codes
constexpr int kI8PerLane = 16;
constexpr int kChunkTensors = 192;     // tensors described per LAMB launch

// Active peers (counts > 0) in ascending peer order, with their weights.
struct PeerTable {
    const void *codes[kMaxPeers];
    const float *scales[kMaxPeers];
    float w[kMaxPeers];
    uint32_t n;
};

// Groups of peers reduced by one launch (one group for a plain shard
// reduce; the groups of one iteration of the group all-reduce).  Group g
// averages table entries [gbegin[g], gbegin[g+1]) (its members with samples,
// ascending) into out[g] (and out_scales[g] for int8); an empty range
// produces nothing.
constexpr int kMaxGroups = 64;
struct GroupTable {
    PeerTable pt;
    uint32_t gbegin[kMaxGroups + 1];
    void *out[kMaxGroups];
    float *out_scales[kMaxGroups];
    uint32_t n_groups;
};

// The local peer of a round: its fp32 gradient is encoded by the pass that
// averages it (the codes it would have sent are written on the way), at
// position `pos` of the launch's peer table (-1: no local peer here).
struct LocalArgs {
    int32_t pos;
    const float *grad;  // the full vector, indexed like the messages
    void *codes;        // its message (output)
    float *scales;      // int8: its block scales (output)
};

// A reduce over more peers than one table holds is a chain of launches
// through an fp32 running sum (stored exactly between launches, so the fma
// chain is the same as in one pass).  Only a single-group reduce chains, and
// only a single-group fp16 reduce has a local peer.
struct ChainArgs {
    const float *acc_in;  // running sum of the peers before this launch (nullable: start at +0)
    float *acc_out;       // the sum after this launch (the mean after the last launch; nullable)
    int final_pass;       // encode into the group outputs
    LocalArgs local;
};

// A run of consecutive tensors handled by one LAMB launch (it spans fewer
// than 2^32 elements).  Tiles never cross a tensor: tensor k of the chunk
// covers elements base + [start[k], start[k+1]) and owns launch blocks
// [tile_begin[k], tile_begin[k+1]).
struct Chunk {
    uint64_t base;                        // absolute offset of the chunk's first element
    uint32_t nt;                          // tensors in this chunk
    uint32_t t0;                          // index of the chunk's first tensor
    uint32_t tile_base;                   // index of the chunk's first tile in the workspace
    uint32_t start[kChunkTensors + 1];    // element offsets relative to base
    uint32_t tile_begin[kChunkTensors + 1];
    uint8_t flags[kChunkTensors];
};

// Optimizer applied after the gather.
enum Opt : int {
    kOptLamb = 0,  // Adam moments + layer-wise trust ratio ||x||/||u||
    kOptLars = 1   // momentum SGD + layer-wise rate eta*||x||/(||g|| + wd*||x||)
};

// Hyper-parameters of either optimizer (host-computed constants included).
struct OptParams {
    float lr, wd;
    float beta1, beta2, omb1, omb2, c1, c2, eps;  // LAMB
    float momentum, trust_coef;                   // LARS
    int32_t unit_trust;
    uint32_t trust_polls;  // pass B: polls of a tensor's published ratio before computing it
};

// Where the LAMB step takes its gradient from.
enum GradSrc : int {
    kSrcF32 = 0,      // fp32 gradient
    kSrcFP16 = 1,     // fp16 message
    kSrcI8 = 2,       // int8 message + block scales
    kSrcPeersFP16 = 3,      // fused: average the fp16 peer messages, encode, decode
    kSrcPeersFP16Chain = 4, // the same, continuing a running sum of earlier peers (and
                            // with the local peer if the launch holds it)
    kSrcPeersFP16Local = 5  // kSrcPeersFP16 with the local peer's encode
};

struct GradArgs {
    const void *grad;        // kSrcF32 / kSrcFP16 / kSrcI8
    const float *scales;     // kSrcI8
    uint16_t *out_codes;     // kSrcPeersFP16*: gathered encoded average
    float *out_mean;         // kSrcPeersFP16*: fp32 average (nullable)
    const float *acc_in;     // kSrcPeersFP16Chain: running sum of the earlier peers
    LocalArgs local;         // kSrcPeersFP16Chain / kSrcPeersFP16Local
};

struct LambWs {
    double *partials;            // 2 per tile: sum x^2, sum u^2
    unsigned long long *trust;   // per tensor: (epoch << 32) | bits of r_t, published inside pass B
    uint32_t *epoch;             // the tag of the current launch: advanced by pass A, read by pass B
};

// Launchers (return hipError_t of the launch).
hipError_t launch_encode_fp16(const float *x, uint64_t n, uint16_t *codes, hipStream_t s);
hipError_t launch_decode_fp16(const uint16_t *codes, uint64_t n, float *out, hipStream_t s);
hipError_t launch_encode_i8(const float *x, uint64_t n, int8_t *codes, float *scales, hipStream_t s);
hipError_t launch_decode_i8(const int8_t *codes, const float *scales, uint64_t n, float *out,
                            hipStream_t s);
hipError_t launch_reduce_fp16(const GroupTable &gt, uint64_t len, const ChainArgs &ca, hipStream_t s);
hipError_t launch_reduce_i8(const GroupTable &gt, uint64_t len, const ChainArgs &ca, hipStream_t s);
hipError_t launch_opt_a(int opt, int src, const Chunk &ch, uint32_t n_tiles, const PeerTable *pt,
                        const GradArgs &ga, const OptParams &op, float *x, float *m, float *v,
                        const LambWs &ws, hipStream_t s);
hipError_t launch_opt_b(int opt, int src, const Chunk &ch, uint32_t n_tiles, const GradArgs &ga,
                        const OptParams &op, float *x, float *m, float *v, const LambWs &ws, uint32_t nonce,
                        float *trust_out, hipStream_t s);
hipError_t launch_accumulate(float *acc, const void *grad, bool fp16, uint64_t n, float b, hipStream_t s);
hipError_t launch_finalize_fp16(float *acc, uint64_t n, float count, uint16_t *codes, int reset, hipStream_t s);
hipError_t launch_finalize_i8(float *acc, uint64_t n, float count, int8_t *codes, float *scales, int reset,
                              hipStream_t s);
hipError_t launch_fill_zero(void *p, size_t bytes, hipStream_t s);

}  // namespace dedloc
