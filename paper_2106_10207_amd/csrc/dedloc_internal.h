// Internal declarations shared by the kernels and the C-ABI layer of
// libdedloc.  Not part of the public interface (include/dedloc.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dedloc {

constexpr int kWG = 256;               // threads per workgroup: 4 wave64
constexpr int kVec = 8;                // fp32/fp16 elements per lane (16 B of fp16, 2x16 B of fp32)
constexpr int kTile = kWG * kVec;      // LAMB tile: 2048 elements of one tensor
constexpr int kMaxPeers = 64;          // peer table lives in the kernel arguments
constexpr int kI8Block = 1024;         // int8 codec block = one wave64 x 16 codes
constexpr int kI8PerLane = 16;
constexpr int kChunkTensors = 64;      // tensors described per LAMB launch

// Active peers (counts > 0) in ascending peer order, with their weights.
struct PeerTable {
    const void *codes[kMaxPeers];
    const float *scales[kMaxPeers];
    float w[kMaxPeers];
    uint32_t n;
};

// A run of consecutive tensors handled by one LAMB launch.  Tiles never cross
// a tensor: tensor k of the chunk owns launch blocks
// [tile_begin[k], tile_begin[k+1]).
struct Chunk {
    uint64_t off[kChunkTensors + 1];      // absolute element offsets
    uint32_t tile_begin[kChunkTensors + 1];
    uint32_t nt;                          // tensors in this chunk
    uint32_t t0;                          // index of the chunk's first tensor
    uint32_t tile_base;                   // index of the chunk's first tile in the workspace
    uint8_t flags[kChunkTensors];
};

struct LambParams {
    float lr, beta1, beta2, omb1, omb2, c1, c2, eps, wd;
    int32_t unit_trust;
};

// Where the LAMB step takes its gradient from.
enum GradSrc : int {
    kSrcF32 = 0,      // fp32 gradient
    kSrcFP16 = 1,     // fp16 message
    kSrcI8 = 2,       // int8 message + block scales
    kSrcPeersFP16 = 3 // fused: average the fp16 peer messages, encode, decode
};

struct GradArgs {
    const void *grad;        // kSrcF32 / kSrcFP16 / kSrcI8
    const float *scales;     // kSrcI8
    uint16_t *out_codes;     // kSrcPeersFP16: gathered encoded average
    float *out_mean;         // kSrcPeersFP16: fp32 average (nullable)
};

struct LambWs {
    double *partials;        // 2 per tile: sum x^2, sum u^2
    float *trust;            // per tensor: r_t, read by pass B
};

// Launchers (return hipError_t of the launch).
hipError_t launch_encode_fp16(const float *x, uint64_t n, uint16_t *codes, hipStream_t s);
hipError_t launch_decode_fp16(const uint16_t *codes, uint64_t n, float *out, hipStream_t s);
hipError_t launch_encode_i8(const float *x, uint64_t n, int8_t *codes, float *scales, hipStream_t s);
hipError_t launch_decode_i8(const int8_t *codes, const float *scales, uint64_t n, float *out,
                            hipStream_t s);
hipError_t launch_reduce_fp16(const PeerTable &pt, uint64_t len, uint16_t *out, float *mean,
                              hipStream_t s);
hipError_t launch_reduce_i8(const PeerTable &pt, uint64_t len, int8_t *out, float *out_scales,
                            float *mean, hipStream_t s);
hipError_t launch_lamb_a(int src, const Chunk &ch, uint32_t n_tiles, const PeerTable *pt,
                         const GradArgs &ga, const LambParams &lp, float *x, float *m, float *v,
                         const LambWs &ws, hipStream_t s);
hipError_t launch_lamb_trust(const Chunk &ch, const LambParams &lp, const LambWs &ws, float *trust_out,
                             hipStream_t s);
hipError_t launch_lamb_b(const Chunk &ch, uint32_t n_tiles, const LambParams &lp, float *x,
                         const float *m, const float *v, const LambWs &ws, hipStream_t s);
hipError_t launch_fill_zero(void *p, size_t bytes, hipStream_t s);

}  // namespace dedloc
