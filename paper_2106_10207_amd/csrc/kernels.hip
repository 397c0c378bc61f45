// gfx950 kernels of libdedloc: wire codecs, the weighted shard average and
// the two LAMB passes.
//
// Every kernel streams HBM in 16-byte vectors per lane; nothing here is a
// dense contraction, so there is no MFMA.  Compiled with -ffp-contract=off:
// every fused multiply-add is an explicit fmaf, every other operation rounds
// once, fp32 division and square root are correctly rounded (the HIP
// defaults), so the results are fixed by the definitions in dedloc.h.
#include <algorithm>
#include <tuple>
#include <utility>

#include "dedloc_internal.h"

namespace dedloc {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- helpers

// Loads of data read once (peer messages) and stores of data written once.
template <typename T>
__device__ __forceinline__ T ld_stream(const T *p) {
    if (DEDLOC_NT_PEERS) return __builtin_nontemporal_load(p);
    return *p;
}
template <typename T>
__device__ __forceinline__ void st_stream(T *p, T v) {
    if (DEDLOC_NT_STORES) __builtin_nontemporal_store(v, p);
    else *p = v;
}
// Stores of encoded messages (read by other peers, not by this kernel).
template <typename T>
__device__ __forceinline__ void st_msg(T *p, T v) {
    if (DEDLOC_NT_MSG_STORES) __builtin_nontemporal_store(v, p);
    else *p = v;
}

__device__ __forceinline__ float h2f(unsigned bits) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
}
__device__ __forceinline__ unsigned f2h(float f) {
    // IEEE round to nearest even, gradual underflow, overflow to infinity
    return __builtin_bit_cast(uint16_t, (_Float16)f);
}

__device__ __forceinline__ void unpack_fp16x8(u32x4 c, float *o) {
#pragma unroll
    for (int i = 0; i < 4; i++) {
        o[2 * i] = h2f(c[i] & 0xffffu);
        o[2 * i + 1] = h2f(c[i] >> 16);
    }
}
__device__ __forceinline__ u32x4 pack_fp16x8(const float *a) {
    u32x4 c;
#pragma unroll
    for (int i = 0; i < 4; i++) c[i] = f2h(a[2 * i]) | (f2h(a[2 * i + 1]) << 16);
    return c;
}

__device__ __forceinline__ float sbyte(unsigned word, int j) {
    return (float)(int)(int8_t)(word >> (8 * j));
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Sum of two doubles over the 256-thread block in a fixed tree; thread 0
// gets the result.
__device__ __forceinline__ void block_sum2(double &a, double &b) {
    __shared__ double red[2][kWG / 64];
    a = wave_sum(a);
    b = wave_sum(b);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) {
        red[0][wave] = a;
        red[1][wave] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
        b = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    }
    __syncthreads();
}

// Encode one int8 block held by a wave: 16 values per lane (lanes or values
// past the end hold zero).  Returns the codes packed in a u32x4 and the
// block scale (same on every lane).
//
// The code is rint of the correctly rounded quotient x / s.  It is taken from
// t = x * rcp(s) instead wherever that provably gives the same integer:
// v_rcp_f32 is within 1 ulp of 1/s, so |t - x/s| < 1.5 * 2^-23 * |x/s| and
// |x/s| <= a / fl(a/127) < 127.00001 bound the error by 2.3e-5, and the
// correctly rounded quotient lies within half an ulp (2^-18 below 128) of
// x/s.  When t is farther than 2^-14 from every half-integer, x/s, its
// rounding and t all lie strictly on the same side of every half-integer,
// so rint(t) is the code.  Lanes holding a value closer to a tie, and blocks
// whose scale is outside [2^-100, 2^100] (where rcp could leave the normal
// range), divide.
__device__ __forceinline__ u32x4 encode_i8_wave(const float *val, float &scale) {
    float a = 0.0f;
#pragma unroll
    for (int j = 0; j < kI8PerLane; j++) a = fmaxf(a, fabsf(val[j]));
    a = wave_max(a);
    const float s = a / 127.0f;
    scale = s;
    u32x4 c = {0u, 0u, 0u, 0u};
    if (s != 0.0f) {  // s == 0: an all-zero block, or a / 127 underflowed; every code is 0
        float q[kI8PerLane];
        bool divide = !(s >= 0x1p-100f && s <= 0x1p100f);  // wave-uniform
        if (!divide) {
            const float y = __builtin_amdgcn_rcpf(s);
#pragma unroll
            for (int j = 0; j < kI8PerLane; j++) {
                const float t = val[j] * y;
                q[j] = rintf(t);
                divide |= fabsf(t - q[j]) > 0.5f - 0x1p-14f;  // t - rint(t) is exact
            }
        }
        if (divide) {
#pragma unroll
            for (int j = 0; j < kI8PerLane; j++) q[j] = rintf(val[j] / s);
        }
#pragma unroll
        for (int j = 0; j < kI8PerLane; j++) {
            const float qc = fminf(fmaxf(q[j], -127.0f), 127.0f);
            c[j >> 2] |= ((unsigned)(int)qc & 0xffu) << (8 * (j & 3));
        }
    }
    return c;
}

// -------------------------------------------------------------- fp16 codec

__global__ __launch_bounds__(kWG) void encode_fp16_kernel(const float *__restrict__ x, uint64_t n,
                                                          uint16_t *__restrict__ codes) {
    const uint64_t e0 = ((uint64_t)blockIdx.x * kWG + threadIdx.x) * kVec;
    if (e0 + kVec <= n) {
        const f32x4 a = ld_stream((const f32x4 *)(x + e0)), b = ld_stream((const f32x4 *)(x + e0 + 4));
        float v[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
        st_msg((u32x4 *)(codes + e0), pack_fp16x8(v));
    } else {
        for (uint64_t e = e0; e < n; e++) codes[e] = (uint16_t)f2h(x[e]);
    }
}

__global__ __launch_bounds__(kWG) void decode_fp16_kernel(const uint16_t *__restrict__ codes, uint64_t n,
                                                          float *__restrict__ out) {
    const uint64_t e0 = ((uint64_t)blockIdx.x * kWG + threadIdx.x) * kVec;
    if (e0 + kVec <= n) {
        float v[8];
        unpack_fp16x8(*(const u32x4 *)(codes + e0), v);
        *(f32x4 *)(out + e0) = f32x4{v[0], v[1], v[2], v[3]};
        *(f32x4 *)(out + e0 + 4) = f32x4{v[4], v[5], v[6], v[7]};
    } else {
        for (uint64_t e = e0; e < n; e++) out[e] = h2f(codes[e]);
    }
}

// -------------------------------------------------------------- int8 codec
// One wave per 1024-element block, 16 elements per lane.  In the standalone
// codec kernels lane l holds elements 256*q + 4*l + r (q, r in 0..3) of its
// block, so that every 16-byte fp32 access of the wave covers 1 KB without
// gaps (the block maximum and the per-element codes do not depend on which
// lane holds which element).

__device__ __forceinline__ uint64_t i8_lane_base(uint64_t blk) { return blk * kI8Block + 4 * (threadIdx.x & 63); }
#define I8_ELEM(b0, q, r) ((b0) + 256 * (q) + (r))

// The lane's 16 fp32 values of block blk (zero past n).
__device__ __forceinline__ void load_i8_lane(const float *__restrict__ x, uint64_t n, uint64_t blk, float *val) {
    const uint64_t b0 = i8_lane_base(blk);
    if ((blk + 1) * kI8Block <= n) {
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const f32x4 a = ld_stream((const f32x4 *)(x + I8_ELEM(b0, q, 0)));
            val[4 * q] = a[0]; val[4 * q + 1] = a[1]; val[4 * q + 2] = a[2]; val[4 * q + 3] = a[3];
        }
    } else {
#pragma unroll
        for (int q = 0; q < 4; q++)
#pragma unroll
            for (int r = 0; r < 4; r++) {
                const uint64_t e = I8_ELEM(b0, q, r);
                val[4 * q + r] = e < n ? x[e] : 0.0f;
            }
    }
}

// Store the lane's 16 codes of block blk (those below n) and the scale.
__device__ __forceinline__ void store_i8_lane(int8_t *__restrict__ codes, float *__restrict__ scales, uint64_t n,
                                              uint64_t blk, u32x4 c, float s) {
    const uint64_t b0 = i8_lane_base(blk);
    if ((blk + 1) * kI8Block <= n) {
#pragma unroll
        // plain stores: with a non-temporal hint the reduce that reads this
        // message next ran 40 us slower on ALBERT-xlarge
        for (int q = 0; q < 4; q++) *(unsigned *)(codes + I8_ELEM(b0, q, 0)) = c[q];
    } else {
#pragma unroll
        for (int q = 0; q < 4; q++)
#pragma unroll
            for (int r = 0; r < 4; r++) {
                const uint64_t e = I8_ELEM(b0, q, r);
                if (e < n) codes[e] = (int8_t)(c[q] >> (8 * r));
            }
    }
    if ((threadIdx.x & 63) == 0) scales[blk] = s;
}

__global__ __launch_bounds__(kWG) void encode_i8_kernel(const float *__restrict__ x, uint64_t n,
                                                        int8_t *__restrict__ codes,
                                                        float *__restrict__ scales) {
    const uint64_t blk = (uint64_t)blockIdx.x * (kWG / 64) + (threadIdx.x >> 6);
    if (blk * kI8Block >= n) return;  // whole wave past the end
    float val[kI8PerLane];
    load_i8_lane(x, n, blk, val);
    float s;
    const u32x4 c = encode_i8_wave(val, s);
    store_i8_lane(codes, scales, n, blk, c, s);
}

__global__ __launch_bounds__(kWG) void decode_i8_kernel(const int8_t *__restrict__ codes,
                                                        const float *__restrict__ scales, uint64_t n,
                                                        float *__restrict__ out) {
    const uint64_t blk = (uint64_t)blockIdx.x * (kWG / 64) + (threadIdx.x >> 6);
    if (blk * kI8Block >= n) return;  // whole wave past the end
    const float s = scales[blk];
    const uint64_t b0 = i8_lane_base(blk);
    if ((blk + 1) * kI8Block <= n) {
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const unsigned c = *(const unsigned *)(codes + I8_ELEM(b0, q, 0));
            *(f32x4 *)(out + I8_ELEM(b0, q, 0)) = f32x4{sbyte(c, 0) * s, sbyte(c, 1) * s, sbyte(c, 2) * s,
                                                        sbyte(c, 3) * s};
        }
    } else {
#pragma unroll
        for (int q = 0; q < 4; q++)
#pragma unroll
            for (int r = 0; r < 4; r++) {
                const uint64_t e = I8_ELEM(b0, q, r);
                if (e < n) out[e] = (float)codes[e] * s;
            }
    }
}

// ------------------------------------------------------------- the reducer
// mean[e] = sum over the active peers of a group (ascending) of
// w_p * dec_p[e], one fma per peer starting from +0.  A launch reduces every
// group of a GroupTable: grid row blockIdx.y is the group.

// Running sums of eight consecutive elements: from acc_in, or +0.
__device__ __forceinline__ void init8(const float *acc_in, uint64_t e0, float *acc) {
    if (acc_in) {
        const f32x4 a = *(const f32x4 *)(acc_in + e0), b = *(const f32x4 *)(acc_in + e0 + 4);
        acc[0] = a[0]; acc[1] = a[1]; acc[2] = a[2]; acc[3] = a[3];
        acc[4] = b[0]; acc[5] = b[1]; acc[6] = b[2]; acc[7] = b[3];
    } else {
#pragma unroll
        for (int i = 0; i < 8; i++) acc[i] = 0.0f;
    }
}

// Eight consecutive fp16 elements starting at e0 (all in range), peers
// [p_lo, p_hi) of the table, added to the running sums in acc.
template <int B = kPeerBatch>  // peer loads kept in flight per lane
__device__ __forceinline__ void reduce_fp16x8(const PeerTable &pt, uint32_t p_lo, uint32_t p_hi,
                                              uint64_t e0, float *acc) {
    for (uint32_t p0 = p_lo; p0 < p_hi; p0 += B) {
        u32x4 c[B];
#pragma unroll
        for (int j = 0; j < B; j++)
            if (p0 + j < p_hi) c[j] = ld_stream((const u32x4 *)((const uint16_t *)pt.codes[p0 + j] + e0));
#pragma unroll
        for (int j = 0; j < B; j++) {
            if (p0 + j < p_hi) {
                const float w = pt.w[p0 + j];
                float d[8];
                unpack_fp16x8(c[j], d);
#pragma unroll
                for (int i = 0; i < 8; i++) acc[i] = fmaf(w, d[i], acc[i]);
            }
        }
    }
}

__device__ __forceinline__ float reduce_fp16_one(const PeerTable &pt, uint32_t p_lo, uint32_t p_hi,
                                                 uint64_t e, float acc) {
    for (uint32_t p = p_lo; p < p_hi; p++)
        acc = fmaf(pt.w[p], h2f(((const uint16_t *)pt.codes[p])[e]), acc);
    return acc;
}

// Peers [0, n) of the table added to acc, the peer at lp (< n) being the
// local one: its eight fp32 values are encoded, the codes stored as its
// message and their decoded values averaged like any peer's.  (Issuing the
// next peers' loads before the local peer's values are used measured the
// same, and keeping the local loads inside a peer batch costs registers.)
__device__ __forceinline__ void reduce_fp16x8_local(const PeerTable &pt, uint32_t n, uint32_t lp,
                                                    const LocalArgs &la, uint64_t e0, float *acc) {
    reduce_fp16x8(pt, 0, lp, e0, acc);
    const f32x4 ga = ld_stream((const f32x4 *)(la.grad + e0)), gb = ld_stream((const f32x4 *)(la.grad + e0 + 4));
    const float v[8] = {ga[0], ga[1], ga[2], ga[3], gb[0], gb[1], gb[2], gb[3]};
    const u32x4 lc = pack_fp16x8(v);
    st_msg((u32x4 *)((uint16_t *)la.codes + e0), lc);
    float d[8];
    unpack_fp16x8(lc, d);
    const float w = pt.w[lp];
#pragma unroll
    for (int i = 0; i < 8; i++) acc[i] = fmaf(w, d[i], acc[i]);
    reduce_fp16x8(pt, lp + 1, n, e0, acc);
}

__device__ __forceinline__ float reduce_fp16_one_local(const PeerTable &pt, uint32_t n, uint32_t lp,
                                                       const LocalArgs &la, uint64_t e, float acc) {
    acc = reduce_fp16_one(pt, 0, lp, e, acc);
    const unsigned c = f2h(la.grad[e]);
    ((uint16_t *)la.codes)[e] = (uint16_t)c;
    acc = fmaf(pt.w[lp], h2f(c), acc);
    return reduce_fp16_one(pt, lp + 1, n, e, acc);
}

// B: peer loads per batch (small groups take a small batch, which keeps
// registers and so more waves in flight).  Only the full batch handles a
// local peer.
template <int B>
__global__ __launch_bounds__(kWG) void reduce_fp16_kernel(const GroupTable gt, uint64_t len,
                                                          const ChainArgs ca) {
    const uint32_t g = blockIdx.y;
    const uint32_t p_lo = gt.gbegin[g], p_hi = gt.gbegin[g + 1];
    if (p_lo == p_hi) return;  // a group without samples produces nothing
    uint16_t *__restrict__ out = (uint16_t *)gt.out[g];
    float *mean = ca.acc_out;  // may alias ca.acc_in (same element, same lane)
    const uint64_t e0 = ((uint64_t)blockIdx.x * kWG + threadIdx.x) * kVec;
    const bool local = B == kPeerBatch && ca.local.pos >= 0;  // single group: p_lo = 0
    if (e0 + kVec <= len) {
        float acc[8];
        init8(ca.acc_in, e0, acc);
        if (local) reduce_fp16x8_local(gt.pt, p_hi, ca.local.pos, ca.local, e0, acc);
        else reduce_fp16x8<B>(gt.pt, p_lo, p_hi, e0, acc);
        if (ca.final_pass) *(u32x4 *)(out + e0) = pack_fp16x8(acc);
        if (mean) {
            *(f32x4 *)(mean + e0) = f32x4{acc[0], acc[1], acc[2], acc[3]};
            *(f32x4 *)(mean + e0 + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
        }
    } else {
        for (uint64_t e = e0; e < len; e++) {
            const float a0 = ca.acc_in ? ca.acc_in[e] : 0.0f;
            const float a = local ? reduce_fp16_one_local(gt.pt, p_hi, ca.local.pos, ca.local, e, a0)
                                  : reduce_fp16_one(gt.pt, p_lo, p_hi, e, a0);
            if (ca.final_pass) out[e] = (uint16_t)f2h(a);
            if (mean) mean[e] = a;
        }
    }
}

// Codes (16 per lane) and block scales of block blk of peers
// [p0, min(p0 + B, p_hi)); `full` if all 16 elements of the lane are in range.
template <int B>
__device__ __forceinline__ void load_i8_batch(const PeerTable &pt, uint32_t p0, uint32_t p_hi, uint64_t blk,
                                              uint64_t e0, uint64_t len, bool full, u32x4 *c, float *s) {
#pragma unroll
    for (int j = 0; j < B; j++) {
        if (p0 + j < p_hi) {
            const int8_t *src = (const int8_t *)pt.codes[p0 + j];
            s[j] = pt.scales[p0 + j][blk];
            if (full) {
                c[j] = ld_stream((const u32x4 *)(src + e0));
            } else {
                c[j] = u32x4{0u, 0u, 0u, 0u};
                for (int k = 0; k < kI8PerLane; k++)
                    if (e0 + k < len) c[j][k >> 2] |= ((unsigned)(uint8_t)src[e0 + k]) << (8 * (k & 3));
            }
        }
    }
}

template <int B>
__device__ __forceinline__ void fma_i8_batch(const PeerTable &pt, uint32_t p0, uint32_t p_hi, const u32x4 *c,
                                             const float *s, float *acc) {
#pragma unroll
    for (int j = 0; j < B; j++) {
        if (p0 + j < p_hi) {
            const float w = pt.w[p0 + j];
#pragma unroll
            for (int k = 0; k < kI8PerLane; k++) {
                const float d = sbyte(c[j][k >> 2], k & 3) * s[j];
                acc[k] = fmaf(w, d, acc[k]);
            }
        }
    }
}

// Peers [p_lo, p_hi) of the table added to the lane's 16 running sums of
// block blk (elements e0..).
template <int B>  // peer loads issued before the batch's fmas
__device__ __forceinline__ void reduce_i8_range(const PeerTable &pt, uint32_t p_lo, uint32_t p_hi, uint64_t blk,
                                                uint64_t e0, uint64_t len, bool full, float *acc) {
    for (uint32_t p0 = p_lo; p0 < p_hi; p0 += B) {
        u32x4 c[B];
        float s[B];
        load_i8_batch<B>(pt, p0, p_hi, blk, e0, len, full, c, s);
        fma_i8_batch<B>(pt, p0, p_hi, c, s, acc);
    }
}

// One wave per 1024-element block; lane holds 16 elements.  B as for
// reduce_fp16_kernel.
template <int B>
__global__ __launch_bounds__(kWG) void reduce_i8_kernel(const GroupTable gt, uint64_t len,
                                                        const ChainArgs ca) {
    const uint32_t g = blockIdx.y;
    const uint32_t p_lo = gt.gbegin[g], p_hi = gt.gbegin[g + 1];
    if (p_lo == p_hi) return;  // a group without samples produces nothing
    int8_t *__restrict__ out = (int8_t *)gt.out[g];
    float *__restrict__ out_scales = gt.out_scales[g];
    const PeerTable &pt = gt.pt;
    const uint64_t blk = (uint64_t)blockIdx.x * (kWG / 64) +
                         (uint64_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (blk * kI8Block >= len) return;  // whole wave past the end
    const uint64_t e0 = blk * kI8Block + (threadIdx.x & 63) * kI8PerLane;
    const bool full = e0 + kI8PerLane <= len;
    float *mean = ca.acc_out;  // may alias ca.acc_in (same element, same lane)
    float acc[kI8PerLane];
    if (ca.acc_in && full) {
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const f32x4 a = *(const f32x4 *)(ca.acc_in + e0 + 4 * q);
            acc[4 * q] = a[0]; acc[4 * q + 1] = a[1]; acc[4 * q + 2] = a[2]; acc[4 * q + 3] = a[3];
        }
    } else {
#pragma unroll
        for (int j = 0; j < kI8PerLane; j++) acc[j] = (ca.acc_in && e0 + j < len) ? ca.acc_in[e0 + j] : 0.0f;
    }
    reduce_i8_range<B>(pt, p_lo, p_hi, blk, e0, len, full, acc);
    if (mean) {
        if (full) {
#pragma unroll
            for (int q = 0; q < 4; q++)
                *(f32x4 *)(mean + e0 + 4 * q) = f32x4{acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
        } else {
            for (int k = 0; k < kI8PerLane; k++)
                if (e0 + k < len) mean[e0 + k] = acc[k];
        }
    }
    if (!ca.final_pass) return;  // wave-uniform
    float s;
    const u32x4 c = encode_i8_wave(acc, s);  // out-of-range lanes hold 0
    if (full) {
        *(u32x4 *)(out + e0) = c;
    } else {
        for (int k = 0; k < kI8PerLane; k++)
            if (e0 + k < len) out[e0 + k] = (int8_t)(c[k >> 2] >> (8 * (k & 3)));
    }
    if ((threadIdx.x & 63) == 0) out_scales[blk] = s;
}

// ------------------------------------------------------- LAMB and LARS

__device__ __forceinline__ float lamb_dir(float mn, float vn, float x, float lam,
                                          const OptParams &op) {
    const float mh = mn / op.c1;
    const float vh = vn / op.c2;
    return mh / (sqrtf(vh) + op.eps) + lam * x;
}

// Tensor of launch block b: the largest k with tile_begin[k] <= b (empty
// tensors own no blocks and are skipped).  All values are wave-uniform.
__device__ __forceinline__ uint32_t chunk_tensor(const Chunk &ch, uint32_t b) {
    uint32_t lo = 0, hi = ch.nt;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (ch.tile_begin[mid] <= b) lo = mid;
        else hi = mid;
    }
    return lo;
}

// Gradient of the elements [e0, e0+cnt), cnt <= 8, for source SRC.
template <int SRC>
__device__ __forceinline__ void load_grad(const GradArgs &ga, const PeerTable &pt, uint64_t e0,
                                          int cnt, float *g) {
    if (cnt == kVec) {
        if (SRC == kSrcF32) {
            const f32x4 a = *(const f32x4 *)((const float *)ga.grad + e0);
            const f32x4 b = *(const f32x4 *)((const float *)ga.grad + e0 + 4);
            g[0] = a[0]; g[1] = a[1]; g[2] = a[2]; g[3] = a[3];
            g[4] = b[0]; g[5] = b[1]; g[6] = b[2]; g[7] = b[3];
        } else if (SRC == kSrcFP16) {
            unpack_fp16x8(*(const u32x4 *)((const uint16_t *)ga.grad + e0), g);
        } else if (SRC == kSrcI8) {
            const u32x2 c = *(const u32x2 *)((const int8_t *)ga.grad + e0);
            const float s = ga.scales[e0 / kI8Block];
#pragma unroll
            for (int j = 0; j < 8; j++) g[j] = sbyte(c[j >> 2], j & 3) * s;
        } else {
            float acc[8];
            init8(SRC == kSrcPeersFP16Chain ? ga.acc_in : nullptr, e0, acc);
            if (SRC != kSrcPeersFP16 && ga.local.pos >= 0) reduce_fp16x8_local(pt, pt.n, ga.local.pos, ga.local, e0, acc);
            else reduce_fp16x8(pt, 0, pt.n, e0, acc);
            const u32x4 c = pack_fp16x8(acc);
            st_msg((u32x4 *)(ga.out_codes + e0), c);
            if (ga.out_mean) {
                *(f32x4 *)(ga.out_mean + e0) = f32x4{acc[0], acc[1], acc[2], acc[3]};
                *(f32x4 *)(ga.out_mean + e0 + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
            }
            unpack_fp16x8(c, g);
        }
    } else {
        for (int j = 0; j < kVec; j++) {
            if (j >= cnt) {
                g[j] = 0.0f;
                continue;
            }
            const uint64_t e = e0 + j;
            if (SRC == kSrcF32) {
                g[j] = ((const float *)ga.grad)[e];
            } else if (SRC == kSrcFP16) {
                g[j] = h2f(((const uint16_t *)ga.grad)[e]);
            } else if (SRC == kSrcI8) {
                g[j] = (float)((const int8_t *)ga.grad)[e] * ga.scales[e / kI8Block];
            } else {
                const float a0 = SRC == kSrcPeersFP16Chain ? ga.acc_in[e] : 0.0f;
                const float a = SRC != kSrcPeersFP16 && ga.local.pos >= 0
                                    ? reduce_fp16_one_local(pt, pt.n, ga.local.pos, ga.local, e, a0)
                                    : reduce_fp16_one(pt, 0, pt.n, e, a0);
                const unsigned c = f2h(a);
                ga.out_codes[e] = (uint16_t)c;
                if (ga.out_mean) ga.out_mean[e] = a;
                g[j] = h2f(c);
            }
        }
    }
}

__device__ __forceinline__ void load8(const float *p, uint64_t e0, int cnt, float *o) {
    if (cnt == kVec) {
        const f32x4 a = *(const f32x4 *)(p + e0), b = *(const f32x4 *)(p + e0 + 4);
        o[0] = a[0]; o[1] = a[1]; o[2] = a[2]; o[3] = a[3];
        o[4] = b[0]; o[5] = b[1]; o[6] = b[2]; o[7] = b[3];
    } else {
        for (int j = 0; j < kVec; j++) o[j] = j < cnt ? p[e0 + j] : 0.0f;
    }
}

__device__ __forceinline__ void store8(float *p, uint64_t e0, int cnt, const float *o) {
    if (cnt == kVec) {
        st_stream((f32x4 *)(p + e0), f32x4{o[0], o[1], o[2], o[3]});
        st_stream((f32x4 *)(p + e0 + 4), f32x4{o[4], o[5], o[6], o[7]});
    } else {
        for (int j = 0; j < cnt; j++) p[e0 + j] = o[j];
    }
}

// Pass A.  LAMB: gradient (optionally the fused average), new moments, and
// the per-tile sums of x^2 and u^2.  LARS: gradient (optionally the fused
// average) and the per-tile sums of x^2 and g^2; nothing else is written.
// Sums are fp64 with a fixed tree inside the tile.
template <int SRC, int OPT>
__global__ __launch_bounds__(kWG) void opt_a_kernel(const Chunk ch, const PeerTable pt,
                                                    const GradArgs ga, const OptParams op,
                                                    const float *__restrict__ x,
                                                    float *__restrict__ m, float *__restrict__ v,
                                                    LambWs ws) {
    const uint32_t b = blockIdx.x;
    const uint32_t k = chunk_tensor(ch, b);
    const uint64_t t_lo = ch.base + ch.start[k], t_hi = ch.base + ch.start[k + 1];
    const uint32_t tile = b - ch.tile_begin[k];
    const float lam = (ch.flags[k] & 1u) ? op.wd : 0.0f;

    double s0 = 0.0, s1 = 0.0;
#pragma unroll
    for (int r = 0; r < kVPL; r++) {
        const uint64_t e0 = t_lo + (uint64_t)tile * kTile + ((uint64_t)r * kWG + threadIdx.x) * kVec;
        if (e0 < t_hi) {
            const int cnt = (int)(t_hi - e0 < (uint64_t)kVec ? t_hi - e0 : (uint64_t)kVec);
            float g[8], xv[8];
            load8(x, e0, cnt, xv);
            if (OPT == kOptLamb) {
                float mv[8], vv[8];
                load8(m, e0, cnt, mv);
                load8(v, e0, cnt, vv);
                load_grad<SRC>(ga, pt, e0, cnt, g);
#pragma unroll
                for (int j = 0; j < 8; j++) {
                    const float mn = fmaf(op.beta1, mv[j], op.omb1 * g[j]);
                    const float vn = fmaf(op.beta2, vv[j], op.omb2 * (g[j] * g[j]));
                    const float u = lamb_dir(mn, vn, xv[j], lam, op);
                    mv[j] = mn;
                    vv[j] = vn;
                    if (j < cnt) {
                        s0 += (double)xv[j] * (double)xv[j];
                        s1 += (double)u * (double)u;
                    }
                }
                store8(m, e0, cnt, mv);
                store8(v, e0, cnt, vv);
            } else {
                load_grad<SRC>(ga, pt, e0, cnt, g);
#pragma unroll
                for (int j = 0; j < 8; j++) {
                    if (j < cnt) {
                        s0 += (double)xv[j] * (double)xv[j];
                        s1 += (double)g[j] * (double)g[j];
                    }
                }
            }
        }
    }
    block_sum2(s0, s1);
    if (threadIdx.x == 0) {
        ws.partials[2 * (ch.tile_base + b)] = s0;
        ws.partials[2 * (ch.tile_base + b) + 1] = s1;
        // a fresh tag for the ratios pass B publishes (the only access to
        // this word during the launch; pass B reads it after the launch)
        if (b == 0) ws.epoch[0] = ws.epoch[0] + 1u;
    }
}

// Sums over tensor k of the chunk of its tile partials (x^2, and u^2 or
// g^2), in a fixed order: lane-strided, then a fixed tree.  Every thread of
// the workgroup calls it; thread 0 gets the sums.
__device__ __forceinline__ void tensor_sums(const Chunk &ch, const LambWs &ws, uint32_t k, double &a0, double &a1) {
    const uint32_t first = ch.tile_base + ch.tile_begin[k];
    const uint32_t ntiles = ch.tile_begin[k + 1] - ch.tile_begin[k];
    typedef double f64x2 __attribute__((ext_vector_type(2)));
    const f64x2 *part = (const f64x2 *)ws.partials + first;
    a0 = 0.0;
    a1 = 0.0;
    constexpr int U = DEDLOC_TRUST_UNROLL;  // loads in flight per lane
    for (uint32_t i0 = 0; i0 < ntiles; i0 += U * kWG) {
        f64x2 q[U];
#pragma unroll
        for (int j = 0; j < U; j++) {
            const uint32_t i = i0 + j * kWG + threadIdx.x;
            q[j] = i < ntiles ? part[i] : f64x2{0.0, 0.0};
        }
#pragma unroll
        for (int j = 0; j < U; j++) {
            a0 += q[j][0];
            a1 += q[j][1];
        }
    }
    block_sum2(a0, a1);
}

// The ratio of tensor k from its sums (r = 1 when disabled or a norm is 0).
//   LAMB: r = ||x|| / ||u||;  LARS: r = eta*||x|| / (||g|| + lambda*||x||).
template <int OPT>
__device__ __forceinline__ float trust_ratio(const Chunk &ch, const OptParams &op, uint32_t k, double a0,
                                             double a1) {
    const double X = sqrt(a0), Y = sqrt(a1);
    float r = 1.0f;
    if (!op.unit_trust && (ch.flags[k] & 2u) && X > 0.0 && Y > 0.0) {
        if (OPT == kOptLamb) {
            r = (float)(X / Y);
        } else {
            const double lam = (ch.flags[k] & 1u) ? (double)op.wd : 0.0;
            r = (float)((double)op.trust_coef * X / (Y + lam * X));
        }
    }
    return r;
}

// The trust ratio of tensor k inside pass B.  One workgroup of the tensor,
// the producer (dispatched ahead of every other tile), sums the partials
// and publishes r in the tensor's workspace word as (epoch << 32 | bits of
// r) with one relaxed device-scope atomic store; the others poll that word
// with relaxed device-scope atomic loads until it carries this launch's
// epoch (a value and its tag in one word: no ordering between two
// locations is needed).  The epoch is a workspace counter that pass A
// advances on every launch plus a value the host draws for every call, so
// every call, graph replays included, has a tag that no word left by an
// earlier call on this workspace carries (and that other contents match
// only by a 2^-32 chance).  The polling is bounded: a workgroup that gives up
// sums the partials itself, in the same order, so r is the same bits on
// every path and every kernel exits.  Every thread calls it.
template <int OPT>
__device__ __forceinline__ float tensor_ratio(const Chunk &ch, const OptParams &op, const LambWs &ws,
                                              uint32_t k, bool producer, uint32_t epoch,
                                              float *__restrict__ trust_out) {
    __shared__ float s_r;
    __shared__ int s_have;
    unsigned long long *word = ws.trust + ch.t0 + k;
    if (!producer) {
        if (threadIdx.x == 0) {
            int have = 0;
            unsigned bits = 0u;
            for (uint32_t i = 0; i < op.trust_polls; i++) {
                const unsigned long long w = __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if ((uint32_t)(w >> 32) == epoch) {
                    have = 1;
                    bits = (uint32_t)w;
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
            }
            s_have = have;
            s_r = __uint_as_float(bits);
        }
        __syncthreads();
        if (s_have) return s_r;  // workgroup-uniform
    }
    double a0, a1;
    tensor_sums(ch, ws, k, a0, a1);
    if (threadIdx.x == 0) {
        const float r = trust_ratio<OPT>(ch, op, k, a0, a1);
        if (producer) {
            __hip_atomic_store(word, ((unsigned long long)epoch << 32) | __float_as_uint(r), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            if (trust_out) trust_out[ch.t0 + k] = r;
        }
        s_r = r;
    }
    __syncthreads();
    return s_r;
}

// Pass B.  LAMB: x' = x - (lr * r_t) * u, with u recomputed from x, m', v' by
// the same operations as pass A.  LARS: v' = fma(mu, v, (lr*r_t)*(g + lambda*x)),
// x' = x - v', with g read again from the gathered message (SRC).  The
// tile's data are loaded and the step direction formed before r_t is known.
template <int SRC, int OPT>
__global__ __launch_bounds__(kWG) void opt_b_kernel(const Chunk ch, const GradArgs ga,
                                                    const OptParams op, float *__restrict__ x,
                                                    float *__restrict__ m, float *__restrict__ v,
                                                    LambWs ws, uint32_t nonce, float *__restrict__ trust_out) {
    // Workgroups [0, nt) are the producers: tile 0 of tensor k = blockIdx.x
    // (the producer of an empty tensor writes r = 1 and exits).  The rest
    // cover every tile b of the chunk (last to first when DEDLOC_B_REVERSE:
    // the re-reads start with what pass A touched last) and skip tile 0.
    uint32_t k, tile;
    const bool producer = blockIdx.x < ch.nt;
    if (producer) {
        k = blockIdx.x;
        tile = 0;
        if (ch.tile_begin[k] == ch.tile_begin[k + 1]) {
            if (threadIdx.x == 0 && trust_out) trust_out[ch.t0 + k] = 1.0f;
            return;
        }
    } else {
        const uint32_t q = blockIdx.x - ch.nt;
        const uint32_t b = DEDLOC_B_REVERSE ? gridDim.x - 1 - ch.nt - q : q;
        k = chunk_tensor(ch, b);
        tile = b - ch.tile_begin[k];
        if (tile == 0) return;
    }
    const uint64_t t_hi = ch.base + ch.start[k + 1];
    const uint64_t base = ch.base + ch.start[k] + (uint64_t)tile * kTile;
    const float lam = (ch.flags[k] & 1u) ? op.wd : 0.0f;
    const uint32_t epoch = ws.epoch[0] + nonce;  // ws.epoch: advanced by this chunk's pass A
    // the producer publishes r_t before touching its own tile (its partial
    // loads would otherwise queue behind the tile's loads)
    float lrr = producer ? op.lr * tensor_ratio<OPT>(ch, op, ws, k, true, epoch, trust_out) : 0.0f;
    float xv[kVPL][8], dv[kVPL][8], vv[kVPL][8];
    int cnt[kVPL];
#pragma unroll
    for (int r = 0; r < kVPL; r++) {
        const uint64_t e0 = base + ((uint64_t)r * kWG + threadIdx.x) * kVec;
        cnt[r] = e0 < t_hi ? (int)(t_hi - e0 < (uint64_t)kVec ? t_hi - e0 : (uint64_t)kVec) : 0;
        if (cnt[r] == 0) continue;
        load8(x, e0, cnt[r], xv[r]);
        load8(v, e0, cnt[r], vv[r]);
        if (OPT == kOptLamb) {
            float mv[8];
            load8(m, e0, cnt[r], mv);
#pragma unroll
            for (int j = 0; j < 8; j++) dv[r][j] = lamb_dir(mv[j], vv[r][j], xv[r][j], lam, op);
        } else {
            float g[8];
            load_grad<SRC>(ga, PeerTable{}, e0, cnt[r], g);
#pragma unroll
            for (int j = 0; j < 8; j++) dv[r][j] = g[j] + lam * xv[r][j];
        }
    }
    if (!producer) lrr = op.lr * tensor_ratio<OPT>(ch, op, ws, k, false, epoch, trust_out);
#pragma unroll
    for (int r = 0; r < kVPL; r++) {
        if (cnt[r] == 0) continue;
        const uint64_t e0 = base + ((uint64_t)r * kWG + threadIdx.x) * kVec;
        if (OPT == kOptLamb) {
#pragma unroll
            for (int j = 0; j < 8; j++) xv[r][j] = xv[r][j] - lrr * dv[r][j];
        } else {
#pragma unroll
            for (int j = 0; j < 8; j++) {
                vv[r][j] = fmaf(op.momentum, vv[r][j], lrr * dv[r][j]);
                xv[r][j] = xv[r][j] - vv[r][j];
            }
            store8(v, e0, cnt[r], vv[r]);
        }
        store8(x, e0, cnt[r], xv[r]);
    }
}

// ------------------------------------------------ local accumulation
// acc = fma(b, g, acc): a micro-batch of b samples with mean gradient g.
template <bool G16>
__global__ __launch_bounds__(kWG) void accumulate_kernel(float *__restrict__ acc, const void *__restrict__ grad,
                                                         uint64_t n, float b) {
    const uint64_t e0 = ((uint64_t)blockIdx.x * kWG + threadIdx.x) * kVec;
    if (e0 >= n) return;
    const int cnt = (int)(n - e0 < (uint64_t)kVec ? n - e0 : (uint64_t)kVec);
    float a[8], g[8];
    load8(acc, e0, cnt, a);
    if (G16) {
        if (cnt == kVec) {
            unpack_fp16x8(ld_stream((const u32x4 *)((const uint16_t *)grad + e0)), g);
        } else {
            for (int j = 0; j < kVec; j++) g[j] = j < cnt ? h2f(((const uint16_t *)grad)[e0 + j]) : 0.0f;
        }
    } else {
        if (cnt == kVec) {
            const f32x4 p = ld_stream((const f32x4 *)((const float *)grad + e0));
            const f32x4 q = ld_stream((const f32x4 *)((const float *)grad + e0 + 4));
            g[0] = p[0]; g[1] = p[1]; g[2] = p[2]; g[3] = p[3];
            g[4] = q[0]; g[5] = q[1]; g[6] = q[2]; g[7] = q[3];
        } else {
            for (int j = 0; j < kVec; j++) g[j] = j < cnt ? ((const float *)grad)[e0 + j] : 0.0f;
        }
    }
#pragma unroll
    for (int j = 0; j < 8; j++) a[j] = fmaf(b, g[j], a[j]);
    store8(acc, e0, cnt, a);
}

// mean = acc / count, encoded fp16; acc zeroed when reset.
__global__ __launch_bounds__(kWG) void finalize_fp16_kernel(float *__restrict__ acc, uint64_t n, float count,
                                                            uint16_t *__restrict__ codes, int reset) {
    const uint64_t e0 = ((uint64_t)blockIdx.x * kWG + threadIdx.x) * kVec;
    if (e0 >= n) return;
    const int cnt = (int)(n - e0 < (uint64_t)kVec ? n - e0 : (uint64_t)kVec);
    float a[8];
    load8(acc, e0, cnt, a);
#pragma unroll
    for (int j = 0; j < 8; j++) a[j] = a[j] / count;
    if (cnt == kVec) {
        st_msg((u32x4 *)(codes + e0), pack_fp16x8(a));
    } else {
        for (int j = 0; j < cnt; j++) codes[e0 + j] = (uint16_t)f2h(a[j]);
    }
    if (reset) {
        const float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        store8(acc, e0, cnt, z);
    }
}

// int8: one wave per 1024-element block, 16 elements per lane.
__global__ __launch_bounds__(kWG) void finalize_i8_kernel(float *__restrict__ acc, uint64_t n, float count,
                                                          int8_t *__restrict__ codes, float *__restrict__ scales,
                                                          int reset) {
    const uint64_t blk = (uint64_t)blockIdx.x * (kWG / 64) + (threadIdx.x >> 6);
    if (blk * kI8Block >= n) return;  // whole wave past the end
    float val[kI8PerLane];
    load_i8_lane(acc, n, blk, val);
#pragma unroll
    for (int j = 0; j < kI8PerLane; j++) val[j] = val[j] / count;
    float s;
    const u32x4 c = encode_i8_wave(val, s);
    store_i8_lane(codes, scales, n, blk, c, s);
    if (reset) {
        const uint64_t b0 = i8_lane_base(blk);
        if ((blk + 1) * kI8Block <= n) {
#pragma unroll
            for (int q = 0; q < 4; q++) st_stream((f32x4 *)(acc + I8_ELEM(b0, q, 0)), f32x4{0.0f, 0.0f, 0.0f, 0.0f});
        } else {
#pragma unroll
            for (int q = 0; q < 4; q++)
#pragma unroll
                for (int r = 0; r < 4; r++) {
                    const uint64_t e = I8_ELEM(b0, q, r);
                    if (e < n) acc[e] = 0.0f;
                }
        }
    }
}

__global__ __launch_bounds__(kWG) void fill_zero_kernel(uint32_t *p, uint64_t n_words) {
    const uint64_t i = (uint64_t)blockIdx.x * kWG + threadIdx.x;
    if (i < n_words) p[i] = 0u;
}

// --------------------------------------------------------------- launchers

static inline unsigned grid_for(uint64_t items, uint64_t per_block) {
    return (unsigned)((items + per_block - 1) / per_block);
}

// Launch through hipLaunchKernel, whose return value is this launch's own
// status (hipGetLastError after a <<<>>> launch would also report an error
// left pending by an earlier, unrelated call of the caller's).  The
// arguments are converted to the kernel's parameter types and held while
// the runtime copies them into the kernel arguments.
template <typename K, typename Held, size_t... I>
static hipError_t launch_held(K kernel, dim3 grid, hipStream_t s, Held &held, std::index_sequence<I...>) {
    void *argv[] = {(void *)&std::get<I>(held)...};
    return hipLaunchKernel((const void *)kernel, grid, dim3(kWG), argv, 0, s);
}

template <typename... KArgs, typename... Args>
static hipError_t launch_kernel(void (*kernel)(KArgs...), dim3 grid, hipStream_t s, Args &&...args) {
    if (grid.x == 0 || grid.y == 0) return hipSuccess;  // nothing to do
    std::tuple<KArgs...> held(std::forward<Args>(args)...);
    return launch_held(kernel, grid, s, held, std::index_sequence_for<KArgs...>{});
}

#define DEDLOC_LAUNCH(grid, kernel, s, ...) return launch_kernel((kernel), (grid), (s), __VA_ARGS__)

hipError_t launch_encode_fp16(const float *x, uint64_t n, uint16_t *codes, hipStream_t s) {
    DEDLOC_LAUNCH(dim3(grid_for(n, (uint64_t)kWG * kVec)), encode_fp16_kernel, s, x, n, codes);
}

hipError_t launch_decode_fp16(const uint16_t *codes, uint64_t n, float *out, hipStream_t s) {
    DEDLOC_LAUNCH(dim3(grid_for(n, (uint64_t)kWG * kVec)), decode_fp16_kernel, s, codes, n, out);
}

hipError_t launch_encode_i8(const float *x, uint64_t n, int8_t *codes, float *scales, hipStream_t s) {
    DEDLOC_LAUNCH(dim3(grid_for(n, (uint64_t)kI8Block * (kWG / 64))), encode_i8_kernel, s, x, n, codes, scales);
}

hipError_t launch_decode_i8(const int8_t *codes, const float *scales, uint64_t n, float *out,
                            hipStream_t s) {
    DEDLOC_LAUNCH(dim3(grid_for(n, (uint64_t)kI8Block * (kWG / 64))), decode_i8_kernel, s, codes, scales, n, out);
}

// Groups of at most this many members take the small peer batch.
constexpr uint32_t kSmallGroup = 4;

static uint32_t largest_group(const GroupTable &gt) {
    uint32_t m = 0;
    for (uint32_t g = 0; g < gt.n_groups; g++) m = std::max(m, gt.gbegin[g + 1] - gt.gbegin[g]);
    return m;
}

hipError_t launch_reduce_fp16(const GroupTable &gt, uint64_t len, const ChainArgs &ca, hipStream_t s) {
    const dim3 grid(grid_for(len, (uint64_t)kWG * kVec), gt.n_groups);
    if (ca.local.pos < 0 && largest_group(gt) <= kSmallGroup)
        DEDLOC_LAUNCH(grid, reduce_fp16_kernel<(int)kSmallGroup>, s, gt, len, ca);
    DEDLOC_LAUNCH(grid, reduce_fp16_kernel<kPeerBatch>, s, gt, len, ca);
}

hipError_t launch_reduce_i8(const GroupTable &gt, uint64_t len, const ChainArgs &ca, hipStream_t s) {
    const dim3 grid(grid_for(len, (uint64_t)kI8Block * (kWG / 64)), gt.n_groups);
    if (largest_group(gt) <= kSmallGroup) DEDLOC_LAUNCH(grid, reduce_i8_kernel<(int)kSmallGroup>, s, gt, len, ca);
    DEDLOC_LAUNCH(grid, reduce_i8_kernel<DEDLOC_I8_BATCH>, s, gt, len, ca);
}

template <int OPT>
static hipError_t launch_a(int src, const Chunk &ch, uint32_t n_tiles, const PeerTable &p, const GradArgs &ga,
                           const OptParams &op, float *x, float *m, float *v, const LambWs &ws, hipStream_t s) {
    switch (src) {
    case kSrcF32: DEDLOC_LAUNCH(dim3(n_tiles), (opt_a_kernel<kSrcF32, OPT>), s, ch, p, ga, op, x, m, v, ws);
    case kSrcFP16: DEDLOC_LAUNCH(dim3(n_tiles), (opt_a_kernel<kSrcFP16, OPT>), s, ch, p, ga, op, x, m, v, ws);
    case kSrcI8: DEDLOC_LAUNCH(dim3(n_tiles), (opt_a_kernel<kSrcI8, OPT>), s, ch, p, ga, op, x, m, v, ws);
    case kSrcPeersFP16: DEDLOC_LAUNCH(dim3(n_tiles), (opt_a_kernel<kSrcPeersFP16, OPT>), s, ch, p, ga, op, x, m, v, ws);
    case kSrcPeersFP16Chain:
        DEDLOC_LAUNCH(dim3(n_tiles), (opt_a_kernel<kSrcPeersFP16Chain, OPT>), s, ch, p, ga, op, x, m, v, ws);
    case kSrcPeersFP16Local:
        DEDLOC_LAUNCH(dim3(n_tiles), (opt_a_kernel<kSrcPeersFP16Local, OPT>), s, ch, p, ga, op, x, m, v, ws);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_opt_a(int opt, int src, const Chunk &ch, uint32_t n_tiles, const PeerTable *pt,
                        const GradArgs &ga, const OptParams &op, float *x, float *m, float *v,
                        const LambWs &ws, hipStream_t s) {
    static const PeerTable empty = {};
    const PeerTable &p = pt ? *pt : empty;
    if (opt == kOptLamb) return launch_a<kOptLamb>(src, ch, n_tiles, p, ga, op, x, m, v, ws, s);
    if (opt == kOptLars) return launch_a<kOptLars>(src, ch, n_tiles, p, ga, op, x, m, v, ws, s);
    return hipErrorInvalidValue;
}

hipError_t launch_opt_b(int opt, int src, const Chunk &ch, uint32_t n_tiles, const GradArgs &ga,
                        const OptParams &op, float *x, float *m, float *v, const LambWs &ws, uint32_t nonce,
                        float *trust_out, hipStream_t s) {
    const dim3 g(ch.nt + n_tiles);  // one producer per tensor, then every tile
    if (opt == kOptLamb)
        DEDLOC_LAUNCH(g, (opt_b_kernel<kSrcF32, kOptLamb>), s, ch, ga, op, x, m, v, ws, nonce, trust_out);
    if (opt != kOptLars) return hipErrorInvalidValue;
    switch (src) {
    case kSrcF32: DEDLOC_LAUNCH(g, (opt_b_kernel<kSrcF32, kOptLars>), s, ch, ga, op, x, m, v, ws, nonce, trust_out);
    case kSrcFP16: DEDLOC_LAUNCH(g, (opt_b_kernel<kSrcFP16, kOptLars>), s, ch, ga, op, x, m, v, ws, nonce, trust_out);
    case kSrcI8: DEDLOC_LAUNCH(g, (opt_b_kernel<kSrcI8, kOptLars>), s, ch, ga, op, x, m, v, ws, nonce, trust_out);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_accumulate(float *acc, const void *grad, bool fp16, uint64_t n, float b, hipStream_t s) {
    if (fp16) DEDLOC_LAUNCH(dim3(grid_for(n, (uint64_t)kWG * kVec)), accumulate_kernel<true>, s, acc, grad, n, b);
    DEDLOC_LAUNCH(dim3(grid_for(n, (uint64_t)kWG * kVec)), accumulate_kernel<false>, s, acc, grad, n, b);
}

hipError_t launch_finalize_fp16(float *acc, uint64_t n, float count, uint16_t *codes, int reset, hipStream_t s) {
    DEDLOC_LAUNCH(dim3(grid_for(n, (uint64_t)kWG * kVec)), finalize_fp16_kernel, s, acc, n, count, codes, reset);
}

hipError_t launch_finalize_i8(float *acc, uint64_t n, float count, int8_t *codes, float *scales, int reset,
                              hipStream_t s) {
    DEDLOC_LAUNCH(dim3(grid_for(n, (uint64_t)kI8Block * (kWG / 64))), finalize_i8_kernel, s, acc, n, count, codes,
                  scales, reset);
}

hipError_t launch_fill_zero(void *p, size_t bytes, hipStream_t s) {
    const uint64_t words = bytes / 4;
    if (words == 0) return hipSuccess;
    DEDLOC_LAUNCH(dim3(grid_for(words, kWG)), fill_zero_kernel, s, (uint32_t *)p, words);
}

}  // namespace dedloc
