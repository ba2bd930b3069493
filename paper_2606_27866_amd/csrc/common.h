// Shared definitions of the FlexMoE HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace flexmoe {

constexpr int kWave = 64;
constexpr int kMaxExperts = 256;
constexpr int kMaxTopK = 16;
constexpr int kRouteTokens = 16;   // tokens per routing block (= dispatch chunk)
constexpr int kSmallAssign = 1024; // T * top_k at or below which one workgroup dispatches
                                   // (every decode-sized batch: T <= 64, top_k <= 16)
constexpr int kSmallWaves = 16;    // waves of that workgroup
constexpr int kSmallRouteT = 64;   // above this many tokens route_kernel routes first (one token
                                   // per wave on several compute units) and the workgroup only
                                   // dispatches.  Up to 64 the workgroup also routes: submitted
                                   // before the shared expert's GEMMs, it holds a compute unit,
                                   // where a second kernel would wait for one behind their
                                   // workgroups (1-2 % per decode step at 17-64 tokens)

typedef uint16_t bf16_t;           // raw bf16 bits in memory
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// Round to nearest even (v_cvt_pk_bf16_f32, which also keeps NaNs NaN and
// fp32 denormals as bf16 denormals: the kernels run with denormals
// preserved).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    return __builtin_bit_cast(bf16_t, (__bf16)f);
}
// Two values rounded as above in one instruction: lo in bits 0-15.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(float2_t{lo, hi}, bf16x2_t));
}

// x * sigmoid(x) in fp32 via the hardware exp2 and reciprocal (1 ulp each).
// For x -> -inf the product tends to -0, for x -> +inf to x.
__device__ __forceinline__ float silu_fast(float x) {
    const float e = __builtin_amdgcn_exp2f(-x * 1.4426950408889634f);
    return x * __builtin_amdgcn_rcpf(1.0f + e);
}

__host__ __device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Per-segment metadata written by the dispatch kernel.  With a shared expert,
// segment 0 is the shared expert (rows = tokens) and segment 1 + e is routed
// expert e; without one, segment e is expert e.  Routed rows are grouped by
// the dispatch permutation.
struct SegMeta {
    int32_t row0;   // first row of the segment in the routed row space
    int32_t rows;   // rows of the segment (0 for inactive experts)
    int32_t kk;     // channels of the segment (k_e, or I_shared)
    int32_t ch0;    // clipped weight layout: the expert's first packed channel
    int32_t kg;     // channels the GEMMs compute: kk, or kk aligned up in the
                    // bucketed forward (the extra channels' activations are 0)
    int32_t e;      // routed expert id (-1: the shared expert)
    int32_t prow0;  // routed segments: first row in the padded row space, where
                    // every segment takes packed_width(rows) rows (the column
                    // offset of the segment in transposed activation copies)
    int32_t rt0;    // routed segments: row tiles (of the gate/up tile height) of
                    // the routed segments before this one
};

// Channels an expert occupies in the clipped (offline) weight layout: k_e
// rounded up to 8, so every packed row starts on a 16-byte boundary.
__host__ __device__ __forceinline__ int packed_width(int k) { return (k + 7) & ~7; }

// Tile shapes of one GEMM-kernel family; the dispatch kernel builds the tile
// tables with the same numbers the GEMM kernels use.
struct TileShape {
    int32_t bm1, bn1;   // gate/up GEMM: rows x channels per tile
    int32_t bm2, bn2;   // down GEMM: rows x output columns per tile
    int32_t ks2;        // > 0: the shared expert's down GEMM is split into
                        // reductions of ks2 channels (one tile set each)
};

// Lane-shift building block of the wave scans: v of the lane DPP control
// CTRL names (row_shr:n within rows of 16 lanes, or the gfx9 row broadcasts
// of lane 15 / lane 31), 0 where that lane is outside the row or the row is
// not in ROW_MASK.  A DPP move costs about as much as an ALU op, where a
// ds_bpermute shuffle waits on the LDS crossbar.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_shift(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, ROW_MASK, 0xf, false);
}

// Wave-wide inclusive prefix sum of an int (64 lanes, all active): a
// Hillis-Steele scan inside each row of 16 lanes (row_shr 1, 2, 4, 8), then
// row 0's total added to row 1 and row 2's to row 3 (row_bcast:15 into rows
// 1 and 3), then the total of rows 0-1 to rows 2 and 3 (row_bcast:31).
__device__ __forceinline__ int wave_incl_scan(int v) {
    v += dpp_shift<0x111, 0xf>(v);
    v += dpp_shift<0x112, 0xf>(v);
    v += dpp_shift<0x114, 0xf>(v);
    v += dpp_shift<0x118, 0xf>(v);
    v += dpp_shift<0x142, 0xa>(v);
    v += dpp_shift<0x143, 0xc>(v);
    return v;
}

// Value of lane 63 (e.g. the total of an inclusive scan), in every lane.
__device__ __forceinline__ int lane63(int v) { return __builtin_amdgcn_readlane(v, 63); }

// Sum of a float over the wave (64 lanes, all active), in every lane: the
// scan above on the float bits, read from lane 63.  The order of the
// additions is fixed, so the sum is deterministic.
__device__ __forceinline__ float wave_total_f(float v) {
#define FLEXMOE_FSTEP(C, M) v += __int_as_float(dpp_shift<C, M>(__float_as_int(v)))
    FLEXMOE_FSTEP(0x111, 0xf);
    FLEXMOE_FSTEP(0x112, 0xf);
    FLEXMOE_FSTEP(0x114, 0xf);
    FLEXMOE_FSTEP(0x118, 0xf);
    FLEXMOE_FSTEP(0x142, 0xa);
    FLEXMOE_FSTEP(0x143, 0xc);
#undef FLEXMOE_FSTEP
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

}  // namespace flexmoe

namespace flexmoe {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Segment owning tile L: the largest s with tstart[s] <= L (segments with no
// tiles share their start with the next one and are skipped).  tstart is
// non-decreasing, so that is one less than the number of entries <= L: each
// lane reads entries lane, lane + 64, ... all at once and ballots count them
// -- one memory round trip at the start of every GEMM workgroup, where a
// binary search took log2(nseg) dependent ones.  All 64 lanes must be active
// (every caller runs it first thing, workgroup-uniform).
__device__ __forceinline__ int find_segment(const int32_t* tstart, int nseg, int L) {
    constexpr int NJ = (kMaxExperts + 1 + 63) / 64;  // segments: the experts and a shared expert
    const int lane = threadIdx.x & 63;
    int v[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) v[j] = tstart[min(j * 64 + lane, nseg)];  // tstart holds nseg + 1 entries
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < NJ; ++j) cnt += __popcll(__ballot(j * 64 + lane < nseg && v[j] <= L));
    return cnt - 1;
}

// Fragment-blocked layout of a [rows][C] bf16 matrix (C a multiple of 8):
// 32-row x 8-column blocks of 512 bytes, block (r/32, c/8) at element
// ((r/32) * (C/8) + c/8) * 256, and inside it element
// (((c/4) % 2) * 32 + r % 32) * 4 + c % 4 -- the order in which a wave's 64
// lanes hold runs of 4 consecutive columns of 32 rows (lane -> row lane % 32,
// columns 4 * (lane / 32) ..), so that the wave's 8-byte accesses cover 512
// contiguous bytes.  R rows take ceil(R/32) * 32 * C elements.
__host__ __device__ __forceinline__ size_t frag_blocked(size_t r, int c, int C) {
    return (((r >> 5) * (size_t)(C >> 3) + (size_t)(c >> 3)) << 8) + (size_t)((((c >> 2) & 1) << 5) + (r & 31)) * 4 +
           (c & 3);
}

// Zero the bf16 elements at positions >= nvalid of an 8-element vector.
__device__ __forceinline__ u32x4 mask_tail_bf16(u32x4 v, int nvalid) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if (2 * i >= nvalid) v[i] = 0u;
        else if (2 * i + 1 >= nvalid) v[i] &= 0xffffu;
    }
    return v;
}

}  // namespace flexmoe
