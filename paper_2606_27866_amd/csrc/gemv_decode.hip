// Weight-streaming GEMMs on the vector ALUs, for batches of at most
// kGemvMaxT tokens.
//
// A routed expert then sees one or two tokens and the shared expert at most
// eight: a handful of products per weight element, far below what the
// vector ALUs sustain at HBM speed, so matrix cores gain nothing.  What
// matters is how fast the kept weights (Eq. 4: the first k_e channels of
// each routed expert, plus the shared expert) stream in.  An MFMA fragment
// would fix the load layout to 64 bytes of each of 16 rows per instruction;
// here each load instruction covers two weight rows of 512 contiguous bytes
// -- whole 128-byte lines -- and carries the non-temporal hint.  On this chip
// that streams at about 7.1 TB/s against 6.3 for plain loads, while
// non-temporal half-line reads fall to 5.8.
//
// A tile is 16 channels (gate/up) or 16 output columns (down) of one
// segment, for every row of the segment.  The four waves split the
// reduction into 256-deep batches (wave q: batches q, q+4, ...).  In a
// batch, lane l holds the 8 consecutive K elements of chunk l%32 of tile
// rows 2i + l/32 (i < 8), and the same 8 elements of every token row, and
// accumulates their products with v_dot2_f32_bf16 in fp32.  A row's partial
// sums end up spread over the 32 lanes of a half-wave and over the waves:
// a butterfly over the half-wave first, then a sum over the waves in wave
// order through LDS (a fixed order: the result is deterministic).
#include "mfma_tile.h"

namespace flexmoe {

namespace {
constexpr int GV_WAVES = 4;
constexpr int GV_KB = 256;                 // K elements per batch (32 chunks of 8)
constexpr int GV_ROWS = kDecBN;            // weight rows per tile
constexpr int GV_NI = GV_ROWS / 2;         // load instructions per weight matrix per batch
constexpr int kNT = 2;                     // cache-policy operand of a buffer load: non-temporal
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
using mfma::kOOB;
using mfma::make_rsrc;

// acc + the dot product of two runs of 8 bf16 (fp32 products and sums).  The
// pairs are taken with shufflevector from the whole 8-element vectors: a
// bit_cast of a single element of the 4-dword vector compiled to element 0
// every time.
__device__ __forceinline__ float dot8(u32x4 a, u32x4 b, float acc) {
    const bf16x8 x = __builtin_bit_cast(bf16x8, a), y = __builtin_bit_cast(bf16x8, b);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(x, x, 0, 1), __builtin_shufflevector(y, y, 0, 1),
                                          acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(x, x, 2, 3), __builtin_shufflevector(y, y, 2, 3),
                                          acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(x, x, 4, 5), __builtin_shufflevector(y, y, 4, 5),
                                          acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(x, x, 6, 7), __builtin_shufflevector(y, y, 6, 7),
                                          acc, false);
    return acc;
}

// Sums each of V values over the 32 lanes of a half-wave (lane bits 0..4).
// Step b pairs lanes whose bit b differs; of the n values a lane still holds,
// the one with bit b clear keeps the lower n/2 (adding its partner's) and the
// one with bit b set the upper n/2, so each step halves the values held and
// the exchanges total about V per lane.  Once a lane holds one value, the
// remaining steps add it to the partner's.  Afterwards value q < max(V/32, 1)
// of lane l is the half-wave total of value index gv_base<V>(l) + q.
template <int V>
__device__ __forceinline__ int gv_base(int lane) {
    int base = 0, n = V;
#pragma unroll
    for (int b = 0; b < 5; ++b) {
        if (n > 1) {
            n >>= 1;
            if ((lane >> b) & 1) base += n;
        }
    }
    return base;
}

template <int N, int B>
struct HalfWaveSum {
    static __device__ __forceinline__ void run(float* v, int lane) {
        if constexpr (B < 5) {
            const bool hi = (lane >> B) & 1;
            if constexpr (N > 1) {
                constexpr int H = N / 2;
#pragma unroll
                for (int j = 0; j < H; ++j) {
                    const float send = hi ? v[j] : v[H + j];
                    const float keep = hi ? v[H + j] : v[j];
                    v[j] = keep + __shfl_xor(send, 1 << B, 64);
                }
                HalfWaveSum<H, B + 1>::run(v, lane);
            } else {
                v[0] += __shfl_xor(v[0], 1 << B, 64);
                HalfWaveSum<1, B + 1>::run(v, lane);
            }
        }
    }
};

// Reduce the V per-lane partial sums of every wave and leave, in red, the
// half-wave totals of each wave: red[(wave * 2 + half) * V + index].
template <int V>
__device__ __forceinline__ void gv_reduce(float (&acc)[V], float* red, int wave, int lane) {
    HalfWaveSum<V, 0>::run(acc, lane);
    constexpr int NQ = V >= 32 ? V / 32 : 1;
    const int base = gv_base<V>(lane);
    // with fewer than 32 values, lanes that differ only in the bits past
    // log2(V) hold the same totals: the lowest of them writes
    const bool writer = V >= 32 || (lane & 31) < V;
    if (writer) {
        float* dst = red + (wave * 2 + (lane >> 5)) * V + base;
#pragma unroll
        for (int q = 0; q < NQ; ++q) dst[q] = acc[q];
    }
    __syncthreads();
}

}  // namespace

// NR: the most rows a segment can hold (the launch's token count rounded up
// to a power of two); R = the segment's rows <= NR.
template <int NR>
__global__ __launch_bounds__(64 * GV_WAVES, NR <= 2 ? 4 : NR == 4 ? 3 : 2) void gemv1_kernel(Gemm1Params<bf16_t> p) {
    constexpr int V = 2 * GV_NI * NR;  // [gate|up][instruction i][row r]
    __shared__ float red[GV_WAVES * 2 * V];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    int s, ntile;
    SegMeta sm;
    if (!tile_of(p, blockIdx.x, s, sm, ntile)) return;  // workgroup-uniform
    const bool shared = sm.e < 0;
    const RoutedWeights rw = shared ? RoutedWeights{0, p.Is, 0} : routed_weights(p, sm);
    const int d = p.d;
    const __amdgpu_buffer_rsrc_t rg = make_rsrc((shared ? p.sg : p.wg) + rw.base, (size_t)rw.rows * d);
    const __amdgpu_buffer_rsrc_t ru = make_rsrc((shared ? p.su : p.wu) + rw.base, (size_t)rw.rows * d);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.x, (size_t)p.tokens * d);
    const int R = min(sm.rows, NR);
    const int ck = (lane & 31) * 8;   // K offset of this lane's chunk inside a batch
    const int half = lane >> 5;
    // byte offsets of the lane's chunk of batch 0 (the batch start is the
    // scalar offset); kOOB (the load returns zeros) for rows past the GEMM
    uint32_t xoff[NR], woff[GV_NI];
    // token of each row: routed rows are gathered through perm, all NR
    // entries requested together (rows past the segment read its last
    // row's, unused)
    int tok[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) tok[r] = r;
    if (!shared) {
        const int32_t* pr = p.perm + sm.row0;
#pragma unroll
        for (int r = 0; r < NR; ++r) tok[r] = pr[max(min(r, R - 1), 0)];
#pragma unroll
        for (int r = 0; r < NR; ++r) tok[r] = (int)min((unsigned)(tok[r] / p.top_k), (unsigned)(p.tokens - 1));
    }
#pragma unroll
    for (int r = 0; r < NR; ++r) xoff[r] = r < R ? (uint32_t)(((size_t)tok[r] * d + ck) * 2) : kOOB;
#pragma unroll
    for (int i = 0; i < GV_NI; ++i) {
        const int c = ntile * GV_ROWS + 2 * i + half;  // channel; the GEMM computes c < kg
        woff[i] = c < sm.kg ? (uint32_t)(((size_t)c * d + ck) * 2) : kOOB;
    }
    float acc[V];
#pragma unroll
    for (int j = 0; j < V; ++j) acc[j] = 0.f;
    for (int kb = wave * GV_KB; kb < d; kb += GV_WAVES * GV_KB) {
        const bool kval = kb + ck < d;  // d % 8 == 0: a chunk is wholly inside or outside
        const uint32_t soff = (uint32_t)kb * 2u;
        u32x4 g[GV_NI], u[GV_NI], xv[NR];
#pragma unroll
        for (int i = 0; i < GV_NI; ++i) {
            const uint32_t o = kval ? woff[i] : kOOB;
            g[i] = __builtin_amdgcn_raw_buffer_load_b128(rg, o, soff, kNT);
            u[i] = __builtin_amdgcn_raw_buffer_load_b128(ru, o, soff, kNT);
        }
#pragma unroll
        for (int r = 0; r < NR; ++r)
            xv[r] = __builtin_amdgcn_raw_buffer_load_b128(rx, kval ? xoff[r] : kOOB, soff, 0);
        // every load of the batch is issued before the first product
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < GV_NI; ++i)
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                if (r > 0 && r >= R) break;  // workgroup-uniform (R >= 1)
                acc[i * NR + r] = dot8(g[i], xv[r], acc[i * NR + r]);
                acc[(GV_NI + i) * NR + r] = dot8(u[i], xv[r], acc[(GV_NI + i) * NR + r]);
            }
    }
    gv_reduce<V>(acc, red, wave, lane);
    // one output (tile row, token row) per thread: H = silu(g) * u; channels
    // in [kk, kk8) are written as zeros (the down GEMM reads 8-wide chunks)
    bf16_t* Hb = shared ? p.Hs : p.H + (size_t)sm.row0 * p.I;
    const int ldh = shared ? p.Is : p.I;
    const int kk8 = min((sm.kg + 7) & ~7, ldh);
    const int o = threadIdx.x;
    if (o < GV_ROWS * R) {
        const int row = o / R, r = o - row * R;  // tile row = 2i + half
        const int i = row >> 1, h = row & 1;
        const int ch = ntile * GV_ROWS + row;
        if (ch < kk8) {
            float gs = 0.f, us = 0.f;
#pragma unroll
            for (int w = 0; w < GV_WAVES; ++w) {
                gs += red[(w * 2 + h) * V + i * NR + r];
                us += red[(w * 2 + h) * V + (GV_NI + i) * NR + r];
            }
            Hb[(size_t)r * ldh + ch] = ch < sm.kk ? f32_to_bf16(silu_fast(gs) * us) : (bf16_t)0;
        }
    }
}

template <int NR>
__global__ __launch_bounds__(64 * GV_WAVES, NR <= 4 ? 4 : 3) void gemv2_kernel(Gemm2Params<bf16_t> p) {
    constexpr int V = GV_NI * NR;  // [instruction i][row r]
    __shared__ float red[GV_WAVES * 2 * V];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    int s, local;
    SegMeta sm;
    if (!tile_of(p, blockIdx.x, s, sm, local)) return;  // workgroup-uniform
    const int d = p.d;
    const int nt = ceil_div(d, GV_ROWS);
    const int split = local / nt, ntile = local % nt;  // split > 0 only for the shared expert
    const bool shared = sm.e < 0;
    const RoutedWeights rw = shared ? RoutedWeights{0, 0, p.Is} : routed_weights(p, sm);
    const int ldh = shared ? p.Is : p.I;  // activation row stride
    const bf16_t* Hb = shared ? p.Hs : p.H + (size_t)sm.row0 * p.I;
    const int kbeg = shared ? split * p.ks2 : 0;
    const int kend = shared ? min(sm.kg, kbeg + p.ks2) : sm.kg;
    const int R = min(sm.rows, NR);
    const __amdgpu_buffer_rsrc_t rwd = make_rsrc(shared ? p.sd : p.wd + rw.base, (size_t)d * rw.ldd);
    const __amdgpu_buffer_rsrc_t rh = make_rsrc(Hb, (size_t)max(R, 1) * ldh);
    const int ck = (lane & 31) * 8;
    const int half = lane >> 5;
    uint32_t hoff[NR], woff[GV_NI];
#pragma unroll
    for (int r = 0; r < NR; ++r) hoff[r] = r < R ? (uint32_t)(((size_t)r * ldh + ck) * 2) : kOOB;
#pragma unroll
    for (int i = 0; i < GV_NI; ++i) {
        const int n = ntile * GV_ROWS + 2 * i + half;  // output column
        woff[i] = n < d ? (uint32_t)(((size_t)n * rw.ldd + ck) * 2) : kOOB;
    }
    float acc[V];
#pragma unroll
    for (int j = 0; j < V; ++j) acc[j] = 0.f;
    // a chunk is read when it starts before kend; the activations are zero
    // from k_e to the chunk-aligned end, and the weights there are real
    // (finite) values, so their products are exact zeros
    for (int kb = kbeg + wave * GV_KB; kb < kend; kb += GV_WAVES * GV_KB) {
        const bool kval = kb + ck < kend;
        const uint32_t soff = (uint32_t)kb * 2u;
        u32x4 w[GV_NI], hv[NR];
#pragma unroll
        for (int i = 0; i < GV_NI; ++i)
            w[i] = __builtin_amdgcn_raw_buffer_load_b128(rwd, kval ? woff[i] : kOOB, soff, kNT);
#pragma unroll
        for (int r = 0; r < NR; ++r)
            hv[r] = __builtin_amdgcn_raw_buffer_load_b128(rh, kval ? hoff[r] : kOOB, soff, 0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < GV_NI; ++i)
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                if (r > 0 && r >= R) break;  // workgroup-uniform (R >= 1)
                acc[i * NR + r] = dot8(w[i], hv[r], acc[i * NR + r]);
            }
    }
    gv_reduce<V>(acc, red, wave, lane);
    bf16_t* Ob = shared ? p.Os + (size_t)split * p.tokens * d : p.O + (size_t)sm.row0 * d;
    const int o = threadIdx.x;
    if (o < GV_ROWS * R) {
        const int row = o / R, r = o - row * R;
        const int i = row >> 1, h = row & 1;
        const int n = ntile * GV_ROWS + row;
        if (n < d) {
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < GV_WAVES; ++w) sum += red[(w * 2 + h) * V + i * NR + r];
            Ob[(size_t)r * d + n] = f32_to_bf16(sum);
        }
    }
}

hipError_t launch_gemm1_decode(const Gemm1Params<bf16_t>& p, int tiles, hipStream_t s) {
    if (tiles <= 0 || p.tokens <= 0 || p.tokens > kGemvMaxT) return hipSuccess;
    if (p.tokens <= 1) gemv1_kernel<1><<<tiles, 64 * GV_WAVES, 0, s>>>(p);
    else if (p.tokens <= 2) gemv1_kernel<2><<<tiles, 64 * GV_WAVES, 0, s>>>(p);
    else if (p.tokens <= 4) gemv1_kernel<4><<<tiles, 64 * GV_WAVES, 0, s>>>(p);
    else gemv1_kernel<8><<<tiles, 64 * GV_WAVES, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_gemm2_decode(const Gemm2Params<bf16_t>& p, int tiles, hipStream_t s) {
    if (tiles <= 0 || p.tokens <= 0 || p.tokens > kGemvMaxT) return hipSuccess;
    if (p.tokens <= 1) gemv2_kernel<1><<<tiles, 64 * GV_WAVES, 0, s>>>(p);
    else if (p.tokens <= 2) gemv2_kernel<2><<<tiles, 64 * GV_WAVES, 0, s>>>(p);
    else if (p.tokens <= 4) gemv2_kernel<4><<<tiles, 64 * GV_WAVES, 0, s>>>(p);
    else gemv2_kernel<8><<<tiles, 64 * GV_WAVES, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace flexmoe
