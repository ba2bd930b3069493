// Weight-streaming grouped GEMMs for decode-sized token counts (T <= 64).
//
// With a few tokens per expert the layer is bound by reading the kept
// weights (Eq. 4: the first k_e channels of each routed expert, plus the
// shared expert), so these kernels read every kept weight byte exactly once,
// straight from HBM into MFMA fragments, with many waves in flight.
//
// A workgroup owns one tile: 16 channels (gate/up) or 16 output columns
// (down) of one segment, for every row (token) of that segment (<= 64 rows =
// up to four 16-wide MFMA column blocks).  Its four waves split the
// reduction: wave q takes the 256-wide K batches q, q+4, q+8, ...; the four
// partial sums are added in wave order through LDS (a fixed order, so the
// result is deterministic).  Small tiles keep all CUs streaming to the end.
//
// The tile's 16 weight rows are the M side of v_mfma_f32_16x16x32_bf16, the
// tokens the N side.  A 256-wide batch is eight MFMA steps of 32: at step j
// lane l holds weight row l%16 and the 8 K elements 32*j + 8*(l/16) .. +8,
// so one load instruction reads 64 contiguous bytes of each of 16 rows and
// the next one the other half of the same cache lines.  Token fragments are
// read with the same K mapping, so every product pairs equal K indices.
//
// gate/up: SwiGLU is applied to the reduced sums; H is written as bf16.
// down: the reduction runs over the segment's kept channels; the shared
//   expert's reduction is split into chunks of I channels (one routed
//   expert's worth), each chunk writing its own partial rows, which the
//   combine sums in a fixed order.
#include <type_traits>

#include "mfma_tile.h"

namespace flexmoe {

namespace {
constexpr int DCH = 16;    // channels (gate/up) or output columns (down) per tile
constexpr int DKB = 256;   // K elements per batch
constexpr int DWAVES = 4;  // waves per workgroup, splitting K
typedef float floatx4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 as_frag(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Sum NACC float4 accumulators per lane over the four waves in wave order;
// wave 0 ends up with the total.  red holds DWAVES * NACC * 64 float4.
template <int NACC>
__device__ __forceinline__ void reduce_waves(floatx4_t (&acc)[NACC], float4* red, int wave, int lane) {
    if (wave > 0) {
#pragma unroll
        for (int i = 0; i < NACC; ++i)
            red[((wave - 1) * NACC + i) * 64 + lane] = make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int w = 1; w < DWAVES; ++w)
#pragma unroll
            for (int i = 0; i < NACC; ++i) {
                const float4 v = red[((w - 1) * NACC + i) * 64 + lane];
                acc[i][0] += v.x;
                acc[i][1] += v.y;
                acc[i][2] += v.z;
                acc[i][3] += v.w;
            }
    }
}
}  // namespace

// NFM: most 16-token blocks a segment can hold (1 for T <= 16: the kernel
// then needs far fewer registers and more workgroups fit per compute unit).
template <int NFM>
__global__ __launch_bounds__(64 * DWAVES, NFM == 1 ? 4 : 1) void gemm1_decode_kernel(Gemm1Params<bf16_t> p) {
    __shared__ float4 red[(DWAVES - 1) * 2 * NFM * 64];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    int s, ntile;  // one row tile per segment (rows <= 64): the local tile is the channel tile
    SegMeta sm;
    if (!tile_of(p, blockIdx.x, s, sm, ntile)) return;  // workgroup-uniform
    const bool shared = sm.e < 0;
    const size_t wofs = shared ? 0 : routed_weights(p, sm).base;
    const bf16_t* Wg = (shared ? p.sg : p.wg) + wofs;
    const bf16_t* Wu = (shared ? p.su : p.wu) + wofs;
    const int d = p.d;
    const int g = lane >> 4;  // K group of this lane
    const int c = ntile * DCH + (lane & 15);
    const bool cval = c < sm.kg;  // channels the GEMM computes
    const int nf = min(ceil_div(sm.rows, 16), NFM);  // token blocks (rows <= 16 * NFM)

    const bf16_t* xrow[NFM];
#pragma unroll
    for (int f = 0; f < NFM; ++f) {
        const int r = f * 16 + (lane & 15);
        xrow[f] = nullptr;
        if (f < nf && r < sm.rows) {
            const int t = shared ? r
                                 : (int)min((unsigned)(p.perm[sm.row0 + r] / p.top_k), (unsigned)(p.tokens - 1));
            xrow[f] = p.x + (size_t)t * d;
        }
    }
    floatx4_t acc[2 * NFM];  // [0, NFM) gate, [NFM, 2 NFM) up, per token block
#pragma unroll
    for (int i = 0; i < 2 * NFM; ++i) acc[i] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    const u32x4 zero = {0u, 0u, 0u, 0u};
    const bf16_t* wgr = Wg + (size_t)c * d;
    const bf16_t* wur = Wu + (size_t)c * d;
    for (int kb = wave * DKB; kb < d; kb += DWAVES * DKB) {
        const int k0 = kb + g * 8;  // + 32*j at step j
        u32x4 wgv[8], wuv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const bool ok = cval && k0 + j * 32 < d;  // d % 8 == 0
            wgv[j] = ok ? *reinterpret_cast<const u32x4*>(wgr + k0 + j * 32) : zero;
            wuv[j] = ok ? *reinterpret_cast<const u32x4*>(wur + k0 + j * 32) : zero;
        }
#pragma unroll
        for (int f = 0; f < NFM; ++f) {
            if (f >= nf) break;  // workgroup-uniform
            u32x4 xv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                xv[j] = (xrow[f] && k0 + j * 32 < d) ? *reinterpret_cast<const u32x4*>(xrow[f] + k0 + j * 32) : zero;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_frag(wgv[j]), as_frag(xv[j]), acc[f], 0, 0, 0);
                acc[NFM + f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_frag(wuv[j]), as_frag(xv[j]), acc[NFM + f], 0, 0,
                                                                       0);
            }
        }
    }
    reduce_waves(acc, red, wave, lane);
    if (wave != 0) return;
    // D[m][n]: lane holds channels m = 4*(lane/16) + i of token n = lane%16
    bf16_t* Hb = shared ? p.Hs : p.H + (size_t)sm.row0 * p.I;
    const int ldh = shared ? p.Is : p.I;
    const int kk8 = min((sm.kg + 7) & ~7, ldh);  // [kk, kk8) written as zeros
#pragma unroll
    for (int f = 0; f < NFM; ++f) {
        if (f >= nf) break;
        const int r = f * 16 + (lane & 15);
        if (r >= sm.rows) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int ch = ntile * DCH + 4 * g + i;
            if (ch < kk8)
                Hb[(size_t)r * ldh + ch] = ch < sm.kk ? f32_to_bf16(silu_fast(acc[f][i]) * acc[NFM + f][i]) : (bf16_t)0;
        }
    }
}

template <int NFM>
__global__ __launch_bounds__(64 * DWAVES) void gemm2_decode_kernel(Gemm2Params<bf16_t> p) {
    __shared__ float4 red[(DWAVES - 1) * NFM * 64];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    int s, local;
    SegMeta sm;
    if (!tile_of(p, blockIdx.x, s, sm, local)) return;  // workgroup-uniform
    const int d = p.d;
    const int nt = ceil_div(d, DCH);
    const int split = local / nt, ntile = local % nt;  // split > 0 only for the shared expert
    const bool shared = sm.e < 0;
    const RoutedWeights rw = shared ? RoutedWeights{0, 0, p.Is} : routed_weights(p, sm);
    const int ldh = shared ? p.Is : p.I;  // H row stride
    const bf16_t* Hb = shared ? p.Hs : p.H + (size_t)sm.row0 * p.I;
    const bf16_t* Wd = shared ? p.sd : p.wd + rw.base;
    const int kbeg = shared ? split * p.ks2 : 0;
    const int kend = shared ? min(sm.kg, kbeg + p.ks2) : sm.kg;
    const int g = lane >> 4;
    const int n = ntile * DCH + (lane & 15);
    const bool nval = n < d;
    const int nf = min(ceil_div(sm.rows, 16), NFM);
    const bf16_t* hrow[NFM];
#pragma unroll
    for (int f = 0; f < NFM; ++f) {
        const int r = f * 16 + (lane & 15);
        hrow[f] = (f < nf && r < sm.rows) ? Hb + (size_t)r * ldh : nullptr;
    }
    floatx4_t acc[NFM];
#pragma unroll
    for (int f = 0; f < NFM; ++f) acc[f] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    const u32x4 zero = {0u, 0u, 0u, 0u};
    const bf16_t* wrow = Wd + (size_t)n * rw.ldd;
    // a chunk is used when it starts before kend; H is zero past k_e within
    // the chunk-aligned end, and W_down columns there are real (finite)
    // weights, so their products are exact zeros
    for (int kb = kbeg + wave * DKB; kb < kend; kb += DWAVES * DKB) {
        const int k0 = kb + g * 8;  // + 32*j at step j
        u32x4 wv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            wv[j] = (nval && k0 + j * 32 < kend) ? *reinterpret_cast<const u32x4*>(wrow + k0 + j * 32) : zero;
#pragma unroll
        for (int f = 0; f < NFM; ++f) {
            if (f >= nf) break;
            u32x4 hv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                hv[j] = (hrow[f] && k0 + j * 32 < kend) ? *reinterpret_cast<const u32x4*>(hrow[f] + k0 + j * 32) : zero;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_frag(wv[j]), as_frag(hv[j]), acc[f], 0, 0, 0);
        }
    }
    reduce_waves(acc, red, wave, lane);
    if (wave != 0) return;
    // D[m][n']: lane holds output columns m = 4*(lane/16) + i of row n' = lane%16
    bf16_t* Ob = shared ? p.Os + (size_t)split * p.tokens * d : p.O + (size_t)sm.row0 * d;
#pragma unroll
    for (int f = 0; f < NFM; ++f) {
        if (f >= nf) break;
        const int r = f * 16 + (lane & 15);
        if (r >= sm.rows) continue;
        const int col = ntile * DCH + 4 * g;
        if (col + 3 < d) {
            const uint32_t lo = (uint32_t)f32_to_bf16(acc[f][0]) | ((uint32_t)f32_to_bf16(acc[f][1]) << 16);
            const uint32_t hi = (uint32_t)f32_to_bf16(acc[f][2]) | ((uint32_t)f32_to_bf16(acc[f][3]) << 16);
            *reinterpret_cast<uint2*>(Ob + (size_t)r * d + col) = make_uint2(lo, hi);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (col + i < d) Ob[(size_t)r * d + col + i] = f32_to_bf16(acc[f][i]);
        }
    }
}

// ---- Wide tiles ------------------------------------------------------------
//
// The 16-channel tiles above read a segment's token rows once per 16 weight
// rows -- at 64 tokens, for the shared expert, four times the weight bytes,
// from L2, one 16-token block after another.  With enough rows per segment
// (the shared expert above kDecodeWideSharedT tokens, routed experts above
// kDecodeWideT tokens once T * k >= 8 E) the GEMMs take tiles of 64
// channels (gate/up) or 64 output columns (down) instead: wave w
// owns 16 of them over the whole reduction, and the four waves share the
// segment's token rows through LDS.  Per 256-deep K batch the workgroup
// copies the rows into LDS once (buffer_load ... lds; as many 16-row blocks
// as T needs, so small batches keep more workgroups per compute unit); the
// next batch's rows and weights are in flight while the current batch is
// multiplied.  LDS row r keeps its 16-B chunk c at position c ^ (r & 15):
// the 16 lanes of one fragment read (16 rows, one chunk) then cover all 64
// banks.
namespace {
constexpr int WCH = kDecWideBN;         // channels / output columns per wide tile
constexpr int WKB = 256;                // K per batch
constexpr int WSTEPS = WKB / 32;        // MFMA steps per batch
constexpr int WROWB = WKB * 2;          // LDS bytes per staged row
constexpr int WCHUNKS = WROWB / 16;     // 16-byte chunks per staged row
constexpr int WRPI = 1024 / WROWB;      // staged rows one DMA instruction (64 lanes x 16 B) fills
static_assert(WCHUNKS % 16 == 0 && 1024 % WROWB == 0,
              "the chunk swizzle XORs with 4 row bits; a DMA instruction fills whole rows");
}  // namespace

// 16-row blocks staged per batch for a launch over T tokens (every segment
// has at most T rows) and the dynamic LDS that takes: two stages.
__host__ __device__ __forceinline__ int wide_blocks(int tokens) { return ceil_div(min(tokens, kDecodeMaxT), 16); }
__host__ __device__ __forceinline__ size_t wide_lds_bytes(int tokens) {
    return (size_t)2 * wide_blocks(tokens) * 16 * WROWB;
}

// SB: 16-row blocks staged per batch, wide_blocks(T) (a template parameter:
// a fixed count of row copies keeps the compiler's count of outstanding loads
// exact).
template <bool kGateUp, int SB>
__device__ __forceinline__ void wide_tile(const Gemm1Params<bf16_t>& p1, const Gemm2Params<bf16_t>& p2,
                                          unsigned char* smem) {
    using namespace mfma;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    int s, local;  // one row tile per segment (rows <= 64): `local` numbers the segment's 64-wide tiles
    SegMeta sm;
    if (!(kGateUp ? tile_of(p1, blockIdx.x, s, sm, local) : tile_of(p2, blockIdx.x, s, sm, local))) return;
    const bool shared = sm.e < 0;
    const int R = sm.rows;  // token rows, <= kDecodeMaxT
    const int d = kGateUp ? p1.d : p2.d;
    // weight rows of the tile: channels c < kg (gate/up) or output columns n < d (down)
    const int nrows = kGateUp ? sm.kg : d;
    int tile = local, split = 0;
    if (!kGateUp) {  // the shared expert's split reduction: chunk `split`
        const int nt = ceil_div(d, WCH);
        split = local / nt;
        tile = local - split * nt;
    }
    // the reduction: all of d (gate/up), the kept channels (routed down) or
    // channel chunk `split` of I_s (shared down)
    const int ks = kGateUp ? d : shared ? (p2.ks2 > 0 ? p2.ks2 : p2.Is) : sm.kg;
    const int kbeg = split * ks;
    const int K = kGateUp ? d : shared ? min(p2.Is - kbeg, ks) : sm.kg;
    if (K <= 0) return;  // workgroup-uniform

    // token rows: x [T][d] (routed rows gathered through perm), the routed
    // activations H [A][I] of the segment, or the shared Hs [T][I_s] from kbeg
    const int lda = kGateUp ? d : shared ? p2.Is : p2.I;
    const bf16_t* A = kGateUp ? p1.x : shared ? p2.Hs + kbeg : p2.H + (size_t)sm.row0 * p2.I;
    const size_t aext = kGateUp ? (size_t)p1.tokens * d : (size_t)R * lda - kbeg;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(A, aext);
    // Staged rows: SB 16-row blocks; each wave issues NDMA DMA instructions
    // per batch, instruction i filling staged rows WRPI*(wave*NDMA + i) ..
    // +WRPI; lane -> row lane/WCHUNKS, LDS chunk lane%WCHUNKS.
    constexpr int stage_bytes = SB * 16 * WROWB;
    constexpr int NDMA = SB * 16 / (DWAVES * WRPI);
    static_assert(NDMA * DWAVES * WRPI == SB * 16, "the waves' DMAs fill the stage");
    uint32_t aoff[NDMA];
    int acol[NDMA];
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
        const int r = WRPI * (wave * NDMA + i) + lane / WCHUNKS;
        const int c = (lane % WCHUNKS) ^ (r & 15);
        acol[i] = c * 8;
        aoff[i] = kOOB;
        if (r < R) {
            int src = r;
            if (kGateUp && !shared)
                src = (int)min((unsigned)(p1.perm[sm.row0 + r] / p1.top_k), (unsigned)(p1.tokens - 1));
            aoff[i] = (uint32_t)(((size_t)src * lda + c * 8) * 2);
        }
    }
    // weights: this wave's 16 rows; lane -> row lane%16, K group lane/16
    const RoutedWeights rw = kGateUp ? (shared ? RoutedWeights{0, p1.Is, 0} : routed_weights(p1, sm))
                                     : (shared ? RoutedWeights{0, 0, p2.Is} : routed_weights(p2, sm));
    const int ldw = kGateUp ? d : rw.ldd;  // weight row stride
    const bf16_t* W0 = kGateUp ? (shared ? p1.sg : p1.wg + rw.base) : (shared ? p2.sd : p2.wd + rw.base);
    const bf16_t* W1 = kGateUp ? (shared ? p1.su : p1.wu + rw.base) : W0;
    const size_t wext = kGateUp ? (size_t)rw.rows * d : (size_t)d * ldw;
    const __amdgpu_buffer_rsrc_t rw0 = make_rsrc(W0, wext);
    const __amdgpu_buffer_rsrc_t rw1 = make_rsrc(W1, wext);
    const int wrow = tile * WCH + wave * 16 + (lane & 15);
    const int g8 = (lane >> 4) * 8;
    const uint32_t woff = wrow < nrows ? (uint32_t)(((size_t)wrow * ldw + kbeg + g8) * 2) : kOOB;

    const int nb = ceil_div(K, WKB);
    constexpr int NW = kGateUp ? 2 : 1;  // weight matrices

    auto issue_rows = [&](int b) {
        unsigned char* st = smem + (b & 1) * stage_bytes + wave * NDMA * 1024;
        const int k0 = b * WKB, lim = K - k0;
#pragma unroll
        for (int i = 0; i < NDMA; ++i)
            load_lds16(ra, acol[i] < lim ? aoff[i] : kOOB, (uint32_t)k0 * 2u, st + i * 1024);
    };
    // weights of step j of batch b into w[.][j]
    auto load_step = [&](int b, int j, u32x4 (&w)[NW][WSTEPS]) {
        const int k0 = b * WKB;
        const uint32_t off = k0 + 32 * j + g8 < K ? woff + (uint32_t)(k0 + 32 * j) * 2u : kOOB;
        w[0][j] = __builtin_amdgcn_raw_buffer_load_b128(rw0, off, 0, 0);
        if constexpr (NW == 2) w[NW - 1][j] = __builtin_amdgcn_raw_buffer_load_b128(rw1, off, 0, 0);
    };

    // The K loop and epilogue for NF 16-token blocks (the rows R fill NF blocks).
    auto run = [&](auto nf_tag) {
        constexpr int NF = decltype(nf_tag)::value;
        floatx4 acc[NW][NF];
#pragma unroll
        for (int m = 0; m < NW; ++m)
#pragma unroll
            for (int f = 0; f < NF; ++f) acc[m][f] = floatx4{0.f, 0.f, 0.f, 0.f};
        // One weight buffer: once step j of batch b has been multiplied, its
        // registers are reloaded with step j of batch b+1, so a batch's
        // weights are requested one batch ahead.  The token fragments of step
        // j+1 are read from LDS while step j multiplies.
        u32x4 w[NW][WSTEPS];
        auto compute = [&](int b) {
            const unsigned char* st = smem + (b & 1) * stage_bytes + (lane & 15) * WROWB;
            bf16x8 xf[2][NF];
            auto read = [&](int j, bf16x8 (&x)[NF]) {
                const int c = (4 * j + (lane >> 4)) ^ (lane & 15);
#pragma unroll
                for (int f = 0; f < NF; ++f)
                    x[f] = as_frag(*reinterpret_cast<const u32x4*>(st + f * 16 * WROWB + c * 16));
            };
            read(0, xf[0]);
#pragma unroll
            for (int j = 0; j < WSTEPS; ++j) {
                if (j + 1 < WSTEPS) read(j + 1, xf[(j + 1) & 1]);
#pragma unroll
                for (int f = 0; f < NF; ++f)
#pragma unroll
                    for (int m = 0; m < NW; ++m)
                        acc[m][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_frag(w[m][j]), xf[j & 1][f],
                                                                            acc[m][f], 0, 0, 0);
                load_step(b + 1, j, w);  // past the last batch: zero-page loads
                // order: next step's LDS reads, this step's MFMAs, the reloads
                if (j + 1 < WSTEPS) __builtin_amdgcn_sched_group_barrier(0x100, NF, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, NF * NW, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, NW, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        issue_rows(0);
#pragma unroll
        for (int j = 0; j < WSTEPS; ++j) load_step(0, j, w);
        for (int b = 0; b < nb; ++b) {
            // batch b's rows are in LDS once every wave's row DMAs are done:
            // only batch b's weight loads (issued after them) may be
            // outstanding; this wave's LDS reads of batch b-1 are finished, so
            // after the barrier batch b+1's rows may refill that stage
            __builtin_amdgcn_s_waitcnt(waitcnt_vm(WSTEPS * NW) & kWaitLgkm0);
            barrier_no_fence();
            // unconditional, so that the compiler's count of outstanding loads
            // stays exact: past the last batch the rows and weights are all
            // masked and read the zero page
            issue_rows(b + 1);
            compute(b);
        }
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // no DMA may outlive the workgroup's LDS

        // D[m][n]: lane holds weight rows 4*(lane/16) + i of token n = lane%16.
        // gate/up writes channels below kk8 = the GEMM width rounded up to 8
        // (the down GEMM reads whole 16-byte chunks), zeros from kk on; col
        // and kk8 are multiples of 4 and 8, so a lane's run of 4 is wholly
        // inside or outside.
        const int col = tile * WCH + wave * 16 + 4 * (lane >> 4);
        const int ldh = kGateUp ? (shared ? p1.Is : p1.I) : d;
        const int lim = kGateUp ? min((sm.kg + 7) & ~7, ldh) : d;  // d % 8 == 0
        if (col >= lim) return;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const int r = f * 16 + (lane & 15);
            if (r >= R) continue;
            uint32_t v[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                float lo, hi;
                if constexpr (kGateUp) {
                    lo = col + 2 * h < sm.kk ? silu_fast(acc[0][f][2 * h]) * acc[1][f][2 * h] : 0.f;
                    hi = col + 2 * h + 1 < sm.kk ? silu_fast(acc[0][f][2 * h + 1]) * acc[1][f][2 * h + 1] : 0.f;
                } else {
                    lo = acc[0][f][2 * h];
                    hi = acc[0][f][2 * h + 1];
                }
                v[h] = (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
            }
            bf16_t* dst;
            if constexpr (kGateUp)
                dst = (shared ? p1.Hs : p1.H + (size_t)sm.row0 * p1.I) + (size_t)r * ldh + col;
            else
                dst = (shared ? p2.Os + (size_t)split * p2.tokens * d : p2.O + (size_t)sm.row0 * d) +
                      (size_t)r * d + col;
            *reinterpret_cast<uint2*>(dst) = make_uint2(v[0], v[1]);
        }
    };
    // R <= tokens, so NF = ceil(R/16) <= SB
    if (SB >= 4 && R > 48) run(std::integral_constant<int, SB >= 4 ? 4 : 1>{});
    else if (SB >= 3 && R > 32) run(std::integral_constant<int, SB >= 3 ? 3 : 1>{});
    else if (SB >= 2 && R > 16) run(std::integral_constant<int, SB >= 2 ? 2 : 1>{});
    else run(std::integral_constant<int, 1>{});
}

// LDS: wide_lds_bytes(tokens), dynamic; SB = wide_blocks(tokens).
template <int SB>
__global__ __launch_bounds__(64 * DWAVES) void gemm1_decode_wide_kernel(Gemm1Params<bf16_t> p) {
    extern __shared__ __attribute__((aligned(1024))) unsigned char wide_smem[];
    wide_tile<true, SB>(p, Gemm2Params<bf16_t>{}, wide_smem);
}

template <int SB>
__global__ __launch_bounds__(64 * DWAVES) void gemm2_decode_wide_kernel(Gemm2Params<bf16_t> p) {
    extern __shared__ __attribute__((aligned(1024))) unsigned char wide_smem[];
    wide_tile<false, SB>(Gemm1Params<bf16_t>{}, p, wide_smem);
}

hipError_t launch_gemm1_decode(const Gemm1Params<bf16_t>& p, int tiles, hipStream_t s) {
    if (tiles <= 0) return hipSuccess;
    if (p.tokens <= kGemvMaxT) return launch_gemv1_decode(p, tiles, s);
    if (p.tokens <= 16) gemm1_decode_kernel<1><<<tiles, 64 * DWAVES, 0, s>>>(p);
    else gemm1_decode_kernel<4><<<tiles, 64 * DWAVES, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_gemm2_decode(const Gemm2Params<bf16_t>& p, int tiles, hipStream_t s) {
    if (tiles <= 0) return hipSuccess;
    if (p.tokens <= kGemvMaxT) return launch_gemv2_decode(p, tiles, s);
    if (p.tokens <= 16) gemm2_decode_kernel<1><<<tiles, 64 * DWAVES, 0, s>>>(p);
    else gemm2_decode_kernel<4><<<tiles, 64 * DWAVES, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_gemm1_decode_wide(const Gemm1Params<bf16_t>& p, int tiles, hipStream_t s) {
    if (tiles <= 0 || p.tokens <= 0 || p.tokens > kDecodeMaxT) return hipSuccess;
    const size_t lds = wide_lds_bytes(p.tokens);
    switch (wide_blocks(p.tokens)) {
        case 1: gemm1_decode_wide_kernel<1><<<tiles, 64 * DWAVES, lds, s>>>(p); break;
        case 2: gemm1_decode_wide_kernel<2><<<tiles, 64 * DWAVES, lds, s>>>(p); break;
        case 3: gemm1_decode_wide_kernel<3><<<tiles, 64 * DWAVES, lds, s>>>(p); break;
        default: gemm1_decode_wide_kernel<4><<<tiles, 64 * DWAVES, lds, s>>>(p); break;
    }
    return hipGetLastError();
}

hipError_t launch_gemm2_decode_wide(const Gemm2Params<bf16_t>& p, int tiles, hipStream_t s) {
    if (tiles <= 0 || p.tokens <= 0 || p.tokens > kDecodeMaxT) return hipSuccess;
    const size_t lds = wide_lds_bytes(p.tokens);
    switch (wide_blocks(p.tokens)) {
        case 1: gemm2_decode_wide_kernel<1><<<tiles, 64 * DWAVES, lds, s>>>(p); break;
        case 2: gemm2_decode_wide_kernel<2><<<tiles, 64 * DWAVES, lds, s>>>(p); break;
        case 3: gemm2_decode_wide_kernel<3><<<tiles, 64 * DWAVES, lds, s>>>(p); break;
        default: gemm2_decode_wide_kernel<4><<<tiles, 64 * DWAVES, lds, s>>>(p); break;
    }
    return hipGetLastError();
}

}  // namespace flexmoe
