// Weight-streaming grouped GEMMs on the matrix cores for decode-sized batches
// of more than kGemvMaxT tokens (up to kDecodeMaxT = 64).
//
// With a few tokens per expert the layer is bound by reading the kept
// weights (Eq. 4: the first k_e channels of each routed expert, plus the
// shared expert), so these kernels read every kept weight byte exactly once.
// A workgroup owns one tile: 64 channels (gate/up) or 64 output columns
// (down) of one segment, for every row (token) of that segment (<= 64 rows =
// up to four 16-token blocks).  The routed experts take these tiles above
// kGemvMaxT tokens, the shared expert above kDecodeWideSharedT; smaller
// batches run the vector-ALU kernels (gemv_decode.hip) on 16-wide tiles.
//
// Both operands are staged through LDS with buffer_load ... lds: per
// 128-deep K batch, the workgroup's four waves copy the 64 weight rows of
// each weight matrix and the segment's token rows (as many 16-row blocks as
// T needs).  Each copy instruction fills four whole 256-byte rows, so the
// weight reads cover whole 128-byte lines, and they carry the non-temporal
// hint (each weight byte is read once per forward; an MFMA fragment loaded
// straight from memory would take 64 bytes of each of 16 rows per
// instruction, and non-temporal half-line reads stream slower than plain
// ones).  Three stages: the copies of batches b+1 and b+2 are in flight
// while batch b is multiplied.  Wave w multiplies weight rows 16w .. 16w+15
// of the tile against every token block (v_mfma_f32_16x16x32_bf16, weights
// on the M side, tokens on the N side; at step j lane l holds logical chunk
// 4j + l/16 of its row of both operands, so every product pairs equal K
// indices).  LDS row r keeps its 16-byte chunk c at position c ^ (r & 15):
// the 16 lanes of one fragment read (16 rows, one chunk) then cover all 64
// banks.
//
// gate/up: SwiGLU is applied to the sums; H is written as bf16, channels
//   from k_e up to the next multiple of 8 as zeros.
// down: the reduction runs over the segment's kept channels; the shared
//   expert's reduction is split into chunks (shared_ks2), each chunk writing
//   its own partial rows, which the combine sums in a fixed order.
#include <type_traits>

#include "mfma_tile.h"

namespace flexmoe {

namespace {
constexpr int DWAVES = 4;  // waves per workgroup
constexpr int WCH = kDecWideBN;         // weight rows (channels / output columns) per wide tile
constexpr int WKB = 128;                // K per batch
constexpr int WSTEPS = WKB / 32;        // MFMA steps per batch
constexpr int WROWB = WKB * 2;          // LDS bytes per staged row
constexpr int WCHUNKS = WROWB / 16;     // 16-byte chunks per staged row
constexpr int WRPI = 1024 / WROWB;      // staged rows one copy instruction (64 lanes x 16 B) fills
constexpr int WSTAGES = 3;
constexpr int WW_DMA = WCH / (DWAVES * WRPI);  // weight copy instructions per wave, matrix and batch
static_assert(WCHUNKS == 16 && 1024 % WROWB == 0 && WW_DMA * DWAVES * WRPI == WCH,
              "the chunk swizzle XORs with 4 row bits; a copy instruction fills whole rows");
constexpr int kNTAux = 2;               // cache-policy operand of a buffer load: non-temporal
}  // namespace

// 16-row token blocks staged per batch for a launch over T tokens (every
// segment has at most T rows), and the LDS of a workgroup with NW weight
// matrices (2: gate/up, 1: down): WSTAGES stages of token and weight rows.
constexpr __host__ __device__ int wide_blocks(int tokens) {
    return ((tokens < kDecodeMaxT ? tokens : kDecodeMaxT) + 15) / 16;
}
constexpr __host__ __device__ size_t wide_lds_bytes(int tokens, int nw) {
    return (size_t)WSTAGES * (wide_blocks(tokens) * 16 + nw * WCH) * WROWB;
}

// SB: 16-row token blocks staged per batch, wide_blocks(T) (a template
// parameter: a fixed count of copies keeps the compiler's count of
// outstanding loads exact).
template <bool kGateUp, int SB>
__device__ __forceinline__ void wide_tile(const Gemm1Params<bf16_t>& p1, const Gemm2Params<bf16_t>& p2,
                                          unsigned char* smem) {
    using namespace mfma;
    constexpr int NW = kGateUp ? 2 : 1;  // weight matrices
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
    // weight matrices: rows of ldw elements, this tile's from kbeg
    const RoutedWeights rw = kGateUp ? (shared ? RoutedWeights{0, p1.Is, 0} : routed_weights(p1, sm))
                                     : (shared ? RoutedWeights{0, 0, p2.Is} : routed_weights(p2, sm));
    const int ldw = kGateUp ? d : rw.ldd;
    const bf16_t* W0 = kGateUp ? (shared ? p1.sg : p1.wg + rw.base) : (shared ? p2.sd : p2.wd + rw.base);
    const bf16_t* W1 = kGateUp ? (shared ? p1.su : p1.wu + rw.base) : W0;
    const size_t wext = kGateUp ? (size_t)rw.rows * d : (size_t)d * ldw;
    const __amdgpu_buffer_rsrc_t rw0 = make_rsrc(W0, wext);
    const __amdgpu_buffer_rsrc_t rw1 = make_rsrc(W1, wext);

    // Stage layout: SB*16 token rows, then WCH rows of each weight matrix,
    // WROWB bytes each.  Copy instruction i of a wave fills WRPI rows; lane
    // -> row lane/WCHUNKS, LDS chunk lane%WCHUNKS, which holds the global
    // chunk (lane%WCHUNKS) ^ (row & 15).
    constexpr int TROWS = SB * 16;
    constexpr int stage_bytes = (TROWS + NW * WCH) * WROWB;
    constexpr int NDMA = TROWS / (DWAVES * WRPI);  // token-row copies per wave per batch
    static_assert(NDMA * DWAVES * WRPI == TROWS, "the waves' copies fill the token rows");
    const int pos = lane % WCHUNKS;
    uint32_t aoff[NDMA], woff[WW_DMA];
    int acol[NDMA], wcol[WW_DMA];
    // source row of each token row: the routed gate/up rows are gathered
    // through perm; every lane loads its entries (rows past the segment read
    // its last row's, unused), so the NDMA loads are in flight together
    int src[NDMA];
#pragma unroll
    for (int i = 0; i < NDMA; ++i) src[i] = WRPI * (wave * NDMA + i) + lane / WCHUNKS;
    if (kGateUp && !shared) {
        const int32_t* pr = p1.perm + sm.row0;
#pragma unroll
        for (int i = 0; i < NDMA; ++i) src[i] = pr[max(min(src[i], R - 1), 0)];
#pragma unroll
        for (int i = 0; i < NDMA; ++i) src[i] = (int)min((unsigned)(src[i] / p1.top_k), (unsigned)(p1.tokens - 1));
    }
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
        const int r = WRPI * (wave * NDMA + i) + lane / WCHUNKS;
        const int c = pos ^ (r & 15);
        acol[i] = c * 8;
        aoff[i] = r < R ? (uint32_t)(((size_t)src[i] * lda + c * 8) * 2) : kOOB;
    }
#pragma unroll
    for (int i = 0; i < WW_DMA; ++i) {
        const int r = WRPI * (wave * WW_DMA + i) + lane / WCHUNKS;  // tile row
        const int c = pos ^ (r & 15);
        const int wr = tile * WCH + r;                                // weight row
        wcol[i] = c * 8;
        woff[i] = wr < nrows ? (uint32_t)(((size_t)wr * ldw + kbeg + c * 8) * 2) : kOOB;
    }

    const int nb = ceil_div(K, WKB);
    auto issue = [&](int b) {
        unsigned char* st = smem + (b % WSTAGES) * stage_bytes;
        const int k0 = b * WKB, lim = K - k0;
        const uint32_t soff = (uint32_t)k0 * 2u;
#pragma unroll
        for (int i = 0; i < NDMA; ++i)
            load_lds16(ra, acol[i] < lim ? aoff[i] : kOOB, soff, st + (wave * NDMA + i) * 1024);
#pragma unroll
        for (int m = 0; m < NW; ++m) {
            unsigned char* sw = st + (TROWS + m * WCH) * WROWB;
#pragma unroll
            for (int i = 0; i < WW_DMA; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(m ? rw1 : rw0, (lds_ptr_t*)(sw + (wave * WW_DMA + i) * 1024),
                                                         16, wcol[i] < lim ? woff[i] : kOOB, soff, 0, kNTAux);
        }
    };
    constexpr int PER_BATCH = NDMA + NW * WW_DMA;  // copy instructions per wave per batch

    // The K loop and epilogue for NF 16-token blocks (the rows R fill NF blocks).
    auto run = [&](auto nf_tag) {
        constexpr int NF = decltype(nf_tag)::value;
        floatx4 acc[NW][NF];
#pragma unroll
        for (int m = 0; m < NW; ++m)
#pragma unroll
            for (int f = 0; f < NF; ++f) acc[m][f] = floatx4{0.f, 0.f, 0.f, 0.f};
        // fragment reads: lane -> row lane%16 (of a token block, or of this
        // wave's 16 weight rows), logical chunk 4j + lane/16 at step j
        auto compute = [&](int b) {
            const unsigned char* st = smem + (b % WSTAGES) * stage_bytes + (lane & 15) * WROWB;
            const unsigned char* sw = st + (TROWS + wave * 16) * WROWB;
            bf16x8 xf[2][NF], wf[2][NW];
            auto read = [&](int j, bf16x8 (&x)[NF], bf16x8 (&w)[NW]) {
                const int c = (4 * j + (lane >> 4)) ^ (lane & 15);
#pragma unroll
                for (int f = 0; f < NF; ++f)
                    x[f] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(st + f * 16 * WROWB + c * 16));
#pragma unroll
                for (int m = 0; m < NW; ++m)
                    w[m] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(sw + m * WCH * WROWB + c * 16));
            };
            read(0, xf[0], wf[0]);
#pragma unroll
            for (int j = 0; j < WSTEPS; ++j) {
                if (j + 1 < WSTEPS) read(j + 1, xf[(j + 1) & 1], wf[(j + 1) & 1]);
#pragma unroll
                for (int f = 0; f < NF; ++f)
#pragma unroll
                    for (int m = 0; m < NW; ++m)
                        acc[m][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j & 1][m], xf[j & 1][f], acc[m][f],
                                                                            0, 0, 0);
            }
        };
        issue(0);
        issue(1);
        for (int b = 0; b < nb; ++b) {
            // batch b is in LDS once every wave's copies of it are done: only
            // batch b+1's may be outstanding; this wave's LDS reads of batch
            // b-1 are finished, so after the barrier batch b+2 may refill
            // that stage
            __builtin_amdgcn_s_waitcnt(waitcnt_vm(PER_BATCH) & kWaitLgkm0);
            barrier_no_fence();
            // unconditional, so that the compiler's count of outstanding
            // loads stays exact: past the last batch every copy is masked
            // and reads the zero page
            issue(b + 2);
            compute(b);
        }
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // no copy may outlive the workgroup's LDS

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
                v[h] = pack_bf16x2(lo, hi);
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

// SB = wide_blocks(tokens); the stages are a static LDS array of
// wide_lds_bytes(tokens, NW) bytes (up to 144 KB for gate/up at SB = 4).
template <int SB>
__global__ __launch_bounds__(64 * DWAVES) void gemm1_decode_wide_kernel(Gemm1Params<bf16_t> p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[wide_lds_bytes(SB * 16, 2)];
    wide_tile<true, SB>(p, Gemm2Params<bf16_t>{}, smem);
}

template <int SB>
__global__ __launch_bounds__(64 * DWAVES) void gemm2_decode_wide_kernel(Gemm2Params<bf16_t> p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[wide_lds_bytes(SB * 16, 1)];
    wide_tile<false, SB>(Gemm1Params<bf16_t>{}, p, smem);
}
static_assert(wide_lds_bytes(kDecodeMaxT, 2) <= 160 * 1024, "the stages fit the compute unit's LDS");

hipError_t launch_gemm1_decode_wide(const Gemm1Params<bf16_t>& p, int tiles, hipStream_t s) {
    if (tiles <= 0 || p.tokens <= 0 || p.tokens > kDecodeMaxT) return hipSuccess;
    switch (wide_blocks(p.tokens)) {
        case 1: gemm1_decode_wide_kernel<1><<<tiles, 64 * DWAVES, 0, s>>>(p); break;
        case 2: gemm1_decode_wide_kernel<2><<<tiles, 64 * DWAVES, 0, s>>>(p); break;
        case 3: gemm1_decode_wide_kernel<3><<<tiles, 64 * DWAVES, 0, s>>>(p); break;
        default: gemm1_decode_wide_kernel<4><<<tiles, 64 * DWAVES, 0, s>>>(p); break;
    }
    return hipGetLastError();
}

hipError_t launch_gemm2_decode_wide(const Gemm2Params<bf16_t>& p, int tiles, hipStream_t s) {
    if (tiles <= 0 || p.tokens <= 0 || p.tokens > kDecodeMaxT) return hipSuccess;
    switch (wide_blocks(p.tokens)) {
        case 1: gemm2_decode_wide_kernel<1><<<tiles, 64 * DWAVES, 0, s>>>(p); break;
        case 2: gemm2_decode_wide_kernel<2><<<tiles, 64 * DWAVES, 0, s>>>(p); break;
        case 3: gemm2_decode_wide_kernel<3><<<tiles, 64 * DWAVES, 0, s>>>(p); break;
        default: gemm2_decode_wide_kernel<4><<<tiles, 64 * DWAVES, 0, s>>>(p); break;
    }
    return hipGetLastError();
}

}  // namespace flexmoe
