// Large-tile ragged grouped GEMMs on bf16 MFMA for prefill-sized token counts.
//
// The gate/up GEMM with fused SwiGLU and the down GEMM with the reduction
// truncated to k_e (FlexMoE Eq. 4), shaped for gfx950:
//   - 256 x 256 workgroup tile (rows x weight rows), K tile 64, 8 waves (two
//     per SIMD: one wave alone cannot keep the matrix core fed) arranged
//     2 x 4, each owning a 128 x 64 block of v_mfma_f32_32x32x16_bf16
//     accumulators (128 registers).  Per K tile the CU reads 192 KB of LDS
//     fragments (256 B/clk) and writes 64 KB (128 B/clk): about 60 % of the
//     LDS time the MFMAs take, with zero bank conflicts.
//   - operands go from global memory straight into LDS (buffer_load ... lds,
//     16 bytes per lane): no VGPRs stage them and no ds_write is issued.
//     Each lane's offset into the operand is fixed for the whole reduction;
//     the K position is a scalar offset.  Rows outside a segment, channels at
//     or past k_e and K chunks past the end use an offset outside the buffer
//     descriptor, for which the hardware returns zeros.
//   - each 128-byte LDS row (64 bf16 of K) stores its eight 16-byte chunks
//     XOR-swizzled by bits 1..3 of the row index, so the 16 lanes served in
//     one LDS cycle of a fragment read hit 64 distinct banks.
//   - two LDS stages of 64 KB: the loads of K tile t+1 are in flight while
//     tile t is multiplied (a launch that may take all of the LDS takes a
//     third token-row stage, 160 KB in all, so that half of each tile's DMAs
//     leave before the barrier).  MFMA operand fragments are read from LDS one
//     16-deep step ahead of their use.  This keeps the kernel near 200 VGPRs:
//     its two waves per SIMD then leave room on every compute unit for the
//     small routing kernels of a concurrently dispatched batch, which a
//     deeper fragment pipeline (about 240 VGPRs) would lock out until a tile
//     finished.
//   - tiles are numbered segment-major (shared expert first: its reductions
//     are the longest), inside a segment in groups of four row tiles (all
//     columns of a group, a column's row tiles consecutive); runs of 8
//     consecutive tiles (32 for a gate/up launch with no concurrent launch
//     beside it) go to one XCD (workgroup b runs on XCD b % 8), interleaving
//     the XCDs run by run, so that the tiles an XCD runs at once share
//     token-row and weight panels in its L2 while the work stays balanced.
// gate/up: a workgroup tile is 256 rows x 128 channels; its B tile holds the
//   128 gate rows then the 128 up rows of those channels, and wave (wm, wn)
//   multiplies gate rows [wn*32, wn*32+32) and the matching up rows, so the
//   gate and up accumulators of a channel sit in the same lane.
// down: a workgroup tile is 256 rows x 256 output columns.  When the shared
//   expert alone has too few tiles to fill the chip, its reduction over I_s
//   is split into chunks whose partial rows the combine adds in chunk order.
// A segment's last row tile often holds far fewer than 256 rows (a routed
// expert gets a few hundred tokens).  A tile with R rows runs the variant in
// which each wave multiplies ceil(R/64) fragments of 32 rows, so MFMA work
// follows the rows at a 64-row granularity; the loads stay the same (rows
// past the segment read the zero page).
#include <type_traits>

#include "mfma_tile.h"

namespace flexmoe {

namespace {
using namespace mfma;
constexpr int BM = 256, BN = 256;
constexpr int NWAVE = 8, THREADS = 64 * NWAVE;
constexpr int WAVES_PER_SIMD = NWAVE / 4;
constexpr int WM = 2, WN = NWAVE / WM;      // wave grid
static_assert(BM == WM * 128, "a full tile gives each M-wave four 32-row fragments");
constexpr int NF = BN / (WN * 32);          // 32-column fragments per wave
constexpr int WCOL = BN / WN;               // weight rows per wave
constexpr int NSB = 2;                      // LDS stages of BK-deep weight (B) tiles
constexpr int NSTEP = BK / 16;              // 16-deep MFMA steps per K tile
static_assert(NSTEP == 4, "the K-loop schedule is laid out for four steps per K tile");
constexpr int RPI = 64 / CHUNKS;            // LDS rows filled per DMA instruction
constexpr int ROWS_PER_WAVE = BM / NWAVE;   // A rows (and B rows) each wave loads
constexpr int NI = ROWS_PER_WAVE / RPI;     // DMA instructions per wave per operand
constexpr int LOADS_PER_TILE = 2 * NI;      // DMA instructions per lane per K tile
constexpr int STAGE_A = BM * ROWB;          // 32 KB
constexpr int STAGE_B = BN * ROWB;          // 32 KB
// LDS of a workgroup with NSA stages of token-row (A) tiles: 128 KB for two,
// 160 KB -- all of a compute unit's LDS -- for three.
template <int NSA>
constexpr int smem_bytes() { return NSA * STAGE_A + NSB * STAGE_B; }
static_assert(smem_bytes<3>() <= 160 * 1024, "the stages fit the compute unit's LDS");
constexpr int XCD_GROUP = 8;                // consecutive tiles kept on one XCD (default)
constexpr int ROW_GROUP = 4;                // row tiles of a segment walked before the next column
}  // namespace

// Saliency forward: the tile's h (256 rows x 128 channels) written
// transposed through an LDS staging tile.  In the accumulator, lane -> row
// lane%32 of a 32-row fragment, register v -> channel (v/4)*8 + (lane/32)*4 +
// v%4 of the wave's 32 gate (jj = 0) and up (jj = NF/2) channels.
constexpr int TROW = 256 + 8;  // staging row pitch (bf16): 4 rows apart = 16 banks apart
static_assert(128 * TROW * 2 <= smem_bytes<2>(), "the staging tile fits in the operand stages");

template <int MFW, typename Acc>
__device__ __forceinline__ void train_store_h_transposed(const Gemm1Params<bf16_t>& p, const SegMeta& sm,
                                                         const Acc& acc, unsigned char* smem, int mtile,
                                                         int ntile, int wave, int lane) {
    constexpr int WR = 32 * MFW;
    const int wm = wave / WN, wn = wave % WN;
    bf16_t* st = reinterpret_cast<bf16_t*>(smem);
    const int tile_rows = sm.rows - mtile * BM;            // real rows of this tile
    const int pvalid = packed_width(sm.rows) - mtile * BM;  // rows written (padding included)
    const int ch_tile = ntile * (BN / 2);
    // the operand stages are free once every wave is past its last fragment read
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    barrier_no_fence();
#pragma unroll
    for (int i = 0; i < MFW; ++i) {
        const int row = wm * WR + i * 32 + (lane & 31);
        const bool real = row < tile_rows;
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int cl = wn * (WCOL / 2) + q * 8 + (lane >> 5) * 4 + r;
                const float g = acc[i][0][q * 4 + r], u = acc[i][NF / 2][q * 4 + r];
                st[cl * TROW + row] = real ? f32_to_bf16(silu_fast(g) * u) : (bf16_t)0;
            }
    }
    __syncthreads();
    bf16_t* out = p.ht + (size_t)sm.prow0 + mtile * BM;
    for (int k = threadIdx.x; k < (BN / 2) * (BM / 8); k += THREADS) {
        const int cl = k / (BM / 8), r0 = (k % (BM / 8)) * 8;
        const int ch = ch_tile + cl;
        if (r0 >= pvalid || ch >= sm.kg) continue;
        *reinterpret_cast<u32x4*>(out + (size_t)ch * p.ldt + r0) =
            *reinterpret_cast<const u32x4*>(st + cl * TROW + r0);
    }
}

// kTrain: 0 = inference; 1 = also g and u of the routed rows
// (fragment-blocked) and their h transposed (channel saliency); 2 = also g
// and u of every row, fragment-blocked (the masked layer's training backward).
// NSA: LDS stages of token-row tiles (2, or 3: token-row tile kt+2 is then
// requested during the first MFMA step of tile kt instead of after the
// barrier, so each barrier releases half as many DMAs).
// XG: consecutive tiles kept on one XCD (XCD_GROUP, or 32 for a gate/up
// launch with the GPU to itself, see gemm1_big_kernel).
template <bool kGateUp, int kTrain = 0, int NSA = 2, int XG = XCD_GROUP>
__device__ __forceinline__ void big_tile(const Gemm1Params<bf16_t>& p1, const Gemm2Params<bf16_t>& p2,
                                         unsigned char* smem) {
    const int d = kGateUp ? p1.d : p2.d;

    // tile numbering: XCD x = b % 8 takes runs of XG consecutive tiles
    const int jb = blockIdx.x >> 3;
    const int L = (jb / XG) * (8 * XG) + (blockIdx.x & 7) * XG + jb % XG;
    int s, local;
    SegMeta sm;
    if (!(kGateUp ? tile_of(p1, L, s, sm, local) : tile_of(p2, L, s, sm, local))) return;
    // A segment's tiles form an mt x nt grid (row tiles x channel or output
    // column tiles); the down GEMM of a split shared expert has one grid per
    // reduction chunk, chunk `split` after chunk split-1.  Inside a grid the
    // tiles go in groups of ROW_GROUP row tiles: all columns of a group, each
    // column's row tiles consecutive, then the next group.  An XCD's 32
    // concurrent tiles (four runs of 8 from consecutive rounds over the 8
    // XCDs, or one run of 32) then share about ROW_GROUP token-row panels
    // and 8 weight panels through its L2, instead of needing up to 32
    // token-row panels and 4 weight panels: the L2 misses of the
    // Mixtral-shaped gate/up launch drop from 13.3 GB (one row tile after
    // another) to 9.5 GB with runs of 8 and 6.8 GB with runs of 32.
    const int mt = ceil_div(sm.rows, BM);
    const int nt = kGateUp ? ceil_div(sm.kg, BN / 2) : ceil_div(d, BN);
    const int split = kGateUp ? 0 : local / (mt * nt);
    const int loc = kGateUp ? local : local - split * mt * nt;
    const int grp = loc / (ROW_GROUP * nt);
    const int rem = loc - grp * ROW_GROUP * nt;
    const int grows = min(ROW_GROUP, mt - grp * ROW_GROUP);  // row tiles of this group
    const int ntile = rem / grows, mtile = grp * ROW_GROUP + rem % grows;
    const bool shared = sm.e < 0;

    // the wave index is uniform: keeping it in a scalar register makes every
    // LDS destination address (M0) scalar arithmetic
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;

    // ---- buffer descriptors and per-lane byte offsets of the A rows and B
    // rows this lane loads.  DMA instruction i of a wave fills LDS rows
    // wave*ROWS_PER_WAVE + i*RPI .. +RPI of each operand; lane -> row
    // lane/CHUNKS, LDS chunk lane%CHUNKS, which holds global chunk
    // swz(row, lane%CHUNKS).  Masked rows (outside the segment, channels at or
    // past k_e, columns past d) get an offset past the descriptor's extent,
    // for which the load returns zeros.
    const int pos = lane % CHUNKS;
    uint32_t aoff[NI], boff[NI];
    int acol[NI];
    int K;
    __amdgpu_buffer_rsrc_t ra, rb;
    if constexpr (kGateUp) {
        K = d;
        const RoutedWeights rw = shared ? RoutedWeights{0, p1.Is, 0} : routed_weights(p1, sm);
        // this wave's B rows are all gate rows or all up rows
        const bf16_t* W = (wave * ROWS_PER_WAVE < BN / 2 ? (shared ? p1.sg : p1.wg) : (shared ? p1.su : p1.wu)) + rw.base;
        ra = make_rsrc(p1.x, (size_t)p1.tokens * d);
        rb = make_rsrc(W, (size_t)rw.rows * d);
        // token of each A row: every lane loads its rows' entries of the
        // permutation (rows past the segment read its last row's, unused), so
        // the NI loads are in flight together rather than one after another
        int tok[NI];
        const int row_l = mtile * BM + wave * ROWS_PER_WAVE + lane / CHUNKS;
        if (shared) {
#pragma unroll
            for (int i = 0; i < NI; ++i) tok[i] = row_l + i * RPI;
        } else {
            const int32_t* pr = p1.perm + sm.row0;
#pragma unroll
            for (int i = 0; i < NI; ++i) tok[i] = pr[min(row_l + i * RPI, sm.rows - 1)];
        }
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int r = wave * ROWS_PER_WAVE + i * RPI + lane / CHUNKS;
            const int row = mtile * BM + r;
            const int c = swz(r, pos) * 8;
            acol[i] = c;
            const int t = shared ? tok[i] : (int)min((unsigned)(tok[i] / p1.top_k), (unsigned)(p1.tokens - 1));
            aoff[i] = row < sm.rows ? (uint32_t)(((size_t)t * d + c) * 2) : kOOB;
            const int ch = ntile * (BN / 2) + (r & (BN / 2 - 1));
            boff[i] = ch < sm.kg ? (uint32_t)(((size_t)ch * d + c) * 2) : kOOB;
        }
    } else {
        const int kbeg = shared && p2.ks2 > 0 ? split * p2.ks2 : 0;
        K = shared && p2.ks2 > 0 ? min(sm.kg - kbeg, p2.ks2) : sm.kg;
        const RoutedWeights rw = shared ? RoutedWeights{0, 0, p2.Is} : routed_weights(p2, sm);
        const int ldh = shared ? p2.Is : p2.I;  // H row stride
        const int ldw = rw.ldd;                 // W_down row stride
        const int hrows = shared ? p2.tokens : sm.rows;
        const bf16_t* Hb = (shared ? p2.Hs : p2.H + (size_t)sm.row0 * p2.I) + kbeg;
        const bf16_t* Wd = (shared ? p2.sd : p2.wd + rw.base) + kbeg;
        ra = make_rsrc(Hb, (size_t)hrows * ldh - kbeg);
        rb = make_rsrc(Wd, (size_t)d * ldw - kbeg);
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int r = wave * ROWS_PER_WAVE + i * RPI + lane / CHUNKS;
            const int row = mtile * BM + r;
            const int c = swz(r, pos) * 8;
            acol[i] = c;
            aoff[i] = row < sm.rows ? (uint32_t)(((size_t)row * ldh + c) * 2) : kOOB;
            const int n = ntile * BN + r;
            boff[i] = n < d ? (uint32_t)(((size_t)n * ldw + c) * 2) : kOOB;
        }
    }

    // DMA of K tile kt into a stage.  Chunks at or past K are masked as well,
    // and tiles past the end load nothing useful (their stage is never read),
    // so every tile issues exactly LOADS_PER_TILE loads.
    // The A stages come first in LDS, then the B stages.
    auto issue_a = [&](int kt, int stage) {
        unsigned char* sa = smem + stage * STAGE_A + wave * ROWS_PER_WAVE * ROWB;
        const int lim = K - kt * BK;
        const uint32_t soff = (uint32_t)(kt * BK) * 2u;
#pragma unroll
        for (int i = 0; i < NI; ++i) load_lds16(ra, acol[i] < lim ? aoff[i] : kOOB, soff, sa + i * RPI * ROWB);
    };
    auto issue_b = [&](int kt, int stage) {
        unsigned char* sb = smem + NSA * STAGE_A + stage * STAGE_B + wave * ROWS_PER_WAVE * ROWB;
        const int lim = K - kt * BK;
        const uint32_t soff = (uint32_t)(kt * BK) * 2u;
#pragma unroll
        for (int i = 0; i < NI; ++i) load_lds16(rb, acol[i] < lim ? boff[i] : kOOB, soff, sb + i * RPI * ROWB);
    };

    const int wm = wave / WN, wn = wave % WN;
    int brow[NF];
#pragma unroll
    for (int j = 0; j < NF; ++j) {
        if constexpr (kGateUp)  // gate rows, then the same channels' up rows
            brow[j] = (j < NF / 2 ? 0 : BN / 2) + wn * (WCOL / 2) + (j % (NF / 2)) * 32;
        else
            brow[j] = wn * WCOL + j * 32;
    }
    const int nk = ceil_div(K, BK);

    // The K loop and epilogue for tiles whose waves multiply MFW 32-row
    // fragments each (the two M-waves then cover 64*MFW rows).
    auto run = [&](auto mfw_tag) {
        constexpr int MFW = decltype(mfw_tag)::value;
        constexpr int WR = 32 * MFW;                    // rows per wave
        constexpr int NMF = MFW * NF;                   // MFMAs per 16-deep step
        constexpr int NRD = MFW + NF;                   // fragment reads per step
        floatx16 acc[MFW][NF];
#pragma unroll
        for (int i = 0; i < MFW; ++i)
#pragma unroll
            for (int j = 0; j < NF; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
        bf16x8 a[2][MFW], b[2][NF];  // fragment buffers of alternate steps
        auto read_frags = [&](int kt, int ks, int buf) {
            const unsigned char* sa = smem + (kt % NSA) * STAGE_A;
            const unsigned char* sb = smem + NSA * STAGE_A + (kt % NSB) * STAGE_B;
            const int chunk = ks * 2 + (lane >> 5);
#pragma unroll
            for (int i = 0; i < MFW; ++i) a[buf][i] = lds_frag(sa, wm * WR + i * 32 + (lane & 31), chunk);
#pragma unroll
            for (int j = 0; j < NF; ++j) b[buf][j] = lds_frag(sb, brow[j] + (lane & 31), chunk);
        };
        auto mfma_step = [&](int buf) {
#pragma unroll
            for (int i = 0; i < MFW; ++i)
#pragma unroll
                for (int j = 0; j < NF; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[buf][j], a[buf][i], acc[i][j], 0, 0, 0);
        };

        // Two weight stages, fragments one step ahead:
        //   steps s < 3: read (kt, s+1) | MFMA (kt, s)
        //   wait for tile kt+1 and this wave's reads, barrier
        //   DMA tile kt+2 into the stages of tile kt | read (kt+1, 0) | MFMA (kt, 3)
        // At the barrier every wave has finished reading tile kt (its last
        // fragments are in registers), so its stages can be refilled, and
        // tile kt+1 has landed, so its fragments can be read.  Every
        // iteration issues one tile's DMAs (zero-page loads once past the
        // end), so at the wait no later tile's loads are outstanding.
        // With two stages each wave issues all 8 of its DMAs right after the
        // barrier, 64 per compute unit at once, and the MFMAs behind them
        // wait for issue.  With three token-row stages, token-row tile kt+2
        // goes into the stage of tile kt-1 (free since the previous barrier)
        // beside the MFMAs of step 0 and only the weight tile's DMAs follow
        // the barrier (the Mixtral-shaped gate/up GEMM runs 3 % faster); at
        // the wait that token-row tile may still be outstanding.
        static_assert(NSA == 2 || NSA == 3, "two or three token-row stages");
        constexpr int EARLY = NSA == 3 ? NI : 0;  // DMAs issued before the barrier
        issue_a(0, 0);
        issue_b(0, 0);
        issue_a(1, 1);
        issue_b(1, 1);
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * NI));  // tile 0 in
        barrier_no_fence();
        read_frags(0, 0, 0);
        for (int kt = 0; kt < nk; ++kt) {
            read_frags(kt, 1, 1);
            if constexpr (NSA == 3) issue_a(kt + 2, (kt + 2) % 3);
            mfma_step(0);
            sched_interleave<NMF, EARLY, NRD>();
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int st = 1; st < NSTEP - 1; ++st) {
                read_frags(kt, st + 1, (st + 1) & 1);
                mfma_step(st & 1);
                sched_interleave<NMF, 0, NRD>();
                __builtin_amdgcn_sched_barrier(0);
            }
            __builtin_amdgcn_s_waitcnt(waitcnt_vm(EARLY) & kWaitLgkm0);  // tile kt+1 in; own reads done
            barrier_no_fence();  // all waves are done reading tile kt: its stages are free
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (NSA == 2) issue_a(kt + 2, kt % 2);
            issue_b(kt + 2, kt % 2);
            // after the last tile this reads stale stages, whose values go unused
            read_frags(kt + 1, 0, 0);
            mfma_step((NSTEP - 1) & 1);
            sched_interleave<NMF, LOADS_PER_TILE - EARLY, NRD>();
            __builtin_amdgcn_sched_barrier(0);
        }
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // no DMA may outlive the workgroup's LDS

        // ---- epilogue.  The weight fragment is the MFMA's first operand, so
        // the accumulator is transposed: lane -> row lane%32 of the fragment,
        // register v -> weight row (v/4)*8 + (lane/32)*4 + v%4.  Each lane
        // thus holds four runs of 4 consecutive channels (or output columns)
        // of one row and stores each run as one 8-byte write.
        const int row_l = mtile * BM + wm * WR + (lane & 31);
        const int sub = (lane >> 5) * 4;
        if constexpr (kGateUp) {
            bf16_t* Hb = shared ? p1.Hs : p1.H + (size_t)sm.row0 * p1.I;
            const int ldh = shared ? p1.Is : p1.I;
            // channels [kk, kk8) are written as zeros, kk8 = the GEMM width
            // rounded up to 8 (the down GEMM reads whole 16-byte chunks); kk8
            // and the runs are multiples of 8 and 4, so a run is wholly inside
            // or outside
            const int kk8 = min((sm.kg + 7) & ~7, ldh);
#pragma unroll
            for (int i = 0; i < MFW; ++i) {
                const int row = row_l + i * 32;
                if (row >= sm.rows) continue;
                bf16_t* hr = Hb + (size_t)row * ldh;
#pragma unroll
                for (int jj = 0; jj < NF / 2; ++jj)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int ch = ntile * (BN / 2) + wn * (WCOL / 2) + jj * 32 + q * 8 + sub;
                    if (ch >= kk8) continue;
                    uint32_t w[2];
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int v = q * 4 + h * 2;
                        const float g0 = acc[i][jj][v], u0 = acc[i][jj + NF / 2][v];
                        const float g1 = acc[i][jj][v + 1], u1 = acc[i][jj + NF / 2][v + 1];
                        const float lo = ch + h * 2 < sm.kk ? silu_fast(g0) * u0 : 0.f;
                        const float hi = ch + h * 2 + 1 < sm.kk ? silu_fast(g1) * u1 : 0.f;
                        w[h] = pack_bf16x2(lo, hi);
                    }
                    *reinterpret_cast<uint2*>(hr + ch) = make_uint2(w[0], w[1]);
                }
            }
            if (kTrain == 2 || (kTrain == 1 && !shared)) {
                // g and u for the training backward, in the fragment-blocked
                // layout (common.h) over the routed row space (or the tokens)
                bf16_t* Gb = shared ? p1.Gs : p1.G;
                bf16_t* Ub = shared ? p1.Us : p1.U;
                const size_t rbase = shared ? 0 : (size_t)sm.row0;
#pragma unroll
                for (int i = 0; i < MFW; ++i) {
                    const int row = row_l + i * 32;
                    if (row >= sm.rows) continue;
#pragma unroll
                    for (int jj = 0; jj < NF / 2; ++jj)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const int ch = ntile * (BN / 2) + wn * (WCOL / 2) + jj * 32 + q * 8 + sub;
                            if (ch >= sm.kg) continue;
                            uint32_t gw[2], uw[2];
#pragma unroll
                            for (int h = 0; h < 2; ++h) {
                                const int v = q * 4 + h * 2;
                                gw[h] = pack_bf16x2(acc[i][jj][v], acc[i][jj][v + 1]);
                                uw[h] = pack_bf16x2(acc[i][jj + NF / 2][v], acc[i][jj + NF / 2][v + 1]);
                            }
                            const size_t off = frag_blocked(rbase + row, ch, ldh);
                            *reinterpret_cast<uint2*>(Gb + off) = make_uint2(gw[0], gw[1]);
                            *reinterpret_cast<uint2*>(Ub + off) = make_uint2(uw[0], uw[1]);
                        }
                }
            }
            if constexpr (kTrain == 1) {
                // h transposed for the weight-gradient GEMMs, element
                // [c][prow0 + row], zero in the rows up to the segment's padded
                // height, staged through LDS as a [128 channels][256 rows] tile
                // so that global stores are whole 16-byte row pieces
                if (!shared) train_store_h_transposed<MFW>(p1, sm, acc, smem, mtile, ntile, wave, lane);
            }
        } else {
            bf16_t* Ob = shared ? p2.Os + (size_t)split * p2.tokens * d : p2.O + (size_t)sm.row0 * d;
#pragma unroll
            for (int i = 0; i < MFW; ++i) {
                const int row = row_l + i * 32;
                if (row >= sm.rows) continue;
                bf16_t* orow = Ob + (size_t)row * d;
#pragma unroll
                for (int j = 0; j < NF; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int n = ntile * BN + wn * WCOL + j * 32 + q * 8 + sub;
                        if (n >= d) continue;
                        const uint32_t w0 = pack_bf16x2(acc[i][j][q * 4], acc[i][j][q * 4 + 1]);
                        const uint32_t w1 = pack_bf16x2(acc[i][j][q * 4 + 2], acc[i][j][q * 4 + 3]);
                        *reinterpret_cast<uint2*>(orow + n) = make_uint2(w0, w1);
                    }
            }
        }
    };

    const int tile_rows = min(BM, sm.rows - mtile * BM);
    if (tile_rows > 3 * 64) run(std::integral_constant<int, 4>{});
    else if (tile_rows > 2 * 64) run(std::integral_constant<int, 3>{});
    else if (tile_rows > 64) run(std::integral_constant<int, 2>{});
    else run(std::integral_constant<int, 1>{});
}

// NSA = 3 (160 KB of LDS) except for the shared expert's side-stream
// launches, which must leave room for the routing kernels beside them.
// XG = 32 when no side-stream launch runs at all: the L2 misses drop by 29 %
// and the layer step by about 1 % (Mixtral and Qwen2-57B shapes); beside a
// side-stream launch the longer runs were 0.5 % slower.  The down GEMM keeps
// runs of 8: its segments' reductions differ, and longer runs left the XCDs
// unevenly loaded at the end.
template <int NSA, int XG>
__global__ __launch_bounds__(THREADS, WAVES_PER_SIMD) void gemm1_big_kernel(Gemm1Params<bf16_t> p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[smem_bytes<NSA>()];
    big_tile<true, 0, NSA, XG>(p, Gemm2Params<bf16_t>{}, smem);
}

// The gate/up GEMM of the training forward: the same tiles, plus the
// transposed g, u and h copies of the routed segments (Gemm1Params).
__global__ __launch_bounds__(THREADS, WAVES_PER_SIMD) void gemm1_big_train_kernel(Gemm1Params<bf16_t> p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[smem_bytes<3>()];
    big_tile<true, 1, 3>(p, Gemm2Params<bf16_t>{}, smem);
}

// The gate/up GEMM of the masked layer's training forward: the same tiles,
// plus g and u of every row (Gemm1Params).
__global__ __launch_bounds__(THREADS, WAVES_PER_SIMD) void gemm1_big_train_rm_kernel(Gemm1Params<bf16_t> p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[smem_bytes<3>()];
    big_tile<true, 2, 3>(p, Gemm2Params<bf16_t>{}, smem);
}

// NSA = 3 as for the gate/up GEMM: the down GEMM's long reductions then run
// 4 % faster on the Mixtral and Qwen2-57B shapes.
template <int NSA>
__global__ __launch_bounds__(THREADS, WAVES_PER_SIMD) void gemm2_big_kernel(Gemm2Params<bf16_t> p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[smem_bytes<NSA>()];
    big_tile<false, 0, NSA>(Gemm1Params<bf16_t>{}, p, smem);
}

hipError_t launch_gemm1_big(const Gemm1Params<bf16_t>& p, int grid, hipStream_t s, bool full_lds, bool alone) {
    if (grid <= 0) return hipSuccess;
    const int xg = alone ? 32 : XCD_GROUP;
    const int g = (grid + 8 * xg - 1) / (8 * xg) * (8 * xg);
    if (alone) gemm1_big_kernel<3, 32><<<g, THREADS, 0, s>>>(p);
    else if (full_lds) gemm1_big_kernel<3, XCD_GROUP><<<g, THREADS, 0, s>>>(p);
    else gemm1_big_kernel<2, XCD_GROUP><<<g, THREADS, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_gemm1_big_train(const Gemm1Params<bf16_t>& p, int grid, hipStream_t s) {
    if (grid <= 0) return hipSuccess;
    const int g = (grid + 8 * XCD_GROUP - 1) / (8 * XCD_GROUP) * (8 * XCD_GROUP);
    gemm1_big_train_kernel<<<g, THREADS, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_gemm1_big_train_rm(const Gemm1Params<bf16_t>& p, int grid, hipStream_t s) {
    if (grid <= 0) return hipSuccess;
    const int g = (grid + 8 * XCD_GROUP - 1) / (8 * XCD_GROUP) * (8 * XCD_GROUP);
    gemm1_big_train_rm_kernel<<<g, THREADS, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_gemm2_big(const Gemm2Params<bf16_t>& p, int grid, hipStream_t s, bool full_lds) {
    if (grid <= 0) return hipSuccess;
    const int g = (grid + 8 * XCD_GROUP - 1) / (8 * XCD_GROUP) * (8 * XCD_GROUP);
    if (full_lds) gemm2_big_kernel<3><<<g, THREADS, 0, s>>>(p);
    else gemm2_big_kernel<2><<<g, THREADS, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace flexmoe
