// Backward GEMMs of the channel saliency (FlexMoE Sec. 3.1, Eq. 2) on bf16
// MFMA.  For the loss L = 1/2 sum_t ||Y_t - Y_target_t||^2 and routed expert
// e with dO_a = w_a dY_t (one row per routed assignment):
//   dgrad:  dH[a][c] = sum_n dO_a[n] W_down[n][c]; fused epilogue
//           dG = dH u silu'(g), dU = dH silu(g)           (SwiGLU backward)
//           (the same kernel serves the masked layer's training backward)
//   wgrad:  dW_gate[c][i] = sum_a dG[a][c] x_a[i], dW_up likewise with dU,
//           dW_down[n][c] = sum_a dO_a[n] h_a[c]; fused epilogue
//           s[e][c] += sum over the tile of (theta * dW)^2  (Eq. 2)
// so the weight gradients are never written: each wgrad tile reduces its
// 256 x 256 block of (theta * g)^2 to one partial sum per channel.
//
// All are "NT" GEMMs: A rows and B rows are contiguous in K, staged by the
// same LDS pipeline as the forward's big tiles (mfma_tile.h: 256 x 256 x 64
// tiles, 8 waves as 2 x 4, direct-to-LDS DMA, three A and two B stages,
// fragments one step ahead).  In the wgrad the MFMA takes the A fragment first, so a lane's
// accumulator holds one B row (a channel) and runs of 4 consecutive A rows,
// and the weight reads of its epilogue are 8-byte accesses.
//   dgrad: A = dO [A][d] (a segment's rows), B = W_down^T [E][I][d] (a
//          transposed copy of the down weights), K = d.
//   wgrad: A = x^T or dO^T [d][ldt], B = dG^T, dU^T or h^T [I][ldt], with a
//          segment's rows as K (columns prow0 .. prow0 + rows of the
//          transposed copies, zero-padded to a multiple of 8).
#include <type_traits>

#include "mfma_tile.h"
#include "saliency.h"
#include "train.h"

namespace flexmoe {

namespace {
using namespace mfma;
constexpr int BM = 256, BN = 256;
constexpr int NWAVE = 8, THREADS = 64 * NWAVE;
constexpr int WAVES_PER_SIMD = NWAVE / 4;
constexpr int WM = 2, WN = NWAVE / WM;      // wave grid
constexpr int NF = BN / (WN * 32);          // 32-row B fragments per wave
constexpr int WCOL = BN / WN;               // B rows per wave
constexpr int NSTEP = BK / 16;
static_assert(NSTEP == 4, "the K-loop schedule is laid out for four steps per K tile");
constexpr int RPI = 64 / CHUNKS;            // LDS rows filled per DMA instruction
constexpr int ROWS_PER_WAVE = BM / NWAVE;   // A rows (and B rows) each wave loads
constexpr int NI = ROWS_PER_WAVE / RPI;     // DMA instructions per wave per operand
constexpr int STAGE_A = BM * ROWB;
constexpr int STAGE_B = BN * ROWB;
constexpr int SMEM3 = 3 * STAGE_A + 2 * STAGE_B;  // the K loop's LDS with three A stages
static_assert(SMEM3 <= 160 * 1024, "three A stages and two B stages fit one compute unit");
constexpr int XCD_GROUP = 8;
static_assert(BM == kSalTile && BN == kSalTile, "host tile counts use kSalTile");

// The operands of one tile: per-lane byte offsets of the A and B rows this
// lane loads (kOOB for rows outside the operand), the chunk column of each,
// and the reduction length.
struct NTOperands {
    __amdgpu_buffer_rsrc_t ra, rb;
    uint32_t aoff[NI], boff[NI];
    int acol[NI];
    int K;
};

// DMA instruction i of a wave fills LDS rows wave*ROWS_PER_WAVE + i*RPI ..
// +RPI; lane -> row lane/CHUNKS, LDS chunk lane%CHUNKS, which holds global
// chunk swz(row, lane%CHUNKS).  Rows at or past `valid` (counted from the
// operand's base) read zeros.
__device__ __forceinline__ void nt_rows(int wave, int lane, int row_base, int valid, int ld, uint32_t* off,
                                        int* acol) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int r = wave * ROWS_PER_WAVE + i * RPI + lane / CHUNKS;
        const int c = swz(r, lane % CHUNKS) * 8;
        const int row = row_base + r;
        acol[i] = c;
        off[i] = row < valid ? (uint32_t)(((size_t)row * ld + c) * 2) : kOOB;
    }
}

// Tail of a K loop that needs nothing after its last K tile: zero-page loads
// keep the count of outstanding DMAs the schedule waits on.
struct ZeroTail {
    __amdgpu_buffer_rsrc_t r;
    // one part (A or B) of a K-tile slot past the end
    __device__ __forceinline__ void operator()(int, bool, unsigned char* dst) const {
#pragma unroll
        for (int i = 0; i < NI; ++i) load_lds16(r, kOOB, 0, dst + i * RPI * ROWB);
    }
};

// The K loop of one tile whose waves multiply MFW 32-row A fragments each:
// acc[i][j] = A rows wm*32*MFW + i*32 .. x B rows wn*WCOL + j*32 ...  The
// schedule is the forward's: three A stages and two B stages (all 160 KB of
// LDS; the A stages first, then the B stages), fragments read one step ahead,
// A tile kt+2 requested beside the first MFMA step of tile kt, so each
// barrier releases only the B tile's DMAs.  The last two DMA slots of each
// part (K tiles nk and nk+1, past the end) go to tail(h, part_a, dst) for
// h = 0, 1, which must issue exactly NI loads into this wave's rows `dst` of
// A stage (nk + h) % 3 or of B stage (nk + h) % 2.
// kSwap: the A fragment is the MFMA's first operand (lane -> B row, registers
// -> runs of 4 A rows); otherwise the B fragment is (lane -> A row, registers
// -> runs of 4 B rows).  zero = false continues accumulating into acc.
template <int MFW, bool kSwap = true, typename Tail>
__device__ __forceinline__ void nt_mainloop(unsigned char* smem, const NTOperands& op, int wave, int lane,
                                            floatx16 (&acc)[MFW][NF], Tail&& tail, bool zero = true) {
    constexpr int WR = 32 * MFW;
    constexpr int NMF = MFW * NF;
    constexpr int NRD = MFW + NF;
    const int wm = wave / WN, wn = wave % WN;
    if (zero) {
#pragma unroll
        for (int i = 0; i < MFW; ++i)
#pragma unroll
            for (int j = 0; j < NF; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    }

    const int nk = ceil_div(op.K, BK);
    bf16x8 a[2][MFW], b[2][NF];
    auto read_frags = [&](int kt, int ks, int buf) {
        const unsigned char* sa = smem + (kt % 3) * STAGE_A;
        const unsigned char* sb = smem + 3 * STAGE_A + (kt % 2) * STAGE_B;
        const int chunk = ks * 2 + (lane >> 5);
#pragma unroll
        for (int i = 0; i < MFW; ++i) a[buf][i] = lds_frag(sa, wm * WR + i * 32 + (lane & 31), chunk);
#pragma unroll
        for (int j = 0; j < NF; ++j) b[buf][j] = lds_frag(sb, wn * WCOL + j * 32 + (lane & 31), chunk);
    };
    auto mfma_step = [&](int buf) {
#pragma unroll
        for (int i = 0; i < MFW; ++i)
#pragma unroll
            for (int j = 0; j < NF; ++j)
                acc[i][j] = kSwap ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[buf][i], b[buf][j], acc[i][j], 0, 0, 0)
                                  : __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[buf][j], a[buf][i], acc[i][j], 0, 0, 0);
    };
    // DMA of K tile kt's A part into A stage kt % 3, or its B part into
    // B stage kt % 2 (masked past K)
    auto issue_part = [&](int kt, bool part_a) {
        unsigned char* dst = (part_a ? smem + (kt % 3) * STAGE_A : smem + 3 * STAGE_A + (kt % 2) * STAGE_B) +
                             wave * ROWS_PER_WAVE * ROWB;
        if (kt >= nk) {
            tail(kt - nk, part_a, dst);
            return;
        }
        const int lim = op.K - kt * BK;
        const uint32_t soff = (uint32_t)(kt * BK) * 2u;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const bool kin = op.acol[i] < lim;
            if (part_a) load_lds16(op.ra, kin ? op.aoff[i] : kOOB, soff, dst + i * RPI * ROWB);
            else load_lds16(op.rb, kin ? op.boff[i] : kOOB, soff, dst + i * RPI * ROWB);
        }
    };
    issue_part(0, true);
    issue_part(0, false);
    issue_part(1, true);
    issue_part(1, false);
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * NI));  // tile 0 in
    barrier_no_fence();
    read_frags(0, 0, 0);
    for (int kt = 0; kt < nk; ++kt) {
        read_frags(kt, 1, 1);
        issue_part(kt + 2, true);  // into the A stage of tile kt-1, free since the last barrier
        mfma_step(0);
        sched_interleave<NMF, NI, NRD>();
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int st = 1; st < NSTEP - 1; ++st) {
            read_frags(kt, st + 1, (st + 1) & 1);
            mfma_step(st & 1);
            sched_interleave<NMF, 0, NRD>();
            __builtin_amdgcn_sched_barrier(0);
        }
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(NI) & kWaitLgkm0);  // tile kt+1 in; own reads done
        barrier_no_fence();
        __builtin_amdgcn_sched_barrier(0);
        issue_part(kt + 2, false);
        read_frags(kt + 1, 0, 0);
        mfma_step((NSTEP - 1) & 1);
        sched_interleave<NMF, NI, NRD>();
        __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // no DMA may outlive the workgroup's LDS
}

// Runs `body` with the fragment count for a tile of `rows` A rows (the two
// M-waves cover 64*MFW rows).
template <typename F>
__device__ __forceinline__ void by_rows(int rows, F&& body) {
    if (rows > 3 * 64) body(std::integral_constant<int, 4>{});
    else if (rows > 2 * 64) body(std::integral_constant<int, 3>{});
    else if (rows > 64) body(std::integral_constant<int, 2>{});
    else body(std::integral_constant<int, 1>{});
}

// Tile of this workgroup when groups of `group` consecutive tiles go to one
// XCD (workgroup b runs on XCD b % 8): tiles that share operands then share
// that XCD's L2.  The grid is a multiple of 8 * group (xcd_grid).
__device__ __forceinline__ int xcd_tile(int group = XCD_GROUP) {
    const int jb = blockIdx.x >> 3;
    return (jb / group) * (8 * group) + (blockIdx.x & 7) * group + jb % group;
}
long long xcd_grid(long long tiles, int group) { return (tiles + 8LL * group - 1) / (8LL * group) * (8LL * group); }
// Tiles per XCD group of the dgrad kernels: about one routed expert (two
// row tiles x all channel tiles), whose tiles share its rows of dO.
__host__ __device__ __forceinline__ int dgrad_group(int n_ct) { return 2 * n_ct; }

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
}  // namespace

// ---- wgrad + saliency: one tile = 256 hidden units x 256 channels of one
// (matrix, expert) ----------------------------------------------------------
__global__ __launch_bounds__(THREADS, WAVES_PER_SIMD) void sal_wgrad_kernel(SalWgradParams p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[SMEM3];
    // all tiles of one (matrix, expert) on one XCD: they share its x^T (or
    // dO^T) rows and its dG^T (dU^T, h^T) rows
    const int L = xcd_tile(p.nI * p.nM);
    if (L >= 3 * p.E * p.nI * p.nM) return;
    const int mtile = L % p.nM;
    int rest = L / p.nM;
    const int ntile = rest % p.nI;
    rest /= p.nI;
    const int e = rest % p.E, mat = rest / p.E;
    const SegMeta sm = p.seg[p.hs + e];
    const int MP = p.nM * WM;  // partial sums per channel
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int wm = wave / WN, wn = wave % WN;
    float* part_out = p.partial + ((size_t)mat * p.E + e) * p.I * MP;

    if (sm.rows == 0) {  // no token reached the expert: its gradient is zero
        if (lane < 32)
#pragma unroll
            for (int j = 0; j < NF; ++j) {
                const int c = ntile * BN + wn * WCOL + j * 32 + lane;
                if (c < p.I) part_out[(size_t)c * MP + mtile * WM + wm] = 0.f;
            }
        return;
    }

    const bf16_t* A = p.a[mat] + sm.prow0;
    const bf16_t* B = p.b[mat] + sm.prow0;
    NTOperands op;
    op.K = sm.rows;
    op.ra = make_rsrc(A, (size_t)p.d * p.ldt - sm.prow0);
    op.rb = make_rsrc(B, (size_t)p.I * p.ldt - sm.prow0);
    int bcol[NI];
    nt_rows(wave, lane, mtile * BM, p.d, p.ldt, op.aoff, op.acol);
    nt_rows(wave, lane, ntile * BN, p.I, p.ldt, op.boff, bcol);

    // theta = W[c][m] of the tile's 256 channels x 256 hidden units (gate, up
    // or the transposed down weight), brought into the operand stages by the
    // loop's last two DMA slots, while its last K tiles are multiplied.
    // Slot h holds channels h*128 .. +128, one 512-byte row each: rows 0..63
    // in A stage (nk + h) % 3, rows 64..127 in B stage (nk + h) % 2; 16-byte
    // chunk pos of row r holds hidden units 8 * (pos ^ (r % 32)) ..
    const bf16_t* W = p.w[mat] + (size_t)e * p.I * p.d;
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(W, (size_t)p.I * p.d);
    auto theta_tail = [&](int h, bool part_a, unsigned char* dst) {
        const int part = part_a ? 0 : 1;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int tr = part * 64 + wave * 8 + 2 * i + (lane >> 5);  // theta row of the slot
            const int c = ntile * BN + h * 128 + tr;
            const int m = mtile * BM + ((lane & 31) ^ (tr & 31)) * 8;
            const uint32_t off = c < p.I && m < p.d ? (uint32_t)(((size_t)c * p.d + m) * 2) : kOOB;
            load_lds16(rw, off, 0, dst + i * RPI * ROWB);
        }
    };
    const int nk = ceil_div(op.K, BK);
    by_rows(p.d - mtile * BM, [&](auto tag) {
        constexpr int MFW = decltype(tag)::value;
        floatx16 acc[MFW][NF];
        nt_mainloop<MFW, true>(smem, op, wave, lane, acc, theta_tail);
        barrier_no_fence();  // every wave's theta DMAs have landed
        // epilogue: lane -> channel c, register v -> hidden unit
        // 8(v/4) + 4(lane/32) + v%4 of a fragment; (theta * dW)^2 summed
        float part[NF];
#pragma unroll
        for (int j = 0; j < NF; ++j) {
            part[j] = 0.f;
            const int cl = wn * WCOL + j * 32 + (lane & 31);  // channel within the tile
            const int h = cl >> 7, tr = cl & 127;
            const unsigned char* trow = (tr < 64 ? smem + ((nk + h) % 3) * STAGE_A
                                                 : smem + 3 * STAGE_A + ((nk + h) % 2) * STAGE_B) +
                                        (tr & 63) * 512;
#pragma unroll
            for (int i = 0; i < MFW; ++i)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int ml = wm * 32 * MFW + i * 32 + q * 8 + (lane >> 5) * 4;
                    const uint2 th = *reinterpret_cast<const uint2*>(
                        trow + (((ml >> 3) ^ (cl & 31)) << 4) + (ml & 7) * 2);
                    const float t0 = lo_bf16(th.x) * acc[i][j][q * 4 + 0];
                    const float t1 = hi_bf16(th.x) * acc[i][j][q * 4 + 1];
                    const float t2 = lo_bf16(th.y) * acc[i][j][q * 4 + 2];
                    const float t3 = hi_bf16(th.y) * acc[i][j][q * 4 + 3];
                    part[j] += (t0 * t0 + t1 * t1) + (t2 * t2 + t3 * t3);
                }
        }
#pragma unroll
        for (int j = 0; j < NF; ++j) part[j] += __shfl_xor(part[j], 32, 64);
        if (lane < 32)
#pragma unroll
            for (int j = 0; j < NF; ++j) {
                const int c = ntile * BN + wn * WCOL + j * 32 + lane;
                if (c < p.I) part_out[(size_t)c * MP + mtile * WM + wm] = part[j];
            }
    });
}

// ---- training backward of the masked layer ---------------------------------
namespace {
// Tile L of the training backward's tile list: the shared expert's tiles
// first (ceil(T/256) row tiles x nsh column tiles), then the routed segments'
// (row tiles numbered by SegMeta::rt0, x nr column tiles).  False past the end.
__device__ __forceinline__ bool train_tile(const SegMeta* seg, int hs, int nseg, int T, int Is, int nsh, int nr,
                                           int L, SegMeta& sm, int& mtile, int& ntile, bool with_shared = true) {
    if (hs && with_shared) {
        const int mt = ceil_div(T, BM), sh = mt * nsh;
        if (L < sh) {
            sm = SegMeta{0, T, Is, 0, Is, -1, 0, 0};
            mtile = L % mt;
            ntile = L / mt;
            return true;
        }
        L -= sh;
    }
    int lo = hs, hi = nseg - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (seg[mid].rt0 * nr <= L) lo = mid;
        else hi = mid - 1;
    }
    sm = seg[lo];
    const int mt = ceil_div(sm.rows, BM);
    const int local = L - sm.rt0 * nr;
    if (local >= mt * nr) return false;
    ntile = local / mt;
    mtile = local % mt;
    return true;
}
}  // namespace

// dgrad + SwiGLU backward; tile = 256 rows x 256 channels.  The B fragment
// goes first: lane -> row, registers -> runs of 4 channels.  g and u are read
// in their fragment-blocked layout (a wave's 8-byte reads cover 512
// contiguous bytes); dG and dU are staged through LDS, half of the tile's
// channels at a time, and stored as whole 16-byte pieces.
//   kMode 2 (masked layer's training backward): shared expert included, the
//     mask gradient's partial sums, dG/dU row-major [rows][C] over the kept
//     channels;
//   kMode 1 (channel saliency): routed segments only, every channel kept,
//     dG/dU transposed -- [c][prow0 + r] of [I][ldt], zero in each segment's
//     padding rows -- for the weight-gradient GEMMs.
constexpr int DG_PITCH = BN / 2 + 8;                  // staged row (bf16): 272 bytes, 16-byte aligned
constexpr int DG_STAGE = BM * DG_PITCH * 2;           // one staged array
constexpr int DG_SMEM = (2 * DG_STAGE > SMEM3) ? 2 * DG_STAGE : SMEM3;
constexpr int DG_TPITCH = BM + 8;                     // transposed staging row (bf16): 4 rows = 16 banks
static_assert(2 * (BN / 2) * DG_TPITCH * 2 <= DG_SMEM, "the transposed staging fits");
static_assert(DG_SMEM <= 160 * 1024, "the dgrad LDS fits one compute unit");

template <int kMode>
__global__ __launch_bounds__(THREADS, WAVES_PER_SIMD) void dgrad_kernel(ActDgradParams p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[DG_SMEM];
    SegMeta sm;
    int mtile, ntile;
    if (!train_tile(p.seg, p.hs, p.nseg, p.T, p.Is, p.nIs, p.nI, xcd_tile(dgrad_group(p.nI)), sm, mtile, ntile,
                    kMode == 2))
        return;
    const bool shared = sm.e < 0;
    const int C = shared ? p.Is : p.I;  // channels (row length of g, u, dG, dU)
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int wm = wave / WN, wn = wave % WN;

    NTOperands op;
    op.K = p.d;
    const bf16_t* A = shared ? p.dYs : p.dO + (size_t)sm.row0 * p.d;
    const bf16_t* B = shared ? p.wsdt : p.wdt + (size_t)sm.e * p.I * p.d;
    op.ra = make_rsrc(A, (size_t)sm.rows * p.d);
    op.rb = make_rsrc(B, (size_t)C * p.d);
    int bcol[NI];
    nt_rows(wave, lane, mtile * BM, sm.rows, p.d, op.aoff, op.acol);
    nt_rows(wave, lane, ntile * BN, C, p.d, op.boff, bcol);

    const size_t rbase = shared ? 0 : (size_t)sm.row0;
    const bf16_t* G = shared ? p.Gs : p.G;
    const bf16_t* U = shared ? p.Us : p.U;
    bf16_t* dG = shared ? p.dGs : p.dG;
    bf16_t* dU = shared ? p.dUs : p.dU;
    const int kk = sm.kk;                        // mask: channels below kk are kept
    const int kk8 = min(packed_width(kk), C);    // dG/dU columns the dx GEMM reads
    bf16_t* stg = reinterpret_cast<bf16_t*>(smem);
    bf16_t* stu = stg + (kMode == 2 ? BM * DG_PITCH : (BN / 2) * DG_TPITCH);
    by_rows(sm.rows - mtile * BM, [&](auto tag) {
        constexpr int MFW = decltype(tag)::value;
        floatx16 acc[MFW][NF];
        nt_mainloop<MFW, false>(smem, op, wave, lane, acc, ZeroTail{op.ra});
        // the stages are free once every wave is past its last fragment read
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
        barrier_no_fence();
        // epilogue: lane -> row (lane%32 of a fragment), register v ->
        // channel 8(v/4) + 4(lane/32) + v%4 of a 32-channel fragment
        float msum[NF][16];
#pragma unroll
        for (int j = 0; j < NF; ++j) {
#pragma unroll
            for (int v = 0; v < 16; ++v) msum[j][v] = 0.f;
#pragma unroll
            for (int i = 0; i < MFW; ++i) {
                const int row = wm * 32 * MFW + i * 32 + (lane & 31);  // row of the tile
                const int grow = mtile * BM + row;                     // row of the segment
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int cl = wn * 32 + q * 8 + (lane >> 5) * 4;  // staged column of this half
                    const int c0 = ntile * BN + wn * WCOL + j * 32 + q * 8 + (lane >> 5) * 4;
                    uint32_t dg[2] = {0u, 0u}, du[2] = {0u, 0u};
                    if (grow < sm.rows && c0 < C) {
                        const size_t off = frag_blocked(rbase + grow, c0, C);
                        const uint2 gv = *reinterpret_cast<const uint2*>(G + off);
                        const uint2 uv = *reinterpret_cast<const uint2*>(U + off);
                        const float g[4] = {lo_bf16(gv.x), hi_bf16(gv.x), lo_bf16(gv.y), hi_bf16(gv.y)};
                        const float u[4] = {lo_bf16(uv.x), hi_bf16(uv.x), lo_bf16(uv.y), hi_bf16(uv.y)};
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const float x = g[r];
                            const float sg = 1.0f / (1.0f + __builtin_amdgcn_exp2f(-x * 1.4426950408889634f));
                            const float dh = acc[i][j][q * 4 + r];
                            if constexpr (kMode == 2) msum[j][q * 4 + r] += dh * (x * sg) * u[r];
                            const bool kept = c0 + r < kk;
                            const float vg = kept ? dh * u[r] * (sg * (1.0f + x * (1.0f - sg))) : 0.f;
                            const float vu = kept ? dh * (x * sg) : 0.f;
                            dg[r >> 1] |= (uint32_t)f32_to_bf16(vg) << (16 * (r & 1));
                            du[r >> 1] |= (uint32_t)f32_to_bf16(vu) << (16 * (r & 1));
                        }
                    }
                    if constexpr (kMode == 2) {
                        *reinterpret_cast<uint2*>(stg + row * DG_PITCH + cl) = make_uint2(dg[0], dg[1]);
                        *reinterpret_cast<uint2*>(stu + row * DG_PITCH + cl) = make_uint2(du[0], du[1]);
                    } else {  // staged transposed: [channel][row]
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            stg[(cl + r) * DG_TPITCH + row] = (bf16_t)(dg[r >> 1] >> (16 * (r & 1)));
                            stu[(cl + r) * DG_TPITCH + row] = (bf16_t)(du[r >> 1] >> (16 * (r & 1)));
                        }
                    }
                }
            }
            __syncthreads();
            // staged column cl of half j is channel ntile*BN + (cl/32)*WCOL + j*32 + cl%32
            if constexpr (kMode == 2) {
                for (int k = threadIdx.x; k < BM * (BN / 2 / 8); k += THREADS) {
                    const int row = k / (BN / 2 / 8), cl = (k % (BN / 2 / 8)) * 8;
                    const int grow = mtile * BM + row;
                    const int c = ntile * BN + (cl / 32) * WCOL + j * 32 + cl % 32;
                    if (grow >= sm.rows || c >= kk8) continue;
                    const size_t o = (rbase + grow) * (size_t)C + c;
                    *reinterpret_cast<u32x4*>(dG + o) = *reinterpret_cast<const u32x4*>(stg + row * DG_PITCH + cl);
                    *reinterpret_cast<u32x4*>(dU + o) = *reinterpret_cast<const u32x4*>(stu + row * DG_PITCH + cl);
                }
            } else {
                // rows up to the segment's padded height (zeros past its rows)
                const int pvalid = packed_width(sm.rows) - mtile * BM;
                const size_t col = (size_t)sm.prow0 + mtile * BM;
                for (int k = threadIdx.x; k < (BN / 2) * (BM / 8); k += THREADS) {
                    const int cl = k / (BM / 8), r0 = (k % (BM / 8)) * 8;
                    const int c = ntile * BN + (cl / 32) * WCOL + j * 32 + cl % 32;
                    if (r0 >= pvalid || c >= C) continue;
                    const size_t o = (size_t)c * p.ldt + col + r0;
                    *reinterpret_cast<u32x4*>(dG + o) = *reinterpret_cast<const u32x4*>(stg + cl * DG_TPITCH + r0);
                    *reinterpret_cast<u32x4*>(dU + o) = *reinterpret_cast<const u32x4*>(stu + cl * DG_TPITCH + r0);
                }
            }
            __syncthreads();
        }
        if (kMode == 1 || shared) return;
        // mask-gradient partial sums: over the 32 rows of the lane group
#pragma unroll
        for (int j = 0; j < NF; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                float t = msum[j][v];
#pragma unroll
                for (int o = 1; o < 32; o <<= 1) t += __shfl_xor(t, o, 64);
                msum[j][v] = t;
            }
        if ((lane & 31) == 0) {
            float* out = p.dmp + ((size_t)(sm.rt0 + mtile) * kTrainWaveM + wm) * p.I;
#pragma unroll
            for (int j = 0; j < NF; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int c = ntile * BN + wn * WCOL + j * 32 + q * 8 + (lane >> 5) * 4 + r;
                        if (c < p.I) out[c] = msum[j][q * 4 + r];
                    }
        }
    });
}

// dX = dG W_gate + dU W_up over the kept channels; tile = 256 rows x 256
// hidden units, two K loops into one accumulator.
__global__ __launch_bounds__(THREADS, WAVES_PER_SIMD) void act_dx_kernel(ActDxParams p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[SMEM3];
    SegMeta sm;
    int mtile, ntile;
    if (!train_tile(p.seg, p.hs, p.nseg, p.T, p.Is, p.nD, p.nD, xcd_tile(dgrad_group(p.nD)), sm, mtile, ntile))
        return;
    const bool shared = sm.e < 0;
    const int C = shared ? p.Is : p.I;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int wm = wave / WN, wn = wave % WN;
    const size_t rbase = shared ? 0 : (size_t)sm.row0;

    NTOperands og, ou;
    og.K = ou.K = sm.kk;
    const bf16_t* Ag = (shared ? p.dGs : p.dG) + rbase * C;
    const bf16_t* Au = (shared ? p.dUs : p.dU) + rbase * C;
    const bf16_t* Bg = shared ? p.wsgt : p.wgt + (size_t)sm.e * p.d * p.I;
    const bf16_t* Bu = shared ? p.wsut : p.wut + (size_t)sm.e * p.d * p.I;
    og.ra = make_rsrc(Ag, (size_t)sm.rows * C);
    ou.ra = make_rsrc(Au, (size_t)sm.rows * C);
    og.rb = make_rsrc(Bg, (size_t)p.d * C);
    ou.rb = make_rsrc(Bu, (size_t)p.d * C);
    int bcol[NI];
    nt_rows(wave, lane, mtile * BM, sm.rows, C, og.aoff, og.acol);
    nt_rows(wave, lane, ntile * BN, p.d, C, og.boff, bcol);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        ou.aoff[i] = og.aoff[i];
        ou.boff[i] = og.boff[i];
        ou.acol[i] = og.acol[i];
    }
    float* out = (shared ? p.dXs : p.dXr) + rbase * p.d;
    by_rows(sm.rows - mtile * BM, [&](auto tag) {
        constexpr int MFW = decltype(tag)::value;
        floatx16 acc[MFW][NF];
        nt_mainloop<MFW, false>(smem, og, wave, lane, acc, ZeroTail{og.ra});
        // every wave is past its last LDS read before the second loop refills the stages
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
        barrier_no_fence();
        nt_mainloop<MFW, false>(smem, ou, wave, lane, acc, ZeroTail{ou.ra}, false);
        // epilogue: lane -> row, registers -> runs of 4 hidden units
#pragma unroll
        for (int i = 0; i < MFW; ++i) {
            const int row = mtile * BM + wm * 32 * MFW + i * 32 + (lane & 31);
            if (row >= sm.rows) continue;
#pragma unroll
            for (int j = 0; j < NF; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int n0 = ntile * BN + wn * WCOL + j * 32 + q * 8 + (lane >> 5) * 4;
                    if (n0 >= p.d) continue;
                    *reinterpret_cast<float4*>(out + (size_t)row * p.d + n0) =
                        make_float4(acc[i][j][q * 4], acc[i][j][q * 4 + 1], acc[i][j][q * 4 + 2],
                                    acc[i][j][q * 4 + 3]);
                }
        }
    });
}

hipError_t launch_act_dgrad(const ActDgradParams& p, long long tiles, hipStream_t s) {
    if (tiles <= 0) return hipSuccess;
    const long long g = xcd_grid(tiles, dgrad_group(p.nI));
    dgrad_kernel<2><<<(int)g, THREADS, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_sal_dgrad(const ActDgradParams& p, long long tiles, hipStream_t s) {
    if (tiles <= 0) return hipSuccess;
    const long long g = xcd_grid(tiles, dgrad_group(p.nI));
    dgrad_kernel<1><<<(int)g, THREADS, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_act_dx(const ActDxParams& p, long long tiles, hipStream_t s) {
    if (tiles <= 0) return hipSuccess;
    const long long g = xcd_grid(tiles, dgrad_group(p.nD));
    act_dx_kernel<<<(int)g, THREADS, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_sal_wgrad(const SalWgradParams& p, hipStream_t s) {
    const long long tiles = 3LL * p.E * p.nI * p.nM;
    if (tiles <= 0) return hipSuccess;
    const long long g = xcd_grid(tiles, p.nI * p.nM);
    sal_wgrad_kernel<<<(int)g, THREADS, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace flexmoe
