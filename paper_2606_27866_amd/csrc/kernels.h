// Kernel declarations and argument blocks of the FlexMoE HIP library.
#pragma once

#include <type_traits>

#include "common.h"

namespace flexmoe {

struct KeepArgs {
    int32_t v[kMaxExperts];
};

// Which segments one GEMM launch covers.  The shared expert needs no routing,
// so its GEMMs can run on a second stream while the routed experts are being
// dispatched; each launch then covers one part of the tile list.
enum GemmPart : int32_t {
    kPartRange = 0,   // segments [seg_lo, seg_hi) (tiles tstart[seg_lo] .. tstart[seg_hi])
    kPartShared = 1   // the shared expert alone; its tile count comes from the host
};

// Gate/up GEMM with fused SwiGLU:
//   H[row][c] = silu(<W_gate[c], x_t>) * <W_up[c], x_t>,  c < k_s
// over every segment s (routed experts, then the shared expert).
template <typename T>
struct Gemm1Params {
    const T* x;                 // [T][d]
    const T* wg;                // routed gate [E][I][d]
    const T* wu;                // routed up   [E][I][d]
    const T* sg;                // shared gate [I_s][d]
    const T* su;                // shared up   [I_s][d]
    const int32_t* perm;        // grouped row -> assignment id
    const SegMeta* seg;         // [nseg]
    const int32_t* tstart;      // [nseg+1] first tile of each segment
    T* H;                       // routed activations [A][I]
    T* Hs;                      // shared activations [T][I_s]
    int d, I, Is, E, top_k, nseg, tokens;
    int part;                   // GemmPart
    int seg_lo, seg_hi;         // kPartRange: the segments covered
    int shared_tiles;           // tiles of the shared segment (kPartShared)
    int clipped;                // routed weights in the clipped layout (see RoutedWeights)
    // Training forwards: g and u for every channel the GEMM computes (c < kg),
    // in the fragment-blocked layout (common.h) of a routed [A][I] and a shared
    // [T][I_s] matrix (launch_gemm1_big_train: routed rows only;
    // launch_gemm1_big_train_rm: all rows).
    T* G;
    T* U;
    T* Gs;
    T* Us;
    // launch_gemm1_big_train only: the routed rows' activations h transposed --
    // element [c][prow0 + r] for row r of a segment -- with zeros in the rows
    // [rows, packed_width(rows)) of each segment.  Row stride ldt.
    T* ht;
    int ldt;
};

// Down GEMM: O[row][n] = sum_{c < k_s} H[row][c] * W_down[n][c].  O holds one
// row per routed assignment (and per token for the shared expert); it is fp32
// in fp32 mode and bf16 (rounded once from the fp32 sum) in bf16 mode.
template <typename T>
struct Gemm2Params {
    typedef typename std::conditional<std::is_same<T, float>::value, float, bf16_t>::type OT;
    const T* H;
    const T* Hs;
    const T* wd;                // routed down [E][d][I]
    const T* sd;                // shared down [d][I_s]
    const SegMeta* seg;
    const int32_t* tstart;
    OT* O;                      // routed rows [A][d]
    OT* Os;                     // shared rows [T][d] (split reductions: [splits][T][d])
    int d, I, Is, E, nseg, tokens;
    int ks2;                    // > 0: the shared reduction is split into chunks of ks2 channels
    int part;                   // GemmPart
    int seg_lo, seg_hi;         // kPartRange: the segments covered
    int shared_tiles;           // tiles of the shared segment (kPartShared)
    int clipped;                // routed weights in the clipped layout (see RoutedWeights)
    // Tile order (kPartRange): tstart, seg_lo and seg_hi count positions in
    // this order of the segments (NULL: segment order).  The dispatch puts the
    // shared expert first, then the routed experts by decreasing GEMM width:
    // the longest reductions start first, so the launch ends evenly.
    const int32_t* order = nullptr;
};

// Where routed expert e's weights live.  Ranked layout (online clipping):
// gate/up [E][I][d], down [E][d][I]; expert e's blocks start at e*I*d and a
// down row holds I channels.  Clipped layout (one budget exported offline):
// the experts' blocks are packed back to back, expert e holding
// packed_width(k_e) channels -- gate/up [kp_e][d], down [d][kp_e] -- from
// packed channel ch0; both blocks start at ch0*d and a down row holds kp_e
// channels.
struct RoutedWeights {
    size_t base;   // element offset of the expert's gate/up block and of its down block
    int rows;      // gate/up rows the block holds
    int ldd;       // elements per down row
};
template <typename P>
__device__ __forceinline__ RoutedWeights routed_weights(const P& p, const SegMeta& sm) {
    if (p.clipped) return RoutedWeights{(size_t)sm.ch0 * p.d, packed_width(sm.kk), packed_width(sm.kk)};
    return RoutedWeights{(size_t)sm.e * p.I * p.d, p.I, p.I};
}

// Segment at tile-order position i (down GEMM: Gemm2Params::order).
__device__ __forceinline__ int order_of(const Gemm1Params<bf16_t>&, int i) { return i; }
__device__ __forceinline__ int order_of(const Gemm1Params<float>&, int i) { return i; }
template <typename T>
__device__ __forceinline__ int order_of(const Gemm2Params<T>& p, int i) {
    return p.order ? min(max(p.order[i], 0), p.nseg - 1) : i;
}

// Tile L of a launch -> segment s, its metadata and the tile's index inside
// the segment.  False when L is past the launch's last tile (the caller's
// workgroup then has nothing to do).  The shared segment's metadata is known
// without the dispatch tables: rows = tokens, channels = I_s.  The shared
// expert, when present, is always segment 0.
template <typename P>
__device__ __forceinline__ bool tile_of(const P& p, int L, int& s, SegMeta& sm, int& local) {
    if (p.part == kPartShared) {
        if (L >= p.shared_tiles) return false;
        // the argument values are pinned in scalar registers here: otherwise
        // the compiler may merge the read of `tokens` with the routed path's
        // read of seg[s].rows into one generic (flat) load, one more memory
        // round trip at the start of every tile
        int tokens = p.tokens, is = p.Is;
        asm volatile("" : "+s"(tokens), "+s"(is));
        s = 0;
        sm = SegMeta{0, tokens, is, 0, is, -1, 0, 0};
        local = L;
        return true;
    }
    const int t_lo = p.tstart[p.seg_lo], t_hi = p.tstart[p.seg_hi];  // both requested before either is used
    L += t_lo;
    if (L >= t_hi) return false;
    const int i = find_segment(p.tstart, p.nseg, L);
    s = order_of(p, i);
    sm = p.seg[s];
    local = L - p.tstart[i];
    return true;
}

// Tile shapes of the kernel families (the dispatch kernel builds tile tables
// with these numbers).
constexpr int kF32BM = 64, kF32BN = 64;
constexpr int kBigBM1 = 256, kBigBN1 = 128, kBigBM2 = 256, kBigBN2 = 256;
constexpr int kDecodeMaxT = 64;     // T at or below which the weight-streaming kernels run
constexpr int kGemvMaxT = 8;        // T at or below which the routed experts' weight-streaming
                                    // GEMMs run on the vector ALUs, in tiles of kDecBN channels /
                                    // output columns (launch_gemm*_decode); above, in tiles of
                                    // kDecWideBN on the matrix cores (launch_gemm*_decode_wide)
constexpr int kDecBN = 16;
constexpr int kDecWideBN = 64;
constexpr int kDecodeWideSharedT = 5;  // above this many tokens the shared expert takes the wide
                                       // tiles too
constexpr int kSharedSplit2T = 16;  // above this many (decode) tokens the shared expert's down
                                    // reduction is split into chunks of 2 I channels, else of I

__global__ void route_kernel(const float* logits, int T, int E, int k, int norm_topk, int32_t* idx,
                             float* wts, int32_t* blockcnt, int NB);
__global__ void dispatch_scan_kernel(const int32_t* blockcnt, int NB, int32_t* blockbase,
                                     int32_t* counts);
// `packed_limit`: in the clipped layout, the packed channels the weight
// buffers hold; an expert whose block would reach past it is treated as
// k_e = 0 (the ranked layout passes INT32_MAX).  `plan` (NULL: experts in id
// order, GEMM width = k_e): the bucketed forward's segment order plan[0..E)
// (expert ids) and GEMM widths plan[E..2E).
__global__ void set_plan_kernel(int32_t* keep, int32_t* plan, KeepArgs k, KeepArgs order, KeepArgs kg, int E);
__global__ void dispatch_scatter_kernel(const int32_t* idx, const int32_t* keep,
                                        const int32_t* counts, const int32_t* blockbase, int T,
                                        int E, int k, int I, int I_shared, int d, int NB,
                                        TileShape ts, int packed_limit, const int32_t* plan,
                                        int32_t* perm, int32_t* pos,
                                        int32_t* offsets, SegMeta* seg, int32_t* t1start,
                                        int32_t* t2start, int32_t* order2);
__global__ void dispatch_small_kernel(const float* logits, int T, int E, int k, int norm_topk,
                                      const int32_t* keep, int I, int I_shared, int d, TileShape ts,
                                      int packed_limit, const int32_t* plan, int pre_routed, int32_t* idx,
                                      float* wts, int32_t* counts,
                                      int32_t* perm, int32_t* pos, int32_t* offsets, SegMeta* seg,
                                      int32_t* t1start, int32_t* t2start, int32_t* order2);
__global__ void set_keep_kernel(int32_t* keep, KeepArgs t, int E);

// Launchers (defined next to their kernels).  Each returns the launch status.
// full_lds: the launch takes all of a compute unit's LDS (a third token-row
// stage).  Not for the shared expert's side-stream launches, which start
// beside the routing kernels and would lock them out of the compute units;
// the routed launches that follow the routing may (they and the side-stream
// launches cannot share a compute unit's LDS either way).
// alone (gate/up): no side-stream launch runs at all; implies full_lds.
hipError_t launch_gemm1_big(const Gemm1Params<bf16_t>& p, int grid, hipStream_t s, bool full_lds, bool alone);
hipError_t launch_gemm2_big(const Gemm2Params<bf16_t>& p, int grid, hipStream_t s, bool full_lds);
// T <= kGemvMaxT: 16-wide tiles on the vector ALUs (gemv_decode.hip).
hipError_t launch_gemm1_decode(const Gemm1Params<bf16_t>& p, int tiles, hipStream_t s);
hipError_t launch_gemm2_decode(const Gemm2Params<bf16_t>& p, int tiles, hipStream_t s);
// T <= kDecodeMaxT: tiles of kDecWideBN channels / output columns on the
// matrix cores (gemm_decode.hip).
hipError_t launch_gemm1_decode_wide(const Gemm1Params<bf16_t>& p, int tiles, hipStream_t s);
hipError_t launch_gemm2_decode_wide(const Gemm2Params<bf16_t>& p, int tiles, hipStream_t s);
hipError_t launch_gemm1_f32(const Gemm1Params<float>& p, int grid, hipStream_t s);
hipError_t launch_gemm2_f32(const Gemm2Params<float>& p, int grid, hipStream_t s);
hipError_t launch_combine(const void* O, const void* Os, const int32_t* pos, const float* wts,
                          int T, int k, int d, int shared_parts, int dtype, void* y, hipStream_t s);
hipError_t launch_rank_reorder(const float* scores, const void* wg, const void* wu,
                               const void* wd, void* wg_r, void* wu_r, void* wd_r,
                               int32_t* perm, int E, int I, int d, int esize, hipStream_t s);
// Packs one budget's ranked weights into the clipped layout (RoutedWeights);
// keep holds the budget, already validated on the host.
hipError_t launch_export_clipped(const KeepArgs& keep, const void* wg_r, const void* wu_r,
                                 const void* wd_r, void* wg_c, void* wu_c, void* wd_c, int E, int I,
                                 int d, int esize, hipStream_t s);

}  // namespace flexmoe
