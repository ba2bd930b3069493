// Argument blocks and launchers of the channel-saliency kernels (FlexMoE
// Sec. 3.1, Eq. 2): the backward of the unpruned layer for a layer-level
// loss, reduced to one score per hidden channel of every routed expert.
#pragma once

#include "train.h"

namespace flexmoe {

constexpr int kSalTile = 256;   // rows x channels of the dgrad and wgrad tiles
constexpr int kSalWaveM = 2;    // partial sums per channel from one wgrad tile

// wgrad of the three routed matrices with the Eq. 2 reduction fused; tile
// (mat, e, channel tile, hidden-unit tile) writes kSalWaveM partial sums per
// channel.
struct SalWgradParams {
    const bf16_t* a[3];     // [d][ldt]: x^T, x^T, dO^T
    const bf16_t* b[3];     // [I][ldt]: dG^T, dU^T, h^T
    const bf16_t* w[3];     // [E][I][d]: W_gate, W_up, W_down^T (theta)
    const SegMeta* seg;
    float* partial;         // [3][E][I][nM * kSalWaveM]
    int hs, d, I, E, ldt, nI, nM;   // nM = ceil(d / kSalTile)
};

// Transposed copies of x and of dO = w_a dY_t for the routed rows, and dO
// itself in dispatch order.
struct SalPrepParams {
    const bf16_t* x;        // [T][d]
    const float* dy;        // [T][d] fp32
    const int32_t* perm;    // dispatch order -> assignment id
    const float* wts;       // [T*k] router weights
    const SegMeta* seg;
    bf16_t* xt;             // [d][ldt]
    bf16_t* dot;            // [d][ldt]
    bf16_t* dO;             // [A][d]
    int d, k, hs, nseg, ldt;
};

hipError_t launch_gemm1_big_train(const Gemm1Params<bf16_t>& p, int grid, hipStream_t s);
hipError_t launch_sal_wgrad(const SalWgradParams& p, hipStream_t s);
hipError_t launch_sal_prep(const SalPrepParams& p, hipStream_t s);
hipError_t launch_sal_reduce(const float* partial, int E, int I, int parts, float scale, float* scores,
                             hipStream_t s);
// dY = (the combined layer output in fp32, before any rounding) - target.
hipError_t launch_combine_residual(const bf16_t* O, const bf16_t* Os, const int32_t* pos, const float* wts,
                                   int T, int k, int d, int shared_parts, const float* target, float* dy,
                                   hipStream_t s);

}  // namespace flexmoe
