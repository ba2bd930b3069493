// Argument blocks and launchers of the masked layer's training step (FlexMoE
// Sec. 3.2): the straight-through Gumbel-softmax action sample (Eq. 5), the
// backward of the sampled subnet -- input, router-logit and mask gradients --
// and the action-logit gradient (Eqs. 6-8).
#pragma once

#include "kernels.h"

namespace flexmoe {

constexpr int kTrainTile = 256;    // rows x channels (or hidden units) of the dgrad and dx tiles
constexpr int kTrainWaveM = 2;     // mask-gradient partial sums per routed row tile and channel
constexpr int kMaxActions = 16;

// dgrad of every segment (shared expert first) with the SwiGLU backward and
// the mask gradient fused: dH' = dO W_down over all channels, then
//   dM partial += dH' * silu(g) * u           (routed, every channel)
//   dG = [c < k] dH' u silu'(g), dU = [c < k] dH' silu(g)
struct ActDgradParams {
    const bf16_t* dO;       // [A][d] routed rows in dispatch order: w_a * dY_t
    const bf16_t* dYs;      // [T][d] dY, the shared expert's output gradient
    const bf16_t* wdt;      // [E][I][d] routed W_down^T
    const bf16_t* wsdt;     // [I_s][d] shared W_down^T
    const bf16_t* G;        // [A][I] forward pre-activations (training forward),
    const bf16_t* U;        //   fragment-blocked (common.h)
    const bf16_t* Gs;       // [T][I_s], fragment-blocked
    const bf16_t* Us;
    const SegMeta* seg;
    bf16_t* dG;             // [A][I]: channels below packed_width(k) written
    bf16_t* dU;
    bf16_t* dGs;            // [T][I_s]
    bf16_t* dUs;
    float* dmp;             // [routed row tiles][kTrainWaveM][I] mask-gradient partial sums
    int hs, nseg, d, I, Is, T, nI, nIs;   // nI = ceil(I / kTrainTile), nIs likewise
    int ldt;                // launch_sal_dgrad: dG, dU are [I][ldt], written transposed
};

// dx rows: dX = dG W_gate + dU W_up, K = k (routed) or I_s (shared).
struct ActDxParams {
    const bf16_t* dG;       // [A][I]
    const bf16_t* dU;
    const bf16_t* dGs;      // [T][I_s]
    const bf16_t* dUs;
    const bf16_t* wgt;      // [E][d][I] routed W_gate^T, W_up^T
    const bf16_t* wut;
    const bf16_t* wsgt;     // [d][I_s] shared W_gate^T, W_up^T
    const bf16_t* wsut;
    const SegMeta* seg;
    float* dXr;             // [A][d]
    float* dXs;             // [T][d]
    int hs, nseg, d, I, Is, T, nD;        // nD = ceil(d / kTrainTile)
};

struct ActionWidths {
    int32_t K;
    int32_t width[kMaxActions];   // ceil(r_k * I)
    float ratio[kMaxActions];
};

hipError_t launch_gemm1_big_train_rm(const Gemm1Params<bf16_t>& p, int grid, hipStream_t s);
hipError_t launch_act_dgrad(const ActDgradParams& p, long long tiles, hipStream_t s);
// The channel saliency's dgrad (the same kernel): routed segments only, no
// mask, dG and dU written transposed -- element [c][prow0 + r] of [I][ldt],
// zeros in each segment's padding rows -- and no mask gradient (dmp unused).
hipError_t launch_sal_dgrad(const ActDgradParams& p, long long tiles, hipStream_t s);
hipError_t launch_act_dx(const ActDxParams& p, long long tiles, hipStream_t s);
// seg[s].kg = seg[s].kk: the down GEMM of the training forward reduces over
// the kept channels only (the gate/up GEMM computed all of them)
hipError_t launch_seg_use_kept(SegMeta* seg, int nseg, hipStream_t s);
// dO = bf16(w_a dY_t) for the *nrouted dispatched rows, dYs = bf16(dY)
hipError_t launch_train_prep(const float* dy, const int32_t* perm, const float* wts, const int32_t* nrouted,
                             int A, int T, int d, int k, bf16_t* dO, bf16_t* dYs, hipStream_t s);
// dx = sum of the token's routed rows + the shared row; dlogits through the
// router's softmax (and renormalisation)
hipError_t launch_combine_backward(const float* dXr, const float* dXs, const bf16_t* O, const int32_t* pos,
                                   const int32_t* idx, const float* wts, const float* logits, const float* dy,
                                   int T, int E, int k, int d, int norm_topk, float* dx, float* dlogits,
                                   hipStream_t s);
hipError_t launch_dmask_reduce(const float* dmp, const SegMeta* seg, int hs, int E, int I, float* dmask,
                               hipStream_t s);
hipError_t launch_sample_actions(const ActionWidths& aw, const float* alpha, const float* gumbel, int E,
                                 int32_t* keep, int32_t* action, hipStream_t s);
// per_expert: [E][2] scratch for the cost and entropy of each expert
hipError_t launch_action_grad(const ActionWidths& aw, const float* alpha, const float* gumbel, float tau,
                              const float* dmask, const int32_t* counts, long long assignments, int E, int I,
                              float lambda_cost, float beta, float* dalpha, float* per_expert, float* stats,
                              hipStream_t s);
hipError_t launch_transpose_batched(const bf16_t* src, bf16_t* dst, int batch, int rows, int cols,
                                    hipStream_t s);

}  // namespace flexmoe
