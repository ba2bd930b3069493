// The small kernels of the masked layer's training step (FlexMoE Sec. 3.2)
// around its GEMMs (gemm_bf16_big.hip, gemm_bwd.hip):
//   - the straight-through Gumbel-softmax sample of one action per expert
//     (Eq. 5), written as the device keep table of the forward;
//   - the backward's input rows dO = w_a dY_t (routed) and dY (shared);
//   - the combine backward: dx per token and the router-logit gradient;
//   - the mask gradient's final sums and the action-logit gradient through
//     the straight-through estimator, plus the cost and entropy terms
//     (Eqs. 6-8).
// Fixed summation orders throughout: repeated calls give identical bits.
#include "train.h"

namespace flexmoe {

namespace {
__device__ __forceinline__ float lo_bf(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
}  // namespace

// One thread per expert: k* = argmax_k (alpha + g) (first index on ties; the
// softmax of Eq. 5 is monotone in its argument), keep = ceil(r_k* I).
__global__ void sample_actions_kernel(ActionWidths aw, const float* __restrict__ alpha,
                                      const float* __restrict__ gumbel, int E, int32_t* __restrict__ keep,
                                      int32_t* __restrict__ action) {
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= E) return;
    const float* a = alpha + (size_t)e * aw.K;
    const float* g = gumbel + (size_t)e * aw.K;
    int best = 0;
    float bv = a[0] + g[0];
    for (int k = 1; k < aw.K; ++k) {
        const float v = a[k] + g[k];
        if (v > bv) {
            bv = v;
            best = k;
        }
    }
    keep[e] = aw.width[best];
    if (action) action[e] = best;
}

__global__ void seg_use_kept_kernel(SegMeta* seg, int nseg) {
    const int s = blockIdx.x * blockDim.x + threadIdx.x;
    if (s < nseg) seg[s].kg = seg[s].kk;
}

// Rows r < A: dO[r] = bf16(w_a dY_t) with a = perm[r]; rows A + t: dYs[t] =
// bf16(dY_t).  Eight columns per thread.
__global__ __launch_bounds__(256) void train_prep_kernel(const float* __restrict__ dy,
                                                         const int32_t* __restrict__ perm,
                                                         const float* __restrict__ wts,
                                                         const int32_t* __restrict__ nrouted, int A, int T,
                                                         int d, int k, bf16_t* __restrict__ dO,
                                                         bf16_t* __restrict__ dYs) {
    const int r = blockIdx.x;
    const int n = (blockIdx.y * blockDim.x + threadIdx.x) * 8;
    if (n >= d) return;
    float w = 1.f;
    int t;
    bf16_t* out;
    if (r < A) {
        if (r >= *nrouted) return;  // rows of experts at k = 0 are not dispatched
        const int a = perm[r];
        t = a / k;
        w = wts[a];
        out = dO + (size_t)r * d + n;
    } else {
        t = r - A;
        if (!dYs) return;
        out = dYs + (size_t)t * d + n;
    }
    const float4 f0 = *reinterpret_cast<const float4*>(dy + (size_t)t * d + n);
    const float4 f1 = *reinterpret_cast<const float4*>(dy + (size_t)t * d + n + 4);
    const float v[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
    uint32_t pk[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
        pk[i] = pack_bf16x2(w * v[2 * i], w * v[2 * i + 1]);
    *reinterpret_cast<uint4*>(out) = make_uint4(pk[0], pk[1], pk[2], pk[3]);
}

// One block per token.  dx[t] = sum_j dXr[pos_j] + dXs[t] (ascending j, then
// the shared row); dw_j = <dY_t, O_pos_j>; then, with p = softmax(logits_t)
// and S = sum_j p_{i_j}:  dp_i = dw_i (or (dw_i - sum_j dw_j w_j) / S with
// norm_topk) for the selected experts, dlogits_e = p_e (dp_e - sum_i dp_i p_i).
constexpr int kCombThreads = 256;
constexpr int kCombWaves = kCombThreads / 64;
__global__ __launch_bounds__(kCombThreads) void combine_backward_kernel(
    const float* __restrict__ dXr, const float* __restrict__ dXs, const bf16_t* __restrict__ O,
    const int32_t* __restrict__ pos, const int32_t* __restrict__ idx, const float* __restrict__ wts,
    const float* __restrict__ logits, const float* __restrict__ dy, int E, int k, int d, int norm_topk,
    float* __restrict__ dx, float* __restrict__ dlogits) {
    __shared__ float red[kMaxTopK + 2][kCombWaves];
    __shared__ float bc[kMaxTopK + 2];
    const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float dwp[kMaxTopK];
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) dwp[j] = 0.f;
    for (int n = tid * 4; n < d; n += kCombThreads * 4) {
        float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 g = *reinterpret_cast<const float4*>(dy + (size_t)t * d + n);
#pragma unroll
        for (int j = 0; j < kMaxTopK; ++j) {
            if (j >= k) break;
            const int p = pos[(size_t)t * k + j];
            if (p < 0) continue;
            const float4 v = *reinterpret_cast<const float4*>(dXr + (size_t)p * d + n);
            r.x += v.x;
            r.y += v.y;
            r.z += v.z;
            r.w += v.w;
            const uint2 o = *reinterpret_cast<const uint2*>(O + (size_t)p * d + n);
            dwp[j] += (g.x * lo_bf(o.x) + g.y * hi_bf(o.x)) + (g.z * lo_bf(o.y) + g.w * hi_bf(o.y));
        }
        if (dXs) {
            const float4 v = *reinterpret_cast<const float4*>(dXs + (size_t)t * d + n);
            r.x += v.x;
            r.y += v.y;
            r.z += v.z;
            r.w += v.w;
        }
        *reinterpret_cast<float4*>(dx + (size_t)t * d + n) = r;
    }
    const float* l = logits + (size_t)t * E;
    float m = -INFINITY;
    for (int e = tid; e < E; e += kCombThreads) m = fmaxf(m, l[e]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
        if (j >= k) break;
        const float v = wave_sum_f(dwp[j]);
        if (lane == 0) red[j][wave] = v;
    }
    if (lane == 0) red[kMaxTopK][wave] = m;
    __syncthreads();
    if (tid < k) {
        float s = 0.f;
        for (int w = 0; w < kCombWaves; ++w) s += red[tid][w];
        bc[tid] = s;
    }
    if (tid == 0) {
        float mm = red[kMaxTopK][0];
        for (int w = 1; w < kCombWaves; ++w) mm = fmaxf(mm, red[kMaxTopK][w]);
        bc[kMaxTopK] = mm;
    }
    __syncthreads();
    const float mx = bc[kMaxTopK];
    float z = 0.f;
    for (int e = tid; e < E; e += kCombThreads) z += expf(l[e] - mx);
    z = wave_sum_f(z);
    if (lane == 0) red[kMaxTopK + 1][wave] = z;
    __syncthreads();
    if (tid == 0) {
        float zz = 0.f;
        for (int w = 0; w < kCombWaves; ++w) zz += red[kMaxTopK + 1][w];
        bc[kMaxTopK + 1] = zz;
    }
    __syncthreads();
    const float zs = bc[kMaxTopK + 1];
    // the selected experts' dL/dp (every thread, k <= 16)
    float S = 0.f, dws = 0.f;
    for (int j = 0; j < k; ++j) {
        S += expf(l[idx[(size_t)t * k + j]] - mx) / zs;
        dws += bc[j] * wts[(size_t)t * k + j];
    }
    float dpp = 0.f;
    for (int j = 0; j < k; ++j) {
        const float pj = expf(l[idx[(size_t)t * k + j]] - mx) / zs;
        const float dp = norm_topk ? (bc[j] - dws) / S : bc[j];
        dpp += dp * pj;
    }
    for (int e = tid; e < E; e += kCombThreads) {
        float dpe = 0.f;
        for (int j = 0; j < k; ++j)
            if (idx[(size_t)t * k + j] == e) dpe = norm_topk ? (bc[j] - dws) / S : bc[j];
        const float pe = expf(l[e] - mx) / zs;
        dlogits[(size_t)t * E + e] = pe * (dpe - dpp);
    }
}

// dmask[e][c] = the sum of the dgrad tiles' partial sums over e's row tiles
// and both M-waves of each, in that order.
__global__ __launch_bounds__(256) void dmask_reduce_kernel(const float* __restrict__ dmp,
                                                           const SegMeta* __restrict__ seg, int hs, int I,
                                                           float* __restrict__ dmask) {
    const int e = blockIdx.y, c = blockIdx.x * 256 + threadIdx.x;
    if (c >= I) return;
    const SegMeta sm = seg[hs + e];
    const int mt = ceil_div(sm.rows, kTrainTile);
    float s = 0.f;
    for (int R = sm.rt0; R < sm.rt0 + mt; ++R)
        for (int w = 0; w < kTrainWaveM; ++w) s += dmp[((size_t)R * kTrainWaveM + w) * I + c];
    dmask[(size_t)e * I + c] = s;
}

// One wave per expert: Eqs. 6-8.
//   dz_k = sum_{c < width_k} dmask[e][c]
//   z = softmax((alpha + g) / tau), dalpha_quality = z (dz - <z, dz>) / tau
//   p = softmax(alpha), rbar = <p, r>, H_e = -<p, log p>, q = counts / (T k)
//   dalpha = dalpha_quality + lambda q p (r - rbar) + beta p (log p + H_e) / E
// per_expert[e] = (q rbar, H_e), summed by action_stats_kernel.
__global__ __launch_bounds__(64) void action_grad_kernel(ActionWidths aw, const float* __restrict__ alpha,
                                                         const float* __restrict__ gumbel, float tau,
                                                         const float* __restrict__ dmask,
                                                         const int32_t* __restrict__ counts, float inv_assign,
                                                         int E, int I, float lambda_cost, float beta,
                                                         float* __restrict__ dalpha, float* __restrict__ per_expert) {
    const int e = blockIdx.x, lane = threadIdx.x;
    const int K = aw.K;
    int wmax = 0;
    for (int k = 0; k < K; ++k) wmax = max(wmax, aw.width[k]);
    float dz[kMaxActions];
#pragma unroll
    for (int k = 0; k < kMaxActions; ++k) dz[k] = 0.f;
#pragma unroll 8
    for (int c = lane; c < wmax; c += 64) {
        const float v = dmask[(size_t)e * I + c];
#pragma unroll
        for (int k = 0; k < kMaxActions; ++k)
            if (k < K && c < aw.width[k]) dz[k] += v;
    }
#pragma unroll
    for (int k = 0; k < kMaxActions; ++k)
        if (k < K) dz[k] = wave_sum_f(dz[k]);
    const float* a = alpha + (size_t)e * K;
    const float* g = gumbel + (size_t)e * K;
    float sm = -INFINITY, am = -INFINITY;
    for (int k = 0; k < K; ++k) {
        sm = fmaxf(sm, (a[k] + g[k]) / tau);
        am = fmaxf(am, a[k]);
    }
    float zsum = 0.f, psum = 0.f;
    for (int k = 0; k < K; ++k) {
        zsum += expf((a[k] + g[k]) / tau - sm);
        psum += expf(a[k] - am);
    }
    float zdz = 0.f, rbar = 0.f, H = 0.f;
#pragma unroll
    for (int k = 0; k < kMaxActions; ++k) {
        if (k >= K) break;
        const float z = expf((a[k] + g[k]) / tau - sm) / zsum;
        const float p = expf(a[k] - am) / psum;
        zdz += z * dz[k];
        rbar += p * aw.ratio[k];
        H -= p > 0.f ? p * logf(p) : 0.f;
    }
    const float q = (float)counts[e] * inv_assign;
#pragma unroll
    for (int k = 0; k < kMaxActions; ++k) {
        if (k >= K) break;
        if (lane == k) {
            const float z = expf((a[k] + g[k]) / tau - sm) / zsum;
            const float p = expf(a[k] - am) / psum;
            const float gq = z * (dz[k] - zdz) / tau;
            const float gc = q * p * (aw.ratio[k] - rbar);
            const float ge = p > 0.f ? p * (logf(p) + H) / (float)E : 0.f;
            dalpha[(size_t)e * K + k] = gq + lambda_cost * gc + beta * ge;
        }
    }
    if (lane == 0) {
        per_expert[2 * e] = q * rbar;
        per_expert[2 * e + 1] = H;
    }
}

// stats = (C = sum_e q rbar, H = mean_e H_e), summed in expert order.
__global__ void action_stats_kernel(const float* __restrict__ per_expert, int E, float* __restrict__ stats) {
    if (threadIdx.x != 0) return;
    float C = 0.f, H = 0.f;
    for (int e = 0; e < E; ++e) {
        C += per_expert[2 * e];
        H += per_expert[2 * e + 1];
    }
    stats[0] = C;
    stats[1] = H / (float)E;
}

hipError_t launch_sample_actions(const ActionWidths& aw, const float* alpha, const float* gumbel, int E,
                                 int32_t* keep, int32_t* action, hipStream_t s) {
    sample_actions_kernel<<<ceil_div(E, 256), 256, 0, s>>>(aw, alpha, gumbel, E, keep, action);
    return hipGetLastError();
}

hipError_t launch_seg_use_kept(SegMeta* seg, int nseg, hipStream_t s) {
    seg_use_kept_kernel<<<ceil_div(nseg, 256), 256, 0, s>>>(seg, nseg);
    return hipGetLastError();
}

hipError_t launch_train_prep(const float* dy, const int32_t* perm, const float* wts, const int32_t* nrouted,
                             int A, int T, int d, int k, bf16_t* dO, bf16_t* dYs, hipStream_t s) {
    const int rows = A + (dYs ? T : 0);
    if (rows <= 0) return hipSuccess;
    const dim3 grid(rows, ceil_div(d, 8 * 256));
    train_prep_kernel<<<grid, 256, 0, s>>>(dy, perm, wts, nrouted, A, T, d, k, dO, dYs);
    return hipGetLastError();
}

hipError_t launch_combine_backward(const float* dXr, const float* dXs, const bf16_t* O, const int32_t* pos,
                                   const int32_t* idx, const float* wts, const float* logits, const float* dy,
                                   int T, int E, int k, int d, int norm_topk, float* dx, float* dlogits,
                                   hipStream_t s) {
    if (T <= 0) return hipSuccess;
    combine_backward_kernel<<<T, kCombThreads, 0, s>>>(dXr, dXs, O, pos, idx, wts, logits, dy, E, k, d,
                                                       norm_topk, dx, dlogits);
    return hipGetLastError();
}

hipError_t launch_dmask_reduce(const float* dmp, const SegMeta* seg, int hs, int E, int I, float* dmask,
                               hipStream_t s) {
    const dim3 grid(ceil_div(I, 256), E);
    dmask_reduce_kernel<<<grid, 256, 0, s>>>(dmp, seg, hs, I, dmask);
    return hipGetLastError();
}

hipError_t launch_action_grad(const ActionWidths& aw, const float* alpha, const float* gumbel, float tau,
                              const float* dmask, const int32_t* counts, long long assignments, int E, int I,
                              float lambda_cost, float beta, float* dalpha, float* per_expert, float* stats,
                              hipStream_t s) {
    action_grad_kernel<<<E, 64, 0, s>>>(aw, alpha, gumbel, tau, dmask, counts, 1.0f / (float)assignments, E, I,
                                        lambda_cost, beta, dalpha, per_expert);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess || !stats) return err;
    action_stats_kernel<<<1, 64, 0, s>>>(per_expert, E, stats);
    return hipGetLastError();
}

}  // namespace flexmoe
