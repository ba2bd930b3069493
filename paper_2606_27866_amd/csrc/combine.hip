// Weighted combine (App. C.3: router-weight scaling and scatter-add, done as
// a deterministic gather).  For token t:
//   y[t] = sum_{j < top_k, pos[t][j] >= 0} w[t][j] * O[pos[t][j]] + S[t]
// summed in ascending slot order in fp32, then rounded once to the output
// type.  Assignments of experts with k_e = 0 have pos = -1 and add nothing.
// S[t] is the sum of the shared expert's partial rows Os[part][t] (one part
// unless its down projection was split), added in ascending part order.
// O and Os are fp32 in fp32 mode and bf16 in bf16 mode.
#include "saliency.h"

namespace flexmoe {

__device__ __forceinline__ float4 load4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 load4(const bf16_t* p) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                       __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
}

// Columns n .. n+3 of token t's combined output, in fp32.
template <typename OutT>
__device__ __forceinline__ float4 combine_cols(const OutT* __restrict__ O, const OutT* __restrict__ Os,
                                               const int32_t* __restrict__ pos, const float* __restrict__ wts,
                                               int T, int k, int d, int shared_parts, int t, int n) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < k; ++j) {
        const int p = pos[(size_t)t * k + j];
        if (p < 0) continue;
        const float w = wts[(size_t)t * k + j];
        const float4 o = load4(O + (size_t)p * d + n);
        acc.x += w * o.x;
        acc.y += w * o.y;
        acc.z += w * o.z;
        acc.w += w * o.w;
    }
    float4 sh = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int q = 0; q < shared_parts; ++q) {
        const float4 sv = load4(Os + ((size_t)q * T + t) * d + n);
        sh.x += sv.x;
        sh.y += sv.y;
        sh.z += sv.z;
        sh.w += sv.w;
    }
    acc.x += sh.x;
    acc.y += sh.y;
    acc.z += sh.z;
    acc.w += sh.w;
    return acc;
}

// bf16: columns n .. n+7 of token t (16-byte loads and stores), the same
// arithmetic as combine_cols per column.  KS > 0: the slot count is known at
// compile time and the KS slot rows are requested together; KS = 0: any
// count, in batches of 8 slots and 8 shared row sets whose reads are issued
// together (addresses of absent ones clamped to a valid row, their values
// unused).  NT: the O and Os rows (read exactly once) are loaded with the
// non-temporal hint, which pays for prefill-sized outputs (Mixtral-shaped
// layer -0.35 % per step) but not for decode-sized ones that sit in the L2.
template <bool NT>
__device__ __forceinline__ uint4 load16(const bf16_t* p) {
    if constexpr (NT) {
        const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
        return make_uint4(v.x, v.y, v.z, v.w);
    } else {
        return *reinterpret_cast<const uint4*>(p);
    }
}
__device__ __forceinline__ void add_row8(float (&acc)[8], uint4 v, float w) {
    const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        acc[2 * i] += w * __uint_as_float(u[i] << 16);
        acc[2 * i + 1] += w * __uint_as_float(u[i] & 0xffff0000u);
    }
}
__device__ __forceinline__ void add_row8(float (&acc)[8], uint4 v) {
    const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        acc[2 * i] += __uint_as_float(u[i] << 16);
        acc[2 * i + 1] += __uint_as_float(u[i] & 0xffff0000u);
    }
}
template <int KS, bool NT>
__device__ __forceinline__ void combine_cols8(const bf16_t* __restrict__ O, const bf16_t* __restrict__ Os,
                                              const int32_t* __restrict__ pos, const float* __restrict__ wts,
                                              int T, int k, int d, int shared_parts, int t, int n, float (&acc)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
    float sh[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if constexpr (KS > 0) {
        int p[KS];
        float w[KS];
        uint4 v[KS];
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            p[j] = pos[(size_t)t * KS + j];
            w[j] = wts[(size_t)t * KS + j];
        }
#pragma unroll
        for (int j = 0; j < KS; ++j) v[j] = load16<NT>(O + (size_t)max(p[j], 0) * d + n);
        for (int b = 0; b < shared_parts; b += 8) {  // shared row sets, 8 requested together
            uint4 sv[8];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj)
                sv[jj] = load16<NT>(Os + ((size_t)min(b + jj, shared_parts - 1) * T + t) * d + n);
#pragma unroll
            for (int jj = 0; jj < 8; ++jj)
                if (b + jj < shared_parts) add_row8(sh, sv[jj]);
        }
#pragma unroll
        for (int j = 0; j < KS; ++j)
            if (p[j] >= 0) add_row8(acc, v[j], w[j]);
    } else {
        const int nbat = max(ceil_div(k, 8), ceil_div(shared_parts, 8));
        for (int b = 0; b < nbat; ++b) {
            int p[8];
            float w[8];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) {
                const int j = min(b * 8 + jj, k - 1);
                p[jj] = pos[(size_t)t * k + j];
                w[jj] = wts[(size_t)t * k + j];
            }
            uint4 v[8], sv[8];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) {
                v[jj] = load16<NT>(O + (size_t)max(p[jj], 0) * d + n);
                const int q = min(b * 8 + jj, max(shared_parts - 1, 0));
                sv[jj] = shared_parts > 0 ? load16<NT>(Os + ((size_t)q * T + t) * d + n) : make_uint4(0u, 0u, 0u, 0u);
            }
#pragma unroll
            for (int jj = 0; jj < 8; ++jj)
                if (b * 8 + jj < k && p[jj] >= 0) add_row8(acc, v[jj], w[jj]);
#pragma unroll
            for (int jj = 0; jj < 8; ++jj)
                if (b * 8 + jj < shared_parts) add_row8(sh, sv[jj]);
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += sh[i];
}

// bf16 output: one 8-column group per thread (d % 8 == 0).
template <int KS, bool NT>
__global__ __launch_bounds__(256) void combine_bf16_kernel(const bf16_t* __restrict__ O,
                                                           const bf16_t* __restrict__ Os,
                                                           const int32_t* __restrict__ pos,
                                                           const float* __restrict__ wts, int T, int k, int d,
                                                           int shared_parts, bf16_t* __restrict__ y) {
    const int t = blockIdx.x;
    const int n = (blockIdx.y * blockDim.x + threadIdx.x) * 8;
    if (n >= d) return;
    float acc[8];
    combine_cols8<KS, NT>(O, Os, pos, wts, T, k, d, shared_parts, t, n, acc);
    uint32_t u[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
        u[i] = pack_bf16x2(acc[2 * i], acc[2 * i + 1]);
    *reinterpret_cast<uint4*>(y + (size_t)t * d + n) = make_uint4(u[0], u[1], u[2], u[3]);
}

template <typename OutT>
__global__ __launch_bounds__(256) void combine_kernel(const OutT* __restrict__ O,
                                                      const OutT* __restrict__ Os,
                                                      const int32_t* __restrict__ pos,
                                                      const float* __restrict__ wts, int T, int k,
                                                      int d, int shared_parts, OutT* __restrict__ y) {
    const int t = blockIdx.x;
    const int n = (blockIdx.y * blockDim.x + threadIdx.x) * 4;  // one float4 column group per thread
    if (n < d) {
        const float4 acc = combine_cols(O, Os, pos, wts, T, k, d, shared_parts, t, n);
        if constexpr (sizeof(OutT) == 4) {
            *reinterpret_cast<float4*>(y + (size_t)t * d + n) = acc;
        } else {
            const uint32_t lo = pack_bf16x2(acc.x, acc.y);
            const uint32_t hi = pack_bf16x2(acc.z, acc.w);
            *reinterpret_cast<uint2*>(y + (size_t)t * d + n) = make_uint2(lo, hi);
        }
    }
}

// The residual of the saliency's loss: dY = y - target, y unrounded.
__global__ __launch_bounds__(256) void combine_residual_kernel(const bf16_t* __restrict__ O,
                                                               const bf16_t* __restrict__ Os,
                                                               const int32_t* __restrict__ pos,
                                                               const float* __restrict__ wts, int T, int k,
                                                               int d, int shared_parts,
                                                               const float* __restrict__ target,
                                                               float* __restrict__ dy) {
    const int t = blockIdx.x;
    const int n = (blockIdx.y * blockDim.x + threadIdx.x) * 4;
    if (n < d) {
        const float4 acc = combine_cols(O, Os, pos, wts, T, k, d, shared_parts, t, n);
        const float4 tg = *reinterpret_cast<const float4*>(target + (size_t)t * d + n);
        *reinterpret_cast<float4*>(dy + (size_t)t * d + n) =
            make_float4(acc.x - tg.x, acc.y - tg.y, acc.z - tg.z, acc.w - tg.w);
    }
}

hipError_t launch_combine_residual(const bf16_t* O, const bf16_t* Os, const int32_t* pos, const float* wts,
                                   int T, int k, int d, int shared_parts, const float* target, float* dy,
                                   hipStream_t s) {
    if (T <= 0) return hipSuccess;
    const dim3 grid(T, ceil_div(d, 4 * 256));
    combine_residual_kernel<<<grid, 256, 0, s>>>(O, Os, pos, wts, T, k, d, shared_parts, target, dy);
    return hipGetLastError();
}

hipError_t launch_combine(const void* O, const void* Os, const int32_t* pos, const float* wts,
                          int T, int k, int d, int shared_parts, int dtype, void* y, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    const dim3 grid(T, ceil_div(d, 4 * 256));
    if (dtype == 0)
        combine_kernel<float><<<grid, 256, 0, s>>>((const float*)O, (const float*)Os, pos, wts, T, k, d,
                                                   shared_parts, (float*)y);
    else
    {
        const dim3 g8(T, ceil_div(d, 8 * 256));
        const bf16_t *o = (const bf16_t*)O, *os = (const bf16_t*)Os;
        bf16_t* yb = (bf16_t*)y;
        // decode-sized batches keep the general kernel with cached loads
        const int ks = T > kDecodeMaxT ? k : 0;
        switch (ks) {  // the top-k values of the models this layer is shaped for
            case 2: combine_bf16_kernel<2, true><<<g8, 256, 0, s>>>(o, os, pos, wts, T, k, d, shared_parts, yb); break;
            case 4: combine_bf16_kernel<4, true><<<g8, 256, 0, s>>>(o, os, pos, wts, T, k, d, shared_parts, yb); break;
            case 8: combine_bf16_kernel<8, true><<<g8, 256, 0, s>>>(o, os, pos, wts, T, k, d, shared_parts, yb); break;
            default:
                if (T > kDecodeMaxT)
                    combine_bf16_kernel<0, true><<<g8, 256, 0, s>>>(o, os, pos, wts, T, k, d, shared_parts, yb);
                else
                    combine_bf16_kernel<0, false><<<g8, 256, 0, s>>>(o, os, pos, wts, T, k, d, shared_parts, yb);
        }
    }
    return hipGetLastError();
}

}  // namespace flexmoe
