// Offline clipping (FlexMoE Sec. 4.4, Table 2): the subnetwork of one budget
// exported as a standalone set of compact weights, which the same GEMM
// kernels read through the clipped layout of RoutedWeights (kernels.h).
//
// Expert e keeps its first k_e ranked channels, padded to kp_e =
// packed_width(k_e) (a multiple of 8, so every packed row is 16-byte
// aligned):
//   gate/up  [kp_e][d]  rows c < k_e copied from the ranked rows, the rest 0
//   down     [d][kp_e]  columns c < k_e copied from the ranked columns, the rest 0
// and the experts' blocks follow one another in expert order, expert e
// starting at packed channel ch0_e = sum_{e' < e} kp_e' (element ch0_e * d of
// every packed matrix).  The padding is never multiplied into a result: the
// gate/up GEMM computes channels below k_e only, and the down GEMM's zero H
// columns meet the zero padding.
#include "kernels.h"

namespace flexmoe {

namespace {
struct ExportArgs {
    KeepArgs keep;  // k_e
    KeepArgs ch0;   // first packed channel of each expert
};

// One expert (blockIdx.y), a grid-stride walk over its packed blocks in
// 16-byte chunks (VEC elements): first the gate and up blocks, then down.
template <typename T>
__global__ __launch_bounds__(256) void export_clipped_kernel(ExportArgs a, const T* __restrict__ wg_r,
                                                             const T* __restrict__ wu_r,
                                                             const T* __restrict__ wd_r, T* __restrict__ wg_c,
                                                             T* __restrict__ wu_c, T* __restrict__ wd_c, int I,
                                                             int d) {
    constexpr int VEC = 16 / sizeof(T);
    const int e = blockIdx.y;
    const int k = a.keep.v[e], kp = packed_width(k);
    const size_t src = (size_t)e * I * d;                // ranked blocks of expert e
    const size_t dst = (size_t)a.ch0.v[e] * d;           // packed blocks of expert e
    const size_t n_chunks = (size_t)kp * d / VEC;        // per packed matrix
    const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_chunks;
         i += (size_t)gridDim.x * blockDim.x) {
        const size_t el = i * VEC;
        // gate/up: packed row el / d is ranked row el / d (d % 8 == 0: a chunk
        // never straddles rows)
        const bool keep_row = el / d < (size_t)k;
        const uint4 g = keep_row ? *reinterpret_cast<const uint4*>(wg_r + src + el) : zero;
        const uint4 u = keep_row ? *reinterpret_cast<const uint4*>(wu_r + src + el) : zero;
        *reinterpret_cast<uint4*>(wg_c + dst + el) = g;
        *reinterpret_cast<uint4*>(wu_c + dst + el) = u;
        // down: packed element (n, c) = ranked (n, c) for c < k, else 0
        const size_t n = el / kp;
        const int c = (int)(el % kp);
        T v[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) v[j] = c + j < k ? wd_r[src + n * I + c + j] : T(0);
        *reinterpret_cast<uint4*>(wd_c + dst + el) = *reinterpret_cast<const uint4*>(v);
    }
}
}  // namespace

hipError_t launch_export_clipped(const KeepArgs& keep, const void* wg_r, const void* wu_r,
                                 const void* wd_r, void* wg_c, void* wu_c, void* wd_c, int E, int I,
                                 int d, int esize, hipStream_t s) {
    ExportArgs a;
    a.keep = keep;
    int c = 0;
    for (int e = 0; e < kMaxExperts; ++e) {
        a.ch0.v[e] = c;
        if (e < E) c += packed_width(keep.v[e]);
    }
    // enough workgroups per expert to stream its blocks; each loops over the rest
    const dim3 grid(64, E);
    if (esize == 2)
        export_clipped_kernel<bf16_t><<<grid, 256, 0, s>>>(a, (const bf16_t*)wg_r, (const bf16_t*)wu_r,
                                                           (const bf16_t*)wd_r, (bf16_t*)wg_c, (bf16_t*)wu_c,
                                                           (bf16_t*)wd_c, I, d);
    else
        export_clipped_kernel<float><<<grid, 256, 0, s>>>(a, (const float*)wg_r, (const float*)wu_r,
                                                          (const float*)wd_r, (float*)wg_c, (float*)wu_c,
                                                          (float*)wd_c, I, d);
    return hipGetLastError();
}

}  // namespace flexmoe
